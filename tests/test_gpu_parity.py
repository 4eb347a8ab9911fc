"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

- transformation: bit-exact against the oracle's Alg. 1 copy, on every
  workload at full size and on edge shapes, with a poisoned workspace (every
  element must be written) and a guard band after it (nothing else may be);
- convolution and fused convolution: element by element within the fp32
  rounding bound (n + 2) * 2^-24 * sum|x*w| (n = C*Fh*Fw terms), and relative
  L2 error <= 1e-5 (fp32) / 1e-2 (bf16), against the fp64 direct convolution
  of the same (bf16-rounded) data: on the whole output at reduced batch and on
  sampled outputs at full size;
- fused and unfused stage identical window strips and run the same matrix-core
  sequence, so their outputs must be bitwise identical.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import Shape
import workloads
import paper_2306_14320_amd as P

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
U32 = 2.0 ** -24
RELL2 = {"f32": 1e-5, "bf16": 1e-2}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    P.load_library()
    yield
    torch.cuda.synchronize()


def _shape(wl):
    return Shape(wl.n, wl.c, wl.h, wl.w, wl.k, wl.fh, wl.fw, wl.sh, wl.sw, wl.ph, wl.pw)


def _desc(wl, n=None):
    return P.im2win_desc(n or wl.n, wl.c, wl.h, wl.w, wl.k, wl.fh, wl.fw, wl.sh, wl.sw, wl.ph,
                         wl.pw, P.IM2WIN_F32 if wl.dtype == "f32" else P.IM2WIN_BF16)


def _bits(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    return (t.view(torch.int32) if t.element_size() == 4 else t.view(torch.int16)).numpy()


def _poisoned(numel, dtype, guard=4096):
    """Device buffer of numel + guard elements, all set to an all-ones NaN pattern."""
    buf = torch.empty(numel + guard, dtype=dtype, device=DEV)
    (buf.view(torch.int32) if buf.element_size() == 4 else buf.view(torch.int16)).fill_(-1)
    return buf


def _label(tag, wl, n=None):
    print(f"[parity] {tag} {wl.label()} n={n or wl.n}", flush=True)


# --------------------------------------------------------------------------
# transformation
# --------------------------------------------------------------------------

def _check_transform(wl, x_cpu, n):
    s = _shape(wl)
    s = Shape(n, s.c, s.h, s.w, s.k, s.fh, s.fw, s.sh, s.sw, s.ph, s.pw)
    d = _desc(wl, n)
    nbytes = P.im2win_workspace_bytes(d)
    numel = nbytes // x_cpu.element_size()
    buf = _poisoned(numel, x_cpu.dtype)
    x = x_cpu.to(DEV)
    P.transform(x, d, ws=buf[:numel].view(s.win_shape))
    torch.cuda.synchronize()
    got = _bits(buf)
    ref = oracle.im2win(s, _bits(x_cpu))
    assert np.array_equal(got[:numel], ref.reshape(-1)), "window tensor differs from the oracle"
    assert np.all(got[numel:] == -1), "transformation wrote past the window tensor"


@pytest.mark.parametrize("wl", workloads.WORKLOADS, ids=lambda wl: wl.name)
def test_transform_bit_exact_full_size(wl):
    _label("transform", wl)
    _check_transform(wl, workloads.make_input(wl), wl.n)


# --------------------------------------------------------------------------
# convolution
# --------------------------------------------------------------------------

def _f64(t):
    return t.detach().to(torch.float64).cpu().numpy()


def _run_conv(wl, x_cpu, w_cpu, n, fused):
    d = _desc(wl, n)
    x, w = x_cpu.to(DEV), w_cpu.to(DEV)
    ho, wo = P.im2win_output_shape(d)
    ybuf = torch.full((n * wl.k * ho * wo + 4096,), float("nan"), dtype=torch.float32, device=DEV)
    y = ybuf[:n * wl.k * ho * wo].view(n, wl.k, ho, wo)
    if fused:
        P.conv2d_fused(x, w, d, y=y)
    else:
        ws = P.transform(x, d)
        P.conv2d(ws, w, d, y=y)
    torch.cuda.synchronize()
    assert torch.isnan(ybuf[y.numel():]).all(), "convolution wrote past the output"
    return y.cpu().numpy().astype(np.float64)


def _assert_close(got, ref, ref_abs, nterms, dtype, what):
    bound = (nterms + 2) * U32 * ref_abs + 1e-30
    err = np.abs(got - ref)
    worst = np.argmax(err - bound)
    assert np.all(err <= bound), (f"{what}: {np.sum(err > bound)} outputs outside the fp32 "
                                  f"rounding bound; worst at {worst}: got {got.flat[worst]}, "
                                  f"ref {ref.flat[worst]}, bound {bound.flat[worst]}")
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)
    assert rel <= RELL2[dtype], f"{what}: relative L2 error {rel:.3e}"
    return rel


REDUCED_N = {"single_3x3_f32": 1, "resnet_3x3_f32": 2, "stem_7x7_s2_f32": 2,
             "deep_3x3_bf16": 2, "rect_3x5_s2_f32": 3}


@pytest.mark.parametrize("fused", [False, True], ids=["unfused", "fused"])
@pytest.mark.parametrize("wl", workloads.WORKLOADS, ids=lambda wl: wl.name)
def test_conv_whole_output_reduced_batch(wl, fused):
    n = REDUCED_N[wl.name]
    _label("conv-fused" if fused else "conv", wl, n)
    x_cpu = workloads.make_input(wl, n_images=n)
    w_cpu = workloads.make_filter(wl)
    got = _run_conv(wl, x_cpu, w_cpu, n, fused)
    s = _shape(wl)
    s = Shape(n, s.c, s.h, s.w, s.k, s.fh, s.fw, s.sh, s.sw, s.ph, s.pw)
    ref, ref_abs = oracle.direct_conv(s, _f64(x_cpu), _f64(w_cpu), with_abs=True)
    rel = _assert_close(got, ref, ref_abs, wl.c * wl.fh * wl.fw, wl.dtype, wl.name)
    print(f"[parity] rel-L2 {rel:.3e}", flush=True)


def _sample_indices(n, k, ho, wo, count, seed):
    rng = np.random.default_rng(seed)
    total = n * k * ho * wo
    idx = [rng.integers(0, total, size=count)]
    # borders of the first and last image for the first and last channel
    for i in (0, n - 1):
        for j in (0, k - 1):
            base = (i * k + j) * ho * wo
            rows = np.arange(ho)
            cols = np.arange(wo)
            idx += [base + cols, base + (ho - 1) * wo + cols, base + rows * wo, base + rows * wo + wo - 1]
    idx.append(np.array([0, total - 1]))
    return np.unique(np.concatenate(idx))


@pytest.mark.parametrize("wl", workloads.WORKLOADS, ids=lambda wl: wl.name)
def test_conv_full_size_sampled_and_fused_identical(wl):
    _label("conv-full", wl)
    x_cpu, w_cpu = workloads.make_input(wl), workloads.make_filter(wl)
    y_unf = _run_conv(wl, x_cpu, w_cpu, wl.n, False)
    y_fus = _run_conv(wl, x_cpu, w_cpu, wl.n, True)
    assert np.array_equal(y_unf, y_fus), "fused and unfused outputs differ"
    s = _shape(wl)
    idx = _sample_indices(wl.n, wl.k, s.ho, s.wo, 4000, 7)
    ref, ref_abs = oracle.direct_conv_at(s, _f64(x_cpu), _f64(w_cpu), idx)
    rel = _assert_close(y_unf.reshape(-1)[idx], ref, ref_abs, wl.c * wl.fh * wl.fw, wl.dtype,
                        wl.name + " (sampled)")
    print(f"[parity] sampled rel-L2 {rel:.3e} over {idx.size} outputs", flush=True)


# --------------------------------------------------------------------------
# edge shapes
# --------------------------------------------------------------------------

EDGE = [
    # (n, c, h, w, k, fh, fw, sh, sw, ph, pw)
    (1, 1, 4, 4, 2, 2, 2, 1, 1, 0, 0),        # the paper's worked example (Fig. 2 geometry)
    (2, 3, 9, 11, 5, 3, 5, 2, 2, 1, 2),       # rectangular, stride 2
    (1, 5, 10, 8, 7, 5, 3, 2, 1, 2, 0),       # tall rectangular, mixed strides
    (2, 17, 13, 13, 33, 3, 3, 1, 1, 1, 1),    # channels not a multiple of the chunk, K ragged
    (1, 2, 9, 9, 3, 2, 2, 3, 3, 0, 0),        # Fh < sh, Fw < sw
    (1, 3, 6, 6, 130, 1, 1, 1, 1, 0, 0),      # 1x1 filter, K above one tile
    (1, 4, 5, 6, 3, 5, 6, 1, 1, 0, 0),        # filter covers the input: Ho = Wo = 1
    (3, 2, 3, 3, 2, 3, 3, 1, 1, 2, 2),        # padding wider than the input
    (2, 1, 1, 17, 4, 1, 3, 1, 2, 0, 1),       # H = 1
    (5, 2, 2, 2, 1, 2, 2, 1, 1, 0, 0),        # one output pixel per image, many images
    (1, 33, 30, 70, 65, 7, 7, 2, 2, 3, 3),    # stem-like with ragged pixel and channel tiles
    (2, 40, 7, 7, 300, 3, 3, 1, 1, 1, 1),     # deep-narrow, 3 channel tiles
    (1, 3, 227, 227, 96, 11, 11, 4, 4, 0, 0), # Table 1 Conv1 at batch 1
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", EDGE, ids=lambda c: "x".join(map(str, c)))
def test_edge_shapes(case, dtype):
    n, c, h, w, k, fh, fw, sh, sw, ph, pw = case
    wl, x_cpu, w_cpu = workloads.random_case(sum(case), n, c, h, w, k, fh, fw, sh, sw, ph, pw, dtype)
    _label("edge", wl)
    assert P.im2win_check_plan(_desc(wl)) == 0, P.im2win_last_error()
    _check_transform(wl, x_cpu, n)
    s = _shape(wl)
    ref, ref_abs = oracle.direct_conv(s, _f64(x_cpu), _f64(w_cpu), with_abs=True)
    y_unf = _run_conv(wl, x_cpu, w_cpu, n, False)
    y_fus = _run_conv(wl, x_cpu, w_cpu, n, True)
    _assert_close(y_unf, ref, ref_abs, c * fh * fw, dtype, "unfused")
    assert np.array_equal(y_unf, y_fus), "fused and unfused outputs differ"


def test_non_default_stream_and_reuse():
    """Calls are ordered on the caller's stream; a second, smaller problem on
    the same buffers gives its own correct result."""
    wl = workloads.BY_NAME["rect_3x5_s2_f32"]
    side = torch.cuda.Stream(device=DEV)
    for n in (3, 1):
        x_cpu = workloads.make_input(wl, n_images=n)
        w_cpu = workloads.make_filter(wl)
        d = _desc(wl, n)
        with torch.cuda.stream(side):
            x, w = x_cpu.to(DEV), w_cpu.to(DEV)
            ws = P.transform(x, d, stream=side)
            y = P.conv2d(ws, w, d, stream=side)
        side.synchronize()
        s = Shape(n, wl.c, wl.h, wl.w, wl.k, wl.fh, wl.fw, wl.sh, wl.sw, wl.ph, wl.pw)
        ref, ref_abs = oracle.direct_conv(s, _f64(x_cpu), _f64(w_cpu), with_abs=True)
        _assert_close(y.cpu().numpy().astype(np.float64), ref, ref_abs, wl.c * 15, "f32", "side stream")


def test_bf16_error_against_unrounded_data():
    """Information on top of parity: against the fp32 (not bf16-rounded) data
    the bf16 path is off by the input rounding, about 2^-8/sqrt(6) per operand."""
    wl = workloads.BY_NAME["deep_3x3_bf16"]
    n = 1
    from dataclasses import replace
    wl32 = replace(wl, dtype="f32")
    x32, w32 = workloads.make_input(wl32, n_images=n), workloads.make_filter(wl32)
    got = _run_conv(wl, x32.to(torch.bfloat16), w32.to(torch.bfloat16), n, True)
    s = Shape(n, wl.c, wl.h, wl.w, wl.k, wl.fh, wl.fw, wl.sh, wl.sw, wl.ph, wl.pw)
    ref = oracle.direct_conv(s, _f64(x32), _f64(w32))
    rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    print(f"[parity] bf16 vs unrounded fp32 data: rel-L2 {rel:.3e}", flush=True)
    assert rel < 1e-2


def test_repacked_filters_share_the_stream_buffer():
    """fp32 filters whose chunk rows are not whole 16-byte vectors (7x7, 5x5,
    11x11) are repacked per call into the same per-stream buffer as the bf16
    fast kernels' filters: fp32 and bf16 convolutions interleaved on two
    streams, with a larger filter replacing a stream's buffer in the middle,
    each result against the oracle."""
    cases = [
        (1, "f32", (2, 3, 30, 30, 64, 7, 7, 2, 2, 3, 3)),
        (2, "bf16", (2, 32, 14, 14, 64, 3, 3, 1, 1, 1, 1)),
        (1, "f32", (1, 6, 24, 24, 96, 5, 5, 1, 1, 0, 0)),
        (2, "f32", (1, 3, 47, 47, 96, 11, 11, 4, 4, 0, 0)),
        (1, "bf16", (1, 64, 10, 12, 128, 3, 3, 1, 1, 1, 1)),
        (2, "f32", (2, 3, 30, 30, 64, 7, 7, 2, 2, 3, 3)),
    ]
    streams = {1: torch.cuda.Stream(device=DEV), 2: torch.cuda.Stream(device=DEV)}
    runs = []
    for i, (sid, dtype, shape) in enumerate(cases):
        wl, x_cpu, w_cpu = workloads.random_case(800 + i, *shape, dtype=dtype)
        _label("repacked-filter stream", wl)
        d = _desc(wl)
        assert P.im2win_check_plan(d) == 0, P.im2win_last_error()
        stream = streams[sid]
        with torch.cuda.stream(stream):
            x, w = x_cpu.to(DEV), w_cpu.to(DEV)
            y_fused = P.conv2d_fused(x, w, d, stream=stream)
            y = P.conv2d(P.transform(x, d, stream=stream), w, d, stream=stream)
        runs.append((wl, x_cpu, w_cpu, y, y_fused))
    torch.cuda.synchronize()
    for wl, x_cpu, w_cpu, y, y_fused in runs:
        ref, ref_abs = oracle.direct_conv(_shape(wl), _f64(x_cpu), _f64(w_cpu), with_abs=True)
        for what, out in (("unfused", y), ("fused", y_fused)):
            _assert_close(out.cpu().numpy().astype(np.float64), ref, ref_abs, wl.c * wl.fh * wl.fw, wl.dtype,
                          f"{wl.name} {what}")


def test_bf16_packed_filter_per_stream():
    """The bf16 fast kernels read a repacked filter that the library keeps per
    stream: two streams with different filters in flight at once, then a
    larger filter on the first stream (its buffer is replaced in stream
    order), each result against the oracle."""
    small = (2, 32, 14, 14, 64, 3, 3, 1, 1, 1, 1)
    large = (1, 64, 10, 12, 128, 3, 3, 1, 1, 1, 1)
    s1, s2 = torch.cuda.Stream(device=DEV), torch.cuda.Stream(device=DEV)
    runs = []
    for seed, shape, stream in ((1, small, s1), (2, small, s2), (3, large, s1), (4, small, s2)):
        wl, x_cpu, w_cpu = workloads.random_case(700 + seed, *shape, dtype="bf16")
        _label("packed-filter stream", wl)
        d = _desc(wl)
        assert P.im2win_check_plan(d) == 0, P.im2win_last_error()
        with torch.cuda.stream(stream):
            x, w = x_cpu.to(DEV), w_cpu.to(DEV)
            y_fused = P.conv2d_fused(x, w, d, stream=stream)
            y = P.conv2d(P.transform(x, d, stream=stream), w, d, stream=stream)
        runs.append((wl, x_cpu, w_cpu, y, y_fused))
    torch.cuda.synchronize()
    for wl, x_cpu, w_cpu, y, y_fused in runs:
        ref, ref_abs = oracle.direct_conv(_shape(wl), _f64(x_cpu), _f64(w_cpu), with_abs=True)
        for what, out in (("unfused", y), ("fused", y_fused)):
            _assert_close(out.cpu().numpy().astype(np.float64), ref, ref_abs, wl.c * wl.fh * wl.fw, "bf16",
                          f"{wl.name} {what}")
