"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

- transformation: bit-exact against the oracle's Alg. 1 copy, on every
  workload at full size and on edge shapes, with a poisoned workspace (every
  element must be written) and a guard band after it (nothing else may be);
- convolution and fused convolution: element by element within the fp32
  rounding bound (n + 2) * 2^-24 * sum|x*w| (n = C*Fh*Fw terms), and relative
  L2 error <= 1e-5 (fp32) / 1e-2 (bf16), against the fp64 direct convolution
  of the same (bf16-rounded) data, on the whole output, at reduced batch and
  at full size;
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


@pytest.mark.parametrize("wl", workloads.WORKLOADS, ids=lambda wl: wl.name)
def test_conv_full_size_whole_output_and_fused_identical(wl):
    """Every output of both convolutions at full size, in the launch
    configuration bench.py times, against the fp64 oracle (Eq. 1)."""
    _label("conv-full", wl)
    x_cpu, w_cpu = workloads.make_input(wl), workloads.make_filter(wl)
    y_unf = _run_conv(wl, x_cpu, w_cpu, wl.n, False)
    y_fus = _run_conv(wl, x_cpu, w_cpu, wl.n, True)
    assert np.array_equal(y_unf, y_fus), "fused and unfused outputs differ"
    del y_fus
    ref, ref_abs = oracle.direct_conv(_shape(wl), _f64(x_cpu), _f64(w_cpu), with_abs=True)
    rel = _assert_close(y_unf, ref, ref_abs, wl.c * wl.fh * wl.fw, wl.dtype, wl.name + " (full size)")
    print(f"[parity] full-size rel-L2 {rel:.3e} over {y_unf.size} outputs", flush=True)


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
    (2, 32, 9, 11, 64, 3, 5, 2, 2, 1, 2),     # bf16 3x5 with 16-byte filter pieces (strips gathered)
    (2, 32, 10, 12, 64, 3, 5, 1, 2, 1, 2),    # bf16 3x5 fast and fused-fast kernels (rows of 48, W even)
    (2, 32, 14, 14, 128, 1, 1, 1, 1, 0, 0),   # 1x1 with 16-byte filter pieces
    (2, 32, 16, 16, 128, 1, 1, 1, 1, 0, 0),   # 1x1 fast and fused-fast kernels
    (3, 64, 16, 14, 128, 3, 3, 1, 1, 0, 1),   # bf16 one-image tiles: 196 pixels, pad (0, 1)
    (2, 32, 27, 14, 128, 3, 3, 2, 1, 1, 1),   # bf16 one-image tiles with row stride 2
    (4, 32, 14, 14, 256, 3, 3, 1, 1, 1, 1),   # bf16 one-image tiles, 2 K tiles, XCD placement
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


# Shapes that the fp32 band kernel takes (at least 85% of whole rounds of 256
# workgroups useful), each in both row layouts; the copy granularity (16-byte
# or 4-byte pieces of the strips) follows from the plane alignment.
F32_BANDS = [
    (2, 16, 28, 28, 4096, 3, 5, 2, 2, 1, 2),   # 3x5 stride 2, whole 14x14 images in 7 blocks
    (8, 32, 14, 14, 1024, 3, 3, 1, 1, 1, 1),   # 196 pixels, two chunk pairs, XCD placement
    (16, 16, 13, 13, 512, 3, 3, 1, 1, 0, 0),   # 121 pixels in 4 blocks
    (4, 16, 13, 23, 2048, 3, 5, 1, 2, 0, 1),   # 121 pixels, rows of 75 (4-byte copies)
    (3, 32, 29, 15, 2720, 3, 3, 2, 1, 1, 0),   # 195 pixels, row stride 2, grid not a multiple of 8
    (2, 16, 56, 56, 1024, 3, 3, 1, 1, 1, 1),   # two-way split: 7-row bands of 56 columns
    (8, 16, 28, 28, 1024, 3, 3, 1, 1, 0, 0),   # two-way split: two bands of 13 rows in 11 blocks
    (8, 16, 55, 55, 1024, 3, 3, 2, 2, 1, 1),   # two-way split, stride 2
    (8, 16, 52, 52, 1024, 3, 3, 2, 2, 1, 1),   # two-way split, stride 2, fused from raw rows
    (2, 16, 28, 32, 4096, 3, 5, 2, 2, 1, 4),   # raw rows with 8 zero columns in front (pw = 4)
    (128, 16, 7, 7, 512, 3, 3, 1, 1, 0, 0),    # bands of 8 whole images of 25 pixels (4-byte copies)
    (124, 16, 7, 7, 512, 3, 3, 1, 1, 0, 0),    # the same, the last band of 4 images
    (128, 16, 12, 12, 512, 3, 3, 1, 1, 0, 0),  # two-way split, bands of 4 images of 100 pixels (16-byte copies)
    (126, 16, 12, 12, 512, 3, 3, 1, 1, 0, 0),  # the same, the last band of 2 images
    (128, 16, 5, 5, 512, 3, 3, 1, 1, 1, 1),    # several padded images: the fused gather's zeros
    (128, 16, 7, 9, 512, 3, 5, 1, 1, 0, 0),    # several images, 3x5
    (128, 16, 14, 14, 256, 3, 3, 1, 1, 0, 0),  # two-way split, bands of 2 images of 144 pixels (9 blocks)
    (127, 16, 14, 14, 256, 3, 3, 1, 1, 0, 0),  # the same, the last band of 1 image
    (9, 16, 112, 112, 128, 3, 3, 1, 1, 0, 0),  # two-way split, 4-row bands of 110 pixels in 14 blocks
    (16, 16, 24, 24, 256, 5, 5, 1, 1, 0, 0),   # 5x5: bands of 11 and 9 rows of 20 pixels
    (16, 16, 20, 20, 256, 5, 5, 1, 1, 2, 2),   # 5x5 with padding 2: the raw rows' zero columns
]


# Shapes that the fp32 small-C band kernel takes (C = 3, 7x7).
F32_BANDS_SMALL_C = [
    (4, 3, 64, 64, 512, 7, 7, 2, 2, 3, 3),     # stem-like: stride 2, padding 3, bands of 7 rows
    (8, 3, 70, 70, 64, 7, 7, 1, 1, 0, 0),      # stride 1, 64 x 64 outputs
    (2, 3, 48, 48, 512, 7, 7, 1, 1, 0, 0),     # ragged last band
    (1, 3, 62, 62, 512, 3, 3, 1, 1, 1, 1),     # 3x3: the middle filter row in both k-slots
    (4, 3, 63, 63, 512, 3, 3, 2, 2, 0, 0),
    (16, 3, 59, 59, 512, 11, 11, 4, 4, 2, 2),  # 11x11 stride 4, input rows not whole 16-byte vectors
    (1, 3, 56, 56, 512, 11, 11, 1, 1, 5, 5),
    (4, 3, 64, 64, 96, 3, 3, 1, 1, 1, 1),      # K = 96: the last group's second block of channels idle
    (8, 3, 83, 83, 96, 7, 7, 2, 2, 3, 3),
    (32, 3, 53, 53, 224, 11, 11, 4, 4, 5, 5),
    (16, 3, 45, 45, 160, 7, 7, 2, 2, 3, 3),    # K = 160: three groups, the last half idle
]


@pytest.mark.parametrize("layout", [P.IM2WIN_ROWS_PADDED, P.IM2WIN_ROWS_TRIMMED], ids=["padded", "trimmed"])
@pytest.mark.parametrize("case", F32_BANDS + F32_BANDS_SMALL_C, ids=lambda c: "x".join(map(str, c)))
def test_fp32_band_kernel(case, layout):
    """Whole output of both convolutions against the fp64 oracle (Eq. 1),
    fused and unfused bitwise identical, nothing written past the output."""
    n, c, h, w, k, fh, fw, sh, sw, ph, pw = case
    wl, x_cpu, w_cpu = workloads.random_case(sum(case) + layout, n, c, h, w, k, fh, fw, sh, sw, ph, pw, "f32")
    _label(f"f32-bands layout={layout}", wl)
    d = P.im2win_desc(n, c, h, w, k, fh, fw, sh, sw, ph, pw, P.IM2WIN_F32, layout)
    want = "f32_bands_small_c" if case in F32_BANDS_SMALL_C else "f32_bands"
    assert P.im2win_conv_kernel(d, False) == P.im2win_conv_kernel(d, True) == want
    assert P.im2win_check_plan(d) == 0, P.im2win_last_error()
    x, wt = x_cpu.to(DEV), w_cpu.to(DEV)
    ho, wo = P.im2win_output_shape(d)
    numel = n * k * ho * wo
    outs = []
    for fused in (False, True):
        ybuf = torch.full((numel + 4096,), float("nan"), dtype=torch.float32, device=DEV)
        y = ybuf[:numel].view(n, k, ho, wo)
        if fused:
            P.conv2d_fused(x, wt, d, y=y)
        else:
            P.conv2d(P.transform(x, d), wt, d, y=y)
        torch.cuda.synchronize()
        assert torch.isnan(ybuf[numel:]).all(), "convolution wrote past the output"
        outs.append(y.cpu().numpy().astype(np.float64))
    assert np.array_equal(outs[0], outs[1]), "fused and unfused outputs differ"
    ref, ref_abs = oracle.direct_conv(_shape(wl), _f64(x_cpu), _f64(w_cpu), with_abs=True)
    rel = _assert_close(outs[0], ref, ref_abs, c * fh * fw, "f32", "band kernel")
    print(f"[parity] rel-L2 {rel:.3e}", flush=True)


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


REPACK_CASES = [
    ("f32", (2, 3, 30, 30, 64, 7, 7, 2, 2, 3, 3)),    # fp32 rows not whole vectors: repacked
    ("bf16", (2, 32, 14, 14, 64, 3, 3, 1, 1, 1, 1)),  # bf16 fast kernels: 8-channel pieces
    ("f32", (1, 6, 24, 24, 96, 5, 5, 1, 1, 0, 0)),
    ("f32", (1, 3, 47, 47, 96, 11, 11, 4, 4, 0, 0)),
    ("bf16", (1, 64, 10, 12, 128, 3, 3, 1, 1, 1, 1)),
]


def _check_runs(runs):
    for wl, x_cpu, w_cpu, y, y_fused in runs:
        ref, ref_abs = oracle.direct_conv(_shape(wl), _f64(x_cpu), _f64(w_cpu), with_abs=True)
        for what, out in (("unfused", y), ("fused", y_fused)):
            _assert_close(out.cpu().numpy().astype(np.float64), ref, ref_abs, wl.c * wl.fh * wl.fw, wl.dtype,
                          f"{wl.name} {what}")


def test_repacked_filters_in_caller_scratch_on_two_streams():
    """Filters that the kernels read repacked go to the scratch each call is
    given: fp32 and bf16 convolutions with different filters interleaved on
    two streams, each call with its own scratch, each result against the
    oracle."""
    streams = [torch.cuda.Stream(device=DEV), torch.cuda.Stream(device=DEV)]
    runs = []
    for i, (dtype, shape) in enumerate(REPACK_CASES + REPACK_CASES[:1]):
        wl, x_cpu, w_cpu = workloads.random_case(800 + i, *shape, dtype=dtype)
        _label("repacked-filter stream", wl)
        d = _desc(wl)
        assert P.im2win_check_plan(d) == 0, P.im2win_last_error()
        stream = streams[i % 2]
        with torch.cuda.stream(stream):
            x, w = x_cpu.to(DEV), w_cpu.to(DEV)
            y_fused = P.conv2d_fused(x, w, d, stream=stream)
            y = P.conv2d(P.transform(x, d, stream=stream), w, d, stream=stream)
        runs.append((wl, x_cpu, w_cpu, y, y_fused))
    torch.cuda.synchronize()
    _check_runs(runs)


def test_two_host_threads_on_the_default_stream():
    """Two host threads call the library at once on the same (default) stream,
    each with its own filters -- fp32 ones that are repacked and bf16 ones for
    the fast kernels -- and its own scratch: the library keeps no state
    between calls, so every result matches the oracle."""
    import threading
    cases = [[REPACK_CASES[0], REPACK_CASES[1], REPACK_CASES[3]],
             [REPACK_CASES[4], REPACK_CASES[2], REPACK_CASES[1]]]
    inputs = [[workloads.random_case(900 + 10 * t + i, *shape, dtype=dtype) for i, (dtype, shape) in enumerate(cs)]
              for t, cs in enumerate(cases)]
    for per in inputs:
        for wl, _, _ in per:
            assert P.im2win_check_plan(_desc(wl)) == 0, P.im2win_last_error()
    results = [[], []]
    errors = []
    barrier = threading.Barrier(2)

    def worker(t):
        try:
            torch.cuda.set_device(0)
            barrier.wait()
            for _ in range(3):
                for wl, x_cpu, w_cpu in inputs[t]:
                    d = _desc(wl)
                    x, w = x_cpu.to(DEV), w_cpu.to(DEV)
                    y_fused = P.conv2d_fused(x, w, d)
                    y = P.conv2d(P.transform(x, d), w, d)
                    results[t].append((wl, x_cpu, w_cpu, y, y_fused))
        except Exception as e:   # reported by the main thread
            errors.append(e)

    print("[parity] two host threads on the default stream", flush=True)
    threads = [threading.Thread(target=worker, args=(t,)) for t in (0, 1)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not errors, errors
    _check_runs(results[0] + results[1])


def test_transform_rows_beyond_lds():
    """Window-tensor rows too long to build in on-chip memory (a 2000-wide
    input with a 9x9 filter: Wp*Fh*4 = 72 KB per row) take the transform's
    direct kernel, one workgroup per row: bit-exact, with a guard band."""
    for dtype in ("f32", "bf16"):
        wl, x_cpu, w_cpu = workloads.random_case(950, 1, 2, 12, 2000, 3, 9, 9, 1, 1, 0, 0, dtype)
        _label("transform-direct", wl)
        assert P.im2win_check_plan(_desc(wl)) == 0, P.im2win_last_error()
        _check_transform(wl, x_cpu, wl.n)


NO_TILE = [
    (1, 2, 3, 4096, 3, 3, 4096, 1, 1, 0, 0),       # filter as wide as the input: Wo = 1
    (2, 1, 5, 20000, 2, 5, 19000, 1, 7, 0, 0),     # 64 windows of one row span 97k elements
    (1, 3, 4, 3000, 2, 3, 2990, 2, 3, 1, 0),       # stride, padding, Wo = 4
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", NO_TILE, ids=lambda c: "x".join(map(str, c)))
def test_shapes_without_an_lds_tile(case, dtype):
    """Window strips no LDS tile holds: both convolutions run on the
    per-output kernel, against the oracle; no filter scratch is needed."""
    wl, x_cpu, w_cpu = workloads.random_case(sum(case), *case, dtype=dtype)
    _label("no-tile", wl)
    d = _desc(wl)
    assert P.im2win_filter_scratch_bytes(d) == 0
    assert P.im2win_check_plan(d) == 0, P.im2win_last_error()
    _check_transform(wl, x_cpu, wl.n)
    ref, ref_abs = oracle.direct_conv(_shape(wl), _f64(x_cpu), _f64(w_cpu), with_abs=True)
    y_unf = _run_conv(wl, x_cpu, w_cpu, wl.n, False)
    y_fus = _run_conv(wl, x_cpu, w_cpu, wl.n, True)
    nterms = wl.c * wl.fh * wl.fw
    _assert_close(y_unf, ref, ref_abs, nterms, dtype, "unfused")
    _assert_close(y_fus, ref, ref_abs, nterms, dtype, "fused")


def test_one_hip_runtime_after_gpu_use():
    assert len(P.hip_runtimes_mapped()) == 1, P.hip_runtimes_mapped()
