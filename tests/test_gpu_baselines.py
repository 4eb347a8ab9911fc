"""GPU checks of the comparison systems that bench.py --baselines times against
the im2win path (Sec. IV-B, Fig. 4): they must compute the same convolution,
or the speedups compare different work.

- direct convolution (the library's im2win_direct_conv2d, no transformation):
  element by element within the fp32 rounding bound against the oracle's
  fp64 direct convolution, on every workload at reduced batch and on edge
  shapes, fp32 and bf16, with a guard band after the output;
- im2col + GEMM (unfold and a batched GEMM): relative L2 error within the
  dtype's bound (fp32 1e-5; bf16 1e-2, its GEMM result is bf16);
- the peak-memory probe: the im2win path's peak is exactly x + w + window
  tensor + y, and im2col's is larger on the workloads.
"""
import numpy as np
import pytest
import torch

import bench
import oracle
from oracle import Shape
import workloads
import paper_2306_14320_amd as P

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
U32 = 2.0 ** -24
RELL2 = {"f32": 1e-5, "bf16": 1e-2}
REDUCED_N = {"single_3x3_f32": 1, "resnet_3x3_f32": 2, "stem_7x7_s2_f32": 2,
             "deep_3x3_bf16": 2, "rect_3x5_s2_f32": 3}
EDGE = [
    # (n, c, h, w, k, fh, fw, sh, sw, ph, pw)
    (1, 1, 4, 4, 2, 2, 2, 1, 1, 0, 0),
    (2, 3, 9, 11, 5, 3, 5, 2, 2, 1, 2),
    (1, 2, 9, 9, 3, 2, 2, 3, 3, 0, 0),        # Fh < sh, Fw < sw
    (1, 4, 5, 6, 3, 5, 6, 1, 1, 0, 0),        # Ho = Wo = 1
    (3, 2, 3, 3, 2, 3, 3, 1, 1, 2, 2),        # padding wider than the input
    (1, 3, 227, 227, 96, 11, 11, 4, 4, 0, 0), # Table 1 Conv1 at batch 1
]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    P.load_library()
    yield
    torch.cuda.synchronize()


def _shape(wl, n):
    return Shape(n, wl.c, wl.h, wl.w, wl.k, wl.fh, wl.fw, wl.sh, wl.sw, wl.ph, wl.pw)


def _desc(wl, n):
    return P.im2win_desc(n, wl.c, wl.h, wl.w, wl.k, wl.fh, wl.fw, wl.sh, wl.sw, wl.ph, wl.pw,
                         P.IM2WIN_F32 if wl.dtype == "f32" else P.IM2WIN_BF16)


def _f64(t):
    return t.detach().to(torch.float64).cpu().numpy()


def _direct(wl, x_cpu, w_cpu, n):
    d = _desc(wl, n)
    ho, wo = P.im2win_output_shape(d)
    numel = n * wl.k * ho * wo
    ybuf = torch.full((numel + 4096,), float("nan"), dtype=torch.float32, device=DEV)
    P.direct_conv2d(x_cpu.to(DEV), w_cpu.to(DEV), d, y=ybuf[:numel].view(n, wl.k, ho, wo))
    torch.cuda.synchronize()
    assert torch.isnan(ybuf[numel:]).all(), "direct convolution wrote past the output"
    return ybuf[:numel].cpu().numpy().astype(np.float64)


def _assert_close(got, ref, ref_abs, nterms, dtype, what):
    bound = (nterms + 2) * U32 * ref_abs + 1e-30
    err = np.abs(got - ref)
    assert np.all(err <= bound), f"{what}: {np.sum(err > bound)} outputs outside the fp32 rounding bound"
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)
    assert rel <= RELL2[dtype], f"{what}: relative L2 error {rel:.3e}"
    return rel


@pytest.mark.parametrize("wl", workloads.WORKLOADS, ids=lambda wl: wl.name)
def test_direct_conv_workloads_reduced_batch(wl):
    n = REDUCED_N[wl.name]
    print(f"[baseline] direct {wl.label()} n={n}", flush=True)
    x_cpu, w_cpu = workloads.make_input(wl, n_images=n), workloads.make_filter(wl)
    got = _direct(wl, x_cpu, w_cpu, n)
    ref, ref_abs = oracle.direct_conv(_shape(wl, n), _f64(x_cpu), _f64(w_cpu), with_abs=True)
    rel = _assert_close(got.reshape(ref.shape), ref, ref_abs, wl.c * wl.fh * wl.fw, wl.dtype, wl.name)
    print(f"[baseline] rel-L2 {rel:.3e}", flush=True)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", EDGE, ids=lambda c: "x".join(map(str, c)))
def test_direct_conv_edge_shapes(case, dtype):
    n, c, h, w, k, fh, fw, sh, sw, ph, pw = case
    wl, x_cpu, w_cpu = workloads.random_case(sum(case) + 7, n, c, h, w, k, fh, fw, sh, sw, ph, pw, dtype)
    print(f"[baseline] direct edge {wl.label()}", flush=True)
    got = _direct(wl, x_cpu, w_cpu, n)
    ref, ref_abs = oracle.direct_conv(_shape(wl, n), _f64(x_cpu), _f64(w_cpu), with_abs=True)
    _assert_close(got.reshape(ref.shape), ref, ref_abs, c * fh * fw, dtype, "direct")


@pytest.mark.parametrize("wl", [workloads.BY_NAME["rect_3x5_s2_f32"], workloads.BY_NAME["deep_3x3_bf16"]],
                         ids=lambda wl: wl.name)
def test_im2col_gemm_baseline(wl):
    n = 2
    print(f"[baseline] im2col+gemm {wl.label()} n={n}", flush=True)
    x_cpu, w_cpu = workloads.make_input(wl, n_images=n), workloads.make_filter(wl)
    y = bench.im2col_conv2d(x_cpu.to(DEV), w_cpu.to(DEV), (wl.sh, wl.sw), (wl.ph, wl.pw))
    torch.cuda.synchronize()
    ref = oracle.direct_conv(_shape(wl, n), _f64(x_cpu), _f64(w_cpu))
    got = _f64(y)
    assert got.shape == ref.shape
    rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert rel <= RELL2[wl.dtype], f"relative L2 error {rel:.3e}"


@pytest.mark.parametrize("name", ["resnet_3x3_f32", "deep_3x3_bf16", "stem_7x7_s2_f32"])
def test_peak_memory_probe(name):
    """Peak device bytes of one call: x + w + window tensor + filter scratch
    + y for transform + conv2d, x + w + scratch + y fused (the repacked filter
    is caller-owned now, so it is counted)."""
    wl = workloads.BY_NAME[name]
    line = bench.compare_baselines(wl, n=2)
    d = _desc(wl, 2)
    ho, wo = P.im2win_output_shape(d)
    e = 4 if wl.dtype == "f32" else 2
    x_bytes = 2 * wl.c * wl.h * wl.w * e
    w_bytes = wl.k * wl.c * wl.fh * wl.fw * e
    y_bytes = 2 * wl.k * ho * wo * 4
    ws_bytes = P.im2win_workspace_bytes(d)
    sc = P.im2win_filter_scratch_bytes(d)
    sc_bytes = max(sc, 16) if sc else 0
    # (which kernels repack the filter is pinned on the CPU; bf16 always does)
    if wl.dtype == "bf16":
        assert sc > 0
    paths = line["paths"]
    # the caching allocator rounds each block up to a multiple of 512 bytes
    assert abs(paths["im2win"]["peak_bytes"] - (x_bytes + w_bytes + ws_bytes + sc_bytes + y_bytes)) < 3072
    assert abs(paths["im2win_fused"]["peak_bytes"] - (x_bytes + w_bytes + sc_bytes + y_bytes)) < 3072
    assert line["im2col_peak_over_im2win"] > 1.0
    for path in ("im2win", "im2win_fused", "im2col_gemm", "direct"):
        assert "ms" in paths[path], (path, paths[path])
