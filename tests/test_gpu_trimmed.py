"""GPU parity of the trimmed window-tensor layout (rows of (Wo-1)*sw + Fw
columns, only those some window reads) through the C ABI, against the
oracle's trimmed transformation and its fp64 direct convolution:

- transformation: bit-exact on every workload at full size and on edge
  shapes, with a poisoned buffer (every element must be written) and a guard
  band after it (nothing else may be);
- convolution from the trimmed window tensor and fused convolution with the
  trimmed descriptor: element by element within the fp32 rounding bound and
  relative L2 within the dtype's bound, whole output at reduced batch; fused
  and unfused bitwise identical.
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
REDUCED_N = {"single_3x3_f32": 1, "resnet_3x3_f32": 2, "stem_7x7_s2_f32": 2,
             "deep_3x3_bf16": 2, "rect_3x5_s2_f32": 3}
EDGE = [
    # (n, c, h, w, k, fh, fw, sh, sw, ph, pw): the trimmed rows end before the
    # last input columns, so those columns are skipped on chip
    (2, 3, 12, 12, 5, 3, 2, 1, 3, 0, 0),      # Wt 11 of 12
    (1, 4, 9, 17, 3, 2, 2, 1, 4, 0, 0),       # Fw < sw: 14 of 17
    (2, 17, 13, 32, 33, 3, 5, 2, 2, 0, 0),    # rectangular, ragged channels: 31 of 32
    (1, 33, 30, 70, 65, 7, 7, 2, 2, 0, 0),    # 7x7 stride 2: 69 of 70
    (2, 8, 10, 16, 16, 3, 3, 1, 4, 1, 1),     # padded: 15 of 18, input columns 14-15 unread
    (2, 32, 14, 16, 64, 3, 3, 1, 2, 0, 0),    # bf16 fast-kernel channels: 15 of 16
    (3, 16, 9, 9, 64, 3, 3, 2, 2, 0, 0),      # nothing to trim: 9 of 9
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
                         P.IM2WIN_F32 if wl.dtype == "f32" else P.IM2WIN_BF16, P.IM2WIN_ROWS_TRIMMED)


def _bits(t):
    t = t.detach().cpu().contiguous()
    return (t.view(torch.int32) if t.element_size() == 4 else t.view(torch.int16)).numpy()


def _check_transform(wl, x_cpu, n):
    s = _shape(wl, n)
    d = _desc(wl, n)
    numel = P.im2win_workspace_bytes(d) // x_cpu.element_size()
    assert numel == oracle.im2win_elems(s, trimmed=True)
    buf = torch.empty(numel + 4096, dtype=x_cpu.dtype, device=DEV)
    (buf.view(torch.int32) if buf.element_size() == 4 else buf.view(torch.int16)).fill_(-1)
    P.transform(x_cpu.to(DEV), d, ws=buf[:numel].view(s.win_shape_of(True)))
    torch.cuda.synchronize()
    got = _bits(buf)
    ref = oracle.im2win(s, _bits(x_cpu), trimmed=True)
    assert np.array_equal(got[:numel], ref.reshape(-1)), "trimmed window tensor differs from the oracle"
    assert np.all(got[numel:] == -1), "transformation wrote past the window tensor"


def _convs(wl, x_cpu, w_cpu, n):
    d = _desc(wl, n)
    assert P.im2win_check_plan(d) == 0, P.im2win_last_error()
    x, w = x_cpu.to(DEV), w_cpu.to(DEV)
    ho, wo = P.im2win_output_shape(d)
    numel = n * wl.k * ho * wo
    outs = []
    for fused in (False, True):
        ybuf = torch.full((numel + 4096,), float("nan"), dtype=torch.float32, device=DEV)
        y = ybuf[:numel].view(n, wl.k, ho, wo)
        if fused:
            P.conv2d_fused(x, w, d, y=y)
        else:
            P.conv2d(P.transform(x, d), w, d, y=y)
        torch.cuda.synchronize()
        assert torch.isnan(ybuf[numel:]).all(), "convolution wrote past the output"
        outs.append(y.cpu().numpy().astype(np.float64))
    return outs


def _assert_close(got, ref, ref_abs, nterms, dtype, what):
    bound = (nterms + 2) * U32 * ref_abs + 1e-30
    err = np.abs(got - ref)
    assert np.all(err <= bound), f"{what}: {np.sum(err > bound)} outputs outside the fp32 rounding bound"
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)
    assert rel <= RELL2[dtype], f"{what}: relative L2 error {rel:.3e}"
    return rel


@pytest.mark.parametrize("wl", workloads.WORKLOADS, ids=lambda wl: wl.name)
def test_trimmed_transform_bit_exact_full_size(wl):
    print(f"[trimmed] transform {wl.label()}", flush=True)
    _check_transform(wl, workloads.make_input(wl), wl.n)


@pytest.mark.parametrize("wl", workloads.WORKLOADS, ids=lambda wl: wl.name)
def test_trimmed_conv_reduced_batch(wl):
    n = REDUCED_N[wl.name]
    print(f"[trimmed] conv {wl.label()} n={n}", flush=True)
    x_cpu, w_cpu = workloads.make_input(wl, n_images=n), workloads.make_filter(wl)
    y_unf, y_fus = _convs(wl, x_cpu, w_cpu, n)
    ref, ref_abs = oracle.direct_conv(_shape(wl, n), x_cpu.double().numpy(), w_cpu.double().numpy(),
                                      with_abs=True)
    rel = _assert_close(y_unf, ref, ref_abs, wl.c * wl.fh * wl.fw, wl.dtype, wl.name)
    assert np.array_equal(y_unf, y_fus), "fused and unfused outputs differ"
    print(f"[trimmed] rel-L2 {rel:.3e}", flush=True)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", EDGE, ids=lambda c: "x".join(map(str, c)))
def test_trimmed_edge_shapes(case, dtype):
    n, c, h, w, k, fh, fw, sh, sw, ph, pw = case
    wl, x_cpu, w_cpu = workloads.random_case(sum(case) + 11, n, c, h, w, k, fh, fw, sh, sw, ph, pw, dtype)
    print(f"[trimmed] edge {wl.label()}", flush=True)
    _check_transform(wl, x_cpu, n)
    y_unf, y_fus = _convs(wl, x_cpu, w_cpu, n)
    ref, ref_abs = oracle.direct_conv(_shape(wl, n), x_cpu.double().numpy(), w_cpu.double().numpy(),
                                      with_abs=True)
    _assert_close(y_unf, ref, ref_abs, c * fh * fw, dtype, "unfused")
    _assert_close(y_fus, ref, ref_abs, c * fh * fw, dtype, "fused")
