"""The entry point that allocates nothing (im2win_conv2d_fused_noalloc):
through the C ABI, its output equals im2win_conv2d_fused's (same kernels,
caller-owned scratch there, the library's static array here) on two calls in
a row on one stream, the second with a smaller problem, for fp32 filters that
are repacked and for bf16 fast-kernel filters; each also within the oracle's
fp32 rounding bound."""
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

# (dtype, (n, c, h, w, k, fh, fw, sh, sw, ph, pw)): larger first, then smaller
SEQUENCES = [
    ("bf16", [(8, 256, 14, 14, 256, 3, 3, 1, 1, 1, 1), (2, 64, 10, 12, 128, 3, 3, 1, 1, 1, 1)]),
    # (five input channels: the three-channel band kernel, which reads the
    # filter as it is, does not take the first)
    ("f32", [(4, 5, 224, 224, 64, 7, 7, 2, 2, 3, 3), (1, 3, 40, 36, 64, 7, 7, 2, 2, 3, 3)]),
]


def _desc(wl):
    return P.im2win_desc(wl.n, wl.c, wl.h, wl.w, wl.k, wl.fh, wl.fw, wl.sh, wl.sw, wl.ph, wl.pw,
                         P.IM2WIN_F32 if wl.dtype == "f32" else P.IM2WIN_BF16)


@pytest.mark.parametrize("dtype,shapes", SEQUENCES, ids=[s[0] for s in SEQUENCES])
def test_noalloc_matches_fused_on_two_calls(dtype, shapes):
    assert torch.cuda.is_available()
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    for i, shape in enumerate(shapes):
        wl, x_cpu, w_cpu = workloads.random_case(1300 + 10 * i + len(dtype), *shape, dtype=dtype)
        print(f"[noalloc] call {i + 1}: {wl.label()}", flush=True)
        d = _desc(wl)
        need = P.im2win_filter_scratch_bytes(d)
        assert 0 < need <= P.IM2WIN_NOALLOC_SCRATCH_BYTES
        assert P.im2win_check_plan(d) == 0, P.im2win_last_error()
        x, w = x_cpu.to(DEV), w_cpu.to(DEV)
        ho, wo = P.im2win_output_shape(d)
        total = wl.n * wl.k * ho * wo
        ybuf = torch.full((total + 4096,), float("nan"), dtype=torch.float32, device=DEV)
        y_ref = torch.empty(total, dtype=torch.float32, device=DEV)
        scratch = torch.empty(need, dtype=torch.uint8, device=DEV)
        P.im2win_conv2d_fused(d, x.data_ptr(), w.data_ptr(), scratch.data_ptr(), need, y_ref.data_ptr(), sp)
        P.im2win_conv2d_fused_noalloc(d, x.data_ptr(), w.data_ptr(), ybuf.data_ptr(), sp)
        torch.cuda.synchronize()
        assert torch.isnan(ybuf[total:]).all(), "wrote past the output"
        got = ybuf[:total].cpu().numpy()
        ref = y_ref.cpu().numpy()
        assert np.array_equal(got.view(np.int32), ref.view(np.int32)), "differs from im2win_conv2d_fused"
        s = Shape(*shape)
        exact, exact_abs = oracle.direct_conv(s, x_cpu.double().numpy(), w_cpu.double().numpy(), with_abs=True)
        err = np.abs(got.astype(np.float64).reshape(exact.shape) - exact)
        assert np.all(err <= (wl.c * wl.fh * wl.fw + 2) * U32 * exact_abs + 1e-30)
