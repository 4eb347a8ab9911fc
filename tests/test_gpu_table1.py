"""GPU parity on the paper's twelve benchmark layers (Sec. IV-A, Table 1), fp32,
no padding, at the paper's batch of 128 (the launch configuration that
`bench.py --table1` times) and at batch 2.

- batch 128: the window tensor of the first and the last image bit-exact
  against the oracle's Alg. 1 copy; the convolution on sampled outputs of four
  images against the fp64 direct convolution, element by element within the
  fp32 rounding bound; fused and unfused outputs bitwise identical over the
  whole tensor;
- batch 2: the whole output of both convolutions against the oracle.
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
RELL2 = 1e-5
SAMPLED_IMAGES = (0, 1, 63, 127)


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
                         P.IM2WIN_F32)


def _assert_close(got, ref, ref_abs, nterms, what):
    bound = (nterms + 2) * U32 * ref_abs + 1e-30
    err = np.abs(got - ref)
    assert np.all(err <= bound), f"{what}: {np.sum(err > bound)} outputs outside the fp32 rounding bound"
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300)
    assert rel <= RELL2, f"{what}: relative L2 error {rel:.3e}"
    return rel


def _run(wl, x, w, n):
    """transform + conv2d and conv2d_fused on device tensors; returns (ws, y, y_fused)."""
    d = _desc(wl, n)
    ws = P.transform(x, d)
    y = P.conv2d(ws, w, d)
    y2 = P.conv2d_fused(x, w, d)
    torch.cuda.synchronize()
    return ws, y, y2


@pytest.mark.parametrize("wl", workloads.TABLE1, ids=lambda wl: wl.name)
def test_table1_full_batch_sampled(wl):
    print(f"[parity] table1 full batch {wl.label()}", flush=True)
    n = wl.n
    s = _shape(wl, n)
    x_cpu, w_cpu = workloads.make_input(wl), workloads.make_filter(wl)
    x, w = x_cpu.to(DEV), w_cpu.to(DEV)
    ws, y, y2 = _run(wl, x, w, n)
    assert torch.equal(y, y2), "fused and unfused outputs differ"
    # window tensor of the first and the last image (each image's rows depend
    # on that image alone)
    s1 = _shape(wl, 1)
    for i in (0, n - 1):
        got = ws[i].contiguous().view(torch.int32).cpu().numpy()
        ref = oracle.im2win(s1, x_cpu[i:i + 1].view(torch.int32).numpy())
        assert np.array_equal(got.reshape(-1), ref.reshape(-1)), f"window tensor of image {i} differs"
    # sampled outputs of four images
    rng = np.random.default_rng(wl.seed_x)
    per = wl.k * s.ho * s.wo
    picks = []
    for slot, i in enumerate(SAMPLED_IMAGES):
        local = np.unique(np.concatenate([rng.integers(0, per, size=500), [0, per - 1]]))
        picks.append((slot, i, local))
    sub = Shape(len(SAMPLED_IMAGES), wl.c, wl.h, wl.w, wl.k, wl.fh, wl.fw, wl.sh, wl.sw, wl.ph, wl.pw)
    idx_sub = np.concatenate([slot * per + loc for slot, _, loc in picks])
    idx_full = np.concatenate([i * per + loc for _, i, loc in picks])
    x_sub = x_cpu[list(SAMPLED_IMAGES)].double().numpy()
    ref, ref_abs = oracle.direct_conv_at(sub, x_sub, w_cpu.double().numpy(), idx_sub)
    got = y.view(-1)[torch.from_numpy(idx_full).to(DEV)].double().cpu().numpy()
    rel = _assert_close(got, ref, ref_abs, wl.c * wl.fh * wl.fw, wl.name + " (sampled)")
    print(f"[parity] sampled rel-L2 {rel:.3e} over {idx_full.size} outputs", flush=True)


@pytest.mark.parametrize("wl", workloads.TABLE1, ids=lambda wl: wl.name)
def test_table1_whole_output_batch2(wl):
    print(f"[parity] table1 batch 2 {wl.name}", flush=True)
    n = 2
    s = _shape(wl, n)
    x_cpu, w_cpu = workloads.make_input(wl, n_images=n), workloads.make_filter(wl)
    _, y, y2 = _run(wl, x_cpu.to(DEV), w_cpu.to(DEV), n)
    ref, ref_abs = oracle.direct_conv(s, x_cpu.double().numpy(), w_cpu.double().numpy(), with_abs=True)
    for what, out in (("unfused", y), ("fused", y2)):
        _assert_close(out.double().cpu().numpy(), ref, ref_abs, wl.c * wl.fh * wl.fw, f"{wl.name} {what}")
