"""Host-side checks of bench.py (no GPU): the one-GPU contract, the rule that
HBM traffic is reported only for the kernel sources it was measured on, and
the im2col + GEMM comparison system's arithmetic (run on the CPU in fp64
against the oracle's direct convolution)."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

import bench
import oracle
from oracle import Shape
from conftest import ROOT


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_reported_only_for_the_measured_sources(tmp_path, monkeypatch):
    f = tmp_path / "traffic.json"
    entry = {"bytes_per_launch": 123, "source_hash": bench.source_hash("conv")}
    f.write_text(json.dumps({"resnet_3x3_f32": {"fused": entry}}))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.measured_traffic("resnet_3x3_f32", "fused") == 123
    assert bench.measured_traffic("resnet_3x3_f32", "conv") is None
    entry["source_hash"] = "0" * 16
    f.write_text(json.dumps({"resnet_3x3_f32": {"fused": entry}}))
    assert bench.measured_traffic("resnet_3x3_f32", "fused") is None


@pytest.mark.parametrize("shape", [
    (2, 3, 9, 11, 5, 3, 5, 2, 2, 1, 2),
    (1, 4, 8, 8, 6, 3, 3, 1, 1, 1, 1),
    (1, 2, 9, 9, 3, 2, 2, 3, 3, 0, 0),
])
def test_im2col_gemm_baseline_computes_the_convolution(shape):
    s = Shape(*shape)
    rng = np.random.default_rng(sum(shape))
    x = rng.uniform(-1, 1, (s.n, s.c, s.h, s.w))
    w = rng.uniform(-1, 1, (s.k, s.c, s.fh, s.fw))
    y = bench.im2col_conv2d(torch.from_numpy(x), torch.from_numpy(w), (s.sh, s.sw), (s.ph, s.pw))
    assert tuple(y.shape) == s.out_shape
    np.testing.assert_allclose(y.double().numpy(), oracle.direct_conv(s, x, w), rtol=0, atol=1e-5)
