"""Seeded synthetic workloads for the im2win convolution.

Shared by the tests, the benchmark and the smoke check.  This module only
describes problem shapes and draws random tensors; it holds none of the
method's arithmetic (no output sizes, no index formulas), so that the oracle
and the HIP library can both be fed from it without sharing any code.

Distributions follow the workload descriptions: U[a,b] is ``a + (b-a)*rand``;
N(0,1) is ``randn``; "N(0, 2/fan_in)" is read as variance 2/fan_in (He
initialisation), i.e. ``randn * sqrt(2/fan_in)`` with fan_in = C*Fh*Fw.
bf16 workloads draw in fp32 and round to bf16 with round-to-nearest-even.
Seeds: workload number c (1-based) draws x from seed 100*c+1 and w from 100*c+2.
"""
from dataclasses import dataclass, replace
import math

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    c: int
    h: int
    w: int
    k: int
    fh: int
    fw: int
    sh: int
    sw: int
    ph: int
    pw: int
    dtype: str            # "f32" or "bf16": dtype of x, w and the window tensor
    x_dist: tuple         # ("uniform", lo, hi) | ("normal", std)
    w_dist: tuple         # ("uniform", lo, hi) | ("he",)
    seed_x: int
    seed_w: int

    def with_batch(self, n: int) -> "Workload":
        """Same layer with another batch size (and so other random draws)."""
        return replace(self, n=n)

    def label(self) -> str:
        return (f"{self.name}: {self.dtype} N={self.n} C={self.c} H={self.h} W={self.w} "
                f"K={self.k} {self.fh}x{self.fw} s=({self.sh},{self.sw}) p=({self.ph},{self.pw})")


WORKLOADS = [
    Workload("single_3x3_f32", 1, 3, 32, 32, 16, 3, 3, 1, 1, 0, 0, "f32",
             ("uniform", -1.0, 1.0), ("uniform", -1.0, 1.0), 101, 102),
    Workload("resnet_3x3_f32", 32, 64, 56, 56, 64, 3, 3, 1, 1, 1, 1, "f32",
             ("uniform", 0.0, 1.0), ("he",), 201, 202),
    Workload("stem_7x7_s2_f32", 32, 3, 224, 224, 64, 7, 7, 2, 2, 3, 3, "f32",
             ("normal", 1.0), ("he",), 301, 302),
    Workload("deep_3x3_bf16", 128, 256, 14, 14, 256, 3, 3, 1, 1, 1, 1, "bf16",
             ("uniform", 0.0, 1.0), ("he",), 401, 402),
    Workload("rect_3x5_s2_f32", 64, 128, 28, 28, 128, 3, 5, 2, 2, 1, 2, "f32",
             ("uniform", -1.0, 1.0), ("he",), 501, 502),
]

BY_NAME = {wl.name: wl for wl in WORKLOADS}

# The paper's twelve benchmark layers (Sec. IV-A, Table 1): input Ci x Hi x Wi,
# filter Co x Hf x Wf with stride s, no padding, batch 128 (Sec. IV-B), fp32.
# The paper states no data distribution; these draw U[-1,1] inputs and
# He-scaled normal weights.  Layer i (1-based) seeds x with 1000+10i+1 and w
# with 1000+10i+2.
_TABLE1_SHAPES = [
    # (Ci, Hi, Wi, Co, Hf, Wf, s)
    (3, 227, 227, 96, 11, 11, 4),
    (3, 231, 231, 96, 11, 11, 4),
    (3, 227, 227, 64, 7, 7, 2),
    (64, 224, 224, 64, 7, 7, 2),
    (96, 24, 24, 256, 5, 5, 1),
    (256, 12, 12, 512, 3, 3, 1),
    (3, 224, 224, 64, 3, 3, 1),
    (64, 112, 112, 128, 3, 3, 1),
    (64, 56, 56, 64, 3, 3, 1),
    (128, 28, 28, 128, 3, 3, 1),
    (256, 14, 14, 256, 3, 3, 1),
    (512, 7, 7, 512, 3, 3, 1),
]
TABLE1_BATCH = 128
TABLE1 = [
    Workload(f"table1_conv{i}", TABLE1_BATCH, ci, hi, wi, co, hf, wf, s, s, 0, 0, "f32",
             ("uniform", -1.0, 1.0), ("he",), 1000 + 10 * i + 1, 1000 + 10 * i + 2)
    for i, (ci, hi, wi, co, hf, wf, s) in enumerate(_TABLE1_SHAPES, start=1)
]
BY_NAME.update({wl.name: wl for wl in TABLE1})

# The workload the benchmark's headline line is quoted on.
HEADLINE = BY_NAME["resnet_3x3_f32"]


def torch_dtype(dt: str):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dt]


def _draw(shape, dist, seed, fan_in):
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    kind = dist[0]
    if kind == "uniform":
        lo, hi = dist[1], dist[2]
        return lo + (hi - lo) * torch.rand(shape, generator=g, dtype=torch.float32)
    if kind == "normal":
        return dist[1] * torch.randn(shape, generator=g, dtype=torch.float32)
    if kind == "he":
        return math.sqrt(2.0 / fan_in) * torch.randn(shape, generator=g, dtype=torch.float32)
    raise ValueError(f"unknown distribution {dist}")


def make_input(wl: Workload, n_images: int = None) -> torch.Tensor:
    """x, N x C x H x W, on the CPU in the workload's dtype.  With n_images,
    the first n_images images of the full draw (a prefix of the same tensor)."""
    x = _draw((wl.n, wl.c, wl.h, wl.w), wl.x_dist, wl.seed_x, wl.c * wl.fh * wl.fw)
    if n_images is not None:
        x = x[:n_images]
    return x.to(torch_dtype(wl.dtype)).contiguous()


def make_filter(wl: Workload) -> torch.Tensor:
    """w, K x C x Fh x Fw, on the CPU in the workload's dtype."""
    w = _draw((wl.k, wl.c, wl.fh, wl.fw), wl.w_dist, wl.seed_w, wl.c * wl.fh * wl.fw)
    return w.to(torch_dtype(wl.dtype)).contiguous()


def random_case(seed: int, n, c, h, w, k, fh, fw, sh=1, sw=1, ph=0, pw=0, dtype="f32"):
    """A small random problem (uniform[-1,1] data) for parity and edge tests."""
    wl = Workload(f"case{seed}", n, c, h, w, k, fh, fw, sh, sw, ph, pw, dtype,
                  ("uniform", -1.0, 1.0), ("uniform", -1.0, 1.0), 2 * seed + 1, 2 * seed + 2)
    return wl, make_input(wl), make_filter(wl)
