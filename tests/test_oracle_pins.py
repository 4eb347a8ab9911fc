"""Pins for the CPU oracle: each test ties an oracle function to something the
paper prints, to a closed form, or to an independent library routine or brute
force, so that a dropped term, a wrong index or a transposed operand fails.

CPU only (no GPU marker).
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import Shape
from conftest import GOLDEN

RNG = np.random.default_rng(2306_14320)


def _rand(shape):
    return RNG.uniform(-1.0, 1.0, size=shape)


# Small shapes covering square and rectangular filters, strides above and
# below the filter size, asymmetric padding, 1-wide outputs and 1x1 filters.
SMALL_SHAPES = [
    Shape(1, 1, 4, 4, 2, 2, 2),                       # Fig. 2 geometry
    Shape(2, 3, 7, 9, 4, 3, 3, 1, 1, 1, 1),
    Shape(2, 2, 9, 11, 3, 3, 5, 2, 2, 1, 2),          # rectangular 3x5, stride 2
    Shape(1, 3, 10, 8, 2, 5, 3, 2, 1, 2, 0),          # rectangular 5x3, mixed stride
    Shape(1, 2, 11, 13, 3, 7, 7, 2, 2, 3, 3),         # stem-like
    Shape(2, 2, 6, 6, 3, 1, 1),                       # 1x1 filter
    Shape(1, 2, 9, 9, 2, 2, 2, 3, 3),                 # Fh < sh, Fw < sw
    Shape(1, 1, 5, 5, 2, 2, 2, 2, 2),                 # Fh = sh
    Shape(1, 2, 5, 6, 2, 5, 6),                       # filter covers the input: Ho=Wo=1
    Shape(1, 1, 3, 3, 1, 3, 3, 1, 1, 2, 2),           # padding wider than the input
    Shape(3, 1, 1, 8, 2, 1, 3, 1, 2, 0, 1),           # H = 1
]


def _ids(shapes):
    return [f"N{s.n}C{s.c}H{s.h}W{s.w}K{s.k}f{s.fh}x{s.fw}s{s.sh}{s.sw}p{s.ph}{s.pw}" for s in shapes]


# --------------------------------------------------------------------------
# Sizes: worked example, Fig. 2, Table 1, the 2.93x average, the delta formula
# --------------------------------------------------------------------------

def test_worked_example_sizes():
    g = json.load(open(os.path.join(GOLDEN, "worked_example.json")))
    n, c, h, w = g["input_nchw"]
    k, _, fh, fw = g["filter_kcfhfw"]
    s = Shape(n, c, h, w, k, fh, fw, g["stride"], g["stride"], g["padding"], g["padding"])
    assert (s.ho, s.wo) == tuple(g["output_hw"])
    assert n * c * h * w == g["input_elems"]
    assert oracle.im2col_elems(s) == g["im2col_elems"]
    assert oracle.im2win_elems(s) == g["im2win_elems"]
    # "one third fewer" elements than im2col
    assert Fraction(g["im2col_elems"] - g["im2win_elems"], g["im2col_elems"]) == Fraction(1, 3)
    # the transformed tensor really has that many elements
    x = np.arange(16, dtype=np.float32).reshape(1, 1, 4, 4)
    assert oracle.im2win(s, x).size == g["im2win_elems"]


def test_table1_output_extents():
    t = json.load(open(os.path.join(GOLDEN, "table1.json")))
    for layer in t["layers"]:
        ci, hi, wi = layer["input"]
        co, hf, wf = layer["filter"]
        st = layer["stride"]
        oc, ho, wo = layer["output"]
        assert oc == co
        assert oracle.out_extent(hi, hf, st, 0) == ho, layer["name"]
        assert oracle.out_extent(wi, wf, st, 0) == wo, layer["name"]


def test_table1_average_size_ratio():
    t = json.load(open(os.path.join(GOLDEN, "table1.json")))
    ratios = []
    for layer in t["layers"]:
        ci, hi, wi = layer["input"]
        co, hf, wf = layer["filter"]
        st = layer["stride"]
        s = Shape(t["batch"], ci, hi, wi, co, hf, wf, st, st)
        ratios.append(oracle.im2col_elems(s) / oracle.im2win_elems(s))
    mean = sum(ratios) / len(ratios)
    assert round(mean, t["im2col_over_im2win_mean_printed_digits"]) == t["im2col_over_im2win_mean"]


def test_im2win_size_formula_and_delta():
    """Sec. III-A: im2win has N*C*Hf*Wi*Ho elements and, for square filters whose
    stride divides Wi - Wf, im2col exceeds it by Hf*C*(Wi-Wf)*Ho*(Wf/s - 1)."""
    for (c, hw, f, st) in [(3, 227, 11, 4), (64, 56, 3, 1), (5, 17, 3, 2), (2, 9, 3, 3), (4, 12, 4, 2)]:
        s = Shape(1, c, hw, hw, 1, f, f, st, st)
        assert oracle.im2win_elems(s) == c * f * hw * s.ho
        if (hw - f) % st == 0:
            delta = Fraction(f * c * (hw - f) * s.ho) * (Fraction(f, st) - 1)
            assert oracle.im2col_elems(s) - oracle.im2win_elems(s) == delta
        if f == st and hw % st == 0:     # Hf = Wf = s: both equal the input size
            assert oracle.im2win_elems(s) == c * hw * hw == oracle.im2col_elems(s)
    # the general identity (any stride, padding, rectangular filter):
    # im2col - im2win = N*C*Fh*Ho*(Fw*Wo - Wp)
    for s in SMALL_SHAPES:
        assert oracle.im2col_elems(s) - oracle.im2win_elems(s) == \
            s.n * s.c * s.fh * s.ho * (s.fw * s.wo - s.wp)


@pytest.mark.parametrize("s", SMALL_SHAPES, ids=_ids(SMALL_SHAPES))
def test_sizes_match_library(s):
    x = torch.from_numpy(_rand((s.n, s.c, s.h, s.w)))
    w = torch.from_numpy(_rand((s.k, s.c, s.fh, s.fw)))
    y = F.conv2d(x, w, stride=(s.sh, s.sw), padding=(s.ph, s.pw))
    assert tuple(y.shape) == s.out_shape
    cols = F.unfold(x, (s.fh, s.fw), stride=(s.sh, s.sw), padding=(s.ph, s.pw))
    assert cols.numel() == oracle.im2col_elems(s)


# --------------------------------------------------------------------------
# The transformation
# --------------------------------------------------------------------------

@pytest.mark.parametrize("s", SMALL_SHAPES, ids=_ids(SMALL_SHAPES))
def test_im2win_windows_match_unfold(s):
    """Every window read by the convolution (row m, start column n*sw, Fw columns
    of Fh values each) equals the im2col column that torch's unfold builds."""
    x = _rand((s.n, s.c, s.h, s.w))
    win = oracle.im2win(s, x.astype(np.float32))
    cols = F.unfold(torch.from_numpy(x.astype(np.float32)), (s.fh, s.fw),
                    stride=(s.sh, s.sw), padding=(s.ph, s.pw)).numpy()
    cols = cols.reshape(s.n, s.c, s.fh, s.fw, s.ho, s.wo)
    for m in range(s.ho):
        for n in range(s.wo):
            for u in range(s.fh):
                for v in range(s.fw):
                    got = win[:, :, m, (n * s.sw + v) * s.fh + u]
                    np.testing.assert_array_equal(got, cols[:, :, u, v, m, n])


@pytest.mark.parametrize("s", SMALL_SHAPES, ids=_ids(SMALL_SHAPES))
def test_im2win_every_element_is_padded_input(s):
    """All Wp*Fh positions of a row, including columns no window reaches, hold
    the zero-padded input column-major over the Fh rows starting at m*sh."""
    x = _rand((s.n, s.c, s.h, s.w)).astype(np.float32)
    win = oracle.im2win(s, x)
    xp = F.pad(torch.from_numpy(x), (s.pw, s.pw, s.ph, s.ph)).numpy()
    for m in range(s.ho):
        strip = xp[:, :, m * s.sh:m * s.sh + s.fh, :]            # N x C x Fh x Wp
        np.testing.assert_array_equal(win[:, :, m, :], strip.transpose(0, 1, 3, 2).reshape(s.n, s.c, -1))


def test_im2win_worked_example_by_hand():
    """4x4 input numbered 0..15, 2x2 windows, stride 1: row m of the window
    tensor interleaves input rows m and m+1 column by column."""
    s = Shape(1, 1, 4, 4, 1, 2, 2)
    x = np.arange(16, dtype=np.float32).reshape(1, 1, 4, 4)
    win = oracle.im2win(s, x)[0, 0]
    for m in range(3):
        expect = [4 * (m + u) + k for k in range(4) for u in range(2)]
        np.testing.assert_array_equal(win[m], np.array(expect, dtype=np.float32))


def test_im2win_copies_bits():
    """bf16 (2-byte) and fp32 (4-byte) elements are copied bit for bit,
    including NaN payloads, infinities and negative zero; padding is +0."""
    s = Shape(1, 2, 5, 5, 1, 3, 3, 1, 1, 1, 1)
    bits32 = RNG.integers(0, 2**32, size=(1, 2, 5, 5), dtype=np.uint64).astype(np.uint32)
    bits32[0, 0, 0, :4] = [0x7FC00001, 0xFF800000, 0x80000000, 0x00000001]
    w32 = oracle.im2win(s, bits32)
    ref = oracle.im2win(s, bits32.view(np.float32)).view(np.uint32)
    np.testing.assert_array_equal(w32, ref)
    assert w32[0, 0, 0, 0] == 0 and w32[0, 0, 0, 4] == 0x7FC00001   # pad, then x[0][0]
    bits16 = RNG.integers(0, 2**16, size=(1, 2, 5, 5), dtype=np.uint64).astype(np.uint16)
    w16 = oracle.im2win(s, bits16)
    xp = np.pad(bits16, ((0, 0), (0, 0), (1, 1), (1, 1)))
    for m in range(s.ho):
        np.testing.assert_array_equal(w16[:, :, m, :],
                                      xp[:, :, m:m + 3, :].transpose(0, 1, 3, 2).reshape(1, 2, -1))


# --------------------------------------------------------------------------
# The convolution
# --------------------------------------------------------------------------

@pytest.mark.parametrize("s", SMALL_SHAPES, ids=_ids(SMALL_SHAPES))
def test_direct_conv_matches_torch_conv2d(s):
    x, w = _rand((s.n, s.c, s.h, s.w)), _rand((s.k, s.c, s.fh, s.fw))
    y = oracle.direct_conv(s, x, w)
    ref = F.conv2d(torch.from_numpy(x), torch.from_numpy(w), stride=(s.sh, s.sw),
                   padding=(s.ph, s.pw)).numpy()
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("s", SMALL_SHAPES, ids=_ids(SMALL_SHAPES))
def test_direct_conv_matches_im2col_gemm(s):
    """Sec. II-B: R' = M x N with the im2col matrix M and the filter matrix N,
    then R(j, m, n) = R'(m*Wo + n, j)."""
    x, w = _rand((s.n, s.c, s.h, s.w)), _rand((s.k, s.c, s.fh, s.fw))
    cols = oracle.im2col(s, x)                                   # N x HoWo x CFhFw
    unf = F.unfold(torch.from_numpy(x), (s.fh, s.fw), stride=(s.sh, s.sw),
                   padding=(s.ph, s.pw)).numpy()                 # N x CFhFw x HoWo
    np.testing.assert_array_equal(cols, unf.transpose(0, 2, 1))
    fmat = w.reshape(s.k, -1).T                                  # CFhFw x K
    r = np.stack([cols[i] @ fmat for i in range(s.n)])           # N x HoWo x K
    y = oracle.direct_conv(s, x, w)
    np.testing.assert_allclose(y, r.transpose(0, 2, 1).reshape(s.out_shape), rtol=0, atol=1e-12)


@pytest.mark.parametrize("s", SMALL_SHAPES, ids=_ids(SMALL_SHAPES))
def test_window_conv_of_im2win_equals_direct_conv(s):
    """Alg. 2 over the transformed tensor gives the direct convolution."""
    x, w = _rand((s.n, s.c, s.h, s.w)), _rand((s.k, s.c, s.fh, s.fw))
    win = oracle.im2win(s, x.astype(np.float64))
    np.testing.assert_allclose(oracle.window_conv(s, win, w), oracle.direct_conv(s, x, w),
                               rtol=0, atol=1e-12)


# --------------------------------------------------------------------------
# Trimmed rows: only the columns some window reads, (Wo-1)*sw + Fw of them
# --------------------------------------------------------------------------

# shapes whose padded rows hold columns no window reaches (the trimmed rows are
# shorter), beside ones where both widths agree
TRIM_SHAPES = SMALL_SHAPES + [
    Shape(2, 3, 12, 10, 2, 3, 2, 1, 3, 1, 1),         # Wo=4: Wt = 11 of Wp = 12
    Shape(1, 2, 9, 28, 3, 3, 5, 2, 2, 1, 2),          # rect-like: 31 of 32
    Shape(1, 2, 9, 17, 2, 2, 2, 1, 4, 0, 0),          # Fw < sw: 14 of 17
]


@pytest.mark.parametrize("s", TRIM_SHAPES, ids=_ids(TRIM_SHAPES))
def test_trimmed_width_is_the_last_window_end(s):
    """The trimmed row ends where the last window ends: the last output
    column's window covers padded columns [(Wo-1)*sw, (Wo-1)*sw + Fw), and the
    padded input has W + 2*pw >= that many columns (floor in Wo)."""
    last = max(n * s.sw + v for n in range(s.wo) for v in range(s.fw)) + 1
    assert s.wt == last <= s.wp
    assert oracle.im2win_elems(s, trimmed=True) == s.n * s.c * s.ho * last * s.fh


@pytest.mark.parametrize("s", TRIM_SHAPES, ids=_ids(TRIM_SHAPES))
def test_trimmed_windows_match_unfold(s):
    """Every window of the trimmed tensor equals the im2col column that torch's
    unfold builds, and every element of a trimmed row is the zero-padded input
    (no column is dropped that a window reads, none is added)."""
    x = _rand((s.n, s.c, s.h, s.w)).astype(np.float32)
    win = oracle.im2win(s, x, trimmed=True)
    assert win.shape == (s.n, s.c, s.ho, s.wt * s.fh)
    cols = F.unfold(torch.from_numpy(x), (s.fh, s.fw), stride=(s.sh, s.sw),
                    padding=(s.ph, s.pw)).numpy().reshape(s.n, s.c, s.fh, s.fw, s.ho, s.wo)
    for m in range(s.ho):
        for n in range(s.wo):
            for u in range(s.fh):
                for v in range(s.fw):
                    np.testing.assert_array_equal(win[:, :, m, (n * s.sw + v) * s.fh + u], cols[:, :, u, v, m, n])
    xp = F.pad(torch.from_numpy(x), (s.pw, s.pw, s.ph, s.ph)).numpy()
    for m in range(s.ho):
        strip = xp[:, :, m * s.sh:m * s.sh + s.fh, :s.wt]          # N x C x Fh x Wt
        np.testing.assert_array_equal(win[:, :, m, :], strip.transpose(0, 1, 3, 2).reshape(s.n, s.c, -1))


@pytest.mark.parametrize("s", TRIM_SHAPES, ids=_ids(TRIM_SHAPES))
def test_trimmed_window_conv_equals_conv2d(s):
    """Alg. 2 over the trimmed tensor gives torch's fp64 conv2d."""
    x, w = _rand((s.n, s.c, s.h, s.w)), _rand((s.k, s.c, s.fh, s.fw))
    win = oracle.im2win(s, x, trimmed=True)
    ref = F.conv2d(torch.from_numpy(x), torch.from_numpy(w), stride=(s.sh, s.sw), padding=(s.ph, s.pw)).numpy()
    np.testing.assert_allclose(oracle.window_conv(s, win, w, trimmed=True), ref, rtol=0, atol=1e-12)


def test_trimmed_size_never_exceeds_im2col_when_fw_at_least_sw():
    """im2col - trimmed = N*C*Fh*Ho*(Wo-1)*(Fw - sw): no larger than im2col
    whenever Fw >= sw (equal when Wo = 1 or Fw = sw), larger only when Fw < sw."""
    rng = np.random.default_rng(77)
    for _ in range(2000):
        fh, fw, sh, sw = (int(v) for v in rng.integers(1, 8, size=4))
        ph, pw = (int(v) for v in rng.integers(0, 4, size=2))
        h = int(rng.integers(max(1, fh - 2 * ph), 40))
        w = int(rng.integers(max(1, fw - 2 * pw), 60))
        s = Shape(int(rng.integers(1, 4)), int(rng.integers(1, 9)), h, w, 1, fh, fw, sh, sw, ph, pw)
        diff = oracle.im2col_elems(s) - oracle.im2win_elems(s, trimmed=True)
        assert diff == s.n * s.c * s.fh * s.ho * (s.wo - 1) * (s.fw - s.sw)
        if fw >= sw:
            assert diff >= 0
        assert oracle.im2win_elems(s, trimmed=True) <= oracle.im2win_elems(s)


def _literal_alg2(s, win, w):
    """Alg. 2 with the window offset exactly as printed, n*s*Wf + v*Hf + u."""
    y = np.zeros(s.out_shape)
    for m in range(s.ho):
        for n in range(s.wo):
            for u in range(s.fh):
                for v in range(s.fw):
                    a = win[:, :, m, n * s.sw * s.fw + v * s.fh + u]          # N x C
                    y[:, :, m, n] += a @ w[:, :, u, v].T
    return y


def test_printed_window_offset_only_holds_for_square_filters():
    """The offset n*s*Wf printed in Alg. 2 agrees with the direct convolution
    for square filters and not for rectangular ones; with n*s*Hf both agree."""
    sq = Shape(1, 2, 8, 8, 2, 3, 3, 1, 1)
    x, w = _rand((1, 2, 8, 8)), _rand((2, 2, 3, 3))
    np.testing.assert_allclose(_literal_alg2(sq, oracle.im2win(sq, x), w),
                               oracle.direct_conv(sq, x, w), atol=1e-12)
    rect = Shape(1, 2, 9, 12, 2, 3, 5, 1, 1)
    x, w = _rand((1, 2, 9, 12)), _rand((2, 2, 3, 5))
    win = oracle.im2win(rect, x)
    wide = np.zeros(win.shape[:3] + (win.shape[3] + 64,))
    wide[..., :win.shape[3]] = win                    # room for the overrun of the printed offset
    literal = _literal_alg2(rect, wide, w)
    assert np.abs(literal - oracle.direct_conv(rect, x, w)).max() > 1e-3
    np.testing.assert_allclose(oracle.window_conv(rect, win, w), oracle.direct_conv(rect, x, w), atol=1e-12)


def test_special_case_1x1_filter_is_channel_matmul():
    s = Shape(2, 5, 4, 6, 3, 1, 1)
    x, w = _rand((2, 5, 4, 6)), _rand((3, 5, 1, 1))
    ref = np.einsum("ichw,kc->ikhw", x, w[:, :, 0, 0])
    np.testing.assert_allclose(oracle.direct_conv(s, x, w), ref, atol=1e-12)


def test_special_case_full_filter_is_dot_product():
    s = Shape(2, 3, 4, 5, 2, 4, 5)
    x, w = _rand((2, 3, 4, 5)), _rand((2, 3, 4, 5))
    ref = np.einsum("ichw,kchw->ik", x, w).reshape(2, 2, 1, 1)
    np.testing.assert_allclose(oracle.direct_conv(s, x, w), ref, atol=1e-12)


def test_special_case_delta_filter_shifts_input():
    """A filter that is 1 at tap (u0, v0) of channel 0 and 0 elsewhere picks the
    input sample at (m*sh + u0 - ph, n*sw + v0 - pw)."""
    s = Shape(1, 2, 7, 9, 1, 3, 5, 2, 1, 1, 2)
    x = _rand((1, 2, 7, 9))
    xp = np.pad(x, ((0, 0), (0, 0), (1, 1), (2, 2)))
    for (u0, v0) in [(0, 0), (1, 3), (2, 4)]:
        w = np.zeros((1, 2, 3, 5))
        w[0, 0, u0, v0] = 1.0
        y = oracle.direct_conv(s, x, w)[0, 0]
        for m in range(s.ho):
            for n in range(s.wo):
                assert y[m, n] == xp[0, 0, m * 2 + u0, n * 1 + v0]


def test_abs_sum_and_points():
    s = Shape(2, 3, 9, 8, 4, 3, 5, 2, 1, 1, 2)
    x, w = _rand((2, 3, 9, 8)), _rand((4, 3, 3, 5))
    y, ya = oracle.direct_conv(s, x, w, with_abs=True)
    np.testing.assert_allclose(ya, oracle.direct_conv(s, np.abs(x), np.abs(w)), atol=1e-12)
    assert np.all(ya >= np.abs(y))
    idx = RNG.choice(y.size, size=50, replace=False)
    yp, yap = oracle.direct_conv_at(s, x, w, idx)
    np.testing.assert_array_equal(yp, y.reshape(-1)[idx])
    np.testing.assert_array_equal(yap, ya.reshape(-1)[idx])


def test_linearity():
    s = Shape(1, 3, 8, 8, 2, 3, 3, 1, 1, 1, 1)
    x1, x2, w = _rand((1, 3, 8, 8)), _rand((1, 3, 8, 8)), _rand((2, 3, 3, 3))
    np.testing.assert_allclose(oracle.direct_conv(s, 2.0 * x1 - x2, w),
                               2.0 * oracle.direct_conv(s, x1, w) - oracle.direct_conv(s, x2, w),
                               atol=1e-12)


def test_workload_shapes_fit_and_shrink_workspace():
    """On the five benchmark workloads the window tensor is smaller than the
    im2col matrix (the condition Wp <= Fw*Wo holds on each)."""
    import workloads
    for wl in workloads.WORKLOADS:
        s = Shape(wl.n, wl.c, wl.h, wl.w, wl.k, wl.fh, wl.fw, wl.sh, wl.sw, wl.ph, wl.pw)
        assert s.wp <= s.fw * s.wo
        assert oracle.im2win_elems(s) < oracle.im2col_elems(s)


def test_table1_workloads_are_the_printed_layers():
    """The Table 1 workloads that the sweep times and the GPU tests check are
    the printed layers (input, filter, stride, no padding) at the paper's batch."""
    import workloads
    t = json.load(open(os.path.join(GOLDEN, "table1.json")))
    assert len(workloads.TABLE1) == len(t["layers"])
    for wl, layer in zip(workloads.TABLE1, t["layers"]):
        assert [wl.c, wl.h, wl.w] == layer["input"], layer["name"]
        assert [wl.k, wl.fh, wl.fw] == layer["filter"], layer["name"]
        assert wl.sh == wl.sw == layer["stride"] and wl.ph == wl.pw == 0, layer["name"]
        assert wl.n == t["batch"] and wl.dtype == "f32"
