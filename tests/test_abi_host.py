"""Host-side tests of the C ABI (no GPU needed): the library loads and exports
every declared symbol, size queries agree with the oracle, invalid arguments
are rejected before any HIP call, and every launch plan stays in bounds."""
import ctypes
import glob
import os
import random
import re

import pytest

import oracle
from oracle import Shape
import workloads
import paper_2306_14320_amd as P
from conftest import ROOT

HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


def _desc(s: Shape, dtype=P.IM2WIN_F32):
    return P.im2win_desc(s.n, s.c, s.h, s.w, s.k, s.fh, s.fw, s.sh, s.sw, s.ph, s.pw, dtype)


def _wl_shape(wl):
    return Shape(wl.n, wl.c, wl.h, wl.w, wl.k, wl.fh, wl.fw, wl.sh, wl.sw, wl.ph, wl.pw)


def _wl_dtype(wl):
    return P.IM2WIN_F32 if wl.dtype == "f32" else P.IM2WIN_BF16


def test_library_exports_every_declared_symbol():
    text = "".join(open(h).read() for h in HEADERS)
    declared = set(re.findall(r"^\s*(?:int|const char\s*\*)\s*(im2win_\w+)\s*\(", text, re.M))
    assert {"im2win_workspace_bytes", "im2win_transform", "im2win_conv2d",
            "im2win_conv2d_fused", "im2win_last_error", "im2win_direct_conv2d"} <= declared
    lib = ctypes.CDLL(P.LIB_PATH)
    for name in sorted(declared):
        assert hasattr(lib, name), name


def test_fastdiv_selftest():
    assert P.im2win_selftest() == 0


SHAPES = [_wl_shape(wl) for wl in workloads.WORKLOADS] + [
    Shape(1, 1, 4, 4, 2, 2, 2), Shape(2, 3, 9, 11, 3, 3, 5, 2, 2, 1, 2),
    Shape(1, 2, 9, 9, 2, 2, 2, 3, 3), Shape(1, 1, 3, 3, 1, 3, 3, 1, 1, 2, 2),
    Shape(128, 3, 227, 227, 96, 11, 11, 4, 4),
]


@pytest.mark.parametrize("s", SHAPES, ids=str)
@pytest.mark.parametrize("dtype", [P.IM2WIN_F32, P.IM2WIN_BF16])
def test_sizes_agree_with_oracle(s, dtype):
    d = _desc(s, dtype)
    e = 4 if dtype == P.IM2WIN_F32 else 2
    assert P.im2win_output_shape(d) == (s.ho, s.wo)
    assert P.im2win_workspace_bytes(d) == oracle.im2win_elems(s) * e
    assert P.im2win_im2col_bytes(d) == oracle.im2col_elems(s) * e
    assert P.workspace_shape(d) == s.win_shape


def test_workspace_not_larger_than_im2col_on_workloads():
    for wl in workloads.WORKLOADS:
        d = _desc(_wl_shape(wl), _wl_dtype(wl))
        assert P.im2win_workspace_bytes(d) < P.im2win_im2col_bytes(d)


def _code(fn, *args):
    with pytest.raises(P.Im2winError) as ei:
        fn(*args)
    return ei.value.code


GOOD = Shape(2, 3, 8, 8, 4, 3, 3, 1, 1, 1, 1)
FAKE = 0x10000   # never dereferenced: every call below is rejected before any HIP call


@pytest.mark.parametrize("field,value", [
    ("n", 0), ("c", 0), ("h", -1), ("w", 0), ("k", 0), ("fh", 0), ("fw", 0),
    ("stride_h", 0), ("stride_w", -2), ("pad_h", -1), ("pad_w", -1), ("dtype", 7),
    ("fh", 11), ("fw", 11),  # filter larger than the padded input: Ho or Wo < 1
])
def test_invalid_descriptor_rejected(field, value):
    d = _desc(GOOD)
    setattr(d, field, value)
    assert _code(P.im2win_workspace_bytes, d) == P.IM2WIN_EINVAL
    assert _code(P.im2win_transform, d, FAKE, FAKE, 1 << 30, 0) == P.IM2WIN_EINVAL
    assert _code(P.im2win_conv2d, d, FAKE, 1 << 30, FAKE, FAKE, 1 << 30, FAKE, 0) == P.IM2WIN_EINVAL
    assert _code(P.im2win_conv2d_fused, d, FAKE, FAKE, FAKE, 1 << 30, FAKE, 0) == P.IM2WIN_EINVAL
    assert _code(P.im2win_direct_conv2d, d, FAKE, FAKE, FAKE, 0) == P.IM2WIN_EINVAL
    assert _code(P.im2win_filter_scratch_bytes, d) == P.IM2WIN_EINVAL
    assert _code(P.im2win_workspace_shape, d) == P.IM2WIN_EINVAL
    assert P.im2win_last_error() != ""


def test_null_misaligned_and_short_workspace_rejected():
    d = _desc(GOOD)
    need = P.im2win_workspace_bytes(d)
    assert _code(P.im2win_transform, d, 0, FAKE, need, 0) == P.IM2WIN_ENULL
    assert _code(P.im2win_transform, d, FAKE, 0, need, 0) == P.IM2WIN_ENULL
    assert _code(P.im2win_transform, d, FAKE + 4, FAKE, need, 0) == P.IM2WIN_EALIGN
    assert _code(P.im2win_transform, d, FAKE, FAKE, need - 1, 0) == P.IM2WIN_EWORKSPACE
    sb = 1 << 20
    assert _code(P.im2win_conv2d, d, FAKE, need - 4, FAKE, FAKE, sb, FAKE, 0) == P.IM2WIN_EWORKSPACE
    assert _code(P.im2win_conv2d, d, FAKE, need, 0, FAKE, sb, FAKE, 0) == P.IM2WIN_ENULL
    assert _code(P.im2win_conv2d, d, FAKE, need, FAKE, FAKE, sb, FAKE + 8, 0) == P.IM2WIN_EALIGN
    assert _code(P.im2win_conv2d_fused, d, FAKE, FAKE, FAKE, sb, 0, 0) == P.IM2WIN_ENULL
    assert _code(P.im2win_conv2d_fused, d, FAKE, FAKE + 2, FAKE, sb, FAKE, 0) == P.IM2WIN_EALIGN
    for i in range(3):   # the direct baseline checks nulls (its pointers need no 16-byte alignment)
        args = [FAKE, FAKE, FAKE]
        args[i] = 0
        assert _code(P.im2win_direct_conv2d, d, *args, 0) == P.IM2WIN_ENULL
    lib = P.load_library()
    assert lib.im2win_workspace_bytes(None, None) == P.IM2WIN_ENULL
    assert lib.im2win_workspace_bytes(ctypes.byref(d), None) == P.IM2WIN_ENULL


def test_oversized_problem_rejected():
    d = _desc(Shape(1 << 20, 4, 1024, 1024, 4, 3, 3, 1, 1, 1, 1))   # N*Ho*Wo >= 2^31
    assert _code(P.im2win_workspace_bytes, d) == P.IM2WIN_EOVERFLOW
    assert _code(P.im2win_conv2d_fused, d, FAKE, FAKE, FAKE, 1 << 30, FAKE, 0) == P.IM2WIN_EOVERFLOW
    assert _code(P.im2win_direct_conv2d, d, FAKE, FAKE, FAKE, 0) == P.IM2WIN_EOVERFLOW


@pytest.mark.parametrize("layout", [P.IM2WIN_ROWS_PADDED, P.IM2WIN_ROWS_TRIMMED], ids=["padded", "trimmed"])
@pytest.mark.parametrize("wl", workloads.WORKLOADS, ids=lambda wl: wl.name)
def test_launch_plans_in_bounds_on_workloads(wl, layout):
    d = _desc(_wl_shape(wl), _wl_dtype(wl))
    d.layout = layout
    assert P.im2win_check_plan(d) == 0, P.im2win_last_error()


@pytest.mark.parametrize("s", SHAPES, ids=str)
@pytest.mark.parametrize("dtype", [P.IM2WIN_F32, P.IM2WIN_BF16])
def test_trimmed_sizes_agree_with_oracle(s, dtype):
    d = _desc(s, dtype)
    d.layout = P.IM2WIN_ROWS_TRIMMED
    e = 4 if dtype == P.IM2WIN_F32 else 2
    assert P.im2win_workspace_bytes(d) == oracle.im2win_elems(s, trimmed=True) * e
    assert P.workspace_shape(d) == s.win_shape_of(True)
    assert P.im2win_output_shape(d) == (s.ho, s.wo)


def test_unknown_layout_rejected():
    d = _desc(GOOD)
    d.layout = 2
    assert _code(P.im2win_workspace_bytes, d) == P.IM2WIN_EINVAL
    assert _code(P.im2win_conv2d_fused, d, FAKE, FAKE, FAKE, 1 << 30, FAKE, 0) == P.IM2WIN_EINVAL
    assert "layout" in P.im2win_last_error()


def test_launch_plans_in_bounds_on_random_shapes():
    rng = random.Random(14320)
    checked = 0
    while checked < 600:
        n, c, h, w = rng.randint(1, 4), rng.randint(1, 40), rng.randint(1, 40), rng.randint(1, 64)
        k, fh, fw = rng.randint(1, 140), rng.randint(1, 9), rng.randint(1, 9)
        sh, sw, ph, pw = rng.randint(1, 4), rng.randint(1, 4), rng.randint(0, 4), rng.randint(0, 4)
        if h + 2 * ph < fh or w + 2 * pw < fw:
            continue
        for dt in (P.IM2WIN_F32, P.IM2WIN_BF16):
            d = P.im2win_desc(n, c, h, w, k, fh, fw, sh, sw, ph, pw, dt, checked % 2)
            assert P.im2win_check_plan(d) == 0, (d, P.im2win_last_error())
            checked += 1


def test_launch_plans_in_bounds_on_paper_layers():
    """Table 1 layers at batch 2 (the plan depends on the batch only through
    the number of tiles)."""
    import json
    from conftest import GOLDEN
    t = json.load(open(os.path.join(GOLDEN, "table1.json")))
    for layer in t["layers"]:
        ci, hi, wi = layer["input"]
        co, hf, wf = layer["filter"]
        st = layer["stride"]
        for dt in (P.IM2WIN_F32, P.IM2WIN_BF16):
            for layout in (P.IM2WIN_ROWS_PADDED, P.IM2WIN_ROWS_TRIMMED):
                d = P.im2win_desc(2, ci, hi, wi, co, hf, wf, st, st, 0, 0, dt, layout)
                assert P.im2win_check_plan(d) == 0, (layer["name"], P.im2win_last_error())


# Shapes that the fp32 band kernel takes (n, c, h, w, k, fh, fw, sh, sw, ph,
# pw): C a multiple of 16, K of 32 (64 with the two-way reduction split), a
# band of output rows of 97-224 pixels (four-way split) or 353-416 (two-way),
# or of several whole images of fewer pixels, at most 4 rounds of 256
# workgroups with at least 85% of them useful.
F32_BANDS = [
    (64, 128, 28, 28, 128, 3, 5, 2, 2, 1, 2),   # the rectangular-window layer: whole images
    (128, 512, 7, 7, 512, 3, 3, 1, 1, 0, 0),    # Table 1 Conv12: bands of 8 images of 25 pixels
    (128, 256, 12, 12, 512, 3, 3, 1, 1, 0, 0),  # Table 1 Conv6: bands of 4 images of 100 pixels
    (124, 16, 7, 7, 512, 3, 3, 1, 1, 0, 0),     # several images, the last band of 4
    (126, 16, 12, 12, 512, 3, 3, 1, 1, 0, 0),   # several images, the last band of 2
    (128, 16, 5, 5, 512, 3, 3, 1, 1, 1, 1),     # several padded images
    (128, 16, 7, 9, 512, 3, 5, 1, 1, 0, 0),     # several images, 3x5
    (127, 16, 14, 14, 256, 3, 3, 1, 1, 0, 0),   # two-way split, 2 images of 144 pixels, the last band of 1
    (128, 64, 112, 112, 128, 3, 3, 1, 1, 0, 0), # Table 1 Conv8: 4-row bands in 14 blocks, 28 rounds of long work
    (9, 16, 112, 112, 128, 3, 3, 1, 1, 0, 0),
    (128, 96, 24, 24, 256, 5, 5, 1, 1, 0, 0),   # Table 1 Conv5: 5x5, 11-row bands, 8 rounds of long work
    (16, 16, 20, 20, 256, 5, 5, 1, 1, 2, 2),
    (32, 64, 56, 56, 64, 3, 3, 1, 1, 1, 1),     # the ResNet-style layer: 7-row bands, two-way split
    (128, 64, 56, 56, 64, 3, 3, 1, 1, 0, 0),    # Table 1 Conv9: ragged last band
    (128, 128, 28, 28, 128, 3, 3, 1, 1, 0, 0),  # Table 1 Conv10
    (128, 256, 14, 14, 256, 3, 3, 1, 1, 0, 0),  # Table 1 Conv11
    (2, 16, 28, 28, 4096, 3, 5, 2, 2, 1, 2),
    (8, 32, 14, 14, 1024, 3, 3, 1, 1, 1, 1),
    (16, 16, 13, 13, 512, 3, 3, 1, 1, 0, 0),
    (4, 16, 13, 23, 2048, 3, 5, 1, 2, 0, 1),
    (3, 32, 29, 15, 2720, 3, 3, 2, 1, 1, 0),
    (16, 16, 28, 28, 512, 3, 3, 1, 1, 1, 1),
    (2, 16, 56, 56, 1024, 3, 3, 1, 1, 1, 1),
    (8, 16, 28, 28, 1024, 3, 3, 1, 1, 0, 0),
    (8, 16, 55, 55, 1024, 3, 3, 2, 2, 1, 1),
    (8, 16, 52, 52, 1024, 3, 3, 2, 2, 1, 1),     # fused from raw rows, stride 2
    (4, 16, 112, 112, 512, 3, 3, 2, 2, 1, 1),
    (2, 16, 28, 32, 4096, 3, 5, 2, 2, 1, 4),     # raw rows with 8 zero columns in front
]


# Shapes that the fp32 small-C band kernel takes: C = 3, 7x7 filters, K a
# multiple of 64, bands of 97-224 pixels, at least 75% of the occupied
# matrix-core work useful.
F32_BANDS_SMALL_C = [
    (32, 3, 224, 224, 64, 7, 7, 2, 2, 3, 3),    # the stem layer: bands of 2 rows
    (128, 3, 227, 227, 64, 7, 7, 2, 2, 0, 0),   # Table 1 Conv3
    (4, 3, 64, 64, 512, 7, 7, 2, 2, 3, 3),
    (8, 3, 70, 70, 64, 7, 7, 1, 1, 0, 0),
    (2, 3, 48, 48, 512, 7, 7, 1, 1, 0, 0),      # ragged last band
    (128, 3, 224, 224, 64, 3, 3, 1, 1, 0, 0),   # Table 1 Conv7: one row per band, y past 1 GiB
    (1, 3, 62, 62, 512, 3, 3, 1, 1, 1, 1),
    (4, 3, 63, 63, 512, 3, 3, 2, 2, 0, 0),
    (16, 3, 59, 59, 512, 11, 11, 4, 4, 2, 2),   # 11x11 stride 4, rows not whole 16-byte vectors
    (1, 3, 56, 56, 512, 11, 11, 1, 1, 5, 5),
    (128, 3, 227, 227, 96, 11, 11, 4, 4, 0, 0),   # Table 1 Conv1: K = 96, the last group's second block idle
    (128, 3, 231, 231, 96, 11, 11, 4, 4, 0, 0),   # Table 1 Conv2
    (4, 3, 64, 64, 96, 3, 3, 1, 1, 1, 1),
    (8, 3, 83, 83, 96, 7, 7, 2, 2, 3, 3),
    (16, 3, 45, 45, 160, 7, 7, 2, 2, 3, 3),
]


@pytest.mark.parametrize("layout", [0, 1], ids=["padded", "trimmed"])
@pytest.mark.parametrize("case", F32_BANDS_SMALL_C, ids=lambda c: "x".join(map(str, c)))
def test_launch_plans_in_bounds_fp32_bands_small_c(case, layout):
    d = P.im2win_desc(*case, P.IM2WIN_F32, layout)
    assert P.im2win_conv_kernel(d, False) == P.im2win_conv_kernel(d, True) == "f32_bands_small_c"
    assert P.im2win_filter_scratch_bytes(d) == 0
    assert P.im2win_check_plan(d) == 0, P.im2win_last_error()


def test_conv_kernel_names_on_workloads():
    got = {}
    for wl in workloads.WORKLOADS:
        d = _desc(_wl_shape(wl), _wl_dtype(wl))
        got[wl.name] = (P.im2win_conv_kernel(d, False), P.im2win_conv_kernel(d, True))
    assert got["rect_3x5_s2_f32"] == ("f32_bands",) * 2
    assert got["resnet_3x3_f32"] == ("f32_bands",) * 2
    assert got["deep_3x3_bf16"] == ("bf16_one_image",) * 2
    assert got["stem_7x7_s2_f32"] == ("f32_bands_small_c",) * 2
    d = P.im2win_desc(1, 3, 4000, 4000, 4, 60, 60, 1, 1, 0, 0, P.IM2WIN_F32)
    assert P.im2win_conv_kernel(d, False) == "per_output"


def test_conv_kernel_names_on_table1():
    """The kernel family each of the paper's twelve layers takes at batch
    128, both variants alike: three-channel layers on the persistent kernel,
    Conv4 (7x7, rows longer than a band slot) on the tiles, the rest on bands
    (Conv6, Conv11, Conv12 as bands of several whole images)."""
    want = {1: "f32_bands_small_c", 2: "f32_bands_small_c", 3: "f32_bands_small_c", 4: "f32_tiles",
            5: "f32_bands", 6: "f32_bands", 7: "f32_bands_small_c", 8: "f32_bands", 9: "f32_bands",
            10: "f32_bands", 11: "f32_bands", 12: "f32_bands"}
    assert len(workloads.TABLE1) == 12
    for i, wl in enumerate(workloads.TABLE1, start=1):
        d = _desc(_wl_shape(wl), P.IM2WIN_F32)
        assert (P.im2win_conv_kernel(d, False), P.im2win_conv_kernel(d, True)) == (want[i],) * 2, wl.name
        # the band kernels read w as it is; Conv4's tiles take repacked filter blocks
        assert (P.im2win_filter_scratch_bytes(d) > 0) == (want[i] == "f32_tiles"), wl.name


@pytest.mark.parametrize("layout", [0, 1], ids=["padded", "trimmed"])
@pytest.mark.parametrize("case", F32_BANDS, ids=lambda c: "x".join(map(str, c)))
def test_launch_plans_in_bounds_fp32_bands(case, layout):
    """The band kernel takes these shapes in both row layouts (and only for
    fp32), and its replayed staging copies, window reads and stores are in
    bounds and hold what Alg. 2 sums."""
    d = P.im2win_desc(*case, P.IM2WIN_F32, layout)
    assert P.im2win_conv_kernel(d, False) == "f32_bands"
    assert P.im2win_conv_kernel(d, True) == "f32_bands"
    assert P.im2win_filter_scratch_bytes(d) == 0
    assert P.im2win_check_plan(d) == 0, P.im2win_last_error()
    assert P.im2win_conv_kernel(P.im2win_desc(*case, P.IM2WIN_BF16, layout), False) != "f32_bands"


def test_fp32_bands_decline_unsupported_shapes():
    base = list(F32_BANDS[0])
    def name(**kw):
        c = dict(zip("n c h w k fh fw sh sw ph pw".split(), base))
        c.update(kw)
        return P.im2win_conv_kernel(P.im2win_desc(*c.values(), P.IM2WIN_F32), False)
    assert name() == "f32_bands"
    assert name(n=56) != "f32_bands"            # 224 workgroups: 77% of one round
    assert name(n=1100, c=16) != "f32_bands"    # more than 4 rounds of short work per workgroup
    assert name(n=1088) == "f32_bands"          # 17 rounds of long work (13.8M multiply-adds each)
    assert name(c=120) != "f32_bands"           # C not a multiple of 16
    assert name(k=112) != "f32_bands"           # K not a multiple of 32
    assert name(fh=5, fw=3, ph=2, pw=1) != "f32_bands"   # 5x3 filter (5x5 is taken: Conv5 above)
    assert name(h=12, w=12, ph=0, pw=0) != "f32_bands"   # 5x4 = 20 pixels


# ---------------------------------------------------------------------------
# Filter scratch (the repacked filter lives in a caller-owned buffer)
# ---------------------------------------------------------------------------

def test_filter_scratch_sizes_on_workloads():
    """Which workloads repack the filter, and how large the scratch is: bf16
    fast kernels take K*C*Fh*Fw*2 bytes exactly; fp32 tile kernels whose
    chunk rows are not whole 16-byte vectors (C*Fh*Fw odd: the single-image
    layer, and the stem layer at a batch the band kernel does not take) take
    padded blocks of about K*C*Fh*Fw*4 bytes; the band kernels none."""
    got = {}
    for wl in workloads.WORKLOADS:
        d = _desc(_wl_shape(wl), _wl_dtype(wl))
        got[wl.name] = P.im2win_filter_scratch_bytes(d)
    kcft = {wl.name: wl.k * wl.c * wl.fh * wl.fw for wl in workloads.WORKLOADS}
    assert got["deep_3x3_bf16"] == kcft["deep_3x3_bf16"] * 2
    assert got["resnet_3x3_f32"] == 0 and got["rect_3x5_s2_f32"] == 0 and got["stem_7x7_s2_f32"] == 0
    name = "single_3x3_f32"
    assert kcft[name] * 4 <= got[name] <= 2 * kcft[name] * 4 + (1 << 16), (name, got[name])
    st = workloads.BY_NAME["stem_7x7_s2_f32"]
    stem1 = P.im2win_desc(1, st.c, st.h, st.w, st.k, st.fh, st.fw, st.sh, st.sw, st.ph, st.pw, P.IM2WIN_F32)
    assert P.im2win_conv_kernel(stem1, False) == "f32_tiles"
    assert kcft["stem_7x7_s2_f32"] * 4 <= P.im2win_filter_scratch_bytes(stem1) <= 2 * kcft["stem_7x7_s2_f32"] * 4 + (1 << 16)


def test_short_or_missing_scratch_rejected():
    wl = workloads.BY_NAME["deep_3x3_bf16"]
    d = _desc(_wl_shape(wl), _wl_dtype(wl))
    need_ws = P.im2win_workspace_bytes(d)
    need = P.im2win_filter_scratch_bytes(d)
    assert need > 0
    assert _code(P.im2win_conv2d, d, FAKE, need_ws, FAKE, FAKE, need - 16, FAKE, 0) == P.IM2WIN_EWORKSPACE
    assert "scratch" in P.im2win_last_error()
    assert _code(P.im2win_conv2d_fused, d, FAKE, FAKE, FAKE, need - 16, FAKE, 0) == P.IM2WIN_EWORKSPACE
    assert _code(P.im2win_conv2d, d, FAKE, need_ws, FAKE, 0, need, FAKE, 0) == P.IM2WIN_ENULL
    assert _code(P.im2win_conv2d_fused, d, FAKE, FAKE, FAKE + 4, need, FAKE, 0) == P.IM2WIN_EALIGN


@pytest.mark.parametrize("s", SHAPES, ids=str)
@pytest.mark.parametrize("dtype", [P.IM2WIN_F32, P.IM2WIN_BF16])
def test_workspace_shape_query(s, dtype):
    d = _desc(s, dtype)
    n, c, ho, row = P.im2win_workspace_shape(d)
    e = 4 if dtype == P.IM2WIN_F32 else 2
    assert (n, c, ho) == (s.n, s.c, s.ho)
    assert n * c * ho * row * e == P.im2win_workspace_bytes(d)
    assert (n, c, ho, row) == s.win_shape


# Shapes whose window strips fit no LDS tile (long rows, few output columns):
# they run on the per-output kernel, which needs no plan and no scratch.
NO_TILE = [Shape(1, 2, 3, 4096, 3, 3, 4096, 1, 1, 0, 0), Shape(2, 1, 5, 20000, 2, 5, 19000, 1, 7, 0, 0)]


@pytest.mark.parametrize("s", NO_TILE, ids=str)
@pytest.mark.parametrize("dtype", [P.IM2WIN_F32, P.IM2WIN_BF16])
def test_shapes_without_a_tile_take_the_plain_kernel(s, dtype):
    d = _desc(s, dtype)
    assert P.im2win_filter_scratch_bytes(d) == 0
    assert P.im2win_check_plan(d) == 0, P.im2win_last_error()


def test_binding_rejects_mismatched_tensors():
    """The tensor helpers check shapes and dtypes before any C call (the C
    ABI takes no tensor sizes)."""
    import torch
    d = P.desc_for((2, 3, 8, 8), (4, 3, 3, 3), 1, 1)
    x = torch.zeros(2, 3, 8, 8)           # a host tensor: refused as not on the device
    with pytest.raises(ValueError):
        P.conv2d_fused(x, torch.zeros(4, 3, 3, 3), d)


def test_one_hip_runtime_mapped():
    """libim2win binds to the HIP runtime torch loaded, not to a second copy."""
    P.load_library()
    maps = P.hip_runtimes_mapped()
    assert len(maps) == 1, maps


def test_noalloc_entry_point_rejects_scratch_beyond_its_array():
    """im2win_conv2d_fused_noalloc keeps the repacked filter in a static
    device array of IM2WIN_NOALLOC_SCRATCH_BYTES; a filter that needs more is
    refused on the host (EWORKSPACE) before any HIP call."""
    d = P.im2win_desc(2, 1024, 14, 14, 1024, 3, 3, 1, 1, 1, 1, P.IM2WIN_BF16)
    assert P.im2win_filter_scratch_bytes(d) > P.IM2WIN_NOALLOC_SCRATCH_BYTES
    assert _code(P.im2win_conv2d_fused_noalloc, d, FAKE, FAKE, FAKE, 0) == P.IM2WIN_EWORKSPACE
    assert "static" in P.im2win_last_error()
    bad = _desc(GOOD)
    bad.k = 0
    assert _code(P.im2win_conv2d_fused_noalloc, bad, FAKE, FAKE, FAKE, 0) == P.IM2WIN_EINVAL
    assert _code(P.im2win_conv2d_fused_noalloc, _desc(GOOD), FAKE, FAKE, FAKE + 4, 0) == P.IM2WIN_EALIGN
