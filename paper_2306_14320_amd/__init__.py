"""MI355X (gfx950) im2win transformation and im2win-based convolution.

Python binding of ``libim2win.so`` (C ABI in ``include/im2win.h``).  The
functions named ``im2win_*`` mirror the C entry points one to one and only
marshal arguments; every step of the computation runs in the HIP kernels.
The tensor helpers below them (``desc_for``, ``transform``, ``conv2d``,
``conv2d_fused``) check that the tensors match the descriptor and use PyTorch
only to allocate device memory (window tensor, filter scratch, output) on the
call's HIP stream.

There is no fallback: if the library is missing or was built for another
target, loading fails with an error.  Build it with
``python -m paper_2306_14320_amd.build``.

Method: Lu, Chu, Liu, "Im2win: Memory Efficient Convolution On SIMD
Architectures", arXiv 2306.14320 (Sec. III, Alg. 1 and Alg. 2).
"""
import ctypes
import os

import torch  # imported first: libim2win then binds to the HIP runtime torch has loaded

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libim2win.so")

IM2WIN_F32, IM2WIN_BF16 = 0, 1
IM2WIN_ROWS_PADDED, IM2WIN_ROWS_TRIMMED = 0, 1   # im2win_layout
IM2WIN_OK = 0
IM2WIN_EINVAL = -1
IM2WIN_ENULL = -2
IM2WIN_EWORKSPACE = -3
IM2WIN_EHIP = -4
IM2WIN_EOVERFLOW = -5
IM2WIN_EALIGN = -6
IM2WIN_NOALLOC_SCRATCH_BYTES = 8 << 20


class im2win_desc(ctypes.Structure):
    """Mirror of the C ``im2win_desc``."""
    _fields_ = [
        ("n", ctypes.c_int64), ("c", ctypes.c_int64), ("h", ctypes.c_int64), ("w", ctypes.c_int64),
        ("k", ctypes.c_int64), ("fh", ctypes.c_int64), ("fw", ctypes.c_int64),
        ("stride_h", ctypes.c_int64), ("stride_w", ctypes.c_int64),
        ("pad_h", ctypes.c_int64), ("pad_w", ctypes.c_int64),
        ("dtype", ctypes.c_int32), ("layout", ctypes.c_int32),
    ]

    def __repr__(self):
        return ("im2win_desc(n=%d, c=%d, h=%d, w=%d, k=%d, fh=%d, fw=%d, stride=(%d,%d), "
                "pad=(%d,%d), dtype=%d, layout=%d)" % (self.n, self.c, self.h, self.w, self.k, self.fh,
                                                       self.fw, self.stride_h, self.stride_w, self.pad_h,
                                                       self.pad_w, self.dtype, self.layout))


class Im2winError(RuntimeError):
    def __init__(self, code, message):
        super().__init__(f"im2win error {code}: {message}")
        self.code = code


_lib = None


def load_library():
    """Load libim2win.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2306_14320_amd.build` (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    runtimes = hip_runtimes_mapped()
    if len(runtimes) > 1:
        raise RuntimeError("libim2win bound a second HIP runtime next to torch's: " + ", ".join(runtimes))
    P, D, SZ, I64P = ctypes.c_void_p, ctypes.POINTER(im2win_desc), ctypes.c_size_t, ctypes.POINTER(ctypes.c_int64)
    sigs = {
        "im2win_workspace_bytes": [D, ctypes.POINTER(SZ)],
        "im2win_im2col_bytes": [D, ctypes.POINTER(SZ)],
        "im2win_output_shape": [D, I64P, I64P],
        "im2win_workspace_shape": [D, I64P],
        "im2win_filter_scratch_bytes": [D, ctypes.POINTER(SZ)],
        "im2win_conv_kernel": [D, ctypes.c_int, ctypes.POINTER(ctypes.c_char_p)],
        "im2win_transform": [D, P, P, SZ, P],
        "im2win_conv2d": [D, P, SZ, P, P, SZ, P, P],
        "im2win_conv2d_fused": [D, P, P, P, SZ, P, P],
        "im2win_direct_conv2d": [D, P, P, P, P],
        "im2win_conv2d_fused_noalloc": [D, P, P, P, P],
        "im2win_selftest": [],
        "im2win_check_plan": [D],
    }
    for name, args in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.im2win_last_error.argtypes = []
    lib.im2win_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def hip_runtimes_mapped():
    """Distinct HIP runtime libraries (libamdhip64) mapped into this process.
    libim2win must bind to the one torch loaded (it is imported first), never
    to a second copy with its own device state."""
    try:
        with open("/proc/self/maps") as f:
            return sorted({l.split()[-1] for l in f if "libamdhip64" in l})
    except OSError:
        return []


def _check(rc):
    if rc != IM2WIN_OK:
        raise Im2winError(rc, im2win_last_error())


# ---------------------------------------------------------------------------
# C entry points, same names and arguments (raising Im2winError on failure)
# ---------------------------------------------------------------------------

def im2win_workspace_bytes(desc: im2win_desc) -> int:
    out = ctypes.c_size_t()
    _check(load_library().im2win_workspace_bytes(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def im2win_im2col_bytes(desc: im2win_desc) -> int:
    out = ctypes.c_size_t()
    _check(load_library().im2win_im2col_bytes(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def im2win_output_shape(desc: im2win_desc):
    ho, wo = ctypes.c_int64(), ctypes.c_int64()
    _check(load_library().im2win_output_shape(ctypes.byref(desc), ctypes.byref(ho), ctypes.byref(wo)))
    return ho.value, wo.value


def im2win_workspace_shape(desc: im2win_desc):
    dims = (ctypes.c_int64 * 4)()
    _check(load_library().im2win_workspace_shape(ctypes.byref(desc), dims))
    return tuple(dims)


def im2win_filter_scratch_bytes(desc: im2win_desc) -> int:
    out = ctypes.c_size_t()
    _check(load_library().im2win_filter_scratch_bytes(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def im2win_conv_kernel(desc: im2win_desc, fused: bool) -> str:
    """Name of the kernel im2win_conv2d (fused False) or im2win_conv2d_fused
    (fused True) launches for desc."""
    out = ctypes.c_char_p()
    _check(load_library().im2win_conv_kernel(ctypes.byref(desc), int(bool(fused)), ctypes.byref(out)))
    return out.value.decode()


def im2win_transform(desc: im2win_desc, x: int, ws: int, ws_bytes: int, stream: int) -> None:
    _check(load_library().im2win_transform(ctypes.byref(desc), x, ws, ws_bytes, stream))


def im2win_conv2d(desc: im2win_desc, ws: int, ws_bytes: int, w: int, scratch: int,
                  scratch_bytes: int, y: int, stream: int) -> None:
    _check(load_library().im2win_conv2d(ctypes.byref(desc), ws, ws_bytes, w, scratch, scratch_bytes,
                                        y, stream))


def im2win_conv2d_fused(desc: im2win_desc, x: int, w: int, scratch: int, scratch_bytes: int,
                        y: int, stream: int) -> None:
    _check(load_library().im2win_conv2d_fused(ctypes.byref(desc), x, w, scratch, scratch_bytes, y,
                                              stream))


def im2win_conv2d_fused_noalloc(desc: im2win_desc, x: int, w: int, y: int, stream: int) -> None:
    _check(load_library().im2win_conv2d_fused_noalloc(ctypes.byref(desc), x, w, y, stream))


def im2win_direct_conv2d(desc: im2win_desc, x: int, w: int, y: int, stream: int) -> None:
    """Comparison baseline (include/im2win_baseline.h): direct convolution, no transformation."""
    _check(load_library().im2win_direct_conv2d(ctypes.byref(desc), x, w, y, stream))


def im2win_last_error() -> str:
    return load_library().im2win_last_error().decode()


def im2win_selftest() -> int:
    return load_library().im2win_selftest()


def im2win_check_plan(desc: im2win_desc) -> int:
    """0 if every kernel index for this descriptor stays in bounds, else the
    number of violations (the first is in im2win_last_error())."""
    return load_library().im2win_check_plan(ctypes.byref(desc))


# ---------------------------------------------------------------------------
# Tensor helpers (marshalling: shapes -> descriptor, tensors -> pointers)
# ---------------------------------------------------------------------------

_DTYPES = {torch.float32: IM2WIN_F32, torch.bfloat16: IM2WIN_BF16}


def _pair(v):
    return (v, v) if isinstance(v, int) else tuple(v)


def desc_for(x_shape, w_shape, stride=1, padding=0, dtype=torch.float32,
             layout=None) -> im2win_desc:
    """Descriptor for input N x C x H x W, filter K x C x Fh x Fw (window-tensor
    rows of the padded width unless layout=IM2WIN_ROWS_TRIMMED)."""
    n, c, h, w = x_shape
    k, c2, fh, fw = w_shape
    if c2 != c:
        raise ValueError(f"filter has {c2} input channels, input has {c}")
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    if dtype not in _DTYPES:
        raise ValueError(f"unsupported dtype {dtype} (float32 or bfloat16)")
    return im2win_desc(n, c, h, w, k, fh, fw, sh, sw, ph, pw, _DTYPES[dtype],
                       IM2WIN_ROWS_PADDED if layout is None else layout)


def _torch_stream(stream):
    """The torch stream a call runs on (the current one when None)."""
    if stream is None:
        return torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream))


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dev(t, name, shape=None, dtype=None):
    """Device pointer of t, after checking that it is a contiguous device
    tensor of the given shape and dtype (the C ABI receives no tensor sizes,
    so a mismatch here would make the kernels read or write out of bounds)."""
    if not isinstance(t, torch.Tensor) or not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous device tensor")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, the descriptor needs {tuple(shape)}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, the descriptor needs {dtype}")
    return t.data_ptr()


def _dtype_of(desc):
    return torch.float32 if desc.dtype == IM2WIN_F32 else torch.bfloat16


def x_shape(desc: im2win_desc):
    return (desc.n, desc.c, desc.h, desc.w)


def w_shape(desc: im2win_desc):
    return (desc.k, desc.c, desc.fh, desc.fw)


def y_shape(desc: im2win_desc):
    ho, wo = im2win_output_shape(desc)
    return (desc.n, desc.k, ho, wo)


def workspace_shape(desc: im2win_desc):
    """N x C x Ho x Wr*Fh (im2win_workspace_shape)."""
    return im2win_workspace_shape(desc)


def _empty(shape, dtype, device, stream):
    """torch.empty on the call's stream (the current one when stream is None)."""
    if stream is None:
        return torch.empty(shape, dtype=dtype, device=device)
    with torch.cuda.stream(_torch_stream(stream)):
        return torch.empty(shape, dtype=dtype, device=device)


def filter_scratch(desc: im2win_desc, device, stream=None, nbytes=None) -> torch.Tensor:
    """A device buffer of im2win_filter_scratch_bytes() bytes (at least 16),
    allocated on the call's stream."""
    if nbytes is None:
        nbytes = im2win_filter_scratch_bytes(desc)
    return _empty(max(nbytes, 16), torch.uint8, device, stream)


def _scratch_args(desc, scratch, device, stream):
    if scratch is None:
        need = im2win_filter_scratch_bytes(desc)
        if need == 0:
            return None, 0, 0
        scratch = filter_scratch(desc, device, stream, need)
    p = _dev(scratch, "scratch")
    return scratch, p, scratch.numel() * scratch.element_size()


def transform(x: torch.Tensor, desc: im2win_desc, ws: torch.Tensor = None, stream=None) -> torch.Tensor:
    """Window tensor of x (N x C x Ho x Wr*Fh, dtype of x)."""
    xp = _dev(x, "x", x_shape(desc), _dtype_of(desc))
    if ws is None:
        ws = _empty(workspace_shape(desc), x.dtype, x.device, stream)
    im2win_transform(desc, xp, _dev(ws, "ws", dtype=_dtype_of(desc)), ws.numel() * ws.element_size(),
                     _stream(stream))
    return ws


def _output(y, desc, device, stream):
    shape = y_shape(desc)
    if y is None:
        y = _empty(shape, torch.float32, device, stream)
    return y, _dev(y, "y", shape, torch.float32)


def conv2d(ws: torch.Tensor, w: torch.Tensor, desc: im2win_desc, y: torch.Tensor = None,
           stream=None, scratch: torch.Tensor = None) -> torch.Tensor:
    """Convolution from a window tensor; returns y (N x K x Ho x Wo, fp32).
    `scratch` is the filter scratch (allocated per call when None)."""
    wsp = _dev(ws, "ws", dtype=_dtype_of(desc))
    wp = _dev(w, "w", w_shape(desc), _dtype_of(desc))
    y, yp = _output(y, desc, ws.device, stream)
    scratch, sp, sbytes = _scratch_args(desc, scratch, ws.device, stream)
    im2win_conv2d(desc, wsp, ws.numel() * ws.element_size(), wp, sp, sbytes, yp, _stream(stream))
    return y


def conv2d_fused(x: torch.Tensor, w: torch.Tensor, desc: im2win_desc, y: torch.Tensor = None,
                 stream=None, scratch: torch.Tensor = None) -> torch.Tensor:
    """Convolution straight from x (window strips built on chip); returns y."""
    xp = _dev(x, "x", x_shape(desc), _dtype_of(desc))
    wp = _dev(w, "w", w_shape(desc), _dtype_of(desc))
    y, yp = _output(y, desc, x.device, stream)
    scratch, sp, sbytes = _scratch_args(desc, scratch, x.device, stream)
    im2win_conv2d_fused(desc, xp, wp, sp, sbytes, yp, _stream(stream))
    return y


def direct_conv2d(x: torch.Tensor, w: torch.Tensor, desc: im2win_desc, y: torch.Tensor = None,
                  stream=None) -> torch.Tensor:
    """Comparison baseline: direct convolution (no data transformation); returns y."""
    xp = _dev(x, "x", x_shape(desc), _dtype_of(desc))
    wp = _dev(w, "w", w_shape(desc), _dtype_of(desc))
    y, yp = _output(y, desc, x.device, stream)
    im2win_direct_conv2d(desc, xp, wp, yp, _stream(stream))
    return y
