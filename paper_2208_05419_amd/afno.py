"""Python binding of the C ABI in include/afno.h (argument marshalling only).

Every step of the filter runs in the HIP kernels of ``libafno_mi355x.so``; this module
only turns torch tensors into pointers, sizes and the current HIP stream.  There is no
fallback: if the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libafno_mi355x.so")

AFNO_OK = 0
AFNO_ERR_INVALID_ARG = -1
AFNO_ERR_UNSUPPORTED = -2
AFNO_ERR_ALIAS = -3
AFNO_ERR_HIP = -4
AFNO_DTYPE_FP32 = 0
AFNO_DTYPE_BF16 = 1
AFNO_STAGE_SPECTRUM = 1
AFNO_STAGE_MIXED = 2
AFNO_STAGE_DELTA = 3

AFNO_PATH_AUTO = 0
AFNO_PATH_GENERIC = 1
AFNO_PATH_VALU_DFT = 2

EXPORTED = ("afno_filter_forward", "afno_filter_forward_noalloc", "afno_filter_forward_hidden",
            "afno_block_forward",
            "afno_filter_stage", "afno_filter_stage_hidden", "afno_filter_backward",
            "afno_profile_begin", "afno_profile_end", "afno_set_kernel_path", "afno_last_error",
            "afno_version")
KERNELS = ("prep", "row_r2c", "column", "row_c2r")

_ERR_NAMES = {AFNO_ERR_INVALID_ARG: "AFNO_ERR_INVALID_ARG", AFNO_ERR_UNSUPPORTED: "AFNO_ERR_UNSUPPORTED",
              AFNO_ERR_ALIAS: "AFNO_ERR_ALIAS", AFNO_ERR_HIP: "AFNO_ERR_HIP"}

_lib = None


class AfnoError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_ERR_NAMES.get(code, code)}: {msg}")
        self.code = code


def load_library():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"AFNO HIP library not built: {LIB_PATH} is missing "
                           "(run `python -c 'import __graft_entry__ as g; g.build()'`)")
    # torch ships its own HIP runtime under the same soname; loading torch first makes the
    # library bind to that runtime, so tensors torch allocated are valid device pointers here
    # (loaded the other way round, the process would hold two runtimes)
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    i64, vp, f32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_float
    lib.afno_filter_forward.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, f32, f32,
                                        ctypes.c_int, vp, vp]
    lib.afno_filter_forward.restype = ctypes.c_int
    lib.afno_filter_forward_noalloc.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, f32,
                                                f32, ctypes.c_int, vp, vp]
    lib.afno_filter_forward_noalloc.restype = ctypes.c_int
    lib.afno_filter_forward_hidden.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, i64,
                                               f32, f32, ctypes.c_int, vp, vp]
    lib.afno_filter_forward_hidden.restype = ctypes.c_int
    lib.afno_block_forward.argtypes = [vp] * 13 + [i64, i64, i64, i64, i64, f32, f32,
                                                   ctypes.c_int, vp, vp]
    lib.afno_block_forward.restype = ctypes.c_int
    lib.afno_filter_stage.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, f32, f32,
                                      ctypes.c_int, ctypes.c_int, vp, vp]
    lib.afno_filter_stage.restype = ctypes.c_int
    lib.afno_filter_stage_hidden.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, i64,
                                             f32, f32, ctypes.c_int, ctypes.c_int, vp, vp]
    lib.afno_filter_stage_hidden.restype = ctypes.c_int
    # the float* gradient outputs are device addresses: passed as plain pointers
    lib.afno_filter_backward.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, f32, f32,
                                         ctypes.c_int, vp, vp, vp, vp, vp, vp]
    lib.afno_filter_backward.restype = ctypes.c_int
    lib.afno_last_error.argtypes = []
    lib.afno_last_error.restype = ctypes.c_char_p
    lib.afno_version.argtypes = []
    lib.afno_version.restype = ctypes.c_int
    lib.afno_profile_begin.argtypes = [ctypes.c_int]
    lib.afno_profile_begin.restype = ctypes.c_int
    lib.afno_profile_end.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
    lib.afno_profile_end.restype = ctypes.c_int
    lib.afno_set_kernel_path.argtypes = [ctypes.c_int]
    lib.afno_set_kernel_path.restype = ctypes.c_int
    _lib = lib
    return lib


def afno_last_error() -> str:
    return load_library().afno_last_error().decode()


def afno_version() -> int:
    return int(load_library().afno_version())


def _check(rc: int):
    if rc != AFNO_OK:
        raise AfnoError(rc, afno_last_error())


def afno_filter_forward(x, w1, b1, w2, b2, B, H, W, C, num_blocks, lam, keep_fraction, dtype,
                        out, stream) -> int:
    """Raw call: pointers as ints (or None), returns the C return code."""
    return load_library().afno_filter_forward(x, w1, b1, w2, b2, B, H, W, C, num_blocks, lam,
                                              keep_fraction, dtype, out, stream)


def afno_filter_forward_noalloc(x, w1, b1, w2, b2, B, H, W, C, num_blocks, lam, keep_fraction,
                                dtype, out, stream) -> int:
    """Raw call of the allocation-free variant: pointers as ints (or None)."""
    return load_library().afno_filter_forward_noalloc(x, w1, b1, w2, b2, B, H, W, C, num_blocks,
                                                      lam, keep_fraction, dtype, out, stream)


def afno_filter_forward_hidden(x, w1, b1, w2, b2, B, H, W, C, num_blocks, hidden, lam,
                               keep_fraction, dtype, out, stream) -> int:
    """Raw call with the block MLP's hidden size: pointers as ints (or None)."""
    return load_library().afno_filter_forward_hidden(x, w1, b1, w2, b2, B, H, W, C, num_blocks,
                                                     hidden, lam, keep_fraction, dtype, out,
                                                     stream)


def afno_filter_stage(x, w1, b1, w2, b2, B, H, W, C, num_blocks, lam, keep_fraction, dtype,
                      stage, dst, stream) -> int:
    return load_library().afno_filter_stage(x, w1, b1, w2, b2, B, H, W, C, num_blocks, lam,
                                            keep_fraction, dtype, stage, dst, stream)


def afno_filter_stage_hidden(x, w1, b1, w2, b2, B, H, W, C, num_blocks, hidden, lam,
                             keep_fraction, dtype, stage, dst, stream) -> int:
    return load_library().afno_filter_stage_hidden(x, w1, b1, w2, b2, B, H, W, C, num_blocks,
                                                   hidden, lam, keep_fraction, dtype, stage, dst,
                                                   stream)


def afno_filter_backward(x, w1, b1, w2, b2, gout, B, H, W, C, num_blocks, lam, keep_fraction,
                         dtype, dx, dw1, db1, dw2, db2, stream) -> int:
    return load_library().afno_filter_backward(x, w1, b1, w2, b2, gout, B, H, W, C, num_blocks,
                                               lam, keep_fraction, dtype, dx, dw1, db1, dw2,
                                               db2, stream)


def afno_profile_begin(max_calls: int) -> int:
    return load_library().afno_profile_begin(max_calls)


def afno_profile_end(kernel_ms, calls) -> int:
    return load_library().afno_profile_end(kernel_ms, calls)


def afno_set_kernel_path(path: int) -> int:
    return load_library().afno_set_kernel_path(path)


def set_kernel_path(path: int):
    """AFNO_PATH_AUTO: specialised kernels where available (bf16 columns with H <= 96 and
    block size 32, 64 or 96 take the matrix-core DFT kernel); AFNO_PATH_VALU_DFT: the same
    without the matrix-core DFT kernel; AFNO_PATH_GENERIC: generic kernels only."""
    _check(afno_set_kernel_path(path))


def profile_begin(max_calls: int):
    _check(afno_profile_begin(max_calls))


def profile_end():
    """-> ({kernel name: summed ms}, timed calls)"""
    ms = (ctypes.c_double * len(KERNELS))()
    calls = ctypes.c_int64()
    _check(afno_profile_end(ms, ctypes.byref(calls)))
    return dict(zip(KERNELS, list(ms))), int(calls.value)


# ---------------------------------------------------------------- torch-level wrappers


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return AFNO_DTYPE_FP32
    if t.dtype == torch.bfloat16:
        return AFNO_DTYPE_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")


def _ptr(t):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    if not t.is_cuda:
        raise ValueError("tensors must be on the GPU")
    return t.data_ptr() or None


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _grid(x, num_blocks: int):
    """x must be a 4-D [B, H, W, C] tensor of a supported dtype with C a multiple of
    num_blocks; returns (B, H, W, C, bs)."""
    if x.dim() != 4:
        raise ValueError(f"x must be [B, H, W, C], got shape {tuple(x.shape)}")
    _dtype_code(x)
    B, H, W, C = (int(d) for d in x.shape)
    if num_blocks <= 0 or C % num_blocks:
        raise ValueError(f"C = {C} must be a positive multiple of num_blocks = {num_blocks}")
    return B, H, W, C, C // num_blocks


def _expect(x, specs):
    """Checks, before any GPU call, that every (name, tensor, shape, dtype) of specs has that
    shape, that dtype (None: x's), x's device and a contiguous layout, and that x is on the
    GPU: the C library trusts the sizes it is given, so a mismatched tensor would be read or
    written beyond its end."""
    for name, t, shape, dt in specs:
        if t is None:
            raise ValueError(f"{name} is missing")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)} "
                             "(weight shapes must match num_blocks, the block size and the "
                             "hidden size)")
        want = x.dtype if dt is None else dt
        if t.dtype != want:
            raise TypeError(f"{name} has dtype {t.dtype}, expected {want}")
        if t.device != x.device:
            raise ValueError(f"{name} is on {t.device}, x on {x.device}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    if not x.is_cuda:
        raise ValueError("tensors must be on the GPU")


def _filter_specs(x, w1, b1, w2, b2, num_blocks: int, hidden_from_w1: bool):
    """(B, H, W, C, bs, hs) and the weight specs; hs from w1 when hidden_from_w1, else bs."""
    B, H, W, C, bs = _grid(x, num_blocks)
    hs = bs
    if hidden_from_w1:
        if w1 is None or w1.dim() != 4:
            raise ValueError("w1 must be [num_blocks, bs, hidden, 2] (weight shapes)")
        hs = int(w1.shape[2])
    nb = num_blocks
    specs = [("w1", w1, (nb, bs, hs, 2), None), ("b1", b1, (nb, hs, 2), None),
             ("w2", w2, (nb, hs, bs, 2), None), ("b2", b2, (nb, bs, 2), None)]
    return (B, H, W, C, bs, hs), specs


def filter_forward(x, w1, b1, w2, b2, num_blocks: int, lam: float, keep_fraction: float = 1.0,
                   out=None, stream=None):
    """out = x + AFNO filter(x) for x [B,H,W,C] (float32 or bfloat16 on the GPU);
    weights w1 [nb,bs,hs,2], b1 [nb,hs,2], w2 [nb,hs,bs,2], b2 [nb,bs,2] of x's dtype, the
    hidden size hs from w1 (hs = bs: afno_filter_forward, else afno_filter_forward_hidden).
    Enqueued on ``stream`` (default: torch's current stream)."""
    import torch
    (B, H, W, C, bs, hs), specs = _filter_specs(x, w1, b1, w2, b2, num_blocks, True)
    if out is not None:
        specs.append(("out", out, tuple(x.shape), None))
    _expect(x, specs)
    if out is None:
        out = torch.empty_like(x)
    if hs == bs:
        rc = afno_filter_forward(_ptr(x), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2), B, H, W, C,
                                 num_blocks, lam, keep_fraction, _dtype_code(x), _ptr(out),
                                 _stream(stream))
    else:
        rc = afno_filter_forward_hidden(_ptr(x), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2), B, H, W,
                                        C, num_blocks, hs, lam, keep_fraction, _dtype_code(x),
                                        _ptr(out), _stream(stream))
    _check(rc)
    return out


def filter_forward_noalloc(x, w1, b1, w2, b2, num_blocks: int, lam: float, keep_fraction: float,
                           out, stream=None):
    """afno_filter_forward_noalloc: out = x + AFNO filter(x) into the caller's out, with no
    device allocation (the library's fixed workspace; hidden size = block size).  Calls that
    overlap in time on one GPU race (see include/afno.h)."""
    (B, H, W, C, bs, hs), specs = _filter_specs(x, w1, b1, w2, b2, num_blocks, False)
    specs.append(("out", out, tuple(x.shape), None))
    _expect(x, specs)
    _check(afno_filter_forward_noalloc(_ptr(x), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2), B, H, W,
                                       C, num_blocks, lam, keep_fraction, _dtype_code(x),
                                       _ptr(out), _stream(stream)))
    return out


def afno_block_forward(x, ln1_g, ln1_b, w1, b1, w2, b2, ln2_g, ln2_b, wa, ba, wb, bb, B, H, W, C,
                       num_blocks, lam, keep_fraction, dtype, out, stream) -> int:
    """Raw call: pointers as ints (or None), returns the C return code."""
    return load_library().afno_block_forward(x, ln1_g, ln1_b, w1, b1, w2, b2, ln2_g, ln2_b, wa,
                                             ba, wb, bb, B, H, W, C, num_blocks, lam,
                                             keep_fraction, dtype, out, stream)


BLOCK_PARAMS = ("ln1_g", "ln1_b", "w1", "b1", "w2", "b2", "ln2_g", "ln2_b", "wa", "ba", "wb", "bb")


def block_forward(x, p: dict, num_blocks: int, lam: float, keep_fraction: float = 1.0, out=None,
                  stream=None):
    """One AFNO block on x [B,H,W,C] bfloat16: p holds the BLOCK_PARAMS tensors (bfloat16, on
    the GPU): the LayerNorm gains and shifts [C], the filter's weights (hidden = block size),
    wa [C,4C], ba [4C], wb [4C,C], bb [C].  Enqueued on ``stream`` (default: torch's current
    stream)."""
    import torch
    missing = [k for k in BLOCK_PARAMS if p.get(k) is None]
    if missing:
        raise ValueError(f"block parameters missing: {missing}")
    (B, H, W, C, bs, hs), specs = _filter_specs(x, p["w1"], p["b1"], p["w2"], p["b2"],
                                                num_blocks, False)
    specs += [(k, p[k], (C,), None) for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "bb")]
    specs += [("wa", p["wa"], (C, 4 * C), None), ("ba", p["ba"], (4 * C,), None),
              ("wb", p["wb"], (4 * C, C), None)]
    if out is not None:
        specs.append(("out", out, tuple(x.shape), None))
    _expect(x, specs)
    if out is None:
        out = torch.empty_like(x)
    rc = afno_block_forward(_ptr(x), *(_ptr(p[k]) for k in BLOCK_PARAMS), B, H, W, C, num_blocks,
                            lam, keep_fraction, _dtype_code(x), _ptr(out), _stream(stream))
    _check(rc)
    return out


def filter_backward(x, w1, b1, w2, b2, gout, num_blocks: int, lam: float, keep_fraction: float = 1.0,
                    stream=None):
    """Gradients through out = x + AFNO filter(x) for dL/dout = gout: returns a dict with dx
    (x's dtype) and dw1, db1, dw2, db2 (float32, the weights' layouts).  The backward runs the
    paper's filter, hidden size = block size: other weight shapes are rejected."""
    import torch
    (B, H, W, C, bs, hs), specs = _filter_specs(x, w1, b1, w2, b2, num_blocks, False)
    specs.append(("gout", gout, tuple(x.shape), None))
    _expect(x, specs)
    f32 = dict(dtype=torch.float32, device=x.device)
    dx = torch.empty_like(x)
    dw1, dw2 = torch.empty((num_blocks, bs, bs, 2), **f32), torch.empty((num_blocks, bs, bs, 2), **f32)
    db1, db2 = torch.empty((num_blocks, bs, 2), **f32), torch.empty((num_blocks, bs, 2), **f32)
    rc = afno_filter_backward(_ptr(x), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2), _ptr(gout), B, H,
                              W, C, num_blocks, lam, keep_fraction, _dtype_code(x), _ptr(dx),
                              _ptr(dw1), _ptr(db1), _ptr(dw2), _ptr(db2), _stream(stream))
    _check(rc)
    return {"dx": dx, "dw1": dw1, "db1": db1, "dw2": dw2, "db2": db2}


def filter_stage(x, w1, b1, w2, b2, num_blocks: int, lam: float, keep_fraction: float, stage: int,
                 stream=None):
    """Diagnostic stage output in float32: spectrum / mixed spectrum [B,H,W/2+1,C,2] or the
    filter output before the residual [B,H,W,C].  The hidden size comes from w1 (hs != bs:
    afno_filter_stage_hidden)."""
    import torch
    (B, H, W, C, bs, hs), specs = _filter_specs(x, w1, b1, w2, b2, num_blocks, True)
    _expect(x, specs)
    shape = (B, H, W, C) if stage == AFNO_STAGE_DELTA else (B, H, W // 2 + 1, C, 2)
    dst = torch.empty(shape, dtype=torch.float32, device=x.device)
    if hs == bs:
        rc = afno_filter_stage(_ptr(x), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2), B, H, W, C,
                               num_blocks, lam, keep_fraction, _dtype_code(x), stage, _ptr(dst),
                               _stream(stream))
    else:
        rc = afno_filter_stage_hidden(_ptr(x), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2), B, H, W,
                                      C, num_blocks, hs, lam, keep_fraction, _dtype_code(x),
                                      stage, _ptr(dst), _stream(stream))
    _check(rc)
    return dst
