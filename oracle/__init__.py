"""Float64 CPU oracle for the AFNO spectral filter -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this package.  The HIP library never imports, links or calls it, and it
shares no code with the HIP path: it is a ctypes wrapper around ``afno_oracle.c``
(plain C, double precision, direct DFTs and naive complex matrix products).

Functions take and return float64 numpy arrays.  Stored bf16 inputs are widened to
float64 exactly (``widen_bf16``), so the oracle only ever sees the quantised values.
Every function cites the passage of the FourCastNet paper it follows in the C file.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libafno_oracle.so")
_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_l = ctypes.c_long


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b  # the checker is C; build it on first use
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.orc_keep_counts.argtypes = [_l, _l, ctypes.c_double, ctypes.POINTER(_l), ctypes.POINTER(_l)]
    lib.orc_keep_counts.restype = None
    lib.orc_mode_kept.argtypes = [_l, _l, _l, _l, _l]
    lib.orc_mode_kept.restype = ctypes.c_int
    lib.orc_dft_w_r2c.argtypes = [_dp, _l, _l, _l, _l, _dp]
    lib.orc_dft_h.argtypes = [_dp, _l, _l, _l, _l, ctypes.c_int, _dp]
    lib.orc_dft_w_c2r.argtypes = [_dp, _l, _l, _l, _l, _dp]
    lib.orc_block_mlp.argtypes = [_dp, _dp, _dp, _dp, _dp, _l, _l, _l, _l, _l, ctypes.c_double,
                                  _l, _l, _dp]
    lib.orc_filter_forward.argtypes = [_dp, _dp, _dp, _dp, _dp, _l, _l, _l, _l, _l,
                                       ctypes.c_double, ctypes.c_double, _dp, _dp, _dp, _dp]
    lib.orc_block_mlp_h.argtypes = [_dp, _dp, _dp, _dp, _dp, _l, _l, _l, _l, _l, _l,
                                    ctypes.c_double, _l, _l, _dp]
    lib.orc_filter_forward_h.argtypes = [_dp, _dp, _dp, _dp, _dp, _l, _l, _l, _l, _l, _l,
                                         ctypes.c_double, ctypes.c_double, _dp, _dp, _dp, _dp]
    lib.orc_dft2_bruteforce.argtypes = [_dp, _l, _l, _l, _l, _dp]
    lib.orc_idft2_bruteforce.argtypes = [_dp, _l, _l, _l, _l, _dp]
    for f in ("orc_dft_w_r2c", "orc_dft_h", "orc_dft_w_c2r", "orc_block_mlp",
              "orc_filter_forward", "orc_block_mlp_h", "orc_filter_forward_h",
              "orc_dft2_bruteforce", "orc_idft2_bruteforce",
              "orc_num_threads"):
        getattr(lib, f).restype = ctypes.c_int
    lib.orc_num_threads.argtypes = []
    _lib = lib
    return lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return ctypes.cast(None, _dp)
    assert a.dtype == np.float64 and a.flags.c_contiguous
    return a.ctypes.data_as(_dp)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _check(rc: int, name: str):
    if rc != 0:
        raise ValueError(f"oracle {name} rejected its arguments (rc={rc})")


def widen_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64, exactly (bf16 is the top half of a float32)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def num_threads() -> int:
    return int(_load().orc_num_threads())


def keep_counts(H: int, W: int, keep: float) -> tuple[int, int]:
    """(kept_h, kept_w) of the hard mode cutoff; keep is taken as the float32 the ABI passes."""
    kh, kw = _l(), _l()
    _load().orc_keep_counts(H, W, float(np.float32(keep)), ctypes.byref(kh), ctypes.byref(kw))
    return kh.value, kw.value


def keep_mask(H: int, W: int, keep: float) -> np.ndarray:
    """Boolean [H, W/2+1] mask of the modes that pass the block MLP."""
    kept_h, kept_w = keep_counts(H, W, keep)
    lib = _load()
    Wm = W // 2 + 1
    return np.array([[bool(lib.orc_mode_kept(a, b, H, kept_h, kept_w)) for b in range(Wm)]
                     for a in range(H)])


def rfft2(x, mid=None) -> np.ndarray:
    """Forward spectrum [B,H,Wm,C] complex128 of real x [B,H,W,C] (direct DFT, W then H).
    mid, if given, maps the W-axis spectrum [B,H,Wm,C,2] (re, im) before the H-axis DFT (a
    storage rounding between the two passes)."""
    x = _f64(x)
    B, H, W, C = x.shape
    Wm = W // 2 + 1
    s1 = np.empty((B, H, Wm, C, 2))
    s2 = np.empty_like(s1)
    lib = _load()
    _check(lib.orc_dft_w_r2c(_ptr(x), B, H, W, C, _ptr(s1)), "dft_w_r2c")
    if mid is not None:
        s1 = _f64(mid(s1))
    _check(lib.orc_dft_h(_ptr(s1), B, H, Wm, C, -1, _ptr(s2)), "dft_h")
    return s2[..., 0] + 1j * s2[..., 1]


def irfft2(Y, W: int) -> np.ndarray:
    """Real [B,H,W,C] from a half spectrum [B,H,Wm,C] (inverse H, then complex-to-real W)."""
    Y = np.asarray(Y)
    B, H, Wm, C = Y.shape
    assert Wm == W // 2 + 1
    s = _f64(np.stack([Y.real, Y.imag], axis=-1))
    s2 = np.empty_like(s)
    y = np.empty((B, H, W, C))
    lib = _load()
    _check(lib.orc_dft_h(_ptr(s), B, H, Wm, C, +1, _ptr(s2)), "dft_h")
    _check(lib.orc_dft_w_c2r(_ptr(s2), B, H, W, C, _ptr(y)), "dft_w_c2r")
    return y


def _hidden(w1, b1, w2, b2, num_blocks: int, C: int) -> int:
    """Hidden units per block, from the weights' shapes: w1 [nb][bs][hs][2], b1 [nb][hs][2],
    w2 [nb][hs][bs][2], b2 [nb][bs][2] (hs = bs is the filter's default)."""
    bs = C // num_blocks
    hs = int(np.shape(w1)[2])
    if (np.shape(w1) != (num_blocks, bs, hs, 2) or np.shape(b1) != (num_blocks, hs, 2)
            or np.shape(w2) != (num_blocks, hs, bs, 2) or np.shape(b2) != (num_blocks, bs, 2)):
        raise ValueError("weight shapes do not match num_blocks, the block size and a hidden size")
    return hs


def block_mlp(X, w1, b1, w2, b2, num_blocks: int, lam: float, keep: float, W: int) -> np.ndarray:
    """MLP + softshrink + cutoff on a spectrum [B,H,Wm,C] complex; returns the same shape.
    The hidden size is w1's third dimension."""
    X = np.asarray(X)
    B, H, Wm, C = X.shape
    hs = _hidden(w1, b1, w2, b2, num_blocks, C)
    kept_h, kept_w = keep_counts(H, W, keep)
    s = _f64(np.stack([X.real, X.imag], axis=-1))
    y = np.empty_like(s)
    _check(_load().orc_block_mlp_h(_ptr(s), _ptr(_f64(w1)), _ptr(_f64(b1)), _ptr(_f64(w2)),
                                   _ptr(_f64(b2)), B, H, Wm, C, num_blocks, hs, float(lam),
                                   kept_h, kept_w, _ptr(y)), "block_mlp")
    return y[..., 0] + 1j * y[..., 1]


def filter_forward(x, w1, b1, w2, b2, num_blocks: int, lam: float, keep: float,
                   stages: bool = False):
    """out = x + filter(x) in float64 (hidden size: w1's third dimension).  With stages=True
    also returns a dict holding 'spec_fwd', 'spec_mlp' (complex [B,H,Wm,C]) and 'delta'
    ([B,H,W,C])."""
    x = _f64(x)
    B, H, W, C = x.shape
    hs = _hidden(w1, b1, w2, b2, num_blocks, C)
    Wm = W // 2 + 1
    lam = float(np.float32(lam))
    keep = float(np.float32(keep))
    out = np.empty_like(x)
    sf = np.empty((B, H, Wm, C, 2)) if stages else None
    sm = np.empty((B, H, Wm, C, 2)) if stages else None
    de = np.empty_like(x) if stages else None
    _check(_load().orc_filter_forward_h(_ptr(x), _ptr(_f64(w1)), _ptr(_f64(b1)), _ptr(_f64(w2)),
                                        _ptr(_f64(b2)), B, H, W, C, num_blocks, hs, lam, keep,
                                        _ptr(out), _ptr(sf), _ptr(sm), _ptr(de)), "filter_forward")
    if not stages:
        return out
    return out, {"spec_fwd": sf[..., 0] + 1j * sf[..., 1],
                 "spec_mlp": sm[..., 0] + 1j * sm[..., 1], "delta": de}


def dft2_bruteforce(x) -> np.ndarray:
    x = _f64(x)
    B, H, W, C = x.shape
    X = np.empty((B, H, W // 2 + 1, C, 2))
    _check(_load().orc_dft2_bruteforce(_ptr(x), B, H, W, C, _ptr(X)), "dft2_bruteforce")
    return X[..., 0] + 1j * X[..., 1]


def idft2_bruteforce(Y, W: int) -> np.ndarray:
    Y = np.asarray(Y)
    B, H, Wm, C = Y.shape
    s = _f64(np.stack([Y.real, Y.imag], axis=-1))
    y = np.empty((B, H, W, C))
    _check(_load().orc_idft2_bruteforce(_ptr(s), B, H, W, C, _ptr(y)), "idft2_bruteforce")
    return y
