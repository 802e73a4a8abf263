"""Float64 CPU oracle for the AFNO filter's backward pass -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg may import
this module; the HIP library never calls it.

The paper's training step runs the forward and the backward pass of the whole network
("Implementation Details" (a) and (e); its FLOP counts in "Performance: Single Model Instance"
cover both).  The filter's backward pass is the transpose of its forward map ("Model
Innovations", the three spatial-mixing steps), taken step by step in reverse order:

  forward  X = F(x)                       2-D real DFT: W-axis R2C then H-axis DFT, 1/sqrt(HW)
           v = X_k W1_k + b1_k            per mode and block k, complex
           h = relu(Re v) + i relu(Im v)
           o = h W2_k + b2_k
           z = S_lam(Re o) + i S_lam(Im o), zero outside the mode cutoff
           y = G(z)                       H-axis inverse DFT then W-axis C2R, weights c_kw
           out = x + y

  backward, for an upstream gradient g = dL/dout (all gradients of the real parts and the
  imaginary parts of complex quantities packed as gr + i gi):
           dz  = G^T g  = c_kw * F(g)     (the transpose of the C2R-with-weights map is the
                                           R2C map times the same weights; of the unitary
                                           inverse H-DFT, the forward H-DFT)
           do  = dz masked by |Re o| > lam, |Im o| > lam, and by the cutoff
           dh  = do W2^H                  (conjugate transpose: dh_j = sum_k do_k conj W2_jk)
           dv  = dh masked by Re v > 0, Im v > 0
           dX  = dv W1^H
           dW2 = sum over modes of conj(h)^T do,   db2 = sum of do
           dW1 = sum over modes of conj(X)^T dv,   db1 = sum of dv
           dx  = g + F^T dX, F^T dX = G(dX / c_kw)  (the transpose of R2C is C2R with unit
                                           weights; G's weights are c_kw, so divide them out)

The masks use the strict inequalities (relu'(0) = 0, S_lam' = 0 on [-lam, lam]).  A complex
weight gradient is returned as (d/dre, d/dim) pairs in the weights' own layout
[nb][in][out][2]; for v = X W, d/dW_re + i d/dW_im = conj(X) dv.

The transforms are the forward oracle's (direct DFTs); the block products are plain complex
einsums in float64.
"""
from __future__ import annotations

import numpy as np

from . import _f64, irfft2, keep_mask, rfft2


def c_weights(W: int) -> np.ndarray:
    """c_kw of the half-spectrum inverse: 1 at kw = 0 and W/2, 2 in between."""
    Wm = W // 2 + 1
    c = np.full(Wm, 2.0)
    c[0] = 1.0
    c[W // 2] = 1.0
    return c


def _cplx(a) -> np.ndarray:
    a = _f64(a)
    return a[..., 0] + 1j * a[..., 1]


def _pairs(z: np.ndarray) -> np.ndarray:
    return np.stack([z.real, z.imag], axis=-1)


def filter_backward(x, w1, b1, w2, b2, gout, num_blocks: int, lam: float, keep: float):
    """Gradients of L with dL/dout = gout: returns dict dx [B,H,W,C], dw1, dw2 [nb,bs,bs,2],
    db1, db2 [nb,bs,2], all float64."""
    x = _f64(x)
    g = _f64(gout)
    B, H, W, C = x.shape
    assert g.shape == x.shape
    nb = num_blocks
    bs = C // nb
    Wm = W // 2 + 1
    lam = float(np.float32(lam))
    keep = float(np.float32(keep))
    W1, W2 = _cplx(w1), _cplx(w2)          # [nb, bs, bs]
    B1, B2 = _cplx(b1), _cplx(b2)          # [nb, bs]
    c = c_weights(W)

    # forward state, block by block
    X = rfft2(x).reshape(B, H, Wm, nb, bs)
    v = np.einsum("bhwki,kij->bhwkj", X, W1) + B1
    h = np.maximum(v.real, 0.0) + 1j * np.maximum(v.imag, 0.0)
    o = np.einsum("bhwkj,kjl->bhwkl", h, W2) + B2
    kept = keep_mask(H, W, keep)[None, :, :, None, None]

    # backward
    dz = (c[None, None, :, None] * rfft2(g)).reshape(B, H, Wm, nb, bs)
    do = (dz.real * (np.abs(o.real) > lam) + 1j * dz.imag * (np.abs(o.imag) > lam)) * kept
    dh = np.einsum("bhwkl,kjl->bhwkj", do, np.conj(W2))
    dv = dh.real * (v.real > 0) + 1j * dh.imag * (v.imag > 0)
    dX = np.einsum("bhwkj,kij->bhwki", dv, np.conj(W1))
    dw2 = np.einsum("bhwkj,bhwkl->kjl", np.conj(h), do)
    dw1 = np.einsum("bhwki,bhwkj->kij", np.conj(X), dv)
    db2 = do.sum(axis=(0, 1, 2))
    db1 = dv.sum(axis=(0, 1, 2))
    dx = g + irfft2(dX.reshape(B, H, Wm, C) / c[None, None, :, None], W)
    return {"dx": dx, "dw1": _pairs(dw1), "db1": _pairs(db1), "dw2": _pairs(dw2),
            "db2": _pairs(db2)}
