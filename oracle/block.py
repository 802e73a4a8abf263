"""Float64 CPU oracle of one AFNO transformer block's forward pass -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline leg may import
this module; the HIP library never calls it.

The paper's transformer layer ("Model Innovations") mixes tokens with the spectral filter and
then channels with a single-hidden-layer MLP whose hidden width is four times the embedding
("Implementation Details" (c): 4,096 hidden units for 1,024 channels), the MLP weights shared
by all tokens.  The paper leaves the normalisation, the activation and the residual
arrangement unstated; the reading taken here is the pre-norm transformer block of the AFNO
layer:

    t   = LN1(x)                       per-token LayerNorm over the C channels
    v   = x + filter(t)                the filter as defined (it adds its own input t)
    w   = LN2(v)
    out = v + GELU(w Wa + ba) Wb + bb  Wa [C][4C], ba [4C], Wb [4C][C], bb [C]

    LN(z) = (z - mean) / sqrt(var + eps) * gamma + beta,  biased variance, eps = 1e-6
    GELU(z) = z * Phi(z) = 0.5 z (1 + erf(z / sqrt 2))   (the exact form)
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

from . import _f64, filter_forward

LN_EPS = 1e-6


def layer_norm(z, gamma, beta, eps: float = LN_EPS) -> np.ndarray:
    """Per-token LayerNorm over the last axis (biased variance)."""
    z = _f64(z)
    mean = z.mean(axis=-1, keepdims=True)
    var = ((z - mean) ** 2).mean(axis=-1, keepdims=True)
    return (z - mean) / np.sqrt(var + eps) * _f64(gamma) + _f64(beta)


def gelu(z) -> np.ndarray:
    """GELU(z) = z Phi(z), Phi the standard normal CDF through erf."""
    z = _f64(z)
    return 0.5 * z * (1.0 + erf(z / np.sqrt(2.0)))


def channel_mlp(w, wa, ba, wb, bb) -> np.ndarray:
    """GELU(w Wa + ba) Wb + bb per token; w [..., C]."""
    h = gelu(_f64(w) @ _f64(wa) + _f64(ba))
    return h @ _f64(wb) + _f64(bb)


def block_forward(x, ln1_g, ln1_b, w1, b1, w2, b2, ln2_g, ln2_b, wa, ba, wb, bb,
                  num_blocks: int, lam: float, keep: float, stages: bool = False):
    """One AFNO block on x [B,H,W,C] in float64; with stages=True also returns t, v, w."""
    x = _f64(x)
    t = layer_norm(x, ln1_g, ln1_b)
    v = x + filter_forward(t, w1, b1, w2, b2, num_blocks, lam, keep)
    w = layer_norm(v, ln2_g, ln2_b)
    out = v + channel_mlp(w, wa, ba, wb, bb)
    if stages:
        return out, {"t": t, "v": v, "w": w}
    return out
