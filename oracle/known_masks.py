"""Inputs with unambiguous mask decisions for the backward parity tests -- TEST
INFRASTRUCTURE ONLY (tests may import it; the HIP library never does).

The filter's gradients are step functions of two decisions per kept mode, block unit and
real component: relu's (v > 0, v = X w1 + b1) and the softshrink's (|o| > lam, o = h w2 + b2).
Where an implementation's v or o lie within its rounding error of such a kink, either branch
is a correct result.  This module builds inputs on which no decision is that close: from x,
w1, w2 as drawn it chooses b1, b2 and lam with the exact float64 forward state of the
oracle, so that on every kept mode |v| >= m1 and ||o| - lam| >= m2, with m1, m2 many times
the error a bf16-storage implementation makes in v and o.  The backward of such inputs has
one correct result, and the GPU's gradients can be compared with the oracle's element by
element, with no allowance.

To make the masks change from mode to mode (rather than hold one value per unit over all
modes), plant_frequencies adds a few strong single-frequency components to x: at those modes
the spectrum is tens of times larger than elsewhere, so for many units the widest gap in v
(and in o) separates the planted modes from the rest, and the bias is put into that gap.

Procedure for one bias (per block k, unit j, component re/im): the forbidden values of the bias
are intervals of half-width m around the points c_m (c_m = -R_m for b1 with R = X w1; c_m =
+-lam - o0_m for b2 with o0 = h w2), one or two per kept mode m.  The bias is the middle of the
widest gap between consecutive sorted points when that gap leaves 2 m on both sides (chosen
with probability `interior`), else a value 3 m beyond the smallest or the largest point.  The
bias is then rounded to the storage dtype and the margin is checked again on the rounded value.
"""
from __future__ import annotations

import numpy as np

from . import keep_mask, rfft2
from .backward import _blocks, _cplx, round_bf16


def _store(a, dtype):
    """Nearest value of the storage dtype (float32 or bf16) of each float64, as float64."""
    if dtype == "bf16":
        return round_bf16(a)
    return np.asarray(a, dtype=np.float64).astype(np.float32).astype(np.float64)


def plant_frequencies(x, dtype: str, keep: float, n_freq: int, amp: float, rng):
    """x [B,H,W,C] float64 plus, per sample, n_freq components amp * cos(2 pi (a h / H + b w / W)
    + phi) * u[c] (u a random +-1 vector over the channels) at kept modes (a, b) with
    0 < b < W/2, rounded to the storage dtype.  Returns (x as stored values in float64,
    the planted (sample, a, b) list)."""
    x = np.array(x, dtype=np.float64)
    B, H, W, C = x.shape
    kept = keep_mask(H, W, keep)
    cand = [(a, b) for a in range(H) for b in range(1, W // 2) if kept[a, b]]
    planted = []
    hh = np.arange(H)[:, None, None]
    ww = np.arange(W)[None, :, None]
    for s in range(B):
        if not cand:
            break
        for t in rng.choice(len(cand), size=min(n_freq, len(cand)), replace=False):
            a, b = cand[int(t)]
            phi = rng.uniform(0, 2 * np.pi)
            u = rng.choice([-1.0, 1.0], size=C)
            x[s] += amp * np.cos(2 * np.pi * (a * hh / H + b * ww / W) + phi) * u[None, None, :]
            planted.append((s, a, b))
    return _store(x, dtype), planted


def _pick(points, m, rng, interior):
    """points [U, N]: per unit, a value at distance >= 2 m from each of its N points (see the
    module docstring); interior: probability of taking the widest interior gap when it
    qualifies."""
    S = np.sort(points, axis=1)
    U = S.shape[0]
    lo, hi = S[:, 0], S[:, -1]
    ext = np.where(rng.random(U) < 0.5, lo - 3 * m, hi + 3 * m)
    if S.shape[1] < 2:
        return ext, np.zeros(U, dtype=bool)
    d = S[:, 1:] - S[:, :-1]
    k = np.argmax(d, axis=1)
    rows = np.arange(U)
    width = d[rows, k]
    mid = 0.5 * (S[rows, k] + S[rows, k + 1])
    use = (width >= 4 * m) & (rng.random(U) < interior)
    return np.where(use, mid, ext), use


def _units(z):
    """complex [M, nb, n] -> real [nb * n * 2, M]: one row per (block, unit, component)."""
    return np.ascontiguousarray(np.stack([z.real, z.imag], axis=-1).reshape(z.shape[0], -1).T)


def _fix(b, points, m, dtype):
    """Round the biases to the storage dtype; where rounding leaves a unit closer than m to one
    of its points ([U, N]), move that unit's bias 4 m beyond the nearer end of its points and
    round again."""
    bq = _store(b, dtype)
    lo, hi = points.min(axis=1), points.max(axis=1)
    for _ in range(4):
        dist = np.min(np.abs(points - bq[:, None]), axis=1)
        bad = dist < m
        if not np.any(bad):
            return bq
        shift = 4 * m + 2.0 ** -7 * np.abs(b)
        b = np.where(bad, np.where(bq < 0.5 * (lo + hi), lo - shift, hi + shift), b)
        bq = _store(b, dtype)
    raise AssertionError("could not place the biases outside the kink bands")


def choose_biases(x, w1, w2, num_blocks: int, keep: float, dtype: str, rng, interior: float = 0.6,
                  margin: float = 12.0):
    """b1 [nb,bs,2], b2 [nb,bs,2] (float64 values exact in the storage dtype) and lam (a float32
    value) for which every kept mode's decisions are unambiguous.

    The margins are `margin` times an estimate of a bf16-storage implementation's error in v
    and o (operands rounded to bf16: relative 2^-8 per element, errors adding in quadrature over
    the 2 bs (2 hs) real terms of a product), and at least 5 % of the spread of v (o).  Returns
    (b1, b2, lam, info) with info: the margins, the smallest distances achieved, the fraction of
    units whose relu and softshrink masks differ between modes."""
    x = np.asarray(x, dtype=np.float64)
    B, H, W, C = x.shape
    nb = num_blocks
    bs = C // nb
    Wm = W // 2 + 1
    W1, W2 = _cplx(w1), _cplx(w2)
    hs = W1.shape[-1]
    kept = keep_mask(H, W, keep)
    X = rfft2(x).reshape(B, H, Wm, nb, bs)[:, kept]          # [B, K, nb, bs]
    X = X.reshape(-1, nb, bs)                                 # [M, nb, bs]
    R = _blocks(X, W1)                                        # [M, nb, hs]
    Rr = _units(R)                                            # [U1, M]
    eps = 2.0 ** -8
    rms = lambda a: float(np.sqrt(np.mean(np.abs(a) ** 2)))  # noqa: E731
    e_v = eps * rms(X) * np.sqrt(2) * rms(W1) * np.sqrt(2 * bs)
    m1 = max(margin * e_v, 0.05 * float(np.std(Rr)))
    p1 = -Rr
    b1, _ = _pick(p1, m1, rng, interior)
    b1 = _fix(b1, p1, m1, dtype)
    v = Rr + b1[:, None]
    h = np.maximum(v, 0.0).T.reshape(-1, nb, hs, 2)
    hc = h[..., 0] + 1j * h[..., 1]
    Or = _units(_blocks(hc, W2))                              # [U2, M]
    e_o = eps * (rms(hc) * np.sqrt(2) + e_v) * rms(W2) * np.sqrt(2 * hs)
    So = np.sort(Or, axis=1)
    n = So.shape[1]
    cen = So - So[:, n // 2:n // 2 + 1]
    m2 = max(margin * e_o, 0.05 * float(np.std(cen)))
    # lam: half the median spread of o over the modes (0.1 % trimmed at both ends), so that
    # for about half of the units the bulk of the modes can sit inside (-lam, lam) while the
    # planted modes pass
    spread = So[:, min(n - 1, int(0.999 * n))] - So[:, int(0.001 * n)]
    lam = float(np.float32(0.5 * float(np.median(spread)) + 3 * m2))
    p2 = np.concatenate([lam - Or, -lam - Or], axis=1)
    b2, _ = _pick(p2, m2, rng, interior)
    b2 = _fix(b2, p2, m2, dtype)
    o = Or + b2[:, None]
    d1 = float(np.min(np.abs(v)))
    d2 = float(np.min(np.abs(np.abs(o) - lam)))
    relu_mixed = float(np.mean(np.any(v > 0, axis=1) & np.any(v < 0, axis=1)))
    soft_mixed = float(np.mean(np.any(np.abs(o) > lam, axis=1) & np.any(np.abs(o) < lam, axis=1)))
    info = {"m1": m1, "m2": m2, "min_dist_v": d1, "min_dist_o": d2, "relu_mixed": relu_mixed,
            "softshrink_mixed": soft_mixed, "lam": lam}
    assert d1 >= m1 and d2 >= m2, info
    shape = (nb, bs, 2)
    return b1.reshape(nb, hs, 2), b2.reshape(shape), lam, info
