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
batched matrix products in float64.
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


def _blocks(A, Wk):
    """Per-block product: A [..., nb, i] times Wk [nb, i, j] -> [..., nb, j] (a batched matmul)."""
    lead = A.shape[:-2]
    nb, ni = A.shape[-2:]
    a = A.reshape(-1, nb, ni).transpose(1, 0, 2)
    return np.matmul(a, Wk).transpose(1, 0, 2).reshape(*lead, nb, Wk.shape[-1])


def _gram(A, Bm):
    """sum over modes of A^T B per block: A [..., nb, i], B [..., nb, j] -> [nb, i, j]."""
    nb = A.shape[-2]
    a = A.reshape(-1, nb, A.shape[-1]).transpose(1, 2, 0)
    b = Bm.reshape(-1, nb, Bm.shape[-1]).transpose(1, 0, 2)
    return np.matmul(a, b)


def round_bf16(a) -> np.ndarray:
    """Nearest bfloat16 value (ties to even) of each float64, through float32 (the value a
    float32 computation stores as bf16)."""
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32).astype(np.float64)
    return np.where(np.isfinite(f), out, f.astype(np.float64))


def _round_c(z, rnd):
    return rnd(z.real) + 1j * rnd(z.imag)


def filter_backward(x, w1, b1, w2, b2, gout, num_blocks: int, lam: float, keep: float,
                    band: float = 0.0, decide: str = "exact", flips=()):
    """Gradients of L with dL/dout = gout: returns dict dx [B,H,W,C], dw1, dw2 [nb,bs,bs,2],
    db1, db2 [nb,bs,2], all float64.

    band > 0 adds the kink allowance: the gradients are step functions of the pre-activations
    at relu's kink (v = 0) and the softshrink's (|o| = lam), so an implementation whose v or o
    differ from the exact ones by up to band * rms(v) (band * rms(o)) may take either branch
    for elements that close to a kink.  allow_<name> bounds, elementwise, how far its gradient
    can move when any set of those ambiguous branches flips (first order: each flip taken
    alone, their magnitudes summed; a flip at one kink does not move another), and n_kinks
    counts the ambiguous elements (v, o).

    decide selects the precision of the two mask decisions (relu's v > 0, the softshrink's
    |o| > lam); the gradient values are float64 either way.  "exact": v and o in float64.
    "bf16" (a CPU diagnostic): v and o from bf16-stored intermediates, as a bf16-storage
    implementation forms them: the W-axis spectrum, the 2-D spectrum X and the hidden layer h
    rounded to bf16 (products and sums then exact).

    flips: decisions to invert, each (kind, part, index) with kind "relu" (v > 0) or "soft"
    (|o| > lam), part 0 (re) or 1 (im) and index (b, kh, kw, block, unit): the other branch at
    an element that sits at a kink (see ambiguous_decisions)."""
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
    v = _blocks(X, W1) + B1
    h = np.maximum(v.real, 0.0) + 1j * np.maximum(v.imag, 0.0)
    o = _blocks(h, W2) + B2
    kept = keep_mask(H, W, keep)[None, :, :, None, None]
    if decide == "exact":
        v_dec, o_dec = v, o
    elif decide == "bf16":
        Xr = _round_c(rfft2(x, mid=round_bf16), round_bf16).reshape(B, H, Wm, nb, bs)
        v_dec = _blocks(Xr, W1) + B1
        hr = _round_c(np.maximum(v_dec.real, 0.0) + 1j * np.maximum(v_dec.imag, 0.0), round_bf16)
        o_dec = _blocks(hr, W2) + B2
    else:
        raise ValueError(f"unknown decide {decide!r}")

    # the two masks, with the requested decisions inverted
    soft = [np.abs(o_dec.real) > lam, np.abs(o_dec.imag) > lam]
    relu = [v_dec.real > 0, v_dec.imag > 0]
    for kind, part, idx in flips:
        if kind not in ("relu", "soft"):
            raise ValueError(f"unknown decision kind {kind!r}")
        m = relu if kind == "relu" else soft
        m[part][tuple(idx)] = not m[part][tuple(idx)]

    # backward
    dz = (c[None, None, :, None] * rfft2(g)).reshape(B, H, Wm, nb, bs)
    do = (dz.real * soft[0] + 1j * dz.imag * soft[1]) * kept
    dh = _blocks(do, np.conj(W2).transpose(0, 2, 1))
    dv = dh.real * relu[0] + 1j * dh.imag * relu[1]
    dX = _blocks(dv, np.conj(W1).transpose(0, 2, 1))
    dw2 = _gram(np.conj(h), do)
    dw1 = _gram(np.conj(X), dv)
    db2 = do.sum(axis=(0, 1, 2))
    db1 = dv.sum(axis=(0, 1, 2))
    dx = g + irfft2(dX.reshape(B, H, Wm, C) / c[None, None, :, None], W)
    res = {"dx": dx, "dw1": _pairs(dw1), "db1": _pairs(db1), "dw2": _pairs(dw2),
           "db2": _pairs(db2)}
    if band > 0.0:
        res.update(_kink_allowance(X, v_dec, h, o_dec, dz, dh, kept, W1, W2, lam, band, H * W))
    return res


def _kink_allowance(X, v, h, o, dz, dh, kept, W1, W2, lam, band, hw):
    """Elementwise bounds on the gradient change from flipping ambiguous mask entries (see
    filter_backward).  A relu flip at (mode, block, j, part) moves dv_j by the part's dh value a:
    dW1[:, j] by |X_i| a, db1[j] by a, dX_i by a |W1_ij|.  A softshrink flip at (..., l, part)
    moves do_l by the part's dz value a: db2[l] by a, dW2[:, l] by |h_j| a, dh_j by at most
    e_j = a |W2_jl|, and so dv_j, db1[j] by e_j, dW1[:, j] by |X_i| e_j, dX_i by sum_j e_j |W1_ij|.
    dX at one mode reaches every pixel of its sample through the half-spectrum inverse with at
    most |dX| / sqrt(H W)."""
    rms_v = np.sqrt(np.mean(v.real ** 2 + v.imag ** 2) / 2)
    rms_o = np.sqrt(np.mean(o.real ** 2 + o.imag ** 2) / 2)
    a1r = np.abs(dh.real) * (np.abs(v.real) <= band * rms_v)
    a1i = np.abs(dh.imag) * (np.abs(v.imag) <= band * rms_v)
    near = lambda t: np.abs(np.abs(t) - lam) <= band * rms_o  # noqa: E731
    a2r = np.abs(dz.real) * near(o.real) * kept
    a2i = np.abs(dz.imag) * near(o.imag) * kept
    s1, s2 = a1r + a1i, a2r + a2i                            # [B, H, Wm, nb, bs]
    e = _blocks(s2, np.abs(W2).transpose(0, 2, 1))           # e_j = sum_l s2_l |W2_jl|
    both = lambda t: np.stack([t, t], axis=-1)  # noqa: E731
    dw1 = _gram(np.abs(X), s1 + e)
    dw2 = _gram(np.abs(h), s2)
    db1 = np.stack([(a1r + e).sum(axis=(0, 1, 2)), (a1i + e).sum(axis=(0, 1, 2))], axis=-1)
    db2 = np.stack([a2r.sum(axis=(0, 1, 2)), a2i.sum(axis=(0, 1, 2))], axis=-1)
    dX = _blocks(s1 + e, np.abs(W1).transpose(0, 2, 1))     # [B, H, Wm, nb, bs]
    B = X.shape[0]
    per_sample = dX.reshape(B, -1, dX.shape[-2] * dX.shape[-1]).sum(axis=1) / np.sqrt(hw)
    n = int(np.count_nonzero(a1r) + np.count_nonzero(a1i) + np.count_nonzero(a2r) +
            np.count_nonzero(a2i))
    return {"allow_dx": per_sample[:, None, None, :], "allow_dw1": both(dw1),
            "allow_db1": db1, "allow_dw2": both(dw2), "allow_db2": db2, "n_kinks": n}


def ambiguous_decisions(x, w1, b1, w2, b2, num_blocks: int, lam: float, keep: float,
                        band: float):
    """The decisions an implementation whose v and o are within band * rms(v) (band * rms(o))
    of the exact float64 values may take either way: relu's at |v| <= band * rms(v) and the
    softshrink's at ||o| - lam| <= band * rms(o), on kept modes, as flips entries (kind, part,
    index) for filter_backward."""
    x = _f64(x)
    B, H, W, C = x.shape
    nb = num_blocks
    bs = C // nb
    Wm = W // 2 + 1
    lam = float(np.float32(lam))
    keep = float(np.float32(keep))
    W1, W2 = _cplx(w1), _cplx(w2)
    B1, B2 = _cplx(b1), _cplx(b2)
    X = rfft2(x).reshape(B, H, Wm, nb, bs)
    v = _blocks(X, W1) + B1
    h = np.maximum(v.real, 0.0) + 1j * np.maximum(v.imag, 0.0)
    o = _blocks(h, W2) + B2
    kept = np.broadcast_to(keep_mask(H, W, keep)[None, :, :, None, None], v.shape)
    rms_v = np.sqrt(np.mean(v.real ** 2 + v.imag ** 2) / 2)
    rms_o = np.sqrt(np.mean(o.real ** 2 + o.imag ** 2) / 2)
    out = []
    for part, (vp, op) in enumerate(((v.real, o.real), (v.imag, o.imag))):
        for idx in zip(*np.nonzero((np.abs(vp) <= band * rms_v) & kept)):
            out.append(("relu", part, tuple(int(i) for i in idx)))
        for idx in zip(*np.nonzero((np.abs(np.abs(op) - lam) <= band * rms_o) & kept)):
            out.append(("soft", part, tuple(int(i) for i in idx)))
    return out
