"""Pins of the AFNO-block oracle (oracle/block.py) against closed forms and invariants: GELU
at points where Phi is known, LayerNorm's defining moments, the block with inert mixers, the
channel MLP in its linear regime, and token locality of the channel mixer.  CPU only."""
import math

import numpy as np
import pytest

import oracle
from oracle import block as ob

RNG = np.random.default_rng(77)


def test_gelu_known_values():
    """GELU(z) = z Phi(z): Phi(0) = 1/2, Phi(1) = 0.841344746068543 (normal table),
    Phi(-z) = 1 - Phi(z); for large |z| GELU tends to relu."""
    z = np.array([0.0, 1.0, -1.0, 2.0, -2.0, 8.0, -8.0])
    phi1, phi2 = 0.8413447460685429, 0.9772498680518208
    want = np.array([0.0, phi1, -(1 - phi1), 2 * phi2, -2 * (1 - phi2), 8.0, -0.0])
    assert np.max(np.abs(ob.gelu(z) - want)) < 1e-12


def test_layer_norm_moments_and_affine():
    """Unit gamma, zero beta: every token has mean 0 and biased variance var/(var + eps);
    gamma, beta then act channelwise."""
    C = 48
    z = RNG.standard_normal((3, 5, C)) * 3.0 + 1.5
    y = ob.layer_norm(z, np.ones(C), np.zeros(C))
    var = z.var(axis=-1)
    assert np.max(np.abs(y.mean(axis=-1))) < 1e-12
    assert np.max(np.abs(y.var(axis=-1) - var / (var + ob.LN_EPS))) < 1e-12
    g, b = RNG.standard_normal(C), RNG.standard_normal(C)
    assert np.max(np.abs(ob.layer_norm(z, g, b) - (y * g + b))) < 1e-12
    # a constant token normalises to beta
    assert np.max(np.abs(ob.layer_norm(np.full((1, C), 7.0), g, b) - b)) < 1e-12


def _filter_weights(nb, bs, s=0.0):
    return [RNG.standard_normal((nb, bs, bs, 2)) * s, RNG.standard_normal((nb, bs, 2)) * s,
            RNG.standard_normal((nb, bs, bs, 2)) * s, RNG.standard_normal((nb, bs, 2)) * s]


def test_inert_block_closed_form():
    """Zero filter weights with lam = 0 make the filter the identity on its input, and zero
    MLP weights make the channel mixer add bb: with unit gamma and zero beta, out - x - bb is
    the normalised token, so it has mean 0 and biased variance var/(var + eps) per token."""
    B, H, W, C, nb = 1, 6, 8, 32, 2
    x = RNG.standard_normal((B, H, W, C)) * 2.0 + 0.7
    bb = RNG.standard_normal(C)
    out = ob.block_forward(x, np.ones(C), np.zeros(C), *_filter_weights(nb, C // nb),
                           np.ones(C), np.zeros(C), np.zeros((C, 4 * C)), np.zeros(4 * C),
                           np.zeros((4 * C, C)), bb, nb, 0.0, 1.0)
    r = out - x - bb
    var = x.var(axis=-1)
    assert np.max(np.abs(r.mean(axis=-1))) < 1e-12
    assert np.max(np.abs(r.var(axis=-1) - var / (var + ob.LN_EPS))) < 1e-12


def test_channel_mlp_linear_regime_and_token_locality():
    """ba large and positive keeps every GELU argument far right of 0, where GELU(z) = z to
    double precision, so the mixer is the affine map w Wa Wb + (ba Wb + bb); and it acts on
    each token alone."""
    C, N = 16, 4 * 16
    w = RNG.standard_normal((2, 3, C))
    wa, wb = RNG.standard_normal((C, N)) * 0.1, RNG.standard_normal((N, C)) * 0.1
    ba, bb = np.full(N, 50.0), RNG.standard_normal(C)
    got = ob.channel_mlp(w, wa, ba, wb, bb)
    assert np.max(np.abs(got - (w @ wa @ wb + ba @ wb + bb))) < 1e-9
    w2 = w.copy()
    w2[1, 2] += 1.0
    got2 = ob.channel_mlp(w2, wa, ba, wb, bb)
    mask = np.ones((2, 3), bool)
    mask[1, 2] = False
    assert np.array_equal(got[mask], got2[mask])


def test_block_uses_the_filter_on_the_normalised_input():
    """With an inert channel mixer (zero weights and biases), out - x equals the filter of
    LN1(x): the spatial mixer sees the normalised tokens and its residual is kept."""
    B, H, W, C, nb = 1, 6, 10, 32, 2
    x = RNG.standard_normal((B, H, W, C)) * 2 + 0.5
    g1, b1 = RNG.standard_normal(C), RNG.standard_normal(C)
    fw = _filter_weights(nb, C // nb, 0.3)
    zc = np.zeros(C)
    out = ob.block_forward(x, g1, b1, *fw, np.ones(C), zc, np.zeros((C, 4 * C)), np.zeros(4 * C),
                           np.zeros((4 * C, C)), zc, nb, 0.01, 0.8)
    t = ob.layer_norm(x, g1, b1)
    assert np.max(np.abs(out - x - oracle.filter_forward(t, *fw, nb, 0.01, 0.8))) < 1e-12
