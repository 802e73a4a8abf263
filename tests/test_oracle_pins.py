"""Pins of the float64 oracle against facts fixed by mathematics, not by the oracle.

Each test names the reading of the paper it pins.  The paper (FourCastNet, section
"Model Innovations" and "Implementation Details" (b)) defines the filter as forward
FFT -> per-token block-diagonal complex MLP -> inverse FFT with real-to-complex /
complex-to-real transforms; softshrink, the hard cutoff and the residual follow the
AFNO layer it builds on.  No test here re-types an oracle formula: the expected
values come from closed forms, invariants, brute force, or numpy's independent FFT.
"""
import json
import os

import numpy as np
import pytest

import oracle

RNG = np.random.default_rng(1234)
TOL = 1e-11


def _rand(*shape):
    return RNG.standard_normal(shape)


def _crand(*shape):
    return RNG.standard_normal(shape) + 1j * RNG.standard_normal(shape)


def _zeros_weights(nb, bs):
    return (np.zeros((nb, bs, bs, 2)), np.zeros((nb, bs, 2)), np.zeros((nb, bs, bs, 2)),
            np.zeros((nb, bs, 2)))


def _cw(a):
    """complex array -> stored (re, im)-fastest float64 array"""
    a = np.asarray(a, dtype=np.complex128)
    return np.stack([a.real, a.imag], axis=-1)


# ---------------------------------------------------------------- transforms


@pytest.mark.parametrize("shape", [(2, 6, 10, 3), (1, 16, 32, 4), (1, 5, 8, 2), (1, 1, 2, 1),
                                   (1, 9, 12, 2)])
def test_round_trip(shape):
    x = _rand(*shape)
    y = oracle.irfft2(oracle.rfft2(x), shape[2])
    assert np.max(np.abs(y - x)) < TOL


@pytest.mark.parametrize("shape", [(2, 6, 10, 3), (1, 15, 20, 2)])
def test_parseval_half_spectrum(shape):
    """Ortho normalisation is unitary: sum x^2 = sum_k c_kw |X|^2 with c_0 = c_{W/2} = 1, else 2."""
    x = _rand(*shape)
    X = oracle.rfft2(x)
    W = shape[2]
    c = np.full(W // 2 + 1, 2.0)
    c[0] = 1.0
    c[-1] = 1.0  # W even
    lhs = np.sum(x * x, axis=(1, 2))
    rhs = np.sum(c[None, None, :, None] * np.abs(X) ** 2, axis=(1, 2))
    assert np.max(np.abs(lhs - rhs)) < 1e-10 * np.max(lhs)


def test_hermitian_symmetry():
    """Real input: X[kh, 0] = conj X[-kh, 0] and X[kh, W/2] = conj X[-kh, W/2]."""
    x = _rand(2, 9, 12, 3)
    X = oracle.rfft2(x)
    H = 9
    neg = (-np.arange(H)) % H
    for kw in (0, 6):
        assert np.max(np.abs(X[:, :, kw] - np.conj(X[:, neg, kw]))) < TOL


@pytest.mark.parametrize("shape", [(1, 4, 8, 3), (1, 16, 32, 2), (2, 6, 10, 2)])
def test_separable_equals_bruteforce_2d(shape):
    x = _rand(*shape)
    assert np.max(np.abs(oracle.rfft2(x) - oracle.dft2_bruteforce(x))) < TOL


@pytest.mark.parametrize("shape", [(1, 4, 8, 3), (1, 6, 10, 2)])
def test_inverse_equals_bruteforce_2d_nonhermitian(shape):
    B, H, W, C = shape
    Y = _crand(B, H, W // 2 + 1, C)  # arbitrary, not Hermitian on kw = 0, W/2
    assert np.max(np.abs(oracle.irfft2(Y, W) - oracle.idft2_bruteforce(Y, W))) < TOL


@pytest.mark.parametrize("shape", [(1, 90, 180, 2), (2, 16, 32, 3), (1, 30, 8, 2)])
def test_forward_matches_numpy_ortho(shape):
    x = _rand(*shape)
    ref = np.fft.rfft2(x, axes=(1, 2), norm="ortho")
    assert np.max(np.abs(oracle.rfft2(x) - ref)) < 1e-10


@pytest.mark.parametrize("shape", [(1, 6, 8, 2), (1, 90, 180, 1), (1, 5, 12, 2)])
def test_inverse_matches_numpy_ortho_nonhermitian(shape):
    """pocketfft's irfft2 drops the imaginary part of the kw=0 and kw=W/2 bins."""
    B, H, W, C = shape
    Y = _crand(B, H, W // 2 + 1, C)
    ref = np.fft.irfft2(Y, s=(H, W), axes=(1, 2), norm="ortho")
    assert np.max(np.abs(oracle.irfft2(Y, W) - ref)) < 1e-10


@pytest.mark.parametrize("a,b", [(2, 3), (0, 5), (3, 0), (0, 0), (4, 8), (7, 1)])
def test_single_frequency_bins(a, b):
    """x = cos(2pi(a h/H + b w/W)) has bins +-(a,b) of value sqrt(HW)/2 (or one bin of
    sqrt(HW) when they coincide); sin(...) gives -i sqrt(HW)/2 at (a,b) (forward sign -)."""
    H, W = 8, 16
    h = np.arange(H)[:, None]
    w = np.arange(W)[None, :]
    th = 2 * np.pi * (a * h / H + b * w / W)
    for fn, val in ((np.cos, 0.5), (np.sin, -0.5j)):
        x = fn(th)[None, :, :, None]
        X = oracle.rfft2(x)[0, :, :, 0]
        expect = np.zeros((H, W // 2 + 1), dtype=complex)
        n = np.sqrt(H * W)
        for (p, q, s) in ((a, b, 1.0), (-a, -b, -1.0)):
            p %= H
            q %= W
            if q <= W // 2:
                # conj bin of sin is +i sqrt(HW)/2
                expect[p, q] += n * (val if s > 0 else np.conj(val))
        assert np.max(np.abs(X - expect)) < 1e-10, (fn.__name__, a, b)


# ---------------------------------------------------------------- cutoff


def test_keep_counts_ensemble_grid():
    """90 x 180 grid, keep 0.5: 23 rows each side of 0 (45 rows) and 45 columns."""
    assert oracle.keep_counts(90, 180, 0.5) == (23, 45)
    m = oracle.keep_mask(90, 180, 0.5)
    rows = np.nonzero(m.any(axis=1))[0]
    assert list(rows) == list(range(0, 23)) + list(range(68, 90))
    assert list(np.nonzero(m.any(axis=0))[0]) == list(range(45))
    assert m.sum() == 2025
    assert oracle.keep_mask(90, 180, 1.0).all()
    assert oracle.keep_mask(16, 32, 1.0).all()


def test_cutoff_zeroes_outside_modes():
    nb, bs, H, W = 2, 4, 12, 16
    x = _rand(1, H, W, nb * bs)
    w = [_rand(nb, bs, bs, 2) * 0.3, _rand(nb, bs, 2) * 0.3, _rand(nb, bs, bs, 2) * 0.3,
         _rand(nb, bs, 2) * 0.3]
    _, full = oracle.filter_forward(x, *w, nb, 0.01, 1.0, stages=True)
    _, cut = oracle.filter_forward(x, *w, nb, 0.01, 0.5, stages=True)
    m = oracle.keep_mask(H, W, 0.5)
    assert 0 < m.sum() < m.size
    assert np.all(cut["spec_mlp"][:, ~m] == 0)
    assert np.max(np.abs(cut["spec_mlp"][:, m] - full["spec_mlp"][:, m])) == 0


def test_nothing_kept_gives_identity():
    nb, bs = 2, 4
    x = _rand(1, 16, 32, nb * bs)
    assert oracle.keep_counts(16, 32, 0.05) == (0, 0)
    w = [_rand(nb, bs, bs, 2), _rand(nb, bs, 2), _rand(nb, bs, bs, 2), _rand(nb, bs, 2)]
    out = oracle.filter_forward(x, *w, nb, 0.0, 0.05)
    assert np.array_equal(out, x)


def test_dc_only_closed_form():
    """Only mode (0,0) kept: out = x + Re(Y00)/sqrt(HW), Y00 = the MLP of the DC bin
    sum(x)/sqrt(HW), computed here with numpy complex arithmetic."""
    nb, bs, H, W = 2, 4, 16, 32
    keep = 0.115
    assert oracle.keep_counts(H, W, keep) == (1, 1)
    x = _rand(1, H, W, nb * bs)
    w1, b1, w2, b2 = (_crand(nb, bs, bs) * 0.4, _crand(nb, bs) * 0.4, _crand(nb, bs, bs) * 0.4,
                      _crand(nb, bs) * 0.4)
    lam = float(np.float32(0.05))  # the filter takes lambda as a float32
    out = oracle.filter_forward(x, _cw(w1), _cw(b1), _cw(w2), _cw(b2), nb,
                                lam, keep)
    n = np.sqrt(H * W)
    dc = x[0].sum(axis=(0, 1)) / n
    y = np.empty(nb * bs)
    for k in range(nb):
        v = b1[k] + dc[k * bs:(k + 1) * bs] @ w1[k]
        hid = np.maximum(v.real, 0) + 1j * np.maximum(v.imag, 0)
        o = b2[k] + hid @ w2[k]
        sr = np.sign(o.real) * np.maximum(np.abs(o.real) - lam, 0)
        y[k * bs:(k + 1) * bs] = sr / n
    assert np.max(np.abs(out - (x + y))) < 1e-12


# ---------------------------------------------------------------- MLP, softshrink, residual


def test_zero_weights_is_exact_identity():
    nb, bs = 3, 4
    x = _rand(2, 10, 12, nb * bs)
    out = oracle.filter_forward(x, *_zeros_weights(nb, bs), nb, 0.0, 1.0)
    assert np.array_equal(out, x)


def test_huge_lambda_is_exact_identity():
    nb, bs = 2, 4
    x = _rand(1, 6, 8, nb * bs)
    w = [_rand(nb, bs, bs, 2), _rand(nb, bs, 2), _rand(nb, bs, bs, 2), _rand(nb, bs, 2)]
    out = oracle.filter_forward(x, *w, nb, 1e6, 1.0)
    assert np.array_equal(out, x)


def _constant_spectrum_response(d, H, W):
    """y for the constant spectrum d on every stored mode (closed form):
    y[0, w] = (H / sqrt(HW)) * (Re d * W * [w == 0] - 2 Im d * sum_{k=1}^{W/2-1} sin(2 pi k w / W)),
    y[h != 0, w] = 0; the sine sum by the product identity
    sum_{k=1}^{n-1} sin(k t) = sin(n t / 2) sin((n - 1) t / 2) / sin(t / 2)."""
    n = W // 2
    w = np.arange(W)
    t = 2 * np.pi * w / W
    ssum = np.zeros(W)
    nz = w != 0
    ssum[nz] = np.sin(n * t[nz] / 2) * np.sin((n - 1) * t[nz] / 2) / np.sin(t[nz] / 2)
    y = np.zeros((H, W) + np.shape(d))
    pre = H / np.sqrt(H * W)
    y[0] = pre * (np.real(d)[None] * (W * (w == 0))[:, None] - 2 * np.imag(d)[None] * ssum[:, None])
    return y


def test_constant_spectrum_softshrink_and_c2r_convention():
    """w1 = w2 = 0, b2 = d, keep 1: every mode's output is S_lam(d); pins b2, the
    softshrink threshold (|v| = lam -> 0), its sign, and the C2R treatment of the
    imaginary parts at kw = 0 and kw = W/2."""
    nb, bs, H, W = 2, 4, 6, 10
    lam = 0.25
    b2 = np.array([[lam, -lam, lam + 0.5, -lam - 1.0], [0.0, 0.1, -0.3, 2.0 + lam]])
    b2i = np.array([[0.75 + lam, 0.0, -lam, -0.5 - lam], [lam + 1e-3, -2.0, 0.3, 0.01]])
    w1, b1, w2, _ = _zeros_weights(nb, bs)
    b1[...] = _rand(nb, bs, 2)
    b2s = np.stack([b2, b2i], axis=-1)
    x = _rand(1, H, W, nb * bs)
    out = oracle.filter_forward(x, w1, b1, w2, b2s, nb, lam, 1.0)

    def shrink(v):
        return np.where(v > lam, v - lam, np.where(v < -lam, v + lam, 0.0))

    d = (shrink(b2) + 1j * shrink(b2i)).reshape(-1)
    y = _constant_spectrum_response(d, H, W)
    assert np.max(np.abs(out[0] - x[0] - y)) < 1e-12


def test_relu_componentwise_and_layer2_complex_product():
    """w1 = 0: hidden = ReLU(Re b1) + i ReLU(Im b1); w2 = g * I (complex g): spectrum
    constant d = hidden * g (true complex product), lam = 0."""
    nb, bs, H, W = 1, 4, 4, 8
    b1 = np.array([[[0.5, -0.7], [-0.2, 0.3], [1.5, 2.0], [-1.0, -1.0]]])
    g = 0.8 - 0.6j
    w2 = np.zeros((nb, bs, bs), dtype=complex)
    w2[0] = g * np.eye(bs)
    w1 = np.zeros((nb, bs, bs, 2))
    x = _rand(1, H, W, bs)
    out = oracle.filter_forward(x, w1, b1, _cw(w2), np.zeros((nb, bs, 2)), nb, 0.0, 1.0)
    hid = np.maximum(b1[0, :, 0], 0) + 1j * np.maximum(b1[0, :, 1], 0)
    y = _constant_spectrum_response(hid * g, H, W)
    assert np.max(np.abs(out[0] - x[0] - y)) < 1e-12


def _linear_regime(w1c, w2c, beta):
    """b1 = beta(1+i) keeps every pre-activation positive (ReLU inactive); b2 cancels
    the bias that passes through layer 2, so the MLP is the linear map X -> X w1 w2."""
    nb, bs, hs = w1c.shape
    b1 = np.full((nb, hs), beta * (1 + 1j))
    b2 = -np.einsum("kj,kji->ki", b1, w2c)
    return _cw(w1c), _cw(b1), _cw(w2c), _cw(b2)


def test_linear_regime_real_block_matrix_is_token_local():
    """With real weights and ReLU inactive, the filter is out = x + x_blk @ (A @ Bm) for
    every token: a real channel map commutes with the 2-D DFT.  Non-symmetric A, Bm pin
    the input-major orientation (x @ W, not W @ x) and the block-diagonal structure."""
    nb, bs, H, W = 3, 4, 6, 8
    A = _rand(nb, bs, bs) * 0.2
    Bm = _rand(nb, bs, bs) * 0.2
    x = _rand(2, H, W, nb * bs)
    w = _linear_regime(A.astype(complex), Bm.astype(complex), 1e3)
    out = oracle.filter_forward(x, *w, nb, 0.0, 1.0)
    expect = x.copy()
    for k in range(nb):
        sl = slice(k * bs, (k + 1) * bs)
        expect[..., sl] += x[..., sl] @ (A[k] @ Bm[k])
    assert np.max(np.abs(out - expect)) < 1e-9


def test_linear_regime_complex_scalar_on_single_frequency():
    """w1 = diag(m), w2 = I, ReLU inactive, x_c = cos(theta): the stored bin (a,b) is
    multiplied by m, so y_c = Re(m e^{i theta}) = Re m cos(theta) - Im m sin(theta).
    Pins the layer-1 complex product and the forward(-)/inverse(+) signs together."""
    H, W, a, b = 8, 16, 3, 5
    m = np.array([0.3 + 0.9j, -0.4 + 0.2j])
    nb, bs = 1, 2
    w1c = np.zeros((nb, bs, bs), dtype=complex)
    w1c[0] = np.diag(m)
    w2c = np.eye(bs, dtype=complex)[None]
    h = np.arange(H)[:, None]
    ww = np.arange(W)[None, :]
    th = 2 * np.pi * (a * h / H + b * ww / W)
    x = np.repeat(np.cos(th)[None, :, :, None], bs, axis=3)
    out = oracle.filter_forward(x, *_linear_regime(w1c, w2c, 1e3), nb, 0.0, 1.0)
    for c in range(bs):
        expect = np.cos(th) + m[c].real * np.cos(th) - m[c].imag * np.sin(th)
        assert np.max(np.abs(out[0, :, :, c] - expect)) < 1e-9


def test_block_locality_exact():
    nb, bs, H, W = 4, 4, 6, 10
    x = _rand(1, H, W, nb * bs)
    w = [_rand(nb, bs, bs, 2) * 0.3, _rand(nb, bs, 2) * 0.3, _rand(nb, bs, bs, 2) * 0.3,
         _rand(nb, bs, 2) * 0.3]
    out = oracle.filter_forward(x, *w, nb, 0.01, 1.0)
    x2 = x.copy()
    x2[..., bs:2 * bs] += _rand(1, H, W, bs)
    out2 = oracle.filter_forward(x2, *w, nb, 0.01, 1.0)
    other = np.r_[0:bs, 2 * bs:nb * bs]
    assert np.array_equal(out[..., other], out2[..., other])
    assert not np.array_equal(out[..., bs:2 * bs], out2[..., bs:2 * bs])


def test_batch_independence_exact():
    nb, bs, H, W = 2, 4, 6, 8
    x = _rand(3, H, W, nb * bs)
    w = [_rand(nb, bs, bs, 2) * 0.3, _rand(nb, bs, 2) * 0.3, _rand(nb, bs, bs, 2) * 0.3,
         _rand(nb, bs, 2) * 0.3]
    out = oracle.filter_forward(x, *w, nb, 0.01, 0.8)
    for b in range(3):
        assert np.array_equal(out[b:b + 1], oracle.filter_forward(x[b:b + 1], *w, nb, 0.01, 0.8))


def test_stage_outputs_are_consistent():
    nb, bs, H, W = 2, 4, 6, 8
    x = _rand(1, H, W, nb * bs)
    w = [_rand(nb, bs, bs, 2) * 0.3, _rand(nb, bs, 2) * 0.3, _rand(nb, bs, bs, 2) * 0.3,
         _rand(nb, bs, 2) * 0.3]
    out, st = oracle.filter_forward(x, *w, nb, 0.02, 1.0, stages=True)
    assert np.max(np.abs(st["spec_fwd"] - np.fft.rfft2(x, axes=(1, 2), norm="ortho"))) < 1e-12
    assert np.max(np.abs(st["delta"] - np.fft.irfft2(st["spec_mlp"], s=(H, W), axes=(1, 2),
                                                    norm="ortho"))) < 1e-12
    assert np.array_equal(out, x + st["delta"])


def test_golden_tiny_fixture():
    """Regression pin: tests/golden/tiny_filter_4x8.json was written by
    tests/golden/make_golden.py, which calls only the oracle."""
    path = os.path.join(os.path.dirname(__file__), "golden", "tiny_filter_4x8.json")
    with open(path) as f:
        g = json.load(f)
    arr = {k: np.array(v, dtype=np.float64) for k, v in g["inputs"].items()}
    out = oracle.filter_forward(arr["x"], arr["w1"], arr["b1"], arr["w2"], arr["b2"],
                                g["num_blocks"], g["lam"], g["keep"])
    assert np.max(np.abs(out - np.array(g["out"]))) < 1e-12


# ---------------------------------------------------------------- hidden size != block size


@pytest.mark.parametrize("hs", [8, 2, 12])
def test_linear_regime_hidden_size(hs):
    """Hidden size hs != bs (w1 [nb][bs][hs], w2 [nb][hs][bs]): with real weights and ReLU
    inactive the filter is out = x + x_blk @ (A @ Bm) per token, A bs x hs, Bm hs x bs."""
    nb, bs, H, W = 2, 4, 6, 8
    A = _rand(nb, bs, hs) * 0.2
    Bm = _rand(nb, hs, bs) * 0.2
    x = _rand(1, H, W, nb * bs)
    out = oracle.filter_forward(x, *_linear_regime(A.astype(complex), Bm.astype(complex), 1e3),
                                nb, 0.0, 1.0)
    expect = x.copy()
    for k in range(nb):
        sl = slice(k * bs, (k + 1) * bs)
        expect[..., sl] += x[..., sl] @ (A[k] @ Bm[k])
    assert np.max(np.abs(out - expect)) < 1e-9


def test_hidden_units_with_zero_input_weights_drop_out():
    """Hidden units whose layer-1 weights and bias are zero stay at ReLU(0) = 0, so their
    layer-2 rows (set to non-zero values here) contribute nothing: an hs = 2 bs MLP whose
    second half is such units equals the hs = bs MLP of the first half, exactly."""
    nb, bs, H, W = 2, 4, 6, 10
    w1 = _rand(nb, bs, bs, 2) * 0.3
    b1 = _rand(nb, bs, 2) * 0.3
    w2 = _rand(nb, bs, bs, 2) * 0.3
    b2 = _rand(nb, bs, 2) * 0.3
    w1p = np.concatenate([w1, np.zeros((nb, bs, bs, 2))], axis=2)
    b1p = np.concatenate([b1, np.zeros((nb, bs, 2))], axis=1)
    w2p = np.concatenate([w2, _rand(nb, bs, bs, 2)], axis=1)
    x = _rand(2, H, W, nb * bs)
    ref = oracle.filter_forward(x, w1, b1, w2, b2, nb, 0.01, 0.8)
    out = oracle.filter_forward(x, w1p, b1p, w2p, b2, nb, 0.01, 0.8)
    assert np.array_equal(out, ref)


def test_hidden_unit_permutation_invariance():
    """Permuting the hidden units (w1 columns, b1 entries, w2 rows together) leaves the
    filter unchanged up to summation order."""
    nb, bs, hs, H, W = 2, 4, 10, 6, 8
    w1 = _rand(nb, bs, hs, 2) * 0.3
    b1 = _rand(nb, hs, 2) * 0.3
    w2 = _rand(nb, hs, bs, 2) * 0.3
    b2 = _rand(nb, bs, 2) * 0.3
    perm = RNG.permutation(hs)
    x = _rand(1, H, W, nb * bs)
    a = oracle.filter_forward(x, w1, b1, w2, b2, nb, 0.01, 1.0)
    b = oracle.filter_forward(x, w1[:, :, perm], b1[:, perm], w2[:, perm], b2, nb, 0.01, 1.0)
    assert np.max(np.abs(a - b)) < 1e-12
    # and a mismatched hidden size is rejected
    with pytest.raises(ValueError):
        oracle.filter_forward(x, w1, b1[:, :hs - 1], w2, b2, nb, 0.01, 1.0)
