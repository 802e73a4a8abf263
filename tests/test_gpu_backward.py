"""GPU parity of the filter's backward pass (afno_filter_backward) against the float64
backward oracle (oracle/backward.py), on the same seeded inputs and upstream gradients.

Metric: max over elements of (|gpu - ref| - allow) / max |ref| per tensor; dx also on its
filter part dx - gout for fp32.  Bars: fp32 1e-4, bf16 storage 2e-2 (the forward's).

The gradients are step functions of the pre-activations at relu's kink (v = 0) and the
softshrink's (|o| = lam).  An element whose pre-activation lies within rounding distance of
a kink may take either branch; allow is the oracle's elementwise bound on what such flips
can move (kink band below, relative to rms(v), rms(o)), zero wherever no ambiguous element
reaches.  The decisions themselves are taken in the kernel's precision: float64 for fp32
storage; for bf16 storage from the bf16-stored W-axis spectrum, spectrum and hidden layer
(without that, bf16 rounding alone moves 3-10 % of the weight gradients' max through
flipped decisions).  Bands: fp32 2e-5 (the kernels' v and o stay within ~5e-6 rms of the
exact values); bf16 3e-3: the spectrum the kernels round to bf16 carries their transform
error (fp32 FFT ~3e-7, the matrix-core split-table DFT ~4e-6 relative), so its rounding lands
one ulp away from the exactly rounded value in up to ~1 % of elements, and one such ulp of an
operand of up to 4 sigma moves o by up to ~1.1e-3 rms through the two weight layers (h's
own rounding likewise); the band covers about three coincident ones."""
import numpy as np
import pytest

import paper_2208_05419_amd as afno
from oracle import backward as ob
from paper_2208_05419_amd import synth
from gpu_util import dev_weights, max_rel as _rel, say, to_dev as _dev, to_f64

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    afno.load_library()


BAND = {"fp32": 2e-5, "bf16": 3e-3}
DECIDE = {"fp32": "exact", "bf16": "bf16"}


def _run(wl, seed=0):
    x_st, w_st = synth.make_x(wl, seed=seed), synth.make_weights(wl, seed=seed)
    rng = np.random.default_rng(1000 + seed)
    g_st = synth.quantize(rng.standard_normal(x_st.shape), wl.dtype)
    wide = lambda a: synth.widen(a, wl.dtype)  # noqa: E731
    ref = ob.filter_backward(wide(x_st), *(wide(w_st[k]) for k in ("w1", "b1", "w2", "b2")),
                             wide(g_st), wl.num_blocks, wl.lam, wl.keep, band=BAND[wl.dtype],
                             decide=DECIDE[wl.dtype])
    w = dev_weights(w_st, wl.dtype)
    got = afno.filter_backward(_dev(x_st, wl.dtype), w["w1"], w["b1"], w["w2"], w["b2"],
                               _dev(g_st, wl.dtype), wl.num_blocks, wl.lam, wl.keep)
    torch.cuda.synchronize()
    return {k: to_f64(v) for k, v in got.items()}, ref, wide(g_st)


def _excess(got, ref, allow):
    """max over elements of (|got - ref| - allow) / max |ref|, floored at 0."""
    den = float(np.max(np.abs(ref))) or 1.0
    return max(0.0, float(np.max(np.abs(got - ref) - allow)) / den)


def _check(wl, tol, seed=0):
    say(f"[backward] {wl.name} B={wl.B} {wl.H}x{wl.W}x{wl.C} nb={wl.num_blocks} {wl.dtype} "
        f"keep={wl.keep} seed={seed}")
    got, ref, g = _run(wl, seed)
    errs, plain = {}, {}
    for k in ("dx", "dw1", "db1", "dw2", "db2"):
        allow = ref.get("allow_" + k, 0.0)
        errs[k] = _excess(got[k], ref[k], allow)
        plain[k] = _rel(got[k], ref[k])
    if wl.dtype == "fp32":  # dx = g + filter part: the filter part alone, at its own scale
        errs["dx-g"] = _excess(got["dx"] - g, ref["dx"] - g, ref.get("allow_dx", 0.0))
        plain["dx-g"] = _rel(got["dx"] - g, ref["dx"] - g)
    say(f"  kinks in band: {ref.get('n_kinks', 0)}")
    say("  beyond allowance: " + "  ".join(f"{k} {v:.2e}" for k, v in errs.items()))
    say("  plain:            " + "  ".join(f"{k} {v:.2e}" for k, v in plain.items()))
    for k, v in errs.items():
        assert v <= tol, (k, v)


def test_backward_small_fp32():
    _check(synth.WORKLOADS["afno16x32_c64_nb4_fp32"], 1e-4)


@pytest.mark.parametrize("path", ["auto", "generic"])
def test_backward_90x180_fp32(path):
    """auto: the size-specialised W-axis kernels; generic: the size-generic ones."""
    afno.set_kernel_path(afno.AFNO_PATH_AUTO if path == "auto" else afno.AFNO_PATH_GENERIC)
    try:
        _check(synth.WORKLOADS["afno90x180_c768_nb8_fp32"], 1e-4)
    finally:
        afno.set_kernel_path(afno.AFNO_PATH_AUTO)


@pytest.mark.parametrize("path", ["auto", "valu"])
def test_backward_90x180_bf16_b2(path):
    """auto: the matrix-core backward column kernel; valu: the size-generic one."""
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"]
    afno.set_kernel_path(afno.AFNO_PATH_AUTO if path == "auto" else afno.AFNO_PATH_VALU_DFT)
    try:
        _check(synth.Workload("bwd_90x180_bf16_b2", 2, wl.H, wl.W, wl.C, wl.num_blocks, "bf16",
                              wl.lam, 1.0), 2e-2)
    finally:
        afno.set_kernel_path(afno.AFNO_PATH_AUTO)


EDGE = [
    # B, H, W, C, nb, dtype, lam, keep
    (2, 6, 10, 32, 2, "fp32", 0.01, 1.0),
    (1, 30, 8, 64, 2, "fp32", 0.02, 0.7),
    (2, 25, 50, 96, 2, "bf16", 0.01, 0.6),
    (1, 1, 2, 16, 1, "fp32", 0.01, 1.0),
    (1, 45, 360, 64, 4, "bf16", 0.01, 1.0),
    (1, 16, 40, 128, 1, "fp32", 0.005, 1.0),
    (3, 12, 16, 48, 1, "bf16", 0.01, 1.0),
    (1, 180, 20, 128, 2, "bf16", 0.01, 1.0),
    (1, 180, 24, 64, 2, "fp32", 0.01, 0.5),
    # bf16 shapes of the matrix-core backward column kernel: bs 32 / 64 / 96, padded heights
    # 32 / 64 / 96, ragged rows, keep < 1
    (2, 20, 24, 64, 2, "bf16", 0.01, 0.6),
    (1, 45, 50, 128, 2, "bf16", 0.01, 1.0),
    (1, 64, 16, 96, 1, "bf16", 0.02, 1.0),
    (2, 96, 8, 64, 1, "bf16", 0.01, 0.8),
    (1, 32, 10, 192, 2, "bf16", 0.01, 1.0),
]


@pytest.mark.parametrize("case", EDGE, ids=lambda c: "B{}_H{}_W{}_C{}_nb{}_{}_k{}".format(
    c[0], c[1], c[2], c[3], c[4], c[5], c[7]))
def test_backward_edge_shapes(case):
    B, H, W, C, nb, dtype, lam, keep = case
    _check(synth.Workload("bwd_edge", B, H, W, C, nb, dtype, lam, keep), 1e-4 if dtype == "fp32" else 2e-2,
           seed=5)


def test_backward_nothing_kept_passes_gradient_through():
    wl = synth.Workload("bwd_none", 1, 8, 8, 32, 2, "fp32", 0.01, 0.1)
    got, ref, g = _run(wl)
    assert np.array_equal(got["dx"], g)
    for k in ("dw1", "db1", "dw2", "db2"):
        assert not np.any(got[k])


def test_backward_at_the_benchmark_configuration():
    """The benchmark's backward: 90 x 180 x 768, 8 blocks of 96, bf16, B = 4, channel-scaled
    fields (the weight gradients sum over the batch, so all four samples are compared)."""
    _check(synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"], 2e-2)
