"""GPU parity of the filter's backward pass (afno_filter_backward) against the float64
backward oracle (oracle/backward.py), element by element with no allowance.

The gradients are step functions of two decisions per kept mode and unit: relu's (v > 0)
and the softshrink's (|o| > lam).  Where v or o sit within rounding distance of such a kink
either branch is correct, so the cases are built to have one correct result:

* known-mask cases (every bf16 case, the fp32 90 x 180 workload, the edge shapes and the
  benchmark configuration): x carries a few planted single-frequency components and b1, b2,
  lam are chosen from the exact forward state (oracle/known_masks.py) so that every kept
  mode's |v| and ||o| - lam| stay a dozen times the bf16 implementation's error away from the
  kinks.  The masks still change from mode to mode (planted modes against the rest).
* enumerated cases (fp32, random biases): the oracle lists the decisions within 2e-5 rms of a
  kink (the fp32 kernels' v and o stay within ~5e-6 rms of the exact values); there are at
  most six, and the GPU's gradients must match the oracle's for one of the 2^k assignments.

Bars (max |gpu - ref| / max |ref| per tensor): fp32 1e-4, bf16 2e-2, on dx, dw1, db1, dw2,
db2, and on the filter part dx - gout at its own scale.  For bf16 storage dx is rounded once
to bf16 after the residual add, so dx - gout is allowed that rounding (half a bf16 ulp of
|dx|) on top of the bar."""
import itertools

import numpy as np
import pytest

import paper_2208_05419_amd as afno
from oracle import backward as ob
from oracle import known_masks as km
from paper_2208_05419_amd import synth
from gpu_util import dev_weights, say, to_dev as _dev, to_f64

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TOL = {"fp32": 1e-4, "bf16": 2e-2}
NAMES = ("dx", "dw1", "db1", "dw2", "db2")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    afno.load_library()


def _gpu_grads(x_st, w_st, g_st, wl, lam):
    w = dev_weights(w_st, wl.dtype)
    got = afno.filter_backward(_dev(x_st, wl.dtype), w["w1"], w["b1"], w["w2"], w["b2"],
                               _dev(g_st, wl.dtype), wl.num_blocks, lam, wl.keep)
    torch.cuda.synchronize()
    return {k: to_f64(v) for k, v in got.items()}


def _errors(got, ref, g, dtype):
    """Relative error of every gradient, and of dx - g (bf16: beyond dx's output rounding)."""
    errs = {}
    for k in NAMES:
        den = float(np.max(np.abs(ref[k]))) or 1.0
        errs[k] = float(np.max(np.abs(got[k] - ref[k]))) / den
    fg, rg = got["dx"] - g, ref["dx"] - g
    den = float(np.max(np.abs(rg))) or 1.0
    slack = 0.0
    if dtype == "bf16":  # half an ulp of the stored dx: 2^-8 of its binade's lower end
        slack = np.ldexp(1.0, np.frexp(np.abs(ref["dx"]))[1] - 9)
    errs["dx-g"] = max(0.0, float(np.max(np.abs(fg - rg) - slack))) / den
    return errs


def _report(tag, wl, lam, errs):
    say(f"  {tag}: " + "  ".join(f"{k} {v:.2e}" for k, v in errs.items()))
    for k, v in errs.items():
        assert v <= TOL[wl.dtype], (k, v)


def _check_known(wl, seed=0, n_freq=4, amp=1.0):
    """Known-mask case: exact decisions, zero allowance."""
    say(f"[backward known-mask] {wl.name} B={wl.B} {wl.H}x{wl.W}x{wl.C} nb={wl.num_blocks} "
        f"{wl.dtype} keep={wl.keep} seed={seed}")
    rng = np.random.default_rng(7000 + seed)
    wide = lambda a: synth.widen(a, wl.dtype)  # noqa: E731
    x = wide(synth.make_x(wl, seed=seed))
    w = {k: wide(v) for k, v in synth.make_weights(wl, seed=seed).items()}
    x, planted = km.plant_frequencies(x, wl.dtype, wl.keep, n_freq, amp, rng)
    b1, b2, lam, info = km.choose_biases(x, w["w1"], w["w2"], wl.num_blocks, wl.keep, wl.dtype, rng)
    say(f"  lam {lam:.4g}; margins v {info['m1']:.3g} (min {info['min_dist_v']:.3g}), o "
        f"{info['m2']:.3g} (min {info['min_dist_o']:.3g}); units with mode-dependent relu / "
        f"softshrink masks {info['relu_mixed']:.2f} / {info['softshrink_mixed']:.2f}; "
        f"{len(planted)} planted modes")
    g = wide(synth.quantize(np.random.default_rng(1000 + seed).standard_normal(x.shape), wl.dtype))
    st = lambda a: synth.quantize(a, wl.dtype)  # noqa: E731 (exact: the values are stored ones)
    w_st = {"w1": st(w["w1"]), "b1": st(b1), "w2": st(w["w2"]), "b2": st(b2)}
    assert all(np.array_equal(wide(w_st[k]), v) for k, v in (("b1", b1), ("b2", b2)))
    got = _gpu_grads(st(x), w_st, st(g), wl, lam)
    ref = ob.filter_backward(x, w["w1"], b1, w["w2"], b2, g, wl.num_blocks, lam, wl.keep)
    _report("rel err", wl, lam, _errors(got, ref, g, wl.dtype))


def _check_enumerated(wl, seed=5, band=2e-5, max_kinks=6):
    """Random biases: the GPU must match the oracle for one assignment of the ambiguous
    decisions."""
    say(f"[backward enumerated] {wl.name} B={wl.B} {wl.H}x{wl.W}x{wl.C} nb={wl.num_blocks} "
        f"{wl.dtype} keep={wl.keep} seed={seed}")
    x_st, w_st = synth.make_x(wl, seed=seed), synth.make_weights(wl, seed=seed)
    g_st = synth.quantize(np.random.default_rng(1000 + seed).standard_normal(x_st.shape), wl.dtype)
    wide = lambda a: synth.widen(a, wl.dtype)  # noqa: E731
    x, g = wide(x_st), wide(g_st)
    w = [wide(w_st[k]) for k in ("w1", "b1", "w2", "b2")]
    amb = ob.ambiguous_decisions(x, *w, wl.num_blocks, wl.lam, wl.keep, band)
    say(f"  {len(amb)} decisions within {band:g} rms of a kink")
    assert len(amb) <= max_kinks, "case too kink-dense for enumeration"
    got = _gpu_grads(x_st, w_st, g_st, wl, wl.lam)
    best = None
    for r in range(len(amb) + 1):
        for sub in itertools.combinations(amb, r):
            ref = ob.filter_backward(x, *w, g, wl.num_blocks, wl.lam, wl.keep, flips=sub)
            errs = _errors(got, ref, g, wl.dtype)
            if best is None or max(errs.values()) < max(best[1].values()):
                best = (sub, errs)
    say(f"  best assignment flips {len(best[0])} of {len(amb)}")
    _report("rel err", wl, wl.lam, best[1])


def test_backward_small_fp32_known_masks():
    _check_known(synth.WORKLOADS["afno16x32_c64_nb4_fp32"])


def test_backward_small_fp32_enumerated():
    _check_enumerated(synth.WORKLOADS["afno16x32_c64_nb4_fp32"], seed=0)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("path", ["auto", "generic"])
def test_backward_90x180_fp32(path):
    """auto: the size-specialised W-axis kernels; generic: the size-generic ones."""
    afno.set_kernel_path(afno.AFNO_PATH_AUTO if path == "auto" else afno.AFNO_PATH_GENERIC)
    try:
        _check_known(synth.WORKLOADS["afno90x180_c768_nb8_fp32"])
    finally:
        afno.set_kernel_path(afno.AFNO_PATH_AUTO)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("path", ["auto", "valu"])
def test_backward_90x180_bf16_b2(path):
    """auto: the matrix-core backward column kernel; valu: the size-generic one."""
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"]
    afno.set_kernel_path(afno.AFNO_PATH_AUTO if path == "auto" else afno.AFNO_PATH_VALU_DFT)
    try:
        _check_known(synth.Workload("bwd_90x180_bf16_b2", 2, wl.H, wl.W, wl.C, wl.num_blocks,
                                    "bf16", wl.lam, 1.0, "channel_scaled"))
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


def _edge_id(c):
    return "B{}_H{}_W{}_C{}_nb{}_{}_k{}".format(c[0], c[1], c[2], c[3], c[4], c[5], c[7])


@pytest.mark.parametrize("case", EDGE, ids=_edge_id)
def test_backward_edge_shapes_known_masks(case):
    B, H, W, C, nb, dtype, lam, keep = case
    _check_known(synth.Workload("bwd_edge", B, H, W, C, nb, dtype, lam, keep), seed=5)


# fp32 shapes with random biases and at most six decisions within 2e-5 rms of a kink
ENUMERATED = [
    (1, 16, 40, 128, 1, "fp32", 0.005, 1.0),
    (1, 180, 24, 64, 2, "fp32", 0.01, 0.5),
    (2, 20, 24, 64, 2, "fp32", 0.01, 0.6),
]


@pytest.mark.parametrize("case", ENUMERATED, ids=_edge_id)
def test_backward_edge_shapes_enumerated(case):
    B, H, W, C, nb, dtype, lam, keep = case
    _check_enumerated(synth.Workload("bwd_enum", B, H, W, C, nb, dtype, lam, keep), seed=5)


def test_backward_nothing_kept_passes_gradient_through():
    wl = synth.Workload("bwd_none", 1, 8, 8, 32, 2, "fp32", 0.01, 0.1)
    x_st, w_st = synth.make_x(wl), synth.make_weights(wl)
    g_st = synth.quantize(np.random.default_rng(1000).standard_normal(x_st.shape), wl.dtype)
    got = _gpu_grads(x_st, w_st, g_st, wl, wl.lam)
    assert np.array_equal(got["dx"], synth.widen(g_st, wl.dtype))
    for k in ("dw1", "db1", "dw2", "db2"):
        assert not np.any(got[k])


@pytest.mark.timeout(1200)
def test_backward_at_the_benchmark_configuration():
    """The benchmark's backward: 90 x 180 x 768, 8 blocks of 96, bf16, B = 4, channel-scaled
    fields (the weight gradients sum over the batch, so all four samples are compared)."""
    _check_known(synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"])


@pytest.mark.parametrize("path,dtype,nb", [("auto", "bf16", 8), ("generic", "bf16", 8),
                                           ("auto", "fp32", 8), ("auto", "bf16", 6)])
def test_backward_repeats_bitwise(path, dtype, nb):
    """The weight and bias gradients are chunk sums stored without atomics and added in a fixed
    order, so two calls give the same bits: the slab weight product after the matrix-core and
    after the generic column kernel (bf16, 96-channel blocks), the size-generic weight product
    (fp32; bf16 with 128-channel blocks).  Random inputs: repeatability only."""
    wl = synth.Workload("bwd_rep", 2, 90, 180, 768, nb, dtype, 0.01, 1.0)
    x_st, w_st = synth.make_x(wl), synth.make_weights(wl)
    g_st = synth.quantize(np.random.default_rng(77).standard_normal(x_st.shape), wl.dtype)
    afno.set_kernel_path(afno.AFNO_PATH_AUTO if path == "auto" else afno.AFNO_PATH_GENERIC)
    try:
        w = dev_weights(w_st, wl.dtype)
        x, g = _dev(x_st, wl.dtype), _dev(g_st, wl.dtype)
        runs = []
        for _ in range(2):
            got = afno.filter_backward(x, w["w1"], w["b1"], w["w2"], w["b2"], g,
                                       wl.num_blocks, wl.lam, wl.keep)
            torch.cuda.synchronize()
            runs.append({k: v.clone() for k, v in got.items()})
    finally:
        afno.set_kernel_path(afno.AFNO_PATH_AUTO)
    for k in NAMES:
        assert torch.equal(runs[0][k], runs[1][k]), k
        assert bool(torch.isfinite(runs[0][k].float()).all()), k
    say(f"backward {path} {dtype} nb={nb}: two calls bitwise equal")
