"""Seeded random shapes against the float64 oracle: grids, channel splits, storage types,
cutoffs and thresholds drawn from fixed ranges with a fixed generator, so that combinations
nobody listed by hand (odd heights beside even widths, block sizes beside padded heights,
cutoffs that keep one row or one column) run through whichever kernels the automatic path
picks for them.  The draw is the same on every run (seed 2208); each case prints its shape.

Bars as the other parity tests: out, the filter's delta (float32 stage output) and the
delta's rows h >= 1 at their own scale within 1e-4 (fp32 storage) or 2e-2 (bf16), metric
max|g - r| / max|r|."""
import numpy as np
import pytest

import paper_2208_05419_amd as afno
from paper_2208_05419_amd import synth
from gpu_util import TOL, dev_weights, max_rel, off_row0_rel, oracle_run, say, to_dev, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

# 2^a 3^b 5^c sizes the kernels accept
SMOOTH_H = [1, 2, 3, 4, 5, 6, 8, 9, 10, 12, 15, 16, 18, 20, 24, 25, 27, 30, 32, 36, 40, 45,
            48, 50, 54, 60, 64, 72, 75, 80, 81, 90, 96]
SMOOTH_W = [2, 4, 6, 8, 10, 12, 16, 18, 20, 24, 30, 32, 36, 40, 48, 50, 54, 60, 64, 72, 90,
            96, 120, 180]


def _draw(n=20, seed=2208):
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        dtype = "bf16" if rng.random() < 0.6 else "fp32"
        if dtype == "bf16":  # mostly the matrix-core transform kernel's block sizes
            bs = int(rng.choice([32, 64, 96, 16, 48], p=[0.25, 0.25, 0.25, 0.125, 0.125]))
        else:
            bs = int(rng.choice([16, 32, 48, 64]))
        nb = int(rng.integers(1, 4))
        H = int(rng.choice(SMOOTH_H))
        W = int(rng.choice(SMOOTH_W))
        B = int(rng.integers(1, 4))
        keep = float(rng.choice([1.0, 1.0, 0.9, 0.5, 0.2]))
        lam = float(rng.choice([0.0, 0.005, 0.01, 0.02]))
        if B * H * W * nb * bs > 2_000_000:  # the oracle finishes each case in seconds
            continue
        cases.append((B, H, W, nb * bs, nb, dtype, lam, keep))
    return cases


CASES = _draw()


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    afno.load_library()


@pytest.mark.parametrize("case", CASES, ids=lambda c: "B{}_H{}_W{}_C{}_nb{}_{}_l{}_k{}".format(*c))
def test_random_shape(case):
    B, H, W, C, nb, dtype, lam, keep = case
    wl = synth.Workload("random", B, H, W, C, nb, dtype, lam, keep)
    say(f"[random] B={B} H={H} W={W} C={C} nb={nb} {dtype} lam={lam} keep={keep}")
    x_st, w_st = synth.make_x(wl, seed=H * 1000 + W), synth.make_weights(wl, seed=C + nb)
    x = to_dev(x_st, dtype)
    w = dev_weights(w_st, dtype)
    out = afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], nb, lam, keep)
    delta = afno.filter_stage(x, w["w1"], w["b1"], w["w2"], w["b2"], nb, lam, keep,
                              afno.AFNO_STAGE_DELTA)
    torch.cuda.synchronize()
    ref, st = oracle_run(x_st, w_st, wl, stages=True)
    e_out = max_rel(to_f64(out), ref)
    e_delta = max_rel(to_f64(delta), st["delta"])
    e_rows = off_row0_rel(to_f64(delta), st["delta"])
    say(f"  out rel {e_out:.3e}  delta rel {e_delta:.3e}  rows h>=1 {e_rows:.3e}  (tol {TOL[dtype]})")
    assert e_out <= TOL[dtype]
    assert e_delta <= TOL[dtype]
    assert e_rows <= TOL[dtype]
