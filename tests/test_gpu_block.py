"""GPU parity of one AFNO block (afno_block_forward: LayerNorm, the filter, LayerNorm, the
channel MLP C -> 4C -> C with GELU, residuals) against the float64 block oracle
(oracle/block.py) on the same stored bf16 inputs.

Bar: bf16 2e-2 (the filter's) on out and on out - x (the block's own contribution, of the
order of x since the filter adds LN1(x)); intermediates are rounded to bf16 four times
(t, the filter output, v, w) and the hidden layer once, each 2^-9 relative."""
import numpy as np
import pytest

import paper_2208_05419_amd as afno
from oracle import block as oblock
from paper_2208_05419_amd import synth
from gpu_util import max_rel, say, to_dev, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    afno.load_library()


CASES = [
    # B, H, W, C, nb, lam, keep, mlp_std
    (1, 6, 8, 128, 2, 0.01, 1.0, 0.02),
    (2, 12, 20, 128, 8, 0.01, 0.7, 0.02),      # 16-channel blocks, keep < 1
    (1, 1, 2, 128, 1, 0.01, 1.0, 0.05),        # two tokens: one ragged 128-row tile
    (3, 30, 36, 384, 4, 0.02, 0.5, 0.05),      # 3240 tokens: ragged last row tile
    (1, 45, 50, 256, 4, 0.01, 1.0, 0.1),       # the MLP dominates out - x
    (1, 90, 180, 768, 8, 0.01, 1.0, 0.02),     # the 90 x 180 x 768 block (16200 tokens)
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "B{}_H{}_W{}_C{}_nb{}_k{}_s{}".format(
    c[0], c[1], c[2], c[3], c[4], c[6], c[7]))
def test_block_parity(case):
    B, H, W, C, nb, lam, keep, mlp_std = case
    wl = synth.Workload("block", B, H, W, C, nb, "bf16", lam, keep)
    say(f"[block] B={B} {H}x{W}x{C} nb={nb} keep={keep} mlp_std={mlp_std}")
    x_st = synth.make_x(wl, seed=4)
    p_st = synth.make_block_params(wl, seed=4, mlp_std=mlp_std)
    x = to_dev(x_st, "bf16")
    p = {k: to_dev(v, "bf16") for k, v in p_st.items()}
    out = afno.block_forward(x, p, nb, lam, keep)
    torch.cuda.synchronize()
    wide = {k: synth.widen(v, "bf16") for k, v in p_st.items()}
    xs = synth.widen(x_st, "bf16")
    ref = oblock.block_forward(xs, *(wide[k] for k in afno.BLOCK_PARAMS), nb, lam, keep)
    got = to_f64(out)
    e_out, e_d = max_rel(got, ref), max_rel(got - xs, ref - xs)
    say(f"  out {e_out:.2e}  out-x {e_d:.2e}")
    assert e_out <= 2e-2 and e_d <= 2e-2


def test_block_deterministic():
    """No atomics: repeated calls are bitwise equal."""
    wl = synth.Workload("block", 1, 12, 20, 256, 4, "bf16", 0.01, 1.0)
    x = to_dev(synth.make_x(wl, seed=1), "bf16")
    p = {k: to_dev(v, "bf16") for k, v in synth.make_block_params(wl, seed=1).items()}
    a = afno.block_forward(x, p, 4, 0.01, 1.0)
    b = afno.block_forward(x, p, 4, 0.01, 1.0)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_block_at_the_benchmark_configuration_sampled():
    """The benchmark's block: 90 x 180 x 768, 8 blocks, B = 4, default parameters.  Samples
    are independent through the block (the filter per sample, LayerNorm and the MLP per
    token), so samples 0 and 3 are compared against the oracle run on those two alone."""
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"]
    x_st = synth.make_x(wl, seed=0)
    p_st = synth.make_block_params(wl, seed=0)
    x = to_dev(x_st, "bf16")
    p = {k: to_dev(v, "bf16") for k, v in p_st.items()}
    out = afno.block_forward(x, p, wl.num_blocks, wl.lam, wl.keep)
    torch.cuda.synchronize()
    got = to_f64(out)[[0, 3]]
    wide = {k: synth.widen(v, "bf16") for k, v in p_st.items()}
    xs = synth.widen(x_st, "bf16")[[0, 3]]
    ref = oblock.block_forward(xs, *(wide[k] for k in afno.BLOCK_PARAMS), wl.num_blocks, wl.lam,
                               wl.keep)
    e_out, e_d = max_rel(got, ref), max_rel(got - xs, ref - xs)
    say(f"[block] benchmark configuration, samples 0 and 3: out {e_out:.2e}  out-x {e_d:.2e}")
    assert e_out <= 2e-2 and e_d <= 2e-2
