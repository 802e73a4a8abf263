"""GPU parity of the block MLP with a hidden size other than the block size
(afno_filter_forward_hidden) against the float64 oracle, whose hidden size comes from the
weights' shapes.  bf16 columns with H <= 96, block size 32, 64 or 96 and hidden = 2 bs run the
matrix-core hidden-size kernel under the automatic path; everything else, and every case
under the generic path, runs the size-generic column kernel.

Bars as the forward's: fp32 1e-4, bf16 2e-2, on out, on the filter's delta y (the float32
AFNO_STAGE_DELTA output of afno_filter_stage_hidden, which runs the same kernels up to the
inverse W-axis transform) and on the delta's rows h >= 1 at their own scale (the biases'
response is a spike on row 0).  The bf16 cases use weights of std 0.1 so that out also shows
the filter."""
import numpy as np
import pytest

import paper_2208_05419_amd as afno
from paper_2208_05419_amd import synth
from gpu_util import dev_weights, max_rel, off_row0_rel, oracle_run, say, to_dev, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    afno.load_library()


CASES = [
    # B, H, W, C, nb, hidden, dtype, lam, keep, weight_std
    (1, 16, 32, 64, 4, 32, "fp32", 0.01, 1.0, 0.02),
    (2, 12, 20, 64, 2, 64, "fp32", 0.01, 0.7, 0.02),
    (1, 30, 24, 128, 2, 32, "fp32", 0.01, 1.0, 0.02),      # hidden < block size
    (1, 45, 16, 128, 2, 128, "fp32", 0.02, 1.0, 0.02),
    (1, 20, 12, 64, 1, 256, "fp32", 0.01, 1.0, 0.02),      # eight waves, four groups each
    (1, 90, 180, 768, 8, 192, "bf16", 0.01, 1.0, 0.1),     # hidden factor 2 at 90 x 180
    (2, 25, 30, 96, 2, 96, "bf16", 0.01, 0.6, 0.1),
    (1, 1, 2, 32, 1, 64, "bf16", 0.01, 1.0, 0.1),
    # the matrix-core hidden-size kernel: each padded height and block size, ragged H, cutoff
    (2, 64, 40, 128, 2, 128, "bf16", 0.01, 0.7, 0.1),      # bs 64, H = HP = 64
    (1, 36, 20, 192, 2, 192, "bf16", 0.01, 1.0, 0.1),      # bs 96, HP 64, ragged
    (3, 18, 10, 64, 2, 64, "bf16", 0.02, 0.5, 0.1),        # bs 32, HP 32, cutoff
    (1, 96, 8, 96, 1, 192, "bf16", 0.01, 0.8, 0.1),        # bs 96, H = HP = 96
    (2, 72, 12, 128, 4, 64, "bf16", 0.01, 1.0, 0.1),       # bs 32, HP 96
]


def _mfma_case(H, C, nb, hs, dtype):
    bs = C // nb
    return dtype == "bf16" and H <= 96 and bs in (32, 64, 96) and hs == 2 * bs


@pytest.mark.parametrize("path", ["auto", "generic"])
@pytest.mark.parametrize("case", CASES, ids=lambda c: "B{}_H{}_W{}_C{}_nb{}_hs{}_{}_k{}".format(*c[:9]))
def test_hidden_parity(case, path):
    B, H, W, C, nb, hs, dtype, lam, keep, wstd = case
    if path == "generic" and not _mfma_case(H, C, nb, hs, dtype):
        pytest.skip("the automatic path already runs the generic kernel")
    wl = synth.Workload("hidden", B, H, W, C, nb, dtype, lam, keep, weight_std=wstd, hidden=hs)
    say(f"[hidden] B={B} {H}x{W}x{C} nb={nb} bs={C // nb} hidden={hs} {dtype} keep={keep} {path}")
    afno.set_kernel_path(afno.AFNO_PATH_AUTO if path == "auto" else afno.AFNO_PATH_GENERIC)
    try:
        _check_case(wl)
    finally:
        afno.set_kernel_path(afno.AFNO_PATH_AUTO)


def _check_case(wl):
    lam, keep, nb, dtype = wl.lam, wl.keep, wl.num_blocks, wl.dtype
    tol = 1e-4 if dtype == "fp32" else 2e-2
    x_st, w_st = synth.make_x(wl, seed=3), synth.make_weights(wl, seed=3)
    w = dev_weights(w_st, dtype)
    x = to_dev(x_st, dtype)
    out = afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], nb, lam, keep)
    delta = afno.filter_stage(x, w["w1"], w["b1"], w["w2"], w["b2"], nb, lam, keep,
                              afno.AFNO_STAGE_DELTA)
    torch.cuda.synchronize()
    ref, st = oracle_run(x_st, w_st, wl, stages=True)
    got, gd = to_f64(out), to_f64(delta)
    e_out = max_rel(got, ref)
    e_delta = max_rel(gd, st["delta"])
    e_rows = off_row0_rel(gd, st["delta"])
    say(f"  out {e_out:.2e}  delta {e_delta:.2e}  delta rows h>=1 {e_rows:.2e}")
    assert e_out <= tol and e_delta <= tol and e_rows <= tol


def test_hidden_equal_to_block_size_is_the_default_filter():
    """hidden == bs through afno_filter_forward_hidden runs the same kernels as
    afno_filter_forward: bitwise equal outputs."""
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"]
    x = to_dev(synth.make_x(wl), "bf16")
    w = dev_weights(synth.make_weights(wl), "bf16")
    a = afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam, wl.keep)
    b = torch.empty_like(x)
    rc = afno.afno_filter_forward_hidden(x.data_ptr(), w["w1"].data_ptr(), w["b1"].data_ptr(),
                                         w["w2"].data_ptr(), w["b2"].data_ptr(), wl.B, wl.H, wl.W,
                                         wl.C, wl.num_blocks, wl.C // wl.num_blocks, wl.lam,
                                         wl.keep, afno.AFNO_DTYPE_BF16, b.data_ptr(),
                                         torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert rc == afno.AFNO_OK
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_hidden_at_the_benchmark_configuration_sampled():
    """The benchmark's hidden-size workload (90 x 180 x 768, 8 blocks of 96, 192 hidden units,
    B = 4, channel-scaled fields, weights of std 0.02 as benchmarked): samples are independent
    through the filter, so samples 0 and 3 are compared against the oracle run on those two
    alone, on out, the delta and the delta's rows h >= 1."""
    wl = synth.WORKLOADS["afno90x180_c768_nb8_hs192_bf16_b4"]
    x_st, w_st = synth.make_x(wl), synth.make_weights(wl)
    w = dev_weights(w_st, "bf16")
    x = to_dev(x_st, "bf16")
    out = afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam, wl.keep)
    delta = afno.filter_stage(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam,
                              wl.keep, afno.AFNO_STAGE_DELTA)
    torch.cuda.synchronize()
    got, gd = to_f64(out)[[0, 3]], to_f64(delta)[[0, 3]]
    ref, st = oracle_run(x_st[[0, 3]], w_st, wl, stages=True)
    e_out = max_rel(got, ref)
    e_delta = max_rel(gd, st["delta"])
    e_rows = off_row0_rel(gd, st["delta"])
    say(f"[hidden] benchmark configuration, samples 0 and 3: out {e_out:.2e}  delta {e_delta:.2e}"
        f"  delta rows h>=1 {e_rows:.2e}")
    assert e_out <= 2e-2 and e_delta <= 2e-2 and e_rows <= 2e-2
