"""GPU parity: the HIP path (through the C ABI) against the float64 oracle, element by
element on the same seeded stored inputs.

Bar (metric: max|g - r| / max|r| over the compared tensor, in float64):
  * fp32 storage: 1e-4 on out, and 1e-4 on the filter's delta y = out - x taken from the
    float32 AFNO_STAGE_DELTA entry point (out ~ x, so out alone barely sees the filter);
  * bf16 storage: 2e-2 on out and 2e-2 on the delta, the same way;
  * both: the delta's rows h >= 1 at their own scale (off_row0_rel): the biases' response is
    a spike on row 0 that would otherwise set the scale of the whole comparison.
Full-size workloads the oracle cannot finish in seconds are compared on sampled
outputs: whole channel blocks (blocks are independent) of the 180 x 360 grid, and
whole ensemble members of the 100-member batch.
"""
import numpy as np
import pytest

import paper_2208_05419_amd as afno
from paper_2208_05419_amd import synth
from gpu_util import TOL, dev_weights, max_rel, off_row0_rel, oracle_run, say, to_dev, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    afno.load_library()


_PATH = {"now": "auto"}


_PATHS = {"auto": afno.AFNO_PATH_AUTO, "valu": afno.AFNO_PATH_VALU_DFT,
          "generic": afno.AFNO_PATH_GENERIC}


@pytest.fixture(params=["auto", "valu", "generic"])
def kernel_path(request):
    """Run a test on the default kernels (auto: bf16 columns with H <= 96 take the
    matrix-core DFT kernel), on the same without that kernel (valu: vector-ALU FFT column
    kernels) and on the size-generic kernels."""
    afno.set_kernel_path(_PATHS[request.param])
    _PATH["now"] = request.param
    yield request.param
    afno.set_kernel_path(afno.AFNO_PATH_AUTO)
    _PATH["now"] = "auto"


def _skip_same_as_auto(kernel_path, dtype, H, bs):
    """valu differs from auto only where auto takes the matrix-core DFT column kernel."""
    if kernel_path == "valu" and not (dtype == "bf16" and H <= 96 and bs in (32, 64, 96)):
        pytest.skip("valu runs the same kernels as auto here")


def _run(x_st, w_st, wl, stage=None, keep=None):
    x = to_dev(x_st, wl.dtype)
    w = dev_weights(w_st, wl.dtype)
    keep = wl.keep if keep is None else keep
    if stage is None:
        out = afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam, keep)
    else:
        out = afno.filter_stage(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam, keep,
                                stage)
    torch.cuda.synchronize()
    return to_f64(out)


def _check_full(wl, x_st, w_st, label):
    say(f"[parity] {label}: B={x_st.shape[0]} H={wl.H} W={wl.W} C={wl.C} nb={wl.num_blocks} "
        f"{wl.dtype} keep={wl.keep} path={_PATH['now']}")
    g = _run(x_st, w_st, wl)
    r, st = oracle_run(x_st, w_st, wl, stages=True)
    x64 = synth.widen(x_st, wl.dtype)
    e_out = max_rel(g, r)
    # the delta through the float32 stage output: out - x would add out's own rounding
    # (half an ulp of |x|), which swamps a small delta
    gd = _run(x_st, w_st, wl, stage=afno.AFNO_STAGE_DELTA)
    e_delta = max_rel(gd, st["delta"])
    e_rows = off_row0_rel(gd, st["delta"])
    if wl.dtype == "fp32":
        assert max_rel(g - x64, st["delta"]) <= 2 * np.finfo(np.float32).eps * np.max(
            np.abs(x64)) / np.max(np.abs(st["delta"])) + TOL["fp32"]
    say(f"  out rel {e_out:.3e}  delta rel {e_delta:.3e}  delta rows h>=1 rel {e_rows:.3e}  "
        f"(tol {TOL[wl.dtype]})")
    assert e_out <= TOL[wl.dtype]
    assert e_delta <= TOL[wl.dtype]
    assert e_rows <= TOL[wl.dtype]
    return g, r, st


# ---------------------------------------------------------------- the five workloads


def test_afno16x32_fp32_full(kernel_path):
    wl = synth.WORKLOADS["afno16x32_c64_nb4_fp32"]
    _skip_same_as_auto(kernel_path, wl.dtype, wl.H, wl.bs)
    _check_full(wl, synth.make_x(wl), synth.make_weights(wl), wl.name)


def test_afno90x180_fp32_full(kernel_path):
    wl = synth.WORKLOADS["afno90x180_c768_nb8_fp32"]
    _skip_same_as_auto(kernel_path, wl.dtype, wl.H, wl.bs)
    _check_full(wl, synth.make_x(wl), synth.make_weights(wl), wl.name)


def test_afno90x180_bf16_b4_full(kernel_path):
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"]
    _skip_same_as_auto(kernel_path, wl.dtype, wl.H, wl.bs)
    _check_full(wl, synth.make_x(wl), synth.make_weights(wl), wl.name)


def test_afno180x360_bf16_sampled_blocks(kernel_path):
    """Full 1 x 180 x 360 x 1024 call; the oracle recomputes blocks 0 and 7 alone."""
    wl = synth.WORKLOADS["afno180x360_c1024_nb8_bf16"]
    _skip_same_as_auto(kernel_path, wl.dtype, wl.H, wl.bs)
    x_st, w_st = synth.make_x(wl), synth.make_weights(wl)
    say(f"[parity] {wl.name}: full GPU call, oracle on blocks 0 and 7")
    g = _run(x_st, w_st, wl)
    gd = _run(x_st, w_st, wl, stage=afno.AFNO_STAGE_DELTA)
    bs = wl.bs
    for k in (0, 7):
        sl = slice(k * bs, (k + 1) * bs)
        sub = synth.Workload(wl.name + f"_blk{k}", wl.B, wl.H, wl.W, bs, 1, wl.dtype, wl.lam, wl.keep)
        r, st = oracle_run(np.ascontiguousarray(x_st[..., sl]),
                           {n: np.ascontiguousarray(v[k:k + 1]) for n, v in w_st.items()}, sub,
                           stages=True)
        e_out, e_delta = max_rel(g[..., sl], r), max_rel(gd[..., sl], st["delta"])
        e_rows = off_row0_rel(gd[..., sl], st["delta"])
        say(f"  block {k}: out rel {e_out:.3e}  delta rel {e_delta:.3e}  rows h>=1 {e_rows:.3e}")
        assert e_out <= TOL["bf16"] and e_delta <= TOL["bf16"] and e_rows <= TOL["bf16"]


def test_afno180x360_nb32_paper_shape_sampled_blocks(kernel_path):
    """The paper's own filter shape (180 x 360 tokens, C = 1024 in 32 blocks of 32): full
    call, the oracle recomputes blocks 0, 13 and 31 alone."""
    wl = synth.WORKLOADS["afno180x360_c1024_nb32_bf16"]
    _skip_same_as_auto(kernel_path, wl.dtype, wl.H, wl.bs)
    x_st, w_st = synth.make_x(wl), synth.make_weights(wl)
    say(f"[parity] {wl.name}: full GPU call, oracle on blocks 0, 13, 31 (path {_PATH['now']})")
    g = _run(x_st, w_st, wl)
    gd = _run(x_st, w_st, wl, stage=afno.AFNO_STAGE_DELTA)
    bs = wl.bs
    for k in (0, 13, 31):
        sl = slice(k * bs, (k + 1) * bs)
        sub = synth.Workload(wl.name + f"_blk{k}", wl.B, wl.H, wl.W, bs, 1, wl.dtype, wl.lam, wl.keep)
        r, st = oracle_run(np.ascontiguousarray(x_st[..., sl]),
                           {n: np.ascontiguousarray(v[k:k + 1]) for n, v in w_st.items()}, sub,
                           stages=True)
        e_out, e_delta = max_rel(g[..., sl], r), max_rel(gd[..., sl], st["delta"])
        e_rows = off_row0_rel(gd[..., sl], st["delta"])
        say(f"  block {k}: out rel {e_out:.3e}  delta rel {e_delta:.3e}  rows h>=1 {e_rows:.3e}")
        assert e_out <= TOL["bf16"] and e_delta <= TOL["bf16"] and e_rows <= TOL["bf16"]


def test_afno90x180_bf16_ensemble100_keep05_sampled_members(kernel_path):
    """Full 100-member call with keep 0.5; the oracle recomputes members 0, 57 and 99."""
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_ens100_keep0.5"]
    say(f"[parity] {wl.name}: generating 100 members")
    x_st, w_st = synth.make_x(wl), synth.make_weights(wl)
    say("  full GPU call")
    g = _run(x_st, w_st, wl)
    gd = _run(x_st, w_st, wl, stage=afno.AFNO_STAGE_DELTA)
    for m in (0, 57, 99):
        assert np.array_equal(x_st[m], synth.make_x(wl, members=[m])[0])
        r, st = oracle_run(x_st[m:m + 1], w_st, wl, stages=True)
        e_out, e_delta = max_rel(g[m:m + 1], r), max_rel(gd[m:m + 1], st["delta"])
        e_rows = off_row0_rel(gd[m:m + 1], st["delta"])
        say(f"  member {m}: out rel {e_out:.3e}  delta rel {e_delta:.3e}  rows h>=1 {e_rows:.3e}")
        assert e_out <= TOL["bf16"] and e_delta <= TOL["bf16"] and e_rows <= TOL["bf16"]


# ---------------------------------------------------------------- per-stage parity


@pytest.mark.parametrize("name", ["afno16x32_c64_nb4_fp32", "afno90x180_c768_nb8_fp32"])
def test_stage_spectra_fp32(name, kernel_path):
    wl = synth.WORKLOADS[name]
    _skip_same_as_auto(kernel_path, wl.dtype, wl.H, wl.bs)
    x_st, w_st = synth.make_x(wl), synth.make_weights(wl)
    say(f"[stage] {name}")
    _, st = oracle_run(x_st, w_st, wl, stages=True)
    sp = _run(x_st, w_st, wl, stage=afno.AFNO_STAGE_SPECTRUM)
    mx = _run(x_st, w_st, wl, stage=afno.AFNO_STAGE_MIXED)
    e1 = max_rel(sp[..., 0] + 1j * sp[..., 1], st["spec_fwd"])
    e2 = max_rel(mx[..., 0] + 1j * mx[..., 1], st["spec_mlp"])
    say(f"  spectrum rel {e1:.3e}  mixed rel {e2:.3e}")
    assert e1 <= 1e-5 and e2 <= 1e-4


def test_stage_spectra_bf16(kernel_path):
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"]
    x_st, w_st = synth.make_x(wl), synth.make_weights(wl)
    x_st = x_st[:1]
    say("[stage] bf16 90x180x768 B=1")
    _, st = oracle_run(x_st, w_st, wl, stages=True)
    sp = _run(x_st, w_st, wl, stage=afno.AFNO_STAGE_SPECTRUM)
    mx = _run(x_st, w_st, wl, stage=afno.AFNO_STAGE_MIXED)
    e1 = max_rel(sp[..., 0] + 1j * sp[..., 1], st["spec_fwd"])
    e2 = max_rel(mx[..., 0] + 1j * mx[..., 1], st["spec_mlp"])
    say(f"  spectrum rel {e1:.3e}  mixed rel {e2:.3e}")
    assert e1 <= 1e-2 and e2 <= 2e-2


def test_stage_mixed_180x360_sampled_blocks(kernel_path):
    """The mixed spectrum Y (after the block MLP, softshrink and cutoff) of the full
    1 x 180 x 360 x 1024 call, blocks 0 and 7 against the oracle run on each block alone."""
    wl = synth.WORKLOADS["afno180x360_c1024_nb8_bf16"]
    _skip_same_as_auto(kernel_path, wl.dtype, wl.H, wl.bs)
    x_st, w_st = synth.make_x(wl), synth.make_weights(wl)
    say(f"[stage] {wl.name}: mixed spectrum, oracle on blocks 0 and 7 (path {_PATH['now']})")
    mx = _run(x_st, w_st, wl, stage=afno.AFNO_STAGE_MIXED)
    bs = wl.bs
    for k in (0, 7):
        sl = slice(k * bs, (k + 1) * bs)
        sub = synth.Workload(wl.name + f"_blk{k}", wl.B, wl.H, wl.W, bs, 1, wl.dtype, wl.lam, wl.keep)
        _, st = oracle_run(np.ascontiguousarray(x_st[..., sl]),
                           {n: np.ascontiguousarray(v[k:k + 1]) for n, v in w_st.items()}, sub,
                           stages=True)
        e2 = max_rel(mx[..., sl, 0] + 1j * mx[..., sl, 1], st["spec_mlp"])
        say(f"  block {k}: mixed rel {e2:.3e}")
        assert e2 <= TOL["bf16"]


def test_stage_mixed_ensemble_sampled_members(kernel_path):
    """The mixed spectrum of ensemble members 0, 57 and 99 (keep 0.5): the stage entry point
    runs the same kernels on those three members as a batch of three (members are independent
    through the filter; the whole 100-member spectrum in float32 would take 5 GB)."""
    wl = synth.WORKLOADS["afno90x180_c768_nb8_bf16_ens100_keep0.5"]
    _skip_same_as_auto(kernel_path, wl.dtype, wl.H, wl.bs)
    x_st, w_st = synth.make_x(wl, members=[0, 57, 99]), synth.make_weights(wl)
    say(f"[stage] {wl.name}: mixed spectrum of members 0, 57, 99 (path {_PATH['now']})")
    mx = _run(x_st, w_st, wl, stage=afno.AFNO_STAGE_MIXED)
    _, st = oracle_run(x_st, w_st, wl, stages=True)
    for n, m in enumerate((0, 57, 99)):
        e2 = max_rel(mx[n:n + 1, ..., 0] + 1j * mx[n:n + 1, ..., 1], st["spec_mlp"][n:n + 1])
        say(f"  member {m}: mixed rel {e2:.3e}")
        assert e2 <= TOL["bf16"]


# ---------------------------------------------------------------- ragged, small and edge shapes

EDGE = [
    # B, H, W, C, nb, dtype, lam, keep
    (3, 6, 10, 32, 2, "fp32", 0.01, 1.0),
    (3, 6, 10, 32, 2, "bf16", 0.01, 1.0),
    (2, 30, 8, 64, 2, "fp32", 0.02, 0.7),
    (1, 1, 2, 16, 1, "fp32", 0.01, 1.0),
    (2, 25, 50, 96, 2, "fp32", 0.01, 1.0),
    (1, 25, 50, 96, 2, "bf16", 0.01, 0.6),
    (1, 192, 64, 128, 1, "bf16", 0.01, 1.0),
    (1, 108, 64, 128, 1, "fp32", 0.01, 1.0),
    (2, 25, 50, 48, 1, "bf16", 0.01, 1.0),
    (1, 4, 1024, 16, 1, "fp32", 0.01, 1.0),
    (1, 45, 360, 64, 4, "bf16", 0.01, 1.0),
    (2, 18, 24, 64, 1, "fp32", 0.005, 1.0),
    (1, 81, 12, 80, 5, "fp32", 0.01, 0.9),
    # grids with size-specialised W kernels but generic column kernels, and the reverse
    (2, 30, 180, 64, 2, "bf16", 0.01, 1.0),
    (1, 90, 32, 192, 2, "fp32", 0.01, 0.8),
    (1, 16, 360, 96, 1, "bf16", 0.01, 0.5),
    (3, 16, 40, 64, 4, "bf16", 0.01, 1.0),
    # bf16 columns on the matrix-core DFT kernel: padded heights 32 / 64 / 96 with block
    # sizes 32 / 64 / 96, padding rows (H < HP), cutoffs, and the degenerate H = 1, 2
    (1, 96, 24, 128, 2, "bf16", 0.01, 1.0),
    (2, 50, 20, 192, 2, "bf16", 0.01, 0.8),
    (1, 64, 16, 64, 2, "bf16", 0.02, 1.0),
    (2, 27, 30, 128, 2, "bf16", 0.01, 1.0),
    (1, 75, 12, 32, 1, "bf16", 0.01, 0.5),
    (1, 60, 32, 128, 2, "bf16", 0.01, 1.0),
    (2, 1, 4, 64, 2, "bf16", 0.01, 1.0),
    (1, 2, 6, 32, 1, "bf16", 0.01, 1.0),
    # more padded-height-96 shapes: odd H, block size 96 with two blocks, block size 32
    (1, 81, 10, 96, 1, "bf16", 0.01, 0.7),
    (2, 72, 8, 192, 2, "bf16", 0.01, 1.0),
    (1, 80, 6, 64, 2, "bf16", 0.01, 1.0),
    # the kept-row matrix-core kernel (bf16, block size 96, 64 < H <= 96, at most 48 kept
    # rows): 45, 27, 7 and 1 kept rows, ragged H, two blocks
    (2, 90, 20, 192, 2, "bf16", 0.01, 0.5),
    (1, 96, 8, 96, 1, "bf16", 0.02, 0.3),
    (1, 81, 10, 96, 1, "bf16", 0.01, 0.1),
    (2, 72, 40, 96, 1, "bf16", 0.01, 0.05),
    (1, 75, 30, 96, 1, "bf16", 0.01, 0.6),
    (1, 80, 16, 192, 2, "bf16", 0.005, 0.55),
    # H = 180 columns with the size-specialised vector-ALU transform kernels at block
    # sizes 32 (fp32 and bf16) and 64 (bf16), with and without a cutoff
    (1, 180, 24, 64, 2, "fp32", 0.01, 1.0),
    (2, 180, 12, 64, 2, "bf16", 0.01, 0.7),
    (1, 180, 20, 128, 2, "bf16", 0.01, 1.0),
    # W-axis slices: the W = 180 forward on 32 channels and inverse on 64 (fp32: full 128-byte
    # lines; channels not a multiple of 64 fall back to the generic W passes), W = 360 on 32
    # channels (bf16 pairs of slices per line, a single slice per row, fp32)
    (1, 20, 180, 128, 2, "fp32", 0.01, 1.0),
    (1, 12, 180, 32, 1, "bf16", 0.01, 1.0),
    (2, 9, 180, 96, 1, "bf16", 0.01, 0.8),
    (1, 12, 360, 32, 1, "fp32", 0.01, 0.7),
    (2, 10, 360, 32, 1, "bf16", 0.01, 1.0),
]


@pytest.mark.parametrize("case", EDGE, ids=lambda c: "B{}_H{}_W{}_C{}_nb{}_{}_k{}".format(
    c[0], c[1], c[2], c[3], c[4], c[5], c[7]))
def test_edge_shapes(case):
    B, H, W, C, nb, dtype, lam, keep = case
    wl = synth.Workload("edge", B, H, W, C, nb, dtype, lam, keep)
    _check_full(wl, synth.make_x(wl, seed=5), synth.make_weights(wl, seed=5), str(case))


def _zero_weights(wl):
    z = lambda *s: synth.quantize(np.zeros(s), wl.dtype)  # noqa: E731
    bs = wl.bs
    return {"w1": z(wl.num_blocks, bs, bs, 2), "b1": z(wl.num_blocks, bs, 2),
            "w2": z(wl.num_blocks, bs, bs, 2), "b2": z(wl.num_blocks, bs, 2)}


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_zero_weights_bit_exact_identity(dtype, kernel_path):
    wl = synth.Workload("zero", 2, 90, 180, 128, 2, dtype, 0.0, 1.0)
    _skip_same_as_auto(kernel_path, dtype, wl.H, wl.bs)
    say(f"[edge] zero weights {dtype}")
    x_st = synth.make_x(wl)
    g = _run(x_st, _zero_weights(wl), wl)
    assert np.array_equal(g, synth.widen(x_st, dtype))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_nothing_kept_bit_exact_identity(dtype, kernel_path):
    wl = synth.Workload("cut", 2, 16, 32, 64, 4, dtype, 0.01, 0.05)
    _skip_same_as_auto(kernel_path, dtype, wl.H, wl.bs)
    say(f"[edge] nothing kept {dtype}")
    x_st = synth.make_x(wl)
    g = _run(x_st, synth.make_weights(wl), wl)
    assert np.array_equal(g, synth.widen(x_st, dtype))


def test_dc_only_cutoff(kernel_path):
    wl = synth.Workload("dc", 2, 16, 32, 64, 4, "fp32", 0.01, 0.115)
    _skip_same_as_auto(kernel_path, wl.dtype, wl.H, wl.bs)
    _check_full(wl, synth.make_x(wl), synth.make_weights(wl), "DC-only cutoff")


def test_matrix_core_and_valu_transforms_both_run():
    """bf16, H = 90, bs = 96: the default path (matrix-core DFT column kernel) and
    AFNO_PATH_VALU_DFT (vector-ALU FFT column kernel) both meet the bar and round
    differently, so each really ran its own kernel."""
    wl = synth.Workload("paths", 1, 90, 32, 192, 2, "bf16", 0.01, 1.0)
    x_st, w_st = synth.make_x(wl, seed=9), synth.make_weights(wl, seed=9)
    r = oracle_run(x_st, w_st, wl)
    got = {}
    try:
        for name in ("auto", "valu"):
            afno.set_kernel_path(_PATHS[name])
            got[name] = _run(x_st, w_st, wl)
            e = max_rel(got[name], r)
            say(f"[paths] {name}: out rel {e:.3e}")
            assert e <= TOL["bf16"]
    finally:
        afno.set_kernel_path(afno.AFNO_PATH_AUTO)
    assert not np.array_equal(got["auto"], got["valu"])


def test_batch_zero_is_noop():
    rc = afno.afno_filter_forward(None, None, None, None, None, 0, 16, 32, 64, 4, 0.01, 1.0,
                                  afno.AFNO_DTYPE_FP32, None, torch.cuda.current_stream().cuda_stream)
    assert rc == afno.AFNO_OK


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_deterministic_bitwise(dtype, kernel_path):
    wl = synth.Workload("det", 2, 90, 180, 192, 2, dtype, 0.01, 1.0)
    _skip_same_as_auto(kernel_path, dtype, wl.H, wl.bs)
    say(f"[edge] determinism {dtype}")
    x = to_dev(synth.make_x(wl), dtype)
    w = dev_weights(synth.make_weights(wl), dtype)
    a = afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam, 1.0)
    b = afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam, 1.0)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16) if dtype == "bf16" else a.view(torch.int32),
                       b.view(torch.int16) if dtype == "bf16" else b.view(torch.int32))


def test_non_default_stream():
    wl = synth.WORKLOADS["afno16x32_c64_nb4_fp32"]
    say("[edge] non-default stream")
    x_st, w_st = synth.make_x(wl), synth.make_weights(wl)
    x = to_dev(x_st, wl.dtype)
    w = dev_weights(w_st, wl.dtype)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        out = afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam,
                                  wl.keep, stream=s)
    s.synchronize()
    r = oracle_run(x_st, w_st, wl)
    assert max_rel(to_f64(out), r) <= TOL["fp32"]


def test_alias_rejected_and_nothing_written():
    wl = synth.WORKLOADS["afno16x32_c64_nb4_fp32"]
    x = to_dev(synth.make_x(wl), wl.dtype)
    w = dev_weights(synth.make_weights(wl), wl.dtype)
    before = x.clone()
    with pytest.raises(afno.AfnoError) as ei:
        afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam, 1.0, out=x)
    assert ei.value.code == afno.AFNO_ERR_ALIAS
    torch.cuda.synchronize()
    assert torch.equal(x, before)
