"""C ABI checks that need no GPU: the library loads, exports every function the header
declares, and rejects bad arguments before any HIP call (validation runs first, so
these calls never reach the device).  Pointers here are fake, aligned integers."""
import math
import os
import re

import pytest

import paper_2208_05419_amd as afno

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# fake device addresses, 256-byte aligned and far apart
X, W1, B1, W2, B2, OUT = (0x10000000 * (i + 1) for i in range(6))


def _header_functions():
    with open(os.path.join(ROOT, "include", "afno.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(afno_\w+)\s*\(", text)))


def test_library_loads_and_exports_header_symbols():
    lib = afno.load_library()
    names = _header_functions()
    assert set(names) == set(afno.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_version():
    assert afno.afno_version() == 100


def call(**kw):
    a = dict(x=X, w1=W1, b1=B1, w2=W2, b2=B2, B=1, H=16, W=32, C=64, nb=4, lam=0.01, keep=1.0,
             dtype=afno.AFNO_DTYPE_FP32, out=OUT, stream=None)
    a.update(kw)
    return afno.afno_filter_forward(a["x"], a["w1"], a["b1"], a["w2"], a["b2"], a["B"], a["H"],
                                    a["W"], a["C"], a["nb"], a["lam"], a["keep"], a["dtype"],
                                    a["out"], a["stream"])


@pytest.mark.parametrize("kw", [
    dict(x=None), dict(w1=None), dict(b1=None), dict(w2=None), dict(b2=None), dict(out=None),
    dict(H=0), dict(W=-2), dict(C=0), dict(nb=0), dict(B=-1), dict(C=64, nb=3),
    dict(lam=-0.1), dict(lam=math.nan), dict(lam=math.inf), dict(keep=0.0), dict(keep=1.5),
    dict(keep=math.nan), dict(keep=-0.5), dict(dtype=2), dict(dtype=-1),
])
def test_invalid_arguments(kw):
    assert call(**kw) == afno.AFNO_ERR_INVALID_ARG
    assert afno.afno_last_error() != ""


@pytest.mark.parametrize("kw", [
    dict(H=7), dict(W=14), dict(W=33), dict(H=11, W=22),          # not 2,3,5-smooth / odd W
    dict(C=96, nb=4),                                              # bs = 24, not a multiple of 16
    dict(C=512, nb=2),                                             # bs = 256 > 128
    dict(H=256),                                                   # H > 192
    dict(W=2048),                                                  # W > 1024
    dict(x=X + 8), dict(out=OUT + 4), dict(w1=W1 + 2),             # misaligned
    dict(dtype=afno.AFNO_DTYPE_FP32, H=192, W=64, C=256, nb=2),   # fp32 tile 192 x 128 over LDS
])
def test_unsupported(kw):
    assert call(**kw) == afno.AFNO_ERR_UNSUPPORTED
    assert afno.afno_last_error() != ""


@pytest.mark.parametrize("kw", [
    dict(out=X), dict(out=X + 16 * 32 * 64 * 4 - 16), dict(out=W1), dict(out=B2 - 16),
    dict(out=X - 16),
])
def test_alias(kw):
    assert call(**kw) == afno.AFNO_ERR_ALIAS


def test_batch_zero_is_ok_without_gpu():
    assert call(B=0, x=None, out=None) == afno.AFNO_OK
    assert afno.afno_last_error() == ""


def test_batch_zero_still_validates_scalars():
    assert call(B=0, C=64, nb=3) == afno.AFNO_ERR_INVALID_ARG


def test_stage_validation():
    f = afno.afno_filter_stage
    assert f(X, W1, B1, W2, B2, 1, 16, 32, 64, 4, 0.01, 1.0, 0, 9, OUT, None) == afno.AFNO_ERR_INVALID_ARG
    assert f(X, W1, B1, W2, B2, 1, 16, 32, 64, 4, 0.01, 1.0, 0, afno.AFNO_STAGE_DELTA, X,
             None) == afno.AFNO_ERR_ALIAS
    assert f(X, W1, B1, W2, B2, 1, 16, 32, 64, 4, 0.01, 1.0, 0, afno.AFNO_STAGE_SPECTRUM,
             OUT + 8, None) == afno.AFNO_ERR_UNSUPPORTED


def test_error_message_is_thread_local_and_cleared():
    import threading
    assert call(H=0) == afno.AFNO_ERR_INVALID_ARG
    msgs = []
    t = threading.Thread(target=lambda: msgs.append(afno.afno_last_error()))
    t.start()
    t.join()
    assert msgs == [""]
    assert afno.afno_last_error() != ""
    assert call(B=0) == afno.AFNO_OK
    assert afno.afno_last_error() == ""


def test_missing_library_raises(monkeypatch, tmp_path):
    import paper_2208_05419_amd.afno as mod
    monkeypatch.setattr(mod, "_lib", None)
    monkeypatch.setattr(mod, "LIB_PATH", str(tmp_path / "nope.so"))
    with pytest.raises(RuntimeError, match="not built"):
        mod.load_library()


def test_kernel_path_switch_validation():
    assert afno.afno_set_kernel_path(7) == afno.AFNO_ERR_INVALID_ARG
    assert afno.afno_set_kernel_path(afno.AFNO_PATH_GENERIC) == afno.AFNO_OK
    assert afno.afno_set_kernel_path(afno.AFNO_PATH_VALU_DFT) == afno.AFNO_OK
    assert afno.afno_set_kernel_path(afno.AFNO_PATH_AUTO) == afno.AFNO_OK


G, DX, DW1, DB1, DW2, DB2 = (0x10000000 * (i + 8) for i in range(6))


def call_bwd(**kw):
    a = dict(x=X, w1=W1, b1=B1, w2=W2, b2=B2, g=G, B=1, H=16, W=32, C=64, nb=4, lam=0.01, keep=1.0,
             dtype=afno.AFNO_DTYPE_FP32, dx=DX, dw1=DW1, db1=DB1, dw2=DW2, db2=DB2)
    a.update(kw)
    return afno.afno_filter_backward(a["x"], a["w1"], a["b1"], a["w2"], a["b2"], a["g"], a["B"],
                                     a["H"], a["W"], a["C"], a["nb"], a["lam"], a["keep"],
                                     a["dtype"], a["dx"], a["dw1"], a["db1"], a["dw2"], a["db2"],
                                     None)


@pytest.mark.parametrize("kw", [dict(g=None), dict(dx=None), dict(dw1=None), dict(db2=None),
                                dict(C=64, nb=3), dict(lam=-1.0)])
def test_backward_invalid_arguments(kw):
    assert call_bwd(**kw) == afno.AFNO_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [dict(g=G + 8), dict(dw1=DW1 + 2), dict(H=7), dict(C=512, nb=2)])
def test_backward_unsupported(kw):
    assert call_bwd(**kw) == afno.AFNO_ERR_UNSUPPORTED


@pytest.mark.parametrize("kw", [dict(dx=G), dict(dx=X), dict(dw1=W1), dict(dw2=DW1 + 64),
                                dict(db1=G + 128), dict(db2=DX)])
def test_backward_alias(kw):
    assert call_bwd(**kw) == afno.AFNO_ERR_ALIAS


def call_hidden(**kw):
    a = dict(x=X, w1=W1, b1=B1, w2=W2, b2=B2, B=1, H=16, W=32, C=64, nb=4, hidden=32, lam=0.01,
             keep=1.0, dtype=afno.AFNO_DTYPE_FP32, out=OUT)
    a.update(kw)
    return afno.afno_filter_forward_hidden(a["x"], a["w1"], a["b1"], a["w2"], a["b2"], a["B"],
                                           a["H"], a["W"], a["C"], a["nb"], a["hidden"], a["lam"],
                                           a["keep"], a["dtype"], a["out"], None)


@pytest.mark.parametrize("kw", [dict(hidden=0), dict(hidden=-16), dict(w1=None), dict(nb=3)])
def test_hidden_invalid_arguments(kw):
    assert call_hidden(**kw) == afno.AFNO_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [dict(hidden=24), dict(hidden=272), dict(H=180, C=256, nb=2, hidden=256)])
def test_hidden_unsupported(kw):
    assert call_hidden(**kw) == afno.AFNO_ERR_UNSUPPORTED


def test_hidden_alias_covers_the_wider_weights():
    # w1 is nb * bs * hidden * 2 * 4 = 4 * 16 * 32 * 8 = 16 KiB: out 12 KiB after w1 overlaps it
    assert call_hidden(out=W1 + 12 * 1024) == afno.AFNO_ERR_ALIAS
    assert call_hidden(out=B1 + 256) == afno.AFNO_ERR_ALIAS   # b1: 4 * 32 * 8 = 1 KiB


LN = [0x10000000 * (i + 20) for i in range(8)]  # ln1_g, ln1_b, ln2_g, ln2_b, wa, ba, wb, bb


def call_block(**kw):
    a = dict(x=X, w1=W1, b1=B1, w2=W2, b2=B2, ln1_g=LN[0], ln1_b=LN[1], ln2_g=LN[2], ln2_b=LN[3],
             wa=LN[4], ba=LN[5], wb=LN[6], bb=LN[7], B=1, H=16, W=32, C=128, nb=4, lam=0.01,
             keep=1.0, dtype=afno.AFNO_DTYPE_BF16, out=OUT)
    a.update(kw)
    return afno.afno_block_forward(a["x"], a["ln1_g"], a["ln1_b"], a["w1"], a["b1"], a["w2"],
                                   a["b2"], a["ln2_g"], a["ln2_b"], a["wa"], a["ba"], a["wb"],
                                   a["bb"], a["B"], a["H"], a["W"], a["C"], a["nb"], a["lam"],
                                   a["keep"], a["dtype"], a["out"], None)


@pytest.mark.parametrize("kw", [dict(ln1_g=None), dict(wb=None), dict(x=None), dict(C=128, nb=3),
                                dict(dtype=7), dict(lam=float("nan"))])
def test_block_invalid_arguments(kw):
    assert call_block(**kw) == afno.AFNO_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [dict(dtype=afno.AFNO_DTYPE_FP32), dict(C=64, nb=4),
                                dict(C=4096, nb=32), dict(ln2_b=LN[3] + 8), dict(H=7)])
def test_block_unsupported(kw):
    assert call_block(**kw) == afno.AFNO_ERR_UNSUPPORTED


@pytest.mark.parametrize("kw", [dict(out=LN[4] + 64), dict(out=X), dict(out=W2 + 16)])
def test_block_alias(kw):
    assert call_block(**kw) == afno.AFNO_ERR_ALIAS


def test_block_empty_batch_is_ok_without_the_gpu():
    assert call_block(B=0, x=None, out=None) == afno.AFNO_OK


def test_binding_rejects_mismatched_weight_shapes_before_any_gpu_call():
    """filter_forward reads the hidden size from w1 and checks every weight shape first."""
    torch = pytest.importorskip("torch")
    x = torch.zeros((1, 4, 8, 32))
    nb, bs, hs = 2, 16, 32
    ok = dict(w1=torch.zeros((nb, bs, hs, 2)), b1=torch.zeros((nb, hs, 2)),
              w2=torch.zeros((nb, hs, bs, 2)), b2=torch.zeros((nb, bs, 2)))
    for bad in (dict(b1=torch.zeros((nb, bs, 2))), dict(w2=torch.zeros((nb, bs, bs, 2))),
                dict(b2=torch.zeros((nb, hs, 2)))):
        w = dict(ok, **bad)
        with pytest.raises(ValueError, match="weight shapes"):
            afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], nb, 0.01)
    with pytest.raises(ValueError, match="GPU"):  # well-formed, but host tensors
        afno.filter_forward(x, ok["w1"], ok["b1"], ok["w2"], ok["b2"], nb, 0.01)


def test_spectrum_column_span_beyond_32_bit_offsets_is_rejected():
    """One column of the spectrum (H rows of kept_w * C complex values) must stay within the
    kernels' 32-bit byte offsets: 90 x 91 x C x 4 bytes (bf16) crosses 2^32 between
    C = 131072 and C = 132096 (block size 128)."""
    bf = afno.AFNO_DTYPE_BF16
    below = dict(H=90, W=180, C=131072, nb=1024, dtype=bf)
    above = dict(H=90, W=180, C=132096, nb=1032, dtype=bf)
    assert 90 * 91 * 131072 * 4 < 2 ** 32 <= 90 * 91 * 132096 * 4
    assert call(**above) == afno.AFNO_ERR_UNSUPPORTED
    assert "4 GiB" in afno.afno_last_error()
    # below the limit the plan is accepted up to the last check (out overlapping x)
    assert call(out=X, **below) == afno.AFNO_ERR_ALIAS
    # keep < 1 shrinks the column: the same C then fits
    assert call(out=X, keep=0.5, **above) == afno.AFNO_ERR_ALIAS


def _host_weights(torch, nb, bs, hs, dtype):
    return dict(w1=torch.zeros((nb, bs, hs, 2), dtype=dtype), b1=torch.zeros((nb, hs, 2), dtype=dtype),
                w2=torch.zeros((nb, hs, bs, 2), dtype=dtype), b2=torch.zeros((nb, bs, 2), dtype=dtype))


def test_binding_backward_rejects_a_hidden_size_other_than_the_block_size():
    """The backward kernels run hidden = block size; weights of another hidden size would be
    read (and gradients written) beyond their ends, so the binding refuses them first."""
    torch = pytest.importorskip("torch")
    x = torch.zeros((1, 4, 8, 192))
    w = _host_weights(torch, 2, 96, 48, torch.float32)
    with pytest.raises(ValueError, match="shape"):
        afno.filter_backward(x, w["w1"], w["b1"], w["w2"], w["b2"], torch.zeros_like(x), 2, 0.01)
    w = _host_weights(torch, 2, 96, 96, torch.float32)
    with pytest.raises(ValueError, match="gout"):
        afno.filter_backward(x, w["w1"], w["b1"], w["w2"], w["b2"], torch.zeros((1, 4, 8, 96)), 2,
                             0.01)


def test_binding_rejects_weights_of_another_dtype_or_device():
    torch = pytest.importorskip("torch")
    x = torch.zeros((1, 4, 8, 32))
    w = _host_weights(torch, 2, 16, 16, torch.bfloat16)   # fp32 x, bf16 weights
    with pytest.raises(TypeError, match="dtype"):
        afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], 2, 0.01)
    with pytest.raises(TypeError, match="dtype"):
        afno.filter_backward(x, w["w1"], w["b1"], w["w2"], w["b2"], torch.zeros_like(x), 2, 0.01)
    xm = torch.zeros((1, 4, 8, 32), device="meta")     # weights on another device than x
    w = _host_weights(torch, 2, 16, 16, torch.float32)
    with pytest.raises(ValueError, match="device|meta"):
        afno.filter_forward(xm, w["w1"], w["b1"], w["w2"], w["b2"], 2, 0.01)
    with pytest.raises(ValueError, match="contiguous"):
        wt = dict(w, w1=torch.zeros((2, 16, 16, 2)).transpose(1, 2))
        afno.filter_forward(x, wt["w1"], wt["b1"], wt["w2"], wt["b2"], 2, 0.01)
    with pytest.raises(ValueError, match="out"):
        afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], 2, 0.01,
                            out=torch.zeros((1, 4, 8, 16)))
    with pytest.raises(ValueError, match="num_blocks"):
        afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], 3, 0.01)
    with pytest.raises(ValueError, match=r"\[B, H, W, C\]"):
        afno.filter_forward(x[0], w["w1"], w["b1"], w["w2"], w["b2"], 2, 0.01)


def test_binding_stage_checks_weights_and_takes_the_hidden_size_from_w1():
    torch = pytest.importorskip("torch")
    x = torch.zeros((1, 4, 8, 32))
    w = _host_weights(torch, 2, 16, 32, torch.float32)
    with pytest.raises(ValueError, match="shape"):
        afno.filter_stage(x, w["w1"], w["b2"], w["w2"], w["b2"], 2, 0.01, 1.0, afno.AFNO_STAGE_DELTA)
    with pytest.raises(ValueError, match="GPU"):   # well-formed hidden weights, host tensors
        afno.filter_stage(x, w["w1"], w["b1"], w["w2"], w["b2"], 2, 0.01, 1.0, afno.AFNO_STAGE_DELTA)


def test_binding_block_checks_every_parameter_shape():
    torch = pytest.importorskip("torch")
    C, nb = 128, 4
    x = torch.zeros((1, 4, 8, C), dtype=torch.bfloat16)
    bf = torch.bfloat16
    p = dict(_host_weights(torch, nb, C // nb, C // nb, bf))
    p.update({k: torch.zeros(C, dtype=bf) for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "bb")})
    p.update(wa=torch.zeros((C, 4 * C), dtype=bf), ba=torch.zeros(4 * C, dtype=bf),
             wb=torch.zeros((4 * C, C), dtype=bf))
    for k, bad in (("wa", torch.zeros((4 * C, C), dtype=bf)), ("ba", torch.zeros(C, dtype=bf)),
                   ("ln2_g", torch.zeros(C + 1, dtype=bf)), ("w1", torch.zeros((nb, 32, 64, 2), dtype=bf))):
        with pytest.raises(ValueError, match=k):
            afno.block_forward(x, dict(p, **{k: bad}), nb, 0.01)
    with pytest.raises(TypeError, match="dtype"):
        afno.block_forward(x, dict(p, bb=torch.zeros(C)), nb, 0.01)
    with pytest.raises(ValueError, match="missing"):
        afno.block_forward(x, {k: v for k, v in p.items() if k != "wb"}, nb, 0.01)
    with pytest.raises(ValueError, match="GPU"):   # well-formed, host tensors
        afno.block_forward(x, p, nb, 0.01)


def call_stage_hidden(**kw):
    a = dict(x=X, w1=W1, b1=B1, w2=W2, b2=B2, B=1, H=16, W=32, C=64, nb=4, hidden=32, lam=0.01,
             keep=1.0, dtype=afno.AFNO_DTYPE_FP32, stage=afno.AFNO_STAGE_DELTA, dst=OUT)
    a.update(kw)
    return afno.afno_filter_stage_hidden(a["x"], a["w1"], a["b1"], a["w2"], a["b2"], a["B"],
                                         a["H"], a["W"], a["C"], a["nb"], a["hidden"], a["lam"],
                                         a["keep"], a["dtype"], a["stage"], a["dst"], None)


def test_stage_hidden_validation():
    assert call_stage_hidden(hidden=0) == afno.AFNO_ERR_INVALID_ARG
    assert call_stage_hidden(stage=7) == afno.AFNO_ERR_INVALID_ARG
    assert call_stage_hidden(hidden=24) == afno.AFNO_ERR_UNSUPPORTED
    assert call_stage_hidden(dst=OUT + 8) == afno.AFNO_ERR_UNSUPPORTED
    # w1 of the hidden size: 4 * 16 * 32 * 8 bytes = 16 KiB, so dst 8 KiB in overlaps it
    assert call_stage_hidden(dst=W1 + 8192) == afno.AFNO_ERR_ALIAS
    assert call_stage_hidden(B=0, x=None, dst=None) == afno.AFNO_OK


def call_noalloc(**kw):
    a = dict(x=X, w1=W1, b1=B1, w2=W2, b2=B2, B=1, H=16, W=32, C=64, nb=4, lam=0.01, keep=1.0,
             dtype=afno.AFNO_DTYPE_FP32, out=OUT, stream=None)
    a.update(kw)
    return afno.afno_filter_forward_noalloc(a["x"], a["w1"], a["b1"], a["w2"], a["b2"], a["B"],
                                            a["H"], a["W"], a["C"], a["nb"], a["lam"], a["keep"],
                                            a["dtype"], a["out"], a["stream"])


def test_noalloc_validates_like_the_forward_and_bounds_its_workspace():
    """Validation before any HIP call: the forward's checks, then the fixed workspace's bound
    (128 MiB; the 90 x 180 x 768 bf16 filter needs B * 100.6 MB of spectrum plus 1.2 MB of
    prepared operands, so B = 6 does not fit)."""
    assert call_noalloc(H=0) == afno.AFNO_ERR_INVALID_ARG
    assert call_noalloc(H=7) == afno.AFNO_ERR_UNSUPPORTED
    assert call_noalloc(out=X) == afno.AFNO_ERR_ALIAS
    assert call_noalloc(B=0, x=None, out=None) == afno.AFNO_OK
    bf = dict(H=90, W=180, C=768, nb=8, dtype=afno.AFNO_DTYPE_BF16)
    assert call_noalloc(B=6, **bf) == afno.AFNO_ERR_UNSUPPORTED
    assert "exceeds" in afno.afno_last_error()
    assert call_noalloc(B=50, **bf) == afno.AFNO_ERR_UNSUPPORTED
