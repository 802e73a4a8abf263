"""The allocation-free entry point (afno_filter_forward_noalloc) through the C ABI: on three
calls in a row -- the 90 x 180 x 768 bf16 workload with B = 4 (about 102 MB of the library's
128 MiB workspace), then smaller inputs that reuse the array the first call left behind -- its
output equals afno_filter_forward's bit for bit (the same kernels on the same inputs)."""
import numpy as np
import pytest

import paper_2208_05419_amd as afno
from paper_2208_05419_amd import synth
from gpu_util import dev_weights, say, to_dev

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    afno.load_library()


def _raw(fn, x, w, out, wl, stream):
    code = afno.AFNO_DTYPE_BF16 if wl.dtype == "bf16" else afno.AFNO_DTYPE_FP32
    return fn(x.data_ptr(), w["w1"].data_ptr(), w["b1"].data_ptr(), w["w2"].data_ptr(),
              w["b2"].data_ptr(), wl.B, wl.H, wl.W, wl.C, wl.num_blocks, wl.lam, wl.keep, code,
              out.data_ptr(), stream)


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


@pytest.mark.parametrize("order", ["large_first"])
def test_noalloc_equals_the_allocating_entry_point_on_calls_in_a_row(order):
    stream = torch.cuda.current_stream().cuda_stream
    cases = [synth.WORKLOADS["afno90x180_c768_nb8_bf16_b4"],
             synth.Workload("noalloc_small", 2, 30, 36, 192, 2, "bf16", 0.01, 0.6),
             synth.WORKLOADS["afno16x32_c64_nb4_fp32"]]
    for n, wl in enumerate(cases):
        say(f"[noalloc] call {n}: {wl.name} B={wl.B} {wl.H}x{wl.W}x{wl.C} nb={wl.num_blocks} "
            f"{wl.dtype} keep={wl.keep}")
        x = to_dev(synth.make_x(wl, seed=n), wl.dtype)
        w = dev_weights(synth.make_weights(wl, seed=n), wl.dtype)
        ref = torch.empty_like(x)
        got = torch.full_like(x, float("nan"))
        assert _raw(afno.afno_filter_forward, x, w, ref, wl, stream) == afno.AFNO_OK
        rc = _raw(afno.afno_filter_forward_noalloc, x, w, got, wl, stream)
        assert rc == afno.AFNO_OK, afno.afno_last_error()
        torch.cuda.synchronize()
        same = torch.equal(_bits(got), _bits(ref))
        say(f"  bitwise equal to afno_filter_forward: {same}")
        assert same


def test_noalloc_torch_wrapper_writes_the_callers_out():
    wl = synth.WORKLOADS["afno16x32_c64_nb4_fp32"]
    x = to_dev(synth.make_x(wl), wl.dtype)
    w = dev_weights(synth.make_weights(wl), wl.dtype)
    out = torch.empty_like(x)
    r = afno.filter_forward_noalloc(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam,
                                    wl.keep, out)
    ref = afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam, wl.keep)
    torch.cuda.synchronize()
    assert r is out and torch.equal(out, ref)
