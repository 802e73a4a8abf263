"""The allocation-free entry point (afno_filter_forward_noalloc) through the C ABI: on three
calls in a row -- the 90 x 180 x 768 bf16 workload with B = 4 (about 102 MB of the library's
128 MiB workspace), then smaller inputs that reuse the array the first call left behind -- its
output equals afno_filter_forward's bit for bit (the same kernels on the same inputs).  It is
for callers that cannot allocate, such as code under graph capture: recorded into a HIP graph
and replayed, it gives the same bits again."""
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


def test_noalloc_replays_from_a_captured_graph():
    """The allocation-free entry point recorded into a HIP graph (torch.cuda.graph) and replayed
    three times, with eager work and synchronisations between the replays and new input values
    before each: every replay's output equals an eager afno_filter_forward call on the same
    input, bit for bit."""
    wl = synth.Workload("noalloc_graph", 2, 30, 36, 192, 2, "bf16", 0.01, 1.0)
    x = to_dev(synth.make_x(wl, seed=7), wl.dtype)
    w = dev_weights(synth.make_weights(wl, seed=7), wl.dtype)
    out = torch.empty_like(x)
    s = torch.cuda.Stream()
    # an eager call first: the library's one-time set-up (kernel attributes, the scratch
    # array's address on this device) happens outside the capture
    assert _raw(afno.afno_filter_forward_noalloc, x, w, out, wl, s.cuda_stream) == afno.AFNO_OK
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    say("[noalloc graph] capture")
    with torch.cuda.graph(g, stream=s):
        rc = _raw(afno.afno_filter_forward_noalloc, x, w, out, wl, s.cuda_stream)
    assert rc == afno.AFNO_OK, afno.afno_last_error()
    torch.cuda.synchronize()
    cur = torch.cuda.current_stream().cuda_stream
    for rep in range(3):
        x.copy_(to_dev(synth.make_x(wl, seed=20 + rep), wl.dtype))  # eager work between replays
        torch.cuda.synchronize()
        say(f"[noalloc graph] replay {rep}")
        g.replay()
        torch.cuda.synchronize()
        ref = torch.empty_like(x)
        assert _raw(afno.afno_filter_forward, x, w, ref, wl, cur) == afno.AFNO_OK
        torch.cuda.synchronize()
        same = torch.equal(_bits(out), _bits(ref))
        say(f"  replay {rep} bitwise equal to afno_filter_forward: {same}")
        assert same
