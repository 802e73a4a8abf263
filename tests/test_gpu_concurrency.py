"""Calls from several host threads at once, each on its own stream (default priority).

The C ABI keeps no per-call state outside the call: each call validates, plans and takes a
stream-ordered workspace of its own, and the kernel path a call uses is fixed when its plan is
made.  So concurrent calls on different streams must give, bit for bit, what the same calls
give one after another; and switching the kernel path while other threads are calling must
leave every call's output equal to the output of one of the two paths."""
import threading

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


def _inputs(wl, seed):
    return to_dev(synth.make_x(wl, seed=seed), wl.dtype), dev_weights(synth.make_weights(wl, seed=seed), wl.dtype)


def _call(wl, x, w, stream):
    return afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam,
                               wl.keep, stream=stream)


def _run_threads(jobs, iters):
    """jobs: [(wl, x, w, want_set)], one thread each; every output must bitwise equal one of
    want_set's tensors.  Returns the failures as strings."""
    errors = []

    def worker(i, wl, x, w, wants):
        s = torch.cuda.Stream()
        try:
            for it in range(iters):
                with torch.cuda.stream(s):
                    out = _call(wl, x, w, s)
                s.synchronize()
                if not any(torch.equal(out.view(torch.int16 if out.dtype == torch.bfloat16
                                                else torch.int32),
                                       ref.view(torch.int16 if ref.dtype == torch.bfloat16
                                                else torch.int32)) for ref in wants):
                    errors.append(f"thread {i} ({wl.name}) iteration {it}: output differs")
                    return
        except Exception as e:  # noqa: BLE001 -- reported to the main thread
            errors.append(f"thread {i} ({wl.name}): {e!r}")

    ts = [threading.Thread(target=worker, args=(i, *job)) for i, job in enumerate(jobs)]
    for t in ts:
        t.start()
    for t in ts:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in ts), "a worker thread did not finish"
    return errors


def test_concurrent_calls_on_separate_streams_match_sequential():
    wls = [synth.Workload("c_bf16", 2, 90, 180, 768, 8, "bf16", 0.01, 1.0),
           synth.Workload("c_fp32", 2, 16, 32, 64, 4, "fp32", 0.01, 0.8),
           synth.Workload("c_bf16_keep", 1, 30, 48, 192, 2, "bf16", 0.02, 0.6)]
    say("[concurrency] three threads, three streams, three shapes")
    jobs = []
    for i, wl in enumerate(wls):
        x, w = _inputs(wl, 20 + i)
        ref = _call(wl, x, w, None)
        torch.cuda.synchronize()
        jobs.append((wl, x, w, [ref.clone()]))
    errors = _run_threads(jobs, iters=12)
    assert not errors, errors


def test_switching_the_kernel_path_during_calls():
    """One thread flips the path between automatic and generic while two others call on
    their own streams: each call runs one path end to end (its workspace was sized for the
    kernels it launches), so every output equals that path's sequential output."""
    wl = synth.Workload("c_switch", 1, 90, 180, 768, 8, "bf16", 0.01, 1.0)
    say("[concurrency] kernel path switched while two threads call")
    x, w = _inputs(wl, 31)
    refs = []
    try:
        for path in (afno.AFNO_PATH_AUTO, afno.AFNO_PATH_GENERIC):
            afno.set_kernel_path(path)
            refs.append(_call(wl, x, w, None).clone())
            torch.cuda.synchronize()
        stop = threading.Event()

        def flipper():
            k = 0
            while not stop.is_set():
                afno.set_kernel_path(afno.AFNO_PATH_GENERIC if k % 2 else afno.AFNO_PATH_AUTO)
                k += 1
                stop.wait(0.002)

        f = threading.Thread(target=flipper)
        f.start()
        try:
            errors = _run_threads([(wl, x, w, refs), (wl, x, w, refs)], iters=10)
        finally:
            stop.set()
            f.join(timeout=10)
    finally:
        afno.set_kernel_path(afno.AFNO_PATH_AUTO)
    assert not errors, errors
