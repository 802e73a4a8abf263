"""The diagnostic per-phase timing (afno_profile_begin / afno_profile_end) on the GPU: the four
phase times of a few calls, the call count, and a preparation phase of exactly zero where the
preparation runs inside the W-axis forward launch."""
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


@pytest.mark.parametrize("path", ["auto", "generic"])
def test_profile_phases(path):
    wl = synth.Workload("profile", 2, 90, 180, 192, 2, "bf16", 0.01, 1.0)
    x = to_dev(synth.make_x(wl), wl.dtype)
    w = dev_weights(synth.make_weights(wl), wl.dtype)
    afno.set_kernel_path(afno.AFNO_PATH_AUTO if path == "auto" else afno.AFNO_PATH_GENERIC)
    try:
        afno.profile_begin(3)
        for _ in range(5):  # calls beyond the three are not timed
            afno.filter_forward(x, w["w1"], w["b1"], w["w2"], w["b2"], wl.num_blocks, wl.lam, wl.keep)
        torch.cuda.synchronize()
        ms, calls = afno.profile_end()
    finally:
        afno.set_kernel_path(afno.AFNO_PATH_AUTO)
    say(f"[profile] {path}: calls {calls}, ms {ms}")
    assert calls == 3
    assert set(ms) == set(afno.KERNELS)
    for k in ("row_r2c", "column", "row_c2r"):
        assert ms[k] > 0.0
    if path == "auto":  # the preparation runs as extra workgroups of the W-axis forward launch
        assert ms["prep"] == 0.0
    else:  # the generic path prepares nothing for its column kernel
        assert ms["prep"] >= 0.0
