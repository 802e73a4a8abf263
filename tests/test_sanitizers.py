"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Two builds into a temporary directory:
  * the HIP library with its host code instrumented (hipcc, each -fsanitize= behind
    -Xarch_host: the device code is built as usual), driven through the C ABI on the argument
    validation and plan paths that run before any HIP call -- invalid arguments, unsupported
    shapes, aliasing, the 32-bit span guard, the allocation-free entry point's bound;
  * the float64 oracle (gcc), run on small filters, stages and backward pieces and compared
    with the regular build.
Each runs in a child process with the sanitizer runtime preloaded; a sanitizer report makes
the child fail.  The HIP build takes about a minute."""
import os
import shutil
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2208_05419_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _clang_asan_runtime():
    out = subprocess.run([HIPCC, "--print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True)
    path = out.stdout.strip()
    if out.returncode == 0 and os.path.isabs(path) and os.path.exists(path):
        return path
    import glob
    found = glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    return found[0] if found else None


@pytest.fixture(scope="module")
def builds(tmp_path_factory):
    if not os.path.exists(HIPCC) or shutil.which("gcc") is None:
        pytest.skip("hipcc or gcc missing")
    rt = _clang_asan_runtime()
    if rt is None:
        pytest.skip("clang ASan runtime missing")
    d = tmp_path_factory.mktemp("sanitized")
    lib = str(d / "libafno_asan.so")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-shared-libsan", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I" + os.path.join(ROOT, "include"), "-I" + CSRC, "-x", "hip", os.path.join(CSRC, "afno_kernels.hip"), "-x", "hip", os.path.join(CSRC, "afno_api.cpp"), "-o", lib]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    olib = str(d / "libafno_oracle_asan.so")
    ocmd = ["gcc", "-O1", "-g", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-o", olib, os.path.join(ROOT, "oracle", "afno_oracle.c"), "-lm"]
    r = subprocess.run(ocmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    gcc_asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                              text=True).stdout.strip()
    return {"lib": lib, "rt": rt, "olib": olib, "gcc_asan": gcc_asan, "dir": str(d)}


def _run_child(script, preload, workdir):
    env = dict(os.environ)
    env["LD_PRELOAD"] = preload
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["PYTHONPATH"] = ROOT
    r = subprocess.run([sys.executable, "-c", textwrap.dedent(script)], capture_output=True,
                       text=True, env=env, cwd=workdir, timeout=600)
    report = "AddressSanitizer" in r.stderr or "runtime error:" in r.stderr
    assert r.returncode == 0 and not report and "CHILD OK" in r.stdout, \
        (r.returncode, r.stdout[-2000:], r.stderr[-4000:])


def test_abi_validation_under_asan_ubsan(builds):
    script = f"""
    import ctypes, math
    lib = ctypes.CDLL({builds['lib']!r})
    i64, vp, f32, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, ctypes.c_int
    fwd = [vp] * 5 + [i64] * 5 + [f32, f32, ci, vp, vp]
    for name in ("afno_filter_forward", "afno_filter_forward_noalloc"):
        getattr(lib, name).argtypes = fwd
        getattr(lib, name).restype = ci
    lib.afno_filter_forward_hidden.argtypes = [vp] * 5 + [i64] * 6 + [f32, f32, ci, vp, vp]
    lib.afno_filter_stage.argtypes = [vp] * 5 + [i64] * 5 + [f32, f32, ci, ci, vp, vp]
    lib.afno_filter_backward.argtypes = [vp] * 6 + [i64] * 5 + [f32, f32, ci] + [vp] * 6
    lib.afno_block_forward.argtypes = [vp] * 13 + [i64] * 5 + [f32, f32, ci, vp, vp]
    lib.afno_set_kernel_path.argtypes = [ci]
    lib.afno_last_error.restype = ctypes.c_char_p
    X, W1, B1, W2, B2, OUT, G = (0x10000000 * (i + 1) for i in range(7))
    base = dict(x=X, w1=W1, b1=B1, w2=W2, b2=B2, B=1, H=16, W=32, C=64, nb=4, lam=0.01,
                keep=1.0, dtype=0, out=OUT)

    def call(fn="afno_filter_forward", **kw):
        a = dict(base, **kw)
        return getattr(lib, fn)(a["x"], a["w1"], a["b1"], a["w2"], a["b2"], a["B"], a["H"],
                                a["W"], a["C"], a["nb"], a["lam"], a["keep"], a["dtype"],
                                a["out"], None)

    INV, UNS, ALI = -1, -2, -3
    cases = [
        (INV, dict(x=None)), (INV, dict(H=0)), (INV, dict(C=64, nb=3)), (INV, dict(lam=-1.0)),
        (INV, dict(lam=math.nan)), (INV, dict(keep=0.0)), (INV, dict(dtype=5)),
        (UNS, dict(H=7)), (UNS, dict(W=33)), (UNS, dict(C=512, nb=2)), (UNS, dict(H=256)),
        (UNS, dict(W=2048)), (UNS, dict(x=X + 8)), (UNS, dict(w1=W1 + 2)),
        (UNS, dict(H=90, W=180, C=132096, nb=1032, dtype=1)),
        (ALI, dict(out=X)), (ALI, dict(out=W1 + 64)), (ALI, dict(keep=0.3, out=X)),
        (ALI, dict(H=90, W=180, C=768, nb=8, dtype=1, B=4, out=X)),
        (ALI, dict(H=180, W=360, C=1024, nb=32, dtype=1, out=X)),
        (0, dict(B=0, x=None, out=None)),
    ]
    for path in (0, 1, 2):
        assert lib.afno_set_kernel_path(path) == 0
        for want, kw in cases:
            for fn in ("afno_filter_forward", "afno_filter_forward_noalloc"):
                rc = call(fn, **kw)
                assert rc == want, (fn, kw, rc, lib.afno_last_error())
    assert lib.afno_set_kernel_path(0) == 0
    assert call("afno_filter_forward_noalloc", H=90, W=180, C=768, nb=8, dtype=1, B=6) == UNS
    # hidden sizes, stages, backward, block: their own checks
    rc = lib.afno_filter_forward_hidden(X, W1, B1, W2, B2, 1, 16, 32, 64, 4, 24, 0.01, 1.0, 0,
                                        OUT, None)
    assert rc == UNS
    rc = lib.afno_filter_stage(X, W1, B1, W2, B2, 1, 16, 32, 64, 4, 0.01, 1.0, 0, 3, X, None)
    assert rc == ALI
    rc = lib.afno_filter_backward(X, W1, B1, W2, B2, G, 1, 16, 32, 64, 4, 0.01, 1.0, 0,
                                  OUT, W1, B1, 0x90000000, 0xa0000000, None)
    assert rc == ALI
    rc = lib.afno_filter_backward(X, W1, B1, W2, B2, G, 1, 90, 180, 768, 8, 0.01, 1.0, 1, X,
                                  0x90000000, 0xa0000000, 0xb0000000, 0xc0000000, None)
    assert rc == ALI
    L = [0x10000000 * (i + 20) for i in range(8)]
    rc = lib.afno_block_forward(X, L[0], L[1], W1, B1, W2, B2, L[2], L[3], L[4], L[5], L[6],
                                L[7], 1, 16, 32, 128, 4, 0.01, 1.0, 1, X, None)
    assert rc == ALI
    print("CHILD OK")
    """
    _run_child(script, builds["rt"], builds["dir"])


def test_oracle_under_asan_ubsan(builds):
    script = f"""
    import numpy as np
    import oracle
    from oracle import backward as ob
    oracle._LIB_PATH = {builds['olib']!r}
    rng = np.random.default_rng(3)
    out = {{}}
    for (B, H, W, C, nb, hs, keep) in ((1, 4, 8, 8, 2, 4, 1.0), (2, 5, 6, 12, 3, 8, 0.7),
                                       (1, 1, 2, 4, 1, 4, 1.0), (1, 6, 10, 8, 2, 4, 0.2)):
        bs = C // nb
        x = rng.standard_normal((B, H, W, C))
        w = [rng.standard_normal(s) * 0.3 for s in ((nb, bs, hs, 2), (nb, hs, 2),
                                                   (nb, hs, bs, 2), (nb, bs, 2))]
        y, st = oracle.filter_forward(x, *w, nb, 0.05, keep, stages=True)
        key = f"{{B}}_{{H}}_{{W}}_{{C}}_{{hs}}_{{keep}}"
        out[key + "_y"] = y
        out[key + "_spec"] = st["spec_mlp"].real + st["spec_mlp"].imag
        out[key + "_bf"] = oracle.dft2_bruteforce(x).real
        if hs == bs:
            g = rng.standard_normal(x.shape)
            out[key + "_dx"] = ob.filter_backward(x, *w, g, nb, 0.05, keep)["dx"]
    np.savez("oracle_asan.npz", **out)
    print("CHILD OK")
    """
    _run_child(script, builds["gcc_asan"], builds["dir"])
    # the same computations with the regular build agree to rounding
    import numpy as np
    import oracle
    from oracle import backward as ob
    got = np.load(os.path.join(builds["dir"], "oracle_asan.npz"))
    rng = np.random.default_rng(3)
    for (B, H, W, C, nb, hs, keep) in ((1, 4, 8, 8, 2, 4, 1.0), (2, 5, 6, 12, 3, 8, 0.7),
                                       (1, 1, 2, 4, 1, 4, 1.0), (1, 6, 10, 8, 2, 4, 0.2)):
        bs = C // nb
        x = rng.standard_normal((B, H, W, C))
        w = [rng.standard_normal(s) * 0.3 for s in ((nb, bs, hs, 2), (nb, hs, 2),
                                                   (nb, hs, bs, 2), (nb, bs, 2))]
        y, st = oracle.filter_forward(x, *w, nb, 0.05, keep, stages=True)
        key = f"{B}_{H}_{W}_{C}_{hs}_{keep}"
        assert np.allclose(got[key + "_y"], y, rtol=0, atol=1e-12)
        assert np.allclose(got[key + "_spec"], st["spec_mlp"].real + st["spec_mlp"].imag,
                           rtol=0, atol=1e-12)
        assert np.allclose(got[key + "_bf"], oracle.dft2_bruteforce(x).real, rtol=0, atol=1e-12)
        if hs == bs:
            g = rng.standard_normal(x.shape)
            assert np.allclose(got[key + "_dx"], ob.filter_backward(x, *w, g, nb, 0.05, keep)["dx"],
                               rtol=0, atol=1e-12)
