"""The library's host-side argument validation under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU).

A build with the host code instrumented (build.build_host_sanitized) is loaded in a
child process with the sanitizer runtime preloaded; the child calls every validating
entry point with invalid arguments (null handles, shapes outside the limits, bad
configs, bad step arguments) and the pure host functions over their edge cases, each
of which must return before any device work.  Any sanitizer report fails the test.
"""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RUNTIME = "/opt/rocm/llvm/lib/clang/22/lib/linux/libclang_rt.asan-x86_64.so"

CHILD = textwrap.dedent(r"""
    import ctypes as C, sys
    sys.path.insert(0, ROOT)
    lib = C.CDLL(SAN)
    # the binding's structures and signatures, applied to the sanitized library
    import importlib.util
    spec = importlib.util.spec_from_file_location("b", ROOT + "/paper_2609_37924_amd/__init__.py")
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    for name, (res, args) in b._SIGS.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    import synth
    INV, ST, UNS = b.TADM_ERR_INVALID, b.TADM_ERR_STATE, b.TADM_ERR_UNSUPPORTED
    cfg = synth.get_config("tiny")
    m = C.c_void_p()
    for field, value in (("n_heads", 3), ("dtype", 7), ("vocab", 262148), ("d_model", 0), ("head_dim", 6),
                         ("fusion_kind", 9), ("max_batch", 0), ("n_anchor", -1)):
        bad = b.make_config(cfg)
        setattr(bad, field, value)
        assert lib.tadm_model_create(C.byref(bad), C.byref(m)) in (INV, UNS), field
        assert len(lib.tadm_last_error()) > 0
    assert lib.tadm_model_create(None, C.byref(m)) == INV
    good = b.make_config(cfg)
    r, k = C.c_int64(), C.c_int64()
    n = lib.tadm_weight_count(C.byref(good))
    assert n > 0
    for i in (-1, n, 1 << 30):
        assert lib.tadm_weight_info(C.byref(good), i, C.byref(r), C.byref(k)) == INV
    for i in range(n):
        assert lib.tadm_weight_info(C.byref(good), i, C.byref(r), C.byref(k)) == 0 and r.value > 0
    assert lib.tadm_generate(None, None, 1, 0, 8, 4, 1, 8, 0, 1.0, None) == INV
    args = b.step_args(1, 4, 1, 0, 0, 1.0)
    assert lib.tadm_sample(None, None, None, 1, 8, 0, 0, C.byref(args), None, None, None) == INV
    assert lib.tadm_sample_noalloc(None, None, None, 1, 8, 0, 0, C.byref(args), None, None, None) == INV
    assert lib.tadm_denoise_step(None, None, None, 1, 8, 0, None, C.byref(args), None, None) == INV
    assert lib.tadm_anchor_forward(None, None, None, 1, 8, 1, 4, None) == INV
    assert lib.tadm_cache_destroy(None) == INV
    assert lib.tadm_context_reset(None) == INV
    assert lib.tadm_context_read(None, 0, None, None, 0) == INV
    assert lib.tadm_model_destroy(None) == INV
    assert lib.tadm_debug_layers(None, None, 0) == INV
    for M0 in (0, 1, 24, 1 << 20):
        for T in (1, 16, 4096):
            assert sum(lib.tadm_unmask_count(M0, i, T) for i in range(1, T + 1)) == M0
    assert lib.tadm_unmask_count(5, 0, 4) == 0 and lib.tadm_unmask_count(-1, 1, 4) == 0
    s, p = C.c_float(), C.c_float()
    for i in (1, 2, 64):
        lib.tadm_remask_probs(i, 64, 0.04, C.byref(s), C.byref(p))
        lib.tadm_loop_probs(i, 64, 0.02, 0.55, 0.05, 0.9, C.byref(s), C.byref(p))
    print("validation ok")
""")


def _san_lib():
    sys.path.insert(0, os.path.join(ROOT, "paper_2609_37924_amd", "csrc"))
    import build  # noqa: E402
    if not os.path.exists(build.SAN_OUT):
        build.build_host_sanitized()
    return build.SAN_OUT


@pytest.mark.skipif(not os.path.exists(RUNTIME), reason="no AddressSanitizer runtime in this image")
def test_host_validation_under_sanitizers():
    san = _san_lib()
    env = dict(os.environ, LD_PRELOAD=RUNTIME, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    code = f"ROOT = {ROOT!r}\nSAN = {san!r}\n" + CHILD
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=300)
    report = r.stdout + r.stderr
    assert r.returncode == 0, report[-4000:]
    assert "validation ok" in r.stdout
    for marker in ("ERROR: AddressSanitizer", "runtime error:", "ERROR: UndefinedBehaviorSanitizer"):
        assert marker not in report, report[-4000:]
