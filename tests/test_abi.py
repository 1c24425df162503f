"""Host-side checks of the C ABI: the library loads, exports every declared symbol,
agrees with the seeded input module on the weight order, and rejects bad arguments
before touching the GPU."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import synth
from oracle import loop

tadm = pytest.importorskip("paper_2609_37924_amd")

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "tadm.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tadm_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert len(names) >= 25
    for n in names:
        assert hasattr(tadm.lib, n), n
    assert set(tadm.EXPORTED) == set(names)


@pytest.mark.parametrize("name", list(synth.CONFIGS))
def test_weight_order_matches_inputs(name):
    cfg = synth.get_config(name)
    c = tadm.make_config(cfg)
    specs = synth.weight_specs(cfg)
    assert tadm.tadm_weight_count(c) == len(specs)
    for i, (nm, shape, _) in enumerate(specs):
        rows, cols = tadm.tadm_weight_info(c, i)
        assert (rows, cols) == (shape[0], shape[1] if len(shape) > 1 else 0), nm


def test_unmask_count_matches_schedule():
    for M0, T in [(24, 16), (256, 64), (64, 32), (1024, 128), (7, 3), (0, 5)]:
        for i in range(1, T + 1):
            assert tadm.tadm_unmask_count(M0, i, T) == loop.unmask_count(M0, i, T)
    assert tadm.tadm_unmask_count(5, 0, 4) == 0


def test_invalid_arguments_fail_before_device_work():
    cfg = synth.get_config("tiny")
    bad = tadm.make_config(cfg)
    bad.n_heads = 3  # not a multiple of n_kv_heads = 4
    m = C.c_void_p()
    assert tadm.lib.tadm_model_create(C.byref(bad), C.byref(m)) == tadm.TADM_ERR_INVALID
    assert "n_kv_heads" in tadm.last_error()
    bad = tadm.make_config(cfg)
    bad.dtype = 7
    assert tadm.lib.tadm_model_create(C.byref(bad), C.byref(m)) == tadm.TADM_ERR_INVALID
    bad = tadm.make_config(cfg)
    bad.vocab = 262144 + 4  # past the sampler's on-chip group partials
    assert tadm.lib.tadm_model_create(C.byref(bad), C.byref(m)) == tadm.TADM_ERR_INVALID
    assert "vocab" in tadm.last_error()
    good = tadm.make_config(cfg)
    r, k = C.c_int64(), C.c_int64()
    assert tadm.lib.tadm_weight_info(C.byref(good), 10_000, C.byref(r), C.byref(k)) == tadm.TADM_ERR_INVALID
    assert tadm.lib.tadm_generate(None, None, 1, 0, 8, 4, 1, 8, 0, 1.0, None) == tadm.TADM_ERR_INVALID
    args = tadm.step_args(1, 4, 1, 0, 0, 1.0)
    assert tadm.lib.tadm_sample(None, None, None, 1, 8, 0, 0, C.byref(args), None, None, None) \
        == tadm.TADM_ERR_INVALID
    assert tadm.lib.tadm_cache_destroy(None) == tadm.TADM_ERR_INVALID
    assert tadm.lib.tadm_context_reset(None) == tadm.TADM_ERR_INVALID
    with pytest.raises(tadm.TadmError):
        tadm.check(tadm.lib.tadm_model_destroy(None))


def test_remask_probs_match_the_oracle():
    """The library's per-step (sigma, p_unmask) are the oracle's float32 numbers."""
    from oracle import loop
    for T in (1, 7, 16, 64, 128, 1024):
        for eta in (0.0, 0.02, 0.04, 0.3, 1.0):
            for i in sorted({1, 2, 3, T // 2 or 1, T - 1 or 1, T}):
                sg, pu = tadm.tadm_remask_probs(i, T, eta)
                rs, rp = loop.remask_probs(i, T, eta)
                assert np.float32(sg) == rs and np.float32(pu) == rp, (i, T, eta)


def test_loop_probs_match_the_oracle():
    """The library's ReMDM-Loop (sigma, p_unmask) are the oracle's float32 numbers at every
    step, including the steps at the plateau's edges."""
    from oracle import loop
    for T in (1, 2, 20, 40, 64, 100, 1024, 4096):
        for params in ((0.02, 0.55, 0.05, 0.9), (0.04, 0.7, 0.2, 0.5), (0.5, 0.55, 0.05, 0.9), (0.0, 0.5, 0.25, 0.6)):
            for i in range(1, T + 1):
                sg, pu = tadm.tadm_loop_probs(i, T, *params)
                rs, rp = loop.loop_probs(i, T, *params)
                assert np.float32(sg) == rs and np.float32(pu) == rp, (i, T, params)


def test_entropy_inv_temp_matches_the_oracle():
    from oracle import usdm
    for T in (1, 7, 48, 100):
        for hi, lo in ((0.8, 0.4), (1.0, 1.0), (2.5, 0.1)):
            for n in range(1, T + 1):
                assert np.float32(tadm.tadm_entropy_inv_temp(n, T, hi, lo)) == usdm.inv_temperature(n, T, hi, lo)


def test_stale_times_match_the_oracle():
    """The library's training times (antithetic t, refresh interval, budget, cache age,
    stale time) are the oracle's bit for bit."""
    from oracle import train
    for B, seed, step, eps in ((1, 0, 0, 1e-3), (16, 7, 3, 1e-3), (512, 2 ** 40 + 5, 99, 0.0), (37, 11, 1, 0.25)):
        got = tadm.tadm_stale_times(B, seed, step, eps)
        ref = train.stale_times(B, seed, step, eps)
        for g, r, name in zip(got, ref, ("t", "t'", "K", "T", "k")):
            assert np.array_equal(np.asarray(g), np.asarray(r).astype(np.asarray(g).dtype)), (name, B, seed)


def test_entropy_sampler_rejects_bad_settings():
    for bad in (dict(eta=-0.1), dict(tau_min=0.0), dict(tau_max=0.3, tau_min=0.4), dict(eta=float("inf"))):
        smp = tadm.entropy_sampler(**bad)
        st = tadm.lib.tadm_generate_sampler(None, None, 1, 0, 8, 4, 1, 8, 0, 1.0, C.byref(smp), None)
        assert st != 0
        assert re.search(rb"entropy bound|temperatures", tadm.lib.tadm_last_error()), bad


def test_loop_sampler_rejects_bad_schedules():
    cfg = synth.get_config("tiny")
    for bad in (dict(t_on=0.05, t_off=0.55), dict(t_on=1.0), dict(t_off=0.0), dict(alpha_on=1.0), dict(eta=1.5)):
        smp = tadm.loop_sampler(**bad)
        st = tadm.lib.tadm_generate_sampler(None, None, 1, 0, 8, 4, 1, 8, 0, 1.0, C.byref(smp), None)
        assert st != 0
        assert re.search(rb"loop schedule|eta", tadm.lib.tadm_last_error()), bad


RUN = os.path.join(os.path.dirname(os.path.dirname(__file__)), "paper_2609_37924_amd", "tadm_run")


def test_kernel_bench_rejects_bad_arguments_before_device_work():
    import subprocess

    kb = os.path.join(os.path.dirname(RUN), "kernel_bench")
    if not os.path.exists(kb):
        pytest.skip("kernel_bench not built")
    for argv, msg in (([], "missing batch"), (["foo"], "bad argument"),
                      (["batch=1", "prompt_len=0", "gen_len=8", "d_model=64", "n_heads=1", "head_dim=32",
                        "d_ffn=64", "vocab=64", "T=4"], "unsupported shape"),
                      (["batch=1", "prompt_len=0", "gen_len=8", "d_model=64", "n_heads=1", "head_dim=64",
                        "d_ffn=64", "vocab=0", "T=4"], "unsupported shape"),
                      (["batch=2", "prompt_len=0", "gen_len=8", "d_model=64", "n_heads=1", "head_dim=64",
                        "d_ffn=64"], "missing vocab"),
                      (["batch=2", "prompt_len=0", "gen_len=8", "d_model=64", "n_heads=1", "head_dim=64",
                        "d_ffn=64", "vocab=64", "T=4", "dtype=0"], "bf16 workloads only")):
        r = subprocess.run([kb] + argv, capture_output=True, text=True, timeout=60)
        assert r.returncode == 1, (argv, r.returncode, r.stderr)
        assert msg in r.stderr, (argv, r.stderr)


def test_native_driver_rejects_bad_arguments_before_device_work():
    """tadm_run (the native program over the C ABI) checks its arguments before it
    touches the GPU: these run on a host without one."""
    import subprocess

    if not os.path.exists(RUN):
        pytest.skip("tadm_run not built")
    for argv, msg in (([], "missing batch"), (["foo"], "bad argument"),
                      (["batch=1", "prompt_len=0", "gen_len=8", "T=0", "vocab=8", "d_model=8", "n_heads=1",
                        "head_dim=8", "d_ffn=8", "n_anchor=1", "n_denoise=1"], "must be positive"),
                      (["batch=x"], "bad value")):
        r = subprocess.run([RUN] + argv, capture_output=True, text=True, timeout=60)
        assert r.returncode == 1, (argv, r.returncode, r.stderr)
        assert msg in r.stderr, (argv, r.stderr)
