"""Pins of the oracle's entropy-bound sampler (Algorithm 2, uniform-state diffusion)."""
import math

import numpy as np
import pytest

import synth
from oracle import loop
from oracle import network
from oracle import sampler as S
from oracle import usdm

F32 = np.float32


def _softmax64(l, inv_temp):
    lp = np.asarray(l, np.float32).astype(np.float64) * float(np.float32(inv_temp))
    p = np.exp(lp - lp.max())
    return p / p.sum()


@pytest.mark.parametrize("V,scale,inv_temp", [(1000, 3.0, 1.25), (50, 0.1, 2.5), (4096, 8.0, 1.0),
                                              (257, 30.0, 1.0), (2, 0.0, 1.0)])
def test_entropy_matches_the_float64_definition(V, scale, inv_temp):
    """H of the fixed-point form equals -sum p log p of the float64 softmax to within
    the float32 rounding of its two terms (a few 1e-7 relative) plus the 2^-40 weights."""
    rng = np.random.default_rng(V)
    for _ in range(5):
        l = (rng.normal(size=V) * scale).astype(np.float32)
        _, _, H, Hq = usdm.entropy_stats(l, inv_temp)
        p = _softmax64(l, inv_temp)
        ref = float(-(p[p > 0] * np.log(p[p > 0])).sum())
        assert abs(float(H) - ref) <= 4e-7 * max(ref, 1.0) + V * 2.0 ** -38, (H, ref)
        assert Hq == round(float(H) * 2.0 ** 40)


def test_entropy_special_rows():
    """Uniform row: H = log V; one dominant entry: H ~ 0 (never below -1e-6)."""
    for V in (2, 3, 64, 1000, 32768):
        H = usdm.entropy_stats(np.zeros(V, np.float32), 1.0)[2]
        assert abs(float(H) - math.log(V)) < 2e-6 * math.log(V) + 1e-6
    l = np.zeros(500, np.float32)
    l[7] = 60.0
    H = usdm.entropy_stats(l, 1.0)[2]
    assert -1e-6 <= float(H) < 1e-6


def test_accept_set_is_the_literal_rule():
    """A = {pi_m : C_m - M_m <= eta} over the ascending argsort, C the running sum and M
    the running maximum, computed in float64 on well separated entropies."""
    rng = np.random.default_rng(5)
    for trial in range(200):
        Lc = int(rng.integers(1, 60))
        H = rng.exponential(0.05 if trial % 2 else 0.5, size=Lc)
        eta = float(rng.choice([0.0, 0.1, 0.3, 2.0]))
        Hq = np.rint(H * 2.0 ** 40).astype(np.int64)
        order = np.argsort(H, kind="stable")
        C = np.cumsum(H[order])
        M = np.maximum.accumulate(H[order])
        lit = np.zeros(Lc, bool)
        margin = np.abs(C - M - float(np.float32(eta)))
        lit[order] = (C - M) <= float(np.float32(eta))
        got = usdm.accept_set(Hq, eta)
        ok = margin > 1e-9
        ok_pos = np.zeros(Lc, bool)
        ok_pos[order] = ok
        assert np.array_equal(got[ok_pos], lit[ok_pos])
        assert got[order[0]]                      # the least uncertain position is always accepted


def test_accept_set_extremes_and_ties():
    Hq = np.array([5, 3, 3, 9, 0], np.int64) << 30
    # eta = 0: the first position in (Hq, position) order, and the next one too because
    # only a zero entropy ranks before it
    acc = usdm.accept_set(Hq, 0.0)
    assert acc.tolist() == [False, True, False, False, True]
    # a large bound accepts everyone
    assert usdm.accept_set(Hq, 1e6).all()
    # tied entropies: the lower position ranks first
    acc = usdm.accept_set(np.array([7, 7, 7], np.int64) << 36, 7 * 2.0 ** -4 + 1e-6)
    assert acc.tolist() == [True, True, False]


def test_temperature_schedule():
    T, hi, lo = 48, 0.8, 0.4
    assert usdm.inv_temperature(T, T, hi, lo) == F32(1 / float(F32(0.8)))
    assert usdm.inv_temperature(1, T, hi, lo) == F32(1 / (float(F32(0.4)) + (float(F32(0.8)) - float(F32(0.4))) / T))
    taus = [1 / float(usdm.inv_temperature(n, T, hi, lo)) for n in range(1, T + 1)]
    assert np.ptp(np.diff(taus)) < 1e-6 and abs(np.diff(taus).mean() - 0.4 / T) < 1e-6


def test_uniform_tokens():
    """Re-noise and initial tokens are uniform over [0, V) and use counters that no
    vocabulary draw or remasking decision reaches."""
    V, n = 7, 70000
    for draw in (usdm.renoise_tokens(np.arange(n), 3, 11, 9, V), usdm.initial_tokens(np.arange(n), 1, 2, 9, V)):
        assert draw.min() >= 0 and draw.max() < V
        cnt = np.bincount(draw, minlength=V)
        chi2 = ((cnt - n / V) ** 2 / (n / V)).sum()
        assert chi2 < 30                              # 6 degrees of freedom: p ~ 1e-4
    assert usdm.RENOISE_WORD0 != S.DECISION_WORD0 and usdm.INIT_WORD0 not in (S.DECISION_WORD0, usdm.RENOISE_WORD0)
    assert min(usdm.RENOISE_WORD0, usdm.INIT_WORD0) >= 2 ** 31   # vocabulary counters stay below 2^31


def test_gumbel_token_is_the_masked_samplers_draw():
    rng = np.random.default_rng(2)
    l = rng.normal(size=333).astype(np.float32)
    for step in range(5):
        assert usdm.gumbel_token(l, 1.3, 17, 2, step, 99) == S.sample_position(l, F32(1.3), 17, 2, step, 99)[0]


def test_selfcond_is_the_expected_embedding():
    rng = np.random.default_rng(1)
    V, d = 40, 8
    E = rng.normal(size=(V + 1, d))
    l = rng.normal(size=(3, V)).astype(np.float32)
    s = usdm.selfcond(l, 1.7, E)
    for r in range(3):
        p = _softmax64(l[r], 1.7)
        assert np.allclose(s[r], sum(p[v] * E[v] for v in range(V)), rtol=1e-12, atol=1e-12)
    one_hot = np.full((1, V), -1e4, np.float32)
    one_hot[0, 5] = 0.0
    assert np.allclose(usdm.selfcond(one_hot, 1.0, E)[0], E[5])


def test_step_next_canvas():
    """Accepted positions take x_tilde, the others the re-noise token; the last step
    leaves x_hat, the argmax of the logits."""
    rng = np.random.default_rng(8)
    Lc, V = 30, 50
    logits = (rng.normal(size=(Lc, V)) * rng.uniform(0.1, 6, size=(Lc, 1))).astype(np.float32)
    r = usdm.entropy_step(logits, 5, F32(1.25), 0.5, 100, 1, 7, 3)
    rn = usdm.renoise_tokens(100 + np.arange(Lc), 1, 7, 3, V)
    assert np.array_equal(r["next"], np.where(r["accept"], r["x_tilde"], rn))
    assert 0 < r["accept"].sum() < Lc
    last = usdm.entropy_step(logits, 1, F32(1.25), 0.5, 100, 1, 7, 3)
    assert np.array_equal(last["next"], logits.argmax(axis=1))


def test_usdm_generation_structure():
    """Generation on the tiny model: a block starts from the initial noise, each step
    feeds back the previous step's self-conditioning, the anchor refreshes every K
    steps, and the result is the last step's argmax canvas."""
    cfg = synth.get_config("tiny", batch=1)
    tensors = synth.make_weights(cfg, perturb=True)
    net = network.Network(network.Weights(cfg, [s[0] for s in synth.weight_specs(cfg)], tensors))
    prompt = synth.make_prompt(cfg, batch=1).numpy()
    P, G, T, K = cfg["prompt_len"], cfg["gen_len"], 6, 4
    trace = []
    out = loop.generate_usdm(net, prompt, G, T, K, G, seed=4, trace=trace)
    assert np.array_equal(trace[0]["canvas"], usdm.initial_tokens(np.arange(P, P + G), 0, 0, 4, cfg["vocab"]))
    assert [t["refresh"] for t in trace] == [(T - n) % K == 0 for n in range(T, 0, -1)]
    assert np.array_equal(out[0, P:], trace[-1]["x_hat"])
    for a, b in zip(trace, trace[1:]):
        assert np.array_equal(b["canvas"], a["next"])
    # self-conditioning changes the decoder's input: rerunning a step without it differs
    c_with = net.shared(out[0], np.arange(P + G), sc=np.ones((P + G, cfg["d_model"])))
    c_without = net.shared(out[0], np.arange(P + G))
    assert not np.allclose(c_with, c_without)
