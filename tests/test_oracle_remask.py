"""Pins of the oracle's remasking posterior (eq. inf-post-TADM with sigma_t > 0)."""
import math

import numpy as np

from oracle import loop
from oracle import sampler as S


def test_sigma_zero_is_the_absorbing_posterior():
    """sigma = 0: the unmask probability is (alpha_s - alpha_t) / (1 - alpha_t) = 1/i on
    the linear schedule, and nothing is ever remasked."""
    for T in (4, 16, 64, 128):
        for i in range(1, T + 1):
            sigma, p = loop.remask_probs(i, T, 0.0)
            assert sigma == 0.0
            assert p == np.float32(1.0 / i)


def test_cap_keeps_the_posterior_a_distribution():
    """sigma = min(eta, (1 - alpha_s)/alpha_t) is the largest remasking probability for
    which every case of the posterior is a probability; the last step (alpha_s = 1)
    unmasks everything and remasks nothing."""
    for T in (8, 16, 64, 128):
        for eta in (0.02, 0.04, 0.5, 1.0):
            for i in range(1, T + 1):
                sigma, p = loop.remask_probs(i, T, eta)
                a_t, a_s = 1 - i / T, 1 - (i - 1) / T
                assert 0.0 <= sigma <= np.float32(eta)
                assert 0.0 <= p <= 1.0
                assert 1 - a_s - float(sigma) * a_t >= -1e-6          # mask probability
                assert a_s - (1 - float(sigma)) * a_t >= -1e-6        # token probability
            assert loop.remask_probs(1, T, eta) == (0.0, 1.0)


def test_decision_uniforms_are_independent_of_vocabulary_draws():
    """The decision uses counter word 0 = 2^31, which no vocabulary draw reaches, and is
    uniform on (0, 1)."""
    u = S.decision_uniforms(np.arange(100000), 3, 7, 11)
    assert u.min() > 0 and u.max() < 1
    assert abs(u.mean() - 0.5) < 5 * math.sqrt(1 / 12 / u.size)
    w = S.philox4x32_10(np.full(4, S.DECISION_WORD0, np.uint32), np.arange(4, dtype=np.uint32), np.uint32(3),
                        np.uint32(7), np.uint32(11), np.uint32(0))
    assert np.array_equal(S.bits_to_uniform(w[0]), S.decision_uniforms(np.arange(4), 3, 7, 11))


def test_move_frequencies_match_sigma_and_p_unmask():
    rng = np.random.default_rng(4)
    Lc, V, mask = 8000, 4, 4
    canvas = rng.integers(0, V, Lc)
    canvas[rng.random(Lc) < 0.5] = mask
    logits = rng.normal(size=(Lc, V)).astype(np.float32)
    sigma, p = np.float32(0.3), np.float32(0.6)
    nxt, choice = S.remask_step(logits, canvas, mask, p, sigma, 100, 2, 5, 9, np.float32(1.0))
    m = canvas == mask
    remasked = (~m) & (nxt == mask)
    unmasked = m & (nxt != mask)
    for frac, n, prob in ((remasked.sum() / (~m).sum(), (~m).sum(), sigma), (unmasked.sum() / m.sum(), m.sum(), p)):
        assert abs(frac - prob) < 5 * math.sqrt(prob * (1 - prob) / n)
    assert np.array_equal(nxt[unmasked], choice[unmasked])                  # the Gumbel-max token
    assert np.array_equal(nxt[(~m) & ~remasked], canvas[(~m) & ~remasked])  # others carried over


def test_chain_preserves_the_forward_marginal():
    """From the all-mask canvas, one step of the posterior keeps P(masked) = 1 - alpha_s:
    (1 - alpha_t)(1 - p_unmask) + alpha_t sigma = 1 - alpha_s for any valid sigma.  The
    simulated chain must follow that marginal at every step and end fully unmasked."""
    rng = np.random.default_rng(1)
    Lc, V, T = 3000, 3, 16
    logits = np.zeros((Lc, V), np.float32)
    for eta in (0.0, 0.3):
        z = np.full(Lc, V)
        for i in range(T, 0, -1):
            sigma, p = loop.remask_probs(i, T, eta)
            a_t = 1 - i / T
            frac_t = (z == V).mean()
            expect = frac_t * (1 - float(p)) + (1 - frac_t) * float(sigma)
            z, _ = S.remask_step(logits, z, V, p, sigma, 0, 0, T - i, 17, np.float32(1.0))
            frac = (z == V).mean()
            assert abs(frac - expect) < 5 * math.sqrt(max(expect * (1 - expect), 1e-9) / Lc) + 1e-9
            assert abs(frac - (i - 1) / T) < 0.06, (eta, i, frac)
        assert (z != V).all()


def test_nucleus_matches_the_sorted_cumulative_definition():
    """Away from the boundary the fixed-point nucleus is the float64 textbook one: the
    smallest set of highest-probability entries whose mass reaches p."""
    rng = np.random.default_rng(8)
    checked = 0
    for trial in range(200):
        V = int(rng.integers(3, 300))
        lp = (rng.normal(size=V) * rng.uniform(0.3, 4)).astype(np.float32)
        p = float(rng.uniform(0.05, 0.99))
        got = S.nucleus(lp, p)
        pr = np.exp(lp.astype(np.float64) - lp.max())
        pr /= pr.sum()
        order = np.argsort(-pr, kind="stable")
        cum = np.cumsum(pr[order])
        k = int(np.searchsorted(cum, p)) + 1               # entries needed to reach p
        if k < V and (cum[k - 1] - p > 1e-6) and (k < 2 or p - cum[k - 2] > 1e-6) and \
                (k == V or pr[order[k - 1]] - pr[order[k]] > 1e-9):
            ref = np.zeros(V, bool)
            ref[order[:k]] = True
            assert np.array_equal(got, ref), trial
            checked += 1
    assert checked > 150


def test_nucleus_extremes():
    lp = np.array([0.5, 2.0, 2.0, -1.0, 1.9], np.float32)
    assert np.array_equal(S.nucleus(lp, 1e-6), [False, True, True, False, False])  # ties at the top kept
    assert S.nucleus(np.full(50, 3.0, np.float32), 0.3).all()                       # all tied: all kept
    big = (np.random.default_rng(2).normal(size=4000) * 2).astype(np.float32)
    tok = S.sample_position(big, 1.0, 5, 1, 3, 9)
    assert S.sample_position(big, 1.0, 5, 1, 3, 9, top_p=1.0) == tok                 # p = 1: untruncated


def test_nucleus_sampling_follows_the_truncated_softmax():
    """Gumbel-max restricted to the nucleus draws from the renormalised truncation:
    chi-square over 20000 step ids."""
    lp = np.array([1.5, 1.0, 0.2, -0.5, 2.0, -2.0], np.float32)
    p = 0.8
    keep = S.nucleus(lp, p)
    pr = np.where(keep, np.exp(lp.astype(np.float64) - lp.max()), 0.0)
    pr /= pr.sum()
    n = 20000
    counts = np.zeros(6)
    for k in range(n):
        counts[S.sample_position(lp, 1.0, 3, 0, k, 41, top_p=p)[0]] += 1
    assert (counts[~keep] == 0).all()
    e = n * pr[keep]
    chi2 = ((counts[keep] - e) ** 2 / e).sum()
    assert chi2 < 25.0  # <= 5 dof, p ~ 1e-4


LOOP = (0.02, 0.55, 0.05, 0.9)  # eta, t_on, t_off, alpha_on of the paper's runs with T >= L


def _loop_marginals(T, params):
    """Expected masked fraction after each reverse step, by the posterior's own
    recursion m_s = m_t (1 - p_unmask) + (1 - m_t) sigma from the all-mask canvas."""
    m, out = 1.0, []
    for i in range(T, 0, -1):
        sigma, p = loop.loop_probs(i, T, *params)
        m = m * (1.0 - float(p)) + (1.0 - m) * float(sigma)
        out.append(((i - 1) / T, m, float(sigma), float(p)))
    return out


def test_loop_schedule_phases():
    """ReMDM-Loop: the masked fraction falls linearly from 1 to 1 - alpha_on while t goes
    from 1 to t_on, holds there (remasking with sigma = eta) down to t_off, and falls
    linearly to 0 at t = 0; sigma is eta exactly on the plateau steps and 0 elsewhere."""
    eta, t_on, t_off, a_on = LOOP
    for T in (20, 64, 100, 1024):
        rows = _loop_marginals(T, LOOP)
        assert rows[-1][1] == 0.0 or abs(rows[-1][1]) < 1e-12           # all decoded at t = 0
        for k, (s, m, sigma, p) in enumerate(rows):
            t = s + 1 / T
            plateau = t <= t_on + 1e-12 and s >= t_off - 1e-12
            assert 0.0 <= p <= 1.0 and 0.0 <= sigma <= 1.0
            if plateau:
                assert sigma == np.float32(eta)
                assert abs(m - (1 - a_on)) < 1e-6, (T, s, m)             # the loop holds the marginal
            else:
                assert sigma == 0.0
        # linear on each side of the plateau: constant decrements per step
        for lo, hi in ((t_on, 1.0), (0.0, t_off)):
            ms = [m for s, m, _, _ in rows if lo + 1e-9 < s + 1 / T and s < hi + 1e-9 and lo - 1e-9 <= s]
            d = np.diff([1.0] + ms) if hi == 1.0 else np.diff(ms)
            if len(d) > 1:
                assert np.ptp(d) < 1e-6, (T, lo, hi)
        # endpoints of the two ramps
        first_plateau = min(s for s, _, sg, _ in rows if sg > 0)
        assert abs(dict((s, m) for s, m, _, _ in rows)[first_plateau] - (1 - a_on)) < 1e-6


def test_loop_with_eta_zero_is_an_absorbing_chain():
    """eta = 0: every step is the absorbing posterior p = (alpha_s - alpha_t)/(1 - alpha_t)
    of the piecewise schedule; the plateau steps then reveal nothing."""
    T = 40
    for i in range(T, 0, -1):
        sigma, p = loop.loop_probs(i, T, 0.0, 0.55, 0.05, 0.9)
        assert sigma == 0.0
        t, s = i / T, (i - 1) / T
        if t <= 0.55 and s >= 0.05:
            assert p == 0.0


def test_loop_chain_follows_its_marginal_and_remasks():
    """Simulated ReMDM-Loop chain through the oracle's reverse step: the masked fraction
    tracks the posterior's recursion, decoded tokens are remasked on the plateau at rate
    sigma, and the chain ends fully decoded."""
    rng = np.random.default_rng(3)
    Lc, V, T = 4000, 3, 40
    logits = rng.normal(size=(Lc, V)).astype(np.float32)
    z = np.full(Lc, V)
    remasked_total = 0
    for i in range(T, 0, -1):
        sigma, p = loop.loop_probs(i, T, *LOOP)
        frac_t = (z == V).mean()
        expect = frac_t * (1 - float(p)) + (1 - frac_t) * float(sigma)
        nxt, _ = S.remask_step(logits, z, V, p, sigma, 0, 1, T - i, 23, np.float32(1.0))
        decoded = z != V
        remasked = (decoded & (nxt == V)).sum()
        if sigma > 0:
            n = decoded.sum()
            assert abs(remasked / n - float(sigma)) < 5 * math.sqrt(float(sigma) * (1 - float(sigma)) / n) + 1e-9
        else:
            assert remasked == 0
        remasked_total += remasked
        z = nxt
        frac = (z == V).mean()
        assert abs(frac - expect) < 5 * math.sqrt(max(expect * (1 - expect), 1e-9) / Lc) + 1e-9
    assert remasked_total > 0
    assert (z != V).all()
