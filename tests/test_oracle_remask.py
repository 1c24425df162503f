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
