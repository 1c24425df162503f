"""Pins of the oracle's training objective (Theorem T-ANELBO, gamma = 0, sigma = 0)."""
import math

import numpy as np

import synth
from oracle import network
from oracle import train

F32 = np.float32


def test_pair_corruption_rates_and_nesting():
    """Positions masked in z_t are masked in z_t'; P(masked at t) = (1 - eps) t and a
    position kept at t is masked at t' with probability 1 - alpha_t'/alpha_t (eq. fwd_t_t');
    unmasked positions keep their token."""
    B, L, V, eps = 4, 20000, 50, 1e-3
    rng = np.random.default_rng(0)
    x = rng.integers(0, V, (B, L))
    t = np.array([0.1, 0.4, 0.7, 1.0], F32)
    ts = np.array([0.1, 0.55, 0.9, 1.0], F32)
    zt, zs = train.corrupt_pair(x, t, ts, eps, seed=3, step=5, mask_id=V)
    for b in range(B):
        mt, ms = zt[b] == V, zs[b] == V
        assert not (mt & ~ms).any()
        assert np.array_equal(zt[b][~mt], x[b][~mt]) and np.array_equal(zs[b][~ms], x[b][~ms])
        p = (1 - eps) * float(t[b])
        assert abs(mt.mean() - p) < 5 * math.sqrt(max(p * (1 - p), 1e-12) / L) + 1e-9
        a_t, a_s = 1 - (1 - eps) * float(t[b]), 1 - (1 - eps) * float(ts[b])
        if a_t > 0 and (~mt).sum() > 0:
            q = 1 - a_s / a_t
            frac = (ms & ~mt).sum() / (~mt).sum()
            assert abs(frac - q) < 5 * math.sqrt(max(q * (1 - q), 1e-12) / (~mt).sum()) + 1e-9
    assert np.array_equal(zt[0], zs[0])           # t' = t: the same canvas


def test_lambda_weight_is_the_continuous_limit():
    """The 1/t weight is lambda_t(i) = (alpha_t - alpha_s)/(1 - alpha_t) of the theorem
    (sigma = 0) per unit time, for alpha_t = 1 - (1 - eps) t as the corruption uses it."""
    eps = 1e-3
    for t in (0.05, 0.3, 0.9):
        for T in (1000, 100000):
            s = t - 1.0 / T
            a_t, a_s = 1 - float(train.mask_threshold(t, eps)), 1 - (1 - eps) * s
            lam = (a_s - a_t) / (1 - a_t)
            assert abs(lam * T - 1 / t) < 2e-6 * T / t + 20.0 / (T * t * t)


def test_stale_times_follow_the_recipe():
    B = 4096
    t, ts, K, T, k = train.stale_times(B, seed=9, step=2, eps=1e-3)
    assert (t >= 1e-3).all() and (t < 1).all()
    gaps = np.diff(np.sort(t.astype(np.float64)))
    assert np.allclose(gaps, (1 - 1e-3) / B, atol=1e-6)          # antithetic: evenly spread
    assert set(K.tolist()) == {1, 2, 4, 8} and set(T.tolist()) == set(train.BUDGETS_T)
    assert (k >= 0).all() and (k < K).all()
    assert (ts <= 1).all() and (ts >= t).all()
    ok = ts < 1
    assert np.allclose(ts[ok].astype(np.float64) - t[ok], k[ok] / T[ok], atol=1e-7)
    for vals, n in ((K, 4), (T, 6)):
        cnt = np.unique(vals, return_counts=True)[1]
        assert ((cnt - B / n) ** 2 / (B / n)).sum() < 25


def test_row_losses_special_cases():
    V = 37
    lg = np.zeros((3, V))
    assert np.allclose(train.row_losses(lg, [0, 5, 36], [True, True, False]), [math.log(V), math.log(V), 0.0])
    lg = np.zeros((1, V))
    lg[0, 4] = 60.0
    assert train.row_losses(lg, [4], [True])[0] < 1e-20
    rng = np.random.default_rng(1)
    lg = rng.normal(size=(5, 11)) * 3
    x = rng.integers(0, 11, 5)
    for r in range(5):                                               # brute force
        z = math.fsum(math.exp(v) for v in lg[r])
        assert abs(train.row_losses(lg[r:r + 1], [x[r]], [True])[0] - (math.log(z) - lg[r, x[r]])) < 1e-12
    assert np.allclose(train.row_losses(lg + 7.5, x, np.ones(5, bool)), train.row_losses(lg, x, np.ones(5, bool)))


def test_train_loss_structure():
    """Fresh anchor (t' = t) equals running the network on z_t alone; the loss sums only
    the positions masked in z_t, weighted by 1/t; a row with nothing masked has loss 0."""
    cfg = synth.get_config("tiny")
    tensors = synth.make_weights(cfg, perturb=True)
    net = network.Network(network.Weights(cfg, [s[0] for s in synth.weight_specs(cfg)], tensors))
    V, L = cfg["vocab"], 24
    x = np.random.default_rng(2).integers(0, V, (3, L))
    t = np.array([0.5, 0.8, 1e-6], F32)
    loss, zt, zs, n = train.train_loss(net, x, t, t, 1e-3, seed=4, step=0)
    assert np.array_equal(zt, zs) and n[2] == 0 and loss[2] == 0.0
    pos = np.arange(L)
    for b in range(2):
        c = net.shared(zt[b], pos)
        logits = net.head(net.denoise(net.fuse(c, {"h": net.anchor_cache(c, pos)["h"], "c": c}), pos))
        m = zt[b] == V
        ref = sum(math.log(math.fsum(math.exp(v) for v in logits[l])) - logits[l, x[b, l]] for l in np.flatnonzero(m))
        assert abs(loss[b] - ref / float(t[b])) < 1e-9 * max(1.0, abs(loss[b]))
    # a stale anchor changes the prediction
    ts = np.array([0.9, 0.95, 0.5], F32)
    loss2 = train.train_loss(net, x, t, ts, 1e-3, seed=4, step=0)[0]
    assert not np.allclose(loss2[:2], loss[:2])
