"""Pins of the oracle's sampler: Philox, float32 log/exp, Gumbel-max, ranking, carry-over."""
import math
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import sampler as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
rng = np.random.default_rng(2)


def _kat():
    rows = []
    for line in open(os.path.join(GOLDEN, "philox_kat.txt")):
        if line.strip() and not line.startswith("#"):
            rows.append([int(x, 16) for x in line.split()])
    return rows


def test_philox_known_answers():
    for r in _kat():
        out = S.philox4x32_10(*r[:6])
        assert [int(x) for x in out] == r[6:]


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
def test_philox_matches_rocrand(tmp_path):
    """Cross-check against rocRAND's independent Philox4x32-10 (run, host side)."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    exe = tmp_path / "rocrand_philox"
    subprocess.run([hipcc, "--offload-arch=gfx950", "-O1", "-o", str(exe),
                    os.path.join(GOLDEN, "rocrand_philox.cpp")], check=True,
                   capture_output=True)
    ctr = rng.integers(0, 2 ** 32, size=(200, 6), dtype=np.uint64)
    text = "\n".join(" ".join(f"{int(v):x}" for v in row) for row in ctr) + "\n"
    res = subprocess.run([str(exe)], input=text, capture_output=True, text=True, check=True)
    ref = np.array([[int(x, 16) for x in line.split()] for line in res.stdout.split("\n") if line])
    out = S.philox4x32_10(*[ctr[:, i].astype(np.uint32) for i in range(6)])
    np.testing.assert_array_equal(np.stack(out, 1).astype(np.int64), ref)


def test_uniform_range_is_open_and_exact():
    x = np.array([0, 511, 512, 2 ** 32 - 1], dtype=np.uint32)
    u = S.bits_to_uniform(x)
    assert u[0] == np.float32(2.0 ** -24) and u[1] == u[0]
    assert u[2] == np.float32(3 * 2.0 ** -24)
    assert u[3] == np.float32(1 - 2.0 ** -24) and u[3] < 1
    k = rng.integers(0, 2 ** 32, size=10000, dtype=np.uint64).astype(np.uint32)
    exact = ((k >> 9).astype(np.float64) * 2 + 1) / 2 ** 24
    np.testing.assert_array_equal(S.bits_to_uniform(k).astype(np.float64), exact)


def _ulp_err(got, ref):
    return np.abs(got.astype(np.float64) - ref) / np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)


# Exhaustive sweeps: every float32 in the domain the sampling contract feeds each
# function (log: the uniforms u in [2^-24, 1), E = -log u up to 17, and the normaliser
# S 2^-40 up to 2^19; exp: every argument in [-30, 0]), against float64 libm, in chunks
# of 2^24 values spread over worker processes.
LOG_LO, LOG_HI = np.float32(2.0 ** -24).view(np.uint32), np.float32(2.0 ** 19).view(np.uint32)
EXP_LO, EXP_HI = np.float32(-0.0).view(np.uint32), np.float32(-30.0).view(np.uint32)
CHUNK = 1 << 24


def _ulp_chunk(args):
    which, a, hi = args
    bits = np.arange(a, min(a + CHUNK, hi + 1), dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    if which == "log":
        x = x[x != 1]
        got, ref = S.log32(x), np.log(x.astype(np.float64))
    else:
        got, ref = S.exp32(x), np.exp(x.astype(np.float64))
    err = _ulp_err(got, ref)
    i = int(np.argmax(err))
    return float(err[i]), float(x[i]), int(x.size)


def _sweep(which, lo, hi):
    import multiprocessing as mp
    jobs = [(which, a, int(hi)) for a in range(int(lo), int(hi) + 1, CHUNK)]
    with mp.get_context("fork").Pool(min(8, os.cpu_count() or 1)) as pool:
        res = pool.map(_ulp_chunk, jobs)
    return max(r[0] for r in res), sum(r[2] for r in res)


def test_log32_within_one_ulp_exhaustive():
    worst, n = _sweep("log", LOG_LO, LOG_HI)
    print(f"log32: max error {worst:.4f} ulp over {n} float32 values in [2^-24, 2^19]")
    assert n > 3.5e8
    assert worst <= 1.0
    assert S.log32(np.float32(1.0)) == 0.0


def test_exp32_within_one_ulp_exhaustive():
    worst, n = _sweep("exp", EXP_LO, EXP_HI)
    print(f"exp32: max error {worst:.4f} ulp over {n} float32 values in [-30, 0]")
    assert n > 1.0e9
    assert worst <= 1.0
    assert S.exp32(np.float32(0.0)) == 1.0
    assert S.exp32(np.float32(-30.5)) == 0.0


def test_sample_matches_float64_on_tiny_vocab():
    """Brute force in float64: argmax(l + G) over an enumerated score table and the
    exact log-softmax; the float32 contract must agree away from near-ties."""
    checked = 0
    for trial in range(300):
        V = int(rng.integers(2, 9))
        lg = (rng.normal(size=V) * 2).astype(np.float32)
        tok, conf = S.sample_position(lg, 1.0, pos=trial, row=3, step_id=7, seed=99)
        u = S.uniforms(V, trial, 3, 7, 99).astype(np.float64)
        score = lg.astype(np.float64) - np.log(-np.log(u))
        best = np.sort(score)[::-1]
        if best[0] - best[1] > 1e-4:
            assert tok == int(np.argmax(score))
            checked += 1
        l64 = lg.astype(np.float64)
        ref = l64[tok] - l64.max() - math.log(np.exp(l64 - l64.max()).sum())
        assert abs(conf - ref) < 2e-6 * (1 + abs(ref))
    assert checked > 250


@pytest.mark.parametrize("V,std", [(63, 1.0), (64, 1.0), (65, 3.0), (1000, 5.0), (4099, 30.0), (130, 0.0)])
def test_grouped_normaliser_matches_float64(V, std):
    """S * 2^-40 approximates sum_v exp(l'_v - m) to float32 accuracy for any number of
    64-entry groups (partial last group, spreads that hit the -30 cut-off), and the
    confidence is the float64 log-softmax of the chosen token within that bound."""
    lg = (rng.normal(size=V) * std).astype(np.float32)
    m, Sx = S.normaliser(lg)
    l64 = lg.astype(np.float64)
    ref = np.exp(l64 - l64.max()).sum()
    assert m == lg.max()
    assert abs(Sx * 2.0 ** -40 - ref) <= 4e-7 * ref
    tok, conf = S.sample_position(lg, 1.0, pos=V, row=1, step_id=2, seed=5)
    lsm = l64[tok] - l64.max() - math.log(ref)
    assert abs(conf - lsm) < 2e-6 * (1 + abs(lsm))


def test_grouped_normaliser_worked_example():
    """Hand-worked: 64 equal logits and one more, 1 lower, in a second group.  Group 0
    sums to 64 * 2^40 exactly; group 1 is 2^40 at its own maximum and is scaled by
    exp(-1) (a power-of-two multiple of a float32, so already an integer)."""
    lg = np.zeros(65, np.float32)
    lg[64] = -1.0
    m, Sx = S.normaliser(lg)
    e1 = S.exp32(np.float32(-1.0))
    assert m == 0.0 and Sx == 64 * 2 ** 40 + int(e1 * np.float32(2.0 ** 40))
    # equal logits: the normaliser is exactly V and the confidence exactly -log V
    for V in (1, 64, 130):
        m, Sx = S.normaliser(np.full(V, 2.5, np.float32))
        assert Sx == V * 2 ** 40
        assert S.sample_position(np.full(V, 2.5, np.float32), 1.0, 0, 0, 0, 1)[1] == -S.log32(np.float32(V))


def test_gumbel_max_frequencies_match_softmax():
    """Gumbel-max draws follow softmax(l / temp): chi-square over 40000 step ids."""
    lg = np.array([0.3, -1.0, 1.2, 0.0, 2.0, -0.5], dtype=np.float32)
    temp = 0.8
    inv = np.float32(1 / temp)
    n = 40000
    counts = np.zeros(6)
    steps = np.arange(n, dtype=np.uint32)
    w = S.philox4x32_10(np.zeros(n, np.uint32), np.uint32(5), np.uint32(1), steps,
                        np.uint32(123), np.uint32(0))
    u = np.stack([S.bits_to_uniform(x) for x in w], 1)  # [n, 4] words 0..3
    w2 = S.philox4x32_10(np.ones(n, np.uint32), np.uint32(5), np.uint32(1), steps,
                         np.uint32(123), np.uint32(0))
    u = np.concatenate([u, np.stack([S.bits_to_uniform(x) for x in w2], 1)[:, :2]], 1)
    score = lg * inv - S.log32(-S.log32(u))
    for t in np.argmax(score, axis=1):
        counts[t] += 1
    # the sampler's own path on a few step ids gives the same draws
    for k in range(20):
        assert S.sample_position(lg, inv, 5, 1, k, 123)[0] == int(np.argmax(score[k]))
    p = np.exp(lg / temp - np.max(lg / temp))
    p /= p.sum()
    chi2 = ((counts - n * p) ** 2 / (n * p)).sum()
    assert chi2 < 25.7  # 5 dof, p ~ 1e-4


def test_rank_order_is_full_sort():
    for _ in range(50):
        Lc = int(rng.integers(1, 40))
        conf = np.round(rng.normal(size=Lc), 1).astype(np.float32)  # many exact ties
        cand = rng.random(Lc) < 0.7
        ref = sorted(np.flatnonzero(cand), key=lambda j: (-float(conf[j]), j))
        assert list(S.rank_order(conf, cand)) == ref


def test_reverse_step_carry_over_and_count():
    V, Lc, mask = 11, 30, 11
    canvas = rng.integers(0, V, size=Lc)
    canvas[rng.random(Lc) < 0.6] = mask
    logits = rng.normal(size=(Lc, V)).astype(np.float32)
    n_masked = int((canvas == mask).sum())
    for n in (0, 1, 5, n_masked, n_masked + 3):
        nxt, choice, conf = S.reverse_step(logits, canvas, mask, n, 100, 0, 4, 7, np.float32(1))
        keep = canvas != mask
        assert np.array_equal(nxt[keep], canvas[keep])                  # never re-mask / change
        revealed = (canvas == mask) & (nxt != mask)
        assert revealed.sum() == min(n, n_masked)                        # clamped count
        assert np.all(nxt[revealed] < V)                                 # zero-masking
        assert np.all(nxt[revealed] == choice[revealed])
        top = S.rank_order(conf, canvas == mask)[: min(n, n_masked)]
        assert set(np.flatnonzero(revealed)) == set(top)
