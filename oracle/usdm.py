"""Entropy-bound sampling of a uniform-state diffusion model (Algorithm 2) -- oracle,
test infrastructure only.

One reverse step n (T .. 1) of one canvas row, given the decoder logits L [Lc, V]:

* temperature tau_n = tau_min + (tau_max - tau_min) n / T; scaled logits
  l' = l * inv_temp with inv_temp = float32(1 / tau_n) (float64 arithmetic on the
  float32 parameters);
* x_hat = argmax_v l_v (ties towards the smaller v), the step's argmax canvas;
* x_tilde ~ Cat(softmax(l')): the Gumbel-max draw of the masked sampler's contract
  (Philox counter (v/4, position, row, step id)), no nucleus;
* entropy of softmax(l'), with m = max l', y_v = l'_v - m, e_v = exp32(y_v):
  A = sum_v rint(e_v 2^40), B = sum_v rint((-y_v * e_v) 2^40) over e_v > 0 (int64,
  order-free),
  H = log32(float(A) 2^-40) + float(B) / float(A) (float32 operations; H = log Z +
  sum_v p_v (-y_v) is the entropy with Z = sum_v e_v), Hq = rint(H 2^40) (int64);
* acceptance: positions ordered by (Hq ascending, position ascending); with C_m the
  sum of the first m entropies and M_m their maximum (the m-th, the order being
  ascending), position pi_m is accepted iff C_m - M_m <= eta, i.e. iff the exact sum
  of the Hq ranked before it is <= rint(eta 2^40) (eta float32);
* next canvas (n > 1): accepted positions take x_tilde, the others a fresh uniform
  token: word 0 w of Philox4x32-10 at counter (2^31 + 1, position, row, step id),
  token = (w * V) >> 32.  At n = 1 the canvas becomes x_hat;
* self-conditioning for the next step: s = p E with p = softmax(l') and E the token
  embedding rows [0, V); the decoder adds s to the embeddings of the canvas positions
  (the reading of "Decoder(z, s)").

A block's starting canvas z_T is uniform noise: token (w * V) >> 32 with w word 0 at
counter (2^31 + 2, position, row, block index).
"""
import numpy as np

from . import sampler as smp

F32 = np.float32
U32 = np.uint32
RENOISE_WORD0 = 0x80000001
INIT_WORD0 = 0x80000002
TWO40 = F32(2.0 ** 40)


def inv_temperature(n, T, tau_max, tau_min):
    """float32(1 / tau_n), tau_n = tau_min + (tau_max - tau_min) n / T in float64."""
    hi, lo = float(F32(tau_max)), float(F32(tau_min))
    return F32(1.0 / (lo + (hi - lo) * n / T))


def entropy_stats(logits_row, inv_temp):
    """(A, B, H, Hq) of one row (module docstring)."""
    lp = np.asarray(logits_row, dtype=F32) * F32(inv_temp)
    m = lp.max()
    y = (lp - m).astype(F32)
    e = smp.exp32(y)
    A = int(np.rint(e * TWO40).astype(np.int64).sum())
    with np.errstate(invalid="ignore"):
        terms = np.where(e > 0, np.rint((-y * e).astype(F32) * TWO40), 0.0)   # p log p -> 0 as p -> 0
    Bs = int(terms.astype(np.int64).sum())
    fA, fB = np.array([A, Bs], dtype=np.int64).astype(F32)      # int64 -> float32, one rounding
    H = F32(smp.log32(np.array([fA * F32(2.0 ** -40)], F32))[0] + F32(fB / fA))
    Hq = int(np.rint(np.float64(H) * 2.0 ** 40))
    return A, Bs, H, Hq


def gumbel_token(logits_row, inv_temp, pos, row, step_id, seed):
    """x_tilde: argmax_v (l'_v + G_v), the masked sampler's draw without a nucleus."""
    lp = np.asarray(logits_row, dtype=F32) * F32(inv_temp)
    u = smp.uniforms(lp.shape[0], pos, row, step_id, seed)
    return int(np.argmax(lp + (-smp.log32(-smp.log32(u)))))


def _word0_tokens(word0, pos, row, c3, seed, V):
    pos = np.asarray(pos, dtype=U32)
    w = smp.philox4x32_10(np.full(pos.shape, word0, dtype=U32), pos, U32(row), U32(c3),
                          U32(seed & 0xFFFFFFFF), U32((seed >> 32) & 0xFFFFFFFF))[0]
    return ((w.astype(np.uint64) * np.uint64(V)) >> np.uint64(32)).astype(np.int64)


def renoise_tokens(pos, row, step_id, seed, V):
    """Uniform tokens for the rejected positions of a step."""
    return _word0_tokens(RENOISE_WORD0, pos, row, step_id, seed, V)


def initial_tokens(pos, row, block, seed, V):
    """z_T of a block: a uniform token per position."""
    return _word0_tokens(INIT_WORD0, pos, row, block, seed, V)


def accept_set(Hq, eta):
    """Boolean mask of the accepted positions for exact entropies Hq (int64)."""
    Hq = np.asarray(Hq, dtype=np.int64)
    etaq = int(np.rint(np.float64(F32(eta)) * 2.0 ** 40))
    order = np.lexsort((np.arange(Hq.size), Hq))           # Hq ascending, then position
    before = np.concatenate([[0], np.cumsum(Hq[order])[:-1]])
    acc = np.zeros(Hq.size, dtype=bool)
    acc[order] = before <= etaq
    return acc


def selfcond(logits, inv_temp, embed):
    """s = softmax(l') E in float64 (E = embed[:V])."""
    lp = np.asarray(logits, dtype=F32).astype(np.float64) * np.float64(F32(inv_temp))
    p = np.exp(lp - lp.max(axis=-1, keepdims=True))
    p /= p.sum(axis=-1, keepdims=True)
    V = lp.shape[-1]
    return p @ np.asarray(embed, dtype=np.float64)[:V]


def entropy_step(logits, n, inv_temp, eta, pos0, row, step_id, seed):
    """One step of Algorithm 2 for one row: returns dict(next, x_hat, x_tilde, H, Hq,
    accept); logits [Lc, V] float32, pos0 = absolute position of entry 0."""
    logits = np.asarray(logits, dtype=F32)
    Lc, V = logits.shape
    x_hat = np.argmax(logits, axis=1).astype(np.int64)   # first maximum: smaller v on ties
    x_tilde = np.array([gumbel_token(logits[j], inv_temp, pos0 + j, row, step_id, seed) for j in range(Lc)],
                       dtype=np.int64)
    stats = [entropy_stats(logits[j], inv_temp) for j in range(Lc)]
    H = np.array([s[2] for s in stats], dtype=F32)
    Hq = np.array([s[3] for s in stats], dtype=np.int64)
    acc = accept_set(Hq, eta)
    if n > 1:
        nxt = np.where(acc, x_tilde, renoise_tokens(pos0 + np.arange(Lc), row, step_id, seed, V))
    else:
        nxt = x_hat.copy()
    return dict(next=nxt, x_hat=x_hat, x_tilde=x_tilde, H=H, Hq=Hq, accept=acc)
