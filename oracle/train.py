"""Training objective of TADM:Pretraining (oracle; test infrastructure only).

Theorem T-ANELBO with gamma = 0 and sigma = 0 (Sec. 5), trained as in the pretraining
details of App. C.2: absorbing-state masked diffusion with the log-linear schedule
alpha_t = 1 - (1 - eps) t, continuous t, and a stale anchor time t' = min(1, t + k/T)
with T drawn from the inference step budgets, K from the refresh intervals and the
cache age k uniform in {0, .., K - 1}.

* Pair corruption (eq. fwd and eq. fwd_t_t'): one uniform u per (row b, position l) --
  word 0 of Philox4x32-10 at counter (2^31 + 3, l, b, step) with the sampler's key and
  mapping to (0, 1) -- masks x^l in z_t iff u < float32((1 - eps) t) and in z_t' iff
  u < float32((1 - eps) t').  Since t' >= t every position masked in z_t is masked in
  z_t', and a position kept at t is masked at t' with probability 1 - alpha_t'/alpha_t,
  the transition of eq. fwd_t_t'.
* Forward: c' = S(z_t'), cache = (A(c'), c'); c = S(z_t); logits = head(D(Phi(c, cache))).
* Loss of row b: w_b * sum over positions masked in z_t of -log softmax(logits_l)[x^l],
  w_b = 1 / t_b, the continuous-time limit of lambda_t(i) = (alpha_t - alpha_s)/(1 - alpha_t)
  per unit of time for the log-linear schedule (positions decoded in z_t carry over and
  contribute nothing).
* Times: t_b = eps + (1 - eps) frac(u0 + b / B) (antithetic over the batch, u0 from row 0),
  K_b = {1, 2, 4, 8}[w1 >> 30], T_b = {128, .., 4096}[(6 w2) >> 32], k_b = (K_b w3) >> 32,
  t'_b = min(1, t_b + k_b / T_b), with (w0, w1, w2, w3) Philox4x32-10 at counter
  (2^31 + 4, b, step, 0) and u0 from w0 of row 0; float64 arithmetic, stored as float32
  (t' is recomputed from the float32 t).
"""
import numpy as np

from . import sampler as smp

F32 = np.float32
U32 = np.uint32
CORRUPT_WORD0 = 0x80000003
TIMES_WORD0 = 0x80000004
REFRESH_K = (1, 2, 4, 8)
BUDGETS_T = (128, 256, 512, 1024, 2048, 4096)


def _key(seed):
    return U32(seed & 0xFFFFFFFF), U32((seed >> 32) & 0xFFFFFFFF)


def mask_threshold(t, eps):
    """float32 probability 1 - alpha_t = (1 - eps) t of the log-linear schedule."""
    return F32((1.0 - float(F32(eps))) * float(F32(t)))


def corrupt_pair(x, t, t_stale, eps, seed, step, mask_id):
    """(z_t, z_t') for clean tokens x [B, L] and per-row times (module docstring)."""
    x = np.asarray(x, dtype=np.int64)
    B, L = x.shape
    zt, zs = x.copy(), x.copy()
    k0, k1 = _key(seed)
    for b in range(B):
        w = smp.philox4x32_10(np.full(L, CORRUPT_WORD0, U32), np.arange(L, dtype=U32), U32(b), U32(step), k0, k1)[0]
        u = smp.bits_to_uniform(w)
        zt[b, u < mask_threshold(t[b], eps)] = mask_id
        zs[b, u < mask_threshold(t_stale[b], eps)] = mask_id
    return zt, zs


def stale_times(B, seed, step, eps):
    """(t, t', K, T, k) for a batch of B rows (module docstring)."""
    k0, k1 = _key(seed)
    w = smp.philox4x32_10(np.full(B, TIMES_WORD0, U32), np.arange(B, dtype=U32), U32(step), U32(0), k0, k1)
    w = [x.astype(np.uint64) for x in w]
    u0 = float(smp.bits_to_uniform(w[0][:1].astype(U32))[0])
    e = float(F32(eps))
    t = np.empty(B, F32)
    ts = np.empty(B, F32)
    K = np.empty(B, np.int64)
    T = np.empty(B, np.int64)
    k = np.empty(B, np.int64)
    for b in range(B):
        frac = (u0 + b / B) % 1.0
        t[b] = F32(e + (1.0 - e) * frac)
        K[b] = REFRESH_K[int(w[1][b] >> np.uint64(30))]
        T[b] = BUDGETS_T[int((w[2][b] * np.uint64(6)) >> np.uint64(32))]
        k[b] = int((w[3][b] * np.uint64(K[b])) >> np.uint64(32))
        ts[b] = F32(min(1.0, float(t[b]) + k[b] / T[b]))
    return t, ts, K, T, k


def row_losses(logits, x, masked):
    """Per-position cross-entropy -log softmax(logits)[x] (float64) where masked."""
    lg = np.asarray(logits, dtype=np.float64)
    m = lg.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(lg - m).sum(axis=1))
    ce = lse - lg[np.arange(lg.shape[0]), np.asarray(x)]
    return np.where(masked, ce, 0.0)


def train_loss(net, x, t, t_stale, eps, seed, step):
    """Per-row weighted loss [B] (float64), the corrupted pair and the per-row masked
    counts, for clean tokens x [B, L]."""
    cfg = net.cfg
    mask_id = cfg["vocab"]
    x = np.asarray(x, dtype=np.int64)
    B, L = x.shape
    zt, zs = corrupt_pair(x, t, t_stale, eps, seed, step, mask_id)
    pos = np.arange(L)
    loss = np.zeros(B)
    for b in range(B):
        cache = net.anchor_cache(net.shared(zs[b], pos), pos)
        xf = net.denoise(net.fuse(net.shared(zt[b], pos), cache), pos)
        logits = net.head(xf)
        ce = row_losses(logits, x[b], zt[b] == mask_id)
        loss[b] = ce.sum() / float(F32(t[b]))
    return loss, zt, zs, (zt == mask_id).sum(axis=1)
