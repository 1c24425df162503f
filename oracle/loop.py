"""Anchor-cache inference, Algorithm 1 (oracle; test infrastructure only).

For i = T .. 1: c_i = S(z_i); if (T - i) mod K == 0 the anchor is refreshed,
h_cache = A(c_i); h~_i = Phi(c_i, h_cache); x^_i = D(h~_i); z_{i-1} ~ P(z_i, x^_i, i).

The sampler P reveals n_i = floor(M0 i / T) - floor(M0 (i-1) / T) masked positions
at step i, so that exactly floor(M0 (i-1)/T) stay masked afterwards: the integer
form of the linear schedule alpha_t = 1 - t on the grid t(i) = i/T (Sec. 2.1), with
alpha_0 = 1 making the last step reveal everything.

Single-canvas mode (block_len == gen_len): the prompt and the canvas form one
bidirectional sequence.  Block mode (block_len < gen_len): the prompt is block 0,
run once as a fresh pass whose per-layer K, V become the context; each block of
``block_len`` positions is then denoised for T steps attending to the context and
to itself, and once finished is appended to the context by another fresh pass
(bidirectional within a block, causal across blocks).  The refresh counter
restarts at each block.  Each reverse step has id block*T + (T - i).

``net`` provides shared / anchor_cache / fuse / denoise / head / fresh_kv on one
row (``oracle.network.Network``); ``counts`` records layer calls in the units of
the paper's compute count (one call per layer per step for the batch).
"""
import numpy as np

from . import sampler as smp


def unmask_count(M0, i, T):
    return (M0 * i) // T - (M0 * (i - 1)) // T


def remask_probs(i, T, eta):
    """(sigma, p_unmask) of reverse step i under the linear schedule alpha_t = 1 - t,
    t = i/T, s = (i-1)/T, with the capped remasking probability
    sigma = min(eta, (1 - alpha_s) / alpha_t): the largest sigma for which the posterior
    of eq. inf-post-TADM keeps a non-negative mask probability 1 - alpha_s - sigma alpha_t.
    p_unmask = (alpha_s - (1 - sigma) alpha_t) / (1 - alpha_t).  Computed in float64
    and returned rounded to float32 (the kernels receive the same two numbers)."""
    a_t = 1.0 - i / T
    a_s = 1.0 - (i - 1) / T
    cap = (1.0 - a_s) / a_t if a_t > 0.0 else float("inf")
    sigma = min(float(np.float32(eta)), cap)  # eta is a float32 parameter
    p = (a_s - (1.0 - sigma) * a_t) / (1.0 - a_t)
    return np.float32(sigma), np.float32(p)


def loop_alpha(t, t_on, t_off, alpha_on):
    """alpha(t) of the ReMDM-Loop schedule (reading of the sampler details, App. C.2, after
    the ReMDM paper): rises linearly from 0 at t = 1 to alpha_on at t_on, stays at
    alpha_on down to t_off, rises linearly to 1 at t = 0."""
    if t >= t_on:
        return alpha_on * (1.0 - t) / (1.0 - t_on)
    if t >= t_off:
        return alpha_on
    return alpha_on + (1.0 - alpha_on) * (t_off - t) / t_off


def loop_probs(i, T, eta, t_on, t_off, alpha_on):
    """(sigma, p_unmask) of reverse step i (t = i/T -> s = (i-1)/T) under ReMDM-Loop.

    Steps wholly inside the plateau [t_off, t_on] (alpha_s = alpha_t = alpha_on) remask
    with sigma = min(eta, (1 - alpha_s) / alpha_t); the other steps are plain absorbing
    steps (sigma = 0).  p_unmask = (alpha_s - (1 - sigma) alpha_t) / (1 - alpha_t) as in
    eq. inf-post-TADM.  eta is a float32 parameter (as for ReMDM-Cap), the schedule's
    times and alpha_on are float64; the arithmetic is float64 and the two results are
    rounded to float32."""
    eta = float(np.float32(eta))
    t, s = i / T, (i - 1) / T
    a_t = loop_alpha(t, t_on, t_off, alpha_on)
    a_s = loop_alpha(s, t_on, t_off, alpha_on)
    sigma = 0.0
    if t <= t_on and s >= t_off:
        sigma = min(eta, (1.0 - a_s) / a_t)
    p = (a_s - (1.0 - sigma) * a_t) / (1.0 - a_t)
    return np.float32(sigma), np.float32(p)


def is_refresh(i, T, K):
    return (T - i) % K == 0


class Counts:
    def __init__(self):
        self.anchor_refreshes = 0
        self.layer_calls = 0
        self.steps = 0


def generate(net, prompt, gen_len, T, K, block_len, seed, temperature, mask_id,
             counts=None, trace=None, sample_fn=None, remask_eta=None, top_p=1.0, loop=None):
    """Run Algorithm 1 on every row of ``prompt`` [B, P]; returns tokens [B, P+gen_len].

    ``remask_eta`` selects the remasking posterior with sigma = min(eta, cap) instead of
    confidence-ranked unmasking; ``loop`` = (eta, t_on, t_off, alpha_on) selects it on
    the ReMDM-Loop schedule; ``top_p`` < 1 samples tokens from the nucleus.
    ``trace`` (list) receives per-step dicts (i, step_id,
    refresh, canvas before the step) for tests; ``sample_fn`` replaces the reverse step
    (used by counting tests).
    """
    cfg = net.cfg
    prompt = np.asarray(prompt, dtype=np.int64)
    B, P = prompt.shape
    if gen_len % block_len != 0 or T < 1 or K < 1:
        raise ValueError("invalid generation arguments")
    Ls, La, Ld = cfg["n_shared"], cfg["n_anchor"], cfg["n_denoise"]
    inv_temp = np.float32(1.0 / float(temperature))
    seq = np.concatenate([prompt, np.full((B, gen_len), mask_id, dtype=np.int64)], axis=1)
    single = block_len == gen_len
    if single:
        windows = [(0, P, P + gen_len)]
        ctx = [None] * B
    else:
        windows = [(P + j * block_len, P + j * block_len, P + (j + 1) * block_len)
                   for j in range(gen_len // block_len)]
        ctx = [net.fresh_kv(seq[b, :P], np.arange(P)) if P > 0 else None for b in range(B)]
        if counts is not None and P > 0:
            counts.layer_calls += Ls + La + Ld
    sample = sample_fn or smp.reverse_step
    for j, (w0, c0, w1) in enumerate(windows):
        pos = np.arange(w0, w1)
        M0 = int((seq[0, c0:w1] == mask_id).sum())
        caches = [None] * B
        for i in range(T, 0, -1):
            step_id = j * T + (T - i)
            n = unmask_count(M0, i, T)
            refresh = is_refresh(i, T, K)
            if trace is not None:
                trace.append(dict(block=j, i=i, step_id=step_id, refresh=refresh, n=n,
                                  canvas=seq[:, w0:w1].copy()))
            if counts is not None:
                counts.steps += 1
                counts.layer_calls += Ls + Ld + (La if refresh else 0)
                counts.anchor_refreshes += int(refresh)
            for b in range(B):
                c = net.shared(seq[b, w0:w1], pos, ctx[b])
                if refresh:
                    caches[b] = net.anchor_cache(c, pos, ctx[b])
                ht = net.fuse(c, caches[b])
                xf = net.denoise(ht, pos, ctx[b])
                logits = net.head(xf[c0 - w0:]).astype(np.float32)
                if remask_eta is None and loop is None:
                    extra = {} if sample_fn else {"top_p": top_p}
                    nxt, _, _ = sample(logits, seq[b, c0:w1], mask_id, n, c0, b, step_id,
                                       seed, inv_temp, **extra)
                else:
                    if loop is not None:
                        sigma, p_unmask = loop_probs(i, T, *loop)
                    else:
                        sigma, p_unmask = remask_probs(i, T, remask_eta)
                    nxt, _ = smp.remask_step(logits, seq[b, c0:w1], mask_id, p_unmask, sigma, c0, b,
                                             step_id, seed, inv_temp, top_p)
                seq[b, c0:w1] = nxt
        if not single:
            for b in range(B):
                kv = net.fresh_kv(seq[b, w0:w1], pos, ctx[b])
                ctx[b] = kv if ctx[b] is None else {
                    li: (np.concatenate([ctx[b][li][0], kv[li][0]]),
                         np.concatenate([ctx[b][li][1], kv[li][1]])) for li in kv}
            if counts is not None:
                counts.layer_calls += Ls + La + Ld
    return seq


def generate_usdm(net, prompt, gen_len, T, K, block_len, seed, eta=0.1, tau_max=0.8, tau_min=0.4, trace=None):
    """Algorithm 1 with the entropy-bound sampler of Algorithm 2 (uniform-state
    diffusion) on every row of ``prompt`` [B, P]; returns tokens [B, P+gen_len].

    Each block starts from uniform noise (``usdm.initial_tokens``) and a zero
    self-conditioning signal; step n uses temperature tau_n and the anchor is refreshed
    iff (T - n) mod K == 0, with the self-conditioning signal of the previous step
    added to the canvas embeddings of every decoder pass (the anchor's included).  The
    last step leaves the argmax canvas.  Step ids and block mode as in ``generate``."""
    from . import usdm
    cfg = net.cfg
    prompt = np.asarray(prompt, dtype=np.int64)
    B, P = prompt.shape
    V, d = cfg["vocab"], cfg["d_model"]
    if gen_len % block_len != 0 or T < 1 or K < 1:
        raise ValueError("invalid generation arguments")
    seq = np.concatenate([prompt, np.zeros((B, gen_len), dtype=np.int64)], axis=1)
    single = block_len == gen_len
    if single:
        windows = [(0, P, P + gen_len)]
        ctx = [None] * B
    else:
        windows = [(P + j * block_len, P + j * block_len, P + (j + 1) * block_len)
                   for j in range(gen_len // block_len)]
        ctx = [net.fresh_kv(seq[b, :P], np.arange(P)) if P > 0 else None for b in range(B)]
    E = net.W["embed"]
    for j, (w0, c0, w1) in enumerate(windows):
        pos = np.arange(w0, w1)
        for b in range(B):
            seq[b, c0:w1] = usdm.initial_tokens(np.arange(c0, w1), b, j, seed, V)
        caches = [None] * B
        sc = np.zeros((B, w1 - w0, d))
        for n in range(T, 0, -1):
            step_id = j * T + (T - n)
            inv_temp = usdm.inv_temperature(n, T, tau_max, tau_min)
            refresh = is_refresh(n, T, K)
            for b in range(B):
                c = net.shared(seq[b, w0:w1], pos, ctx[b], sc=sc[b])
                if refresh:
                    caches[b] = net.anchor_cache(c, pos, ctx[b])
                xf = net.denoise(net.fuse(c, caches[b]), pos, ctx[b])
                logits = net.head(xf[c0 - w0:]).astype(np.float32)
                r = usdm.entropy_step(logits, n, inv_temp, eta, c0, b, step_id, seed)
                if trace is not None:
                    trace.append(dict(block=j, n=n, row=b, step_id=step_id, refresh=refresh,
                                      canvas=seq[b, c0:w1].copy(), **r))
                if n > 1:
                    sc[b, c0 - w0:] = usdm.selfcond(logits, inv_temp, E)
                seq[b, c0:w1] = r["next"]
        if not single:
            for b in range(B):
                kv = net.fresh_kv(seq[b, w0:w1], pos, ctx[b])
                ctx[b] = kv if ctx[b] is None else {
                    li: (np.concatenate([ctx[b][li][0], kv[li][0]]),
                         np.concatenate([ctx[b][li][1], kv[li][1]])) for li in kv}
    return seq


def layer_call_count(T, K, L_shared, L_anchor, L_denoise):
    """Closed form of eq. anchor-cache-compute: T (L_S + L_D) + ceil(T/K) L_A."""
    return T * (L_shared + L_denoise) + -(-T // K) * L_anchor
