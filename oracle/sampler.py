"""Masked-diffusion reverse step with confidence-ranked unmasking (oracle).

Semantics (App. B.1.1, MDLM posterior with zero-masking and carry-over, sigma_t = 0):
a position that is already decoded keeps its token; a masked position may only
become a real token (the head has no column for the mask id).  Which masked
positions are revealed at step i follows the linear schedule: n_i positions, the
ones whose sampled token is most confident.

Sampling contract, identical on CPU and GPU so that token choices and unmask
order can be compared bit for bit.  Every decision is taken in IEEE float32 with
individually rounded +, -, *, / (no fused multiply-add):

* uniform u for (row b, absolute position l, vocab entry v, step id) is word
  (v mod 4) of Philox4x32-10 (Salmon et al., SC'11) at counter
  (v div 4, l, b, step_id) with key (seed low 32 bits, seed high 32 bits), mapped
  to u = (2*(x >> 9) + 1) * 2^-24, which lies in [2^-24, 1 - 2^-24];
* Gumbel noise G = -log(-log u); the token is argmax_v (l_v * inv_temp + G_v) with
  ties broken towards the smaller v (Gumbel-max sampling from softmax(l/temp));
* confidence = log-softmax of the chosen token at temperature temp, with the
  normaliser summed exactly in 64-bit fixed point over groups of 64 consecutive
  vocabulary entries (g = v div 64; the last group may be shorter):
  m_g = max_{v in g} l'_v, S_g = sum_{v in g} rint(exp(l'_v - m_g) * 2^40),
  S = sum_g rint(float(S_g) * exp(m_g - m)), conf = (l'_x - m) - log(float(S) * 2^-40),
  where l' = l * inv_temp, m = max l' = max_g m_g, float() rounds to nearest even and
  exp of an argument below -30 is 0.  Every sum is over integers, so any summation
  order gives the same bits, and a group only needs its own 64 logits: a kernel
  that sees the vocabulary one tile at a time (the vocabulary projection's own
  output tiles) computes the same confidence as one that sees the whole row;
* ranking key: confidence descending, then position ascending.

Nucleus truncation (top-p, used with the remasking sampler): with m = max l', each
entry has the fixed-point weight q_v = rint(exp(l'_v - m) 2^40) (int64) and Q = sum_v q_v.
The nucleus is {v : q_v >= tau}, tau the largest weight whose tail sum
sum_{q_v >= tau} q_v reaches ceil(p Q) (p a float32, the product exact), i.e. the
highest-probability entries until their mass reaches p, with every entry tied at the
boundary kept.  The token is the Gumbel-max over the nucleus; the confidence stays the
untruncated log-probability.

Remasking posterior (eq. inf-post-TADM, the ReMDM form with sigma_t > 0), an
alternative reverse step: each position of the active canvas decides on its own
with one more uniform, word 0 of Philox4x32-10 at counter (2^31, l, b, step_id) --
word 0 of the counter never reaches 2^31 for the vocabulary draws.  A decoded
position becomes the mask with probability sigma_t; a masked position takes its
Gumbel-max token with probability (alpha_s - (1 - sigma_t) alpha_t) / (1 - alpha_t)
and stays masked otherwise.  Both probabilities are float32 numbers that the caller
computes once per step (``loop.remask_probs``); a position moves iff u < probability.

``log32`` and ``exp32`` are this module's own float32 logarithm and exponential:
exponent/mantissa split with the mantissa in [sqrt(1/2), sqrt(2)] and the series
log m = 2 atanh(s), s = (m-1)/(m+1); exponential by Cody-Waite reduction with
ln2 split into a 15-bit head and a tail, and the degree-7 Taylor polynomial.
"""
import numpy as np

U32 = np.uint32
F32 = np.float32

# Philox4x32 round multipliers and Weyl key increments (Salmon et al., SC'11).
PHILOX_M0, PHILOX_M1 = 0xD2511F53, 0xCD9E8D57
PHILOX_W0, PHILOX_W1 = 0x9E3779B9, 0xBB67AE85


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Ten Philox4x32 rounds; all arguments uint32 (broadcastable arrays)."""
    c = [np.asarray(x, dtype=np.uint64) for x in (c0, c1, c2, c3)]
    k0 = np.uint64(k0) if np.isscalar(k0) else np.asarray(k0, dtype=np.uint64)
    k1 = np.uint64(k1) if np.isscalar(k1) else np.asarray(k1, dtype=np.uint64)
    mask = np.uint64(0xFFFFFFFF)
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + np.uint64(PHILOX_W0)) & mask
            k1 = (k1 + np.uint64(PHILOX_W1)) & mask
        p0 = np.uint64(PHILOX_M0) * c[0]
        p1 = np.uint64(PHILOX_M1) * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & mask
        hi1, lo1 = p1 >> np.uint64(32), p1 & mask
        c = [hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0]
    return [x.astype(U32) for x in c]


def bits_to_uniform(x):
    """u = (2*(x >> 9) + 1) * 2^-24 (exact in float32; never 0 or 1)."""
    k = (np.asarray(x, dtype=U32) >> U32(9)).astype(np.int64) * 2 + 1
    return k.astype(F32) * F32(2.0 ** -24)


# float32 constants, given by their bit patterns.
def _f(bits):
    return np.array([bits], dtype=U32).view(F32)[0]


LN2_HI = _f(0x3F317200)      # 0.693145751953125 (15 significant bits)
LN2_LO = _f(0x35BFBE8E)      # ln 2 - LN2_HI
INV_LN2 = _f(0x3FB8AA3B)     # 1/ln 2
SQRT2_BITS = 0x3FB504F3      # float32 nearest sqrt(2)
# log: 2 atanh(s) = 2 s + s R(z), z = s^2, R = 2/3 z + 2/5 z^2 + 2/7 z^3 + 2/9 z^4 + 2/11 z^5
# (the atanh series), coefficients from the highest down
LOG_C = [_f(0x3E3A2E8C), _f(0x3E638E39), _f(0x3E924925), _f(0x3ECCCCCD), _f(0x3F2AAAAB)]
# exp: e^r = 1 + r + r^2 c(r), c = 1/2 + r/6 + ... + r^5/7! (Taylor), from the highest down
EXP_C = [_f(0x39500D01), _f(0x3AB60B61), _f(0x3C088889), _f(0x3D2AAAAB), _f(0x3E2AAAAB), F32(0.5)]
EXP_CUTOFF = F32(-30.0)


def log32(x):
    """Natural log of positive normal float32 values, in float32 arithmetic (within
    1 ulp: the exhaustive sweep of the tests).

    x = 2^e m with m in [sqrt(1/2), sqrt(2)), f = m - 1 (exact), s = f / (2 + f), and
    log(1 + f) = 2 atanh(s) = 2 s + s R(s^2).  Since 2 s = f - s f and
    s f = f^2 / 2 - s f^2 / 2, the sum is taken as f - (f^2/2 - s (f^2/2 + R)): the exact
    f leads and every rounded term is small beside it (the arrangement of Sun's fdlibm
    logarithm).  e ln 2 is added in two parts (Cody-Waite)."""
    x = np.asarray(x, dtype=F32)
    bits = x.view(U32)
    e = (bits >> U32(23)).astype(np.int32) - 127
    mb = (bits & U32(0x007FFFFF)) | U32(0x3F800000)
    big = mb > U32(SQRT2_BITS)
    mb = np.where(big, mb - U32(0x00800000), mb).astype(U32)
    e = e + big.astype(np.int32)
    m = mb.view(F32)
    f = m - F32(1.0)
    s = f / (F32(2.0) + f)
    z = s * s
    c = LOG_C[0]
    for k in LOG_C[1:]:
        c = c * z + k
    R = z * c
    hfsq = F32(0.5) * f * f
    ef = e.astype(F32)
    return (ef * LN2_HI - ((hfsq - (s * (hfsq + R) + ef * LN2_LO)) - f)).astype(F32)


def exp32(y):
    """exp(y) for float32 y <= 0, in float32 arithmetic (within 1 ulp: the exhaustive
    sweep of the tests); 0 below -30.

    k = rint(y / ln 2), r = y - k ln 2 with ln 2 in two parts (Cody-Waite): rh = y - k
    ln2_hi is exact, r = rh - k ln2_lo.  e^r = 1 + r + r^2 c(r), summed as
    1 + (rh + (r^2 c(r) - k ln2_lo)) so that the rounding of r does not enter the linear
    term; then times 2^k (exact)."""
    y = np.asarray(y, dtype=F32)
    yc = np.maximum(y, EXP_CUTOFF)
    k = np.rint(yc * INV_LN2).astype(F32)
    rh = yc - k * LN2_HI
    kl = k * LN2_LO
    r = rh - kl
    c = EXP_C[0]
    for q in EXP_C[1:]:
        c = c * r + q
    q = (r * r) * c
    p = F32(1.0) + (rh + (q - kl))
    scale = ((k.astype(np.int32) + 127).astype(U32) << U32(23)).view(F32)
    return np.where(y < EXP_CUTOFF, F32(0.0), p * scale).astype(F32)


def uniforms(V, pos, row, step_id, seed):
    """u[v] for one (row, position, step): Philox words laid out over the vocabulary."""
    n_ctr = (V + 3) // 4
    c0 = np.arange(n_ctr, dtype=U32)
    w = philox4x32_10(c0, U32(pos), U32(row), U32(step_id),
                      U32(seed & 0xFFFFFFFF), U32((seed >> 32) & 0xFFFFFFFF))
    words = np.stack(w, axis=1).reshape(-1)[:V]
    return bits_to_uniform(words)


GROUP = 64  # vocabulary entries per normaliser group


def normaliser(lp):
    """(m, S): the row maximum of the scaled logits lp and the two-level fixed-point
    normaliser, S ~ 2^40 * sum_v exp(lp_v - m).  The row is padded with -inf to whole
    groups (exp of -inf - m_g is 0); every group holds at least one real entry."""
    V = lp.shape[0]
    ng = -(-V // GROUP)
    padded = np.full(ng * GROUP, -np.inf, dtype=F32)
    padded[:V] = lp
    seg = padded.reshape(ng, GROUP)
    mg = seg.max(axis=1)                                                     # m_g
    Sg = np.rint(exp32(seg - mg[:, None]) * F32(2.0 ** 40)).astype(np.int64).sum(axis=1)
    m = mg.max()
    terms = np.rint((Sg.astype(F32) * exp32((mg - m).astype(F32))).astype(F32)).astype(np.int64)
    return m, int(terms.sum())


def nucleus(lp, top_p):
    """Boolean mask of the top-p nucleus of the scaled logits lp (module docstring)."""
    m = lp.max()
    q = np.rint(exp32(lp - m) * F32(2.0 ** 40)).astype(np.int64)
    Q = int(q.sum())
    num, den = float(np.float32(top_p)).as_integer_ratio()
    target = -(-(num * Q) // den)                         # ceil(p Q), exact
    qs = np.sort(q)[::-1]
    idx = int(np.searchsorted(np.cumsum(qs), target))     # first prefix whose sum >= target
    tau = int(qs[min(idx, qs.size - 1)])
    return q >= tau


def sample_position(logits_row, inv_temp, pos, row, step_id, seed, top_p=1.0):
    """(token, confidence) for one masked position; logits_row is float32 [V]."""
    lg = np.asarray(logits_row, dtype=F32)
    V = lg.shape[0]
    lp = lg * F32(inv_temp)
    u = uniforms(V, pos, row, step_id, seed)
    gumbel = -log32(-log32(u))
    score = lp + gumbel
    if np.float32(top_p) < 1.0:
        score = np.where(nucleus(lp, top_p), score, -np.inf)
    tok = int(np.argmax(score))            # first maximum: smallest v on ties
    m, S = normaliser(lp)
    norm = F32(np.int64(S).astype(F32)) * F32(2.0 ** -40)
    conf = F32(lp[tok] - m) - log32(np.array([norm], dtype=F32))[0]
    return tok, F32(conf)


def rank_order(conf, candidates):
    """Candidate positions ordered by (confidence desc, position asc)."""
    cand = np.flatnonzero(candidates)
    order = np.lexsort((cand, -conf[cand].astype(np.float64)))
    return cand[order]


def reverse_step(logits, canvas, mask_id, n_unmask, pos0, row, step_id, seed, inv_temp, top_p=1.0):
    """One reverse step for one row of the active canvas.

    logits [Lc, V] float32 (all canvas positions), canvas [Lc] ints, pos0 = absolute
    position of canvas entry 0.  Returns (next canvas, choice, conf); choice/conf
    are -1 / -inf at positions that are not masked.
    """
    canvas = np.asarray(canvas)
    Lc = canvas.shape[0]
    masked = canvas == mask_id
    choice = np.full(Lc, -1, dtype=np.int64)
    conf = np.full(Lc, -np.inf, dtype=F32)
    for j in np.flatnonzero(masked):
        choice[j], conf[j] = sample_position(logits[j], inv_temp, pos0 + j, row, step_id, seed, top_p)
    n = min(int(n_unmask), int(masked.sum()))
    sel = rank_order(conf, masked)[:n]
    nxt = canvas.copy()
    nxt[sel] = choice[sel]
    return nxt, choice, conf


DECISION_WORD0 = 0x80000000  # Philox counter word 0 of the per-position decision uniform


def decision_uniforms(pos, row, step_id, seed):
    """One uniform per absolute position in ``pos`` (array) for row ``row`` at a step."""
    pos = np.asarray(pos, dtype=U32)
    w = philox4x32_10(np.full(pos.shape, DECISION_WORD0, dtype=U32), pos, U32(row), U32(step_id),
                      U32(seed & 0xFFFFFFFF), U32((seed >> 32) & 0xFFFFFFFF))
    return bits_to_uniform(w[0])


def remask_step(logits, canvas, mask_id, p_unmask, sigma, pos0, row, step_id, seed, inv_temp, top_p=1.0):
    """One reverse step of the remasking posterior for one row of the active canvas.

    logits [Lc, V] float32, canvas [Lc], pos0 = absolute position of canvas entry 0,
    p_unmask / sigma float32.  Returns (next canvas, choice) with choice -1 where the
    entry was not masked.
    """
    canvas = np.asarray(canvas)
    Lc = canvas.shape[0]
    u = decision_uniforms(pos0 + np.arange(Lc), row, step_id, seed)
    nxt = canvas.copy()
    choice = np.full(Lc, -1, dtype=np.int64)
    for j in range(Lc):
        if canvas[j] == mask_id:
            choice[j] = sample_position(logits[j], inv_temp, pos0 + j, row, step_id, seed, top_p)[0]
            if u[j] < F32(p_unmask):
                nxt[j] = choice[j]
        elif u[j] < F32(sigma):
            nxt[j] = mask_id
    return nxt, choice
