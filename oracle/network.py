"""TADM networks in float64 (oracle; test infrastructure only).

Decomposition (Sec. 3.1): c = S(z), h = A(c), h~ = Phi(c, h'), x = D(h~).
S is the token embedding plus ``n_shared`` transformer layers, A is ``n_anchor``
layers with no final norm, D is ``n_denoise`` layers, a final RMSNorm and an
untied vocabulary head with one column per real token (the mask id has an
embedding row but no output column: zero-masking, App. B.1.1).

Transformer layers are pre-norm blocks without time conditioning (the DiT blocks
of App. C.2 with time conditioning disabled): RMSNorm, multi-head attention with
rotary positions (rotate-half, base 10^4) and grouped KV heads, residual, RMSNorm,
feed-forward (GELU, SwiGLU or GeGLU), residual.

Precision.  Weights are the stored values (bf16 or fp32) and all arithmetic is
float64.  A bf16 model (config dtype "bf16") additionally takes every operand of a
matrix product in bf16: activations are rounded to bf16 (round to nearest even)
where they enter a product -- the normalised input of each projection, Q and K after
the rotary embedding, V, the softmax probabilities, the attention output, the
feed-forward hidden state, the fusion input u and hidden state, the head input --
while accumulation, norms, softmax, residual stream and elementwise maths stay in
float64.  That is the mixed-precision bf16 model (bf16 operands, wide accumulation);
a float32 model has no rounding.

Each function works on one batch row (arrays [L, ...]); rows are independent.
"""
import numpy as np
from scipy.special import erf


# --------------------------------------------------------------------------- ops
def round_bf16(x):
    """Round to the nearest bf16 value (8 significant bits), ties to even."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                       # x = m 2^e, |m| in [0.5, 1)
    return np.ldexp(np.round(m * 256.0) / 256.0, e)


def operand(cfg, x):
    """A matrix-product operand in the model's precision (identity for fp32 models)."""
    return round_bf16(x) if cfg.get("dtype") == "bf16" else x


def rms_norm(x, g, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def layer_norm(x, w, b, eps):
    mu = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * w + b


def gelu(x):
    """Exact (erf) GELU."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def sigmoid(x):
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-x))


def silu(x):
    return x * sigmoid(x)


def rope(x, pos, theta):
    """Rotate-half rotary embedding. x [L, nh, dh], pos [L] absolute positions."""
    dh = x.shape[-1]
    half = dh // 2
    inv_freq = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / dh)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    cos, sin = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def attention(q, k, v, op=lambda x: x):
    """Softmax attention where every query sees every key.

    q [Lq, H, dh]; k, v [Lk, Hkv, dh]; query head h reads KV head floor(h*Hkv/H).
    ``op`` maps a matrix-product operand to the model precision.
    """
    H, Hkv, dh = q.shape[1], k.shape[1], q.shape[2]
    q, k, v = op(q), op(k), op(v)
    out = np.empty((q.shape[0], H, v.shape[2]))
    for h in range(H):
        kh = (h * Hkv) // H
        s = q[:, h, :] @ k[:, kh, :].T / np.sqrt(dh)
        s = s - s.max(axis=-1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=-1, keepdims=True)
        out[:, h, :] = op(p) @ v[:, kh, :]
    return out


# ------------------------------------------------------------------ weights view
class Weights:
    """float64 view of the seeded weights, indexed by tensor name."""

    def __init__(self, cfg, names, tensors):
        self.cfg = cfg
        self.t = {}
        for n, t in zip(names, tensors):
            a = t.float().cpu().numpy() if hasattr(t, "float") else np.asarray(t)
            self.t[n] = a.astype(np.float64)

    def __getitem__(self, k):
        return self.t[k]


# ------------------------------------------------------------- transformer layer
def attention_sublayer(W, li, x, pos, ctx_kv=None):
    """The attention half of one pre-norm layer on one row: x + O Attn(RoPE(Q, K), V) of
    the RMS-normed x.  x [L, d]; ctx_kv = (k, v) of earlier context.

    Returns (x_mid, (k, v)) where k already carries its rotary embedding.
    """
    cfg = W.cfg
    H, Hkv, dh = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    eps, theta = cfg["rms_eps"], cfg["rope_theta"]
    p = f"layer{li}."
    L = x.shape[0]
    op = lambda t: operand(cfg, t)  # noqa: E731
    xn = op(rms_norm(x, W[p + "attn_norm"], eps))
    q = (xn @ W[p + "wq"].T).reshape(L, H, dh)
    k = (xn @ W[p + "wk"].T).reshape(L, Hkv, dh)
    v = (xn @ W[p + "wv"].T).reshape(L, Hkv, dh)
    q, k = rope(q, pos, theta), rope(k, pos, theta)
    if ctx_kv is not None:
        k_all = np.concatenate([ctx_kv[0], k], axis=0)
        v_all = np.concatenate([ctx_kv[1], v], axis=0)
    else:
        k_all, v_all = k, v
    o = op(attention(q, k_all, v_all, op).reshape(L, H * dh))
    return x + o @ W[p + "wo"].T, (k, v)


def ffn_sublayer(W, li, x):
    """The feed-forward half of one pre-norm layer on one row: x + FFN of the RMS-normed x
    (GeLU, SwiGLU or GeGLU)."""
    cfg = W.cfg
    p = f"layer{li}."
    op = lambda t: operand(cfg, t)  # noqa: E731
    xn = op(rms_norm(x, W[p + "ffn_norm"], cfg["rms_eps"]))
    kind = cfg["ffn_kind"]
    if kind == "gelu":
        f = gelu(xn @ W[p + "w_up"].T)
    elif kind == "swiglu":
        f = silu(xn @ W[p + "w_gate"].T) * (xn @ W[p + "w_up"].T)
    elif kind == "geglu":
        f = gelu(xn @ W[p + "w_gate"].T) * (xn @ W[p + "w_up"].T)
    else:
        raise ValueError(kind)
    return x + op(f) @ W[p + "w_down"].T


def transformer_layer(W, li, x, pos, ctx_kv=None):
    """One pre-norm layer on one row (App. C.2: DiT block, no time conditioning): the
    attention half, then the feed-forward half.  x [L, d]; ctx_kv = (k, v) of earlier
    context.

    Returns (x_out, (k, v)) where k already carries its rotary embedding.
    """
    x, kv = attention_sublayer(W, li, x, pos, ctx_kv)
    return ffn_sublayer(W, li, x), kv


def layer_ids(cfg, part):
    Ls, La, Ld = cfg["n_shared"], cfg["n_anchor"], cfg["n_denoise"]
    return {"shared": range(0, Ls), "anchor": range(Ls, Ls + La),
            "denoise": range(Ls + La, Ls + La + Ld)}[part]


def run_layers(W, part, x, pos, ctx=None, kv_out=None):
    """Apply the layers of one part (shared/anchor/denoise); ctx maps layer -> (k, v)."""
    for li in layer_ids(W.cfg, part):
        x, kv = transformer_layer(W, li, x, pos, None if ctx is None else ctx.get(li))
        if kv_out is not None:
            kv_out[li] = kv
    return x


# ------------------------------------------------------------------- S, A, D, head
def shared(W, z, pos, ctx=None, kv_out=None, sc=None):
    """c = S(z): embedding lookup (the embedding has a row for the mask id).  sc, the
    self-conditioning signal of Algorithm 2 ([len(z), d] or None), is added to the
    embeddings."""
    c = W["embed"][np.asarray(z)]
    if sc is not None:
        c = c + np.asarray(sc, dtype=np.float64)
    return run_layers(W, "shared", c, pos, ctx, kv_out)


def anchor(W, c, pos, ctx=None, kv_out=None):
    """h = A(c); the anchor output is the raw residual stream (no final norm)."""
    return run_layers(W, "anchor", c, pos, ctx, kv_out)


def denoiser(W, ht, pos, ctx=None, kv_out=None):
    """Denoiser layers followed by the final RMSNorm."""
    x = run_layers(W, "denoise", ht, pos, ctx, kv_out)
    return rms_norm(x, W["final_norm"], W.cfg["rms_eps"])


def head(W, xf):
    """Vocabulary projection: one logit per real token (mask id excluded)."""
    return operand(W.cfg, xf) @ W["w_out"].T


# ----------------------------------------------------------------------- fusion
def fusion_gated_mlp(W, c, h):
    """Gated residual MLP fusion of App. C.2.

    s = LN(c), a = LN(h'), u = [s; a];  g = sigmoid(W_g u + b_g);
    Delta = W_2 GELU(W_1 u + b_1) + b_2;  h~ = LN(h' + g * Delta).
    """
    eps = W.cfg["ln_eps"]
    s = layer_norm(c, W["fusion.ln_s_w"], W["fusion.ln_s_b"], eps)
    a = layer_norm(h, W["fusion.ln_a_w"], W["fusion.ln_a_b"], eps)
    u = operand(W.cfg, np.concatenate([s, a], axis=-1))
    g = sigmoid(u @ W["fusion.wg"].T + W["fusion.bg"])
    hid = operand(W.cfg, gelu(u @ W["fusion.w1"].T + W["fusion.b1"]))
    delta = hid @ W["fusion.w2"].T + W["fusion.b2"]
    return layer_norm(h + g * delta, W["fusion.ln_o_w"], W["fusion.ln_o_b"], eps)


def paired_mixer(W, Z, U):
    """Shared mixer phi(Z, U) of the paired-attention fusion (App. C.1).

    J = [Z, U] (feature concatenation); Q, K, V = J W_Q, J W_K, J W_V;
    R = Z + MHA(Q, K, V) W_O (bidirectional over the positions of the call);
    phi = R + SiLU(R W_1) W_2.
    """
    nh = W.cfg["paired_heads"]
    op = lambda t: operand(W.cfg, t)  # noqa: E731
    r = Z.shape[1]
    J = op(np.concatenate([Z, U], axis=-1))
    L = J.shape[0]
    q = (J @ W["fusion.w_q"].T).reshape(L, nh, r // nh)
    k = (J @ W["fusion.w_k"].T).reshape(L, nh, r // nh)
    v = (J @ W["fusion.w_v"].T).reshape(L, nh, r // nh)
    R = Z + op(attention(q, k, v, op).reshape(L, r)) @ W["fusion.w_o"].T
    return R + op(silu(op(R) @ W["fusion.w_f1"].T)) @ W["fusion.w_f2"].T


def fusion_paired(W, C, C0, H0):
    """Paired-attention fusion (App. C.1).

    s_C, s_H: token-wise RMS of the cached C0, H0 (eps 1e-6);
    Z = (C/s_C) W_C, Z0 = (C0/s_C) W_C, U = (H0/s_H) W_H;
    M = phi(Z, U) - phi(Z0, U);  F = [U; Z0; Z - Z0; M];
    g = sigmoid(SiLU(F W_g1) W_g2 + b_g) (one scalar per token);
    H~ = H0 + g * s_H * (M W_up).
    """
    eps = W.cfg["rms_eps"]
    op = lambda t: operand(W.cfg, t)  # noqa: E731
    sC = np.sqrt(np.mean(C0 * C0, axis=-1, keepdims=True) + eps)
    sH = np.sqrt(np.mean(H0 * H0, axis=-1, keepdims=True) + eps)
    Z = op(C / sC) @ W["fusion.w_c"].T
    Z0 = op(C0 / sC) @ W["fusion.w_c"].T
    U = op(H0 / sH) @ W["fusion.w_h"].T
    M = paired_mixer(W, Z, U) - paired_mixer(W, Z0, U)
    F = op(np.concatenate([U, Z0, Z - Z0, M], axis=-1))
    g = sigmoid(op(silu(F @ W["fusion.w_g1"].T)) @ W["fusion.w_g2"].T + W["fusion.b_g"])
    return H0 + g * sH * (op(M) @ W["fusion.w_up"].T)


def fuse(W, c, cache):
    """h~ = Phi(c, cached anchor); the cache holds h' (and c' for paired attention)."""
    if W.cfg["fusion_kind"] == "gated_mlp":
        return fusion_gated_mlp(W, c, cache["h"])
    return fusion_paired(W, c, cache["c"], cache["h"])


# ---------------------------------------------------------------- whole passes
class Network:
    """Row-wise TADM network over a window of positions with an optional context.

    ``ctx`` is a dict layer -> (k, v) for the context preceding the window (block
    mode), or None.
    """

    def __init__(self, W):
        self.W = W
        self.cfg = W.cfg

    def shared(self, z, pos, ctx=None, sc=None):
        return shared(self.W, z, pos, ctx, sc=sc)

    def anchor_cache(self, c, pos, ctx=None):
        """Anchor refresh: the cache stores h' = A(c') and c' itself."""
        return {"h": anchor(self.W, c, pos, ctx), "c": c.copy()}

    def fuse(self, c, cache):
        return fuse(self.W, c, cache)

    def denoise(self, ht, pos, ctx=None):
        return denoiser(self.W, ht, pos, ctx)

    def head(self, xf):
        return head(self.W, xf)

    def fresh_kv(self, z, pos, ctx=None):
        """Fresh pass (a refresh step) over clean tokens, keeping every layer's K, V."""
        kv = {}
        c = shared(self.W, z, pos, ctx, kv)
        h = anchor(self.W, c, pos, ctx, kv)
        ht = fuse(self.W, c, {"h": h, "c": c})
        denoiser(self.W, ht, pos, ctx, kv)
        return kv
