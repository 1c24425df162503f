"""Pins of the oracle's two fusion modules (App. C.2 gated MLP, App. C.1 paired attention).

Each test fixes weights so that the module reduces to a closed form stated by the
paper (zero-initialised output projection, C = C0) or to library routines.
"""
import numpy as np
import torch
import torch.nn.functional as F

import synth
from oracle import network as N

rng = np.random.default_rng(1)


def _weights(name, **over):
    cfg = synth.get_config(name, **over)
    specs = synth.weight_specs(cfg)
    W = N.Weights(cfg, [s[0] for s in specs], synth.make_weights(cfg, perturb=True))
    return cfg, W


def T(a):
    return torch.from_numpy(np.ascontiguousarray(a))


def _ln(W, x, key):
    return F.layer_norm(T(x), (x.shape[-1],), T(W[f"fusion.{key}_w"]), T(W[f"fusion.{key}_b"]),
                        eps=W.cfg["ln_eps"])


def test_gated_zero_init_update_is_output_ln_of_anchor():
    """W2 = 0, b2 = 0 (the paper's initialisation): h~ = LN(h')."""
    cfg, W = _weights("tiny")
    d = cfg["d_model"]
    W.t["fusion.w2"][:] = 0.0
    W.t["fusion.b2"][:] = 0.0
    c, h = rng.normal(size=(9, d)), rng.normal(size=(9, d)) * 2
    np.testing.assert_allclose(N.fusion_gated_mlp(W, c, h), _ln(W, h, "ln_o").numpy(),
                               rtol=1e-12, atol=1e-12)


def test_gated_closed_gate_is_output_ln_of_anchor():
    cfg, W = _weights("tiny")
    d = cfg["d_model"]
    W.t["fusion.wg"][:] = 0.0
    W.t["fusion.bg"][:] = -1e4
    c, h = rng.normal(size=(9, d)), rng.normal(size=(9, d))
    np.testing.assert_allclose(N.fusion_gated_mlp(W, c, h), _ln(W, h, "ln_o").numpy(),
                               rtol=1e-12, atol=1e-12)


def _selector(rows, cols, pairs):
    m = np.zeros((rows, cols))
    for r, c in pairs:
        m[r, c] = 1.0
    return m


def test_gated_open_gate_wiring():
    """g = 1, W1 picks one half of u = [s; a], W2 picks the first d hidden units.

    Then h~ = LN_o(h + GELU(LN_s(c))) (first half) or LN_o(h + GELU(LN_a(h))) (second).
    """
    cfg, W = _weights("tiny")
    d = cfg["d_model"]
    c, h = rng.normal(size=(9, d)), rng.normal(size=(9, d))
    W.t["fusion.wg"][:] = 0.0
    W.t["fusion.bg"][:] = 1e4
    W.t["fusion.b1"][:] = 0.0
    W.t["fusion.b2"][:] = 0.0
    W.t["fusion.w2"][:] = _selector(d, 4 * d, [(i, i) for i in range(d)])
    for half, key, src in ((0, "ln_s", c), (1, "ln_a", h)):
        W.t["fusion.w1"][:] = _selector(4 * d, 2 * d, [(i, half * d + i) for i in range(d)])
        ref = _ln(W, T(h) + F.gelu(_ln(W, src, key)), "ln_o")
        np.testing.assert_allclose(N.fusion_gated_mlp(W, c, h), ref.numpy(), rtol=1e-12, atol=1e-12)


def test_gated_gate_multiplies_update():
    """W1 = 0, b1 = 0 => Delta = b2; W_g picks s => h~ = LN_o(h + sigmoid(s + b_g) * b2)."""
    cfg, W = _weights("tiny")
    d = cfg["d_model"]
    c, h = rng.normal(size=(9, d)), rng.normal(size=(9, d))
    W.t["fusion.w1"][:] = 0.0
    W.t["fusion.b1"][:] = 0.0
    W.t["fusion.wg"][:] = _selector(d, 2 * d, [(i, i) for i in range(d)])
    s = _ln(W, c, "ln_s")
    ref = _ln(W, T(h) + torch.sigmoid(s + T(W["fusion.bg"])) * T(W["fusion.b2"]), "ln_o")
    np.testing.assert_allclose(N.fusion_gated_mlp(W, c, h), ref.numpy(), rtol=1e-12, atol=1e-12)


def _paired():
    return _weights("tiny", fusion_kind="paired", fusion_rank=32, paired_heads=4)


def test_paired_fresh_anchor_is_identity_bitwise():
    """C = C0 => Z = Z0 => M = 0 => H~ = H0 exactly (App. C.1)."""
    cfg, W = _paired()
    d = cfg["d_model"]
    C0, H0 = rng.normal(size=(10, d)), rng.normal(size=(10, d)) * 3
    out = N.fusion_paired(W, C0.copy(), C0, H0)
    assert np.array_equal(out, H0)


def test_paired_zero_up_projection_is_identity():
    cfg, W = _paired()
    d = cfg["d_model"]
    W.t["fusion.w_up"][:] = 0.0
    C, C0, H0 = rng.normal(size=(10, d)), rng.normal(size=(10, d)), rng.normal(size=(10, d))
    assert np.array_equal(N.fusion_paired(W, C, C0, H0), H0)


def test_paired_matches_library_formulation():
    """W_g1 = 0 => g = sigmoid(b_g); W_f1 = 0 => phi = R.  Rebuilt with torch rms_norm/SDPA."""
    cfg, W = _paired()
    d, r, nh = cfg["d_model"], cfg["fusion_rank"], cfg["paired_heads"]
    W.t["fusion.w_g1"][:] = 0.0
    W.t["fusion.w_f1"][:] = 0.0
    L = 10
    C, C0, H0 = (T(rng.normal(size=(L, d))) for _ in range(3))
    Wt = {k: T(v) for k, v in W.t.items()}
    eps = cfg["rms_eps"]
    sH = torch.sqrt((H0 * H0).mean(-1, keepdim=True) + eps)
    # C/s_C uses the cached-state scale: rms_norm(C0) = C0/s_C, so 1/s_C = <rms_norm(C0), C0>/<C0, C0>
    c0n = F.rms_norm(C0, (d,), eps=eps)
    scale_c = ((c0n * C0).sum(-1, keepdim=True) / (C0 * C0).sum(-1, keepdim=True))
    Z = F.linear(C * scale_c, Wt["fusion.w_c"])
    Z0 = F.linear(c0n, Wt["fusion.w_c"])
    U = F.linear(F.rms_norm(H0, (d,), eps=eps), Wt["fusion.w_h"])

    def phi(Zx):
        J = torch.cat([Zx, U], -1)
        q, k, v = (F.linear(J, Wt[f"fusion.w_{n}"]).view(L, nh, r // nh).transpose(0, 1)
                   for n in "qkv")
        a = F.scaled_dot_product_attention(q, k, v).transpose(0, 1).reshape(L, r)
        return Zx + F.linear(a, Wt["fusion.w_o"])

    M = phi(Z) - phi(Z0)
    g = torch.sigmoid(Wt["fusion.b_g"])
    ref = H0 + g * sH * F.linear(M, Wt["fusion.w_up"])
    out = N.fusion_paired(W, C.numpy(), C0.numpy(), H0.numpy())
    np.testing.assert_allclose(out, ref.numpy(), rtol=1e-9, atol=1e-11)
