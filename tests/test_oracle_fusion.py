"""Pins of the oracle's two fusion modules (App. C.2 gated MLP, App. C.1 paired attention).

Each test fixes weights so that the module reduces to a closed form stated by the
paper (zero-initialised output projection, C = C0) or to library routines.
"""
import math

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


# ---------------------------------------------------------------------------
# Pins with every fusion weight and bias non-zero.  The reference formulations below
# are written with torch's library ops (F.linear with its bias, F.gelu, F.silu,
# F.layer_norm, F.rms_norm, scaled_dot_product_attention, torch.cat in the order the
# appendix prints), so a swapped concatenation, a wrong activation or a dropped bias
# in the oracle makes them disagree.

def _paired_all_random():
    """Seeded weights with the gate MLP and the mixer FFN scaled up (std 0.02 -> 0.5), so
    that at this small width both change the result by far more than the tolerance."""
    cfg, W = _paired()
    for k in ("fusion.w_g1", "fusion.w_g2", "fusion.w_f1", "fusion.w_f2"):
        W.t[k] *= 25.0
        assert np.count_nonzero(W[k]) == W[k].size
    assert W["fusion.b_g"][0] != -3.0  # perturbed away from the paper's -3
    return cfg, W


def _paired_reference(W, C, C0, H0):
    """App. C.1 written with library ops: s_C, s_H token-wise RMS of the cached C0, H0;
    Z = (C/s_C) W_C, Z0 = (C0/s_C) W_C, U = (H0/s_H) W_H; J = [Z, U];
    R = Z + MHA(J W_Q, J W_K, J W_V) W_O; phi = R + SiLU(R W_1) W_2;
    M = phi(Z, U) - phi(Z0, U); F = [U; Z0; Z - Z0; M];
    g = sigmoid(SiLU(F W_g1) W_g2 + b_g); H~ = H0 + g s_H (M W_up)."""
    cfg = W.cfg
    d, r, nh, eps = cfg["d_model"], cfg["fusion_rank"], cfg["paired_heads"], cfg["rms_eps"]
    Wt = {k: T(v) for k, v in W.t.items()}
    C, C0, H0 = T(C), T(C0), T(H0)
    L = C.shape[0]
    sC = torch.sqrt(torch.mean(C0 ** 2, -1, keepdim=True) + eps)
    sH = torch.sqrt(torch.mean(H0 ** 2, -1, keepdim=True) + eps)
    Z = F.linear(C / sC, Wt["fusion.w_c"])
    Z0 = F.linear(F.rms_norm(C0, (d,), eps=eps), Wt["fusion.w_c"])
    U = F.linear(F.rms_norm(H0, (d,), eps=eps), Wt["fusion.w_h"])

    def phi(Zx):
        J = torch.cat([Zx, U], dim=-1)
        q, k, v = (F.linear(J, Wt[f"fusion.w_{n}"]).view(L, nh, r // nh).transpose(0, 1) for n in "qkv")
        att = F.scaled_dot_product_attention(q, k, v).transpose(0, 1).reshape(L, r)
        R = Zx + F.linear(att, Wt["fusion.w_o"])
        return R + F.linear(F.silu(F.linear(R, Wt["fusion.w_f1"])), Wt["fusion.w_f2"])

    M = phi(Z) - phi(Z0)
    Fcat = torch.cat([U, Z0, Z - Z0, M], dim=-1)
    g = torch.sigmoid(F.linear(F.silu(F.linear(Fcat, Wt["fusion.w_g1"])), Wt["fusion.w_g2"], Wt["fusion.b_g"]))
    return (H0 + g * sH * F.linear(M, Wt["fusion.w_up"])).numpy(), g.numpy(), M, (U, Z0, Z - Z0)


def test_paired_all_weights_nonzero_matches_library_formulation():
    cfg, W = _paired_all_random()
    d = cfg["d_model"]
    C, C0, H0 = rng.normal(size=(12, d)), rng.normal(size=(12, d)), rng.normal(size=(12, d)) * 2
    ref, g, _, _ = _paired_reference(W, C, C0, H0)
    # the gate is a genuine function of the token here, not a constant
    assert g.std() > 1e-3
    np.testing.assert_allclose(N.fusion_paired(W, C, C0, H0), ref, rtol=1e-9, atol=1e-11)


def test_paired_zero_gate_output_layer_gives_bias_gate():
    """W_g2 = 0 => g = sigmoid(b_g) for every token, whatever W_g1 and F are."""
    cfg, W = _paired_all_random()
    d = cfg["d_model"]
    W.t["fusion.w_g2"][:] = 0.0
    C, C0, H0 = rng.normal(size=(12, d)), rng.normal(size=(12, d)), rng.normal(size=(12, d))
    _, _, M, _ = _paired_reference(W, C, C0, H0)
    sH = np.sqrt(np.mean(H0 ** 2, -1, keepdims=True) + cfg["rms_eps"])
    g = 1.0 / (1.0 + np.exp(-W["fusion.b_g"][0]))
    ref = H0 + g * sH * (M.numpy() @ W["fusion.w_up"].T)
    np.testing.assert_allclose(N.fusion_paired(W, C, C0, H0), ref, rtol=1e-9, atol=1e-11)


def test_paired_zero_mixer_output_gives_residual_branch():
    """W_f2 = 0 => phi(Z, U) = R = Z + MHA(.) W_O: the result equals the formulation
    whose mixer stops at R, with W_f1 left non-zero."""
    cfg, W = _paired_all_random()
    d = cfg["d_model"]
    W.t["fusion.w_f2"][:] = 0.0
    C, C0, H0 = rng.normal(size=(12, d)), rng.normal(size=(12, d)), rng.normal(size=(12, d))
    ref, _, _, _ = _paired_reference(W, C, C0, H0)
    W2 = N.Weights(cfg, [], [])
    W2.t = {k: v.copy() for k, v in W.t.items()}
    W2.t["fusion.w_f1"][:] = 0.0  # with W_f2 = 0, W_f1 must not matter
    np.testing.assert_allclose(N.fusion_paired(W, C, C0, H0), N.fusion_paired(W2, C, C0, H0), rtol=0, atol=1e-13)
    np.testing.assert_allclose(N.fusion_paired(W, C, C0, H0), ref, rtol=1e-9, atol=1e-11)


def test_paired_gate_reads_the_four_blocks_in_order():
    """W_g1 selects one r-wide block of F = [U; Z0; Z - Z0; M] (identity on that block,
    zero elsewhere) and W_g2 = 1/r: then g = sigmoid(mean(SiLU(block)) + b_g), with the
    block computed from its own definition.  Each block gives a different gate, so an
    oracle that concatenates in another order fails."""
    cfg, W = _paired_all_random()
    d, r, eps = cfg["d_model"], cfg["fusion_rank"], cfg["rms_eps"]
    C, C0, H0 = rng.normal(size=(12, d)), rng.normal(size=(12, d)), rng.normal(size=(12, d))
    _, _, M, (U, Z0, dZ) = _paired_reference(W, C, C0, H0)
    blocks = [U.numpy(), Z0.numpy(), dZ.numpy(), M.numpy()]
    sH = np.sqrt(np.mean(H0 ** 2, -1, keepdims=True) + eps)
    MWup = M.numpy() @ W["fusion.w_up"].T
    gates = []
    for j, blk in enumerate(blocks):
        W.t["fusion.w_g1"][:] = 0.0
        W.t["fusion.w_g1"][:, j * r:(j + 1) * r] = np.eye(r)
        W.t["fusion.w_g2"][:] = 1.0 / r
        silu = blk / (1.0 + np.exp(-blk))
        g = 1.0 / (1.0 + np.exp(-(silu.mean(-1, keepdims=True) + W["fusion.b_g"][0])))
        gates.append(g)
        np.testing.assert_allclose(N.fusion_paired(W, C, C0, H0), H0 + g * sH * MWup, rtol=1e-9, atol=1e-11)
    for a in range(4):
        for b in range(a + 1, 4):
            assert np.abs(gates[a] - gates[b]).max() > 1e-4


def test_gated_all_weights_nonzero_matches_library_formulation():
    """App. C.2 with every weight and bias non-zero (b1, b2, b_g, LN gains and biases
    perturbed), against F.layer_norm / F.linear with bias / F.gelu / torch.sigmoid."""
    cfg, W = _weights("tiny")
    d = cfg["d_model"]
    assert np.abs(W["fusion.b1"]).max() > 0.05 and np.abs(W["fusion.b2"]).max() > 0.05
    Wt = {k: T(v) for k, v in W.t.items()}
    c, h = rng.normal(size=(9, d)), rng.normal(size=(9, d)) * 2
    u = torch.cat([_ln(W, c, "ln_s"), _ln(W, h, "ln_a")], dim=-1)
    g = torch.sigmoid(F.linear(u, Wt["fusion.wg"], Wt["fusion.bg"]))
    delta = F.linear(F.gelu(F.linear(u, Wt["fusion.w1"], Wt["fusion.b1"])), Wt["fusion.w2"], Wt["fusion.b2"])
    ref = _ln(W, T(h) + g * delta, "ln_o")
    np.testing.assert_allclose(N.fusion_gated_mlp(W, c, h), ref.numpy(), rtol=1e-11, atol=1e-12)


def test_gated_hidden_bias_enters_before_the_gelu():
    """W1 = 0, open gate: the hidden state is GELU(b1) for every token, so
    h~ = LN_o(h + W2 GELU(b1) + b2).  A dropped b1 (GELU(0) = 0) or a b1 added after
    the GELU gives a different value."""
    cfg, W = _weights("tiny")
    d = cfg["d_model"]
    W.t["fusion.w1"][:] = 0.0
    W.t["fusion.wg"][:] = 0.0
    W.t["fusion.bg"][:] = 1e4
    c, h = rng.normal(size=(9, d)), rng.normal(size=(9, d))
    b1 = W["fusion.b1"]
    hid = 0.5 * b1 * (1.0 + np.vectorize(math.erf)(b1 / math.sqrt(2.0)))
    delta = W["fusion.w2"] @ hid + W["fusion.b2"]
    ref = _ln(W, T(h + delta[None, :]), "ln_o").numpy()
    np.testing.assert_allclose(N.fusion_gated_mlp(W, c, h), ref, rtol=1e-11, atol=1e-12)
    wrong = _ln(W, T(h + (W["fusion.w2"] @ (hid * 0) + W["fusion.b2"])[None, :]), "ln_o").numpy()
    assert np.abs(wrong - ref).max() > 1e-3
