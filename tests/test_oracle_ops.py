"""Pins of the oracle's network ops against library routines and closed forms."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import network as N

rng = np.random.default_rng(0)


def t64(a):
    return torch.from_numpy(np.ascontiguousarray(a))


def test_rms_norm_matches_torch():
    x, g = rng.normal(size=(7, 48)), rng.normal(size=48)
    ref = F.rms_norm(t64(x), (48,), t64(g), eps=1e-6).numpy()
    np.testing.assert_allclose(N.rms_norm(x, g, 1e-6), ref, rtol=1e-12, atol=1e-12)


def test_layer_norm_matches_torch():
    x, w, b = rng.normal(size=(5, 40)) * 3 + 1, rng.normal(size=40), rng.normal(size=40)
    ref = F.layer_norm(t64(x), (40,), t64(w), t64(b), eps=1e-5).numpy()
    np.testing.assert_allclose(N.layer_norm(x, w, b, 1e-5), ref, rtol=1e-12, atol=1e-12)


def test_activations_match_torch():
    x = rng.normal(size=1000) * 4
    np.testing.assert_allclose(N.gelu(x), F.gelu(t64(x)).numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(N.silu(x), F.silu(t64(x)).numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(N.sigmoid(x), torch.sigmoid(t64(x)).numpy(), rtol=1e-12)


def test_rope_is_complex_rotation():
    """Pair (x_j, x_{j+dh/2}) rotates by angle pos * theta^(-2j/dh) (rotate-half RoPE)."""
    L, nh, dh, theta = 6, 3, 16, 10000.0
    x = rng.normal(size=(L, nh, dh))
    pos = np.array([0, 1, 5, 17, 100, 1023])
    z = x[..., : dh // 2] + 1j * x[..., dh // 2:]
    freq = theta ** (-2.0 * np.arange(dh // 2) / dh)
    zr = z * np.exp(1j * pos[:, None, None] * freq[None, None, :])
    ref = np.concatenate([zr.real, zr.imag], axis=-1)
    np.testing.assert_allclose(N.rope(x, pos, theta), ref, rtol=1e-12, atol=1e-12)
    # position 0 is the identity; scores depend only on relative position
    np.testing.assert_array_equal(N.rope(x[:1], [0], theta), x[:1])
    q, k = rng.normal(size=(1, 1, dh)), rng.normal(size=(1, 1, dh))
    s1 = np.sum(N.rope(q, [3], theta) * N.rope(k, [10], theta))
    s2 = np.sum(N.rope(q, [103], theta) * N.rope(k, [110], theta))
    assert abs(s1 - s2) < 1e-10


@pytest.mark.parametrize("H,Hkv", [(4, 4), (8, 2), (6, 3)])
def test_attention_matches_sdpa(H, Hkv):
    Lq, Lk, dh = 9, 13, 16
    q, k, v = rng.normal(size=(Lq, H, dh)), rng.normal(size=(Lk, Hkv, dh)), rng.normal(size=(Lk, Hkv, dh))
    rep = H // Hkv
    kt = t64(k).permute(1, 0, 2).repeat_interleave(rep, 0)
    vt = t64(v).permute(1, 0, 2).repeat_interleave(rep, 0)
    ref = F.scaled_dot_product_attention(t64(q).permute(1, 0, 2), kt, vt).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(N.attention(q, k, v), ref, rtol=1e-10, atol=1e-12)


def _torch_layer(cfg, Wt, li, x, pos, ctx=None):
    """Independent formulation of one layer from torch library ops (complex RoPE, SDPA)."""
    H, Hkv, dh = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    p = f"layer{li}."
    L = x.shape[0]
    xn = F.rms_norm(x, (x.shape[1],), Wt[p + "attn_norm"], eps=cfg["rms_eps"])

    def rot(t):
        tc = torch.complex(t[..., : dh // 2], t[..., dh // 2:])
        freq = cfg["rope_theta"] ** (-2.0 * torch.arange(dh // 2, dtype=torch.float64) / dh)
        tc = tc * torch.polar(torch.ones(L, 1, dh // 2, dtype=torch.float64),
                              torch.tensor(pos, dtype=torch.float64)[:, None, None] * freq)
        return torch.cat([tc.real, tc.imag], -1)

    q = rot(F.linear(xn, Wt[p + "wq"]).view(L, H, dh))
    k = rot(F.linear(xn, Wt[p + "wk"]).view(L, Hkv, dh))
    v = F.linear(xn, Wt[p + "wv"]).view(L, Hkv, dh)
    if ctx is not None:
        k, v = torch.cat([ctx[0], k]), torch.cat([ctx[1], v])
    o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                       enable_gqa=True).transpose(0, 1).reshape(L, H * dh)
    x = x + F.linear(o, Wt[p + "wo"])
    xn = F.rms_norm(x, (x.shape[1],), Wt[p + "ffn_norm"], eps=cfg["rms_eps"])
    if cfg["ffn_kind"] == "gelu":
        f = F.gelu(F.linear(xn, Wt[p + "w_up"]))
    elif cfg["ffn_kind"] == "swiglu":
        f = F.silu(F.linear(xn, Wt[p + "w_gate"])) * F.linear(xn, Wt[p + "w_up"])
    else:
        f = F.gelu(F.linear(xn, Wt[p + "w_gate"])) * F.linear(xn, Wt[p + "w_up"])
    return x + F.linear(f, Wt[p + "w_down"])


@pytest.mark.parametrize("ffn", ["gelu", "swiglu", "geglu"])
@pytest.mark.parametrize("kv", [4, 2])
def test_transformer_layer_matches_torch_formulation(ffn, kv):
    cfg = synth.get_config("tiny", ffn_kind=ffn, n_kv_heads=kv)
    specs = synth.weight_specs(cfg)
    ws = synth.make_weights(cfg, perturb=True)
    W = N.Weights(cfg, [s[0] for s in specs], ws)
    Wt = {s[0]: torch.from_numpy(W[s[0]]) for s in specs}
    L = 11
    x = rng.normal(size=(L, cfg["d_model"]))
    pos = list(range(5, 5 + L))
    out, (k, v) = N.transformer_layer(W, 1, x, np.array(pos))
    ref = _torch_layer(cfg, Wt, 1, t64(x), pos).numpy()
    np.testing.assert_allclose(out, ref, rtol=1e-9, atol=1e-11)
    # with a context prefix (block mode): context K/V enter the softmax
    ctx = (rng.normal(size=(7, kv, 16)), rng.normal(size=(7, kv, 16)))
    out, _ = N.transformer_layer(W, 1, x, np.array(pos), ctx)
    ref = _torch_layer(cfg, Wt, 1, t64(x), pos, (t64(ctx[0]), t64(ctx[1]))).numpy()
    np.testing.assert_allclose(out, ref, rtol=1e-9, atol=1e-11)


def test_round_bf16_is_round_to_nearest_even():
    x = (rng.normal(size=20000) * 10.0 ** rng.integers(-3, 4, size=20000)).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(N.round_bf16(x.astype(np.float64)), ref)
    # exact ties go to the even neighbour: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7
    assert N.round_bf16(1.0 + 2.0 ** -8) == 1.0
    assert N.round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6


def test_bf16_model_rounds_only_product_operands():
    """A bf16 layer equals the float64 layer up to bf16 operand rounding, and with
    operands that are already bf16 values the rounding is a no-op."""
    cfg32 = synth.get_config("tiny", dtype="f32")
    cfg16 = synth.get_config("tiny", dtype="bf16")
    specs = synth.weight_specs(cfg16)
    ws = synth.make_weights(cfg16, perturb=True)
    W16 = N.Weights(cfg16, [s[0] for s in specs], ws)
    W32 = N.Weights(cfg32, [s[0] for s in specs], ws)
    x = rng.normal(size=(12, 64))
    a, _ = N.transformer_layer(W16, 0, x, np.arange(12))
    b, _ = N.transformer_layer(W32, 0, x, np.arange(12))
    assert 0 < np.abs(a - b).max() < 2e-2
    v = N.round_bf16(rng.normal(size=100))
    assert np.array_equal(N.operand(cfg16, v), v) and np.array_equal(N.operand(cfg32, x), x)
