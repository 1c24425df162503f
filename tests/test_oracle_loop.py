"""Pins of the oracle's Algorithm 1 loop: schedule, refresh rule, call counts, cache,
carry-over, K=1 reduction and the block-diffusion context decomposition."""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import loop, network as N, sampler as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _net(name, **over):
    cfg = synth.get_config(name, **over)
    specs = synth.weight_specs(cfg)
    W = N.Weights(cfg, [s[0] for s in specs], synth.make_weights(cfg, perturb=True))
    return N.Network(W)


# ----------------------------------------------------------------- schedule
@pytest.mark.parametrize("M0,T", [(24, 16), (256, 64), (64, 32), (1024, 128), (7, 16), (1, 5),
                                  (256, 48), (1000, 1000)])
def test_unmask_schedule(M0, T):
    n = [loop.unmask_count(M0, i, T) for i in range(T, 0, -1)]
    assert sum(n) == M0
    remaining = M0
    for i, ni in zip(range(T, 0, -1), n):
        remaining -= ni
        assert remaining == (M0 * (i - 1)) // T     # floor(M0 * s(i)) stay masked
    assert remaining == 0                           # alpha_0 = 1: nothing masked at the end


def test_unmask_schedule_small_case_alternates():
    assert [loop.unmask_count(24, i, 16) for i in range(16, 0, -1)] == [2, 1] * 8


# -------------------------------------------------------- call counting (stub)
class _StubNet:
    """Network stand-in with the loop's interface: zero work, tiny arrays."""

    def __init__(self, Ls, La, Ld):
        self.cfg = dict(n_shared=Ls, n_anchor=La, n_denoise=Ld)

    def shared(self, z, pos, ctx=None):
        return np.zeros((len(z), 1))

    def anchor_cache(self, c, pos, ctx=None):
        return {"h": c, "c": c}

    def fuse(self, c, cache):
        return c

    def denoise(self, ht, pos, ctx=None):
        return ht

    def head(self, xf):
        return np.zeros((xf.shape[0], 2))

    def fresh_kv(self, z, pos, ctx=None):
        return {}


def _first_n(logits, canvas, mask_id, n, *args):
    nxt = canvas.copy()
    idx = np.flatnonzero(canvas == mask_id)[:n]
    nxt[idx] = 0
    return nxt, None, None


def _count(T, K, Ls, La, Ld, L=4):
    cnt = loop.Counts()
    loop.generate(_StubNet(Ls, La, Ld), np.zeros((1, 0), np.int64), L, T, K, L, 0, 1.0, 9,
                  counts=cnt, sample_fn=_first_n)
    return cnt


def test_layer_calls_match_table2():
    g = json.load(open(os.path.join(GOLDEN, "layer_calls.json")))
    for row in g["table2"]:
        cnt = _count(row["T"], row["K"], row["L_shared"], row["L_anchor"], row["L_denoise"])
        assert cnt.layer_calls == row["calls"], row
        assert cnt.anchor_refreshes == -(-row["T"] // row["K"])
    for row in g["table2_mdlm_ratio"]:
        cnt = _count(row["T"], row["K"], 0, 12, 6)
        assert round(cnt.layer_calls / (row["mdlm_layers"] * row["T"]), 2) == row["ratio"]


def test_compute_ratio_matches_table1():
    g = json.load(open(os.path.join(GOLDEN, "layer_calls.json")))
    for row in g["table1"]:
        Ls, La, Ld, T = row["L_shared"], row["L_anchor"], row["L_denoise"], row["T"]
        cnt = _count(T, row["K"], Ls, La, Ld)
        assert round(cnt.layer_calls / (T * (Ls + La + Ld)), 2) == row["ratio"]


@pytest.mark.parametrize("T,K", [(16, 4), (64, 8), (10, 3), (5, 1), (7, 10)])
def test_refresh_steps(T, K):
    tr = []
    loop.generate(_StubNet(0, 2, 1), np.zeros((1, 0), np.int64), 4, T, K, 4, 0, 1.0, 9,
                  trace=tr, sample_fn=_first_n)
    got = [t["i"] for t in tr if t["refresh"]]
    assert got[0] == T                                   # the first step always refreshes
    assert got == [i for i in range(T, 0, -1) if (T - i) % K == 0]
    assert len(got) == -(-T // K)


# ------------------------------------------------------------- real network
class _Recorder(N.Network):
    def __init__(self, W):
        super().__init__(W)
        self.cache_bytes = []

    def fuse(self, c, cache):
        self.cache_bytes.append(cache["h"].tobytes())
        return super().fuse(c, cache)


def _tiny_run(K, **over):
    cfg = synth.get_config("tiny", **over)
    specs = synth.weight_specs(cfg)
    net = _Recorder(N.Weights(cfg, [s[0] for s in specs], synth.make_weights(cfg, perturb=True)))
    prompt = synth.make_prompt(cfg).numpy()
    tr = []
    out = loop.generate(net, prompt, cfg["gen_len"], cfg["T"], K, cfg["block_len"], 2, 1.0,
                        synth.mask_id(cfg), trace=tr)
    return cfg, net, prompt, out, tr


def test_cache_constant_between_refreshes_and_carry_over():
    cfg, net, prompt, out, tr = _tiny_run(4)
    mask = synth.mask_id(cfg)
    P, M0, T = cfg["prompt_len"], cfg["gen_len"], cfg["T"]
    for k, t in enumerate(tr):
        if not t["refresh"]:
            assert net.cache_bytes[k] == net.cache_bytes[k - 1]
        else:
            assert k == 0 or net.cache_bytes[k] != net.cache_bytes[k - 1]
    canv = [t["canvas"] for t in tr] + [out]
    for a, b in zip(canv, canv[1:]):
        assert np.array_equal(a[:, :P], prompt)                 # prompt untouched
        dec = a[:, P:] != mask
        assert np.array_equal(a[:, P:][dec], b[:, P:][dec])       # never re-masked or changed
    for t, nxt in zip(tr, canv[1:]):
        assert int((nxt[:, P:] == mask).sum()) == (M0 * (t["i"] - 1)) // T
    assert not np.any(out == mask) and np.all(out < cfg["vocab"])


def test_k1_paired_reduces_to_full_network_bitwise():
    """K=1 refreshes every step; with paired attention Phi is then exactly the identity,
    so generation equals the backbone D(A(S(z))) evaluated in full at every step."""
    over = dict(fusion_kind="paired", fusion_rank=32)
    cfg, net, prompt, out, tr = _tiny_run(1, **over)
    assert all(t["refresh"] for t in tr)

    class Backbone(N.Network):
        def fuse(self, c, cache):
            return cache["h"]

    specs = synth.weight_specs(cfg)
    bb = Backbone(N.Weights(cfg, [s[0] for s in specs], synth.make_weights(cfg, perturb=True)))
    out2 = loop.generate(bb, prompt, cfg["gen_len"], cfg["T"], 1, cfg["block_len"], 2, 1.0,
                         synth.mask_id(cfg))
    assert np.array_equal(out, out2)


def test_k1_gated_is_fresh_pass_every_step():
    cfg, net, prompt, out, tr = _tiny_run(1)
    W = net.W
    # replay the teacher canvases with an explicit fresh pass D(Phi(c, A(c)))
    mask = synth.mask_id(cfg)
    P = cfg["prompt_len"]
    pos = np.arange(P + cfg["gen_len"])
    for t, nxt in zip(tr, [x["canvas"] for x in tr[1:]] + [out]):
        c = N.shared(W, t["canvas"][0], pos)
        xf = N.denoiser(W, N.fusion_gated_mlp(W, c, N.anchor(W, c, pos)), pos)
        lg = N.head(W, xf[P:]).astype(np.float32)
        got, _, _ = S.reverse_step(lg, t["canvas"][0, P:], mask, t["n"], P, 0, t["step_id"], 2,
                                   np.float32(1))
        assert np.array_equal(got, nxt[0, P:])


def test_generation_deterministic():
    a = _tiny_run(4)[3]
    b = _tiny_run(4)[3]
    assert np.array_equal(a, b)


# ------------------------------------------------------------- block mode
def _torch_stack_blockcausal(W, z, block_of):
    """Full-sequence fresh pass with an explicit block-causal mask, from torch ops."""
    cfg = W.cfg
    H, Hkv, dh = cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    L = len(z)
    Wt = {k: torch.from_numpy(v) for k, v in W.t.items()}
    blk = torch.tensor(block_of)
    allowed = blk[None, :] <= blk[:, None]
    pos = torch.arange(L, dtype=torch.float64)

    def rot(t):
        tc = torch.complex(t[..., : dh // 2], t[..., dh // 2:])
        freq = cfg["rope_theta"] ** (-2.0 * torch.arange(dh // 2, dtype=torch.float64) / dh)
        tc = tc * torch.polar(torch.ones(L, 1, dh // 2, dtype=torch.float64), pos[:, None, None] * freq)
        return torch.cat([tc.real, tc.imag], -1)

    def layer(li, x):
        p = f"layer{li}."
        xn = F.rms_norm(x, (x.shape[1],), Wt[p + "attn_norm"], eps=cfg["rms_eps"])
        q = rot(F.linear(xn, Wt[p + "wq"]).view(L, H, dh)).transpose(0, 1)
        k = rot(F.linear(xn, Wt[p + "wk"]).view(L, Hkv, dh)).transpose(0, 1)
        v = F.linear(xn, Wt[p + "wv"]).view(L, Hkv, dh).transpose(0, 1)
        o = F.scaled_dot_product_attention(q, k, v, attn_mask=allowed, enable_gqa=True)
        x = x + F.linear(o.transpose(0, 1).reshape(L, H * dh), Wt[p + "wo"])
        xn = F.rms_norm(x, (x.shape[1],), Wt[p + "ffn_norm"], eps=cfg["rms_eps"])
        return x + F.linear(F.gelu(F.linear(xn, Wt[p + "w_up"])), Wt[p + "w_down"])

    c = Wt["embed"][torch.as_tensor(z)]
    h = c
    for li in N.layer_ids(cfg, "anchor"):
        h = layer(li, h)
    ht = torch.from_numpy(N.fusion_gated_mlp(W, c.numpy(), h.numpy()))
    x = ht
    for li in N.layer_ids(cfg, "denoise"):
        x = layer(li, x)
    return F.rms_norm(x, (x.shape[1],), Wt["final_norm"], eps=cfg["rms_eps"])


def test_block_context_equals_block_causal_full_pass():
    """Prefilling the context KV block by block equals one pass with a block-causal mask
    (bidirectional within a block, causal across blocks)."""
    net = _net("tiny", n_kv_heads=2)
    W = net.W
    rng = np.random.default_rng(5)
    z = rng.integers(0, 257, size=8 + 6 + 6)
    block_of = [0] * 8 + [1] * 6 + [2] * 6
    ref = _torch_stack_blockcausal(W, z, block_of).numpy()
    ctx = net.fresh_kv(z[:8], np.arange(8))
    kv1 = net.fresh_kv(z[8:14], np.arange(8, 14), ctx)
    ctx = {li: (np.concatenate([ctx[li][0], kv1[li][0]]), np.concatenate([ctx[li][1], kv1[li][1]]))
           for li in ctx}
    pos = np.arange(14, 20)
    c = net.shared(z[14:], pos, ctx)
    xf = net.denoise(net.fuse(c, net.anchor_cache(c, pos, ctx)), pos, ctx)
    np.testing.assert_allclose(xf, ref[14:], rtol=1e-9, atol=1e-10)


def test_block_mode_generation_invariants():
    cfg = synth.get_config("tiny", block_len=8)
    specs = synth.weight_specs(cfg)
    net = N.Network(N.Weights(cfg, [s[0] for s in specs], synth.make_weights(cfg)))
    prompt = synth.make_prompt(cfg).numpy()
    tr = []
    cnt = loop.Counts()
    out = loop.generate(net, prompt, cfg["gen_len"], 8, 4, 8, 2, 1.0, synth.mask_id(cfg),
                        trace=tr, counts=cnt)
    assert not np.any(out == synth.mask_id(cfg))
    assert np.array_equal(out[:, :8], prompt)
    assert [t["step_id"] for t in tr] == list(range(24))
    assert [t["i"] for t in tr if t["refresh"]] == [8, 4] * 3      # counter restarts per block
    assert cnt.anchor_refreshes == 6
