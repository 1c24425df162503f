"""GPU parity of the entropy-bound sampler (Algorithm 2) against the oracle."""
import numpy as np
import pytest
import torch

import synth
from helpers import dev, gpu_model, oracle_net, rows_close
from oracle import loop
from oracle import usdm

tadm = pytest.importorskip("paper_2609_37924_amd")
pytestmark = pytest.mark.gpu


def sync():
    torch.cuda.synchronize()


@pytest.mark.parametrize("V,B,L,off,inv_temp,eta,i,std,ties", [
    (256, 2, 40, 8, 1.25, 0.1, 5, 2.0, False),
    (1001, 2, 24, 0, 1.0, 0.5, 3, 1.0, False),        # vocabulary not a multiple of 4 or 64
    (64, 2, 32, 0, 2.5, 0.3, 2, 2.0, True),           # planted ties, duplicated rows
    (300, 3, 20, 4, 1.0, 0.2, 4, 0.0, False),         # flat rows: equal entropies, ranked by position
    (32768, 1, 12, 2, 1.6, 1.0, 7, 3.0, False),
    (50304, 1, 6, 0, 2.0, 0.05, 9, 30.0, False),      # peaked: entropies near 0
    (262144, 1, 3, 0, 1.0, 0.1, 2, 1.0, False),       # largest vocabulary
    (500, 2, 16, 0, 1.25, 0.0, 3, 1.0, False),        # eta = 0: only the most certain position(s)
    (500, 2, 16, 3, 1.25, 0.1, 1, 1.0, True),         # last step: the argmax canvas
    (128, 2, 1100, 0, 1.0, 5.0, 6, 1.0, False),       # canvas longer than one block of threads
])
def test_entropy_step_bit_exact(V, B, L, off, inv_temp, eta, i, std, ties):
    """Entropy-bound step from given logits: x_tilde, the entropy bits and the next canvas
    (acceptance, re-noise tokens, x_hat at the last step) equal the oracle's."""
    cfg = synth.get_config("tiny", vocab=V)
    m = tadm.tadm_model_create(tadm.make_config(cfg, max_batch=B, max_seq=L))
    tadm.tadm_set_stream(m, torch.cuda.current_stream().cuda_stream)
    try:
        Lc = L - off
        g = torch.Generator().manual_seed(V + 7)
        canvas = torch.randint(0, V, (B, L), generator=g, dtype=torch.int32)
        logits = synth.make_logits(B * Lc, V, seed=V + 3, std=std, ties=ties).view(B, Lc, V)
        if std == 0.0:
            logits[:, ::3] += 1.0   # two distinct entropy levels, many ties within each
        pos0, step_id, seed = 11, 29, 0xC0FFEE
        args = tadm.step_args(i, 12, 0, step_id, seed, float(np.float32(inv_temp)), entropy_eta=float(np.float32(eta)))
        d_can = canvas.to(dev())
        nxt = torch.empty_like(d_can)
        choice = torch.empty(B, Lc, dtype=torch.int32, device=dev())
        conf = torch.empty(B, Lc, dtype=torch.float32, device=dev())
        tadm.tadm_sample(m, logits.to(dev()), d_can, B, L, off, pos0, args, nxt, choice, conf)
        sync()
        got_next, got_choice, got_H = nxt.cpu().numpy(), choice.cpu().numpy(), conf.cpu().numpy()
        for b in range(B):
            r = usdm.entropy_step(logits[b].numpy(), i, np.float32(inv_temp), np.float32(eta), pos0 + off, b,
                                  step_id, seed)
            np.testing.assert_array_equal(got_choice[b], r["x_tilde"])
            np.testing.assert_array_equal(got_H[b].view(np.int32), r["H"].view(np.int32))
            np.testing.assert_array_equal(got_next[b, off:], r["next"])
            np.testing.assert_array_equal(got_next[b, :off], canvas[b, :off].numpy())
            if i > 1:
                assert 0 < r["accept"].sum() <= Lc
    finally:
        tadm.tadm_model_destroy(m)


@pytest.mark.parametrize("name,overrides,rtol,atol", [
    ("tiny", {}, 1e-4, 1e-5),
    ("small", dict(vocab=4096, n_anchor=1, n_denoise=1), 2e-2, 2e-2),
])
def test_selfcond_matches_oracle(name, overrides, rtol, atol):
    """s = softmax(l * inv_temp) E from the GEMM over the step's weights, against the
    float64 expectation (fp32 model: 1e-4; bf16 model: the 2e-2 bar)."""
    cfg = synth.get_config(name, **overrides)
    B, L, off = 2, 40, 8
    Lc, V, d = L - off, cfg["vocab"], cfg["d_model"]
    tensors = synth.make_weights(cfg)
    m = gpu_model(cfg, tensors, B, L)
    try:
        logits = synth.make_logits(B * Lc, V, seed=5, std=2.0).view(B, Lc, V)
        canvas = torch.randint(0, V, (B, L), generator=torch.Generator().manual_seed(1), dtype=torch.int32)
        sc = torch.empty(B, Lc, d, device=dev())
        args = tadm.step_args(4, 8, 0, 3, 9, float(np.float32(1.25)), entropy_eta=0.1, sc_out=sc)
        nxt = torch.empty(B, L, dtype=torch.int32, device=dev())
        tadm.tadm_sample(m, logits.to(dev()), canvas.to(dev()), B, L, off, 0, args, nxt)
        sync()
        E = tensors[[sp[0] for sp in synth.weight_specs(cfg)].index("embed")]
        ref = usdm.selfcond(logits.numpy(), np.float32(1.25), E.float().numpy())
        if name != "tiny":  # s is ~1e-2 in size: the bar's atol is taken relative to it (stricter)
            atol = atol * float(np.sqrt((ref ** 2).mean()))
        rows_close(sc.cpu().numpy(), ref, rtol, atol, f"{name} self-conditioning")
    finally:
        tadm.tadm_model_destroy(m)


def test_anchor_and_step_with_selfcond_match_oracle():
    """Teacher-forced refresh and entropy step with a self-conditioning input (fp32 tiny
    model): logits within 1e-4 of the oracle's decoder with s added to the embeddings,
    and the step's canvas equal to the oracle's step on the GPU's own logits."""
    cfg = synth.get_config("tiny")
    B, P, G = 2, cfg["prompt_len"], cfg["gen_len"]
    L, V, d = P + G, cfg["vocab"], cfg["d_model"]
    tensors = synth.make_weights(cfg, perturb=True)
    net = oracle_net(cfg, tensors)
    m = gpu_model(cfg, tensors, B, L)
    cache = tadm.tadm_cache_create(m, B, L)
    try:
        canvas = torch.randint(0, V, (B, L), generator=torch.Generator().manual_seed(3), dtype=torch.int32)
        sc = (torch.randn(B, G, d, generator=torch.Generator().manual_seed(4)) * 0.3).float()
        d_sc = sc.to(dev())
        tadm.tadm_anchor_forward_sc(m, None, canvas.to(dev()), B, L, 5, 8, d_sc, P, cache)
        logits = torch.empty(B, G, V, device=dev())
        nxt = torch.empty(B, L, dtype=torch.int32, device=dev())
        args = tadm.step_args(5, 8, 0, 3, 77, float(np.float32(1.5)), entropy_eta=0.2, sc_in=d_sc)
        tadm.tadm_denoise_step(m, None, canvas.to(dev()), B, L, P, cache, args, logits, nxt)
        sync()
        got = logits.cpu().numpy()
        pos = np.arange(L)
        for b in range(B):
            full_sc = np.zeros((L, d))
            full_sc[P:] = sc[b].numpy()
            c = net.shared(canvas[b].numpy(), pos, sc=full_sc)
            anchor = net.anchor_cache(c, pos)
            xf = net.denoise(net.fuse(c, anchor), pos)
            ref = net.head(xf[P:]).astype(np.float32)
            rows_close(got[b], ref, 1e-4, 1e-4, f"row {b} logits with self-conditioning")
            r = usdm.entropy_step(got[b], 5, np.float32(1.5), np.float32(0.2), P, b, 3, 77)
            np.testing.assert_array_equal(nxt[b].cpu().numpy()[P:], r["next"])
    finally:
        tadm.tadm_cache_destroy(cache)
        tadm.tadm_model_destroy(m)


@pytest.mark.parametrize("T,K,block", [(8, 1, False), (8, 3, False), (6, 2, True)])
def test_tiny_entropy_generation_matches_oracle(T, K, block):
    """Whole uniform-state generations (entropy-bound sampler, self-conditioning, anchor
    refresh every K steps) are token-identical to the oracle's."""
    cfg = synth.get_config("tiny", batch=2, n_kv_heads=2 if block else 4)
    B, P, G = 2, cfg["prompt_len"], cfg["gen_len"]
    bl = 8 if block else G
    tensors = synth.make_weights(cfg, perturb=True)
    prompt = synth.make_prompt(cfg, batch=B)
    m = gpu_model(cfg, tensors, B, P + G)
    try:
        out = torch.empty(B, P + G, dtype=torch.int32, device=dev())
        tadm.tadm_generate_sampler(m, prompt.to(dev()), B, P, G, T, K, bl, 6, 1.0, tadm.entropy_sampler(), out)
        sync()
        got = out.cpu().numpy()
    finally:
        tadm.tadm_model_destroy(m)
    net = oracle_net(cfg, tensors)
    ref = loop.generate_usdm(net, prompt.numpy(), G, T, K, bl, 6)
    np.testing.assert_array_equal(got, ref)
