"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Floating point: hidden states and logits within rtol = atol = 1e-4 (float32 models)
or 2e-2 (bf16 models).  Integers (token choices, unmask order, canvases): bit-exact
given identical logits; the confidence is compared bit for bit as well.
"""
import numpy as np
import pytest
import torch

import synth
from helpers import dev, gpu_model, oracle_net, oracle_sample_rows, oracle_step, rows_close
from oracle import loop
from oracle import sampler as S

pytestmark = pytest.mark.gpu

tadm = pytest.importorskip("paper_2609_37924_amd")

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

FP32_TOL = dict(rtol=1e-4, atol=1e-4)
BF16_TOL = dict(rtol=2e-2, atol=2e-2)


def sync():
    torch.cuda.synchronize()


# ------------------------------------------------------------------ sampler
@pytest.mark.parametrize("V,B,L,off,temp,ties,std", [
    (256, 2, 40, 8, 1.0, False, 2.0),
    (1001, 3, 33, 0, 0.7, False, 2.0),    # vocab not a multiple of 4: scalar path
    (32768, 2, 24, 4, 1.0, False, 2.0),
    (64, 4, 64, 0, 1.0, True, 2.0),       # duplicated rows and planted exact ties
    (8, 32, 1024, 0, 1.0, False, 1e-3),   # near-equal scores: many rows take the exact fallback
    (4, 16, 256, 0, 1.0, False, 0.0),     # all logits equal: the Gumbel noise alone decides
    (50304, 1, 6, 2, 1.3, False, 30.0),   # wide, peaked distribution
    (65, 2, 16, 0, 1.0, False, 2.0),      # one normaliser group and one entry
    (1025, 2, 8, 0, 0.9, False, 4.0),     # one 1024-entry chunk and one entry
    (262144, 1, 3, 0, 1.0, False, 3.0),   # largest vocabulary: 4096 groups
])
def test_sampler_bit_exact(V, B, L, off, temp, ties, std):
    cfg = synth.get_config("tiny", vocab=V)
    m = tadm.tadm_model_create(tadm.make_config(cfg, max_batch=B, max_seq=L))
    tadm.tadm_set_stream(m, torch.cuda.current_stream().cuda_stream)
    try:
        g = torch.Generator().manual_seed(V + L)
        canvas = torch.randint(0, V, (B, L), generator=g, dtype=torch.int32)
        canvas[:, off:][torch.rand(B, L - off, generator=g) < 0.7] = V
        canvas[0, off:] = V  # one fully masked row
        if ties:
            canvas[1] = canvas[0]
        logits = synth.make_logits(B * (L - off), V, seed=V, std=std, ties=ties).view(B, L - off, V)
        if ties:
            logits[1] = logits[0]
        inv_temp = float(np.float32(1.0 / temp))
        pos0, step_id, seed, n = 17, 5, 0x1234_5678_9ABC, 6
        args = tadm.step_args(3, 8, n, step_id, seed, inv_temp)
        d_log, d_can = logits.to(dev()), canvas.to(dev())
        nxt = torch.empty_like(d_can)
        choice = torch.empty(B, L - off, dtype=torch.int32, device=dev())
        conf = torch.empty(B, L - off, dtype=torch.float32, device=dev())
        tadm.tadm_sample(m, d_log, d_can, B, L, off, pos0, args, nxt, choice, conf)
        sync()
        r_next, r_choice, r_conf = oracle_sample_rows(logits.numpy(), canvas.numpy().astype(np.int64),
                                                      V, n, pos0, off, step_id, seed, inv_temp)
        masked = canvas[:, off:].numpy() == V
        np.testing.assert_array_equal(choice.cpu().numpy()[masked], r_choice[masked])
        np.testing.assert_array_equal(conf.cpu().numpy().view(np.int32)[masked],
                                      r_conf.view(np.int32)[masked])
        np.testing.assert_array_equal(nxt.cpu().numpy(), r_next)
    finally:
        tadm.tadm_model_destroy(m)


# --------------------------------------------------------- one teacher step
def _teacher_step_parity(cfg, B, tol, rows=None, seed=0, n_masked=(None, None), tensors=None):
    """Refresh on canvas z0, then one stale step on canvas z1 (teacher forcing)."""
    P, G = cfg["prompt_len"], cfg["gen_len"]
    L = P + G
    tensors = tensors or synth.make_weights(cfg, perturb=True)
    net = oracle_net(cfg, tensors)
    m = gpu_model(cfg, tensors, B, L)
    try:
        tadm.tadm_debug_taps(m, 1)
        z0 = synth.make_teacher_canvas(cfg, n_masked[0] or G, batch=B, seed=seed + 11)
        z1 = synth.make_teacher_canvas(cfg, n_masked[1] or (2 * G) // 3, batch=B, seed=seed + 12)
        T, i = 16, 13
        cache = tadm.tadm_cache_create(m, B, L)
        d = cfg["d_model"]
        d0, d1 = z0.to(dev()), z1.to(dev())
        tadm.tadm_anchor_forward(m, None, d0, B, L, 16, T, cache)
        h_gpu = torch.empty(B, L, d, device=dev())
        tadm.tadm_cache_read(cache, tadm.CACHE_H, h_gpu)
        n = tadm.tadm_unmask_count(G, i, T)
        args = tadm.step_args(i, T, n, T - i, 77, 1.0)
        logits = torch.empty(B, G, cfg["vocab"], device=dev())
        nxt = torch.empty_like(d1)
        tadm.tadm_denoise_step(m, None, d1, B, L, P, cache, args, logits, nxt)
        taps = {}
        for tap, shape in ((tadm.TAP_EMBED, (B, L, d)), (tadm.TAP_FUSED, (B, L, d)),
                           (tadm.TAP_FINAL, (B, G, d))):
            taps[tap] = torch.empty(shape, device=dev())
            tadm.tadm_debug_read(m, tap, taps[tap])
        sync()
        pos = np.arange(L)
        rows = range(B) if rows is None else rows
        ref_logits = np.zeros((B, G, cfg["vocab"]), np.float32)
        for b in rows:
            cache_ref = net.anchor_cache(net.shared(z0[b].numpy(), pos), pos)
            rows_close(h_gpu[b].cpu().numpy(), cache_ref["h"], what=f"anchor h row {b}", **tol)
            c, ht, xf, lg = oracle_step(net, z1[b].numpy(), pos, cache_ref, P)
            rows_close(taps[tadm.TAP_EMBED][b].cpu().numpy(), c, what=f"embed row {b}", **tol)
            rows_close(taps[tadm.TAP_FUSED][b].cpu().numpy(), ht, what=f"fused row {b}", **tol)
            rows_close(taps[tadm.TAP_FINAL][b].cpu().numpy(), xf, what=f"final row {b}", **tol)
            rows_close(logits[b].cpu().numpy(), lg, what=f"logits row {b}", **tol)
            ref_logits[b] = lg
        # the GPU reverse step on the oracle's logits is bit-exact with the oracle's
        r_next, _, _ = oracle_sample_rows(ref_logits, z1.numpy().astype(np.int64), cfg["vocab"], n, 0, P,
                                          T - i, 77, 1.0)
        nxt2 = torch.empty_like(d1)
        tadm.tadm_sample(m, torch.from_numpy(ref_logits).to(dev()), d1, B, L, P, 0, args, nxt2)
        sync()
        for b in rows:
            np.testing.assert_array_equal(nxt2[b].cpu().numpy(), r_next[b])
        tadm.tadm_cache_destroy(cache)
    finally:
        tadm.tadm_model_destroy(m)


@pytest.mark.parametrize("V,B,L,off,top_p,std,ties", [
    (256, 2, 40, 8, 0.9, 2.0, False),
    (1001, 2, 24, 0, 0.5, 1.0, False),      # vocabulary not a multiple of 4
    (64, 2, 32, 0, 0.3, 2.0, True),         # planted ties, duplicated rows
    (4, 4, 64, 0, 0.5, 0.0, False),         # all logits equal: the whole vocabulary is the nucleus
    (32768, 1, 12, 2, 0.95, 0.5, False),    # largest row kept in registers
    (50304, 1, 6, 0, 0.9, 30.0, False),     # peaked: a nucleus of a few entries
    (128, 2, 16, 0, 1e-7, 1.0, False),      # tiny p: the top entries only
    (4096, 2, 8, 0, 0.9999, 3.0, False),    # threshold deep in the small weights (digit 0 of each pass)
    (65536, 1, 4, 0, 0.8, 3.0, False),      # weights recomputed per pass
    (131072, 1, 4, 0, 0.9, 1.0, False),
])
def test_nucleus_sampler_bit_exact(V, B, L, off, top_p, std, ties):
    """Confidence-ranked step with top-p tokens: choice, confidence and next canvas equal
    the oracle's bit for bit (threshold by four radix passes over exact int64 weights)."""
    cfg = synth.get_config("tiny", vocab=V)
    m = tadm.tadm_model_create(tadm.make_config(cfg, max_batch=B, max_seq=L))
    tadm.tadm_set_stream(m, torch.cuda.current_stream().cuda_stream)
    try:
        g = torch.Generator().manual_seed(V + 1)
        canvas = torch.randint(0, V, (B, L), generator=g, dtype=torch.int32)
        canvas[:, off:][torch.rand(B, L - off, generator=g) < 0.7] = V
        logits = synth.make_logits(B * (L - off), V, seed=V + 1, std=std, ties=ties).view(B, L - off, V)
        tp = float(np.float32(top_p))
        args = tadm.step_args(3, 8, 5, 6, 0x5EED, 1.0, top_p=tp)
        d_can = canvas.to(dev())
        nxt = torch.empty_like(d_can)
        choice = torch.empty(B, L - off, dtype=torch.int32, device=dev())
        conf = torch.empty(B, L - off, dtype=torch.float32, device=dev())
        tadm.tadm_sample(m, logits.to(dev()), d_can, B, L, off, 9, args, nxt, choice, conf)
        sync()
        r_next, r_choice, r_conf = oracle_sample_rows(logits.numpy(), canvas.numpy().astype(np.int64), V, 5, 9, off,
                                                      6, 0x5EED, 1.0, top_p=tp)
        masked = canvas[:, off:].numpy() == V
        np.testing.assert_array_equal(choice.cpu().numpy()[masked], r_choice[masked])
        np.testing.assert_array_equal(conf.cpu().numpy().view(np.int32)[masked], r_conf.view(np.int32)[masked])
        np.testing.assert_array_equal(nxt.cpu().numpy(), r_next)
    finally:
        tadm.tadm_model_destroy(m)


def test_sampler_per_row_counts():
    """Per-row unmask counts from a device array (clamped to each row's masked count,
    negative counts reveal nothing) against the oracle step with each row's own n."""
    V, B, L, off = 512, 5, 48, 6
    cfg = synth.get_config("tiny", vocab=V)
    m = tadm.tadm_model_create(tadm.make_config(cfg, max_batch=B, max_seq=L))
    tadm.tadm_set_stream(m, torch.cuda.current_stream().cuda_stream)
    try:
        g = torch.Generator().manual_seed(7)
        canvas = torch.randint(0, V, (B, L), generator=g, dtype=torch.int32)
        canvas[:, off:][torch.rand(B, L - off, generator=g) < 0.6] = V
        logits = synth.make_logits(B * (L - off), V, seed=3, std=2.0).view(B, L - off, V)
        counts = torch.tensor([0, 3, 1000, -2, 7], dtype=torch.int32)
        d_counts = counts.to(dev())
        args = tadm.step_args(3, 8, 99, 4, 77, 1.0, n_unmask_rows=d_counts)
        d_can = canvas.to(dev())
        nxt = torch.empty_like(d_can)
        tadm.tadm_sample(m, logits.to(dev()), d_can, B, L, off, 5, args, nxt)
        sync()
        got = nxt.cpu().numpy()
        for b in range(B):
            n = max(int(counts[b]), 0)
            ref_b = S.reverse_step(logits[b].numpy(), canvas[b, off:].numpy().astype(np.int64), V, n, 5 + off, b, 4,
                                   77, np.float32(1.0))[0]
            assert np.array_equal(got[b, off:], ref_b), b
            assert np.array_equal(got[b, :off], canvas[b, :off].numpy())
    finally:
        tadm.tadm_model_destroy(m)


@pytest.mark.parametrize("V,off,sigma,p_unmask", [(300, 5, 0.3, 0.6), (64, 0, 0.0, 0.125), (1001, 3, 0.04, 1.0)])
def test_remask_step_bit_exact(V, off, sigma, p_unmask):
    """Remasking posterior on given logits: every entry's move (unmask to its Gumbel-max
    token, stay masked, keep, remask) equals the oracle's bit for bit."""
    B, L = 4, 40
    cfg = synth.get_config("tiny", vocab=V)
    m = tadm.tadm_model_create(tadm.make_config(cfg, max_batch=B, max_seq=L))
    tadm.tadm_set_stream(m, torch.cuda.current_stream().cuda_stream)
    try:
        g = torch.Generator().manual_seed(V)
        canvas = torch.randint(0, V, (B, L), generator=g, dtype=torch.int32)
        canvas[:, off:][torch.rand(B, L - off, generator=g) < 0.5] = V
        logits = synth.make_logits(B * (L - off), V, seed=V, std=2.0).view(B, L - off, V)
        sg, pu = np.float32(sigma), np.float32(p_unmask)
        args = tadm.step_args(5, 16, 0, 9, 0xABCDEF, 1.0, remask=(float(pu), float(sg)))
        d_can = canvas.to(dev())
        nxt = torch.empty_like(d_can)
        tadm.tadm_sample(m, logits.to(dev()), d_can, B, L, off, 12, args, nxt)
        sync()
        for b in range(B):
            ref, _ = S.remask_step(logits[b].numpy(), canvas[b, off:].numpy().astype(np.int64), V, pu, sg, 12 + off, b,
                                   9, 0xABCDEF, np.float32(1.0))
            assert np.array_equal(nxt[b, off:].cpu().numpy(), ref), b
            assert np.array_equal(nxt[b, :off].cpu().numpy(), canvas[b, :off].numpy())
    finally:
        tadm.tadm_model_destroy(m)


def test_tiny_fp32_step_parity():
    _teacher_step_parity(synth.get_config("tiny", batch=2), 2, FP32_TOL)


def test_tiny_fp32_swiglu_gqa_step_parity():
    cfg = synth.get_config("tiny", ffn_kind="swiglu", n_kv_heads=2, prompt_len=5, gen_len=70)
    _teacher_step_parity(cfg, 2, FP32_TOL)


def test_small_shape_bf16_step_parity():
    """The small model's widths (d=768, 12x64 heads, SwiGLU 2048, V=32768) with fewer
    layers and a ragged sequence (90 positions: 64-row tiles plus a tail)."""
    cfg = synth.get_config("small", n_anchor=2, n_denoise=2, prompt_len=40, gen_len=50)
    _teacher_step_parity(cfg, 2, BF16_TOL)


def test_small_config_full_size_sampled_rows():
    """Full small workload (12 anchor + 2 denoiser layers, B=8, 384 positions) in the
    launch configuration of the benchmark; the oracle checks rows 0 and 7."""
    cfg = synth.get_config("small")
    _teacher_step_parity(cfg, 8, BF16_TOL, rows=[0, 7], n_masked=(256, 200))


def test_gelu_bf16_step_parity():
    """GELU feed-forward, d=2048 / 128-wide heads as in the 1B-class model, few layers."""
    cfg = synth.get_config("1b", n_anchor=1, n_denoise=1, vocab=4096, prompt_len=16, gen_len=112)
    _teacher_step_parity(cfg, 2, BF16_TOL)


@pytest.mark.parametrize("dh,H,Hkv,B,gen", [(64, 12, 12, 2, 100), (128, 16, 16, 2, 100), (128, 16, 4, 2, 100),
                                             (128, 16, 16, 16, 100), (64, 12, 12, 24, 100), (128, 16, 4, 2, 2),
                                             (128, 16, 16, 2, 3), (128, 16, 16, 8, 100), (128, 16, 4, 8, 100)])
def test_attention_dominated_layer(dh, H, Hkv, B, gen):
    """One anchor layer whose output is dominated by attention (feed-forward off,
    V and O projections scaled up twofold: the attention output, rms ~1, is ~50 times
    the embedding it is added to), so that an attention error cannot hide behind the
    residual stream.  Covers both head widths and grouped KV heads.  At B = 16 / 24 the
    grid is large enough for two 16-query strips per wave (128-query blocks), and the
    130 positions leave a ragged second block of 2 queries.  At head width 128 and
    B = 2 the keys of each 64-key tile are split between two wave groups of one strip
    each, at B = 8 of two strips each; the 130 keys leave a last tile of 2 keys, which
    the second group skips, 32 keys give that group no key at all, and 33 keys give it
    one."""
    cfg = synth.get_config("1b", n_anchor=1, n_denoise=1, vocab=512, n_heads=H, n_kv_heads=Hkv,
                           head_dim=dh, d_model=H * dh, prompt_len=30, gen_len=gen)
    tensors = synth.make_weights(cfg, perturb=True)
    names = [s[0] for s in synth.weight_specs(cfg)]
    for li in range(2):
        tensors[names.index(f"layer{li}.wv")] = (tensors[names.index(f"layer{li}.wv")].float() * 2).bfloat16()
        tensors[names.index(f"layer{li}.wo")] = (tensors[names.index(f"layer{li}.wo")].float() * 2).bfloat16()
        tensors[names.index(f"layer{li}.w_down")] = torch.zeros_like(tensors[names.index(f"layer{li}.w_down")])
    _teacher_step_parity(cfg, B, BF16_TOL, tensors=tensors, rows=None if B == 2 else [0, B - 1])


def test_tiny_fp32_paired_step_parity():
    cfg = synth.get_config("tiny", fusion_kind="paired", fusion_rank=32, batch=2)
    _teacher_step_parity(cfg, 2, FP32_TOL)


def test_paired_bf16_step_parity():
    """Paired-attention fusion at rank 256 (4 heads of 64) with GQA and GeGLU as in the
    26B-class shape, narrower model and few layers."""
    cfg = synth.get_config("26b", d_model=1024, n_heads=8, n_kv_heads=4, head_dim=128, d_ffn=2048,
                           n_anchor=2, n_denoise=1, vocab=4096, prompt_len=20, gen_len=100, block_len=100)
    _teacher_step_parity(cfg, 2, BF16_TOL)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_paired_fresh_anchor_identity_bitwise(dtype):
    """At a refresh step C = C0, so the fused state must equal the cached anchor H0
    exactly (App. C.1): both mixer evaluations run the same deterministic kernels."""
    over = dict(fusion_kind="paired", batch=2, dtype=dtype)
    if dtype == "bf16":
        over.update(d_model=512, n_heads=8, n_kv_heads=8, head_dim=64, d_ffn=1024, fusion_rank=256)
    else:
        over.update(fusion_rank=32)
    cfg = synth.get_config("tiny", **over)
    B, P, G = 2, cfg["prompt_len"], cfg["gen_len"]
    L = P + G
    tensors = synth.make_weights(cfg, perturb=True)
    m = gpu_model(cfg, tensors, B, L)
    try:
        tadm.tadm_debug_taps(m, 1)
        cache = tadm.tadm_cache_create(m, B, L)
        z = synth.make_teacher_canvas(cfg, 11, batch=B, seed=8).to(dev())
        tadm.tadm_anchor_forward(m, None, z, B, L, 5, 5, cache)
        args = tadm.step_args(5, 5, 2, 0, 1, 1.0)
        nz = torch.empty_like(z)
        tadm.tadm_denoise_step(m, None, z, B, L, P, cache, args, None, nz)
        fused = torch.empty(B, L, cfg["d_model"], device=dev())
        h0 = torch.empty_like(fused)
        tadm.tadm_debug_read(m, tadm.TAP_FUSED, fused)
        tadm.tadm_cache_read(cache, tadm.CACHE_H, h0)
        sync()
        assert torch.equal(fused, h0)
        tadm.tadm_cache_destroy(cache)
    finally:
        tadm.tadm_model_destroy(m)


def test_tiny_paired_generation_matches_oracle():
    cfg = synth.get_config("tiny", batch=2, fusion_kind="paired", fusion_rank=32)
    tensors, prompt, got = _generate(cfg, 4)
    net = oracle_net(cfg, tensors)
    ref = loop.generate(net, prompt.numpy(), cfg["gen_len"], cfg["T"], 4, cfg["block_len"], 2, 1.0,
                        synth.mask_id(cfg))
    np.testing.assert_array_equal(got, ref)


def test_block_mode_bf16_step_parity():
    """Block diffusion with GQA at bf16: the prompt is prefilled into the context KV
    (a fresh pass through every layer), then a refresh and a stale step run on the
    active block attending to [context | block] (App. C.1 encoder/decoder split)."""
    cfg = synth.get_config("block", d_model=512, n_heads=8, n_kv_heads=2, head_dim=64, d_ffn=1024,
                           n_anchor=2, n_denoise=2, vocab=4096, batch=2, prompt_len=70, gen_len=128,
                           block_len=64)
    B, P, bl = 2, cfg["prompt_len"], cfg["block_len"]
    tensors = synth.make_weights(cfg, perturb=True)
    net = oracle_net(cfg, tensors)
    m = gpu_model(cfg, tensors, B, P + cfg["gen_len"])
    try:
        ctx = tadm.tadm_context_create(m, B, P + cfg["gen_len"])
        prompt = synth.make_prompt(cfg, batch=B)
        tadm.tadm_context_append(m, ctx, prompt.to(dev()), B, P)
        assert tadm.tadm_context_length(ctx) == P
        g = torch.Generator().manual_seed(3)
        z0 = torch.full((B, bl), cfg["vocab"], dtype=torch.int32)
        z1 = torch.randint(0, cfg["vocab"], (B, bl), generator=g, dtype=torch.int32)
        z1[torch.rand(B, bl, generator=g) < 0.6] = cfg["vocab"]
        cache = tadm.tadm_cache_create(m, B, bl)
        tadm.tadm_anchor_forward(m, ctx, z0.to(dev()), B, bl, 8, 8, cache)
        args = tadm.step_args(6, 8, 5, 2, 4, 1.0)
        logits = torch.empty(B, bl, cfg["vocab"], device=dev())
        nxt = torch.empty(B, bl, dtype=torch.int32, device=dev())
        tadm.tadm_denoise_step(m, ctx, z1.to(dev()), B, bl, 0, cache, args, logits, nxt)
        sync()
        pos = np.arange(P, P + bl)
        for b in range(B):
            kv = net.fresh_kv(prompt[b].numpy(), np.arange(P))
            cache_ref = net.anchor_cache(net.shared(z0[b].numpy(), pos, kv), pos, kv)
            c = net.shared(z1[b].numpy(), pos, kv)
            xf = net.denoise(net.fuse(c, cache_ref), pos, kv)
            rows_close(logits[b].cpu().numpy(), net.head(xf), what=f"block logits row {b}", **BF16_TOL)
        tadm.tadm_cache_destroy(cache)
        tadm.tadm_context_destroy(ctx)
    finally:
        tadm.tadm_model_destroy(m)


# -------------------------------------------------------------- generation
def _generate(cfg, K, block_len=None, B=None):
    B = B or cfg["batch"]
    P, G, T = cfg["prompt_len"], cfg["gen_len"], cfg["T"]
    bl = block_len or cfg["block_len"]
    tensors = synth.make_weights(cfg, perturb=True)
    prompt = synth.make_prompt(cfg, batch=B)
    m = gpu_model(cfg, tensors, B, P + G)
    try:
        out = torch.empty(B, P + G, dtype=torch.int32, device=dev())
        tadm.tadm_generate(m, prompt.to(dev()) if P else None, B, P, G, T, K, bl, 2, 1.0, out)
        sync()
        return tensors, prompt, out.cpu().numpy()
    finally:
        tadm.tadm_model_destroy(m)


@pytest.mark.parametrize("K", [4, 1])
def test_tiny_generation_matches_oracle(K):
    cfg = synth.get_config("tiny", batch=2)
    tensors, prompt, got = _generate(cfg, K)
    net = oracle_net(cfg, tensors)
    ref = loop.generate(net, prompt.numpy(), cfg["gen_len"], cfg["T"], K, cfg["block_len"], 2, 1.0,
                        synth.mask_id(cfg))
    np.testing.assert_array_equal(got, ref)


@pytest.mark.parametrize("eta,block,top_p", [(0.04, False, 0.0), (0.5, False, 0.0), (0.3, True, 0.0),
                                             (0.04, False, 0.9), (0.3, True, 0.6)])
def test_tiny_remask_generation_matches_oracle(eta, block, top_p):
    """Whole generations with the remasking sampler (capped sigma) are token-identical
    to the oracle's Algorithm 1 with the same posterior, and end fully unmasked."""
    cfg = synth.get_config("tiny", batch=2, n_kv_heads=2 if block else 4)
    K = 4
    B, P, G, T = 2, cfg["prompt_len"], cfg["gen_len"], cfg["T"]
    bl = 8 if block else G
    tensors = synth.make_weights(cfg, perturb=True)
    prompt = synth.make_prompt(cfg, batch=B)
    m = gpu_model(cfg, tensors, B, P + G)
    try:
        out = torch.empty(B, P + G, dtype=torch.int32, device=dev())
        tadm.tadm_generate_sampler(m, prompt.to(dev()), B, P, G, T, K, bl, 2, 1.0, tadm.remask_sampler(eta, top_p),
                                   out)
        sync()
        got = out.cpu().numpy()
    finally:
        tadm.tadm_model_destroy(m)
    net = oracle_net(cfg, tensors)
    ref = loop.generate(net, prompt.numpy(), G, T, K, bl, 2, 1.0, synth.mask_id(cfg), remask_eta=eta,
                        top_p=float(np.float32(top_p)) if top_p else 1.0)
    np.testing.assert_array_equal(got, ref)
    assert (got != synth.mask_id(cfg)).all()


@pytest.mark.parametrize("T,block,top_p,params", [
    (32, False, 0.0, (0.02, 0.55, 0.05, 0.9)),   # the paper's ReMDM-Loop settings, T >= L
    (48, True, 0.9, (0.02, 0.55, 0.05, 0.9)),
    (40, False, 0.0, (0.3, 0.7, 0.2, 0.5)),      # long plateau, strong remasking
])
def test_tiny_loop_generation_matches_oracle(T, block, top_p, params):
    """Whole generations with the ReMDM-Loop schedule are token-identical to the oracle's
    Algorithm 1 with the same posterior, and end fully unmasked."""
    cfg = synth.get_config("tiny", batch=2, n_kv_heads=2 if block else 4)
    K = 4
    B, P, G = 2, cfg["prompt_len"], cfg["gen_len"]
    bl = 8 if block else G
    tensors = synth.make_weights(cfg, perturb=True)
    prompt = synth.make_prompt(cfg, batch=B)
    m = gpu_model(cfg, tensors, B, P + G)
    eta, t_on, t_off, a_on = params
    try:
        out = torch.empty(B, P + G, dtype=torch.int32, device=dev())
        tadm.tadm_generate_sampler(m, prompt.to(dev()), B, P, G, T, K, bl, 5, 1.0,
                                   tadm.loop_sampler(eta, t_on, t_off, a_on, top_p), out)
        sync()
        got = out.cpu().numpy()
    finally:
        tadm.tadm_model_destroy(m)
    net = oracle_net(cfg, tensors)
    ref = loop.generate(net, prompt.numpy(), G, T, K, bl, 5, 1.0, synth.mask_id(cfg), loop=params,
                        top_p=float(np.float32(top_p)) if top_p else 1.0)
    np.testing.assert_array_equal(got, ref)
    assert (got != synth.mask_id(cfg)).all()


@pytest.mark.parametrize("T,K,block_len,temp", [
    (1, 1, None, 1.0),     # a single reverse step reveals everything
    (40, 3, None, 0.5),    # more steps than positions: many steps reveal nothing; K does not divide T
    (16, 50, None, 2.0),   # K > T: only the first step refreshes the anchor
    (6, 2, 1, 1.0),        # one-token blocks, each appended to the context
])
def test_degenerate_schedules_match_oracle(T, K, block_len, temp):
    """Schedule edge cases of Algorithm 1 and the linear unmask count, token-identical to
    the oracle."""
    cfg = synth.get_config("tiny", batch=2, n_kv_heads=2)
    B, P, G = 2, cfg["prompt_len"], cfg["gen_len"]
    bl = block_len or G
    tensors = synth.make_weights(cfg, perturb=True)
    prompt = synth.make_prompt(cfg, batch=B)
    m = gpu_model(cfg, tensors, B, P + G)
    try:
        out = torch.empty(B, P + G, dtype=torch.int32, device=dev())
        tadm.tadm_generate(m, prompt.to(dev()), B, P, G, T, K, bl, 5, temp, out)
        sync()
        got = out.cpu().numpy()
    finally:
        tadm.tadm_model_destroy(m)
    ref = loop.generate(oracle_net(cfg, tensors), prompt.numpy(), G, T, K, bl, 5, temp, synth.mask_id(cfg))
    np.testing.assert_array_equal(got, ref)
    assert (got != synth.mask_id(cfg)).all()


def test_tiny_block_generation_matches_oracle():
    cfg = synth.get_config("tiny", batch=2, n_kv_heads=2)
    tensors, prompt, got = _generate(cfg, 4, block_len=8)
    net = oracle_net(cfg, tensors)
    ref = loop.generate(net, prompt.numpy(), cfg["gen_len"], cfg["T"], 4, 8, 2, 1.0, synth.mask_id(cfg))
    np.testing.assert_array_equal(got, ref)


def test_bf16_generation_invariants():
    cfg = synth.get_config("small", n_anchor=2, n_denoise=1, batch=3)
    _, prompt, got = _generate(cfg, 4)
    P = cfg["prompt_len"]
    assert np.array_equal(got[:, :P], prompt.numpy())
    assert (got >= 0).all() and (got < cfg["vocab"]).all()


@pytest.mark.parametrize("block_len", [None, 16])
def test_bf16_generation_step_by_step_matches_oracle_sampler(block_len):
    """A whole bf16 generation (single canvas, and block mode with context KV), replayed
    step by step through the C ABI with the product path (masked-only head with the
    sampling epilogue, device-side row compaction): at every step the sampled tokens,
    the confidences and the next canvas equal, bit for bit, the oracle's reverse step
    on that step's GPU logits (the same step run once more with a logits buffer), and
    the replay's final tokens equal tadm_generate's."""
    cfg = synth.get_config("small", n_anchor=2, n_denoise=1, prompt_len=40, gen_len=48, T=12)
    B, P, G, T, K, V = 3, 40, 48, 12, 4, cfg["vocab"]
    bl = block_len or G
    single = bl == G
    seed, inv_temp = 0x51CE, 1.0
    tensors = synth.make_weights(cfg, perturb=True)
    prompt = synth.make_prompt(cfg, batch=B)
    m = gpu_model(cfg, tensors, B, P + G)
    try:
        tadm.tadm_debug_taps(m, 1)
        out = torch.empty(B, P + G, dtype=torch.int32, device=dev())
        tadm.tadm_generate(m, prompt.to(dev()), B, P, G, T, K, bl, seed, inv_temp, out)
        seq = torch.cat([prompt, torch.full((B, G), V, dtype=torch.int32)], 1).to(dev())
        ctx = None
        if not single:
            ctx = tadm.tadm_context_create(m, B, P + G)
            tadm.tadm_context_append(m, ctx, seq[:, :P].contiguous(), B, P)
        windows = [(0, P, P + G)] if single else [(P + j * bl, P + j * bl, P + (j + 1) * bl) for j in range(G // bl)]
        steps = 0
        for j, (w0, c0, w1) in enumerate(windows):
            Lw, off = w1 - w0, c0 - w0
            Lc = w1 - c0
            cache = tadm.tadm_cache_create(m, B, Lw)
            for i in range(T, 0, -1):
                z = seq[:, w0:w1].contiguous()
                if (T - i) % K == 0:
                    tadm.tadm_anchor_forward(m, ctx, z, B, Lw, i, T, cache)
                n = tadm.tadm_unmask_count(Lc, i, T)
                step_id = j * T + (T - i)
                args = tadm.step_args(i, T, n, step_id, seed, inv_temp)
                logits = torch.empty(B, Lc, V, device=dev())
                nz_full = torch.empty_like(z)
                tadm.tadm_denoise_step(m, ctx, z, B, Lw, off, cache, args, logits, nz_full)
                nz = torch.empty_like(z)
                tadm.tadm_denoise_step(m, ctx, z, B, Lw, off, cache, args, None, nz)
                choice = torch.empty(B, Lc, dtype=torch.int32, device=dev())
                conf = torch.empty(B, Lc, dtype=torch.float32, device=dev())
                tadm.tadm_debug_read(m, tadm.TAP_CHOICE, choice)
                tadm.tadm_debug_read(m, tadm.TAP_CONF, conf)
                sync()
                zc = z.cpu().numpy().astype(np.int64)
                r_next, r_choice, r_conf = oracle_sample_rows(logits.cpu().numpy(), zc, V, n, c0 - off, off,
                                                              step_id, seed, inv_temp)
                masked = zc[:, off:] == V
                np.testing.assert_array_equal(choice.cpu().numpy()[masked], r_choice[masked])
                np.testing.assert_array_equal(conf.cpu().numpy().view(np.int32)[masked],
                                              r_conf.view(np.int32)[masked])
                np.testing.assert_array_equal(nz.cpu().numpy(), r_next, err_msg=f"block {j} step i={i}")
                assert torch.equal(nz, nz_full)
                seq[:, w0:w1] = nz
                steps += 1
            tadm.tadm_cache_destroy(cache)
            if ctx is not None and j + 1 < len(windows):
                tadm.tadm_context_append(m, ctx, seq[:, w0:w1].contiguous(), B, Lw)
        sync()
        assert steps == T * len(windows)
        assert not (seq == V).any()
        assert torch.equal(seq, out), "the step-by-step replay differs from tadm_generate"
        if ctx is not None:
            tadm.tadm_context_destroy(ctx)
    finally:
        tadm.tadm_model_destroy(m)


# -------------------------------------------------------------- invariants
def test_cache_unchanged_between_refreshes_and_split_equals_generate():
    cfg = synth.get_config("tiny", batch=2)
    B, P, G, T, K = 2, cfg["prompt_len"], cfg["gen_len"], cfg["T"], 4
    L = P + G
    tensors = synth.make_weights(cfg, perturb=True)
    prompt = synth.make_prompt(cfg, batch=B)
    m = gpu_model(cfg, tensors, B, L)
    try:
        cache = tadm.tadm_cache_create(m, B, L)
        z = torch.cat([prompt, torch.full((B, G), cfg["vocab"], dtype=torch.int32)], 1).to(dev())
        snap = torch.empty(B, L, cfg["d_model"], device=dev())
        for i in range(T, 0, -1):
            if (T - i) % K == 0:
                tadm.tadm_anchor_forward(m, None, z, B, L, i, T, cache)
                tadm.tadm_cache_read(cache, tadm.CACHE_H, snap)
                ref = snap.clone()
            args = tadm.step_args(i, T, tadm.tadm_unmask_count(G, i, T), T - i, 2, 1.0)
            nz = torch.empty_like(z)
            tadm.tadm_denoise_step(m, None, z, B, L, P, cache, args, None, nz)
            tadm.tadm_cache_read(cache, tadm.CACHE_H, snap)
            sync()
            assert torch.equal(snap, ref)
            assert tadm.tadm_cache_refresh_step(cache) == T - ((T - i) // K) * K
            z = nz
        out = torch.empty(B, L, dtype=torch.int32, device=dev())
        tadm.tadm_generate(m, prompt.to(dev()), B, P, G, T, K, G, 2, 1.0, out)
        out2 = torch.empty_like(out)
        tadm.tadm_generate(m, prompt.to(dev()), B, P, G, T, K, G, 2, 1.0, out2)
        sync()
        assert torch.equal(out, z)        # explicit step loop == one-shot generate
        assert torch.equal(out, out2)     # deterministic
        tadm.tadm_cache_destroy(cache)
    finally:
        tadm.tadm_model_destroy(m)


def test_masked_only_head_equals_full_head():
    """Without caller logits the head runs on the masked positions only; the reverse
    step must be bit-identical to the one computed from the full logits."""
    cfg = synth.get_config("small", n_anchor=1, n_denoise=1, prompt_len=40, gen_len=50)
    B, P, G = 3, 40, 50
    L = P + G
    tensors = synth.make_weights(cfg, perturb=True)
    m = gpu_model(cfg, tensors, B, L)
    try:
        cache = tadm.tadm_cache_create(m, B, L)
        z0 = synth.make_teacher_canvas(cfg, G, batch=B, seed=3).to(dev())
        tadm.tadm_anchor_forward(m, None, z0, B, L, 8, 8, cache)
        for n_masked, seed in ((37, 4), (1, 5), (0, 6)):
            z = synth.make_teacher_canvas(cfg, n_masked, batch=B, seed=seed).to(dev())
            args = tadm.step_args(7, 8, 3, 1, 9, 1.0)
            full, part = torch.empty_like(z), torch.empty_like(z)
            logits = torch.empty(B, G, cfg["vocab"], device=dev())
            tadm.tadm_denoise_step(m, None, z, B, L, P, cache, args, logits, full)
            tadm.tadm_denoise_step(m, None, z, B, L, P, cache, args, None, part)
            sync()
            assert torch.equal(full, part), n_masked
        tadm.tadm_cache_destroy(cache)
    finally:
        tadm.tadm_model_destroy(m)


@pytest.mark.parametrize("vocab,d,masked", [
    (1000, 256, (37, 1)),      # 128 x 128 head tiles; last normaliser group has 40 entries
    (32768, 768, (50, 9)),     # the small workload's head
    (262144, 256, (20, 3)),    # largest vocabulary: 256 x 256 head tiles, 4096 groups
    (50304, 256, (41, 7)),     # 393 (fused) and 197 (logits) tile columns: no even split
                               # into 8 XCD regions, so both products take the banded walk
])
def test_fused_head_sampler_matches_unfused(vocab, d, masked):
    """The masked-only bf16 head samples in its epilogue.  Token and confidence of every
    masked position must equal, bit for bit, the standalone sampler on the full logits
    of the same step, and the oracle's sampling contract applied to those logits."""
    H = d // 64
    cfg = synth.get_config("small", n_anchor=1, n_denoise=1, prompt_len=24, gen_len=50, vocab=vocab,
                           d_model=d, n_heads=H, n_kv_heads=H, d_ffn=2 * d)
    B, P, G = 3, 24, 50
    L = P + G
    tensors = synth.make_weights(cfg, perturb=True)
    m = gpu_model(cfg, tensors, B, L)
    try:
        cache = tadm.tadm_cache_create(m, B, L)
        z0 = synth.make_teacher_canvas(cfg, G, batch=B, seed=3).to(dev())
        tadm.tadm_anchor_forward(m, None, z0, B, L, 8, 8, cache)
        for n_masked in masked:
            z = synth.make_teacher_canvas(cfg, n_masked, batch=B, seed=n_masked).to(dev())
            args = tadm.step_args(5, 8, 4, 11, 0xDEAD_BEEF_0042, float(np.float32(1 / 0.9)))
            got = {}
            logits = torch.empty(B, G, vocab, device=dev())
            for name, lg in (("unfused", logits), ("fused", None)):
                nxt = torch.empty_like(z)
                ch = torch.empty(B, G, dtype=torch.int32, device=dev())
                cf = torch.empty(B, G, dtype=torch.float32, device=dev())
                tadm.tadm_denoise_step(m, None, z, B, L, P, cache, args, lg, nxt)
                tadm.tadm_debug_read(m, tadm.TAP_CHOICE, ch)
                tadm.tadm_debug_read(m, tadm.TAP_CONF, cf)
                sync()
                got[name] = (nxt.cpu().numpy(), ch.cpu().numpy(), cf.cpu().numpy())
            msk = z[:, P:].cpu().numpy() == vocab
            assert msk.sum() == B * n_masked
            for k in range(3):
                a, b = got["unfused"][k], got["fused"][k]
                assert np.array_equal(a.view(np.int32), b.view(np.int32)), (n_masked, k)
            r_next, r_choice, r_conf = oracle_sample_rows(logits.cpu().numpy(), z.cpu().numpy().astype(np.int64),
                                                          vocab, 4, 0, P, 11, 0xDEAD_BEEF_0042, args.inv_temp)
            np.testing.assert_array_equal(got["fused"][1][msk], r_choice[msk])
            np.testing.assert_array_equal(got["fused"][2].view(np.int32)[msk], r_conf.view(np.int32)[msk])
            np.testing.assert_array_equal(got["fused"][0], r_next)
            # the remasking posterior on top of the fused head: same bits as from the logits
            rargs = tadm.step_args(5, 8, 0, 11, 0xDEAD_BEEF_0042, float(np.float32(1 / 0.9)), remask=(0.4, 0.2))
            nx = {}
            for name, lg in (("unfused", logits), ("fused", None)):
                nx[name] = torch.empty_like(z)
                tadm.tadm_denoise_step(m, None, z, B, L, P, cache, rargs, lg, nx[name])
            sync()
            assert torch.equal(nx["unfused"], nx["fused"]), n_masked
            r_next = np.stack([S.remask_step(logits[b].cpu().numpy(), z[b, P:].cpu().numpy().astype(np.int64), vocab,
                                             np.float32(0.4), np.float32(0.2), P, b, 11, 0xDEAD_BEEF_0042,
                                             np.float32(rargs.inv_temp))[0] for b in range(B)])
            np.testing.assert_array_equal(nx["fused"][:, P:].cpu().numpy(), r_next)
        tadm.tadm_cache_destroy(cache)
    finally:
        tadm.tadm_model_destroy(m)


def test_state_errors():
    cfg = synth.get_config("tiny")
    tensors = synth.make_weights(cfg)
    m = gpu_model(cfg, tensors, 1, 32)
    try:
        cache = tadm.tadm_cache_create(m, 1, 32)
        z = torch.zeros(1, 32, dtype=torch.int32, device=dev())
        args = tadm.step_args(1, 4, 1, 0, 0, 1.0)
        with pytest.raises(tadm.TadmError) as e:     # never refreshed
            tadm.tadm_denoise_step(m, None, z, 1, 32, 8, cache, args, None, z)
        assert e.value.status == tadm.TADM_ERR_STATE
        with pytest.raises(tadm.TadmError) as e:     # shape mismatch
            tadm.tadm_anchor_forward(m, None, z, 1, 16, 1, 4, cache)
        assert e.value.status == tadm.TADM_ERR_STATE
        with pytest.raises(tadm.TadmError) as e:     # batch too large
            tadm.tadm_anchor_forward(m, None, z, 2, 32, 1, 4, cache)
        assert e.value.status == tadm.TADM_ERR_INVALID
        tadm.tadm_cache_destroy(cache)
    finally:
        tadm.tadm_model_destroy(m)


def test_profile_stages_count_every_launch():
    """Stage timers: one interval per launch of each single-kernel stage over a whole
    generation (refresh iff (T - i) mod K == 0), each positive, nested inside its layer
    stages."""
    cfg = synth.get_config("tiny", batch=2)
    K, T = 4, cfg["T"]
    tensors = synth.make_weights(cfg)
    P, G = cfg["prompt_len"], cfg["gen_len"]
    m = gpu_model(cfg, tensors, 2, P + G)
    try:
        prompt = synth.make_prompt(cfg, batch=2).to(dev())
        out = torch.empty(2, P + G, dtype=torch.int32, device=dev())
        tadm.tadm_profile_reset(m)
        tadm.tadm_profile_enable(m, -1)
        tadm.tadm_generate(m, prompt, 2, P, G, T, K, G, 2, 1.0, out)
        tadm.tadm_profile_enable(m, 0)
        got = {name: tadm.tadm_profile_read(m, si) for si, name in enumerate(tadm.STAGES)}
        n_ref = -(-T // K)
        per_layer = n_ref * (cfg["n_shared"] + cfg["n_anchor"]) + T * (cfg["n_shared"] + cfg["n_denoise"])
        expect = {"qkv": per_layer, "attn": per_layer, "oproj": per_layer, "ffn_up": per_layer,
                  "ffn_down": per_layer, "fusion1": T, "fusion2": T, "head": T, "sample": T, "select": T,
                  "anchor": n_ref, "denoise": T}
        for name, n in expect.items():
            tot, cnt = got[name]
            assert cnt == n, (name, cnt, n)
            assert tot > 0, name
        inner = sum(got[n][0] for n in ("qkv", "attn", "oproj", "ffn_up", "ffn_down"))
        assert inner <= got["anchor"][0] + got["denoise"][0] + 1e-3
        tadm.tadm_profile_reset(m)
        assert tadm.tadm_profile_read(m, tadm.STAGES.index("head")) == (0.0, 0)
    finally:
        tadm.tadm_model_destroy(m)
