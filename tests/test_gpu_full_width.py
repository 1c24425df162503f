"""Full-width, full-batch parity of the benchmark workloads (GPU).

The block-diffusion, 1B-class and 26B-class workloads at their full width, vocabulary,
batch and sequence sizes, so that every kernel runs in the launch configuration the
benchmark times (GEMM tile shapes follow the row count, attention the context length,
the fused head the vocabulary), with one anchor and one denoiser layer so that the
float64 oracle can follow a sampled row in seconds.  Per sampled row: the anchor
state, the fused state, the final hidden state and the logits against the oracle,
judged against the oracle's own bf16 noise floor at that shape (the spread between two
equally valid bf16 evaluations of the row); over the whole batch: the step with the
sampling epilogue equals, bit for bit, the step computed from the full logits.
"""
import numpy as np
import pytest
import torch

import paper_2609_37924_amd as tadm
import synth
from helpers import dev, gpu_model, oracle_net, unnormalised_attention, within_noise_floor
from oracle import network as N

pytestmark = pytest.mark.gpu



def say(msg):
    print(f"[full-width] {msg}", flush=True)


def _full_width(name, rows):
    cfg = synth.get_config(name, n_anchor=1, n_denoise=1)
    B, P, G, bl, V, d = (cfg[k] for k in ("batch", "prompt_len", "gen_len", "block_len", "vocab", "d_model"))
    single = bl == G
    Lw = P + G if single else bl          # positions of one call
    off = P if single else 0
    Lc = Lw - off
    say(f"{name}: B={B} P={P} G={G} block={bl} d={d} V={V}; generating weights")
    tensors = synth.make_weights(cfg, perturb=True)
    m = gpu_model(cfg, tensors, B, P + G)
    say("weights on the GPU")
    try:
        tadm.tadm_debug_taps(m, 1)
        prompt = synth.make_prompt(cfg, batch=B) if P else None
        ctx = None
        g = torch.Generator().manual_seed(5)
        if single:
            z0 = synth.make_teacher_canvas(cfg, (3 * G) // 4, batch=B, seed=21)
            z1 = synth.make_teacher_canvas(cfg, (2 * G) // 3, batch=B, seed=22)
            pos = np.arange(Lw)
        else:
            ctx = tadm.tadm_context_create(m, B, P + G)
            tadm.tadm_context_append(m, ctx, prompt.to(dev()), B, P)
            z0 = torch.full((B, bl), V, dtype=torch.int32)
            z1 = torch.randint(0, V, (B, bl), generator=g, dtype=torch.int32)
            z1[torch.rand(B, bl, generator=g) < 0.6] = V
            pos = np.arange(P, P + bl)
        T, i = 16, 11
        cache = tadm.tadm_cache_create(m, B, Lw)
        tadm.tadm_anchor_forward(m, ctx, z0.to(dev()), B, Lw, T, T, cache)
        h_gpu = torch.empty(B, Lw, d, device=dev())
        tadm.tadm_cache_read(cache, tadm.CACHE_H, h_gpu)
        args = tadm.step_args(i, T, tadm.tadm_unmask_count(Lc, i, T), T - i, 91, 1.0)
        d1 = z1.to(dev())
        logits = torch.empty(B, Lc, V, device=dev())
        nxt_full, nxt_fused = torch.empty_like(d1), torch.empty_like(d1)
        tadm.tadm_denoise_step(m, ctx, d1, B, Lw, off, cache, args, logits, nxt_full)
        fused = torch.empty(B, Lw, d, device=dev())
        final = torch.empty(B, Lc, d, device=dev())
        tadm.tadm_debug_read(m, tadm.TAP_FUSED, fused)
        tadm.tadm_debug_read(m, tadm.TAP_FINAL, final)
        tadm.tadm_denoise_step(m, ctx, d1, B, Lw, off, cache, args, None, nxt_fused)
        torch.cuda.synchronize()
        assert torch.equal(nxt_full, nxt_fused), "sampling epilogue differs from the full-logits step"
        say("GPU step done; fused-head step equals the full-logits step")
        net = oracle_net(cfg, tensors)
        del tensors
        orig = N.attention

        def oracle_row(b, attention):
            N.attention = attention
            try:
                kv = None if single else net.fresh_kv(prompt[b].numpy(), np.arange(P))
                cache_ref = net.anchor_cache(net.shared(z0[b].numpy(), pos, kv), pos, kv)
                ht = net.fuse(net.shared(z1[b].numpy(), pos, kv), cache_ref)
                xf = net.denoise(ht, pos, kv)[off:]
                return {"anchor h": cache_ref["h"], "fused": ht, "final": xf, "logits": net.head(xf)}
            finally:
                N.attention = orig

        for b in rows:
            say(f"oracle row {b} (two bf16 evaluations)")
            ref, alt = oracle_row(b, orig), oracle_row(b, unnormalised_attention(orig))
            got = {"anchor h": h_gpu[b], "fused": fused[b], "final": final[b], "logits": logits[b]}
            for k in ref:
                within_noise_floor(got[k].cpu().numpy(), ref[k], alt[k], f"{name} {k} row {b}")
        tadm.tadm_cache_destroy(cache)
        if ctx is not None:
            tadm.tadm_context_destroy(ctx)
    finally:
        tadm.tadm_model_destroy(m)


def test_block_workload_full_width():
    """Block diffusion: d=2048, 16 heads / 4 KV heads of 128, SwiGLU 8192, V=128256,
    B=16, 512-token prompt prefilled into the context, 64-position blocks."""
    _full_width("block", rows=[0, 15])


def test_1b_workload_full_width():
    """1B-class: d=2048, 16 heads of 128, GELU 8192, V=50304, B=32, 1024 positions."""
    _full_width("1b", rows=[0, 31])


def test_26b_workload_full_width():
    """26B-class post-trained shape: d=4608, 32 heads / 16 KV heads of 128, GeGLU 36864,
    paired-attention fusion of rank 256, V=262144, B=4, 1024-token prompt, 256-position
    blocks."""
    _full_width("26b", rows=[3])
