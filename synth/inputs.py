"""Seeded prompts, canvases and logits.

Prompts are uniform token ids in [0, vocab).  Generated positions start as the
mask id.  Timing canvases for per-step measurement draw t ~ U(0,1) per row, set
i = ceil(t*T) and mask exactly floor(M0*i/T) of the M0 generated positions
(uniformly chosen), filling the rest with uniform tokens: the forward-corruption
marginal conditioned to lie on the linear unmask schedule.
"""
import math

import torch

from .configs import mask_id


def _gen(seed, device="cpu"):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) & 0x7FFFFFFFFFFFFFFF)
    return g


def make_prompt(cfg, batch=None, prompt_len=None, seed=None, device="cpu"):
    B = cfg["batch"] if batch is None else batch
    P = cfg["prompt_len"] if prompt_len is None else prompt_len
    seed = cfg["input_seed"] if seed is None else seed
    return torch.randint(0, cfg["vocab"], (B, P), generator=_gen(seed, device),
                         device=device, dtype=torch.int32)


def make_timing_canvas(cfg, T, batch=None, seed=None):
    """[B, prompt+gen] canvas at random per-row times on the linear schedule."""
    B = cfg["batch"] if batch is None else batch
    P, M0 = cfg["prompt_len"], cfg["gen_len"]
    seed = cfg["input_seed"] if seed is None else seed
    g = _gen(seed + 17)
    prompt = make_prompt(cfg, batch=B, seed=seed)
    gen = torch.randint(0, cfg["vocab"], (B, M0), generator=g, dtype=torch.int32)
    t = torch.rand(B, generator=g, dtype=torch.float64)
    steps = []
    for b in range(B):
        i = max(1, math.ceil(float(t[b]) * T))
        steps.append(i)
        n_mask = (M0 * i) // T
        perm = torch.randperm(M0, generator=g)[:n_mask]
        gen[b, perm] = mask_id(cfg)
    return torch.cat([prompt, gen], dim=1).contiguous(), steps


def make_teacher_canvas(cfg, n_masked, batch=None, seed=None):
    """Canvas whose generated part has exactly ``n_masked`` masked positions per row."""
    B = cfg["batch"] if batch is None else batch
    P, M0 = cfg["prompt_len"], cfg["gen_len"]
    seed = cfg["input_seed"] if seed is None else seed
    g = _gen(seed + 29)
    prompt = make_prompt(cfg, batch=B, seed=seed)
    gen = torch.randint(0, cfg["vocab"], (B, M0), generator=g, dtype=torch.int32)
    for b in range(B):
        perm = torch.randperm(M0, generator=g)[:n_masked]
        gen[b, perm] = mask_id(cfg)
    return torch.cat([prompt, gen], dim=1).contiguous()


def make_logits(rows, vocab, seed, std=1.0, ties=False):
    """fp32 logits [rows, vocab]; ``ties`` plants repeated maxima and duplicate rows."""
    g = _gen(seed)
    x = torch.randn(rows, vocab, generator=g, dtype=torch.float32) * std
    if ties and rows >= 4 and vocab >= 8:
        x[1] = x[0]
        x[2, 3] = x[2].max() + 1.0
        x[2, 5] = x[2, 3]
        x[3] = torch.round(x[3] * 2.0) / 2.0
    return x.contiguous()
