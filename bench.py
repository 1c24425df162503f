"""Benchmark: denoised tokens/s of TADM anchor-cache generation on one MI355X.

One step = one whole generation (Algorithm 1 over all T reverse steps, anchor
refreshes included) of a batch of synthetic prompts, enqueued by tadm_generate with
inputs already resident in HBM.  value = B * gen_len / time per step at the headline
refresh interval; the other refresh intervals of the workload are reported beside it.

Prints one JSON line.  Extra fields: the K sweep, per-stage time, the roofline of
the dominant kernel (algorithmic flops over its HIP-event-timed duration) and the
CPU oracle timed on a bounded sample.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="small")
    ap.add_argument("--K", type=int, default=4, help="headline refresh interval")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-sweep", action="store_true", help="only the headline K")
    ap.add_argument("--out", default=None, help="also write the JSON line to this file")
    return ap.parse_args()


def head_flops(cfg, B):
    """Algorithmic flops of the average vocabulary-projection launch, 2 * rows * d * V,
    where rows = the masked positions entering step i: B * floor(M0 * i / T) with M0
    the block length (the head only runs on masked positions)."""
    M0, T = cfg["block_len"], cfg["T"]
    rows = sum(B * ((M0 * i) // T) for i in range(1, T + 1)) / T
    return 2.0 * rows * cfg["d_model"] * cfg["vocab"]


def workload_name(cfg):
    return (f"{cfg['name']}: d{cfg['d_model']} {cfg['n_heads']}x{cfg['head_dim']} heads "
            f"({cfg['n_kv_heads']} kv) {cfg['ffn_kind']}{cfg['d_ffn']} V{cfg['vocab']}, "
            f"{cfg['n_anchor']} anchor + {cfg['n_denoise']} denoiser layers, {cfg['fusion_kind']} fusion, "
            f"B={cfg['batch']}, prompt {cfg['prompt_len']} + {cfg['gen_len']} generated "
            f"(block {cfg['block_len']}), T={cfg['T']}")


def cpu_baseline(cfg, K):
    """The oracle on one row of the workload's first block: one refresh step and one
    stale step (the first two reverse steps), each timed, scaled to the whole job
    (rows x blocks x (ceil(T/K) refresh steps + the other steps)).  Context prefill
    of block mode is not part of the sample."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import synth
    from oracle import loop, network as N, sampler as S

    specs = synth.weight_specs(cfg)
    tensors = synth.make_weights(cfg)
    net = N.Network(N.Weights(cfg, [s[0] for s in specs], tensors))
    del tensors
    P, G, T, bl = cfg["prompt_len"], cfg["gen_len"], cfg["T"], cfg["block_len"]
    single = bl == G
    mask = synth.mask_id(cfg)
    prompt = synth.make_prompt(cfg, batch=1).numpy()[0]
    if single:
        seq = np.concatenate([prompt, np.full(G, mask)])
        pos, off, ctx = np.arange(P + G), P, None
    else:  # first block after the prompt; the prompt context is built outside the timing
        seq = np.full(bl, mask)
        pos, off = np.arange(P, P + bl), 0
        ctx = net.fresh_kv(prompt, np.arange(P))
    times = []
    cache = None
    for k, refresh in enumerate((True, False)):
        i = T - k
        t0 = time.perf_counter()
        c = net.shared(seq, pos, ctx)
        if refresh:
            cache = net.anchor_cache(c, pos, ctx)
        xf = net.denoise(net.fuse(c, cache), pos, ctx)
        lg = net.head(xf[off:]).astype(np.float32)
        seq[off:], _, _ = S.reverse_step(lg, seq[off:], mask, loop.unmask_count(bl, i, T),
                                         pos[0] + off, 0, T - i, 2, np.float32(1.0))
        times.append(time.perf_counter() - t0)
    n_ref = math.ceil(T / K)
    job_s = cfg["batch"] * (G // bl) * (n_ref * times[0] + (T - n_ref) * times[1])
    threads = max([t.get("num_threads", 1) for t in threadpool_info()] + [1])
    return {"value": cfg["batch"] * G / job_s, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"1 of {cfg['batch']} rows, first block: one refresh step ({times[0]:.1f} s) and one "
                      f"stale step ({times[1]:.1f} s) at the full shape; scaled to rows x blocks x "
                      f"({n_ref} refresh + {T - n_ref} stale steps) per block, context prefill excluded"}


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build runs the path on a single MI355X "
              "(multi-GPU sharding is design only).", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2609_37924_amd as tadm
    import synth

    cfg = synth.get_config(args.config)
    dev = torch.device("cuda:0")
    B, P, G, T, bl = cfg["batch"], cfg["prompt_len"], cfg["gen_len"], cfg["T"], cfg["block_len"]
    stream = torch.cuda.current_stream()
    m = tadm.tadm_model_create(tadm.make_config(cfg, max_batch=B, max_seq=P + G))
    tadm.tadm_set_stream(m, stream.cuda_stream)
    t_load = time.perf_counter()
    for i, spec in enumerate(synth.weight_specs(cfg)):  # one tensor at a time: bounded memory
        t = synth.make_tensor(cfg, i, spec, device=dev)
        tadm.tadm_model_load_weight(m, i, t)
        del t
    torch.cuda.empty_cache()
    print(f"[bench] weights generated and loaded in {time.perf_counter() - t_load:.1f} s", file=sys.stderr,
          flush=True)
    prompt = synth.make_prompt(cfg, device=dev) if P else None
    out = torch.empty(B, P + G, dtype=torch.int32, device=dev)

    def gen(K):
        tadm.tadm_generate(m, prompt, B, P, G, T, K, bl, cfg["sampler_seed"], cfg["temperature"], out)

    def timed(K, steps, warmup, profile=0):
        """profile: stage bit mask recorded with HIP events inside the timed region."""
        for _ in range(warmup):
            gen(K)
        torch.cuda.synchronize()
        tadm.tadm_profile_reset(m)
        tadm.tadm_profile_enable(m, profile)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(steps):
            gen(K)
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        tadm.tadm_profile_enable(m, 0)
        ms = e0.elapsed_time(e1) / steps
        stages = {}
        if profile:
            for si, name in enumerate(tadm.STAGES):
                tot, n = tadm.tadm_profile_read(m, si)
                if n:
                    stages[name] = {"ms_per_step": tot / steps, "launches": n // steps, "avg_ms": tot / n}
        return ms, wall / steps * 1e3, stages

    K0 = args.K
    print(f"[bench] {workload_name(cfg)}", file=sys.stderr, flush=True)
    head_bit = 1 << tadm.STAGES.index("head")
    ms, wall_ms, head_only = timed(K0, args.steps, args.warmup, profile=head_bit)
    tokens = B * G
    value = tokens / (ms / 1e3)
    print(f"[bench] K={K0}: {ms:.3f} ms/generation ({wall_ms:.3f} wall) -> {value:.1f} tokens/s",
          file=sys.stderr, flush=True)
    # stage breakdown from a separate pass (events around every stage perturb timing)
    _, _, stages = timed(K0, max(1, args.steps // 2), 0, profile=-1)
    sweep = {}
    if not args.no_sweep:
        for K in cfg["Ks"]:
            kms, _, _ = timed(K, max(2, args.steps // 2), 1)
            sweep[f"K={K}"] = {"tokens_per_s": tokens / (kms / 1e3), "ms_per_step": kms}
            print(f"[bench] K={K}: {kms:.3f} ms -> {tokens / (kms / 1e3):.1f} tokens/s", file=sys.stderr,
                  flush=True)
    head = head_only.get("head")
    roof = None
    if head:
        flops = head_flops(cfg, B)
        achieved = flops / (head["avg_ms"] / 1e3) / 1e12
        roof = {"kernel": "vocabulary projection GEMM (bf16 MFMA, fp32 logits)", "bound": "mfma",
                "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None,
                "avg_launch_ms": head["avg_ms"], "flops_per_launch": flops}
    cpu = None
    if not args.no_cpu:
        try:
            cpu = cpu_baseline(cfg, K0)
        except Exception as e:  # the GPU number stands on its own
            print(f"[bench] cpu baseline failed: {e}", file=sys.stderr)
    tadm.tadm_model_destroy(m)
    line = {
        "metric": f"denoised tokens/s per MI355X at K={K0} (vs K=1 in k_sweep)",
        "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg["dtype"], "data": "synthetic (uniform-random prompts, seeded random-init weights)",
        "config": {"workload": workload_name(cfg), "global_batch": B, "seq_len": P + G, "K": K0,
                   "parallelism": "none (1 GPU)"},
        "k_sweep": sweep,
        "stages_ms_per_step": {k: v["ms_per_step"] for k, v in stages.items()},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(json.dumps(line) + "\n")


if __name__ == "__main__":
    main()
