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
    """The oracle on one row of the workload, one refresh cycle (1 anchor refresh and
    K reverse steps at the start of generation), scaled to tokens/s of the whole job."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import synth
    from oracle import loop, network as N, sampler as S

    specs = synth.weight_specs(cfg)
    tensors = synth.make_weights(cfg)
    net = N.Network(N.Weights(cfg, [s[0] for s in specs], tensors))
    prompt = synth.make_prompt(cfg, batch=1).numpy()
    P, G, T = cfg["prompt_len"], cfg["gen_len"], cfg["T"]
    mask = synth.mask_id(cfg)
    seq = np.concatenate([prompt[0], np.full(G, mask)])
    pos = np.arange(P + G)
    t0 = time.perf_counter()
    steps = min(K, T)
    cache = None
    for k in range(steps):
        i = T - k
        c = net.shared(seq, pos)
        if loop.is_refresh(i, T, K):
            cache = net.anchor_cache(c, pos)
        xf = net.denoise(net.fuse(c, cache), pos)
        lg = net.head(xf[P:]).astype(np.float32)
        seq[P:], _, _ = S.reverse_step(lg, seq[P:], mask, loop.unmask_count(G, i, T), P, 0, T - i, 2,
                                       np.float32(1.0))
    dt = time.perf_counter() - t0
    # whole job: B rows x ceil(T/K) such cycles
    job_s = dt * cfg["batch"] * math.ceil(T / K) * (K / steps)
    threads = max([t.get("num_threads", 1) for t in threadpool_info()] + [1])
    return {"value": cfg["batch"] * G / job_s, "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"1 of {cfg['batch']} rows, one refresh cycle ({steps} reverse steps incl. 1 anchor "
                      f"refresh) of the K={K} generation, {dt:.1f} s; scaled by rows x ceil(T/K) cycles"}


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
    tensors = synth.make_weights(cfg, device=dev)
    stream = torch.cuda.current_stream()
    m = tadm.load_model(cfg, tensors, max_batch=B, max_seq=P + G, stream=stream.cuda_stream)
    del tensors
    torch.cuda.empty_cache()
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


if __name__ == "__main__":
    main()
