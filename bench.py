"""Benchmark: denoised tokens/s of TADM anchor-cache generation on one MI355X.

One step = one whole generation (Algorithm 1 over all T reverse steps, anchor
refreshes included) of a batch of synthetic prompts, enqueued by tadm_generate with
inputs already resident in HBM.  value = B * gen_len / time per step at the headline
refresh interval; the other refresh intervals of the workload are reported beside it.

Prints one JSON line.  Extra fields: the K sweep, per-stage time, a table of the
timed kernels (algorithmic flops or bytes of the schedule over their event-timed
durations), the roofline of the dominant kernel and the CPU oracle timed on a bounded
sample.  The per-kernel table comes from a pass of its own with timers on every
stage; the dominant kernel is then timed again inside the headline timed region, on
its launches of the last generation (each timed launch adds a few microseconds).
Its HBM traffic comes from the committed counter summary of the workload while the
kernel's sources are unchanged since the counters were taken.

--render-stats and --render-counters turn rocprofv3 output into those summaries.
"""
import argparse
import csv
import glob
import hashlib
import json
import math
import os
import re
import sys
import time
from collections import defaultdict

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 vector (the float32 models' products and attention run on the VALU)
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="26b",
                    help="workload: 26b (default, the largest that fits one GPU), 1b, block, small, tiny")
    ap.add_argument("--K", type=int, default=4, help="headline refresh interval")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-sweep", action="store_true", help="only the headline K")
    ap.add_argument("--extras", action="store_true",
                    help="also time the remasking, loop and entropy-bound samplers and the training forward")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle work in the CPU sample")
    ap.add_argument("--out", default=None, help="also write the JSON line to this file")
    ap.add_argument("--render-stats", metavar="DIR", default=None,
                    help="print a markdown summary of the rocprofv3 --stats output under DIR and exit")
    ap.add_argument("--render-counters", nargs="+", metavar="DIR", default=None,
                    help="print per-kernel HBM traffic from two rocprofv3 --pmc runs (FETCH_SIZE, then "
                         "WRITE_SIZE) and, given a third run with MfmaUtil, the MFMA busy share; then exit")
    ap.add_argument("--command", default="", help="command line quoted in a rendered summary")
    ap.add_argument("--run-args", action="store_true",
                    help="print the workload as key=value arguments of the native tadm_run program and exit")
    return ap.parse_args()


# --------------------------------------------------------------- work model ----
# Algorithmic work of one generation per timed kernel stage: flops of each launch
# summed over the schedule of Algorithm 1 (refresh iff (T - i) mod K == 0, one head
# launch per step over the masked rows, block mode with its context passes), and the
# number of launches.  Matrix products count 2 flops per multiply-add; attention counts
# QK^T and PV (4 * L * Lk * head_dim per head); the sampler counts the bytes of one
# read of the masked rows' logits (the bound of an HBM-bound kernel).
def layer_work(cfg, B, L, Lk):
    d, H, Hk, dh, F = (cfg[k] for k in ("d_model", "n_heads", "n_kv_heads", "head_dim", "d_ffn"))
    N = B * L
    glu = 2 if cfg["ffn_kind"] != "gelu" else 1
    return {"qkv": 2.0 * N * d * (H + 2 * Hk) * dh, "attn": 4.0 * B * H * L * Lk * dh,
            "oproj": 2.0 * N * H * dh * d, "ffn_up": 2.0 * N * d * F * glu, "ffn_down": 2.0 * N * F * d}


def schedule_work(cfg, B, K):
    work, launches = defaultdict(float), defaultdict(int)
    d, V = cfg["d_model"], cfg["vocab"]
    P, G, T, bl = cfg["prompt_len"], cfg["gen_len"], cfg["T"], cfg["block_len"]

    def layers(count, L, Lk):
        for name, w in layer_work(cfg, B, L, Lk).items():
            work[name] += count * w
            launches[name] += count

    def fusion(L):
        if cfg["fusion_kind"] == "gated_mlp":  # the paired fusion has no single-kernel stages
            work["fusion1"] += 2.0 * B * L * (2 * d) * (5 * d)
            work["fusion2"] += 2.0 * B * L * (4 * d) * d
            launches["fusion1"] += 1
            launches["fusion2"] += 1

    def step(i, L, Lk):
        ns, na, nd = cfg["n_shared"], cfg["n_anchor"], cfg["n_denoise"]
        if (T - i) % K == 0:
            layers(ns + na, L, Lk)
        layers(ns + nd, L, Lk)
        fusion(L)
        rows = B * ((bl * i) // T)
        work["head"] += 2.0 * rows * d * V
        # bf16: the head samples in its epilogue and the sampler stage merges one
        # 24-byte partial per (row, 64-entry group); fp32: the sampler reads the logits
        work["sample"] += rows * (24.0 * -(-V // 64) if cfg["dtype"] == "bf16" else 4.0 * V)
        launches["head"] += 1
        launches["sample"] += 1

    all_layers = cfg["n_shared"] + cfg["n_anchor"] + cfg["n_denoise"]
    if bl == G:
        for i in range(T, 0, -1):
            step(i, P + G, P + G)
    else:
        layers(all_layers, P, P)  # prompt prefill into the context
        fusion(P)
        ctx = P
        for j in range(G // bl):
            for i in range(T, 0, -1):
                step(i, bl, ctx + bl)
            if j + 1 < G // bl:  # fresh pass appending the finished block
                layers(all_layers, bl, ctx + bl)
                fusion(bl)
                ctx += bl
    return work, launches


# Kernel groups: the stages that launch one kernel on these workloads (the attention
# output and FFN down projections share the residual-epilogue GEMM), the bound, the
# pattern of its rocprofv3 kernel name and the source it is built from.
KERNELS = [
    ("residual-epilogue GEMM (attention output + FFN down projections, bf16 MFMA)", ("oproj", "ffn_down"),
     "mfma", r"gemm_bf16_kernel<.*EpiKind\)2>", "gemm.hip"),
    ("FFN gate/up GEMM with GLU epilogue (bf16 MFMA)", ("ffn_up",), "mfma",
     r"gemm_bf16_kernel<.*EpiKind\)[345]>", "gemm.hip"),
    ("q/k/v GEMM with rotary epilogue (bf16 MFMA)", ("qkv",), "mfma", r"gemm_bf16_kernel<.*EpiKind\)13>",
     "gemm.hip"),
    ("attention (bf16 MFMA)", ("attn",), "mfma", r"attn_bf16_kernel", "attention.hip"),
    ("vocabulary projection with the sampling epilogue (bf16 MFMA + Gumbel-max/normaliser partials)", ("head",),
     "mfma", r"gemm_bf16_kernel<.*EpiKind\)14>", "head_sample.hip"),
    ("fusion GEMM 1 (LN inputs -> hidden + gate, bf16 MFMA)", ("fusion1",), "mfma",
     r"gemm_bf16_kernel<.*EpiKind\)6>", "gemm.hip"),
    ("fusion GEMM 2 (gated residual, bf16 MFMA)", ("fusion2",), "mfma", r"gemm_bf16_kernel<.*EpiKind\)7>",
     "gemm.hip"),
    ("sampler finalize: merge of the group partials into token + confidence", ("sample",), "hbm",
     r"finalize_kernel", "head_sample.hip"),
]


# The fp32 K-slice products of split residual products (the only fp32-output products
# on the bf16 workloads' layer path; the kernel_bench programs run nothing else of that kind)
SLICE_PATTERN = r"gemm_bf16_kernel<(256, 256|128, 128).*EpiKind\)1>"


def kernel_table(cfg, B, K, stages):
    """Per kernel group: time per generation, launches, algorithmic work and roofline."""
    work, launches = schedule_work(cfg, B, K)
    out = []
    for desc, names, bound, _, _ in KERNELS:
        ms = sum(stages[n]["ms_per_step"] for n in names if n in stages)
        n = sum(stages[n]["launches"] for n in names if n in stages)
        w = sum(work[n] for n in names)
        if not n or not w:
            continue
        expect = sum(launches[x] for x in names)
        if bound == "mfma" and cfg["dtype"] != "bf16":  # float32 kernels: VALU arithmetic
            desc, bound = desc.replace("bf16 MFMA", "fp32 VALU"), "alu"
        peak, unit, scale = ((PEAK_BF16_TFLOPS if bound == "mfma" else PEAK_FP32_TFLOPS), "TFLOP/s", 1e12) \
            if bound != "hbm" else (PEAK_HBM_GBS, "GB/s", 1e9)
        achieved = w / (ms / 1e3) / scale
        out.append({"kernel": desc, "stages": list(names), "bound": bound, "ms_per_step": ms,
                    "launches": n, "launches_expected": expect, "achieved": achieved, "peak": peak,
                    "unit": unit, "frac": achieved / peak, "work_per_launch": w / expect})
    return sorted(out, key=lambda r: -r["ms_per_step"])


# the stage launched right before a stage in every layer / step (when it is a stage)
PRED = {"oproj": "attn", "ffn_down": "ffn_up", "attn": "qkv", "fusion2": "fusion1", "sample": "head"}


def source_digest(source):
    """Hash of the sources a kernel is built from: a stored traffic figure is used only
    while it matches."""
    src = os.path.join(ROOT, "paper_2609_37924_amd", "csrc")
    h = hashlib.sha256()
    for f in ("common.h", "kernels.h", "gemm_kernel.h", "sampler_math.h", source):
        with open(os.path.join(src, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_path(config, K):
    return os.path.join(ROOT, "profiles", f"{config}_k{K}_hbm_traffic.md")


TRAFFIC_LINE = re.compile(r"^traffic stage=(\S+) bytes_per_launch=(\S+)(?: mfma_busy=(\S+))? sources=(\S+)$")


def stored_counters(config, K, stage, source):
    """(HBM bytes per launch, MFMA busy %) of a kernel group from the committed counter
    summary of this workload; (None, None) when there is none or the kernel's sources
    changed since (the busy share is None where the summary has none)."""
    path = traffic_path(config, K)
    if not os.path.exists(path):
        return None, None
    with open(path) as f:
        for line in f:
            mt = TRAFFIC_LINE.match(line.strip())
            if mt and mt.group(1) == stage and mt.group(4) == source_digest(source):
                return float(mt.group(2)), (float(mt.group(3)) if mt.group(3) else None)
    return None, None


def stored_traffic(config, K, stage, source):
    """HBM bytes per launch of a kernel from the committed counter summary of this
    workload, or None when there is none or the kernel's sources changed since."""
    return stored_counters(config, K, stage, source)[0]


def attach_counters(config, K, kernels):
    """Per kernel group, the achieved HBM bandwidth (counter bytes per launch x launches
    / stage time) and the MFMA busy share, from the committed counter summary."""
    for r in kernels:
        # by stage: the float32 workloads' rows carry a renamed description
        source = next(k[4] for k in KERNELS if k[1][0] == r["stages"][0])
        b, busy = stored_counters(config, K, r["stages"][0], source)
        if b is not None:
            gbs = b * r["launches"] / (r["ms_per_step"] / 1e3) / 1e9
            r["hbm_bytes_per_launch"], r["hbm_gbs"], r["hbm_frac"] = b, gbs, gbs / PEAK_HBM_GBS
        if busy is not None:
            r["mfma_busy_pct"] = busy
    return kernels


# ------------------------------------------------------------ profile render ---
def short_name(n):
    n = re.sub(r"\(tadm::GemmProblem, tadm::EpiParams\)", "", n)
    n = n.replace("void ", "").replace("tadm::(anonymous namespace)::", "")
    if "gemm" not in n:
        n = re.sub(r"\(.*$", "", n)
    n = n.replace("(tadm::EpiKind)", "epi")
    mt = re.match(r"_ZN4tadm12_GLOBAL__N_1\d+(\w+?)(I|E)", n)
    if mt:
        n = mt.group(1)
    return n[:90]


def render_stats(d, command):
    files = glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True)
    rows = list(csv.DictReader(open(files[0])))
    print("rocprofv3 `--kernel-trace --stats` summary (kernel_stats.csv, every dispatch of the run, top 16 by "
          "total time).  Command, from the repository root on one MI355X:\n")
    print(f"```\n{command}\n```\n")
    print("| kernel | calls | total ms | avg us | % |\n|---|---|---|---|---|")
    for r in rows[:16]:
        print(f"| `{short_name(r['Name'])}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
              f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['Percentage']):.1f} |")


def counter_rows(d, counter):
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    return [r for r in csv.DictReader(open(files[0])) if r["Counter_Name"] == counter]


def render_counter_summary(fetch_dir, write_dir, mfma_dir=None, command=""):
    """HBM traffic per dispatch from FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each
    scaled by the ratio of known bytes to the same counter on copy_kernel (one thread per
    16 bytes, grid = bytes / 16 on these shapes) in the same run."""
    fetch, write = counter_rows(fetch_dir, "FETCH_SIZE"), counter_rows(write_dir, "WRITE_SIZE")

    def scale(rows):
        cp = [r for r in rows if r["Kernel_Name"].startswith("tadm::(anonymous namespace)::copy_kernel(")]
        known = sum(int(r["Grid_Size"]) * 16 for r in cp)
        return known / (sum(float(r["Counter_Value"]) for r in cp) * 1024.0), len(cp)

    sf, ncf = scale(fetch)
    sw, ncw = scale(write)
    per = defaultdict(lambda: [0, 0.0, 0, 0.0])
    for r in fetch:
        e = per[r["Kernel_Name"]]
        e[0] += 1
        e[1] += float(r["Counter_Value"]) * 1024.0 * sf
    for r in write:
        e = per[r["Kernel_Name"]]
        e[2] += 1
        e[3] += float(r["Counter_Value"]) * 1024.0 * sw
    print("HBM traffic per dispatch from two rocprofv3 `--pmc` runs, FETCH_SIZE then WRITE_SIZE (KiB per "
          "dispatch), each scaled by known bytes / counter on copy_kernel of the same run "
          f"(FETCH x{sf:.4f} over {ncf} copies, WRITE x{sw:.4f} over {ncw} copies).  Commands, from the "
          "repository root on one MI355X:\n")
    print(f"```\n{command}\n```\n")
    util = defaultdict(list)
    if mfma_dir:
        for r in counter_rows(mfma_dir, "MfmaUtil"):
            util[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    print("| kernel | dispatches | read MB | written MB | total MB per dispatch | MFMA busy % |\n"
          "|---|---|---|---|---|---|")
    order = sorted(per.items(), key=lambda kv: -(kv[1][1] + kv[1][3]))
    for name, (nf, bf, nw, bw) in order[:16]:
        rd, wr = bf / max(nf, 1) / 1e6, bw / max(nw, 1) / 1e6
        u = f"{sum(util[name]) / len(util[name]):.1f}" if util.get(name) else "-"
        print(f"| `{short_name(name)}` | {nf} | {rd:.3f} | {wr:.3f} | {rd + wr:.3f} | {u} |")
    if mfma_dir:
        print("\nMFMA busy %: rocprofv3's derived MfmaUtil per dispatch (MFMA-busy SIMD cycles over active GPU "
              "cycles x SIMDs), averaged over the kernel's dispatches in a third run.")
    print("\nPer kernel group (the lines bench.py reads; `sources` hashes the group's kernel sources):\n")
    for desc, names, _, pat, source in KERNELS:
        rx = re.compile(pat)
        fk = [r for r in fetch if rx.search(r["Kernel_Name"])]
        wk = [r for r in write if rx.search(r["Kernel_Name"])]
        calls = len(fk)
        if "oproj" in names:
            # a residual product split over K is two kernels, the fp32 slices and their
            # ordered reduction (with or without the RMSNorm that follows): its bytes are
            # both kernels', and it is one launch of the stage (the reduction marks it)
            red = [r for r in fetch if "resid_reduce" in r["Kernel_Name"]]
            if red:
                sx = re.compile(SLICE_PATTERN)
                fk += red + [r for r in fetch if sx.search(r["Kernel_Name"])]
                wk += [r for r in write if "resid_reduce" in r["Kernel_Name"] or sx.search(r["Kernel_Name"])]
                calls += len(red)
        if not fk or len(fk) != len(wk):
            continue
        b = (sum(float(r["Counter_Value"]) for r in fk) * sf + sum(float(r["Counter_Value"]) for r in wk) * sw) \
            * 1024.0 / calls
        # MFMA busy share of the group's products (its dispatches other than a slice reduction)
        busy = [u for n, us in util.items() if rx.search(n) or ("oproj" in names and re.search(SLICE_PATTERN, n))
                for u in us]
        mb = f" mfma_busy={sum(busy) / len(busy):.1f}" if busy else ""
        print(f"    traffic stage={names[0]} bytes_per_launch={b:.0f}{mb} sources={source_digest(source)}")
        print(f"      ({desc}: {calls} launches, {len(fk)} dispatches, {b / 1e6:.3f} MB per launch)")


def run_args(config, K):
    """The workload as key=value arguments of paper_2609_37924_amd/tadm_run, the native
    program that runs generations through the C ABI (no Python in the process)."""
    import synth

    cfg = synth.get_config(config)
    enums = {"ffn_kind": {"gelu": 0, "swiglu": 1, "geglu": 2}, "fusion_kind": {"gated_mlp": 0, "paired": 1},
             "dtype": {"f32": 0, "bf16": 1}}
    keys = ("vocab", "d_model", "n_heads", "n_kv_heads", "head_dim", "d_ffn", "ffn_kind", "n_shared", "n_anchor",
            "n_denoise", "fusion_kind", "fusion_rank", "paired_heads", "dtype", "rms_eps", "ln_eps", "rope_theta",
            "batch", "prompt_len", "gen_len", "block_len", "T")
    out = [f"{k}={enums[k][cfg[k]] if k in enums else cfg[k]}" for k in keys]
    return out + [f"K={K}", f"seed={cfg['sampler_seed']}", f"temperature={cfg['temperature']}"]


def workload_name(cfg):
    return (f"{cfg['name']}: d{cfg['d_model']} {cfg['n_heads']}x{cfg['head_dim']} heads "
            f"({cfg['n_kv_heads']} kv) {cfg['ffn_kind']}{cfg['d_ffn']} V{cfg['vocab']}, "
            f"{cfg['n_anchor']} anchor + {cfg['n_denoise']} denoiser layers, {cfg['fusion_kind']} fusion, "
            f"B={cfg['batch']}, prompt {cfg['prompt_len']} + {cfg['gen_len']} generated "
            f"(block {cfg['block_len']}), T={cfg['T']}")


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(cfg, K, budget_s=10.0):
    """The oracle's own Algorithm 1 (oracle.loop.generate) on whole rows of the workload,
    one row after another until about budget_s seconds have passed (at least one row):
    complete generations, nothing extrapolated.  Rows are independent, so the rate of
    the rows run is the job's rate.  Workloads whose full generation of one row fits
    the budget at every refresh interval (the tiny one) also get each interval's rate."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import synth
    from oracle import loop, network as N

    specs = synth.weight_specs(cfg)
    print("[bench] cpu baseline: building the oracle's float64 weights", file=sys.stderr, flush=True)
    tensors = synth.make_weights(cfg)
    net = N.Network(N.Weights(cfg, [s[0] for s in specs], tensors))
    del tensors
    B, P, G, T, bl = cfg["batch"], cfg["prompt_len"], cfg["gen_len"], cfg["T"], cfg["block_len"]
    prompts = synth.make_prompt(cfg).numpy() if P else np.zeros((B, 0), dtype=np.int64)

    def rate(Kx, budget, done=0, spent=0.0):
        """rows * G / seconds: rows done, done + 1, ... (row r uses prompt r mod B; rows are
        independent, so a short workload repeats them) until `budget` s have passed, counting
        `done` rows already run in `spent` s"""
        t_start = time.perf_counter() - spent
        rows = done
        while rows == 0 or time.perf_counter() - t_start < budget:
            r = rows % B
            loop.generate(net, prompts[r:r + 1], G, T, Kx, bl, cfg["sampler_seed"], cfg["temperature"],
                          synth.mask_id(cfg))
            rows += 1
        el = time.perf_counter() - t_start
        return rows * G / el, rows, el

    # the first row also pays one-off costs (thread pools, first touches); when a row is
    # short it runs once untimed, otherwise it is the first timed row
    t0 = time.perf_counter()
    loop.generate(net, prompts[0:1], G, T, K, bl, cfg["sampler_seed"], cfg["temperature"], synth.mask_id(cfg))
    t_first = time.perf_counter() - t0
    value, rows, el = rate(K, budget_s) if 4 * t_first < budget_s else rate(K, budget_s, 1, t_first)
    per_k = one_thread = None
    k_note = ""
    if el / rows * len(cfg["Ks"]) * 4 < budget_s:  # each interval's rate on its own share of the budget
        per_k = {f"K={Kx}": rate(Kx, budget_s / len(cfg["Ks"]))[0] for Kx in cfg["Ks"]}
        # short rows: also the rate on one thread (the oracle's results do not depend on it)
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            one_thread = rate(K, budget_s / 4)[0]
    elif el / rows <= 40.0:
        # rows of up to ~40 s (the small workload): one complete row at each other interval
        per_k = {f"K={Kx}": value if Kx == K else rate(Kx, 0.0)[0] for Kx in cfg["Ks"]}
        k_note = "; k_sweep: one complete row at each other interval"
    threads = max([t.get("num_threads", 1) for t in threadpool_info()] + [1])
    return {"value": value, "unit": "tokens/s", "cores": threads, "kind": "oracle", "extrapolated": False,
            "cpu_model": cpu_model(), "host_cpus_available": len(os.sched_getaffinity(0)),
            "k_sweep": per_k, "one_thread": one_thread,
            "sample": f"{rows} rows (prompts of the workload's {B}, in turn), each a complete generation by the "
                      f"oracle's Algorithm 1 at K={K} ({G} positions, T={T}), {el:.1f} s in all; rate of those rows "
                      f"(rows are independent){k_note}"}


STREAM_HEAD_ROWS = 16384  # vocabulary rows of the head in the streamed sample


def cpu_baseline_streamed(cfg, K, tensors, budget_s=20.0):
    """The oracle on a bounded sample of a workload whose float64 weights do not fit
    (or take minutes to build on) the host: one transformer layer (the first anchor
    layer, at the real per-row shape of one call: one block, or the whole canvas, with
    its context keys), the fusion module, the vocabulary head on its first
    STREAM_HEAD_ROWS rows and the reverse step on a few masked positions, each timed by
    itself on one batch row.  A whole generation is then extrapolated from those times
    over Algorithm 1's schedule: per block, ceil(T/K) refresh steps (anchor layers) and
    T steps of denoiser layers, fusion, head and sampler over the positions still
    masked, the prompt prefill and block appends as fresh passes; times the batch
    (rows are independent).  Layer times are taken at the first block's context length;
    the embedding gather is not timed.  The result is labelled as extrapolated."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import synth
    from oracle import network as N, sampler as S

    B, P, G, T, bl, V, d = (cfg[k] for k in ("batch", "prompt_len", "gen_len", "T", "block_len", "vocab",
                                               "d_model"))
    Hkv, dh = cfg["n_kv_heads"], cfg["head_dim"]
    single = bl == G
    L = P + G if single else bl
    ctx_len = 0 if single else P
    li = cfg["n_shared"]
    names = list(tensors)
    W = N.Weights(cfg, names, [tensors[n] for n in names])
    rng = np.random.default_rng(cfg["input_seed"])
    pos = np.arange(ctx_len, ctx_len + L)
    ctx = None
    if ctx_len:  # context K (rotary applied) and V of the prompt, random values of the right shape
        ctx = (rng.standard_normal((ctx_len, Hkv, dh)), rng.standard_normal((ctx_len, Hkv, dh)))
    x = rng.standard_normal((L, d)) * 0.02
    t_start = time.perf_counter()

    # every piece once, then again until the budget is spent; each piece keeps its best time
    best = {}

    def timed(key, fn):
        t0 = time.perf_counter()
        out = fn()
        dt = time.perf_counter() - t0
        best[key] = min(best.get(key, dt), dt)
        return out

    n_s = 4
    cv = np.full(n_s, synth.mask_id(cfg), dtype=np.int64)
    rounds = 0
    while rounds == 0 or time.perf_counter() - t_start < budget_s:
        h, _ = timed("layer", lambda: N.transformer_layer(W, li, x, pos, ctx))
        ht = timed("fusion", lambda: N.fuse(W, x, {"h": h, "c": x + 0.01}))
        xf = N.rms_norm(ht, W["final_norm"], cfg["rms_eps"])
        lg_part = timed("head", lambda: N.operand(cfg, xf) @ W["w_out"].T)
        # the reverse step on full-width logit rows, drawn like the head's output
        lg = (rng.standard_normal((n_s, V)) * float(lg_part.std())).astype(np.float32)
        timed("sampler", lambda: S.reverse_step(lg, cv, synth.mask_id(cfg), 1, ctx_len, 0, 0,
                                                cfg["sampler_seed"], np.float32(1.0)))
        rounds += 1
    t_layer, t_fuse = best["layer"], best["fusion"]
    t_head_row = best["head"] * (V / W["w_out"].shape[0]) / L
    t_samp_row = best["sampler"] / n_s
    sample_s = time.perf_counter() - t_start
    # extrapolation over the schedule (one row)
    La, Ld, Ls = cfg["n_anchor"], cfg["n_denoise"], cfg["n_shared"]
    n_ref = math.ceil(T / K)
    per_block = 0.0
    for i in range(T, 0, -1):
        masked = (G if single else bl) * i // T
        per_block += (Ls + Ld) * t_layer + t_fuse + masked * (t_head_row + t_samp_row)
    per_block += n_ref * La * t_layer
    n_blocks = G // bl
    fresh = (Ls + La + Ld) * t_layer + t_fuse  # a fresh pass over one block's positions
    extra = 0.0 if single else (P / bl) * fresh + (n_blocks - 1) * fresh
    row_s = n_blocks * per_block + extra
    job_s = B * row_s
    threads = max([t.get("num_threads", 1) for t in threadpool_info()] + [1])
    return {"value": B * G / job_s, "unit": "tokens/s", "cores": threads, "kind": "oracle", "extrapolated": True,
            "cpu_model": cpu_model(), "host_cpus_available": len(os.sched_getaffinity(0)),
            "per_row_ms": {"layer": 1e3 * t_layer, "fusion": 1e3 * t_fuse, "head_per_position": 1e3 * t_head_row,
                           "sampler_per_position": 1e3 * t_samp_row},
            "sample": f"EXTRAPOLATED from a layer-streamed sample ({sample_s:.1f} s of oracle work, {rounds} rounds, "
                      f"best of each): one transformer "
                      f"layer on one row of {L} positions with {ctx_len} context keys ({1e3 * t_layer:.0f} ms), the "
                      f"{cfg['fusion_kind']} fusion ({1e3 * t_fuse:.0f} ms), the head on {W['w_out'].shape[0]} of "
                      f"{V} vocabulary rows (scaled), the reverse step on {n_s} masked positions; "
                      f"scaled to B={B} rows x {n_blocks} blocks x ({n_ref} refresh + {T} denoiser steps), "
                      f"prefill and appends as fresh passes; the real weights of those tensors, context K/V and "
                      f"layer inputs random of the right shape; embedding gather not timed"}


def main():
    args = parse()
    if args.render_stats:
        render_stats(args.render_stats, args.command)
        return
    if args.render_counters:
        render_counter_summary(*args.render_counters[:3], command=args.command)
        return
    if args.run_args:
        print(" ".join(run_args(args.config, args.K)))
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the path runs on a single MI355X "
              "(sharding over several GPUs is described, not implemented).", file=sys.stderr)
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
    # the layer-streamed oracle sample of the large workloads keeps float64 host copies of
    # the tensors it runs: the fusion, the final norm, the first anchor layer and the first
    # STREAM_HEAD_ROWS rows of the vocabulary head
    streamed = {} if (not args.no_cpu and cfg["dtype"] == "bf16" and cfg["d_model"] >= 2048) else None
    keep_layer = f"layer{cfg['n_shared']}."
    for i, spec in enumerate(synth.weight_specs(cfg)):  # one tensor at a time: bounded memory
        t = synth.make_tensor(cfg, i, spec, device=dev)
        tadm.tadm_model_load_weight(m, i, t)
        if streamed is not None and (spec[0].startswith(("fusion.", keep_layer)) or spec[0] in ("final_norm", "w_out")):
            src = t[:STREAM_HEAD_ROWS] if spec[0] == "w_out" else t
            streamed[spec[0]] = src.to(torch.float64).cpu().numpy()
        del t
    torch.cuda.empty_cache()
    print(f"[bench] weights generated and loaded in {time.perf_counter() - t_load:.1f} s", file=sys.stderr,
          flush=True)
    prompt = synth.make_prompt(cfg, device=dev) if P else None
    out = torch.empty(B, P + G, dtype=torch.int32, device=dev)

    sampler = [None]  # None: confidence-ranked (the headline); else a tadm_sampler

    T_run = [T]

    def gen(K):
        tadm.tadm_generate_sampler(m, prompt, B, P, G, T_run[0], K, bl, cfg["sampler_seed"], cfg["temperature"],
                                   sampler[0], out)

    def timed(K, steps, warmup, profile=0, profiled_steps=None):
        """Time `steps` generations.  profile: stage bit mask timed during the last
        `profiled_steps` of them (all by default); the timers add a little GPU time per
        timed launch, so the headline pass times only its last generation."""
        profiled_steps = steps if profiled_steps is None else profiled_steps
        for _ in range(warmup):
            gen(K)
        torch.cuda.synchronize()
        tadm.tadm_profile_reset(m)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record(stream)
        for k in range(steps):
            if k == steps - profiled_steps:
                tadm.tadm_profile_enable(m, profile)
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
                    stages[name] = {"ms_per_step": tot / profiled_steps, "launches": n // profiled_steps,
                                    "avg_ms": tot / n}
        return ms, wall / steps * 1e3, stages

    K0 = args.K
    tokens = B * G
    # passes other than the headline (the stage table, the other refresh intervals): half
    # the headline's generations, at most 3 on the workloads whose generations take seconds
    long_gen = T * (P + G) >= 2 ** 16
    n_aux = max(1, args.steps // 2)
    if long_gen:
        n_aux = min(n_aux, 3)
    print(f"[bench] {workload_name(cfg)}", file=sys.stderr, flush=True)
    # 1. per-stage breakdown (HIP events around every stage, so a pass of its own)
    _, _, stages = timed(K0, n_aux, min(args.warmup, 1) if long_gen else args.warmup, profile=-1)
    kernels = attach_counters(args.config, K0, kernel_table(cfg, B, K0, stages))
    for k in kernels:
        print(f"[bench]   {k['ms_per_step']:8.3f} ms  {k['achieved']:8.1f} {k['unit']:7s} ({100 * k['frac']:.1f}% "
              f"of peak)  {k['launches']} launches  {k['kernel']}", file=sys.stderr, flush=True)
    # 2. headline; the dominant kernel's launches of its last generation carry timers,
    # and so do the launches right before them (a kernel timed after an untimed one is
    # charged part of its predecessor's tail)
    dom = kernels[0] if kernels else None
    timed_stages = set(dom["stages"]) | {PRED[n] for n in dom["stages"] if n in PRED} if dom else set()
    mask = sum(1 << tadm.STAGES.index(n) for n in timed_stages)
    ms, wall_ms, dom_stages = timed(K0, args.steps, 1, profile=mask, profiled_steps=1)
    value = tokens / (ms / 1e3)
    print(f"[bench] K={K0}: {ms:.3f} ms/generation ({wall_ms:.3f} wall) -> {value:.1f} tokens/s",
          file=sys.stderr, flush=True)
    sweep = {f"K={K0}": {"tokens_per_s": value, "ms_per_step": ms}}
    if not args.no_sweep:
        for K in cfg["Ks"]:
            if K == K0:
                continue
            kms, _, _ = timed(K, n_aux, 0 if long_gen else 1)
            sweep[f"K={K}"] = {"tokens_per_s": tokens / (kms / 1e3), "ms_per_step": kms}
            print(f"[bench] K={K}: {kms:.3f} ms -> {tokens / (kms / 1e3):.1f} tokens/s", file=sys.stderr,
                  flush=True)
    # per-step timing on canvases at random times (the 1B-class workload's per-step leg):
    # t_b ~ U(0,1) per row, i_b = ceil(t_b T), floor(M0 i_b / T) positions masked; an anchor
    # refresh on the canvas, then stale steps (S, fusion, D, head, reverse step) with each
    # row's own unmask count
    per_step = None
    if cfg["name"] == "1b":
        canvas, steps_b = synth.make_timing_canvas(cfg, T)
        d_canvas = canvas.to(dev)
        n_rows = torch.tensor([tadm.tadm_unmask_count(G, i, T) for i in steps_b], dtype=torch.int32, device=dev)
        cache = tadm.tadm_cache_create(m, B, P + G)
        nxt = torch.empty_like(d_canvas)
        sargs = tadm.step_args(T // 2, T, 0, 7, cfg["sampler_seed"], 1.0, n_unmask_rows=n_rows)
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        tadm.tadm_anchor_forward(m, None, d_canvas, B, P + G, T, T, cache)
        tadm.tadm_denoise_step(m, None, d_canvas, B, P + G, P, cache, sargs, None, nxt)
        torch.cuda.synchronize()
        reps = max(3, args.steps)
        e0.record(stream)
        for _ in range(reps):
            tadm.tadm_anchor_forward(m, None, d_canvas, B, P + G, T, T, cache)
        e1.record(stream)
        for _ in range(reps):
            tadm.tadm_denoise_step(m, None, d_canvas, B, P + G, P, cache, sargs, None, nxt)
        e2.record(stream)
        torch.cuda.synchronize()
        a_ms, s_ms = e0.elapsed_time(e1) / reps, e1.elapsed_time(e2) / reps
        masked = int(sum((G * i) // T for i in steps_b))
        per_step = {"canvas": f"B={B} x {P + G} positions at t_b ~ U(0,1), {masked} masked in all",
                    "anchor_refresh_ms": a_ms, "stale_step_ms": s_ms,
                    "stale_step_tokens_per_s": B * (P + G) / (s_ms / 1e3),
                    "what": "a stale step processes every position of the canvas; the head and sampler run on "
                            "the masked ones"}
        tadm.tadm_cache_destroy(cache)
        print(f"[bench] random-t canvases: anchor refresh {a_ms:.3f} ms, stale step {s_ms:.3f} ms",
              file=sys.stderr, flush=True)
    # the remasking posterior (capped sigma, eta = 0.04) without and with the nucleus p = 0.9
    # of the paper's ReMDM-Cap runs
    remask = None
    if args.extras:
        remask = {}
        for top_p in (0.0, 0.9):
            sampler[0] = tadm.remask_sampler(0.04, top_p)
            rms, _, _ = timed(K0, max(2, args.steps // 2), 1)
            key = f"eta=0.04,top_p={top_p or 1.0}"
            remask[key] = {"K": K0, "tokens_per_s": tokens / (rms / 1e3), "ms_per_step": rms}
            print(f"[bench] remasking sampler {key}, K={K0}: {rms:.3f} ms -> {tokens / (rms / 1e3):.1f} tokens/s",
                  file=sys.stderr, flush=True)
        # ReMDM-Loop, the paper's sampler when the step budget reaches the generation
        # length: T = block length, eta = 0.02, t_on = 0.55, t_off = 0.05, alpha_on = 0.9
        sampler[0] = tadm.loop_sampler(0.02, 0.55, 0.05, 0.9, 0.9)
        T_run[0] = max(T, bl)
        gen(K0)  # warm-up, reported so that a long generation is not taken for a hang
        torch.cuda.synchronize()
        print(f"[bench] remasking sampler loop, T={T_run[0]}: warm-up generation done", file=sys.stderr, flush=True)
        rms, _, _ = timed(K0, 1, 0)
        key = f"loop,T={T_run[0]},eta=0.02,top_p=0.9"
        remask[key] = {"K": K0, "T": T_run[0], "tokens_per_s": tokens / (rms / 1e3), "ms_per_step": rms}
        print(f"[bench] remasking sampler {key}, K={K0}: {rms:.3f} ms -> {tokens / (rms / 1e3):.1f} tokens/s",
              file=sys.stderr, flush=True)
        T_run[0] = T
        # the entropy-bound sampler of uniform-state diffusion (eta = 0.1, tau 0.8 -> 0.4,
        # T = 48, self-conditioning) at the refresh intervals the paper pairs with it
        sampler[0] = tadm.entropy_sampler(0.1, 0.8, 0.4)
        T_run[0] = 48
        for K in (1, 2, 3):
            rms, _, _ = timed(K, 2, 1)
            key = f"entropy,T=48,eta=0.1,K={K}"
            remask[key] = {"K": K, "T": 48, "tokens_per_s": tokens / (rms / 1e3), "ms_per_step": rms}
            print(f"[bench] entropy-bound sampler T=48, K={K}: {rms:.3f} ms -> {tokens / (rms / 1e3):.1f} tokens/s",
                  file=sys.stderr, flush=True)
        T_run[0] = T
        sampler[0] = None
    # the pretraining objective's forward pass (stale pair, anchor on z_t', denoiser on
    # z_t, 1/t-weighted masked cross-entropy) over B sequences of P + G tokens
    train_line = None
    if args.extras:
        Ltr = P + G
        xtr = torch.randint(0, cfg["vocab"], (B, Ltr), generator=torch.Generator().manual_seed(5),
                            dtype=torch.int32).to(dev)
        tt, tts, _, _, _ = tadm.tadm_stale_times(B, 11, 0, 1e-3)
        d_t, d_ts = torch.from_numpy(tt).to(dev), torch.from_numpy(tts).to(dev)
        loss = torch.empty(B, device=dev)
        for _ in range(2):
            tadm.tadm_train_loss(m, xtr, B, Ltr, d_t, d_ts, 1e-3, 11, 0, loss)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = max(3, args.steps)
        e0.record(stream)
        for r in range(reps):
            tadm.tadm_train_loss(m, xtr, B, Ltr, d_t, d_ts, 1e-3, 11, r, loss)
        e1.record(stream)
        torch.cuda.synchronize()
        tms = e0.elapsed_time(e1) / reps
        train_line = {"tokens_per_s": B * Ltr / (tms / 1e3), "ms_per_batch": tms, "batch": B, "seq_len": Ltr,
                      "what": "forward of the T-ANELBO objective (gamma = 0), no backward"}
        print(f"[bench] training objective forward, {B}x{Ltr} tokens: {tms:.3f} ms -> "
              f"{B * Ltr / (tms / 1e3):.1f} tokens/s", file=sys.stderr, flush=True)
    roof = None
    if dom and cfg["dtype"] != "bf16":
        # the float32 tiny workload is a latency measurement (a few 10 us kernels per step,
        # on the VALU path): it has no roofline target
        roof = {"bound": "latency", "note": "float32 tiny workload: latency per generation only, no roofline target",
                "achieved": None, "peak": None, "unit": None, "frac": None, "traffic": None}
        dom = None
    if dom:
        live = next(r for r in kernel_table(cfg, B, K0, dom_stages) if r["kernel"] == dom["kernel"])
        source = next(k[4] for k in KERNELS if k[1][0] == dom["stages"][0])
        traffic = stored_traffic(args.config, K0, dom["stages"][0], source)
        avg_ms = live["ms_per_step"] / live["launches"]
        roof = {"kernel": live["kernel"], "bound": live["bound"], "achieved": live["achieved"],
                "peak": live["peak"], "unit": live["unit"], "frac": live["frac"], "traffic": traffic,
                "avg_launch_ms": avg_ms, "launches_per_step": live["launches"],
                "timed_in": "the last generation of the headline timed region",
                ("flops_per_launch" if live["bound"] == "mfma" else "bytes_per_launch"): live["work_per_launch"]}
    cpu = None
    if not args.no_cpu:
        try:
            if streamed is not None:
                cpu = cpu_baseline_streamed(cfg, K0, streamed, args.cpu_budget)
            else:
                cpu = cpu_baseline(cfg, K0, args.cpu_budget)
        except Exception as e:  # the GPU number stands on its own
            print(f"[bench] cpu baseline skipped: {e}", file=sys.stderr)
            cpu = {"value": None, "unit": "tokens/s", "kind": "oracle", "skipped": str(e)}
    tadm.tadm_model_destroy(m)
    line = {
        "metric": f"denoised tokens/s per MI355X at K={K0} (vs K=1 in k_sweep)",
        "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg["dtype"], "data": "synthetic (uniform-random prompts, seeded random-init weights)",
        "config": {"workload": workload_name(cfg), "global_batch": B, "seq_len": P + G, "K": K0,
                   "parallelism": "none (1 GPU)"},
        "k_sweep": sweep,
        "k4_over_k1": (sweep["K=4"]["tokens_per_s"] / sweep["K=1"]["tokens_per_s"]
                       if "K=4" in sweep and "K=1" in sweep else None),
        "latency_ms_per_generation": {k: v["ms_per_step"] for k, v in sweep.items()},
        "per_step_random_t": per_step,
        "samplers": remask,
        "train_forward": train_line,
        "stages_ms_per_step": {k: v["ms_per_step"] for k, v in stages.items()},
        "kernels": [{k: v for k, v in r.items() if k != "stages"} for r in kernels],
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(json.dumps(line) + "\n")


if __name__ == "__main__":
    main()
