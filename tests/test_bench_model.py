"""The benchmark's work model and its command-line contract, on the CPU.

The per-kernel rates in the benchmark line are algorithmic work divided by measured
time, so the work model is checked here against what the paper fixes: the number of
transformer-layer calls of Algorithm 1 (the anchor network on ceil(T/K) of the T
steps of a block, the denoiser on every step; eq. anchor-cache-compute), the rows the
head sees (the positions still masked under the linear schedule), and the flops of a
matrix product (2 per multiply-add).  Block mode adds one fresh pass for the prompt
and one per finished block but the last (App. C.1 encoder / decoder split).
"""
import math
import os
import subprocess
import sys

import pytest

import bench
import synth

CONFIGS = ["tiny", "small", "block", "1b", "26b"]


def layer_calls(cfg, K):
    """Transformer-layer calls of one row's generation, written from Algorithm 1."""
    LS, LA, LD = cfg["n_shared"], cfg["n_anchor"], cfg["n_denoise"]
    T, G, bl = cfg["T"], cfg["gen_len"], cfg["block_len"]
    blocks = G // bl
    per_block = math.ceil(T / K) * (LS + LA) + T * (LS + LD)
    passes = 0 if bl == G else blocks  # the prompt prefill, then blocks - 1 appends
    return blocks * per_block + passes * (LS + LA + LD)


@pytest.mark.parametrize("name", CONFIGS)
def test_layer_launches_follow_algorithm_1(name):
    cfg = synth.get_config(name)
    for K in cfg["Ks"]:
        work, launches = bench.schedule_work(cfg, cfg["batch"], K)
        expect = layer_calls(cfg, K)
        for stage in ("qkv", "attn", "oproj", "ffn_up", "ffn_down"):
            assert launches[stage] == expect, (name, K, stage)


def test_layer_calls_reproduce_table_2():
    """The model's count for TADM:Pretraining's 6 + 12 split at the T, K pairs the
    paper prints (Table 2: 1536, 6144, 7680, 18432, 36864)."""
    cfg = dict(synth.get_config("small"), n_shared=0, n_anchor=12, n_denoise=6, prompt_len=0, gen_len=1024,
               block_len=1024)
    for T, K, calls in [(128, 2, 1536), (512, 2, 6144), (1024, 8, 7680), (2048, 4, 18432), (4096, 4, 36864)]:
        assert layer_calls(dict(cfg, T=T), K) == calls
        _, launches = bench.schedule_work(dict(cfg, T=T), 1, K)
        assert launches["ffn_up"] == calls


@pytest.mark.parametrize("name", CONFIGS)
def test_head_rows_follow_the_schedule(name):
    """One head launch per reverse step, over the positions still masked before it:
    floor(M0 i / T) of each block's M0 = block_len positions at step i (R11)."""
    cfg = synth.get_config(name)
    B, T, G, bl, d, V = (cfg[k] for k in ("batch", "T", "gen_len", "block_len", "d_model", "vocab"))
    K = cfg["Ks"][0]
    work, launches = bench.schedule_work(cfg, B, K)
    rows = (G // bl) * sum(B * ((bl * i) // T) for i in range(1, T + 1))
    assert launches["head"] == (G // bl) * T
    assert work["head"] == pytest.approx(2.0 * rows * d * V, rel=1e-12)


@pytest.mark.parametrize("name", CONFIGS)
def test_product_flops_are_two_per_multiply_add(name):
    """Per launch of a single-canvas denoiser pass (or a block-mode step), each layer
    product counts 2 M N K with M = rows x positions of the pass; attention counts the
    two products QK^T and PV, 4 L L_k d_h per head."""
    cfg = synth.get_config(name)
    B = cfg["batch"]
    d, H, Hk, dh, F = (cfg[k] for k in ("d_model", "n_heads", "n_kv_heads", "head_dim", "d_ffn"))
    L, Lk = 37, 91
    w = bench.layer_work(cfg, B, L, Lk)
    M = B * L
    up_rows = F if cfg["ffn_kind"] == "gelu" else 2 * F  # gated FFNs multiply gate and up rows
    assert w["qkv"] == 2.0 * M * d * (H + 2 * Hk) * dh
    assert w["oproj"] == 2.0 * M * (H * dh) * d
    assert w["ffn_up"] == 2.0 * M * d * up_rows
    assert w["ffn_down"] == 2.0 * M * F * d
    assert w["attn"] == 4.0 * B * H * L * Lk * dh


def test_bench_refuses_several_gpus(root):
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       cwd=root, timeout=120)
    assert r.returncode == 2
    assert "single" in r.stderr and r.stdout == ""


def test_bench_prints_native_driver_arguments(root):
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--config", "block", "--run-args"],
                       capture_output=True, text=True, cwd=root, timeout=120)
    assert r.returncode == 0
    kv = dict(a.split("=", 1) for a in r.stdout.split())
    cfg = synth.get_config("block")
    assert int(kv["batch"]) == cfg["batch"] and int(kv["block_len"]) == cfg["block_len"]
    assert int(kv["n_kv_heads"]) == cfg["n_kv_heads"] and int(kv["vocab"]) == cfg["vocab"]


@pytest.mark.parametrize("name", ["tiny"] + CONFIGS)
def test_kernel_table_takes_counters_for_every_workload(name):
    """The per-kernel table and its counter fields build for every workload, the float32
    one included (its rows are described as VALU kernels, so counters are looked up by
    stage); a stored figure is attached only where the committed summary matches."""
    cfg = synth.get_config(name)
    K = cfg["Ks"][0]
    _, launches = bench.schedule_work(cfg, cfg["batch"], K)
    stages = {s: {"ms_per_step": 1.0 + i, "launches": n} for i, (s, n) in enumerate(sorted(launches.items())) if n}
    rows = bench.attach_counters(name, K, bench.kernel_table(cfg, cfg["batch"], K, stages))
    assert rows
    for r in rows:
        src = next(k[4] for k in bench.KERNELS if k[1][0] == r["stages"][0])
        b, busy = bench.stored_counters(name, K, r["stages"][0], src)
        assert r.get("hbm_bytes_per_launch") == b
        assert r.get("mfma_busy_pct") == busy
        if b is not None:
            assert r["hbm_gbs"] == pytest.approx(b * r["launches"] / (r["ms_per_step"] / 1e3) / 1e9)
