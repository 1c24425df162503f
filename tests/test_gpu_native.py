"""The native driver of the C ABI (paper_2609_37924_amd/tadm_run): whole generations
from C++ without Python in the process, on the tiny (fp32) and small (bf16)
workloads.  The program itself checks that the prompt survives and that every
generated id is a real token, and exits non-zero otherwise."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RUN = os.path.join(ROOT, "paper_2609_37924_amd", "tadm_run")
sys.path.insert(0, ROOT)


@pytest.mark.gpu
@pytest.mark.parametrize("config", ["tiny", "small"])
def test_native_driver_generates(config):
    import bench

    if not os.path.exists(RUN):
        pytest.fail("tadm_run is not built")
    argv = [RUN] + bench.run_args(config, 4) + ["gens=2"]
    print("running", " ".join(argv), flush=True)
    r = subprocess.run(argv, capture_output=True, text=True, timeout=300)
    print(r.stdout[-2000:], r.stderr[-2000:], flush=True)
    assert r.returncode == 0, r.stderr
    assert r.stdout.count("tadm_run: generation ") == 2
    assert ", 0 invalid" in r.stdout


KB = os.path.join(ROOT, "paper_2609_37924_amd", "kernel_bench")


@pytest.mark.gpu
@pytest.mark.parametrize("config", ["small", "block"])
def test_kernel_bench_runs_every_stage(config):
    """kernel_bench launches one denoiser pass's kernels at the workload's shapes (the
    program the hardware counters are taken on); every stage completes and is timed."""
    import bench

    if not os.path.exists(KB):
        pytest.fail("kernel_bench is not built")
    argv = [KB] + bench.run_args(config, 4) + ["reps=2"]
    print("running", " ".join(argv), flush=True)
    r = subprocess.run(argv, capture_output=True, text=True, timeout=300)
    print(r.stdout[-2000:], r.stderr[-2000:], flush=True)
    assert r.returncode == 0, r.stderr
    for stage in ("copy", "qkv", "attn", "oproj", "ffn_up", "ffn_down"):
        assert f"kernel_bench: {stage} " in r.stdout, stage
