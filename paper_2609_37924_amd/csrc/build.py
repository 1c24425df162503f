"""Builds libtadm.so (gfx950) from the HIP sources next to this file.

Usage: python build.py [--jobs N].  Each source compiles to an object with hipcc
(-O3, --offload-arch=gfx950, packed-fp32 instructions disabled); the samplers and
the vocabulary projection with the sampling epilogue are compiled without
floating-point contraction and with correctly rounded division, so that their
float32 arithmetic is exactly the documented sequence of rounded operations.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
SOURCES = ["runtime.hip", "gemm.hip", "attention.hip", "norm.hip", "sampler.hip", "head_sample.hip", "fusion.hip",
           "usdm.hip", "train.hip"]
CONTRACT = ["-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt"]
EXTRA = {"sampler.hip": CONTRACT, "head_sample.hip": CONTRACT, "usdm.hip": CONTRACT, "train.hip": CONTRACT}
OUT = os.path.join(PKG, "libtadm.so")


def hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return "hipcc"


def flags():
    return ["--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-result",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include"), "-I", HERE]


def compile_one(src, objdir):
    obj = os.path.join(objdir, src.replace(".hip", ".o"))
    cmd = [hipcc(), "-c", os.path.join(HERE, src), "-o", obj] + flags() + EXTRA.get(src, [])
    r = subprocess.run(cmd, capture_output=True, text=True)
    errs = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                     if "packed-fp32-ops" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{errs}")
    return obj, errs


def build(jobs=8, verbose=False):
    objdir = os.path.join(ROOT, "_build")
    os.makedirs(objdir, exist_ok=True)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        results = list(ex.map(lambda s: compile_one(s, objdir), SOURCES))
    if verbose:
        for _, e in results:
            if e:
                print(e)
    tmp = OUT + ".tmp"
    cmd = [hipcc(), "-shared", "-o", tmp, "--offload-arch=gfx950"] + [o for o, _ in results] + \
        ["-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-Wl,-rpath,/opt/rocm/lib"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(tmp, OUT)
    build_run()
    return OUT


# Native programs linked against the library next to them: tadm_run (whole generations
# through the C ABI) and kernel_bench (one denoiser pass's kernels through the library's
# launchers, the program hardware counters are taken on).
PROGRAMS = ["tadm_run", "kernel_bench"]
RUN_OUT = os.path.join(PKG, "tadm_run")


def build_run():
    for name in PROGRAMS:
        out = os.path.join(PKG, name)
        tmp = out + ".tmp"
        cmd = [hipcc(), os.path.join(HERE, name + ".hip"), "-o", tmp] + flags() + \
            ["-L", PKG, "-l:libtadm.so", "-Wl,-rpath,$ORIGIN"]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {name}.hip:\n" + r.stderr)
        os.replace(tmp, out)
    return RUN_OUT


# Host-side sanitizer build: the same sources with the host code instrumented by
# AddressSanitizer and UndefinedBehaviorSanitizer (the device code is not), for running
# the library's argument validation on the CPU under the sanitizers.
SAN_OUT = os.path.join(ROOT, "_build", "san", "libtadm_san.so")
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-omit-frame-pointer"]


def build_host_sanitized(jobs=8):
    objdir = os.path.join(ROOT, "_build", "san")
    os.makedirs(objdir, exist_ok=True)

    def one(src):
        obj = os.path.join(objdir, src.replace(".hip", ".o"))
        cmd = [hipcc(), "-c", os.path.join(HERE, src), "-o", obj] + flags() + EXTRA.get(src, []) + SAN_FLAGS
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc (host sanitizers) failed on {src}:\n{r.stderr}")
        return obj

    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(one, SOURCES))
    cmd = [hipcc(), "-shared", "-o", SAN_OUT, "--offload-arch=gfx950"] + objs + SAN_FLAGS + \
        ["-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-Wl,-rpath,/opt/rocm/lib"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link (host sanitizers) failed:\n" + r.stderr)
    return SAN_OUT


if __name__ == "__main__":
    jobs = int(sys.argv[sys.argv.index("--jobs") + 1]) if "--jobs" in sys.argv else 8
    print(build(jobs, verbose=True))
    if "--sanitize" in sys.argv:
        print(build_host_sanitized(jobs))
