"""Build libattt.so for gfx950 with hipcc (in-tree, no JIT cache).

    python -m paper_2607_03441_amd.build        # or __graft_entry__.build()
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libattt.so")

DEVICE_SOURCES = ["ngram.hip", "ngram_set.hip", "ce.hip", "ce_fused.hip", "lora.hip", "repetition.hip", "attention.hip", "lora_serve.hip"]
HOST_SOURCES = ["api.cpp"]
ARCH = "gfx950"


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the gfx950 library)")


def _common():
    return ["-O3", "-std=c++17", "-fPIC", "-Wall", "-I", INCLUDE, "-I", CSRC]


def _compile(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    return r.stderr


def build(verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    cc = hipcc()
    jobs = []
    objs = []
    for src in DEVICE_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        # packed fp32 ops stay off: ordinary float code only, no v_pk_*_f32
        cmd = [cc, f"--offload-arch={ARCH}", *_common(), "-Xclang", "-target-feature", "-Xclang",
               "-packed-fp32-ops", "-c", os.path.join(CSRC, src), "-o", obj]
        jobs.append(cmd)
        objs.append(obj)
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        cmd = [cc, *_common(), "-D__HIP_PLATFORM_AMD__", "-c", os.path.join(CSRC, src), "-o", obj]
        jobs.append(cmd)
        objs.append(obj)
    with ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        logs = list(ex.map(_compile, jobs))
    tmp = LIB + ".tmp"
    _compile([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    if verbose:
        for log in logs:
            filtered = "\n".join(l for l in log.splitlines() if "packed-fp32-ops" not in l)
            if filtered.strip():
                print(filtered, file=sys.stderr)
        print(f"built {LIB}", file=sys.stderr)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
