"""Build librq.so in-tree with hipcc for gfx950 (cross-compiles without a GPU).

    python -m paper_2605_06675_amd.build
"""
import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "librq.so")
BUILD = os.path.join(HERE, "_build")

SOURCES = ["rq_host.cpp", "rq_alloc.cpp", "rq_quant.hip", "rq_attn.hip",
           "rq_calib.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
    # the quantizer decides codes with separately rounded fp32 steps
    "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
]


def _compile(src):
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *COMMON, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def _check_no_calls(src):
    """Kernels must be call-free: device functions are force-inlined (a
    called function that needs long-branch relaxation may reuse its
    return-address registers).  Compile to device assembly and reject any
    call instruction."""
    asm = os.path.join(BUILD, os.path.splitext(src)[0] + ".s")
    cmd = [HIPCC, *COMMON, "--cuda-device-only", "-S", os.path.join(CSRC, src),
           "-o", asm]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc -S failed for {src}:\n{r.stderr}")
    with open(asm) as f:
        if "s_swappc" in f.read():
            raise RuntimeError(f"{src}: device code contains a function call")
    return asm


def build(verbose=False):
    """Compile every source and link librq.so (always rebuilds)."""
    os.makedirs(BUILD, exist_ok=True)
    hip = [s for s in SOURCES if s.endswith(".hip")]
    with concurrent.futures.ThreadPoolExecutor(len(SOURCES) + len(hip)) as ex:
        checks = [ex.submit(_check_no_calls, s) for s in hip]
        objs = list(ex.map(_compile, SOURCES))
        for c in checks:
            c.result()
    tmp = OUT + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, OUT)
    if verbose:
        print("built", OUT)
    return OUT


def clean():
    shutil.rmtree(BUILD, ignore_errors=True)


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
