"""Build librq.so in-tree with hipcc for gfx950 (cross-compiles without a GPU).

    python -m paper_2605_06675_amd.build
"""
import concurrent.futures
import os
import re
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "librq.so")
BUILD = os.path.join(HERE, "_build")

SOURCES = ["rq_host.cpp", "rq_alloc.cpp", "rq_codebook.cpp"] + sorted(
    f for f in os.listdir(CSRC) if f.endswith(".hip"))

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
    # the quantizer decides codes with separately rounded fp32 steps
    "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # keep each atomic as written: the atomic optimizer turns a uniform-
    # address atomic into a single-lane one whose result is broadcast at
    # once, which waits for it where the attention kernel means to overlap
    "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
]


def _compile(src):
    """Compile one source; for HIP sources keep the device assembly
    (-save-temps) and reject any call instruction in it: device functions
    are force-inlined (a called function that needs long-branch relaxation
    may reuse its return-address registers)."""
    stem = os.path.splitext(src)[0]
    obj = os.path.join(BUILD, stem + ".o")
    cmd = [HIPCC, *COMMON, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".hip"):
        cmd.insert(-4, "-save-temps=obj")
    r = subprocess.run(cmd, capture_output=True, text=True, cwd=BUILD)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    if src.endswith(".hip"):
        asm = [f for f in os.listdir(BUILD)
               if f.startswith(stem + "-hip-amdgcn") and f.endswith(".s")]
        if not asm:
            raise RuntimeError(f"{src}: device assembly not found")
        with open(os.path.join(BUILD, asm[0])) as f:
            text = f.read()
        if "s_swappc" in text:
            raise RuntimeError(f"{src}: device code contains a function call")
        if src.startswith("rq_attn"):
            _check_claim_registers(src, text)
    return obj


_VREG = re.compile(r"\bv(\d+)\b|\bv\[(\d+):(\d+)\]")
_CLAIM_REGS = {166, 167}


def _check_claim_registers(src, text):
    """The attention kernels keep their block claims in v[166:167], written
    and read only by inline assembly: reject code in which the compiler
    itself uses one of those registers."""
    in_asm = False
    for line in text.split("\n"):
        t = line.strip()
        if t.startswith(";;#ASMSTART"):
            in_asm = True
        elif t.startswith(";;#ASMEND"):
            in_asm = False
        elif not in_asm and line.startswith("\t") and t and t[0] not in ".;":
            for m in _VREG.finditer(t.split(";")[0]):
                lo = int(m.group(1) or m.group(2))
                hi = int(m.group(1) or m.group(3))
                if _CLAIM_REGS & set(range(lo, hi + 1)):
                    raise RuntimeError(f"{src}: compiler-generated use of a "
                                       f"claim register: {t}")


def build(verbose=False):
    """Compile every source and link librq.so (always rebuilds)."""
    os.makedirs(BUILD, exist_ok=True)
    # the attention variants for widths up to 8 instantiate the most
    # kernels: start them first, they bound the wall time
    order = sorted(SOURCES, key=lambda f: (0 if "_b8" in f else 1, f))
    with concurrent.futures.ThreadPoolExecutor(os.cpu_count() or 8) as ex:
        objs = list(ex.map(_compile, order))
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
