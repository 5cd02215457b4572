"""In-tree build of libsr.so for gfx950 (hipcc).  ``python -m paper_2607_02829_amd.build``."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
OUT = os.path.join(HERE, "libsr.so")
BUILD = os.path.join(ROOT, "_build")

SOURCES = ["select.hip", "routing.hip", "rowops.hip", "gemv.hip", "gemm.hip", "attention.hip", "cross_attention.hip",
           "edm.hip", "stack.cpp", "api.cpp", "profile.cpp"]
# Files whose floating-point results are part of a bit-exact contract (top-k score,
# scatter rounding): no multiply-add contraction anywhere in them.
NO_CONTRACT = {"select.hip", "routing.hip"}
# Files whose arithmetic never meets a NaN (softmax of finite scores, -inf masks): max/min
# without NaN canonicalisation.
NO_NANS = {"attention.hip"}
# Files whose kernels read LDS fragments with inline assembly: their gfx950 assembly is kept
# and checked (isa_scan) for registers touched while such a read is in flight.
ASYNC_READS = {"attention.hip", "gemm.hip"}

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    # packed fp32 arithmetic stays off (its instructions are not generated)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src + ".o")
    cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if src in NO_CONTRACT:
        cmd.insert(1, "-ffp-contract=off")
    if src in NO_NANS:
        cmd.insert(1, "-fno-honor-nans")
    if src in ASYNC_READS:
        cmd.insert(1, "-save-temps=obj")
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    return obj


def device_asm_path(src: str) -> str:
    """Where build() keeps the gfx950 assembly of an ASYNC_READS source."""
    return os.path.join(BUILD, os.path.splitext(src)[0] + "-hip-amdgcn-amd-amdhsa-gfx950.s")


def check_async_reads() -> dict:
    """Kernels of the ASYNC_READS sources that touch a register while an LDS read into it is in
    flight (empty when sound)."""
    from .isa_scan import kernel_hazards
    bad = {}
    for src in sorted(ASYNC_READS):
        with open(device_asm_path(src)) as f:
            bad.update({k: v for k, v in kernel_hazards(f.read()).items() if v})
    return bad


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    bad = check_async_reads()
    if bad:
        raise RuntimeError(f"registers touched while their LDS reads are in flight: {bad}")
    tmp = OUT + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    # a kernel whose host-side launch stub was not emitted (the host pass drops it without an
    # error when the kernel body does not compile for the host) leaves an undefined symbol of
    # the library's own namespace: refuse such a library
    nm = shutil.which("nm")
    if nm:
        r = subprocess.run([nm, "-D", "--undefined-only", tmp], capture_output=True, text=True)
        own = [ln.split()[-1] for ln in r.stdout.splitlines() if "_ZN2sr" in ln]
        if own:
            os.remove(tmp)
            raise RuntimeError("undefined symbols of libsr's own code:\n" + "\n".join(own[:10]))
    os.replace(tmp, OUT)
    if verbose:
        print(f"built {OUT}")
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
