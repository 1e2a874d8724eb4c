"""Build the HIP library libxdit.so in-tree for gfx950 with hipcc.

    python -m paper_2411_01738_amd.build

Every HIP translation unit is compiled with packed-fp32 instruction
generation disabled (-Xclang -target-feature -Xclang -packed-fp32-ops).
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIBRARY = os.path.join(HERE, "libxdit.so")
SOURCES = ["xdit_api.cpp", "attn_bf16.hip", "attn_w64.hip", "attn_f32.hip", "merge_update.hip"]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas"]


# Per-source flags.  The attention kernels are scheduled by LLVM's iterative
# ILP strategy, which interleaves their matrix products and softmax VALU work
# better than the default occupancy strategy (measured 1-3 % faster at head
# dims 64, 72 and 128, same register counts within a few).
EXTRA = {"attn_bf16.hip": ["-mllvm", "-amdgpu-sched-strategy=iterative-ilp"]}


ATTN_SOURCES = ("attn_bf16.hip", "attn_w64.hip", "attn_common.h")


def kernel_fingerprint(srcs=ATTN_SOURCES) -> str:
    """sha256 prefix of the attention kernels' sources and compile flags:
    measurements taken on one build of the kernels are matched to it by this
    value."""
    import hashlib

    h = hashlib.sha256()
    for src in ([srcs] if isinstance(srcs, str) else srcs):
        with open(os.path.join(CSRC, src), "rb") as f:
            h.update(f.read())
        h.update(" ".join(FLAGS + EXTRA.get(src, [])).encode())
    return h.hexdigest()[:16]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *EXTRA.get(src, []), "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature and says so; that is harmless
    noise = "is not a recognized feature for this target"
    msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{msgs}")
    if msgs.strip():
        print(msgs, file=sys.stderr)
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link libxdit.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIBRARY + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs,
           "-L/opt/rocm/lib", "-Wl,-rpath,/opt/rocm/lib", "-lhipblaslt"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIBRARY)
    if verbose:
        print(f"built {LIBRARY}")
    return LIBRARY


if __name__ == "__main__":
    build(verbose=True)
