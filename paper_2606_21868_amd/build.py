"""Build the native parts in-tree: ``libwisp.so`` (HIP, gfx950) and ``libwisp_datagen.so`` (host C).

``python -m paper_2606_21868_amd.build`` or ``__graft_entry__.build()``.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Packed-fp32 instructions are disabled for all device code (they have given silent wrong results
# on this hardware); hipcc's host pass warns that it does not know the feature, which is harmless.
HIP_FLAGS = [
    "-std=c++17", "-O3", "-fPIC", f"--offload-arch={ARCH}", "-ffp-contract=fast",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-result", f"-I{INCLUDE}", f"-I{CSRC}",
]

HIP_SOURCES = ["abi.cpp", "slot_table.cpp", "staging.cpp", "copy_pool.cpp", "mvwsa.cpp", "predictor.cpp", "router.hip", "expert_ffn.hip", "combine.hip", "probe.hip", "fill.hip",
               "pager.hip", "grouped_gemm.hip", "noalloc.cpp"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}")
    return r.stdout


def build_datagen():
    src = os.path.join(HERE, "datagen", "datagen.c")
    out = os.path.join(HERE, "datagen", "libwisp_datagen.so")
    _run(["gcc", "-O3", "-mavx2", "-ffp-contract=off", "-fno-math-errno", "-fopenmp", "-fPIC", "-shared",
          "-Wall", "-o", out + ".tmp", src, "-lm"])
    os.replace(out + ".tmp", out)
    return out


def build_wisp(jobs=8):
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = [s for s in HIP_SOURCES if os.path.exists(os.path.join(CSRC, s))]
    objs = [os.path.join(BUILD_DIR, s + ".o") for s in srcs]

    def compile_one(pair):
        s, o = pair
        lang = [] if s.endswith(".hip") else ["-x", "hip"]
        _run([HIPCC, *HIP_FLAGS, *lang, "-c", os.path.join(CSRC, s), "-o", o])
        return o

    with cf.ThreadPoolExecutor(max_workers=max(1, min(jobs, len(srcs)))) as ex:
        list(ex.map(compile_one, zip(srcs, objs)))
    out = os.path.join(HERE, "libwisp.so")
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out + ".tmp", *objs])
    os.replace(out + ".tmp", out)
    return out


def build_all(jobs=8):
    if not shutil.which(HIPCC) and not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    outs = [build_datagen(), build_wisp(jobs)]
    return outs


if __name__ == "__main__":
    for p in build_all(int(sys.argv[1]) if len(sys.argv) > 1 else 8):
        print(p)
