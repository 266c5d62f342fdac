"""Build libdkv.so (the C-ABI library) for gfx950 with hipcc, in-tree.

    python paper_2609_32663_amd/build.py [--jobs N]

(run as a script: importing the package loads the library, which this builds).

Every kernel source is compiled for gfx950 only.  Packed-fp32 VALU
instructions are disabled (`-target-feature -packed-fp32-ops`); hipcc's host
pass warns that it does not know that feature, which is harmless.
"""

import argparse
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
LIB_NAME = "libdkv.so"
LIB_PATH = os.path.join(HERE, LIB_NAME)
BUILD_DIR = os.path.join(os.path.dirname(HERE), "_build")

ARCH = "gfx950"
COMMON_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", "-Wall", "-Wno-unused-function",
]
# Per-file additions.  Query-block attention runs with IEEE mode off and no
# NaN semantics, so its row maxima need no NaN canonicalisation (its kernels
# form no NaN from finite inputs; see the file's header).
FILE_FLAGS = {"query_attn.hip": ["-mno-amdgpu-ieee", "-fno-honor-nans"]}
SOURCES = ["map_pattern.hip", "compact.hip", "decode_attn.hip", "dkv_api.cpp", "bw_probe.hip",
           "query_attn.hip", "dkv_query_api.cpp", "page_select.hip", "dkv_paged_api.cpp",
           "topk_pattern.hip", "dkv_pattern_api.cpp"]


def _hipcc():
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the ROCm toolchain is required to build libdkv.so")


def _compile(src, hipcc, verbose):
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [hipcc, *COMMON_FLAGS, *FILE_FLAGS.get(src, []), *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{out}")
    if out.strip() and verbose:
        print(out)
    return obj


def build(verbose=False, jobs=4):
    """Compile every source and link libdkv.so; returns the library path."""
    hipcc = _hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, hipcc, verbose), SOURCES))
    tmp = LIB_PATH + ".tmp"
    cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=4)
    ap.add_argument("-q", "--quiet", action="store_true")
    a = ap.parse_args()
    print(build(verbose=not a.quiet, jobs=a.jobs))
    sys.exit(0)
