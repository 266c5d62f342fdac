"""Build libdkv.so (the C-ABI library) for gfx950 with hipcc, in-tree.

    python paper_2609_32663_amd/build.py [--jobs N] [--phase-stamps]

(run as a script: importing the package loads the library, which this builds).
With --phase-stamps it builds libdkv_phase.so instead: the same sources with
DKV_PHASE_STAMPS=1, whose decode kernels record per-workgroup clock stamps
(bench.py --phase-budget reads them); the product library never has them.

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
PHASE_LIB_PATH = os.path.join(HERE, "libdkv_phase.so")
PHASE_BUILD_DIR = os.path.join(os.path.dirname(HERE), "_build_phase")

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
SOURCES = ["map_pattern.hip", "compact.hip", "compact_bins.hip", "decode_attn.hip", "dkv_api.cpp", "bw_probe.hip",
           "query_attn.hip", "dkv_query_api.cpp", "page_select.hip", "dkv_paged_api.cpp",
           "topk_pattern.hip", "dkv_pattern_api.cpp"]


def _hipcc():
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the ROCm toolchain is required to build libdkv.so")


def _compile(src, hipcc, verbose, build_dir=BUILD_DIR, extra=()):
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [hipcc, *COMMON_FLAGS, *extra, *FILE_FLAGS.get(src, []), *lang, "-c", os.path.join(CSRC, src), "-o", obj]
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


def build(verbose=False, jobs=4, phase_stamps=False):
    """Compile every source and link libdkv.so (or, with phase_stamps, the
    stamped libdkv_phase.so); returns the library path."""
    hipcc = _hipcc()
    build_dir = PHASE_BUILD_DIR if phase_stamps else BUILD_DIR
    lib_path = PHASE_LIB_PATH if phase_stamps else LIB_PATH
    extra = ["-DDKV_PHASE_STAMPS=1"] if phase_stamps else []
    os.makedirs(build_dir, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, hipcc, verbose, build_dir, extra), SOURCES))
    tmp = lib_path + ".tmp"
    cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, lib_path)
    return lib_path


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=4)
    ap.add_argument("-q", "--quiet", action="store_true")
    ap.add_argument("--phase-stamps", action="store_true",
                    help="build libdkv_phase.so (decode kernels with per-workgroup clock stamps)")
    a = ap.parse_args()
    print(build(verbose=not a.quiet, jobs=a.jobs, phase_stamps=a.phase_stamps))
    sys.exit(0)
