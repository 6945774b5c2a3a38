"""Build libmxfp4.so in-tree with hipcc for gfx950.

Usage: python -m paper_2502_20586_amd.build   (or call build()).
Every call recompiles; objects go to <repo>/_build/ and the library to
paper_2502_20586_amd/libmxfp4.so.
"""

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB_PATH = os.path.join(PKG, "libmxfp4.so")
SOURCES = ["mx_quant_rht_sr.hip", "mx_quant_sr8.hip", "mx_quant_ablation.hip", "mx_quant.hip", "mx_gemm.hip",
           "mx_abi.hip", "mx_profile.hip"]
ARCH = "gfx950"

# -packed-fp32-ops off: no v_pk_*_f32 from the compiler. Denormals kept and no
# FP contraction: the quantiser's FP32 arithmetic must be exactly the
# documented sequence of IEEE operations.
HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fno-gpu-flush-denormals-to-zero", "-ffp-contract=off",
    "-Wall", "-Wno-unused-function",
]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    out = res.stdout + res.stderr
    # hipcc's host pass does not know the packed-fp32 target feature; that warning is expected.
    lines = [l for l in out.splitlines() if "packed-fp32-ops" not in l and l.strip()]
    if res.returncode != 0:
        raise RuntimeError("command failed: %s\n%s" % (" ".join(cmd), "\n".join(lines)))
    return "\n".join(lines)


def build(verbose=False):
    cc = hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(BUILD_DIR, src.replace(".hip", ".o"))
        objs.append(obj)
        cmds.append([cc, *HIPCC_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj])
    with ThreadPoolExecutor(max_workers=len(cmds)) as pool:
        logs = list(pool.map(_run, cmds))
    tmp = LIB_PATH + ".tmp"
    logs.append(_run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]))
    os.replace(tmp, LIB_PATH)
    if verbose:
        for l in logs:
            if l:
                print(l)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
