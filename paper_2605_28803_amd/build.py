"""Build the HIP library liboq.so in-tree for gfx950 with hipcc.

Every source under csrc/ is compiled (in parallel) to an object under _build/
and linked into paper_2605_28803_amd/liboq.so.  Always recompiles.  Before
linking, the gfx950 code of every object is disassembled and checked for MFMAs
that could run under an empty EXEC mask (isa_check).
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "liboq.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed-fp32 VALU forms are disabled for all device code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# Per-source extra device flags.  The rotate-quantize kernels keep their
# matrix-core results in ordinary VGPRs (the accumulator-register form makes
# the compiler copy every value back and forth between the two files).
EXTRA = {"rotate_quant.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
          "-Wall", "-Wno-unused-function", "-Wno-unused-variable"]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    extra = EXTRA.get(os.path.basename(src), [])
    cmd = [HIPCC] + COMMON + DEVICE_FLAGS + extra + lang + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    if not shutil.which(HIPCC) and not os.path.exists(HIPCC):
        raise RuntimeError("hipcc not found")
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))
    jobs = min(len(srcs), max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, srcs))
    # Matrix-core instructions ignore EXEC: refuse code in which an MFMA can
    # run under a narrowed EXEC mask with no branch around it.
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)  # run as a script
    from paper_2605_28803_amd import isa_check
    bad = isa_check.check_objects(objs)
    if bad:
        raise RuntimeError("MFMA under a possibly-empty EXEC mask (no s_cbranch_execz around it):\n" +
                           "\n".join(f"  {o}: {f}: {i}" for o, f, i in bad[:20]))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs + ["-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB} from {len(srcs)} sources")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
