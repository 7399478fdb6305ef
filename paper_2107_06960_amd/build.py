"""Builds libmafat.so (the HIP library) in-tree for gfx950.

    python -m paper_2107_06960_amd.build            # libmafat.so
    python -m paper_2107_06960_amd.build --trace    # libmafat_trace.so

Every source under csrc/ is compiled with hipcc for gfx950 and linked into
paper_2107_06960_amd/libmafat.so.  Packed fp32 instructions are disabled
for all device code.  The trace variant (MAFAT_TUNING) adds wall-clock
stamps per workgroup and per kernel phase, printed by the runtime when
MAFAT_WG_DUMP / MAFAT_TRACE_DUMP are set (bench.py --phase-trace); it is a
measurement build, never the product library.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libmafat.so")
BUILD = os.path.join(HERE, "_build")
ARCH = "gfx950"


def hipcc():
    for p in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if p and os.path.exists(p):
            return p
    raise RuntimeError("hipcc not found")


COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          # matrix-core accumulators in ordinary VGPRs (no AGPR copies in
          # the epilogues)
          "-mllvm", "-amdgpu-mfma-vgpr-form",
          "-I", os.path.join(HERE, "..", "include")]


TRACE_LIB = os.path.join(HERE, "libmafat_trace.so")


def _compile(src, build_dir=BUILD, extra=()):
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    cmd = [hipcc()] + COMMON + list(extra) + ["-x", "hip", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    warn = "\n".join(ln for ln in r.stderr.splitlines() if "packed-fp32-ops" not in ln)
    return obj, warn.strip()


def build(verbose: bool = True, trace: bool = False) -> str:
    build_dir = os.path.join(BUILD, "trace") if trace else BUILD
    lib = TRACE_LIB if trace else LIB
    extra = ("-DMAFAT_TUNING",) if trace else ()
    os.makedirs(build_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.cpp")) + glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        results = list(ex.map(lambda src: _compile(src, build_dir, extra), srcs))
    for obj, warn in results:
        if warn and verbose:
            print(warn, file=sys.stderr)
    tmp = lib + f".tmp{os.getpid()}"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + [o for o, _ in results]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build(trace="--trace" in sys.argv[1:])
