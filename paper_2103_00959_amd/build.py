"""Build libcogdl_mi355.so (HIP for gfx950) in-tree with hipcc.

    python -m paper_2103_00959_amd.build

Every translation unit is compiled for gfx950 only, with packed-fp32
instructions disabled, and linked into one shared library next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libcogdl_mi355.so")
# counter-calibration kernels (known traffic), a library of their own
CALIB_LIB = os.path.join(HERE, "libcogdl_calib.so")
CALIB_SOURCES = ["calib.hip"]
SOURCES = ["primitives.hip", "plan.hip", "spmm.hip", "gspmm.hip", "gat.hip", "gat_proj.hip", "gat_bwd.hip", "dense.hip", "codec.hip", "csc.hip", "trace.hip"]

ARCH = "gfx950"
FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", INCLUDE, "-I", CSRC,
]


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = True, jobs: int | None = None) -> str:
    os.makedirs(BUILD, exist_ok=True)
    cc = hipcc()
    t0 = time.time()
    procs = []
    objs = []
    for src in SOURCES + CALIB_SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        objs.append(obj)
        cmd = [cc, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        # hipcc's host pass does not know the packed-fp32 feature; that note is harmless
        lines = [l for l in text.splitlines() if "packed-fp32-ops" not in l]
        if p.returncode != 0:
            failed.append(src)
            print("\n".join(lines), file=sys.stderr)
        elif verbose and lines:
            print("\n".join(lines))
    if failed:
        raise RuntimeError(f"hipcc failed for {failed}")
    calib_objs = objs[len(SOURCES):]
    objs = objs[:len(SOURCES)]
    for lib_path, lib_objs in ((LIB, objs), (CALIB_LIB, calib_objs)):
        tmp = lib_path + f".tmp{os.getpid()}"
        subprocess.run([cc, "-shared", f"--offload-arch={ARCH}", "-o", tmp, *lib_objs], check=True)
        os.replace(tmp, lib_path)
    if verbose:
        print(f"[build] {LIB} in {time.time() - t0:.1f}s")
    return LIB


if __name__ == "__main__":
    build()
