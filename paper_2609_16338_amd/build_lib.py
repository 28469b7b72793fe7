"""Build libbitcos.so in-tree for gfx950 with hipcc.

Every HIP source is compiled to an object under ``_build/`` (in parallel),
the host packers with the same compiler, and everything is linked into
``paper_2609_16338_amd/libbitcos.so``.  Run ``python -m
paper_2609_16338_amd.build_lib`` or call :func:`build`.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libbitcos.so")
ARCH = "gfx950"

HIP_SOURCES = [
    "gemv_bitcos.hip", "gemv_bitcos_s4.hip", "gemv_bitcos_s8.hip", "gemv_bitcos_s16.hip",
    "gemv_bitcos_s32.hip", "gemv_bitcos_s64.hip", "gemv_fixed.hip", "fixed_trit5.hip", "fixed_bit2.hip",
    "gemv_bitcos_d4.hip", "gemv_bitcos_d8.hip", "gemv_bitcos_d16.hip", "gemv_bitcos_d32.hip", "gemv_bitcos_d64.hip",
    "gemv_bitcos_mfma.hip", "batch.hip", "quantize.hip", "pack_device.hip", "partials.hip",
]
HOST_SOURCES = ["host.cpp"]

COMMON = ["-O3", "-fPIC", "-std=c++20", "-Wall", "-Wno-unused-function", f"-I{ROOT}/include"]
# Packed fp32 instructions stay off in every device compile.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libbitcos)")


def _run(cmd: list[str]) -> tuple[list[str], int, str]:
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # The host pass does not know the packed-fp32 feature; that note is noise.
    out = "\n".join(l for l in p.stdout.splitlines() if "packed-fp32-ops" not in l)
    return cmd, p.returncode, out


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every source and link libbitcos.so; returns the library path."""
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    cmds = []
    objs = []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        cmds.append([hipcc, *COMMON, *DEVICE, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src.replace(".cpp", ".host.o"))
        cmds.append([hipcc, *COMMON, "-x", "c++", "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    jobs = jobs or min(len(cmds), max(1, os.cpu_count() or 1))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        for cmd, rc, out in ex.map(_run, cmds):
            if verbose or rc:
                print(" ".join(cmd), file=sys.stderr)
                if out.strip():
                    print(out, file=sys.stderr)
            if rc:
                raise RuntimeError(f"compile failed: {cmd[-3]}")
    tmp = LIB + ".tmp"
    cmd, rc, out = _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    if rc:
        print(out, file=sys.stderr)
        raise RuntimeError("link failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
