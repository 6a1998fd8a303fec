"""Build libcast.so (gfx950) in-tree with hipcc.

    python -m paper_2609_34144_amd.build

Each translation unit is compiled to an object with its own flags, then linked
into paper_2609_34144_amd/libcast.so.  Packed-fp32 instructions are disabled for
all device code.  The PAR unit is built with -fno-signed-zeros so that the
literal zero imaginary parts of real-input tile transforms fold away; the
attention unit selects the VGPR form of the MFMA instructions.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libcast.so")
CLIENT = os.path.join(HERE, "cast_client")
BUILD = os.path.join(os.path.dirname(HERE), "_build")

ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-function", "-Wno-unused-variable"]
# (source, object name, extra flags), longest first; par_fused.hip is compiled
# once per bottom-remainder height of the 8x8 tiling (one row of the
# fused-kernel table)
UNITS = [("par.hip", "par", ["-fno-signed-zeros"])] + [
    ("par_fused.hip", f"par_fused_{hr}", ["-fno-signed-zeros", f"-DCAST_PAR_HR={hr}"])
    for hr in range(8, 0, -1)
] + [
    # MFMA accumulators in VGPRs: the softmax reads S directly, and the Q operands
    # are parked in AGPRs by the kernel itself
    ("anchor_attn.hip", "anchor_attn", ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]),
    ("route_kv.hip", "route_kv", []),
    ("route_coupled.hip", "route_coupled", []),
    ("frame_select.hip", "frame_select", []),
    ("diag.hip", "diag", []),
] + [
    ("diag_fixed.hip", f"diag_fixed_{hp}", ["-fno-signed-zeros", f"-DCAST_DIAG_HP={hp}"])
    for hp in range(8, 0, -1)
] + [
    ("capi.hip", "capi", []),
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def build(verbose: bool = True, jobs: int = 0) -> str:
    jobs = jobs or max(1, min(8, os.cpu_count() or 1))
    os.makedirs(BUILD, exist_ok=True)
    cc = hipcc()
    procs = []
    objs = []
    t0 = time.time()
    for src, name, extra in UNITS:
        obj = os.path.join(BUILD, name + ".o")
        objs.append(obj)
        cmd = [cc, "-c", os.path.join(CSRC, src), "-o", obj] + COMMON + extra
        if verbose:
            print("[build]", " ".join(cmd), flush=True)
        procs.append((name, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        while sum(p.poll() is None for _, p in procs) >= jobs:
            time.sleep(0.05)
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        # the host pass does not know the device-only target feature; that line is noise
        text = "\n".join(l for l in text.splitlines() if "packed-fp32-ops" not in l)
        if text.strip() and verbose:
            print(text, flush=True)
        if p.returncode != 0:
            failed.append(src)
    if failed:
        raise RuntimeError(f"hipcc failed for {failed}")
    tmp = OUT + ".tmp"
    cmd = [cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    if verbose:
        print("[build]", " ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, OUT)
    # a C-ABI client with no Python (tests/test_gpu_c_client.py runs it)
    ctmp = CLIENT + ".tmp"
    cmd = [cc, "-O2", "-std=c++17", f"--offload-arch={ARCH}", os.path.join(CSRC, "cast_client.cpp"),
           "-o", ctmp, "-L" + HERE, "-lcast", "-Wl,-rpath,$ORIGIN"]
    if verbose:
        print("[build]", " ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(ctmp, CLIENT)
    if verbose:
        print(f"[build] {OUT} and {CLIENT} ({time.time() - t0:.1f} s)", flush=True)
    return OUT


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)
