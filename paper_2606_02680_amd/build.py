"""Build libpbb.so in-tree with hipcc for gfx950.

``python -m paper_2606_02680_amd.build`` compiles ``csrc/pbb_api.cpp``,
``csrc/pbb_kernels.hip`` (decode), ``csrc/pbb_prefill.hip`` (prefill) and
``csrc/pbb_backward.hip`` (training backward) into ``paper_2606_02680_amd/libpbb.so`` (and the
streaming-read probe ``csrc/pbb_probe.hip``, a measurement helper, into ``libpbbprobe.so``) and
writes the compiler's
per-kernel resource report (VGPRs, AGPRs, SGPRs, LDS, scratch) to ``_build/resource_usage.txt``
(an untracked build output next to the library).
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libpbb.so")
PROBE_LIB = os.path.join(PKG, "libpbbprobe.so")   # measurement helper (include/pbb_probe.h)
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    # Keep the compiler from emitting packed fp32 arithmetic (v_pk_fma_f32 and friends).
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def build(verbose: bool = False) -> str:
    sources = [os.path.join(CSRC, "pbb_api.cpp"), os.path.join(CSRC, "pbb_kernels.hip"),
               os.path.join(CSRC, "pbb_prefill.hip"), os.path.join(CSRC, "pbb_backward.hip")]
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, "-Rpass-analysis=kernel-resource-usage", *sources, "-o", tmp]
    proc = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    report = [ln for ln in proc.stdout.splitlines() if "remark:" in ln]
    other = [ln for ln in proc.stdout.splitlines()
             if "remark:" not in ln and "packed-fp32-ops" not in ln and ln.strip()]
    if proc.returncode != 0:
        sys.stderr.write("\n".join(other) + "\n")
        raise RuntimeError(f"hipcc failed ({proc.returncode}): {' '.join(cmd)}")
    os.replace(tmp, LIB)
    os.makedirs(os.path.join(PKG, "_build"), exist_ok=True)
    with open(os.path.join(PKG, "_build", "resource_usage.txt"), "w") as f:
        for ln in report:
            f.write(ln.split("remark: ", 1)[-1].strip() + "\n")
    if verbose and other:
        print("\n".join(other))
    build_probe()
    return LIB


def build_probe() -> str:
    """Compile the streaming-read probe (``csrc/pbb_probe.hip``) into ``libpbbprobe.so``."""
    tmp = PROBE_LIB + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, os.path.join(CSRC, "pbb_probe.hip"), "-o", tmp]
    proc = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if proc.returncode != 0:
        sys.stderr.write(proc.stdout + "\n")
        raise RuntimeError(f"hipcc failed ({proc.returncode}): {' '.join(cmd)}")
    os.replace(tmp, PROBE_LIB)
    return PROBE_LIB


if __name__ == "__main__":
    print(build(verbose=True))
