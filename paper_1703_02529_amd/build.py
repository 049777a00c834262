"""Builds the HIP libraries for gfx950 in-tree with hipcc.

    python -m paper_1703_02529_amd.build

produces paper_1703_02529_amd/libnsc.so (the cascade) and synth/libsynth.so
(the synthetic-video renderer used by tests and the benchmark, and the
benchmark's peak probes).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIBNSC = os.path.join(PKG, "libnsc.so")
SYNTH_DIR = os.path.join(ROOT, "synth")
LIBSYNTH = os.path.join(SYNTH_DIR, "libsynth.so")
OBJ_DIR = os.path.join(ROOT, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # no packed-FP32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in ordinary VGPRs: with accumulation registers the
    # compiler shuffles loop-carried accumulators between register files
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wall", "-Wno-unused-function",
]
SOURCES = ["api.hip", "area_diff.hip", "compact_resolve.hip", "cnn.hip", "sweep.hip"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass warns about the device-only target feature; drop that line
    err = "\n".join(l for l in r.stderr.splitlines()
                    if "packed-fp32-ops" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError(f"command failed: {' '.join(cmd)}\n{err}")
    if err:
        sys.stderr.write(err + "\n")


def build_nsc() -> str:
    os.makedirs(OBJ_DIR, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    objs, cmds = [], []
    for s in SOURCES:
        o = os.path.join(OBJ_DIR, s.replace(".hip", ".o"))
        objs.append(o)
        cmds.append([HIPCC, *HIP_FLAGS, *inc, "-c", os.path.join(CSRC, s), "-o", o])
    with cf.ThreadPoolExecutor(max_workers=len(cmds)) as ex:
        list(ex.map(_run, cmds))
    tmp = LIBNSC + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIBNSC)
    return LIBNSC


def build_synth() -> str:
    tmp = LIBSYNTH + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-shared", os.path.join(SYNTH_DIR, "synth_kernel.hip"),
          os.path.join(SYNTH_DIR, "probe_kernel.hip"), "-o", tmp])
    os.replace(tmp, LIBSYNTH)
    return LIBSYNTH


def build_all() -> list:
    with cf.ThreadPoolExecutor(max_workers=2) as ex:
        f1 = ex.submit(build_nsc)
        f2 = ex.submit(build_synth)
        return [f1.result(), f2.result()]


if __name__ == "__main__":
    for p in build_all():
        print(p)
