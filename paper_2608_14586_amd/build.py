"""Compile the HIP kernels and the C-ABI runtime into ``libvlaprefix.so``
(gfx950 only) with hipcc.  Objects go to ``_build/`` next to this file."""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libvlaprefix.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed-fp32 VALU ops are switched off for all device code.
DEVICE_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-fPIC", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
                "-packed-fp32-ops", "-Wno-unused-result"]
HOST_FLAGS = ["-O2", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-result"]

SOURCES = ["gemm_bf16.hip", "attention_bf16.hip", "decode_bf16.hip", "norm.hip", "fp32_path.hip", "vision.hip",
           "static_scratch.hip",
           "runtime.cpp",
           "ops.cpp",
           "host_suffix.cpp", "host_suffix_api.cpp", "sched.cpp"]
# Attention keeps its score and output accumulators in VGPRs: the softmax
# touches them every key tile, and AGPR accumulators would cost a copy each way.
EXTRA = {"attention_bf16.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
         # the host suffix executor: AVX-512 BF16 kernels, entered only after a CPU check
         "host_suffix.cpp": ["--offload-host-only", "-O3", "-mavx512f", "-mavx512bw", "-mavx512vl", "-mavx512bf16",
                             "-mfma"],
         "host_suffix_api.cpp": ["--offload-host-only"],
         "sched.cpp": ["--offload-host-only"]}


def _compile(src: str) -> str:
    path = os.path.join(CSRC, src)
    obj = os.path.join(OUT_DIR, src + ".o")
    if src.endswith(".hip"):
        cmd = [HIPCC] + DEVICE_FLAGS + EXTRA.get(src, []) + ["-c", path, "-o", obj]
    else:
        cmd = [HIPCC] + HOST_FLAGS + EXTRA.get(src, []) + ["-c", path, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr[-6000:]))
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link the shared library; returns its path."""
    os.makedirs(OUT_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr[-4000:]))
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
