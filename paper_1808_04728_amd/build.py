"""Build the gfx950 shared library ``libcosmoflow_hip.so`` in-tree with hipcc.

    python -m paper_1808_04728_amd.build        # compile every source, link

Each source in csrc/ is compiled to an object (in parallel), then linked into
paper_1808_04728_amd/libcosmoflow_hip.so next to this file.  Packed fp32 ops
are disabled for all device code.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libcosmoflow_hip.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wno-unused-command-line-argument", "-I", CSRC,
          "-I", os.path.join(os.path.dirname(HERE), "include")]


# Per-source extra flags.  -amdgpu-mfma-vgpr-form keeps MFMA accumulators in
# ordinary VGPRs: for kernels whose epilogue runs vector arithmetic on every
# accumulator (the fused first layer) it saves one AGPR read per value.
# The fp32 kernels need it for another reason: with AGPR accumulators the
# compiler shuttles them through VGPRs around the streamed loads (measured:
# 120 accvgpr moves in the 16 -> 32 forward's loop, none in VGPR form).
EXTRA = {
    "conv_smallc.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    "conv_smallc_pair.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    "conv_f32.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    "conv_f32_wgrad.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)
                  if f.endswith((".hip", ".cpp")))


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC, *COMMON, *EXTRA.get(os.path.basename(src), []), *lang, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(jobs: int | None = None) -> str:
    """Compile every source and link the shared library; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 2)))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
    sys.exit(0)
