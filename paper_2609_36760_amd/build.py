"""Build ``libmla_lowbit.so`` in-tree for gfx950.

The HIP translation units are compiled by ``hipcc --offload-arch=gfx950``;
the host ABI translation unit is plain C++ and is compiled by ``g++`` against
the HIP runtime headers only.  Flags that matter for results:

* ``-fhip-fp32-correctly-rounded-divide-sqrt`` and ``-ffp-contract=off`` on
  the writer: the quantizer's divisions and additions are single IEEE
  roundings, so packed codes and fp16 metadata are bit-exact;
* ``-fno-gpu-flush-denormals-to-zero``: fp16 subnormal scales survive;
* ``-Xclang -target-feature -Xclang -packed-fp32-ops``: no packed fp32 ALU
  instructions are generated.

Run ``python -m paper_2609_36760_amd.build`` (or ``build()``); it always
recompiles.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(PKG, "libmla_lowbit.so")
BUILD_DIR = os.path.join(ROOT, "_build")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fno-gpu-flush-denormals-to-zero",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Wall", "-Wno-unused-function",
    "-I", INCLUDE, "-I", CSRC,
]
PER_FILE = {
    "quant_append.hip": ["-ffp-contract=off"],
}
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
              "-I", os.path.join(ROCM, "include"), "-I", INCLUDE, "-I", CSRC]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r.stderr


def build(verbose: bool = False) -> str:
    hipcc = os.path.join(ROCM, "bin", "hipcc")
    gxx = shutil.which("g++") or "g++"
    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs = []
    for name in sorted(os.listdir(CSRC)):
        src = os.path.join(CSRC, name)
        obj = os.path.join(BUILD_DIR, name + ".o")
        if name.endswith(".hip"):
            jobs.append([hipcc, *HIP_FLAGS, *PER_FILE.get(name, []), "-c", src, "-o", obj])
        elif name.endswith(".cpp"):
            jobs.append([gxx, *HOST_FLAGS, "-c", src, "-o", obj])
    with ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        logs = list(ex.map(_run, jobs))
    objs = [j[-1] for j in jobs]
    tmp = OUT + ".tmp"
    _run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, OUT)
    if verbose:
        for log in logs:
            if log.strip():
                print(log, file=sys.stderr)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
