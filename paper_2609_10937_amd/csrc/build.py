"""Build libattn.so (HIP kernels + C ABI) for gfx950 with hipcc.

Every translation unit is compiled in parallel into _build/ at the repository
root and linked into paper_2609_10937_amd/libattn.so.  The compiler's
per-kernel resource report (registers, scratch, LDS, occupancy) is saved as
_build/kernel_resources.json.
"""
from __future__ import annotations

import concurrent.futures as cf
import json
import os
import re
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libattn.so")

SOURCES = [
    "capi.cpp",
    "tile_derive.cpp",
    "combine.hip",
    "noalloc.hip",
    "probe.hip",
    "unfused.hip",
    "softmax.hip",
    "fwd_bf16_d64.hip",
    "fwd_bf16_d128.hip",
    "fwd_f16_d64.hip",
    "fwd_f16_d128.hip",
    "fwd_bf16_d256.hip",
    "fwd_f16_d256.hip",
    "fwd_bf16_d96.hip",
    "fwd_f16_d96.hip",
    "gemm_bf16.hip",
    "gemm_f16.hip",
    "gemm_f32.hip",
    "gemm_unfused_bf16.hip",
    "gemm_unfused_f16.hip",
]

ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", os.path.join(ROOT, "include"),
          "-I", HERE, "-Wall", "-Wno-unused-function"]
# Packed fp32 VALU forms are kept out of the device code.
DEVICE = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Rpass-analysis=kernel-resource-usage",
          # No NaN operands are relied on (infinities are): max/min need no
          # NaN-quieting canonicalisation.
          "-fno-honor-nans"]


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def _compile(src):
    hipcc = _hipcc()
    path = os.path.join(HERE, src)
    obj = os.path.join(BUILD, src.replace(".", "_") + ".o")
    cmd = [hipcc, *COMMON]
    if src.endswith(".hip"):
        cmd += ["-x", "hip", *DEVICE]
    cmd += ["-c", path, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stderr}")
    return obj, r.stderr


_KEYS = {
    "VGPRs": "vgpr", "AGPRs": "agpr", "ScratchSize [bytes/lane]": "scratch",
    "Occupancy [waves/SIMD]": "occupancy", "LDS Size [bytes/block]": "lds", "SGPRs": "sgpr",
}


def _parse_resources(text):
    out, cur = {}, None
    for line in text.splitlines():
        m = re.search(r"remark:\s+(.*?)\s*\[-Rpass-analysis", line)
        if not m:
            continue
        body = m.group(1)
        if body.startswith("Function Name:"):
            cur = body.split(":", 1)[1].strip()
            out[cur] = {}
            continue
        if cur is None or ":" not in body:
            continue
        k, v = body.rsplit(":", 1)
        k = k.strip()
        if k in _KEYS:
            try:
                out[cur][_KEYS[k]] = int(v.strip())
            except ValueError:
                pass
    return out


def build(jobs: int | None = None, verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = jobs or min(8, len(SOURCES), os.cpu_count() or 1)
    resources = {}
    objs = []
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        for obj, err in ex.map(_compile, SOURCES):
            objs.append(obj)
            resources.update(_parse_resources(err))
            if verbose:
                print(f"built {os.path.basename(obj)}", flush=True)
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stderr}")
    os.replace(tmp, LIB)
    with open(os.path.join(BUILD, "kernel_resources.json"), "w") as f:
        json.dump(resources, f, indent=1, sort_keys=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
