"""In-tree build of libkvg.so (and the input generator's libkvg_synth.so) for gfx950.

    python -m paper_2607_14431_amd.build

Every call recompiles.  Objects go to _build/ (not committed); the shared libraries land
next to their sources so that they travel with the tree.
"""

from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2607_14431_amd")
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")

KVG_SOURCES = ["kvg_api.cpp", "kvg_api_digest.cpp", "kvg_api_logits.cpp", "kvg_api_noalloc.cpp", "kvg_append.hip",
               "kvg_copy.hip",
               "kvg_attn_valu.hip", "kvg_prefill_mfma.hip", "kvg_digest.hip", "kvg_logits.hip"]
ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Packed fp32 VALU instructions are disabled for all device code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall", "-Wno-unused-function"]
# Per-source extras.  The MFMA prefill keeps its accumulators in VGPRs: left to choose, the
# register allocator splits them between AGPRs and VGPRs and copies them every key tile.
EXTRA = {"kvg_prefill_mfma.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return res


def _compile(src, obj, includes):
    cmd = [HIPCC, *COMMON, *DEVICE_FLAGS, *EXTRA.get(os.path.basename(src), []), *[f"-I{i}" for i in includes],
           "-c", src, "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    _run(cmd)
    return obj


def _link(objs, out):
    tmp = out + ".tmp"
    # -z defs: a symbol left undefined (say a kernel whose host stub was not emitted) fails here,
    # not at load time
    _run([HIPCC, "-shared", f"--offload-arch={ARCH}", "-Wl,-z,defs", "-o", tmp, *objs])
    os.replace(tmp, out)


def build_kvg(jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    includes = [os.path.join(ROOT, "include"), CSRC]
    with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
        futs = [ex.submit(_compile, os.path.join(CSRC, s), os.path.join(BUILD, s + ".o"), includes)
                for s in KVG_SOURCES]
        objs = [f.result() for f in futs]
    out = os.path.join(PKG, "libkvg.so")
    _link(objs, out)
    return out


def build_synth() -> str:
    os.makedirs(BUILD, exist_ok=True)
    src = os.path.join(ROOT, "synth", "gen.hip")
    obj = _compile(src, os.path.join(BUILD, "synth_gen.o"), [])
    out = os.path.join(ROOT, "synth", "libkvg_synth.so")
    _link([obj], out)
    return out


def build_all() -> list[str]:
    if shutil.which(HIPCC) is None and not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    with concurrent.futures.ThreadPoolExecutor(max_workers=2) as ex:
        a = ex.submit(build_kvg)
        b = ex.submit(build_synth)
        return [a.result(), b.result()]


if __name__ == "__main__":
    for p in build_all():
        print(p)
    sys.exit(0)
