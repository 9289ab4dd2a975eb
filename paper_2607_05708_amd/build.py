"""Build the HIP libraries in-tree with hipcc for gfx950.

* ``libmemattn.so``  -- the retrieval/gather library (C ABI in include/memattn.h)
* ``libmeminputs.so`` -- the device payload generator used to fill large
  synthetic page pools (input generation, not part of the method)

Usage: ``python -m paper_2607_05708_amd.build``.  Objects go to ``_build/``.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
BUILD = os.path.join(ROOT, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# -packed-fp32-ops: no v_pk_{add,mul,fma}_f32 in generated code.
DEVICE_FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-mcode-object-version=5",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wall", "-Wno-unused-result", "-fvisibility=hidden"]

LIBS = {
    "libmemattn.so": ["csrc/api.cpp", "csrc/topk_valu.hip", "csrc/topk_mfma.hip", "csrc/gather_append.hip",
                      "csrc/compact.hip"],
    "libmeminputs.so": ["inputs_hip/fill_payload.hip"],
}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src.replace("/", "_") + ".o")
    cmd = [HIPCC, *DEVICE_FLAGS, "-I", os.path.join(ROOT, "include"), "-c", os.path.join(HERE, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip():
        print(err, file=sys.stderr)
    return obj


def device_asm(src: str) -> str:
    """gfx950 assembly of one source file (device code only), built with the
    library's flags; used by host-side code-generation checks."""
    cmd = [HIPCC, *DEVICE_FLAGS, "-I", os.path.join(ROOT, "include"), "--cuda-device-only", "-S",
           os.path.join(HERE, src), "-o", "-"]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc -S failed for {src}:\n{res.stderr}")
    return res.stdout


def build(verbose: bool = True) -> dict:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted({s for v in LIBS.values() for s in v})
    with ThreadPoolExecutor(min(8, len(srcs))) as ex:
        objs = dict(zip(srcs, ex.map(_compile, srcs)))
    out = {}
    for lib, lsrcs in LIBS.items():
        path = os.path.join(HERE, lib)
        tmp = path + ".tmp"
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *[objs[s] for s in lsrcs]]
        subprocess.run(cmd, check=True, capture_output=True, text=True)
        os.replace(tmp, path)
        out[lib] = path
        if verbose:
            print(f"built {path}")
    return out


if __name__ == "__main__":
    build()
