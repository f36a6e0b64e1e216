"""Build libakvs.so (HIP, gfx950) in-tree with hipcc.

Every call recompiles all sources; objects go to _build/ beside this file and the
shared library to libakvs.so beside this file.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libakvs.so")
SOURCES = ["api.hip", "k_misc.hip", "k_reuse.hip", "k_gemm.hip", "k_attn.hip", "k_decode.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed fp32 instructions are kept out of the generated code on purpose.
CFLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
          "-Wno-unused-function", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("command failed: " + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    return r.stderr


def build(verbose: bool = False, jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs = [os.path.join(BUILD, os.path.splitext(s)[0] + ".o") for s in SOURCES]

    def compile_one(src_obj):
        src, obj = src_obj
        err = _run([HIPCC, *CFLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
        return src, err

    with ThreadPoolExecutor(max_workers=max(1, min(jobs, len(SOURCES)))) as ex:
        for src, err in ex.map(compile_one, zip(SOURCES, objs)):
            noise = [l for l in err.splitlines() if "packed-fp32-ops" not in l and l.strip()]
            if verbose and noise:
                print(f"[{src}]\n" + "\n".join(noise), file=sys.stderr)
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
