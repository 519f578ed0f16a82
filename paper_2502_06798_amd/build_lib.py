"""Build libapc.so (gfx950) in-tree with hipcc.

Each source compiles to an object in parallel, then one link step.  Always
compiles when called; the binding only loads what is built.
"""
from __future__ import annotations

import concurrent.futures
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libapc.so")
BUILD = os.path.join(HERE, "_build")
SOURCES = ["apc.cpp", "rowfactor.hip", "simtopk.hip", "stream.hip", "qs.hip", "qs_f16.hip", "qs_bf16.hip", "qs_e4m3.hip", "qs8_f16.hip", "qs8_bf16.hip", "qs8_e4m3.hip", "assign.hip", "gather.hip", "resident.hip", "shards.hip", "quantize.hip", "f32small.hip"]

# Kernels in these sources load into LDS with asm and wait for those loads by
# counting vector-memory operations themselves; a register spill would add
# scratch loads to the count, so their code must not use scratch memory.
COUNTED = ["qs_f16.hip", "qs_bf16.hip", "qs_e4m3.hip", "qs8_f16.hip", "qs8_bf16.hip", "qs8_e4m3.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
         # no packed fp32 instructions: hipcc would otherwise form them from plain float code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         # MFMA results in VGPRs: no copies of the accumulators between register files
         "-mllvm", "-amdgpu-mfma-vgpr-form"]
# Per-source additions.  The query-stationary kernels keep their per-lane lists
# as separate registers: promoted to one vector, a list is copied whole on
# every pass of the insertion loop.
SOURCE_FLAGS = {src: ["-mllvm", "-disable-promote-alloca-to-vector"]
                for src in ("qs_f16.hip", "qs_bf16.hip", "qs_e4m3.hip", "qs8_f16.hip", "qs8_bf16.hip", "qs8_e4m3.hip")}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *SOURCE_FLAGS.get(src, []), "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=900)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def _check_no_scratch(src: str) -> None:
    asm = os.path.join(BUILD, os.path.splitext(src)[0] + ".s")
    cmd = [HIPCC, *FLAGS, *SOURCE_FLAGS.get(src, []), "--cuda-device-only", "-S", "-x", "hip",
           os.path.join(CSRC, src), "-o", asm]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=900)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc -S failed for {src}:\n{r.stderr}")
    text = open(asm).read()
    bad = [(m.group(1), int(m.group(2))) for m in re.finditer(
        r"\.amdhsa_kernel (\S+)(?:.|\n)*?\.amdhsa_private_segment_fixed_size (\d+)", text) if int(m.group(2)) > 0]
    if bad:
        raise RuntimeError(f"{src}: kernels using scratch memory (their LDS-load waits would be wrong): {bad}")


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=8) as ex:
        checks = [ex.submit(_check_no_scratch, src) for src in COUNTED]
        objs = list(ex.map(_compile, SOURCES))
        for c in checks:
            c.result()
    tmp = OUT + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, OUT)
    if verbose:
        print(f"built {OUT}")
    return OUT


# Host code of the library (argument checks, tables, the host planner) under
# AddressSanitizer and UndefinedBehaviorSanitizer: apc.cpp compiled with the
# sanitizers on its host side only, linked with the other objects of the
# normal build (their device code is unchanged).
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
            "-Xarch_host", "-g"]


def build_sanitized(out_dir: str) -> str:
    """libapc.so in out_dir with apc.cpp's host code instrumented; needs a
    normal build's objects (build() first)."""
    os.makedirs(out_dir, exist_ok=True)
    obj = os.path.join(out_dir, "apc_san.o")
    cmd = [HIPCC, *FLAGS, *SAN_HOST, "-x", "hip", "-c", os.path.join(CSRC, "apc.cpp"), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=900)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for the sanitized apc.cpp:\n{r.stderr}")
    objs = [obj] + [os.path.join(BUILD, os.path.splitext(src)[0] + ".o") for src in SOURCES if src != "apc.cpp"]
    out = os.path.join(out_dir, "libapc.so")
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libasan", *SAN_HOST, "-o", out, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized link failed:\n{r.stderr}")
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
