"""Builds libtasq.so (the C-ABI library) and libtasq_probe.so (the benchmark's
measurement probe) for gfx950 with hipcc, in-tree."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libtasq.so")
# The benchmark's measurement probe, a library of its own (not the TASQ ABI).
PROBE_LIB = os.path.join(HERE, "libtasq_probe.so")
PROBE_SOURCES = ["probe.hip"]
OBJDIR = os.path.join(ROOT, "_build")

SOURCES = [
    "tile_256x256_k128_w8_pf1.hip",
    "tile_256x256_k64_w8_pf2.hip",
    "tile_128x128_k128_w4_pf2.hip",
    "tile_64x64_k128_w4_pf2.hip",
    "tile_256x128_k64_w4_pf2.hip",
    "tile_128x256_k64_w4_pf2.hip",
    "ptile_256x256_k128_w8.hip",
    "ptile_256x256_k64_w8.hip",
    "ptile_128x256_k128_w4.hip",
    "ptile_128x256_k64_w4.hip",
    "ptile_256x128_k64_w4.hip",
    "ptile_128x128_k64_w4.hip",
    "ptile_64x64_k128_w4.hip",
    "pack_planes.hip",
    "pack_weights.hip",
    "act_quant.hip",
    "weight_quant.hip",
    "skinny.hip",
    "splitk.hip",
    "tiles.cpp",
    "cost.cpp",
    "tasq_api.cpp",
]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Packed-FP32 instructions are switched off for every HIP source.
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", INCLUDE, "-I", CSRC]


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"]
    cmd = [HIPCC, *COMMON, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    subprocess.check_call(cmd)
    return obj


def _link(objs, out):
    tmp = out + ".tmp"
    subprocess.check_call([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs,
                           "-o", tmp])
    os.replace(tmp, out)


def build() -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    srcs = SOURCES + PROBE_SOURCES
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = dict(zip(srcs, ex.map(_compile, srcs)))
    _link([objs[s] for s in SOURCES], LIB)
    _link([objs[s] for s in PROBE_SOURCES], PROBE_LIB)
    return LIB


if __name__ == "__main__":
    print(build(), file=sys.stderr)
