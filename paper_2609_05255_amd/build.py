"""Builds libgsraster.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2609_05255_amd.build

Each csrc/*.hip is compiled to an object under _build/ and the objects are
linked into paper_2609_05255_amd/libgsraster.so. Objects are rebuilt in
parallel; the link always runs.
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libgsraster.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-munsafe-fp-atomics",                       # hardware float atomics in the blend backward
    "-fhip-fp32-correctly-rounded-divide-sqrt",  # the preprocess geometry needs IEEE / and sqrt
    "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # the blend backward's atomics come from one lane per wave: no wave-level
    # pre-reduction loop around them
    "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
    "-I", os.path.join(HERE, "..", "include"),
]


# Per-file options. preprocess.hip: the decoder kernels loop over chunks of
# Gaussians, and machine-level loop-invariant code motion hoists the fp64
# exp's polynomial constants (the activations) out of that loop into vector
# register pairs, which then spill; without it the latent kernel needs 117
# registers and no spills instead of 128 and 28 bytes of scratch per lane, the
# neural one 97 instead of 123 (latent preprocess 0.138 -> 0.127 ms, neural
# 0.161 -> 0.140 ms; the other kernels' times unchanged). blend.hip: the
# scheduler's instruction-level-parallelism strategy, which keeps more loads in
# flight in the per-splat loops at the same occupancy (blend forward 0.192 ->
# 0.188 ms, backward 0.331 -> 0.324 ms at 3M Gaussians; for the other files it
# is neutral or slower, the latent decoder backward by 20 us).
PER_FILE = {
    "preprocess.hip": ["-mllvm", "-disable-machine-licm"],
    "blend.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
}


def sources():
    return sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src.replace(".hip", ".o"))
    cmd = [HIPCC, *COMMON, *PER_FILE.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr))
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(_compile, sources()))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
