"""Build libuniquan.so (all HIP sources, gfx950) in-tree with hipcc.

Each source compiles to its own object in parallel (``_build/``, not kept in
history); the objects are then linked into paper_2506_03781_amd/libuniquan.so.
Every call recompiles every source.

Numerics flags: no FMA contraction, IEEE correctly rounded fp32 division and
square root, fp32 subnormals kept (codes are decided bit-exactly in fp32);
compiler-generated packed-fp32 instructions disabled.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(os.path.dirname(HERE), "_build")
LIB = os.path.join(HERE, "libuniquan.so")
SOURCES = ["abi.hip", "fq_fwd.hip", "fq_bwd.hip", "gemm.hip", "init_unified.hip", "bcq_deploy.hip", "block_mlp.hip",
           "block_attn.hip", "attn_fused.hip", "probe.hip"]

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-fno-gpu-flush-denormals-to-zero", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if c and (os.path.sep not in c or os.path.exists(c)):
            return c
    raise RuntimeError("hipcc not found")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed with status {r.returncode}: {' '.join(cmd[-3:])}")


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every HIP source (in parallel) and link libuniquan.so."""
    os.makedirs(OBJ, exist_ok=True)
    cc = hipcc()
    objs, cmds = [], []
    for s in SOURCES:
        o = os.path.join(OBJ, s.replace(".hip", ".o"))
        objs.append(o)
        cmds.append([cc, *FLAGS, "-c", "-o", o, os.path.join(CSRC, s)])
    n = jobs or min(len(cmds), max(1, min(8, os.cpu_count() or 1)))
    with ThreadPoolExecutor(n) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    tmp = LIB + ".tmp"
    _run([cc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
