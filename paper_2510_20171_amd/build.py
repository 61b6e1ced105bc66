"""Build libxred.so for gfx950 with hipcc (in-tree, no JIT cache).

    python -m paper_2510_20171_amd.build

Every .hip file under csrc/ is compiled to an object in parallel, then linked
into paper_2510_20171_amd/libxred.so; ceiling/xred_ceiling.hip (a measuring
tool for bench.py) becomes paper_2510_20171_amd/libxred_ceiling.so.  Flags:
  --offload-arch=gfx950      MI355X only
  -ffp-contract=off          no fused multiply-add: one IEEE op per float op
  -fno-gpu-flush-denormals-to-zero   binary32 subnormals are kept
  -packed-fp32-ops (off)     no v_pk_{add,mul,fma}_f32 generated
  -fvisibility=hidden        only the xred_* C ABI is exported
  -mllvm -amdgpu-atomic-optimizer-strategy=None
                             single-lane atomics stay single-lane: the
                             optimizer turns them into wave-wide sequences
                             that wait for the atomic's result at once
                             (the batched queue claims tiles ahead)
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

PKG = Path(__file__).resolve().parent
CSRC = PKG / "csrc"
OUT = PKG / "libxred.so"
# the traffic-only ceiling kernel bench.py measures beside libxred (its own
# library: not part of libxred's interface)
CEILING_SRC = PKG / "ceiling" / "xred_ceiling.hip"
CEILING_OUT = PKG / "libxred_ceiling.so"
BUILD = PKG / "_build"
HIPCC = "/opt/rocm/bin/hipcc"

HIPFLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    "-ffp-contract=off", "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
    "-Wall", "-Wno-unused-function",
]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the gfx950 feature name; that warning is noise
    err = "\n".join(l for l in r.stderr.splitlines()
                    if "not a recognized feature for this target" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed: {' '.join(cmd)}\n{err}")
    if err.strip():
        print(err, file=sys.stderr)


def build(jobs: int = 0, verbose: bool = False) -> Path:
    """Compile every csrc/*.hip and link libxred.so; returns its path."""
    BUILD.mkdir(exist_ok=True)
    sources = sorted(CSRC.glob("*.hip"))
    objs = [BUILD / (s.stem + ".o") for s in sources]
    cmds = [[HIPCC, *HIPFLAGS, "-c", str(s), "-o", str(o)] for s, o in zip(sources, objs)]
    ceiling_tmp = CEILING_OUT.with_suffix(".so.tmp")
    cmds.append([HIPCC, *HIPFLAGS, "-shared", str(CEILING_SRC), "-o", str(ceiling_tmp)])
    if jobs <= 0:
        jobs = min(16, os.cpu_count() or 4)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        list(ex.map(_run, cmds))
    tmp = OUT.with_suffix(".so.tmp")
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *map(str, objs), "-o", str(tmp)])
    tmp.replace(OUT)
    ceiling_tmp.replace(CEILING_OUT)
    if verbose:
        print(f"built {OUT} and {CEILING_OUT}")
    return OUT


if __name__ == "__main__":
    build(verbose=True)
