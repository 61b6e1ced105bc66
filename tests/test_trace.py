"""The optional launch trace (XRED_TRACE in the environment, read once per
process): entry points log their arguments, failures their message and
launches their kernel and grid, on stderr; unset, nothing is printed.  Each
case runs in a child process, since the setting is read once."""
import os
import subprocess
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]

CPU_CALL = """
import ctypes
import paper_2510_20171_amd as xr
L = xr.load()
# nsrc = 0 fails validation before any HIP call
st = L.xred_allreduce_local(None, 0, None, 16, 1, 0, None)
assert st == xr.INVALID_ARGUMENT, st
"""

GPU_CALL = """
import torch
import paper_2510_20171_amd as xr
srcs = [torch.ones(4096, dtype=torch.bfloat16, device="cuda") for _ in range(3)]
out = torch.empty_like(srcs[0])
xr.allreduce_local(srcs, out)
torch.cuda.synchronize()
assert bool((out.float() == 3).all())
"""


def run(code, trace):
    env = dict(os.environ)
    env.pop("XRED_TRACE", None)
    if trace is not None:
        env["XRED_TRACE"] = trace
    return subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True,
                          text=True, timeout=300)


@pytest.fixture(scope="module", autouse=True)
def built():
    import paper_2510_20171_amd as xr
    if not xr._lib.LIB_PATH.exists():
        from paper_2510_20171_amd import build
        build.build()


def test_trace_logs_calls_and_failures():
    r = run(CPU_CALL, "1")
    assert r.returncode == 0, r.stderr
    lines = [l for l in r.stderr.splitlines() if l.startswith("[xred] ")]
    assert lines[0] == ("[xred] xred_allreduce_local nsrc=0 count=16 dtype=1 op=0 "
                        "stream=(nil)"), lines
    assert lines[1].startswith("[xred] failed (status 1): nsrc = 0 outside 1..64"), lines


@pytest.mark.parametrize("value", [None, "0", ""])
def test_trace_off(value):
    r = run(CPU_CALL, value)
    assert r.returncode == 0, r.stderr
    assert "[xred]" not in r.stderr


@pytest.mark.gpu
def test_trace_logs_launches():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    r = run(GPU_CALL, "1")
    assert r.returncode == 0, r.stderr
    lines = [l for l in r.stderr.splitlines() if l.startswith("[xred] ")]
    assert lines[0].startswith("[xred] xred_allreduce_local nsrc=3 count=4096 dtype=1 op=0"), lines
    launch = [l for l in lines if l.startswith("[xred] launch ")]
    assert len(launch) == 1, lines
    assert "reduce_vec_kernel" in launch[0] and launch[0].endswith("-> hipSuccess"), launch
