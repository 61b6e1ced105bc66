"""The C ABI from a plain C program (tests/c/allreduce_example.c): built
with gcc against include/xred.h, libxred.so and the HIP C runtime API, with
no Python or PyTorch in the process.  Compiling and linking runs on the CPU;
running it needs a GPU (it is started as a child process)."""
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
SRC = ROOT / "tests" / "c" / "allreduce_example.c"
LIBDIR = ROOT / "paper_2510_20171_amd"


def _build(out: Path) -> Path:
    if not (LIBDIR / "libxred.so").exists():
        pytest.skip("libxred.so is not built")
    cmd = ["gcc", "-std=c11", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I/opt/rocm/include", f"-I{ROOT / 'include'}", str(SRC), f"-L{LIBDIR}", "-lxred",
           "-L/opt/rocm/lib", "-lamdhip64", f"-Wl,-rpath,{LIBDIR}", "-Wl,-rpath,/opt/rocm/lib",
           "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return out


def test_c_program_builds(tmp_path):
    assert _build(tmp_path / "xred_example").exists()


@pytest.mark.gpu
def test_c_program_runs(tmp_path):
    exe = _build(tmp_path / "xred_example")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert "sum exact" in r.stdout and "overlap rejected" in r.stdout, r.stdout
