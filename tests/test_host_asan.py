"""The library's host code under AddressSanitizer (CPU only): xred_api.hip,
where all argument validation, dispatch and batch staging live, is rebuilt
with its host half instrumented (`-Xarch_host -fsanitize=address`; device
code is unaffected) and linked with the other objects into a private copy of
libxred.so, which tests/c/host_validation.c then drives through every entry
point with exact-size heap arrays.  Runs only where no GPU is visible: its
pointers are not real device memory."""
import os
import shutil
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
SRC = ROOT / "tests" / "c" / "host_validation.c"
CLANG = "/opt/rocm/llvm/bin/clang"


def _gpu_visible() -> bool:
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return False


def test_host_code_under_asan(tmp_path):
    from paper_2510_20171_amd import build
    if _gpu_visible():
        pytest.skip("a GPU is visible: the driver's pointers are not device memory")
    if not Path(CLANG).exists() or shutil.which(build.HIPCC) is None and not Path(build.HIPCC).exists():
        pytest.skip("no ROCm clang / hipcc")
    objs = sorted(build.BUILD.glob("*.o"))
    if not objs:
        build.build()
        objs = sorted(build.BUILD.glob("*.o"))
    api_obj = tmp_path / "xred_api.o"
    subprocess.run([build.HIPCC, *build.HIPFLAGS, "-Xarch_host", "-fsanitize=address",
                    "-Xarch_host", "-fno-omit-frame-pointer", "-c",
                    str(build.CSRC / "xred_api.hip"), "-o", str(api_obj)],
                   check=True, capture_output=True, text=True)
    lib = tmp_path / "libxred.so"
    others = [str(o) for o in objs if o.name != "xred_api.o"]
    subprocess.run([build.HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *others,
                    str(api_obj), "-o", str(lib)], check=True, capture_output=True, text=True)
    exe = tmp_path / "host_validation"
    subprocess.run([CLANG, "-std=c11", "-Wall", "-Werror", "-fsanitize=address",
                    "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    f"-I{ROOT / 'include'}", str(SRC), f"-L{tmp_path}", "-lxred",
                    "-L/opt/rocm/lib", "-lamdhip64", f"-Wl,-rpath,{tmp_path}",
                    "-Wl,-rpath,/opt/rocm/lib", "-o", str(exe)],
                   check=True, capture_output=True, text=True)
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"
    env.pop("XRED_TRACE", None)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all host checks passed" in r.stdout, r.stdout + r.stderr
    assert "AddressSanitizer" not in r.stderr, r.stderr
