"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, the header is valid C, and argument validation rejects bad calls
before any HIP call is made (so these run on a CPU-only machine)."""
import ctypes
import re
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
HEADER = ROOT / "include" / "xred.h"


@pytest.fixture(scope="module")
def L():
    import paper_2510_20171_amd as xr
    if not xr._lib.LIB_PATH.exists():
        from paper_2510_20171_amd import build
        build.build()
    return xr.load()


def declared_functions():
    text = HEADER.read_text()
    return re.findall(r"XRED_API\s+[\w\s\*]+?\b(xred_\w+)\s*\(", text)


def test_header_declares_the_boundary():
    names = set(declared_functions())
    assert {"xred_allreduce_local", "xred_reduce_scatter_local", "xred_reduce_copy_step",
            "xred_acc_cast", "xred_batched_reduce"} <= names


def test_exports_every_declared_symbol(L):
    import paper_2510_20171_amd as xr
    names = declared_functions()
    assert sorted(names) == sorted(xr.EXPORTS)
    for n in names:
        assert hasattr(L, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", str(xr._lib.LIB_PATH)],
                         capture_output=True, text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    assert exported == set(names), exported ^ set(names)


def test_measuring_library_exports(L):
    """bench.py's measuring kernels (stream-mix ceiling, flag handoff) are a
    library of their own, not part of libxred's interface."""
    from paper_2510_20171_amd import build
    lib = build.CEILING_OUT
    assert lib.exists()
    out = subprocess.run(["nm", "-D", "--defined-only", str(lib)],
                         capture_output=True, text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    assert {"xred_ceiling_mix", "xred_ceiling_handoff", "xred_ceiling_placement"} <= exported, \
        exported
    C = ctypes.CDLL(str(lib))
    f = C.xred_ceiling_handoff
    f.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_void_p]
    # argument checks come before any HIP call (hipErrorInvalidValue = 1)
    assert f(0, 0, 1000, None, None, None, None) == 1
    assert f(4, 0, 0, None, None, None, None) == 1
    g = C.xred_ceiling_placement
    g.argtypes = [ctypes.c_void_p, ctypes.c_uint, ctypes.c_void_p]
    assert g(None, 16, None) == 1
    assert g(ctypes.c_void_p(4096), 0, None) == 1


@pytest.mark.parametrize("compiler,lang", [("gcc", "c"), ("g++", "c++")])
def test_header_compiles(tmp_path, compiler, lang):
    src = tmp_path / ("t.c" if lang == "c" else "t.cpp")
    src.write_text('#include "xred.h"\nint main(void){ xred_item it; (void)it; '
                   'return (int)sizeof(xred_item) == 32 ? 0 : 1; }\n')
    exe = tmp_path / "t"
    subprocess.run([compiler, "-std=c11" if lang == "c" else "-std=c++17", "-Wall", "-Werror",
                    f"-I{ROOT / 'include'}", str(src), "-o", str(exe)], check=True)
    assert subprocess.run([str(exe)]).returncode == 0


def test_constants(L):
    assert L.xred_version() == 20301   # 2.3.1: major*10000 + minor*100 + patch
    assert L.xred_acc_elem_size(0) == 4 and L.xred_acc_elem_size(1) == 4
    assert L.xred_acc_elem_size(2) == 4 and L.xred_acc_elem_size(7) == 4
    assert L.xred_acc_elem_size(5) == 8 and L.xred_acc_elem_size(6) == 8
    assert L.xred_acc_elem_size(9) == 8                                  # fp64: binary64
    assert L.xred_acc_elem_size(10) == 4 and L.xred_acc_elem_size(11) == 4   # int8/uint8: uint32
    assert L.xred_acc_elem_size(12) == 0 and L.xred_acc_elem_size(99) == 0
    assert L.xred_status_string(0) == b"success"
    assert L.xred_status_string(3) == b"buffers overlap"


# Fake device addresses: validation never dereferences them.
A = 0x7F0000000000
S = ctypes.c_void_p


def ptrs(*xs):
    return (ctypes.c_void_p * len(xs))(*xs)




@pytest.mark.parametrize("case,expect", [
    (lambda L: L.xred_allreduce_local(ptrs(A), 0, S(A + 4096), 16, 0, 0, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(A), 65, S(A + 4096), 16, 0, 0, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(A), 1, S(A + 4096), 16, 99, 0, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(A), 1, S(A + 4096), 16, 0, 9, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(A), 1, S(A + 4096), 16, 3, 4, None), 2),  # int AVG
    (lambda L: L.xred_allreduce_local(ptrs(A), 1, S(A + 4096), 16, 12, 0, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(A + 4), 1, S(A + 4096), 16, 9, 0, None), 1),  # f64 align
    (lambda L: L.xred_allreduce_local(ptrs(A), 1, S(A + 4096), 16, 10, 4, None), 2),  # int8 AVG
    (lambda L: L.xred_allreduce_local(ptrs(A), 1, S(A + 4096), 16, 11, 4, None), 2),  # uint8 AVG
    (lambda L: L.xred_allreduce_local(ptrs(A), 1, S(A + 4096), 16, 0, 5, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(A + 4), 1, S(A + 4096), 16, 5, 0, None), 1),  # i64 align
    (lambda L: L.xred_allreduce_local(None, 1, S(A + 4096), 16, 0, 0, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(0), 1, S(A + 4096), 16, 0, 0, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(A), 1, S(0), 16, 0, 0, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(A + 2), 1, S(A + 4096), 16, 0, 0, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(A + 1), 1, S(A + 4096), 16, 1, 0, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(A), 1, S(A + 4096), 2**62, 0, 0, None), 1),
    (lambda L: L.xred_allreduce_local(ptrs(A, A + 8), 2, S(A + 4), 4, 0, 0, None), 3),
    (lambda L: L.xred_allreduce_local(ptrs(A, A + 1024), 2, S(A + 1020), 4, 0, 0, None), 3),
    (lambda L: L.xred_reduce_scatter_local(ptrs(A, A + 4096), 2, 2, S(A + 8192), 4, 0, 0, None), 1),
    (lambda L: L.xred_reduce_scatter_local(ptrs(A, A + 4096), 2, -1, S(A + 8192), 4, 0, 0, None), 1),
    (lambda L: L.xred_reduce_scatter_local(ptrs(A, A + 4096), 2, 1, S(A + 4), 4, 0, 0, None), 3),
    (lambda L: L.xred_reduce_scatter_local(ptrs(A, A + 4096), 2, 0, S(A + 4096 - 8), 4, 0, 0, None), 3),
    (lambda L: L.xred_reduce_copy_step(S(A), S(A + 4096), S(0), 16, 0, 0, 4, None), 1),
    (lambda L: L.xred_reduce_copy_step(S(A), S(0), S(0), 16, 1, 0, 0, None), 1),
    (lambda L: L.xred_reduce_copy_step(S(A), S(A + 4096), S(0), 16, 1, 0, 2, None), 1),
    (lambda L: L.xred_reduce_copy_step(S(A), S(A + 16), S(0), 16, 1, 0, 0, None), 3),
    (lambda L: L.xred_reduce_copy_step(S(A), S(A + 4096), S(A + 4096 + 8), 16, 1, 0, 2, None), 3),
    (lambda L: L.xred_reduce_copy_step(S(A), S(A + 4096), S(A + 8193), 16, 1, 0, 2, None), 1),
    (lambda L: L.xred_acc_cast(S(A), S(A + 8), 16, 1, None), 3),
    (lambda L: L.xred_acc_cast(S(A + 2), S(A + 4096), 16, 1, None), 1),
    (lambda L: L.xred_batched_reduce(None, -1, 1, 0, 0, None), 1),
    (lambda L: L.xred_batched_reduce(None, 1, 1, 0, 0, None), 1),
    (lambda L: L.xred_batched_reduce(None, 1, 1, 0, 4, None), 1),
    (lambda L: L.xred_ring_reduce(ptrs(A), 0, S(A + 4096), 16, 1, 0, None, 1, 0, None, None), 1),
    (lambda L: L.xred_ring_reduce(ptrs(A), 65, S(A + 4096), 16, 1, 0, None, 1, 0, None, None), 1),
    (lambda L: L.xred_ring_reduce(ptrs(A + 2, A + 4096), 2, S(A + 8192), 16, 1, 0, None, 1, 0, None,
                                  None), 2),
    (lambda L: L.xred_ring_reduce(ptrs(A), 1, S(A + 8), 16, 1, 0, None, 1, 0, None, None), 3),
    (lambda L: L.xred_ring_reduce(ptrs(A), 1, S(A + 4096), 16, 1, 0, S(A + 1), 1, 0, None, None), 1),
    (lambda L: L.xred_ring_reduce(ptrs(A), 1, S(A + 4096), 16, 1, 4, None, 1, 0, None, None), 2),
    (lambda L: L.xred_reduce_copy_step(S(A), S(A + 4096), S(0), 16, 0, 4, 0, None), 2),  # AVG
    (lambda L: L.xred_reduce_copy_step(S(A), S(A + 4100), S(0), 16, 5, 0, 0, None), 1),  # u64 acc
    (lambda L: L.xred_reduce_copy_step(S(A), S(A + 4100), S(0), 16, 9, 0, 0, None), 1),  # f64 acc
    (lambda L: L.xred_reduce_copy_step(S(A), S(A + 4098), S(0), 16, 10, 0, 0, None), 1),  # i8 acc
    (lambda L: L.xred_reduce_copy_step(S(A), S(A + 4096), S(0), 16, 9, 4, 0, None), 2),  # f64 AVG
    # xred_allreduce_sim(sends, recvs, nranks, count, dtype, op, schedule, stream)
    (lambda L: L.xred_allreduce_sim(ptrs(A), ptrs(A + 8192), 0, 16, 1, 0, 0, None), 1),
    (lambda L: L.xred_allreduce_sim(ptrs(A), ptrs(A + 8192), 65, 16, 1, 0, 0, None), 1),
    (lambda L: L.xred_allreduce_sim(ptrs(A), ptrs(A + 8192), 1, 16, 1, 0, 4, None), 1),
    (lambda L: L.xred_allreduce_sim(ptrs(A), ptrs(A + 8192), 1, 16, 1, 0, -1, None), 1),
    (lambda L: L.xred_allreduce_sim(ptrs(A, A + 4096, A + 8192), ptrs(A + 16384, A + 20480, A + 24576),
                                    3, 16, 1, 0, 1, None), 1),
    (lambda L: L.xred_allreduce_sim(ptrs(A, A + 4096, A + 8192), ptrs(A + 16384, A + 20480, A + 24576),
                                    3, 16, 1, 0, 3, None), 1),
    (lambda L: L.xred_allreduce_sim(ptrs(A, A + 4096), ptrs(A + 8192, A + 12288), 2, 16, 1, 4, 2,
                                    None), 2),
    (lambda L: L.xred_allreduce_sim(None, ptrs(A + 8192), 1, 16, 1, 0, 0, None), 1),
    (lambda L: L.xred_allreduce_sim(ptrs(A, A + 4096), ptrs(A + 8192, 0), 2, 16, 1, 0, 0, None), 1),
    (lambda L: L.xred_allreduce_sim(ptrs(A, A + 4097), ptrs(A + 8192, A + 12288), 2, 16, 1, 0, 0,
                                    None), 1),
    (lambda L: L.xred_allreduce_sim(ptrs(A, A + 4096), ptrs(A + 8192, A + 16), 2, 16, 1, 0, 0, None), 3),
    (lambda L: L.xred_allreduce_sim(ptrs(A, A + 4096), ptrs(A + 8192, A + 8200), 2, 16, 1, 0, 0,
                                    None), 3),
    (lambda L: L.xred_allreduce_sim(ptrs(A, A + 4096), ptrs(A + 8, A + 12288), 2, 16, 1, 0, 0, None), 3),
    (lambda L: L.xred_allreduce_sim(ptrs(A, A + 4096), ptrs(A + 8192, A + 12288), 2, 16, 1, 4, 0,
                                    None), 2),
    (lambda L: L.xred_allreduce_sim(ptrs(A), ptrs(A + 8192), 1, 2**62, 0, 0, 0, None), 1),
])
def test_validation_rejects_before_launch(L, case, expect):
    assert case(L) == expect
    assert L.xred_last_error() != b""


def _item(srcs, dst, count, nsrc, reserved=0):
    import paper_2510_20171_amd as xr
    it = xr.XredItem()
    it.srcs = ctypes.cast(srcs, ctypes.c_void_p) if srcs is not None else None
    it.dst, it.count, it.nsrc, it.reserved = dst, count, nsrc, reserved
    return it


@pytest.mark.parametrize("make,expect", [
    (lambda p: [_item(p, A + 8192, 16, 1, reserved=1)], 1),
    (lambda p: [_item(p, A + 8192, 16, 0)], 1),
    (lambda p: [_item(p, A + 8192, 16, 65)], 1),
    (lambda p: [_item(None, A + 8192, 16, 1)], 1),
    (lambda p: [_item(p, 0, 16, 1)], 1),
    (lambda p: [_item(p, A + 4, 16, 1)], 3),
    (lambda p: [_item(p, A + 8192, 2**62, 1)], 1),
])
def test_batched_host_validation(L, make, expect):
    p = ptrs(A)
    items = make(p)
    arr = (type(items[0]) * len(items))(*items)
    assert L.xred_batched_reduce(arr, len(items), 0, 0, 0, None) == expect


def test_zero_counts_succeed_without_launch(L):
    assert L.xred_allreduce_local(ptrs(A), 1, S(A + 4096), 0, 1, 0, None) == 0
    assert L.xred_reduce_scatter_local(ptrs(A), 1, 0, S(A + 4096), 0, 1, 0, None) == 0
    assert L.xred_reduce_copy_step(S(A), S(A + 4096), S(0), 0, 1, 0, 0, None) == 0
    assert L.xred_acc_cast(S(A), S(A + 4096), 0, 1, None) == 0
    assert L.xred_batched_reduce(None, 0, 1, 0, 0, None) == 0
    p = ptrs(A)
    it = (type(_item(p, A, 0, 1)) * 2)(_item(p, A + 4096, 0, 1), _item(None, 0, 0, 0))
    assert L.xred_batched_reduce(it, 2, 1, 0, 0, None) == 0
    assert L.xred_allreduce_sim(ptrs(A, A + 4096), ptrs(A + 8192, A + 12288), 2, 0, 1, 0, 0,
                                None) == 0


def test_partition_argument_checks(L):
    """The CU partition's argument checks that need no device: a NULL stream
    slot or a CU count below one is rejected, and nothing is written to the
    slots but NULL."""
    a, b = ctypes.c_void_p(1234), ctypes.c_void_p(5678)
    assert L.xred_stream_create_partition(16, None, ctypes.byref(b)) == 1
    assert L.xred_stream_create_partition(0, ctypes.byref(a), ctypes.byref(b)) == 1
    assert a.value is None and b.value is None
    a = ctypes.c_void_p(1234)
    assert L.xred_stream_create_partition(-8, ctypes.byref(a), None) == 1
    assert a.value is None
    assert L.xred_stream_destroy(None) == 1


def test_sim_chunk_rule(L):
    """ceil(count / G) rounded up to 64 elements, as the oracle's schedules use."""
    import pins
    for count in (0, 1, 63, 64, 65, 1000, 64 * 8 + 70, (1 << 26) + 5):
        for G in (1, 2, 3, 7, 8, 64):
            assert L.xred_sim_chunk(count, G) == pins.sim_chunk_len(count, G)
    assert L.xred_sim_chunk(100, 0) == 0


def test_python_layer_raises(L):
    import paper_2510_20171_amd as xr
    with pytest.raises(xr.XredError) as e:
        xr._lib.check(L.xred_allreduce_local(ptrs(A), 0, S(A), 16, 0, 0, None))
    assert e.value.name == "XRED_INVALID_ARGUMENT"
    assert "nsrc" in str(e.value)


def test_torch_dtypes_map_to_codes():
    """Element types taken from tensors: the new ones included."""
    torch = pytest.importorskip("torch")
    import paper_2510_20171_amd as xr
    cases = {torch.float32: "f32", torch.bfloat16: "bf16", torch.float16: "f16",
             torch.int32: "i32", torch.int64: "i64", torch.float64: "f64", torch.int8: "i8",
             torch.uint8: "u8"}
    for name, code in (("float8_e4m3fn", "e4m3"), ("float8_e5m2", "e5m2"), ("uint32", "u32"),
                       ("uint64", "u64")):
        if hasattr(torch, name):
            cases[getattr(torch, name)] = code
    for dt, code in cases.items():
        assert xr._torch_dtype_name(torch.empty(1, dtype=dt)) == code
        assert xr._dtype(torch.empty(1, dtype=dt), None) == xr.DTYPE[code]
    with pytest.raises(xr.XredError):
        xr._torch_dtype_name(torch.empty(1, dtype=torch.complex64))


def test_product_does_not_import_oracle():
    """The product package never refers to the oracle."""
    pkg = ROOT / "paper_2510_20171_amd"
    for f in list(pkg.rglob("*.py")) + list(pkg.rglob("*.hip")) + list(pkg.rglob("*.hpp")):
        text = f.read_text()
        assert "oracle" not in text.lower().replace("oracle-exact", ""), f
