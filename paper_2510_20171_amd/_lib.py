"""ctypes loader for libxred.so (the HIP C ABI declared in include/xred.h).

There is no fallback: if the library is not built this module raises on
first use, so no computation can silently happen anywhere but in the HIP
kernels.
"""
from __future__ import annotations

import ctypes
from pathlib import Path

import numpy as np

LIB_PATH = Path(__file__).resolve().parent / "libxred.so"

# Values of the enums in include/xred.h.
DTYPE = {"f32": 0, "bf16": 1, "f16": 2, "i32": 3, "u32": 4, "i64": 5, "u64": 6, "e4m3": 7,
         "e5m2": 8, "f64": 9, "i8": 10, "u8": 11}
ELEM_SIZE = {"f32": 4, "bf16": 2, "f16": 2, "i32": 4, "u32": 4, "i64": 8, "u64": 8, "e4m3": 1,
             "e5m2": 1, "f64": 8, "i8": 1, "u8": 1}
ACC_SIZE = {d: 8 if d in ("i64", "u64", "f64") else 4 for d in DTYPE}
OP = {"sum": 0, "prod": 1, "max": 2, "min": 3, "avg": 4}
STATUS = {0: "XRED_SUCCESS", 1: "XRED_INVALID_ARGUMENT", 2: "XRED_UNSUPPORTED", 3: "XRED_ALIAS",
          4: "XRED_HIP_ERROR", 5: "XRED_OUT_OF_MEMORY"}
SUCCESS, INVALID_ARGUMENT, UNSUPPORTED, ALIAS, HIP_ERROR, OUT_OF_MEMORY = range(6)
MAX_SRC = 64
STEP_INIT, STEP_FINAL = 1, 2
ITEMS_ON_DEVICE = 1
SCHEDULE = {"ring": 0, "rhd": 1, "ring1": 2, "rhd1": 3}   # 1: every step in one launch

# struct xred_item (32 bytes)
ITEM_DTYPE = np.dtype([("srcs", "<u8"), ("dst", "<u8"), ("count", "<u8"), ("nsrc", "<u4"),
                       ("reserved", "<u4")])
assert ITEM_DTYPE.itemsize == 32


class XredItem(ctypes.Structure):
    _fields_ = [("srcs", ctypes.c_void_p), ("dst", ctypes.c_void_p), ("count", ctypes.c_uint64),
                ("nsrc", ctypes.c_uint32), ("reserved", ctypes.c_uint32)]


EXPORTS = ("xred_allreduce_local", "xred_reduce_scatter_local", "xred_reduce_copy_step",
           "xred_acc_cast", "xred_batched_reduce", "xred_batched_reduce_noalloc",
           "xred_ring_reduce", "xred_ring_max_count",
           "xred_allreduce_sim", "xred_sim_chunk", "xred_set_max_workgroups",
           "xred_stream_create_partition", "xred_stream_destroy", "xred_acc_elem_size",
           "xred_status_string",
           "xred_last_error", "xred_version", "xred_release")

_lib = None


class XredError(RuntimeError):
    """A libxred call returned a status other than XRED_SUCCESS."""

    def __init__(self, status: int, detail: str):
        self.status = status
        self.name = STATUS.get(status, f"status {status}")
        super().__init__(f"{self.name}: {detail}")


def load(path: Path = LIB_PATH) -> ctypes.CDLL:
    """Load libxred.so (once) and declare the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not Path(path).exists():
        raise ImportError(f"{path} is not built: run `python -m paper_2510_20171_amd.build` "
                          "(there is no CPU fallback)")
    # The binding hands over torch's device pointers and streams, so the
    # library must resolve libamdhip64 to the runtime torch already holds.
    # Loaded first, it would map the system ROCm runtime as a second HIP
    # runtime in the process, one that knows none of torch's allocations or
    # streams (and may fail to open the device torch has open).
    import torch  # noqa: F401
    L = ctypes.CDLL(str(path))
    vp, i32, sz, u32 = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_uint
    L.xred_allreduce_local.argtypes = [vp, i32, vp, sz, i32, i32, vp]
    L.xred_reduce_scatter_local.argtypes = [vp, i32, i32, vp, sz, i32, i32, vp]
    L.xred_reduce_copy_step.argtypes = [vp, vp, vp, sz, i32, i32, u32, vp]
    L.xred_acc_cast.argtypes = [vp, vp, sz, i32, vp]
    L.xred_batched_reduce.argtypes = [vp, i32, i32, i32, u32, vp]
    L.xred_batched_reduce_noalloc.argtypes = [vp, i32, i32, i32, vp]
    L.xred_ring_reduce.argtypes = [vp, i32, vp, sz, i32, i32, vp, ctypes.c_uint32,
                                   ctypes.c_uint64, vp, vp]
    L.xred_allreduce_sim.argtypes = [vp, vp, i32, sz, i32, i32, i32, vp]
    L.xred_sim_chunk.argtypes = [sz, i32]
    L.xred_sim_chunk.restype = sz
    L.xred_ring_max_count.argtypes = [i32]
    L.xred_ring_max_count.restype = sz
    for f in ("xred_allreduce_local", "xred_reduce_scatter_local", "xred_reduce_copy_step",
              "xred_acc_cast", "xred_batched_reduce", "xred_batched_reduce_noalloc",
              "xred_ring_reduce", "xred_allreduce_sim", "xred_stream_create_partition",
              "xred_stream_destroy"):
        getattr(L, f).restype = ctypes.c_int
    L.xred_stream_create_partition.argtypes = [i32, ctypes.POINTER(vp), ctypes.POINTER(vp)]
    L.xred_stream_destroy.argtypes = [vp]
    L.xred_set_max_workgroups.argtypes = [ctypes.c_uint]
    L.xred_set_max_workgroups.restype = ctypes.c_uint
    L.xred_acc_elem_size.argtypes = [i32]
    L.xred_acc_elem_size.restype = sz
    L.xred_status_string.argtypes = [i32]
    L.xred_status_string.restype = ctypes.c_char_p
    L.xred_last_error.argtypes = []
    L.xred_last_error.restype = ctypes.c_char_p
    L.xred_version.argtypes = []
    L.xred_version.restype = ctypes.c_int
    L.xred_release.argtypes = []
    L.xred_release.restype = None
    _lib = L
    return L


def check(status: int) -> None:
    """Raise XredError for a non-success status, with the library's detail."""
    if status != SUCCESS:
        raise XredError(status, (load().xred_last_error() or b"").decode())


def ptr_array(ptrs) -> ctypes.Array:
    """A host array of device pointers (void*[n])."""
    return (ctypes.c_void_p * max(1, len(ptrs)))(*[int(p) for p in ptrs])
