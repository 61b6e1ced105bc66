"""libxred: one rank's reduce step of ReduceScatter / AllReduce on MI355X.

Thin Python binding over the C ABI in include/xred.h (argument marshalling
only; every step runs in the HIP kernels of libxred.so).  PyTorch supplies
device memory and streams: tensors are passed as data pointers and the
current HIP stream of the tensor's device is used unless one is given.

    import torch, paper_2510_20171_amd as xr
    srcs = [torch.randn(1 << 20, device="cuda", dtype=torch.bfloat16) for _ in range(8)]
    out = torch.empty_like(srcs[0])
    xr.allreduce_local(srcs, out)                     # out = srcs[0] + ... + srcs[7]

Element types are taken from the tensors (float32, bfloat16, float16,
float8_e4m3fn, float8_e5m2, int32, uint32, int64, uint64) or forced with
``dtype=`` ("f32", "bf16", "f16", "e4m3", "e5m2", "i32", "u32", "i64",
"u64"), e.g. to treat int32 storage as uint32.  Ops: "sum", "prod", "max",
"min" and, for float types where the whole fold is one call, "avg".
"""
from __future__ import annotations

import ctypes

from ._lib import (ACC_SIZE, ALIAS, DTYPE, ELEM_SIZE, EXPORTS, HIP_ERROR, INVALID_ARGUMENT,
                   ITEM_DTYPE,
                   ITEMS_ON_DEVICE, MAX_SRC, OP, OUT_OF_MEMORY, SCHEDULE, STEP_FINAL, STEP_INIT,
                   SUCCESS, UNSUPPORTED, XredError, XredItem, check, load, ptr_array)

__all__ = ["allreduce_local", "reduce_scatter_local", "reduce_copy_step", "acc_cast",
           "batched_reduce_noalloc",
           "batched_reduce", "ring_reduce", "ring_max_count", "allreduce_sim", "sim_chunk",
           "set_max_workgroups", "stream_create_partition", "stream_destroy", "pack_items", "acc_elem_size", "version", "release",
           "XredError", "load", "EXPORTS"]


def _torch_dtype_name(t) -> str:
    import torch
    m = {torch.float32: "f32", torch.bfloat16: "bf16", torch.int32: "i32",
         torch.float16: "f16", torch.int64: "i64", torch.float64: "f64", torch.int8: "i8",
         torch.uint8: "u8"}
    for name, code in (("uint32", "u32"), ("uint64", "u64"), ("float8_e4m3fn", "e4m3"),
                       ("float8_e5m2", "e5m2")):
        if hasattr(torch, name):
            m[getattr(torch, name)] = code
    try:
        return m[t.dtype]
    except KeyError:
        raise XredError(INVALID_ARGUMENT, f"tensor dtype {t.dtype} is not supported") from None


def _dtype_name(t, dtype) -> str:
    name = dtype if dtype is not None else _torch_dtype_name(t)
    if name not in DTYPE:
        raise XredError(INVALID_ARGUMENT, f"unknown dtype {name!r}")
    return name


def _dtype(t, dtype):
    return DTYPE[_dtype_name(t, dtype)]


def _require(tensors, n, es, what, device, host_ok=False):
    """Every tensor: on `device` (or pinned host memory when host_ok),
    contiguous, elements of es bytes and n elements (at least n when host_ok),
    so that the kernels never touch memory outside it."""
    for k, t in enumerate(tensors):
        if t is None:
            continue
        if t.is_cuda:
            if t.device != device:
                raise XredError(INVALID_ARGUMENT, f"{what}[{k}] is on {t.device}, not {device}")
        elif not (host_ok and t.is_pinned()):
            raise XredError(INVALID_ARGUMENT, f"{what}[{k}] is not in GPU"
                            + (" or pinned host" if host_ok else "") + " memory")
        if not t.is_contiguous():
            raise XredError(INVALID_ARGUMENT, f"{what}[{k}] is not contiguous")
        if t.element_size() != es:
            raise XredError(INVALID_ARGUMENT, f"{what}[{k}] has {t.element_size()}-byte elements,"
                            f" the dtype needs {es}")
        if t.numel() < n if host_ok else t.numel() != n:
            raise XredError(INVALID_ARGUMENT, f"{what}[{k}] has {t.numel()} elements, expected "
                            f"{'at least ' if host_ok else ''}{n}")


def _stream(t, stream):
    if stream is not None:
        return ctypes.c_void_p(int(getattr(stream, "cuda_stream", stream)))
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def allreduce_local(srcs, out, op: str = "sum", *, dtype=None, stream=None) -> None:
    """out[i] = fold_op(srcs[0][i], ..., srcs[P-1][i]) in source order (xred_allreduce_local)."""
    L = load()
    n = out.numel()
    dt = _dtype_name(out, dtype)
    _require([out], n, ELEM_SIZE[dt], "out", out.device)
    _require(srcs, n, ELEM_SIZE[dt], "srcs", out.device)
    check(L.xred_allreduce_local(ptr_array([s.data_ptr() for s in srcs]), len(srcs), _ptr(out),
                                 n, DTYPE[dt], OP[op], _stream(out, stream)))


def reduce_scatter_local(srcs, rank: int, out, op: str = "sum", *, dtype=None,
                         stream=None) -> None:
    """Shard `rank` of a ReduceScatter over full send buffers srcs (xred_reduce_scatter_local)."""
    L = load()
    dt = _dtype_name(out, dtype)
    _require([out], out.numel(), ELEM_SIZE[dt], "out", out.device)
    _require(srcs, out.numel() * len(srcs), ELEM_SIZE[dt], "srcs", out.device)
    check(L.xred_reduce_scatter_local(ptr_array([s.data_ptr() for s in srcs]), len(srcs), rank,
                                      _ptr(out), out.numel(), DTYPE[dt], OP[op],
                                      _stream(out, stream)))


def reduce_copy_step(inp, acc, out=None, op: str = "sum", *, init: bool = False,
                     final: bool = False, dtype=None, stream=None) -> None:
    """One ring ReduceCopy step into a 4-byte accumulator (xred_reduce_copy_step)."""
    L = load()
    flags = (STEP_INIT if init else 0) | (STEP_FINAL if final else 0)
    n = inp.numel()
    dt = _dtype_name(inp, dtype)
    _require([inp], n, ELEM_SIZE[dt], "in", inp.device)
    if not (init and final):
        if acc is None:
            raise XredError(INVALID_ARGUMENT, "acc is required unless init and final")
        _require([acc], n, ACC_SIZE[dt], "acc", inp.device)
    if final:
        if out is None:
            raise XredError(INVALID_ARGUMENT, "out is required with final")
        _require([out], n, ELEM_SIZE[dt], "out", inp.device)
    check(L.xred_reduce_copy_step(_ptr(inp), _ptr(acc), _ptr(out), n, DTYPE[dt], OP[op], flags,
                                  _stream(inp, stream)))


def acc_cast(acc, out, *, dtype=None, stream=None) -> None:
    """out = down(acc): closing cast of a step-wise sequence (xred_acc_cast)."""
    L = load()
    dt = _dtype_name(out, dtype)
    _require([out], out.numel(), ELEM_SIZE[dt], "out", out.device)
    _require([acc], out.numel(), ACC_SIZE[dt], "acc", out.device)
    check(L.xred_acc_cast(_ptr(acc), _ptr(out), out.numel(), DTYPE[dt], _stream(out, stream)))


def pack_items(items):
    """Host xred_item array for [(srcs_pointer_array_address, dst_ptr, count, nsrc), ...]."""
    arr = (XredItem * max(1, len(items)))()
    for k, (srcs_addr, dst, count, nsrc) in enumerate(items):
        arr[k].srcs = srcs_addr
        arr[k].dst = dst
        arr[k].count = count
        arr[k].nsrc = nsrc
        arr[k].reserved = 0
    return arr


def batched_reduce(items, op: str = "sum", *, dtype: str, stream=None, device=None) -> None:
    """Many reductions in one launch (xred_batched_reduce).

    items: list of (srcs, out) tensor pairs (descriptors built on the host,
    passed by value), or a CUDA uint8/int64 tensor holding packed xred_item
    descriptors in device memory (metadata by reference; each item's srcs
    field must point to a device array of source pointers)."""
    L = load()
    import torch
    if isinstance(items, torch.Tensor):
        if not items.is_cuda:
            raise XredError(INVALID_ARGUMENT, "device descriptors must be a CUDA tensor")
        n = items.numel() * items.element_size() // ITEM_DTYPE.itemsize
        st = _stream(items, stream)
        check(L.xred_batched_reduce(_ptr(items), n, DTYPE[dtype], OP[op], ITEMS_ON_DEVICE, st))
        return
    keep = []
    rows = []
    es = ELEM_SIZE[_dtype_name(None, dtype)]
    dev = items[0][1].device if items else None
    for k, (srcs, out) in enumerate(items):
        _require([out], out.numel(), es, f"items[{k}].out", dev)
        _require(srcs, out.numel(), es, f"items[{k}].srcs", dev)
        pa = ptr_array([s.data_ptr() for s in srcs])
        keep.append(pa)
        rows.append((ctypes.addressof(pa), out.data_ptr(), out.numel(), len(srcs)))
    arr = pack_items(rows)
    dev_t = items[0][1] if items else None
    st = _stream(dev_t, stream) if dev_t is not None else ctypes.c_void_p(0)
    check(L.xred_batched_reduce(arr, len(rows), DTYPE[dtype], OP[op], 0, st))


def batched_reduce_noalloc(items, op: str = "sum", *, dtype: str, stream=None) -> None:
    """Device-descriptor batch with no allocation (xred_batched_reduce_noalloc).

    items: a CUDA uint8/int64 tensor of packed xred_item descriptors in device
    memory, as for batched_reduce.  Calls that overlap on one GPU race."""
    L = load()
    import torch
    if not isinstance(items, torch.Tensor) or not items.is_cuda:
        raise XredError(INVALID_ARGUMENT, "device descriptors must be a CUDA tensor")
    n = items.numel() * items.element_size() // ITEM_DTYPE.itemsize
    check(L.xred_batched_reduce_noalloc(_ptr(items), n, DTYPE[dtype], OP[op],
                                        _stream(items, stream)))


def ring_reduce(chunks, out, op: str = "sum", *, ready=None, epoch: int = 1,
                timeout_us: int = 0, status=None, dtype=None, stream=None) -> None:
    """All steps of a ring ReduceCopy in one launch (xred_ring_reduce).

    ready: None, or a tensor of len(chunks) uint32/int32 flags in pinned host
    or device memory; status: None or a 1-element int32 tensor (pinned or
    device) that receives 1 if a wait timed out."""
    L = load()
    dt = _dtype_name(out, dtype)
    _require([out], out.numel(), ELEM_SIZE[dt], "out", out.device)
    _require(chunks, out.numel(), ELEM_SIZE[dt], "chunks", out.device)
    _require([ready], len(chunks), 4, "ready", out.device, host_ok=True)
    _require([status], 1, 4, "status", out.device, host_ok=True)
    check(L.xred_ring_reduce(ptr_array([c.data_ptr() for c in chunks]), len(chunks), _ptr(out),
                             out.numel(), DTYPE[dt], OP[op], _ptr(ready), epoch & 0xFFFFFFFF,
                             timeout_us, _ptr(status), _stream(out, stream)))


def allreduce_sim(sends, recvs, op: str = "sum", *, schedule: str = "ring", dtype=None,
                  stream=None) -> None:
    """A whole AllReduce over len(sends) simulated ranks on this GPU
    (xred_allreduce_sim): recvs[r] receives the reduced buffer at every rank.
    schedule: "ring" or "rhd" (recursive halving-doubling), one launch per step, or
    "ring1" / "rhd1", every step in one launch (same bits)."""
    L = load()
    if len(sends) != len(recvs):
        raise XredError(INVALID_ARGUMENT, "one recv buffer per send buffer")
    out = recvs[0]
    dt = _dtype_name(out, dtype)
    _require(recvs, out.numel(), ELEM_SIZE[dt], "recvs", out.device)
    _require(sends, out.numel(), ELEM_SIZE[dt], "sends", out.device)
    check(L.xred_allreduce_sim(ptr_array([s.data_ptr() for s in sends]),
                               ptr_array([r.data_ptr() for r in recvs]), len(sends), out.numel(),
                               DTYPE[dt], OP[op], SCHEDULE[schedule], _stream(out, stream)))


def sim_chunk(count: int, nranks: int) -> int:
    return int(load().xred_sim_chunk(count, nranks))


def ring_max_count(dtype: str) -> int:
    return int(load().xred_ring_max_count(DTYPE[dtype]))


def set_max_workgroups(n: int) -> int:
    """CU budget for later launches (0 = none); returns the previous value."""
    return int(load().xred_set_max_workgroups(n))


def stream_create_partition(ncu: int, rest: bool = True):
    """Streams on a CU partition of the current device (xred_stream_create_partition):
    (handle on ncu CUs, handle on the other CUs or None), as integers."""
    a, b = ctypes.c_void_p(), ctypes.c_void_p()
    check(load().xred_stream_create_partition(ncu, ctypes.byref(a),
                                              ctypes.byref(b) if rest else None))
    return a.value, (b.value if rest else None)


def stream_destroy(handle: int) -> None:
    """xred_stream_destroy: waits for the stream's work, then destroys it."""
    check(load().xred_stream_destroy(handle))


def acc_elem_size(dtype: str) -> int:
    return int(load().xred_acc_elem_size(DTYPE[dtype]))


def version() -> int:
    return int(load().xred_version())


def release() -> None:
    load().xred_release()
