"""CU partitions (xred_stream_create_partition) on the GPU.

- Where the workgroups of a launch ran, read by the measuring library's
  placement kernel from the hardware's XCC_ID and HW_ID registers: on the
  partition's stream exactly ncu CUs, ncu / X on each of the X XCDs; on the
  rest's stream exactly the other CUs; on an ordinary stream every CU.
- Entry points on the two streams give the oracle's bits: the fused reduce
  (and, on the smallest partition, the ring in one launch, whose grid is
  sized for the whole chip and so runs in rounds there) on the partition's
  stream, a host-descriptor batch on the rest's, all enqueued before any is
  waited for; on 8 CUs also the ring gated by host flags and a batch with
  device descriptors, whose grids are sized for the whole chip.
- CU counts that are not a multiple of the XCD count, or not below the CU
  count, are rejected and create nothing.
"""
import ctypes
from collections import Counter

import numpy as np
import pytest

import gpu_util as gu
import pins
from test_gpu_ring import PinnedWords

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def env():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    from paper_2510_20171_amd import build
    xr.load()
    C = ctypes.CDLL(str(build.CEILING_OUT))
    C.xred_ceiling_placement.argtypes = [ctypes.c_void_p, ctypes.c_uint, ctypes.c_void_p]
    yield xr, C


def placement(C, stream_handle, grid):
    """{(xcd, cu address within the XCD)} used by a launch of `grid` workgroups."""
    out = torch.full((grid,), -1, dtype=torch.int32, device="cuda")
    assert C.xred_ceiling_placement(ctypes.c_void_p(out.data_ptr()), grid,
                                    ctypes.c_void_p(stream_handle)) == 0
    torch.cuda.synchronize()
    v = out.cpu().numpy().view(np.uint32)
    assert not (v == 0xFFFFFFFF).any(), "a workgroup did not record"
    return {(int(w) >> 16, int(w) & 0xFFFF) for w in v}


def every_cu(C):
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    used = placement(C, torch.cuda.current_stream().cuda_stream, 16 * cus)
    assert len(used) == cus, (len(used), cus)
    return used, len({x for x, _ in used})


@pytest.mark.parametrize("ncu", [8, 16, 64])
def test_partition_places_and_reduces(env, orc, ncu):
    xr, C = env
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    every, X = every_cu(C)
    if ncu % X:
        pytest.skip(f"{X} XCDs")
    a, b = xr.stream_create_partition(ncu)
    try:
        mine = placement(C, a, 16 * cus)
        other = placement(C, b, 16 * cus)
        assert len(mine) == ncu, sorted(mine)
        assert Counter(x for x, _ in mine) == {x: ncu // X for x in range(X)}
        assert len(other) == cus - ncu
        assert not (mine & other) and (mine | other) == every

        rng = np.random.default_rng(71 + ncu)
        n = 3 * 512 * 8 * 8 + 13
        srcs_np = [pins.random_column_values(rng, "bf16", n) for _ in range(8)]
        srcs = [gu.to_dev(s, "bf16") for s in srcs_np]
        out = torch.empty(n, dtype=torch.bfloat16, device="cuda")
        sizes = [int(x) for x in rng.integers(1, 40000, size=70)]
        bsrc_np = [[pins.random_column_values(rng, "f32", m) for _ in range(3)] for m in sizes]
        bsrc = [[gu.to_dev(s, "f32") for s in row] for row in bsrc_np]
        bout = [torch.empty(m, dtype=torch.float32, device="cuda") for m in sizes]
        torch.cuda.synchronize()
        xr.allreduce_local(srcs, out, stream=a)
        xr.batched_reduce(list(zip(bsrc, bout)), "sum", dtype="f32", stream=b)
        if ncu == 8:
            # a grid sized for the whole chip on 8 CUs: the ring with and
            # without host flags (the poller is workgroup 0, dispatched first;
            # tile workgroups wait only for it), and a device-descriptor batch
            # (the queue kernel: most of its workgroups start once the first
            # ones have taken every tile)
            chunks = [gu.to_dev(s, "bf16") for s in srcs_np[:4]]
            rout = torch.empty(n, dtype=torch.bfloat16, device="cuda")
            xr.ring_reduce(chunks, rout, stream=a)
            flags = PinnedWords(4)
            for i in range(4):
                flags.set(i, 1)
            fout = torch.empty(n, dtype=torch.bfloat16, device="cuda")
            L = xr.load()
            xr._lib.check(L.xred_ring_reduce(
                xr._lib.ptr_array([c.data_ptr() for c in chunks]), 4,
                ctypes.c_void_p(fout.data_ptr()), n, xr.DTYPE["bf16"], xr.OP["sum"], flags.dev, 1,
                2_000_000, None, ctypes.c_void_p(a)))
            dsizes = [int(x) for x in rng.integers(1, 30000, size=300)]
            dsrc_np = [[pins.random_column_values(rng, "bf16", m) for _ in range(5)] for m in dsizes]
            dsrc = [[gu.to_dev(x, "bf16") for x in row] for row in dsrc_np]
            dout = [torch.empty(m, dtype=torch.bfloat16, device="cuda") for m in dsizes]
            ptrs = [torch.tensor([x.data_ptr() for x in row], dtype=torch.int64, device="cuda")
                    for row in dsrc]
            rows = np.zeros(len(dsizes), xr.ITEM_DTYPE)
            for k, (pa, o) in enumerate(zip(ptrs, dout)):
                rows[k] = (pa.data_ptr(), o.data_ptr(), o.numel(), 5, 0)
            ditems = torch.from_numpy(rows.view(np.uint8).copy()).to("cuda")
            torch.cuda.synchronize()
            xr.batched_reduce(ditems, "sum", dtype="bf16", stream=a)
        for s in (a, b):
            torch.cuda.ExternalStream(s).synchronize()
        gu.assert_parity(out, orc.allreduce_local(srcs_np, "bf16", "sum"), "bf16", "sum",
                         f"fused on {ncu} CUs")
        for k, (row, o) in enumerate(zip(bsrc_np, bout)):
            gu.assert_parity(o, orc.allreduce_local(row, "f32", "sum"), "f32", "sum",
                             f"batch item {k} on the other {cus - ncu} CUs")
        if ncu == 8:
            ring_exp = orc.allreduce_local(srcs_np[:4], "bf16", "sum")
            gu.assert_parity(rout, ring_exp, "bf16", "sum", "one-launch ring on 8 CUs")
            gu.assert_parity(fout, ring_exp, "bf16", "sum", "flagged ring on 8 CUs")
            flags.free()
            for k, (row, o) in enumerate(zip(dsrc_np, dout)):
                gu.assert_parity(o, orc.allreduce_local(row, "bf16", "sum"), "bf16", "sum",
                                 f"device-descriptor item {k} on 8 CUs")
    finally:
        xr.stream_destroy(a)
        xr.stream_destroy(b)


def test_partition_rejects_bad_counts(env):
    xr, C = env
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    _, X = every_cu(C)
    bad = [cus, cus + X, 3 * cus]
    if X > 1:
        bad += [X - 1, X + 1, 2 * X + 3]
    for ncu in bad:
        a, b = ctypes.c_void_p(77), ctypes.c_void_p(88)
        st = xr.load().xred_stream_create_partition(ncu, ctypes.byref(a), ctypes.byref(b))
        assert st == xr.INVALID_ARGUMENT, (ncu, st)
        assert a.value is None and b.value is None
    # only the partition's stream, no rest
    a, none = xr.stream_create_partition(X, rest=False)
    try:
        assert none is None
        assert len(placement(C, a, 8 * cus)) == X
    finally:
        xr.stream_destroy(a)
