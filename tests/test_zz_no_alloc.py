"""xred_batched_reduce_noalloc: the device-descriptor batched reduce with its
tile counters in the library's fixed device array instead of memory the
library allocates.

Two calls in a row on one stream, with no synchronisation between them, the
second with a smaller batch (fewer items and tiles, so a counter left
nonzero by the first call would skip part of it), each compared element by
element with xred_batched_reduce (XRED_ITEMS_ON_DEVICE) on the same inputs
and with the oracle: bit-exact, NaN payloads of float sums compared by
NaN-ness only.  Both calls go through the C ABI (ctypes).
"""
import ctypes

import numpy as np
import pytest

import gpu_util as gu
import pins

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def xr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    xr.load()
    return xr


class DeviceBatch:
    """K items of random sources on the device; two output sets, one per entry
    point; descriptors (one table per output set) in device memory."""

    def __init__(self, xr, rng, dtype, K):
        tile = 512 * (16 // gu.NP_BITS[dtype]().itemsize)
        self.dtype, self.host, self.keep = dtype, [], []
        self.outs = ([], [])
        rows = ([], [])
        for k in range(K):
            n = int(rng.choice([1, 7, tile - 1, tile + 3, 3 * tile, 5 * tile + 11]))
            P = int(rng.choice([1, 2, 3, 8, 9]))
            srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
            dev = [gu.to_dev(s, dtype) for s in srcs]
            pa = torch.tensor([d.data_ptr() for d in dev], dtype=torch.int64, device="cuda")
            self.keep += dev + [pa]
            self.host.append(srcs)
            for j in range(2):
                out = torch.zeros(n, dtype=gu.torch_dtype(dtype), device="cuda")
                self.outs[j].append(out)
                rows[j].append((pa.data_ptr(), out.data_ptr(), n, P, 0))
        self.items = []
        for j in range(2):
            arr = np.zeros(K, xr.ITEM_DTYPE)
            for k, r in enumerate(rows[j]):
                arr[k] = r
            self.items.append(torch.from_numpy(arr.view(np.uint8).copy()).to("cuda"))
        self.K = K


def _call(fn, xr, items, K, dtype, stream, *extra):
    st = fn(ctypes.c_void_p(items.data_ptr()), K, xr.DTYPE[dtype], xr.OP["sum"], *extra,
            ctypes.c_void_p(stream.cuda_stream))
    xr._lib.check(st)


def test_noalloc_matches_device_entry_point_twice(xr, orc):
    L = xr.load()
    rng = np.random.default_rng(7700)
    big = DeviceBatch(xr, rng, "bf16", 300)
    small = DeviceBatch(xr, rng, "bf16", 70)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    # the two calls back to back on one stream, then the existing entry point
    _call(L.xred_batched_reduce_noalloc, xr, big.items[0], big.K, "bf16", stream)
    _call(L.xred_batched_reduce_noalloc, xr, small.items[0], small.K, "bf16", stream)
    _call(L.xred_batched_reduce, xr, big.items[1], big.K, "bf16", stream, xr.ITEMS_ON_DEVICE)
    _call(L.xred_batched_reduce, xr, small.items[1], small.K, "bf16", stream, xr.ITEMS_ON_DEVICE)
    torch.cuda.synchronize()
    for name, b in (("first call", big), ("second call", small)):
        for k in range(b.K):
            ref = b.outs[1][k]
            gu.assert_parity(b.outs[0][k], ref, "bf16", "sum", f"{name}, item {k} vs entry point")
            gu.assert_parity(b.outs[0][k], orc.allreduce_local(b.host[k], "bf16", "sum"),
                             "bf16", "sum", f"{name}, item {k} vs oracle")


def test_noalloc_limits(xr):
    """Past 16384 items the call is refused before anything is enqueued;
    zero items succeed without a launch."""
    L = xr.load()
    items = torch.zeros(32 * 16385, dtype=torch.uint8, device="cuda")
    st = L.xred_batched_reduce_noalloc(ctypes.c_void_p(items.data_ptr()), 16385, xr.DTYPE["f32"],
                                       xr.OP["sum"], None)
    assert st == xr.UNSUPPORTED
    assert b"16384" in L.xred_last_error()
    assert L.xred_batched_reduce_noalloc(ctypes.c_void_p(items.data_ptr()), 0, xr.DTYPE["f32"],
                                         xr.OP["sum"], None) == 0
