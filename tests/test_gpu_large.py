"""Buffers larger than 4 GiB: byte offsets past 2^32 on the fused, reduce-scatter
and batched paths.  Inputs are random bit patterns drawn on the device by
PyTorch's seeded generator (values from neither the oracle nor libxred); the
oracle computes sampled columns one by one: random indices plus the elements
around the 4 GiB byte boundary and the ragged tail.
"""
import numpy as np
import pytest

import gpu_util as gu

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def xr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    xr.load()
    return xr


def _random_bits(n, es, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    view = {1: torch.uint8, 2: torch.int16, 8: torch.int64}[es]
    lo, hi = (0, 256) if es == 1 else (-(2 ** (8 * es - 1)), 2 ** (8 * es - 1) - 1)
    return torch.randint(lo, hi, (n,), generator=g, dtype=view, device="cuda")


def _samples(n, es, rng):
    edge = (1 << 32) // es                       # first element past 4 GiB
    idx = set(rng.integers(0, n, 1 << 16).tolist())
    idx |= {i for i in range(edge - 64, edge + 64)} | {i for i in range(n - 64, n)} | {0}
    return torch.tensor(sorted(i for i in idx if 0 <= i < n), dtype=torch.int64, device="cuda")


@pytest.mark.parametrize("dtype,op,n", [("bf16", "sum", (1 << 31) + (1 << 20) + 3),
                                        ("e4m3", "max", (1 << 32) + 4099),
                                        ("i64", "sum", (1 << 29) + 777)])
def test_fused_past_4gib(xr, orc, dtype, op, n):
    es = {"bf16": 2, "e4m3": 1, "i64": 8}[dtype]
    srcs = [_random_bits(n, es, 900 + p) for p in range(2)]
    out = torch.empty_like(srcs[0])
    xr.allreduce_local(srcs, out, op, dtype=dtype)
    torch.cuda.synchronize()
    idx = _samples(n, es, np.random.default_rng(5))
    cols = [gu.bits(s[idx], dtype).copy() for s in srcs]
    exp = orc.allreduce_local([c.view(gu.NP_BITS[dtype]) if dtype != "i64" else c.view(np.int64)
                               for c in cols], dtype, op)
    gu.assert_parity(out[idx], exp, dtype, op, f"{dtype} {op} n={n} (sampled)")
    del srcs, out
    torch.cuda.empty_cache()


def test_reduce_scatter_and_batched_past_4gib(xr, orc):
    """Rank 1's shard of P=2 send buffers of 2 x 2^31 + 10 bf16 (the shard starts
    past 4 GiB), and the same reduction as one batched item."""
    rc = (1 << 31) + 5
    srcs = [_random_bits(2 * rc, 2, 950 + p) for p in range(2)]
    out = torch.empty(rc, dtype=torch.int16, device="cuda")
    xr.reduce_scatter_local(srcs, 1, out, "sum", dtype="bf16")
    out_b = torch.empty(rc, dtype=torch.int16, device="cuda")
    xr.batched_reduce([([s[rc:] for s in srcs], out_b)], "sum", dtype="bf16")
    torch.cuda.synchronize()
    idx = _samples(rc, 2, np.random.default_rng(6))
    cols = [gu.bits(s[rc:][idx], "bf16").copy() for s in srcs]
    exp = orc.allreduce_local(cols, "bf16", "sum")
    gu.assert_parity(out[idx], exp, "bf16", "sum", "rs rank 1 past 4 GiB (sampled)")
    gu.assert_parity(out_b[idx], exp, "bf16", "sum", "batched past 4 GiB (sampled)")
    del srcs, out, out_b
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mib", [256, 400])
def test_fused_eight_large_sources(xr, orc, mib):
    """Eight sources of several hundred MiB each (the launches with the larger
    occupancy caps), ragged length, sampled columns."""
    n = (mib << 20) // 2 + 5
    srcs = [_random_bits(n, 2, 1200 + mib + p) for p in range(8)]
    out = torch.empty_like(srcs[0])
    xr.allreduce_local(srcs, out, "sum", dtype="bf16")
    torch.cuda.synchronize()
    idx = _samples(n, 2, np.random.default_rng(mib))
    cols = [gu.bits(s[idx], "bf16").copy() for s in srcs]
    exp = orc.allreduce_local(cols, "bf16", "sum")
    gu.assert_parity(out[idx], exp, "bf16", "sum", f"P=8 x {mib} MiB (sampled)")
    del srcs, out
    torch.cuda.empty_cache()


def test_batched_beyond_table_and_round_robin_limits(xr, orc):
    """A host batch whose tile table would pass its size limit (2^19 tiles of
    4096 bf16) and whose item count passes the round-robin plan's (8192): the
    range-walking kernel runs it.  8200 items of 65 tiles each, one source;
    sampled items checked whole."""
    n, K = 65 * 4096, 8200
    src = _random_bits(n * K, 2, 1500)
    dst = torch.zeros(n * K, dtype=torch.int16, device="cuda")
    items = [([src[k * n:(k + 1) * n]], dst[k * n:(k + 1) * n]) for k in range(K)]
    xr.batched_reduce(items, "sum", dtype="bf16")
    torch.cuda.synchronize()
    rng = np.random.default_rng(15)
    for k in sorted({0, K - 1} | set(rng.integers(0, K, 32).tolist())):
        col = gu.bits(src[k * n:(k + 1) * n], "bf16").copy()
        gu.assert_parity(dst[k * n:(k + 1) * n], orc.allreduce_local([col], "bf16", "sum"),
                         "bf16", "sum", f"item {k}")
    del src, dst, items
    torch.cuda.empty_cache()


def test_batched_table_at_its_limit(xr, orc):
    """Exactly 2^19 tiles (two items of 2^30 bf16, one source each): the
    largest batch the tile list takes; sampled columns of both items."""
    n = 1 << 30
    srcs = [_random_bits(n, 2, 1600 + k) for k in range(2)]
    outs = [torch.empty(n, dtype=torch.int16, device="cuda") for _ in range(2)]
    xr.batched_reduce([([s], o) for s, o in zip(srcs, outs)], "sum", dtype="bf16")
    torch.cuda.synchronize()
    for k in range(2):
        idx = _samples(n, 2, np.random.default_rng(20 + k))
        col = gu.bits(srcs[k][idx], "bf16").copy()
        gu.assert_parity(outs[k][idx], orc.allreduce_local([col], "bf16", "sum"), "bf16", "sum",
                         f"item {k} (sampled)")
    del srcs, outs
    torch.cuda.empty_cache()


def test_device_batch_with_an_item_past_4gib(xr, orc):
    """Device descriptors, 70 items (two runs of the grouped kernel): item 0
    holds 2^31 + 5 bf16 elements per source (past 4 GiB, over 2^19 tiles), the
    others up to 9000; sampled columns of item 0, every other item whole."""
    n0 = (1 << 31) + 5
    big = [_random_bits(n0, 2, 1700 + p) for p in range(2)]
    out0 = torch.empty(n0, dtype=torch.int16, device="cuda")
    rng = np.random.default_rng(31)
    small = []
    for k in range(69):
        n = int(rng.integers(1, 9000))
        small.append(([_random_bits(n, 2, 1800 + 2 * k + p) for p in range(2)],
                      torch.zeros(n, dtype=torch.int16, device="cuda")))
    keep, rows = [], []
    for srcs, out in [(big, out0)] + small:
        pa = torch.tensor([s.data_ptr() for s in srcs], dtype=torch.int64, device="cuda")
        keep.append(pa)
        rows.append((pa.data_ptr(), out.data_ptr(), out.numel(), len(srcs), 0))
    arr = np.zeros(len(rows), xr.ITEM_DTYPE)
    for k, r in enumerate(rows):
        arr[k] = r
    xr.batched_reduce(torch.from_numpy(arr.view(np.uint8).copy()).to("cuda"), "sum",
                      dtype="bf16")
    torch.cuda.synchronize()
    idx = _samples(n0, 2, np.random.default_rng(32))
    cols = [gu.bits(s[idx], "bf16").copy() for s in big]
    gu.assert_parity(out0[idx], orc.allreduce_local(cols, "bf16", "sum"), "bf16", "sum",
                     "item 0")
    for k, (srcs, out) in enumerate(small):
        cols = [gu.bits(s, "bf16").copy() for s in srcs]
        gu.assert_parity(out, orc.allreduce_local(cols, "bf16", "sum"), "bf16", "sum",
                         f"item {k + 1}")
    del big, out0, small, keep
    torch.cuda.empty_cache()
