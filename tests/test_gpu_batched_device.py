"""Device-resident batch descriptors past one run of items (the queue and
grouped kernels).

A batch of more than 64 items whose descriptors live in device memory runs,
when launched eagerly, on the queue kernel: a persistent grid whose
workgroups scan every item's tile count into an LDS prefix and take tiles in
order from a counter that the stream's slot keeps in device memory (two
counters used alternately by successive launches on the stream).  Under
graph capture, or past the queue's 16384 items, the batch is cut into runs
of consecutive items, each run dealt tile by tile to its own set of
workgroups that plan their tiles from the descriptors in the kernel (the
grouped kernel).  These tests drive both paths across their boundaries
against the CPU oracle:

- batch sizes on both sides of whole runs (65, 127, 128, 129 items) and many
  runs (700 items), items of 0, 1 and a few elements, items ending just
  before, on and after a 512-vector tile, items of many tiles, 1..9, 17 and
  64 sources, element-aligned (not 16-byte aligned) items, and descriptors
  that must be skipped (dst untouched);
- workgroup budgets of 1, 3, 100 and 513 (fewer workgroups than one run's
  set, and sets striding over the runs): results bit-identical;
- graph capture of such a batch, replayed with eager work in between;
- batches enqueued back to back on one stream and alternately on two streams
  (the counters of each stream's slot handed from launch to launch);
- 16384 and 16385 items (the last batch the queue takes, the first past it).
"""
import numpy as np
import pytest

import gpu_util as gu
import pins

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

ES = {"f32": 4, "bf16": 2, "f16": 2, "e4m3": 1, "e5m2": 1, "i32": 4, "u32": 4, "i64": 8,
      "u64": 8, "f64": 8, "i8": 1, "u8": 1}


@pytest.fixture(scope="module")
def xr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    xr.load()
    yield xr
    xr.set_max_workgroups(0)


def _sizes(rng, dtype, K):
    tile = 512 * (16 // ES[dtype])          # elements of one 512-vector tile
    pool = [0, 1, 3, 7, tile - 1, tile, tile + 1, 3 * tile + 5, 9 * tile - 2]
    out = [int(rng.choice(pool)) if rng.random() < 0.7 else int(rng.integers(1, 5 * tile))
           for _ in range(K)]
    out[0] = 40 * tile + 3                  # one item much longer than the others
    return out


class Batch:
    """K items of random sources on the device, descriptors on the device."""

    def __init__(self, xr, rng, dtype, K, skip_rows=True):
        self.dtype = dtype
        sizes = _sizes(rng, dtype, K)
        nsrc = [int(rng.choice([1, 2, 3, 5, 8, 8, 8, 9, 17])) for _ in range(K)]
        nsrc[1] = 64
        self.host, self.outs, self.keep, rows = [], [], [], []
        for k, (n, P) in enumerate(zip(sizes, nsrc)):
            shift = 1 if k % 5 == 2 else 0          # element-aligned only
            srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
            dev = [gu.to_dev(np.concatenate([np.zeros(shift, s.dtype), s]), dtype)[shift:]
                   for s in srcs]
            out = torch.zeros(n + shift, dtype=gu.torch_dtype(dtype), device="cuda")[shift:]
            pa = torch.tensor([d.data_ptr() for d in dev], dtype=torch.int64, device="cuda")
            self.keep += dev + [pa]
            self.host.append(srcs)
            self.outs.append(out)
            rows.append((pa.data_ptr(), out.data_ptr(), n, P, 0))
        # descriptors that must be skipped, spread through the batch
        self.bad = torch.full((4096,), 7, dtype=gu.torch_dtype(dtype), device="cuda")
        if skip_rows:
            nullp = torch.zeros(3, dtype=torch.int64, device="cuda")
            good = self.keep[-1]
            self.keep.append(nullp)
            bad = self.bad.data_ptr()
            for pos, row in zip((3, K // 2, K + 4),
                                ((nullp.data_ptr(), bad, 4096, 3, 0),      # NULL sources
                                 (good.data_ptr(), bad, 4096, 0, 0),       # nsrc 0
                                 (good.data_ptr(), bad, 4096, 1, 1))):     # reserved != 0
                rows.insert(pos, row)
        arr = np.zeros(len(rows), xr.ITEM_DTYPE)
        for k, r in enumerate(rows):
            arr[k] = r
        self.items = torch.from_numpy(arr.view(np.uint8).copy()).to("cuda")
        self.nitems = len(rows)

    def expected(self, orc, op):
        return [orc.allreduce_local(s, self.dtype, op) if s[0].size else None for s in self.host]

    def check(self, exps, op, what):
        for k, (out, exp) in enumerate(zip(self.outs, exps)):
            if exp is not None:
                gu.assert_parity(out, exp, self.dtype, op, f"{what}: item {k}")
        assert torch.all(self.bad == 7), what


@pytest.mark.parametrize("dtype,op,K", [
    ("bf16", "sum", 65), ("f32", "max", 127), ("i32", "sum", 128), ("e4m3", "sum", 129),
    ("f16", "min", 200), ("i64", "prod", 130), ("u32", "max", 66), ("bf16", "avg", 700),
])
def test_device_batch_runs(xr, orc, dtype, op, K):
    rng = np.random.default_rng(5100 + K)
    b = Batch(xr, rng, dtype, K)
    print(f"{dtype} {op}: {b.nitems} device descriptors", flush=True)
    xr.batched_reduce(b.items, op, dtype=dtype)
    torch.cuda.synchronize()
    b.check(b.expected(orc, op), op, f"{dtype} {op} K={K}")


def test_device_batch_runs_under_budgets(xr, orc):
    rng = np.random.default_rng(5200)
    b = Batch(xr, rng, "bf16", 300)
    exps = b.expected(orc, "sum")
    for budget in (1, 3, 100, 513, 0):
        for o in b.outs:
            o.zero_()
        print(f"budget {budget}", flush=True)
        prev = xr.set_max_workgroups(budget)
        try:
            xr.batched_reduce(b.items, "sum", dtype="bf16")
            torch.cuda.synchronize()
        finally:
            xr.set_max_workgroups(prev)
        b.check(exps, "sum", f"budget {budget}")


def test_device_batch_runs_graph_replay(xr, orc):
    rng = np.random.default_rng(5300)
    b = Batch(xr, rng, "f32", 150, skip_rows=False)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        xr.batched_reduce(b.items, "sum", dtype="f32")
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        xr.batched_reduce(b.items, "sum", dtype="f32")
    torch.cuda.synchronize()
    for r in range(3):
        # new inputs in place: scale the first source of every item
        with np.errstate(over="ignore", invalid="ignore"):    # inf and NaN inputs
            for k in range(len(b.host)):
                b.host[k][0] = (b.host[k][0] * np.float32(0.5 + r)).astype(np.float32)
        _upload_first_sources(b)
        for o in b.outs:
            o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        b.check(b.expected(orc, "sum"), "sum", f"replay {r}")


def _upload_first_sources(b):
    """Copy each item's (changed) first host source into its device buffer."""
    # keep holds, per item, its P device sources followed by its pointer array
    pos = 0
    for srcs in b.host:
        dev0 = b.keep[pos]
        if srcs[0].size:
            dev0.copy_(gu.to_dev(srcs[0], b.dtype))
        pos += len(srcs) + 1


def test_device_batches_back_to_back(xr, orc):
    """Eight batches of different shapes enqueued without synchronisation,
    first all on one stream, then alternating over two: each launch must take
    every tile of its own batch exactly once from its stream's counters."""
    rng = np.random.default_rng(5400)
    batches = [Batch(xr, rng, "bf16", int(K), skip_rows=(K % 2 == 0))
               for K in (70, 300, 65, 129, 500, 66, 200, 90)]
    exps = [b.expected(orc, "sum") for b in batches]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for mode in ("one stream", "two streams"):
        for b in batches:
            for o in b.outs:
                o.zero_()
        torch.cuda.synchronize()
        for r in range(3):
            for i, b in enumerate(batches):
                st = streams[0] if mode == "one stream" else streams[(i + r) % 2]
                with torch.cuda.stream(st):
                    xr.batched_reduce(b.items, "sum", dtype="bf16")
        torch.cuda.synchronize()
        for i, (b, e) in enumerate(zip(batches, exps)):
            b.check(e, "sum", f"{mode}: batch {i}")


@pytest.mark.parametrize("K", [16384, 16385])
def test_device_batch_queue_item_limit(xr, orc, K):
    """K int32 items of 1..40 elements over two sources, laid end to end, so
    the concatenated outputs equal one oracle reduction of the concatenated
    sources: the largest batch the queue kernel plans in LDS, and one more
    item (the grouped kernel)."""
    rng = np.random.default_rng(5500 + K)
    sizes = rng.integers(1, 41, size=K)
    sizes[-1] = 3 * 512 * 4 + 1             # the last item spans several tiles
    total = int(sizes.sum())
    srcs_np = [pins.random_column_values(rng, "i32", total) for _ in range(2)]
    d = [gu.to_dev(x, "i32") for x in srcs_np]
    out = torch.zeros(total, dtype=torch.int32, device="cuda")
    starts = np.concatenate([[0], np.cumsum(sizes)[:-1]]).astype(np.uint64)
    ptrs = torch.tensor(np.stack([d[0].data_ptr() + 4 * starts, d[1].data_ptr() + 4 * starts],
                                 axis=1).astype(np.int64).reshape(-1), device="cuda")
    arr = np.zeros(K, xr.ITEM_DTYPE)
    arr["srcs"] = ptrs.data_ptr() + 16 * np.arange(K, dtype=np.uint64)
    arr["dst"] = out.data_ptr() + 4 * starts
    arr["count"] = sizes
    arr["nsrc"] = 2
    items = torch.from_numpy(arr.view(np.uint8).copy()).to("cuda")
    xr.batched_reduce(items, "sum", dtype="i32")
    torch.cuda.synchronize()
    gu.assert_parity(out, orc.allreduce_local(srcs_np, "i32", "sum"), "i32", "sum", f"K={K}")


RAND_DTYPES = ("f32", "bf16", "f16", "e4m3", "e5m2", "i32", "u32", "i64", "u64", "f64",
               "i8", "u8")


@pytest.mark.parametrize("seed", range(4))
def test_random_queue_batches(xr, orc, seed):
    """Seeded random device batches of 65..400 items (the queue kernel): every
    dtype, op (AVG on float types), 1..17 sources, sizes from one element to
    several tiles, element-aligned (not 16-byte aligned) items, under random
    CU budgets, alternating xred_batched_reduce and
    xred_batched_reduce_noalloc, each against the oracle."""
    rng = np.random.default_rng(5600 + seed)
    for case in range(6):
        dtype = RAND_DTYPES[rng.integers(0, len(RAND_DTYPES))]
        ops = ["sum", "prod", "max", "min"] + (["avg"] if dtype in gu.FLOATS else [])
        op = ops[rng.integers(0, len(ops))]
        K = int(rng.integers(65, 401))
        tile = 2 * 512 * (16 // ES[dtype])
        sizes = [int(rng.choice([1, 3, tile - 1, tile, tile + 1, 2 * tile + 5]))
                 if rng.random() < 0.5 else int(rng.integers(1, 3 * tile)) for _ in range(K)]
        nsrc = [int(rng.choice([1, 2, 3, 8, 9, 17])) for _ in range(K)]
        budget = int(rng.choice([0, 0, 1, 7, 100]))
        noalloc = case % 2 == 1
        print(f"case {case}: {dtype} {op} K={K} budget={budget} noalloc={noalloc}", flush=True)
        host, outs, keep, rows = [], [], [], []
        for k, (n, P) in enumerate(zip(sizes, nsrc)):
            shift = 1 if k % 4 == 3 else 0
            srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
            dev = [gu.to_dev(np.concatenate([np.zeros(shift, s.dtype), s]), dtype)[shift:]
                   for s in srcs]
            out = torch.zeros(n + shift, dtype=gu.torch_dtype(dtype), device="cuda")[shift:]
            pa = torch.tensor([d.data_ptr() for d in dev], dtype=torch.int64, device="cuda")
            keep += dev + [pa]
            host.append(srcs)
            outs.append(out)
            rows.append((pa.data_ptr(), out.data_ptr(), n, P, 0))
        arr = np.zeros(K, xr.ITEM_DTYPE)
        for k, r in enumerate(rows):
            arr[k] = r
        items = torch.from_numpy(arr.view(np.uint8).copy()).to("cuda")
        prev = xr.set_max_workgroups(budget)
        try:
            if noalloc:
                xr.batched_reduce_noalloc(items, op, dtype=dtype)
            else:
                xr.batched_reduce(items, op, dtype=dtype)
            torch.cuda.synchronize()
        finally:
            xr.set_max_workgroups(prev)
        for k in range(K):
            gu.assert_parity(outs[k], orc.allreduce_local(host[k], dtype, op), dtype, op,
                             f"case {case} item {k}")


def test_noalloc_graph_replay(xr, orc):
    """xred_batched_reduce_noalloc captured in a HIP graph: its kernel leaves
    the tile counters at zero, so every replay, with eager calls of both
    device-descriptor entry points between replays, folds the whole batch."""
    rng = np.random.default_rng(5700)
    b = Batch(xr, rng, "f32", 180, skip_rows=False)
    other = Batch(xr, rng, "f32", 90, skip_rows=False)
    exp_other = other.expected(orc, "sum")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        xr.batched_reduce_noalloc(b.items, "sum", dtype="f32")   # looks the array up eagerly
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        xr.batched_reduce_noalloc(b.items, "sum", dtype="f32")
    torch.cuda.synchronize()
    for r in range(3):
        with np.errstate(over="ignore", invalid="ignore"):
            for k in range(len(b.host)):
                b.host[k][0] = (b.host[k][0] * np.float32(0.5 + r)).astype(np.float32)
        _upload_first_sources(b)
        for o in b.outs:
            o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        b.check(b.expected(orc, "sum"), "sum", f"replay {r}")
        for o in other.outs:
            o.zero_()
        if r % 2:
            xr.batched_reduce_noalloc(other.items, "sum", dtype="f32")
        else:
            xr.batched_reduce(other.items, "sum", dtype="f32")
        torch.cuda.synchronize()
        other.check(exp_other, "sum", f"eager call after replay {r}")
    del g
