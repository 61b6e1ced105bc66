"""GPU parity: every entry point of libxred against the CPU oracle, element by
element, on the same seeded inputs.  The bar is bit-exact equality (the fold
order is fixed, so float results are deterministic); NaN payloads of float
sum/prod are not specified and compare by NaN-ness only.

Covered: the six workloads at full size in the launch configuration the
benchmark times (c1, c2, c3, c4 with host and with device descriptors, c5a,
c5b: every output element), and an edge matrix of sizes
(empty, ragged, several tiles), source counts 1..64, every dtype x op with
special values (+-0, +-inf, subnormals, NaN, overflow), misaligned buffers,
in-place calls, guard bands around outputs, and every step-wise flag.
"""
import ctypes
import os

import numpy as np
import pytest

import gpu_util as gu
import pins
import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

DTYPES = ("f32", "bf16", "i32", "u32")
OPS = ("sum", "prod", "max", "min")
CORES = min(16, len(os.sched_getaffinity(0)))


@pytest.fixture(scope="module")
def xr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    xr.load()   # raises if libxred.so is missing: there is no fallback
    return xr


def _run_allreduce(xr, srcs_np, dtype, op, **kw):
    srcs = [gu.to_dev(s, dtype) for s in srcs_np]
    out = torch.empty_like(srcs[0])
    xr.allreduce_local(srcs, out, op, dtype=dtype, **kw)
    torch.cuda.synchronize()
    return out


def test_native_library_is_loaded(xr):
    maps = open("/proc/self/maps").read()
    assert str(xr._lib.LIB_PATH) in maps or "libxred.so" in maps


# ------------------------------------------------------------ workloads --

def test_c1_full(xr, orc):
    w = wl.WORKLOADS["c1"]
    srcs = wl.sources(w)
    got = _run_allreduce(xr, srcs, w.dtype, w.op)
    exp = orc.allreduce_local(srcs, w.dtype, w.op, nthreads=CORES)
    gu.assert_parity(got, exp, w.dtype, w.op, "c1")


@pytest.fixture(scope="module")
def c2_sources():
    return wl.sources(wl.WORKLOADS["c2"])


def test_c2_full(xr, orc, c2_sources):
    w = wl.WORKLOADS["c2"]
    got = _run_allreduce(xr, c2_sources, w.dtype, w.op)
    exp = orc.allreduce_local(c2_sources, w.dtype, w.op, nthreads=CORES)
    gu.assert_parity(got, exp, w.dtype, w.op, "c2")


@pytest.mark.parametrize("op", ["prod", "max", "min", "avg"])
def test_c2_full_other_ops(xr, orc, c2_sources, op):
    """The bucket's inputs and launch configuration with every other op."""
    got = _run_allreduce(xr, c2_sources, "bf16", op)
    exp = orc.allreduce_local(c2_sources, "bf16", op, nthreads=CORES)
    gu.assert_parity(got, exp, "bf16", op, f"c2 {op}")


@pytest.mark.parametrize("name", ["c5a", "c5b"])
def test_c5_full(xr, orc, name):
    w = wl.WORKLOADS[name]
    srcs = wl.sources(w)
    got = _run_allreduce(xr, srcs, w.dtype, w.op)
    exp = orc.allreduce_local(srcs, w.dtype, w.op, nthreads=CORES)
    gu.assert_parity(got, exp, w.dtype, w.op, name)
    if name == "c5b":
        # the structured blocks: +-0 columns give +0 unless all -0; one +inf wins
        b = gu.bits(got, "f32")
        assert np.all(b[wl.C5B_BLOCK:2 * wl.C5B_BLOCK] == 0x7F800000)


def test_c3_stepwise_full(xr, orc):
    w = wl.WORKLOADS["c3"]
    chunks = wl.stepwise_chunks(w)
    d = [gu.to_dev(c, w.dtype) for c in chunks]
    acc = torch.empty(w.count, dtype=torch.float32, device="cuda")
    out = torch.empty_like(d[0])
    xr.reduce_copy_step(d[0], acc, None, w.op, init=True)
    for c in d[1:]:
        xr.reduce_copy_step(c, acc, None, w.op)
    xr.acc_cast(acc, out)
    # the same sequence with the last step fused into FINAL
    acc2 = torch.empty_like(acc)
    out2 = torch.empty_like(out)
    xr.reduce_copy_step(d[0], acc2, None, w.op, init=True)
    for c in d[1:-1]:
        xr.reduce_copy_step(c, acc2, None, w.op)
    xr.reduce_copy_step(d[-1], acc2, out2, w.op, final=True)
    torch.cuda.synchronize()
    oacc = orc.reduce_copy_step(chunks[0], None, w.dtype, w.op, init=True)
    for c in chunks[1:]:
        oacc = orc.reduce_copy_step(c, oacc, w.dtype, w.op)
    gu.assert_parity(acc, oacc, "f32", w.op, "c3 accumulator")
    exp = orc.acc_cast(oacc, w.dtype)
    gu.assert_parity(out, exp, w.dtype, w.op, "c3 cast")
    gu.assert_parity(out2, exp, w.dtype, w.op, "c3 final")
    # and it equals the fused 16-source reduce of the chunks
    fused = torch.empty_like(out)
    xr.allreduce_local(d, fused, w.op)
    torch.cuda.synchronize()
    gu.assert_parity(fused, exp, w.dtype, w.op, "c3 fused")


def _c4_device_descriptors(xr, arena_dev, offs, sizes, outs, es):
    """Device-resident xred_item array + per-item device pointer arrays."""
    base = arena_dev.data_ptr()
    P = offs.shape[1]
    ptrs = torch.tensor((base + offs * es).reshape(-1).astype(np.int64), device="cuda")
    items = np.zeros(len(sizes), xr.ITEM_DTYPE)
    items["srcs"] = ptrs.data_ptr() + 8 * P * np.arange(len(sizes), dtype=np.uint64)
    items["dst"] = [o.data_ptr() for o in outs]
    items["count"] = sizes
    items["nsrc"] = P
    dev_items = torch.from_numpy(items.view(np.uint8).copy()).to("cuda")
    return dev_items, ptrs


def _assert_items(got_flat, exp_flat, sizes, dtype, op, what):
    """Every element of every item against the oracle; on a mismatch, name the
    first item that differs."""
    ends = np.cumsum(sizes)
    try:
        gu.assert_parity(got_flat, exp_flat, dtype, op, what)
    except AssertionError:
        g, e = gu.bits(got_flat, dtype), gu.bits(exp_flat, dtype)
        bad = g != e
        if dtype in gu.FLOATS and op in ("sum", "prod", "avg"):
            bad &= ~(gu.nan_mask(g, dtype) & gu.nan_mask(e, dtype))
        i = int(np.flatnonzero(bad)[0])
        k = int(np.searchsorted(ends, i, side="right"))
        raise AssertionError(f"{what}: item {k} (count {int(sizes[k])}) differs first, at "
                             f"element {i - (int(ends[k - 1]) if k else 0)}") from None


def test_c4_batched_full(xr, orc):
    """The small-message batch (4096 items, P=8 bf16, 8 KiB-1 MiB per source):
    every output element of every item, with host descriptors and with
    device-resident descriptors, compared with the oracle's per-item
    reduction (the oracle splits each item's elements over the host's cores,
    which does not change any element's fold)."""
    w = wl.WORKLOADS["c4"]
    sizes = wl.batched_sizes(w)
    arena, offs = wl.batched_arena(w, sizes)
    es = wl.ELEM_SIZE[w.dtype]
    arena_dev = gu.to_dev(arena, w.dtype)
    outs = [torch.empty(int(n), dtype=torch.bfloat16, device="cuda") for n in sizes]
    items = [([arena_dev[o:o + int(n)] for o in offs[k]], outs[k])
             for k, n in enumerate(sizes)]
    xr.batched_reduce(items, w.op, dtype=w.dtype)
    outs2 = [torch.full_like(o, float("nan")) for o in outs]
    dev_items, keep = _c4_device_descriptors(xr, arena_dev, offs, sizes, outs2, es)
    xr.batched_reduce(dev_items, w.op, dtype=w.dtype)
    torch.cuda.synchronize()
    got_host = torch.cat(outs).cpu()
    got_dev = torch.cat(outs2).cpu()
    del outs, outs2, items, keep, dev_items, arena_dev
    exp = orc.batched_reduce([[arena[o:o + int(n)] for o in offs[k]]
                              for k, n in enumerate(sizes)],
                             w.dtype, w.op, nthreads=CORES)
    exp_flat = np.concatenate(exp)
    assert exp_flat.size == int(sizes.sum()) == got_host.numel()
    _assert_items(got_host, exp_flat, sizes, w.dtype, w.op, "c4 host descriptors")
    _assert_items(got_dev, exp_flat, sizes, w.dtype, w.op, "c4 device descriptors")


# ---------------------------------------------------------- edge matrix --

SIZES = [1, 7, 8, 9, 63, 64, 65, 1023, 4096 + 5, (1 << 17) + 3]
NSRCS = [1, 2, 3, 4, 5, 7, 8, 9, 16, 31, 32, 33, 64]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("op", OPS)
def test_edge_matrix(xr, orc, dtype, op):
    rng = np.random.default_rng(10 * DTYPES.index(dtype) + OPS.index(op))
    for P in NSRCS:
        for n in SIZES:
            if P * n > (1 << 21):
                continue
            srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
            got = _run_allreduce(xr, srcs, dtype, op)
            exp = orc.allreduce_local(srcs, dtype, op)
            gu.assert_parity(got, exp, dtype, op, f"{dtype} {op} P={P} n={n}")


@pytest.mark.parametrize("dtype,op", [("bf16", "sum"), ("f32", "max"), ("i32", "sum")])
def test_tile_shapes_at_one_round_threshold(xr, orc, dtype, op):
    """The fused launcher uses 512-thread tiles of one vector per thread while
    every tile fits on the chip in one round (4 per CU), then (up to 8
    sources) 512-thread tiles of two vectors per thread while those fit in one
    round, and occupancy-capped 128-thread tiles above; sizes at and around
    both switches, with ragged tails, on compile-time and runtime source
    counts."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    vec = 16 // (2 if dtype == "bf16" else 4)
    edge = cus * 4 * 512 * vec               # elements at the first switch
    rng = np.random.default_rng(77 + DTYPES.index(dtype))
    nmax = 2 * edge + 128 * vec * 3 + 1
    # random columns (specials included) repeated with an odd period, so no
    # misplaced tile or vector lines up with an equal value
    full = [np.resize(pins.random_column_values(rng, dtype, 65536 + 13 + 2 * p), nmax)
            for p in range(32)]
    for P in (3, 8, 12, 32):
        for n in (edge - 3, edge + 5, 2 * edge, 2 * edge + 5, nmax):
            srcs = [f[:n] for f in full[:P]]
            got = _run_allreduce(xr, srcs, dtype, op)
            exp = orc.allreduce_local(srcs, dtype, op, nthreads=CORES)
            gu.assert_parity(got, exp, dtype, op, f"{dtype} {op} P={P} n={n}")


def test_empty_is_noop(xr):
    a = torch.zeros(0, dtype=torch.bfloat16, device="cuda")
    xr.allreduce_local([a, a], a)
    acc = torch.zeros(0, dtype=torch.float32, device="cuda")
    xr.reduce_copy_step(a, acc, None, init=True)
    xr.acc_cast(acc, a)
    xr.batched_reduce([], dtype="bf16")
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype", DTYPES)
def test_misaligned_and_guard_bands(xr, orc, dtype):
    rng = np.random.default_rng(5)
    n = 70001
    G = 4096          # guard elements on each side of dst
    for P in (1, 3, 8, 33):
        for shift in (1, 3):
            srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
            big = [gu.to_dev(np.concatenate([np.zeros(shift, s.dtype), s]), dtype) for s in srcs]
            views = [b[shift:] for b in big]
            canary = 0x5A
            store = torch.full((n + 2 * G,), 0, dtype=gu.torch_dtype(dtype), device="cuda")
            store.view(torch.uint8).fill_(canary)
            out = store[G + shift:G + shift + n]
            xr.allreduce_local(views, out, "sum", dtype=dtype)
            torch.cuda.synchronize()
            exp = orc.allreduce_local(srcs, dtype, "sum")
            gu.assert_parity(out, exp, dtype, "sum", f"misaligned {dtype} P={P} shift={shift}")
            raw = store.view(torch.uint8).cpu().numpy()
            es = out.element_size()
            assert np.all(raw[:(G + shift) * es] == canary)
            assert np.all(raw[(G + shift + n) * es:] == canary)


@pytest.mark.parametrize("dtype", ["bf16", "f32", "u8", "f64"])
def test_element_offsets_within_16_bytes(xr, orc, dtype):
    """Buffers that are element- but not 16-byte aligned: when every pointer
    sits at the same offset within 16 bytes, the first elements up to the
    next boundary are folded one by one and the rest takes the vector path
    (lengths at, below and just past that lead, and long ones); sources at
    different offsets take the scalar path, the output at another offset
    the vector loads with split stores.  Canaries around the output stay
    untouched."""
    rng = np.random.default_rng(17)
    es = {"bf16": 2, "f32": 4, "u8": 1, "f64": 8}[dtype]
    G = 64
    cases = []
    for m in range(es, 16, es):                 # every element offset within 16 B
        lead = (16 - m) // es
        for n in (1, lead - 1, lead, lead + 1, lead + 16 // es + 3, 70001, 600011):
            if n >= 1:
                cases.append(("common", m, n))
    cases += [("sources differ", es, 70001), ("output differs", es, 70001),
              ("sources differ", es, 5), ("output differs", 16 - es, 600011)]
    for k, (kind, m, n) in enumerate(cases):
        P = (2, 3, 8, 17)[k % 4]
        srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
        keep, views = [], []
        for p, a in enumerate(srcs):
            o = m if kind != "sources differ" or p % 2 == 0 else (m + es) % 16
            big = torch.zeros(o + n * es + 16, dtype=torch.uint8, device="cuda")
            v = big[o:o + n * es].view(gu.torch_dtype(dtype))
            v.copy_(gu.to_dev(a, dtype))
            keep.append(big)
            views.append(v)
        do = m if kind != "output differs" else (m + es) % 16
        store = torch.full((G + do + n * es + G,), 0x5A, dtype=torch.uint8, device="cuda")
        out = store[G + do:G + do + n * es].view(gu.torch_dtype(dtype))
        xr.allreduce_local(views, out, "sum", dtype=dtype)
        torch.cuda.synchronize()
        what = f"{kind} {dtype} P={P} offset={m} n={n}"
        gu.assert_parity(out, orc.allreduce_local(srcs, dtype, "sum"), dtype, "sum", what)
        raw = store.cpu().numpy()
        assert np.all(raw[:G + do] == 0x5A), what
        assert np.all(raw[G + do + n * es:] == 0x5A), what


@pytest.mark.parametrize("dtype", ["bf16", "f32", "u8", "f64", "e5m2", "i64"])
def test_output_at_another_offset(xr, orc, dtype):
    """Sources at one offset within 16 bytes and the output at another (the
    shard of every rank but some of a reduce-scatter with an odd shard
    length): the sources are read in vectors after the lead and each result
    vector is stored in aligned pieces of 1, 2, 4 or 8 bytes.  Every pair of
    element offsets; lengths just past the lead, past one vector, across a
    few tiles with a ragged tail, long, and past one round of wide
    workgroups; 1 to 17 sources (every first and last group size of the
    runtime-count fold); sum, and max / avg / prod on some.  Canaries around
    the output stay untouched."""
    rng = np.random.default_rng(19)
    es = xr.ELEM_SIZE[dtype]
    G = 64
    offs = list(range(0, 16, es))
    cases = []
    for ms in offs:
        for md in offs:
            if md == ms:
                continue
            lead = (16 - ms) % 16 // es
            for n in (lead + 1, lead + 16 // es + 3, 128 * 3 * 16 // es + 7):
                cases.append((ms, md, n))
    big = [(ms, md, 600011) for ms, md in ((offs[1], 0), (0, offs[-1]), (offs[-1], offs[1]))
           if ms != md]
    # past one round of 512-thread workgroups: two vectors per thread (P=2),
    # and 128-thread workgroups (P=9)
    wide = [(offs[1], 0, (9 << 20) // es + 5), (offs[-1], 0, (9 << 20) // es + 3)]
    ops = ["sum", "max", "avg" if dtype in gu.FLOATS else "min", "prod"]
    for k, (ms, md, n) in enumerate(cases + big + wide):
        P = (1, 3, 8, 9, 17, 5, 16, 2)[k % 8]
        op = ops[k % 4] if n < 600011 else "sum"
        if k >= len(cases) + len(big):
            P = (2, 9)[k - len(cases) - len(big)]
        srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
        keep, views = [], []
        for a in srcs:
            b = torch.zeros(ms + n * es + 16, dtype=torch.uint8, device="cuda")
            v = b[ms:ms + n * es].view(gu.torch_dtype(dtype))
            v.copy_(gu.to_dev(a, dtype))
            keep.append(b)
            views.append(v)
        store = torch.full((G + md + n * es + G,), 0x5A, dtype=torch.uint8, device="cuda")
        out = store[G + md:G + md + n * es].view(gu.torch_dtype(dtype))
        xr.allreduce_local(views, out, op, dtype=dtype)
        torch.cuda.synchronize()
        what = f"{dtype} {op} P={P} sources at {ms} output at {md} n={n}"
        gu.assert_parity(out, orc.allreduce_local(srcs, dtype, op), dtype, op, what)
        raw = store.cpu().numpy()
        assert np.all(raw[:G + md] == 0x5A), what
        assert np.all(raw[G + md + n * es:] == 0x5A), what


@pytest.mark.parametrize("dtype", ["bf16", "f32", "u8", "f64", "e4m3", "i32"])
def test_sources_at_different_offsets(xr, orc, dtype):
    """Sources at different offsets within 16 bytes (each at the very start
    of its own allocation, so nothing before it may be read): every source's
    vectors are realigned to the output's grid, the lead and the tail are
    folded element by element.  Offsets drawn per source and for the output;
    lengths below, at and just past the shortest vector launch, a few tiles
    with a ragged tail, and long; 2 to 17 sources; sum, max, avg / min and
    prod.  Canaries around the output stay untouched."""
    rng = np.random.default_rng(29)
    es = xr.ELEM_SIZE[dtype]
    G = 64
    ops = ["sum", "max", "avg" if dtype in gu.FLOATS else "min", "prod"]
    cases = []
    for k in range(48):
        offs = [int(rng.integers(0, 16 // es)) * es for _ in range(17)]
        offs[1] = (offs[0] + es) % 16            # at least two offsets differ
        do = int(rng.integers(0, 16 // es)) * es
        lead = (((16 - do) % 16) + 16) // es
        n = (lead + 32 // es - 1, lead + 32 // es, lead + 32 // es + 1, lead + 48 // es + 3,
             3 * 128 * 16 // es + 7, 600011)[k % 6]
        cases.append((offs, do, n, (2, 3, 8, 9, 17, 8)[k % 6]))
    for k, (offs, do, n, P) in enumerate(cases):
        op = ops[k % 4] if n < 600011 else "sum"
        srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
        keep, views = [], []
        for p, a in enumerate(srcs):
            o = offs[p]
            b = torch.zeros(o + n * es, dtype=torch.uint8, device="cuda")
            v = b[o:o + n * es].view(gu.torch_dtype(dtype))
            v.copy_(gu.to_dev(a, dtype))
            keep.append(b)
            views.append(v)
        store = torch.full((G + do + n * es + G,), 0x5A, dtype=torch.uint8, device="cuda")
        out = store[G + do:G + do + n * es].view(gu.torch_dtype(dtype))
        xr.allreduce_local(views, out, op, dtype=dtype)
        torch.cuda.synchronize()
        what = f"{dtype} {op} P={P} sources at {offs[:P]} output at {do} n={n}"
        gu.assert_parity(out, orc.allreduce_local(srcs, dtype, op), dtype, op, what)
        raw = store.cpu().numpy()
        assert np.all(raw[:G + do] == 0x5A), what
        assert np.all(raw[G + do + n * es:] == 0x5A), what


@pytest.mark.parametrize("dtype", ["bf16", "u8", "f32"])
def test_reduce_scatter_odd_shards(xr, orc, dtype):
    """A reduce-scatter with an odd shard length: every rank's shard (rank 0
    aligned, the others at other offsets within 16 bytes) against the
    oracle, P = 8 and 16, one shard of a few tiles and one of 4 MiB."""
    rng = np.random.default_rng(23)
    for P, rc in ((8, 12345), (16, 3001), (8, (1 << 21) + 1)):
        if rc > 1 << 20 and dtype != "bf16":
            continue
        srcs = [pins.random_column_values(rng, dtype, P * rc) for _ in range(P)]
        d = [gu.to_dev(s, dtype) for s in srcs]
        for r in range(P):
            out = torch.empty(rc, dtype=d[0].dtype, device="cuda")
            xr.reduce_scatter_local(d, r, out, "sum", dtype=dtype)
            torch.cuda.synchronize()
            gu.assert_parity(out, orc.reduce_scatter_local(srcs, r, dtype, "sum"), dtype, "sum",
                             f"rs P={P} recvcount={rc} rank {r}")


@pytest.mark.parametrize("dtype", ["bf16", "f32", "u8", "f64"])
def test_line_misaligned_buffers(xr, orc, dtype):
    """16-byte-aligned buffers that start inside a 128-byte line take the
    vector path with a short first tile up to the first source's next line:
    every byte offset of 16..112, lengths shorter than that first tile, equal
    to it, one vector past it, around one tile of each launch shape past it
    and past one round of workgroups (ragged tails included); the sources
    sharing one offset or not, the output at another; canaries around the
    output stay untouched."""
    rng = np.random.default_rng(13)
    es = {"bf16": 2, "f32": 4, "u8": 1, "f64": 8}[dtype]
    vec = 16 // es
    G = 256           # guard bytes on each side of the output
    cases = []
    for off in range(16, 128, 16):
        head = (128 - off) // es
        for n in (1, vec - 1, head - vec, head, head + 1, head + vec, head + 128 * vec - 3,
                  head + 128 * vec + 5, head + 512 * vec + 1, head + 1024 * vec + 7,
                  head + 300000 * vec // 8 + 3):
            if n >= 1:
                cases.append((off, n, (1, 3, 8, 17)[len(cases) % 4]))
    # past one round of workgroups: the multi-round 128-thread tiles
    cases += [(48, (128 - 48) // es + 1100000 * vec + 5, 3),
              (80, (128 - 80) // es + 600000 * vec + 9, 17)]
    for k, (off, n, P) in enumerate(cases):
        same = k % 3 != 2
        srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
        views = []
        for p, a in enumerate(srcs):
            o = off if same or p == 0 else (off + 16 * p) % 128
            big = torch.zeros(o + n * es + 128, dtype=torch.uint8, device="cuda")
            assert big.data_ptr() % 128 == 0
            v = big[o:o + n * es].view(gu.torch_dtype(dtype))
            v.copy_(gu.to_dev(a, dtype))
            views.append((big, v))
        dofs = (off + 48) % 128
        store = torch.full((G + dofs + n * es + G,), 0x5A, dtype=torch.uint8, device="cuda")
        out = store[G + dofs:G + dofs + n * es].view(gu.torch_dtype(dtype))
        xr.allreduce_local([v for _, v in views], out, "sum", dtype=dtype)
        torch.cuda.synchronize()
        what = f"line-misaligned {dtype} P={P} offset={off} n={n} same={same}"
        gu.assert_parity(out, orc.allreduce_local(srcs, dtype, "sum"), dtype, "sum", what)
        raw = store.cpu().numpy()
        assert np.all(raw[:G + dofs] == 0x5A), what
        assert np.all(raw[G + dofs + n * es:] == 0x5A), what


@pytest.mark.parametrize("dtype", DTYPES)
def test_in_place(xr, orc, dtype):
    rng = np.random.default_rng(8)
    n = (1 << 16) + 5
    for P in (2, 8, 20):
        for k in (0, P - 1):
            srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
            d = [gu.to_dev(s, dtype) for s in srcs]
            xr.allreduce_local(d, d[k], "sum", dtype=dtype)
            torch.cuda.synchronize()
            exp = orc.allreduce_local(srcs, dtype, "sum")
            gu.assert_parity(d[k], exp, dtype, "sum", f"in place k={k} P={P}")


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("recvcount", [1000003, 1 << 18, 1])
def test_reduce_scatter(xr, orc, dtype, recvcount):
    rng = np.random.default_rng(recvcount)
    P = 5
    srcs = [pins.random_column_values(rng, dtype, P * recvcount) for _ in range(P)]
    d = [gu.to_dev(s, dtype) for s in srcs]
    full = _run_allreduce(xr, srcs, dtype, "max")
    shards = []
    for r in range(P):
        out = torch.empty(recvcount, dtype=d[0].dtype, device="cuda")
        xr.reduce_scatter_local(d, r, out, "max", dtype=dtype)
        torch.cuda.synchronize()
        exp = orc.reduce_scatter_local(srcs, r, dtype, "max")
        gu.assert_parity(out, exp, dtype, "max", f"rs rank {r}")
        shards.append(out)
    gu.assert_parity(torch.cat(shards), gu.bits(full, dtype), dtype, "max", "rs concat")
    # in place: rank r's result lands in its own slice of srcs[r]
    r = 2
    d2 = [gu.to_dev(s, dtype) for s in srcs]
    xr.reduce_scatter_local(d2, r, d2[r][r * recvcount:(r + 1) * recvcount], "sum", dtype=dtype)
    torch.cuda.synchronize()
    exp = orc.reduce_scatter_local(srcs, r, dtype, "sum")
    gu.assert_parity(d2[r][r * recvcount:(r + 1) * recvcount], exp, dtype, "sum", "rs in place")


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("op", OPS)
def test_step_all_flags(xr, orc, dtype, op):
    rng = np.random.default_rng(3)
    for n, shift in ((4096 * 3 + 7, 0), (1 << 15, 0), (999, 1)):
        chunks = [pins.random_column_values(rng, dtype, n) for _ in range(6)]
        dev = []
        for c in chunks:
            b = gu.to_dev(np.concatenate([np.zeros(shift, c.dtype), c]), dtype)
            dev.append(b[shift:])
        accbuf = torch.empty(n + shift, dtype=torch.float32 if dtype in ("f32", "bf16")
                             else torch.int32, device="cuda")
        acc = accbuf[shift:]
        xr.reduce_copy_step(dev[0], acc, None, op, init=True, dtype=dtype)
        for c in dev[1:-1]:
            xr.reduce_copy_step(c, acc, None, op, dtype=dtype)
        outbuf = torch.empty(n + shift, dtype=dev[0].dtype, device="cuda")
        out = outbuf[shift:]
        acc_before = acc.clone()
        xr.reduce_copy_step(dev[-1], acc, out, op, final=True, dtype=dtype)
        single = torch.empty_like(out)
        xr.reduce_copy_step(dev[0], None, single, op, init=True, final=True, dtype=dtype)
        torch.cuda.synchronize()
        assert torch.equal(acc.view(torch.int32), acc_before.view(torch.int32)), "FINAL wrote acc"
        oacc = orc.reduce_copy_step(chunks[0], None, dtype, op, init=True)
        for c in chunks[1:-1]:
            oacc = orc.reduce_copy_step(c, oacc, dtype, op)
        accd = "f32" if dtype in ("f32", "bf16") else "u32"
        gu.assert_parity(acc, oacc, accd, op, f"step acc {dtype} {op} n={n}")
        exp = orc.reduce_copy_step(chunks[-1], oacc.copy(), dtype, op, final=True)
        gu.assert_parity(out, exp, dtype, op, f"step final {dtype} {op} n={n}")
        gu.assert_parity(single, orc.reduce_copy_step(chunks[0], None, dtype, op, init=True,
                                                      final=True), dtype, op, "init|final")
        cast = torch.empty_like(out)
        xr.acc_cast(acc, cast, dtype=dtype)
        torch.cuda.synchronize()
        gu.assert_parity(cast, orc.acc_cast(oacc, dtype), dtype, op, "cast")


@pytest.mark.parametrize("dtype", ("bf16", "f32", "i32"))
def test_batched_mixed(xr, orc, dtype):
    """Mixed source counts, ragged and misaligned items, zero-length items,
    host and device descriptors."""
    rng = np.random.default_rng(21)
    specs = []
    for k in range(300):
        P = int(rng.choice([1, 2, 3, 8, 9, 17, 64]))
        n = int(rng.choice([0, 1, 7, 100, 4095, 4096, 4097, 20000, 70001]))
        shift = int(rng.integers(0, 2)) if k % 3 == 0 else 0
        specs.append((P, n, shift))
    host_srcs, items, outs = [], [], []
    for P, n, shift in specs:
        s = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
        host_srcs.append(s)
        d = [gu.to_dev(np.concatenate([np.zeros(shift, x.dtype), x]), dtype)[shift:] for x in s]
        ob = torch.zeros(n + shift, dtype=gu.torch_dtype(dtype), device="cuda")
        outs.append(ob[shift:])
        items.append((d, outs[-1]))
    xr.batched_reduce(items, "sum", dtype=dtype)
    torch.cuda.synchronize()
    for k, (s, o) in enumerate(zip(host_srcs, outs)):
        if s[0].size == 0:
            continue
        gu.assert_parity(o, orc.allreduce_local(s, dtype, "sum"), dtype, "sum", f"item {k}")
    # device descriptors, plus items that must be skipped (dst untouched)
    keep, rows = [], []
    outs2 = [torch.zeros_like(o) for o in outs]
    for (d, _), o in zip(items, outs2):
        pa = torch.tensor([x.data_ptr() for x in d], dtype=torch.int64, device="cuda")
        keep.append(pa)
        rows.append((pa.data_ptr(), o.data_ptr(), o.numel(), len(d), 0))
    bad_out = torch.full((4096,), 7, dtype=gu.torch_dtype(dtype), device="cuda")
    nullp = torch.zeros(3, dtype=torch.int64, device="cuda")
    good_p = keep[0]
    rows += [(good_p.data_ptr(), bad_out.data_ptr(), 4096, 0, 0),      # nsrc 0
             (good_p.data_ptr(), bad_out.data_ptr(), 4096, 65, 0),     # nsrc > 64
             (good_p.data_ptr(), bad_out.data_ptr(), 4096, 1, 1),      # reserved != 0
             (0, bad_out.data_ptr(), 4096, 1, 0),                      # srcs NULL
             (nullp.data_ptr(), bad_out.data_ptr(), 4096, 3, 0)]       # NULL source
    arr = np.zeros(len(rows), xr.ITEM_DTYPE)
    for k, r in enumerate(rows):
        arr[k] = r
    dev_items = torch.from_numpy(arr.view(np.uint8).copy()).to("cuda")
    xr.batched_reduce(dev_items, "sum", dtype=dtype)
    torch.cuda.synchronize()
    # against the oracle (NaN payloads of float sums are unspecified, and the
    # two descriptor modes run different kernels)
    for k, (s, o2) in enumerate(zip(host_srcs, outs2)):
        if s[0].size == 0:
            continue
        gu.assert_parity(o2, orc.allreduce_local(s, dtype, "sum"), dtype, "sum",
                         f"device item {k}")
    assert torch.all(bad_out == 7)
    del keep


@pytest.mark.skip(reason="written for a by-value batch path (descriptors in the kernel "
                         "arguments) whose first run faulted the GPU; the path was removed "
                         "without a found cause, so this case stays off the GPU")
@pytest.mark.parametrize("dtype", ["bf16", "e4m3", "i64"])
def test_batched_argument_limits(xr, orc, dtype):
    """Batches on both sides of 32 non-empty items and of 320 source pointers,
    with zero-length and element-aligned items mixed in, against the oracle."""
    rng = np.random.default_rng(31)
    layouts = {
        "32 items": [(int(rng.integers(1, 9)), int(rng.integers(1, 20000))) for _ in range(32)],
        "33 items": [(int(rng.integers(1, 9)), int(rng.integers(1, 20000))) for _ in range(33)],
        "320 pointers": [(40, int(rng.integers(1, 5000))) for _ in range(8)],
        "321 pointers": [(40, int(rng.integers(1, 5000))) for _ in range(7)] + [(41, 777)],
    }
    for name, shapes in layouts.items():
        shapes = shapes[:5] + [(3, 0), (1, 0)] + shapes[5:]     # zero-length items
        host_srcs, items = [], []
        for k, (P, n) in enumerate(shapes):
            shift = 1 if k % 3 == 0 else 0
            srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
            host_srcs.append(srcs)
            d = [gu.to_dev(np.concatenate([np.zeros(shift, x.dtype), x]), dtype)[shift:]
                 for x in srcs]
            out = torch.zeros(n + shift, dtype=gu.torch_dtype(dtype), device="cuda")[shift:]
            items.append((d, out))
        xr.batched_reduce(items, "sum", dtype=dtype)
        torch.cuda.synchronize()
        for k, (srcs, (_, out)) in enumerate(zip(host_srcs, items)):
            if srcs[0].size:
                gu.assert_parity(out, orc.allreduce_local(srcs, dtype, "sum"), dtype, "sum",
                                 f"{name}: item {k}")


def test_specials_exact(xr):
    """Hand-picked columns through the GPU: -0 columns, overflow, subnormal sums,
    NaN canonicalisation for max/min, bf16 ties."""
    cases = [
        ("f32", "sum", [0x80000000, 0x80000000], 0x80000000),
        ("f32", "sum", [0x00000001, 0x00000001], 0x00000002),
        ("f32", "sum", [0x7F7FFFFF, 0x7F7FFFFF, 0xFF7FFFFF], 0x7F800000),
        ("f32", "sum", [0x3F800000, 0x33800000, 0x33800000], 0x3F800000),
        ("f32", "max", [0x80000000, 0x00000000], 0x00000000),
        ("f32", "min", [0x00000000, 0x80000000], 0x80000000),
        ("f32", "max", [0x3F800000, 0x7FC00001], 0x7FC00000),
        ("f32", "min", [0xFFC00000, 0x3F800000], 0x7FC00000),
        ("bf16", "sum", [0x3F80, 0x3B80, 0x3B80], 0x3F81),
        ("bf16", "sum", [0x3F80, 0x3B80], 0x3F80),
        ("bf16", "sum", [0x7F7F, 0x7F7F], 0x7F80),
        ("bf16", "sum", [0x0001, 0x0001], 0x0002),
        ("bf16", "max", [0x8000, 0x0000], 0x0000),
        ("bf16", "max", [0x7FC1, 0x0000], 0x7FC0),
    ]
    for dtype, op, col, expect in cases:
        n = 4096 + 3   # vector body and scalar tail both see the column
        srcs = [np.full(n, v, gu.NP_BITS[dtype]).view(wl.NP_TYPES[dtype]) for v in col]
        got = gu.bits(_run_allreduce(xr, srcs, dtype, op), dtype)
        assert np.all(got == expect), (dtype, op, [hex(c) for c in col], hex(int(got[0])),
                                       hex(int(got[-1])))


@pytest.mark.parametrize("on_device", [False, True])
def test_batched_beyond_round_robin_limit(xr, orc, on_device):
    """More items than the round-robin plan holds (8192): host descriptors
    take the tile table (or, past its size, the host-planned range kernel),
    device descriptors the grouped kernel (141 runs of 64 items); every item
    against the oracle."""
    rng = np.random.default_rng(77)
    K = 9000
    sizes = rng.integers(1, 600, size=K)
    nsrcs = rng.integers(1, 5, size=K)
    total_in = int(sum(int(n) * int(p) for n, p in zip(sizes, nsrcs)))
    flat = pins.random_column_values(rng, "bf16", total_in)
    src_dev = gu.to_dev(flat, "bf16")
    out_dev = torch.zeros(int(sizes.sum()), dtype=torch.bfloat16, device="cuda")
    items, host_srcs, outs = [], [], []
    pos = opos = 0
    for n, P in zip(sizes.tolist(), nsrcs.tolist()):
        s = [flat[pos + q * n: pos + (q + 1) * n] for q in range(P)]
        d = [src_dev[pos + q * n: pos + (q + 1) * n] for q in range(P)]
        pos += n * P
        o = out_dev[opos: opos + n]
        opos += n
        host_srcs.append(s)
        items.append((d, o))
        outs.append(o)
    if on_device:
        keep, rows = [], []
        for d, o in items:
            pa = torch.tensor([x.data_ptr() for x in d], dtype=torch.int64, device="cuda")
            keep.append(pa)
            rows.append((pa.data_ptr(), o.data_ptr(), o.numel(), len(d), 0))
        arr = np.zeros(len(rows), xr.ITEM_DTYPE)
        for k, r in enumerate(rows):
            arr[k] = r
        xr.batched_reduce(torch.from_numpy(arr.view(np.uint8).copy()).to("cuda"), "sum",
                          dtype="bf16")
    else:
        xr.batched_reduce(items, "sum", dtype="bf16")
    torch.cuda.synchronize()
    got = gu.bits(out_dev, "bf16")
    exp = np.concatenate([orc.allreduce_local(s, "bf16", "sum") for s in host_srcs])
    gu.assert_parity(got, exp, "bf16", "sum", f"{K} items, device={on_device}")


@pytest.mark.parametrize("K", [65536, 65537])
def test_batched_tile_list_entry_width(xr, orc, K):
    """Host descriptors on both sides of the tile list's 16-bit entries (at
    most 65536 items) and its 32-bit ones: K int32 items of 1..40 elements
    over two sources, laid end to end, so the concatenated outputs equal one
    oracle reduction of the concatenated sources."""
    rng = np.random.default_rng(K)
    sizes = rng.integers(1, 41, size=K)
    sizes[-1] = 4097                        # the last item spans two tiles
    total = int(sizes.sum())
    srcs_np = [pins.random_column_values(rng, "i32", total) for _ in range(2)]
    d = [gu.to_dev(s, "i32") for s in srcs_np]
    out = torch.zeros(total, dtype=torch.int32, device="cuda")
    items, pos = [], 0
    for n in sizes.tolist():
        items.append(([x[pos:pos + n] for x in d], out[pos:pos + n]))
        pos += n
    xr.batched_reduce(items, "sum", dtype="i32")
    torch.cuda.synchronize()
    gu.assert_parity(out, orc.allreduce_local(srcs_np, "i32", "sum"), "i32", "sum", f"K={K}")


def _staged_bytes(sizes, nsrc, tile_elems):
    """Bytes a host batch stages when it takes the tile-list layout: 32 per
    item, the item of every tile (2 bytes each up to 65536 items, padded to
    8 bytes) and 8 per source pointer."""
    tiles = int(((np.asarray(sizes) + tile_elems - 1) // tile_elems).sum())
    width = 2 if len(sizes) <= 65536 else 4
    return 32 * len(sizes) + (width * tiles + 7) // 8 * 8 + 8 * nsrc * len(sizes)


@pytest.mark.parametrize("dtype", ["bf16", "f32", "u8", "f64"])
@pytest.mark.parametrize("mode", ["host", "device", "device_small"])
def test_batched_element_offsets(xr, orc, dtype, mode):
    """Batch items whose buffers are element- but not 16-byte aligned: items
    whose pointers all sit at one offset within 16 bytes fold the elements
    before the next boundary one by one and take the vector path for the
    rest (every offset; lengths below, at and past that lead, several tiles;
    up to 8 sources and the general tile's 9-17); items whose sources share
    an offset and whose output sits at another read in vectors and store
    realigned (every pair of offsets, lengths from just past the lead to
    several tiles); items whose sources sit at different offsets read
    vectors realigned to the output's grid, or go element by element when
    too short.  Host descriptors (the tile-table kernel), device
    descriptors past 64 items (the queue kernel; under graph capture runs
    dealt tile by tile) and a device batch of at most 64 items (one run:
    the round-robin kernel); canaries between the outputs stay untouched."""
    on_device = mode != "host"
    rng = np.random.default_rng(19 + on_device + (mode == "device_small"))
    es = {"bf16": 2, "f32": 4, "u8": 1, "f64": 8}[dtype]
    items_np, specs = [], []
    for m in range(es, 16, es):
        lead = (16 - m) // es
        for n in (1, lead - 1, lead, lead + 1, lead + 16 // es + 3, 9000, 40001):
            if n >= 1:
                specs.append(("common", m, n, m))
    specs += [("sources differ", es, 9000, es), ("sources differ", 16 - es, 3, 16 - es)]
    split = []
    for m in range(0, 16, es):
        lead = (16 - m) % 16 // es
        for j, do in enumerate(d for d in range(0, 16, es) if d != m):
            split.append(("output differs", m, (lead + 1, lead + 16 // es + 3, 9000, 40001)[j % 4], do))
    # sources at two offsets, lengths on both sides of the shortest realigned
    # launch (the lead is 16 to 31 bytes, then two vectors) and long
    differ = [("sources differ", m, n, (m + 3 * es) % 16)
              for m in sorted({0, es, 16 - es}) for n in (48 // es + 2, 64 // es + 5, 40001)]
    if mode == "device_small":
        specs = split[::max(1, len(split) // 50)][:50] + differ[:10]
    else:
        specs += split + differ
    if mode == "device":   # past 64 items: the queue kernel, not the one-run kernel
        specs = (specs * (70 // len(specs) + 1))[:max(70, len(specs))]
    keep, items, rows, outs, G = [], [], [], [], 64
    for k, (kind, m, n, do) in enumerate(specs):
        P = (1, 3, 8, 9, 17)[k % 5]
        srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
        items_np.append(srcs)
        views = []
        for p, a in enumerate(srcs):
            o = m if kind != "sources differ" or p % 2 == 0 else (m + es) % 16
            big = torch.zeros(o + n * es + 16, dtype=torch.uint8, device="cuda")
            v = big[o:o + n * es].view(gu.torch_dtype(dtype))
            v.copy_(gu.to_dev(a, dtype))
            keep.append(big)
            views.append(v)
        store = torch.full((G + do + n * es + G,), 0x5A, dtype=torch.uint8, device="cuda")
        out = store[G + do:G + do + n * es].view(gu.torch_dtype(dtype))
        outs.append((store, out, do, n, kind, m, P))
        items.append((views, out))
        if on_device:
            pa = torch.tensor([v.data_ptr() for v in views], dtype=torch.int64, device="cuda")
            keep.append(pa)
            rows.append((pa.data_ptr(), out.data_ptr(), n, P, 0))
    torch.cuda.synchronize()
    if on_device:
        arr = np.zeros(len(rows), xr.ITEM_DTYPE)
        for k, r in enumerate(rows):
            arr[k] = r
        desc = torch.from_numpy(arr.view(np.uint8).copy()).to("cuda")
        xr.batched_reduce(desc, "sum", dtype=dtype)
    else:
        xr.batched_reduce(items, "sum", dtype=dtype)
    torch.cuda.synchronize()
    exps = [orc.allreduce_local(srcs, dtype, "sum") for srcs in items_np]

    def check(how):
        for exp, (store, out, do, n, kind, m, P) in zip(exps, outs):
            what = f"{kind} {dtype} P={P} offset={m} output offset={do} n={n} {how}"
            gu.assert_parity(out, exp, dtype, "sum", what)
            raw = store.cpu().numpy()
            assert np.all(raw[:G + do] == 0x5A), what
            assert np.all(raw[G + do + n * es:] == 0x5A), what

    check(f"{mode} descriptors")
    if on_device:
        # under graph capture the batch runs as runs of items dealt tile by
        # tile (not the queue kernel); replayed twice over zeroed outputs
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            xr.batched_reduce(desc, "sum", dtype=dtype)
        for r in range(2):
            for _, out, *_ in outs:
                out.view(torch.uint8).zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            check(f"graph replay {r}")


def test_batched_host_caller_stream_destroyed(xr, orc):
    """Host batches on streams the caller destroys as soon as each call has
    finished (more such streams than the library has staging slots; batches
    read in place, copied on the caller's stream and copied on the library's
    side stream), then host batches on the current stream: every call
    succeeds and every item matches the oracle.  The library keeps no event
    on a caller's stream (waiting later for an event last recorded on a
    destroyed stream fails in the runtime)."""
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipStreamCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    hip.hipStreamSynchronize.argtypes = [ctypes.c_void_p]
    rng = np.random.default_rng(77)
    for r in range(12):
        K, nsrc = ((20, 3), (2000, 3), (3000, 8))[r % 3]
        sizes = rng.integers(1, 300, size=K)
        srcs_np = [[pins.random_column_values(rng, "f32", int(n)) for _ in range(nsrc)]
                   for n in sizes]
        total = int(sizes.sum())
        flat = [gu.to_dev(np.concatenate([row[p] for row in srcs_np]), "f32")
                for p in range(nsrc)]
        out = torch.zeros(total, dtype=torch.float32, device="cuda")
        items, pos = [], 0
        for n in sizes.tolist():
            items.append(([f[pos:pos + n] for f in flat], out[pos:pos + n]))
            pos += n
        torch.cuda.synchronize()
        if r < 9 and r % 2 == 0:
            h = ctypes.c_void_p()
            assert hip.hipStreamCreate(ctypes.byref(h)) == 0
            xr.batched_reduce(items, "sum", dtype="f32", stream=h.value)
            assert hip.hipStreamSynchronize(h) == 0
            assert hip.hipStreamDestroy(h) == 0
        elif r < 9:
            # a CU-masked stream (a hardware queue of its own), destroyed
            # through the library, with other runtime objects made and freed
            # after it
            a, b = xr.stream_create_partition(8)
            xr.batched_reduce(items, "sum", dtype="f32", stream=b)
            xr.stream_destroy(a)
            xr.stream_destroy(b)
            junk = [torch.empty(1 << 16).pin_memory() for _ in range(4)]
            side = torch.cuda.Stream()
            with torch.cuda.stream(side):
                torch.ones(16, device="cuda").add_(1)
            side.synchronize()
            del junk
        else:
            xr.batched_reduce(items, "sum", dtype="f32")
            torch.cuda.synchronize()
        exp = np.concatenate([orc.allreduce_local(row, "f32", "sum") for row in srcs_np])
        gu.assert_parity(out, exp, "f32", "sum", f"round {r} (K={K}, nsrc={nsrc})")


@pytest.mark.parametrize("K,nruns,maxn,nsrc", [(3000, 12, 300, 8), (40, 12, 300, 3)])
def test_batched_host_batches_back_to_back(xr, orc, K, nruns, maxn, nsrc):
    """Host batches enqueued back to back on two alternating caller streams
    with no synchronisation in between, so the four staging slots are reused
    while earlier batches may still run: 3000 items of 8 sources (staged data
    past 256 KiB, copied on the library's own stream, which the caller's
    stream then waits for) and 40 items of 3 sources (one round of
    workgroups and at most 64 KiB: read by the kernel from the pinned slot
    itself).  Every batch must still see its own descriptors."""
    rng = np.random.default_rng(61 + K)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    runs = []
    for r in range(nruns):
        sizes = rng.integers(1, maxn, size=K)
        need = _staged_bytes(sizes, nsrc, 512 * 8)
        if K == 3000:
            assert need >= 256 << 10, need          # the side-stream copy
        else:
            assert need <= 64 << 10 and K <= 2 * cus, need   # read in place
        total = int(sizes.sum())
        srcs_np = [pins.random_column_values(rng, "bf16", total) for _ in range(nsrc)]
        d = [gu.to_dev(s, "bf16") for s in srcs_np]
        out = torch.zeros(total, dtype=torch.bfloat16, device="cuda")
        items, pos = [], 0
        for n in sizes.tolist():
            items.append(([x[pos:pos + n] for x in d], out[pos:pos + n]))
            pos += n
        runs.append((srcs_np, d, out, items))
    torch.cuda.synchronize()
    for r, (_, _, _, items) in enumerate(runs):
        with torch.cuda.stream(streams[r % 2]):
            xr.batched_reduce(items, "sum", dtype="bf16")
    torch.cuda.synchronize()
    for r, (srcs_np, _, out, _) in enumerate(runs):
        gu.assert_parity(out, orc.allreduce_local(srcs_np, "bf16", "sum"), "bf16", "sum",
                         f"batch {r}")
