"""GPU parity of the further element types (fp16, OCP fp8 e4m3 / e5m2, int64,
uint64, fp64, int8, uint8) and of AVG, against the CPU oracle, bit for bit
(NaN payloads of float sum/prod/avg compare by NaN-ness only).

Covered for every new dtype x op: the fused reduce over source counts 1..33
and sizes from one element to several tiles with ragged tails; a size past
the one-round tile-shape switch; element-aligned buffers (scalar path);
reduce-scatter; every step-wise flag with the closing cast (binary32,
binary64, uint32 or uint64 accumulator); batched items; all steps in one launch (ring); the
simulated ring and halving-doubling schedules.  AVG runs on every float type
through the fused, reduce-scatter and batched paths.
"""
import os

import numpy as np
import pytest

import gpu_util as gu
import pins
import workloads as wl

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

NEW = ("f16", "e4m3", "e5m2", "i64", "u64", "f64", "i8", "u8")
CORES = min(16, len(os.sched_getaffinity(0)))


def ops_for(dtype):
    return pins.ops_for(dtype)


@pytest.fixture(scope="module")
def xr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    xr.load()
    return xr


def _fused(xr, srcs_np, dtype, op):
    srcs = [gu.to_dev(s, dtype) for s in srcs_np]
    out = torch.empty_like(srcs[0])
    xr.allreduce_local(srcs, out, op, dtype=dtype)
    torch.cuda.synchronize()
    return out


SIZES = (1, 15, 16, 17, 63, 4099, (1 << 17) + 5)
NSRC = (1, 2, 3, 5, 8, 9, 16, 33)


@pytest.mark.parametrize("dtype", NEW + ("f32", "bf16"))
def test_fused_matrix(xr, orc, dtype):
    rng = np.random.default_rng(101 + NEW.index(dtype) if dtype in NEW else 120 + len(dtype))
    ops = ops_for(dtype) if dtype in NEW else ("avg",)
    for op in ops:
        for P in NSRC:
            for n in SIZES:
                if P * n > (1 << 21):
                    continue
                srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
                got = _fused(xr, srcs, dtype, op)
                gu.assert_parity(got, orc.allreduce_local(srcs, dtype, op), dtype, op,
                                 f"{dtype} {op} P={P} n={n}")


@pytest.mark.parametrize("dtype,op", [("e4m3", "sum"), ("f16", "avg"), ("i64", "max"),
                                      ("e5m2", "prod"), ("f64", "avg"), ("f64", "min"),
                                      ("i8", "sum"), ("u8", "max")])
def test_past_one_round(xr, orc, dtype, op):
    """Sizes beyond the one-round launch (occupancy-capped tiles), ragged."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    vec = {"f16": 8, "e4m3": 16, "e5m2": 16, "i64": 2, "f64": 2, "i8": 16, "u8": 16}[dtype]
    n = cus * 4 * 512 * vec * 2 + 77
    rng = np.random.default_rng(7)
    base = [pins.random_column_values(rng, dtype, 65536 + 13 + 2 * p) for p in range(8)]
    srcs = [np.resize(b, n) for b in base]
    got = _fused(xr, srcs, dtype, op)
    gu.assert_parity(got, orc.allreduce_local(srcs, dtype, op, nthreads=CORES), dtype, op,
                     f"{dtype} {op} n={n}")


@pytest.mark.parametrize("dtype", NEW)
def test_element_aligned(xr, orc, dtype):
    rng = np.random.default_rng(9)
    n = 5000
    for P in (1, 3, 8):
        for op in ops_for(dtype):
            srcs_np = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
            big = [gu.to_dev(np.concatenate([np.zeros(1, s.dtype), s]), dtype) for s in srcs_np]
            outb = torch.empty_like(big[0])
            xr.allreduce_local([b[1:] for b in big], outb[1:], op, dtype=dtype)
            torch.cuda.synchronize()
            gu.assert_parity(outb[1:], orc.allreduce_local(srcs_np, dtype, op), dtype, op,
                             f"element-aligned {dtype} {op} P={P}")


@pytest.mark.parametrize("dtype", NEW)
def test_reduce_scatter(xr, orc, dtype):
    rng = np.random.default_rng(11)
    P, rc = 4, 12345
    for op in ("max", "avg" if dtype in gu.FLOATS else "sum"):
        srcs = [pins.random_column_values(rng, dtype, P * rc) for _ in range(P)]
        d = [gu.to_dev(s, dtype) for s in srcs]
        for r in range(P):
            out = torch.empty(rc, dtype=d[0].dtype, device="cuda")
            xr.reduce_scatter_local(d, r, out, op, dtype=dtype)
            torch.cuda.synchronize()
            gu.assert_parity(out, orc.reduce_scatter_local(srcs, r, dtype, op), dtype, op,
                             f"rs {dtype} {op} rank {r}")


@pytest.mark.parametrize("dtype", NEW)
def test_stepwise(xr, orc, dtype):
    rng = np.random.default_rng(13)
    acc_t, acc_bits = {"i64": (torch.int64, "u64"), "u64": (torch.int64, "u64"),
                       "f64": (torch.float64, "f64"), "i8": (torch.int32, "u32"),
                       "u8": (torch.int32, "u32")}.get(dtype, (torch.float32, "f32"))
    for op in ("sum", "max", "prod"):
        for n in (4096 * 3 + 7, 999):
            chunks = [pins.random_column_values(rng, dtype, n) for _ in range(5)]
            d = [gu.to_dev(c, dtype) for c in chunks]
            acc = torch.empty(n, dtype=acc_t, device="cuda")
            out = torch.empty_like(d[0])
            out2 = torch.empty_like(d[0])
            xr.reduce_copy_step(d[0], acc, None, op, init=True, dtype=dtype)
            for c in d[1:-1]:
                xr.reduce_copy_step(c, acc, None, op, dtype=dtype)
            acc2 = acc.clone()
            xr.reduce_copy_step(d[-1], acc, out, op, final=True, dtype=dtype)
            xr.reduce_copy_step(d[-1], acc2, None, op, dtype=dtype)
            xr.acc_cast(acc2, out2, dtype=dtype)
            torch.cuda.synchronize()
            oacc = orc.reduce_copy_step(chunks[0], None, dtype, op, init=True)
            for c in chunks[1:]:
                oacc = orc.reduce_copy_step(c, oacc, dtype, op)
            gu.assert_parity(acc2, oacc, acc_bits, op, f"step acc {dtype} {op}")
            exp = orc.allreduce_local(chunks, dtype, op)
            gu.assert_parity(out, exp, dtype, op, f"step final {dtype} {op} n={n}")
            gu.assert_parity(out2, exp, dtype, op, f"step cast {dtype} {op} n={n}")


@pytest.mark.parametrize("dtype", NEW + ("bf16",))
def test_batched(xr, orc, dtype):
    rng = np.random.default_rng(17)
    for op in ("sum", "avg" if dtype in gu.FLOATS else "max"):
        items_np, items = [], []
        for k, (P, n) in enumerate(((1, 10), (3, 4097), (8, 70001), (9, 333), (2, 1))):
            srcs = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
            items_np.append(srcs)
            items.append(([gu.to_dev(s, dtype) for s in srcs],
                          torch.empty(n, dtype=gu.torch_dtype(dtype), device="cuda")))
        xr.batched_reduce(items, op, dtype=dtype)
        torch.cuda.synchronize()
        for k, ((_, o), srcs) in enumerate(zip(items, items_np)):
            gu.assert_parity(o, orc.allreduce_local(srcs, dtype, op), dtype, op,
                             f"batched {dtype} {op} item {k}")


@pytest.mark.parametrize("dtype", NEW)
def test_ring_and_sim(xr, orc, dtype):
    rng = np.random.default_rng(19)
    for op in ("sum", "min"):
        n = 4096 * 4 + 3
        chunks = [pins.random_column_values(rng, dtype, n) for _ in range(9)]
        d = [gu.to_dev(c, dtype) for c in chunks]
        out = torch.empty_like(d[0])
        xr.ring_reduce(d, out, op, dtype=dtype)
        torch.cuda.synchronize()
        gu.assert_parity(out, orc.allreduce_local(chunks, dtype, op), dtype, op,
                         f"ring {dtype} {op}")
        for schedule, G in (("ring", 5), ("rhd", 8), ("ring1", 5), ("rhd1", 8)):
            sends = [pins.random_column_values(rng, dtype, 64 * G + 70 + 4096) for _ in range(G)]
            sd = [gu.to_dev(s, dtype) for s in sends]
            recvs = [torch.empty_like(x) for x in sd]
            xr.allreduce_sim(sd, recvs, op, schedule=schedule, dtype=dtype)
            torch.cuda.synchronize()
            exp = orc.allreduce_sim(sends, dtype, op, schedule.rstrip("1"))
            for r in range(G):
                gu.assert_parity(recvs[r], exp[r], dtype, op, f"sim {schedule} {dtype} {op} r={r}")


def test_fp8_bucket_full(xr, orc):
    """The fp8 bucket the benchmark times: P=8 x 2^27 e4m3, sum."""
    w = wl.WORKLOADS["c2fp8"]
    srcs = wl.sources(w)
    got = _fused(xr, srcs, w.dtype, w.op)
    gu.assert_parity(got, orc.allreduce_local(srcs, w.dtype, w.op, nthreads=CORES), w.dtype,
                     w.op, "c2fp8")
