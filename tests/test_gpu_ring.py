"""GPU parity and flag protocol of xred_ring_reduce (all ring steps in one
launch, accumulator on chip, producer flags).

The result must equal the oracle's left fold over the chunks bit for bit,
whether the chunks are ready at launch, gated by flags set before the launch,
or released one by one by a host thread while the kernel runs.  Flags live in
host memory allocated with hipHostMalloc and are passed to the kernel through
hipHostGetDevicePointer.  The timeout case uses a flag the host never sets
and a tiny spin limit, so the kernel still exits normally.
"""
import ctypes
import threading
import time

import numpy as np
import pytest

import gpu_util as gu
import pins
import workloads as wl

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

DTYPES = ("f32", "bf16", "i32", "u32")
OPS = ("sum", "prod", "max", "min")


@pytest.fixture(scope="module")
def xr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2510_20171_amd as xr
    xr.load()
    return xr


class PinnedWords:
    """n uint32 words of host memory the GPU reads coherently."""

    def __init__(self, n: int):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipHostMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t,
                                           ctypes.c_uint]
        self.hip.hipHostGetDevicePointer.argtypes = [ctypes.POINTER(ctypes.c_void_p),
                                                     ctypes.c_void_p, ctypes.c_uint]
        self.hip.hipHostFree.argtypes = [ctypes.c_void_p]
        self.n = n
        self.host = ctypes.c_void_p()
        assert self.hip.hipHostMalloc(ctypes.byref(self.host), 4 * n, 0) == 0
        self.dev = ctypes.c_void_p()
        assert self.hip.hipHostGetDevicePointer(ctypes.byref(self.dev), self.host, 0) == 0
        self.words = (ctypes.c_uint32 * n).from_address(self.host.value)
        for i in range(n):
            self.words[i] = 0

    def set(self, i: int, v: int) -> None:
        self.words[i] = v & 0xFFFFFFFF

    def get(self, i: int) -> int:
        return int(self.words[i])

    def free(self) -> None:
        if self.host:
            self.hip.hipHostFree(self.host)
            self.host = None


def _ring(xr, chunks_np, dtype, op, ready=None, epoch=1, timeout_us=2_000_000, status=None,
          out=None):
    L = xr.load()
    d = [gu.to_dev(c, dtype) for c in chunks_np]
    if out is None:
        out = torch.empty_like(d[0])
    arr = xr._lib.ptr_array([c.data_ptr() for c in d])
    st = L.xred_ring_reduce(arr, len(d), ctypes.c_void_p(out.data_ptr()), out.numel(),
                            xr.DTYPE[dtype], xr.OP[op],
                            ready.dev if ready is not None else None, epoch, timeout_us,
                            status.dev if status is not None else None,
                            ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    xr._lib.check(st)
    return out, d


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("op", OPS)
def test_ring_parity_no_flags(xr, orc, dtype, op):
    rng = np.random.default_rng(31 + 10 * DTYPES.index(dtype) + OPS.index(op))
    for nchunks in (1, 2, 3, 8, 9, 16, 33, 64):
        for n in (1, 9, 4096 * 8 + 3, 1 << 17):
            if n * nchunks > (1 << 21):
                continue
            chunks = [pins.random_column_values(rng, dtype, n) for _ in range(nchunks)]
            out, _ = _ring(xr, chunks, dtype, op)
            torch.cuda.synchronize()
            gu.assert_parity(out, orc.allreduce_local(chunks, dtype, op), dtype, op,
                             f"ring {dtype} {op} chunks={nchunks} n={n}")


def test_ring_c3_full_and_multi_tile(xr, orc):
    """The step-wise workload (16 x 2^20 bf16) in one launch, and a chunk large
    enough that each workgroup holds several accumulator tiles."""
    w = wl.WORKLOADS["c3"]
    chunks = [c.copy() for c in wl.stepwise_chunks(w)]
    out, _ = _ring(xr, chunks, "bf16", "sum")
    torch.cuda.synchronize()
    gu.assert_parity(out, orc.allreduce_local(chunks, "bf16", "sum", nthreads=8), "bf16", "sum",
                     "c3 ring")
    cap = xr.ring_max_count("bf16")
    n = min(cap, 3 << 21) - 5
    big = [wl.draw("normal", n, 3100 + s, "bf16") for s in range(4)]
    out, _ = _ring(xr, big, "bf16", "sum")
    torch.cuda.synchronize()
    gu.assert_parity(out, orc.allreduce_local(big, "bf16", "sum", nthreads=8), "bf16", "sum",
                     f"ring n={n} (capacity {cap})")


def test_ring_capacity_is_enforced(xr):
    cap = xr.ring_max_count("bf16")
    assert cap >= (1 << 20)
    a = torch.empty(cap + 8, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(xr.XredError) as e:
        xr.ring_reduce([a, a], torch.empty_like(a))
    assert e.value.name == "XRED_UNSUPPORTED"


def test_ring_flags_preset_and_ahead(xr, orc):
    rng = np.random.default_rng(5)
    chunks = [pins.random_column_values(rng, "bf16", 70001 * 8) for _ in range(12)]
    exp = orc.allreduce_local(chunks, "bf16", "sum")
    flags = PinnedWords(12)
    try:
        for epoch, val in ((5, 5), (9, 12)):      # equal, and producer ahead of epoch
            for s in range(12):
                flags.set(s, val)
            out, _ = _ring(xr, chunks, "bf16", "sum", ready=flags, epoch=epoch)
            torch.cuda.synchronize()
            gu.assert_parity(out, exp, "bf16", "sum", f"flags preset epoch={epoch}")
    finally:
        flags.free()


def test_ring_host_producer(xr, orc):
    """A host thread releases the chunks one by one while the kernel runs."""
    rng = np.random.default_rng(6)
    nchunks = 16
    chunks = [pins.random_column_values(rng, "f32", 1 << 18) for _ in range(nchunks)]
    exp = orc.allreduce_local(chunks, "f32", "sum")
    flags = PinnedWords(nchunks)
    status = PinnedWords(1)
    try:
        epoch = 3
        for s in range(nchunks):
            flags.set(s, epoch - 1)
        out, keep = _ring(xr, chunks, "f32", "sum", ready=flags, epoch=epoch, status=status,
                          timeout_us=5_000_000)

        def produce():
            for s in range(nchunks):
                time.sleep(0.0005)
                flags.set(s, epoch)
        th = threading.Thread(target=produce)
        th.start()
        th.join()
        torch.cuda.synchronize()
        assert status.get(0) == 0, "a wait timed out"
        gu.assert_parity(out, exp, "f32", "sum", "host producer")
    finally:
        flags.free()
        status.free()


def test_ring_timeout_exits(xr):
    """Flags the host never sets: every workgroup gives up after the spin limit,
    reports it in *status, and the kernel ends normally."""
    chunks = [np.ones(1 << 16, np.float32) for _ in range(4)]
    flags = PinnedWords(4)
    status = PinnedWords(1)
    try:
        flags.set(0, 1)                      # chunk 0 ready, chunk 1 never
        t0 = time.perf_counter()
        _ring(xr, chunks, "f32", "sum", ready=flags, epoch=1, timeout_us=2000, status=status)
        torch.cuda.synchronize()
        assert time.perf_counter() - t0 < 5.0
        assert status.get(0) == 1
        # the library and the stream are still usable afterwards
        out, _ = _ring(xr, chunks, "f32", "sum")
        torch.cuda.synchronize()
        assert torch.all(out == 4.0)
    finally:
        flags.free()
        status.free()
