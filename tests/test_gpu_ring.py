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


@pytest.mark.parametrize("dtype", ["bf16", "f32", "u8"])
def test_ring_element_offsets(xr, orc, dtype):
    """Chunks that are element- but not 16-byte aligned, all at one offset m
    within 16 bytes: the elements before the next boundary are folded one by
    one with the tail, the rest in vectors; dst at the same offset, aligned,
    or at a third one (realigned stores).  Every offset; lengths within the
    lead, just past it, across several tiles with a ragged tail; without
    flags and with every flag set before the launch.  Canaries around dst
    stay untouched; chunks at different offsets are refused."""
    rng = np.random.default_rng(41)
    es = {"bf16": 2, "f32": 4, "u8": 1}[dtype]
    G = 64
    L = xr.load()
    cases = []
    for m in range(0, 16, es):
        lead = (16 - m) % 16 // es
        for k, do in enumerate(sorted({m, 0, (m + 3 * es) % 16})):
            n = (max(lead, 1), lead + 1, 3 * 512 * 16 // es + 5)[k % 3]
            cases.append((m, do, n))
    cases.append((es, 0, 70001))
    for k, (m, do, n) in enumerate(cases):
        P = (1, 3, 8, 16)[k % 4]
        flagged = k % 2 == 1
        chunks = [pins.random_column_values(rng, dtype, n) for _ in range(P)]
        keep, arr = [], []
        for a in chunks:
            b = torch.zeros(m + n * es + 16, dtype=torch.uint8, device="cuda")
            v = b[m:m + n * es].view(gu.torch_dtype(dtype))
            v.copy_(gu.to_dev(a, dtype))
            keep.append(b)
            arr.append(v.data_ptr())
        store = torch.full((G + do + n * es + G,), 0x5A, dtype=torch.uint8, device="cuda")
        out = store[G + do:G + do + n * es]
        flags = PinnedWords(P) if flagged else None
        if flagged:
            for i in range(P):
                flags.set(i, 1)
        torch.cuda.synchronize()
        xr._lib.check(L.xred_ring_reduce(
            xr._lib.ptr_array(arr), P, ctypes.c_void_p(out.data_ptr()), n, xr.DTYPE[dtype],
            xr.OP["sum"], flags.dev if flagged else None, 1, 2_000_000, None,
            ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)))
        torch.cuda.synchronize()
        if flagged:
            flags.free()
        what = f"ring {dtype} P={P} chunks at {m} dst at {do} n={n} flags={flagged}"
        gu.assert_parity(out.view(gu.torch_dtype(dtype)), orc.allreduce_local(chunks, dtype, "sum"),
                         dtype, "sum", what)
        raw = store.cpu().numpy()
        assert np.all(raw[:G + do] == 0x5A), what
        assert np.all(raw[G + do + n * es:] == 0x5A), what
    # one chunk at another offset: refused, nothing launched
    a = torch.zeros(4096, dtype=torch.uint8, device="cuda")
    out = torch.zeros(1024, dtype=torch.uint8, device="cuda")
    st = L.xred_ring_reduce(xr._lib.ptr_array([a.data_ptr(), a.data_ptr() + 2048 + es]), 2,
                            ctypes.c_void_p(out.data_ptr()), 64 // es, xr.DTYPE[dtype],
                            xr.OP["sum"], None, 1, 0, None,
                            ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == xr.UNSUPPORTED, st


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


def test_ring_flagged_launches_reuse_relay_slots(xr, orc):
    """Flagged launches hand readiness on through a relay word bound to their
    stream (64 per device; launches on one stream share theirs, each with its
    own ticket).  Launches enqueued back to back on one stream, alternating
    over two streams, and one on each of 72 streams (more than there are
    slots: the rest poll without a relay), each with its own output: every
    launch must fold all of its chunks, and none may take a relay value an
    earlier launch left for its own."""
    rng = np.random.default_rng(8)
    nchunks, n = 6, 3 * 4096 + 16       # several tiles; whole 16-byte vectors
    chunks = [pins.random_column_values(rng, "bf16", n) for _ in range(nchunks)]
    exp = orc.allreduce_local(chunks, "bf16", "sum")
    L = xr.load()
    d = [gu.to_dev(c, "bf16") for c in chunks]
    arr = xr._lib.ptr_array([c.data_ptr() for c in d])
    flags = PinnedWords(nchunks)
    status = PinnedWords(1)
    streams = [torch.cuda.Stream() for _ in range(72)]
    try:
        for s in range(nchunks):
            flags.set(s, 7)
        outs = [torch.full_like(d[0], float("nan")) for _ in range(232)]
        torch.cuda.synchronize()
        for k, o in enumerate(outs):
            st = streams[0] if k < 80 else streams[k % 2] if k < 160 else streams[k - 160]
            xr._lib.check(L.xred_ring_reduce(arr, nchunks, ctypes.c_void_p(o.data_ptr()), n,
                                             xr.DTYPE["bf16"], xr.OP["sum"], flags.dev, 7,
                                             2_000_000, status.dev,
                                             ctypes.c_void_p(st.cuda_stream)))
        torch.cuda.synchronize()
        assert status.get(0) == 0, "a wait timed out"
        for k, o in enumerate(outs):
            gu.assert_parity(o, exp, "bf16", "sum", f"flagged launch {k}")
    finally:
        flags.free()
        status.free()


def test_ring_flags_under_graph_capture(xr, orc):
    """Under capture there is no relay (a replay would repeat the captured
    relay ticket): each workgroup polls the flags itself.  Replays with the
    flags set, with eager work in between, give the eager bits each time."""
    rng = np.random.default_rng(9)
    nchunks, n = 5, 2 * 4096 * 8
    chunks = [pins.random_column_values(rng, "f32", n) for _ in range(nchunks)]
    exp = orc.allreduce_local(chunks, "f32", "sum")
    L = xr.load()
    d = [gu.to_dev(c, "f32") for c in chunks]
    arr = xr._lib.ptr_array([c.data_ptr() for c in d])
    flags = PinnedWords(nchunks)
    try:
        for s in range(nchunks):
            flags.set(s, 1)
        out = torch.empty_like(d[0])
        eager = torch.empty_like(d[0])
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            cs = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
            xr._lib.check(L.xred_ring_reduce(arr, nchunks, ctypes.c_void_p(out.data_ptr()), n,
                                             xr.DTYPE["f32"], xr.OP["sum"], flags.dev, 1,
                                             2_000_000, None, cs))
        for r in range(3):
            out.zero_()
            g.replay()
            torch.cuda.synchronize()
            gu.assert_parity(out, exp, "f32", "sum", f"replay {r}")
            _ring(xr, chunks, "f32", "sum", ready=flags, epoch=1, out=eager)
            torch.cuda.synchronize()
            gu.assert_parity(eager, exp, "f32", "sum", f"eager after replay {r}")
        del g
    finally:
        flags.free()
