"""Seeded synthetic inputs for the reduce-step workloads.

This module is shared by the tests, the benchmark and the smoke check, and
holds none of the reduction's arithmetic: it only draws random numbers and
lays them out.  The shapes follow the message sizes the paper quotes for its
collectives (8 MB FTAR chunks, gradient buckets, small inference messages;
Sections 5 and 6), since the paper's own workloads are proprietary traces.

Generator: a stream ``seed`` of n values is cut into chunks of 2^22
elements; chunk c is drawn from numpy ``Generator(PCG64(SeedSequence([seed,
c])))``, so chunks can be drawn in parallel threads and any prefix of a
stream is the same whatever n is.  Float values are drawn in binary32; bf16
inputs are those binary32 draws converted by PyTorch's CPU
``to(torch.bfloat16)`` (a library conversion, round to nearest even).  bf16
arrays are carried as uint16 bit patterns.

Workloads (M = 2^20, K = 2^10 elements):
  c1   allreduce_local  P=4  x 1M  f32  sum   U[-1,1]
  c2   allreduce_local  P=8  x 64M bf16 sum   N(0,1)*1e-3       (gradient bucket)
  c3   step-wise        16 chunks x 1M bf16 sum N(0,1), INIT + 15 steps + cast
  c4   batched_reduce   4096 items, P=8, bf16 sum U[-1,1], per-source size
                        log-uniform on [8 KiB, 1 MiB]
  c5a  allreduce_local  P=32 x 8M  i32  sum   uniform over all int32
  c5b  allreduce_local  P=32 x 8M  f32  max   N(0,1) with +-inf and +-0 mixed in
  c2fp8 allreduce_local P=8  x 128M fp8 e4m3 sum, random sign, magnitudes
                        log-uniform over [2^-9, 4) (the gradient bucket's
                        footprint, 128 MiB per source, in e4m3)
  sim  allreduce_sim    G=8 ranks x 64M bf16 sum N(0,1)*1e-3 per rank (a c2-sized
                        gradient bucket AllReduced over 8 simulated ranks; the
                        send buffer of rank r is source r), ring schedule, one
                        launch per step
  sim1 allreduce_sim    the same inputs, ring schedule with every step in one
                        launch (messages forwarded in registers)
"""
from __future__ import annotations

import math
import threading
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

M = 1 << 20

NP_TYPES = {"f32": np.float32, "bf16": np.uint16, "i32": np.int32, "u32": np.uint32,
            "e4m3": np.uint8}
ELEM_SIZE = {"f32": 4, "bf16": 2, "i32": 4, "u32": 4, "e4m3": 1}


@dataclass(frozen=True)
class Workload:
    name: str
    kind: str          # "allreduce" | "stepwise" | "batched" | "sim"
    dtype: str
    op: str
    nsrc: int
    count: int         # elements per source (per chunk for stepwise; 0 for batched)
    dist: str
    seed_base: int
    nitems: int = 0
    schedule: str = ""  # sim: "ring", "rhd", "ring1", "rhd1"

    def alg_bytes(self, sizes=None) -> int:
        """(P+1)*N*sizeof bytes of one pass (sizes: per-item counts for batched)."""
        es = ELEM_SIZE[self.dtype]
        if self.kind == "batched":
            return int(sum((self.nsrc + 1) * int(n) * es for n in sizes))
        if self.kind == "sim" and self.schedule.endswith("1"):
            # every step in one launch: each rank's send buffer read once,
            # each rank's recv buffer written once
            return 2 * self.nsrc * self.count * es
        if self.kind == "sim":
            # G-1 reduce steps reading two chunks and writing one, G-1 copy
            # steps reading one and writing one, every chunk once per step
            return 5 * (self.nsrc - 1) * self.count * es
        return (self.nsrc + 1) * self.count * es


WORKLOADS = {
    "c1": Workload("c1", "allreduce", "f32", "sum", 4, M, "uniform", 1000),
    "c2": Workload("c2", "allreduce", "bf16", "sum", 8, 64 * M, "normal_1e-3", 2000),
    "c3": Workload("c3", "stepwise", "bf16", "sum", 16, M, "normal", 3000),
    "c4": Workload("c4", "batched", "bf16", "sum", 8, 0, "uniform", 4000, nitems=4096),
    "c5a": Workload("c5a", "allreduce", "i32", "sum", 32, 8 * M, "int32", 5000),
    "c5b": Workload("c5b", "allreduce", "f32", "max", 32, 8 * M, "normal_specials", 5100),
    "sim": Workload("sim", "sim", "bf16", "sum", 8, 64 * M, "normal_1e-3", 7000,
                    schedule="ring"),
    "sim1": Workload("sim1", "sim", "bf16", "sum", 8, 64 * M, "normal_1e-3", 7000,
                     schedule="ring1"),
    "c2fp8": Workload("c2fp8", "allreduce", "e4m3", "sum", 8, 128 * M, "fp8_loguniform", 8000),
}


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """binary32 array -> bf16 bit patterns, using PyTorch's CPU conversion."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


CHUNK = 1 << 22
_tls = threading.local()


def _scratch(n: int) -> np.ndarray:
    """Per-thread float32 scratch of at least n elements (reused across chunks)."""
    buf = getattr(_tls, "buf", None)
    if buf is None or buf.size < n:
        buf = np.empty(max(n, CHUNK), np.float32)
        _tls.buf = buf
    return buf[:n]


def _fill_chunk(dist: str, out: np.ndarray, seed: int, c: int, dtype: str) -> None:
    """Draw chunk c of stream ``seed`` into ``out`` (len(out) values)."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, c])))
    n = out.size
    if dist == "int32":
        v = g.integers(-(2**31), 2**31, size=n, dtype=np.int32)
        out[:] = v if dtype == "i32" else v.view(np.uint32)
        return
    if dist == "fp8_loguniform":
        # e4m3 bytes drawn as fields: random sign, exponent field 0..8 and
        # fraction uniform, i.e. magnitudes log-uniform over [2^-9, 4)
        code = g.integers(0, 9 * 8, size=n, dtype=np.uint8)
        sign = g.integers(0, 2, size=n, dtype=np.uint8) << 7
        out[:] = code | sign
        return
    x = out if dtype == "f32" else _scratch(n)
    if dist == "uniform":                       # U[-1, 1)
        g.random(out=x, dtype=np.float32)
        x *= np.float32(2.0)
        x -= np.float32(1.0)
    elif dist == "normal":
        g.standard_normal(out=x, dtype=np.float32)
    elif dist == "normal_1e-3":
        g.standard_normal(out=x, dtype=np.float32)
        x *= np.float32(1e-3)
    elif dist == "normal_specials":
        # per element: 1% +-inf, 1% +-0.0 (signs 50/50), otherwise N(0,1)
        g.standard_normal(out=x, dtype=np.float32)
        u = g.random(size=n, dtype=np.float32)
        neg = g.random(size=n, dtype=np.float32) < 0.5
        x[u < 0.01] = np.float32(np.inf)
        x[(u >= 0.01) & (u < 0.02)] = np.float32(0.0)
        flip = (u < 0.02) & neg
        x[flip] = -x[flip]
    elif dist == "ones":
        x[:] = np.float32(1.0)
    else:
        raise ValueError(dist)
    if dtype == "bf16":
        out[:] = to_bf16_bits(x)
    elif dtype != "f32":
        raise ValueError(f"float distribution {dist} for {dtype}")


def draw(dist: str, n: int, seed: int, dtype: str, threads: int = 16) -> np.ndarray:
    """n values of distribution ``dist`` from stream ``seed`` in element type ``dtype``."""
    out = np.empty(n, NP_TYPES[dtype])
    nchunks = (n + CHUNK - 1) // CHUNK

    def fill(c):
        lo = c * CHUNK
        _fill_chunk(dist, out[lo:min(n, lo + CHUNK)], seed, c, dtype)

    if nchunks <= 1:
        for c in range(nchunks):
            fill(c)
    else:
        with ThreadPoolExecutor(max_workers=min(threads, nchunks)) as ex:
            list(ex.map(fill, range(nchunks)))
    return out


# Blocks of structured extremes in c5b: [0, 64K) every source is +-0.0 with a
# random sign; [64K, 128K) every source is -inf except one random source per
# column, which is +inf.
C5B_BLOCK = 65536


def c5b_structured(p: int, nsrc: int, seed_base: int, x: np.ndarray) -> None:
    """Overwrite the two structured blocks of source ``p`` (in place)."""
    if x.size < 2 * C5B_BLOCK:
        return
    zsign = _rng(seed_base + 900 + p).random(C5B_BLOCK) < 0.5
    z = np.zeros(C5B_BLOCK, np.float32)
    z[zsign] = np.float32(-0.0)
    x[:C5B_BLOCK] = z
    pick = _rng(seed_base + 999).integers(0, nsrc, size=C5B_BLOCK)
    blk = np.full(C5B_BLOCK, -np.inf, np.float32)
    blk[pick == p] = np.inf
    x[C5B_BLOCK:2 * C5B_BLOCK] = blk


def sources(w: Workload, count: int | None = None, nsrc: int | None = None):
    """The P source buffers of an allreduce workload (count may be shrunk for tests)."""
    n = w.count if count is None else count
    P = w.nsrc if nsrc is None else nsrc
    out = []
    for p in range(P):
        x = draw(w.dist, n, w.seed_base + p, w.dtype)
        if w.dist == "normal_specials":
            c5b_structured(p, P, w.seed_base, x)
        out.append(x)
    return out


def stepwise_chunks(w: Workload, nchunks: int | None = None, chunk: int | None = None):
    """One buffer of nchunks*chunk elements, returned as its chunk views."""
    C = w.nsrc if nchunks is None else nchunks
    n = w.count if chunk is None else chunk
    buf = draw(w.dist, C * n, w.seed_base, w.dtype)
    return [buf[c * n:(c + 1) * n] for c in range(C)]


def batched_sizes(w: Workload, nitems: int | None = None, min_bytes=8192, max_bytes=1 << 20):
    """Per-item element counts: source size log-uniform in bytes on [min_bytes, max_bytes]."""
    k = w.nitems if nitems is None else nitems
    g = _rng(w.seed_base + 999)
    u = g.uniform(math.log(min_bytes), math.log(max_bytes), size=k)
    es = ELEM_SIZE[w.dtype]
    return np.maximum(1, np.rint(np.exp(u) / es)).astype(np.int64)


ARENA_ALIGN = 256  # bytes


def batched_layout(sizes, nsrc: int, dtype: str):
    """Offsets (in elements) of every item's sources in one arena, each 256 B aligned.

    Returns (src_off[k][p], arena_elems)."""
    es = ELEM_SIZE[dtype]
    step = ARENA_ALIGN // es
    offs = np.empty((len(sizes), nsrc), np.int64)
    pos = 0
    for k, n in enumerate(sizes):
        for p in range(nsrc):
            offs[k, p] = pos
            pos += (int(n) + step - 1) // step * step
    return offs, pos


def batched_arena(w: Workload, sizes, nsrc: int | None = None):
    """The whole source arena of a batched workload, drawn as one stream."""
    P = w.nsrc if nsrc is None else nsrc
    offs, total = batched_layout(sizes, P, w.dtype)
    arena = draw(w.dist, total, w.seed_base, w.dtype)
    return arena, offs
