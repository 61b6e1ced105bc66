"""CPU oracle for one rank's reduce step (test infrastructure only).

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg may import this package.  The product library never
imports, links or calls it, and it shares no code with the HIP path.

The arithmetic lives in ``xred_oracle.c`` (plain C, binary32 with
round-to-nearest-even, no contraction, subnormals kept); this module only
builds it with gcc and marshals numpy arrays through ctypes.  Every function
follows the definition in the C file's header: a left fold in source order
0..P-1 of up-converted elements, converted back with round-to-nearest-even
(the per-rank reduce of the FTAR ring, Section 5, and the ReduceScatter /
AllReduce semantics of Section 2.2).

Element arrays are numpy arrays: float32 for ``f32``, float64 for ``f64``,
uint16 bit patterns for ``bf16`` and ``f16``, uint8 bit patterns for ``e4m3``
and ``e5m2``, int8 / uint8 / int32 / uint32 / int64 / uint64 for the integer
types.  Step-wise accumulators are float32 arrays for the binary32-accumulated
float dtypes, float64 for ``f64``, uint32 for 8- and 32-bit and uint64 for
64-bit integer dtypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

HERE = Path(__file__).resolve().parent
SRC = HERE / "xred_oracle.c"
LIB = HERE / "libxred_oracle.so"

# -ffp-contract=off: no fused multiply-add; no fast-math: IEEE binary32
# semantics with subnormals and NaNs honoured.
CFLAGS = [
    "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
    "-ffp-contract=off", "-fno-fast-math", "-fno-finite-math-only",
]

DTYPES = {"f32": (10, np.float32), "bf16": (11, np.uint16), "f16": (12, np.uint16),
          "i32": (13, np.int32), "u32": (14, np.uint32), "i64": (15, np.int64),
          "u64": (16, np.uint64), "e4m3": (17, np.uint8), "e5m2": (18, np.uint8),
          "f64": (30, np.float64), "i8": (31, np.int8), "u8": (32, np.uint8)}
OPS = {"sum": 20, "prod": 21, "max": 22, "min": 23, "avg": 24}
ACC_NP = {"f32": np.float32, "bf16": np.float32, "f16": np.float32, "e4m3": np.float32,
          "e5m2": np.float32, "i32": np.uint32, "u32": np.uint32, "i64": np.uint64,
          "u64": np.uint64, "f64": np.float64, "i8": np.uint32, "u8": np.uint32}
_INIT, _FINAL = 1, 2


def build(src: Path = SRC, out: Path = LIB, extra_flags=()) -> Path:
    """Compile the oracle (gcc) to a shared library and return its path."""
    cmd = ["gcc", *CFLAGS, *extra_flags, str(src), "-o", str(out), "-lm"]
    subprocess.run(cmd, check=True)
    return out


class OracleError(RuntimeError):
    pass


def _ptr(a: np.ndarray) -> ctypes.c_void_p:
    return ctypes.c_void_p(a.ctypes.data)


class Oracle:
    """ctypes wrapper around one built copy of the oracle library."""

    def __init__(self, path: Path = LIB):
        self.path = Path(path)
        L = ctypes.CDLL(str(self.path))
        vp, u64, i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int
        L.xo_allreduce_local.argtypes = [vp, i32, vp, u64, i32, i32, i32]
        L.xo_reduce_scatter_local.argtypes = [vp, i32, i32, vp, u64, i32, i32, i32]
        L.xo_reduce_copy_step.argtypes = [vp, vp, vp, u64, i32, i32, ctypes.c_uint]
        L.xo_acc_cast.argtypes = [vp, vp, u64, i32]
        L.xo_batched_reduce.argtypes = [i32, vp, vp, vp, vp, vp, i32, i32, i32]
        L.xo_sim_chunk.argtypes = [u64, i32]
        L.xo_sim_chunk.restype = u64
        L.xo_ring_allreduce_sim.argtypes = [vp, vp, i32, u64, i32, i32, i32]
        L.xo_rhd_allreduce_sim.argtypes = [vp, vp, i32, u64, i32, i32, i32]
        L.xo_f32_bits_to_bf16.argtypes = [vp, vp, u64]
        L.xo_small_to_f32_bits.argtypes = [vp, i32, vp, u64, i32]
        L.xo_f32_bits_to_small.argtypes = [vp, vp, u64, i32]
        L.xo_bf16_to_f32_bits.argtypes = [vp, vp, u64]
        for fn in ("xo_allreduce_local", "xo_reduce_scatter_local", "xo_reduce_copy_step",
                   "xo_acc_cast", "xo_batched_reduce", "xo_ring_allreduce_sim",
                   "xo_rhd_allreduce_sim", "xo_selfcheck", "xo_max_threads", "xo_version"):
            getattr(L, fn).restype = ctypes.c_int
        self._L = L

    # -- helpers ---------------------------------------------------------
    @staticmethod
    def _check_arrays(arrs, dtype):
        np_t = DTYPES[dtype][1]
        for a in arrs:
            if a.dtype != np_t or not a.flags.c_contiguous:
                raise OracleError(f"expected contiguous {np.dtype(np_t)} array for {dtype}")

    @staticmethod
    def _ptr_table(arrs):
        tbl = (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])
        return tbl

    def selfcheck(self) -> int:
        return self._L.xo_selfcheck()

    def max_threads(self) -> int:
        return self._L.xo_max_threads()

    # -- the definition --------------------------------------------------
    def allreduce_local(self, srcs, dtype: str, op: str, nthreads: int = 1, out=None):
        """out[i] = down(fold_op(up(srcs[0][i]), ..., up(srcs[P-1][i])))."""
        srcs = list(srcs)
        self._check_arrays(srcs, dtype)
        n = srcs[0].size
        if any(s.size != n for s in srcs):
            raise OracleError("sources differ in length")
        if out is None:
            out = np.empty(n, DTYPES[dtype][1])
        tbl = self._ptr_table(srcs)
        rc = self._L.xo_allreduce_local(ctypes.cast(tbl, ctypes.c_void_p), len(srcs), _ptr(out),
                                        n, DTYPES[dtype][0], OPS[op], nthreads)
        if rc != 0:
            raise OracleError(f"xo_allreduce_local rc={rc}")
        return out

    def reduce_scatter_local(self, srcs, rank: int, dtype: str, op: str, nthreads: int = 1):
        """Shard ``rank`` of the ReduceScatter: srcs[p] holds nsrc*recvcount elements."""
        srcs = list(srcs)
        self._check_arrays(srcs, dtype)
        total = srcs[0].size
        if total % len(srcs):
            raise OracleError("send buffer length is not nsrc*recvcount")
        rc_n = total // len(srcs)
        out = np.empty(rc_n, DTYPES[dtype][1])
        tbl = self._ptr_table(srcs)
        rc = self._L.xo_reduce_scatter_local(ctypes.cast(tbl, ctypes.c_void_p), len(srcs), rank,
                                             _ptr(out), rc_n, DTYPES[dtype][0], OPS[op], nthreads)
        if rc != 0:
            raise OracleError(f"xo_reduce_scatter_local rc={rc}")
        return out

    def reduce_copy_step(self, inp, acc, dtype: str, op: str, init=False, final=False):
        """One ring ReduceCopy step; updates ``acc`` in place or returns dst on FINAL."""
        self._check_arrays([inp], dtype)
        n = inp.size
        if acc is None:
            acc = np.zeros(n, ACC_NP[dtype])
        if acc.dtype != ACC_NP[dtype] or acc.size != n:
            raise OracleError("accumulator has the wrong type or length")
        dst = np.zeros(n, DTYPES[dtype][1])
        flags = (_INIT if init else 0) | (_FINAL if final else 0)
        rc = self._L.xo_reduce_copy_step(_ptr(inp), _ptr(acc), _ptr(dst), n, DTYPES[dtype][0],
                                         OPS[op], flags)
        if rc != 0:
            raise OracleError(f"xo_reduce_copy_step rc={rc}")
        return dst if final else acc

    def acc_cast(self, acc, dtype: str):
        n = acc.size
        if acc.dtype != ACC_NP[dtype]:
            raise OracleError("accumulator has the wrong type")
        dst = np.empty(n, DTYPES[dtype][1])
        rc = self._L.xo_acc_cast(_ptr(acc), _ptr(dst), n, DTYPES[dtype][0])
        if rc != 0:
            raise OracleError(f"xo_acc_cast rc={rc}")
        return dst

    def batched_reduce(self, items, dtype: str, op: str, nthreads: int = 1):
        """items: list of source lists; returns one output array per item."""
        flat, offs, nsrc, outs, counts = [], [], [], [], []
        for srcs in items:
            self._check_arrays(srcs, dtype)
            offs.append(len(flat))
            flat.extend(srcs)
            nsrc.append(len(srcs))
            outs.append(np.empty(srcs[0].size, DTYPES[dtype][1]))
            counts.append(srcs[0].size)
        k = len(items)
        tbl = self._ptr_table(flat) if flat else (ctypes.c_void_p * 1)()
        offs_a = np.asarray(offs, np.uint64)
        nsrc_a = np.asarray(nsrc, np.int32)
        outs_t = self._ptr_table(outs) if outs else (ctypes.c_void_p * 1)()
        cnt_a = np.asarray(counts, np.uint64)
        rc = self._L.xo_batched_reduce(k, ctypes.cast(tbl, ctypes.c_void_p), _ptr(offs_a),
                                       _ptr(nsrc_a), ctypes.cast(outs_t, ctypes.c_void_p),
                                       _ptr(cnt_a), DTYPES[dtype][0], OPS[op], nthreads)
        if rc != 0:
            raise OracleError(f"xo_batched_reduce rc={rc}")
        return outs

    def sim_chunk(self, count: int, nranks: int) -> int:
        """Chunk length of the simulated schedules (ceil(count/G) rounded up to 64)."""
        return int(self._L.xo_sim_chunk(count, nranks))

    def allreduce_sim(self, sends, dtype: str, op: str, algo: str = "ring", nthreads: int = 1):
        """A whole AllReduce over len(sends) simulated ranks, message by message
        (``algo`` "ring" or "rhd"); returns every rank's output buffer."""
        sends = list(sends)
        self._check_arrays(sends, dtype)
        n = sends[0].size
        if any(s.size != n for s in sends):
            raise OracleError("send buffers differ in length")
        outs = [np.empty(n, DTYPES[dtype][1]) for _ in sends]
        fn = {"ring": self._L.xo_ring_allreduce_sim, "rhd": self._L.xo_rhd_allreduce_sim}[algo]
        rc = fn(ctypes.cast(self._ptr_table(sends), ctypes.c_void_p),
                ctypes.cast(self._ptr_table(outs), ctypes.c_void_p), len(sends), n,
                DTYPES[dtype][0], OPS[op], nthreads)
        if rc != 0:
            raise OracleError(f"{algo} allreduce simulation rc={rc}")
        return outs

    def f32_bits_to_bf16(self, bits: np.ndarray) -> np.ndarray:
        bits = np.ascontiguousarray(bits, np.uint32)
        out = np.empty(bits.size, np.uint16)
        self._L.xo_f32_bits_to_bf16(_ptr(bits), _ptr(out), bits.size)
        return out

    def small_to_f32_bits(self, h: np.ndarray, dtype: str) -> np.ndarray:
        """Exact widening of f16 / e4m3 / e5m2 bit patterns to binary32 bits."""
        np_t = DTYPES[dtype][1]
        h = np.ascontiguousarray(h, np_t)
        out = np.empty(h.size, np.uint32)
        self._L.xo_small_to_f32_bits(_ptr(h), np.dtype(np_t).itemsize, _ptr(out), h.size,
                                     DTYPES[dtype][0])
        return out

    def f32_bits_to_small(self, bits: np.ndarray, dtype: str) -> np.ndarray:
        """binary32 bits -> f16 / e4m3 / e5m2 bits (round to nearest even)."""
        bits = np.ascontiguousarray(bits, np.uint32)
        out = np.empty(bits.size, DTYPES[dtype][1])
        self._L.xo_f32_bits_to_small(_ptr(bits), _ptr(out), bits.size, DTYPES[dtype][0])
        return out

    def bf16_to_f32_bits(self, h: np.ndarray) -> np.ndarray:
        h = np.ascontiguousarray(h, np.uint16)
        out = np.empty(h.size, np.uint32)
        self._L.xo_bf16_to_f32_bits(_ptr(h), _ptr(out), h.size)
        return out


_default = None


def load() -> Oracle:
    """Load the built oracle, building it with gcc only if nothing is built."""
    global _default
    if _default is None:
        if not LIB.exists() or LIB.stat().st_mtime < SRC.stat().st_mtime:
            build()
        _default = Oracle(LIB)
        if _default.selfcheck() != 0:
            raise OracleError("floating-point environment flushes subnormals or does not "
                              f"round to nearest (selfcheck {_default.selfcheck()})")
    return _default


def host_cores() -> int:
    """Number of cores this process may run on."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1
