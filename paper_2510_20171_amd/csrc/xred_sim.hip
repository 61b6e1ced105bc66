// xred_sim.hip -- a whole AllReduce over G simulated ranks on one GPU
// (xred_allreduce_sim): one launch per step of the schedule, or every step in
// one launch (see "one launch" below).
//
// Ring (the FTAR pipeline's ring, Section 5).  Rank q receives from q-1.
// ReduceScatter step j = 1..G-1: rank q folds chunk c = q-1-j, reading the
// message from rank q-1 and its own contribution, and stores the result in
// recv[q] at chunk c:
//   j = 1        the message is send[q-1] at chunk c (sendCopy is zero-copy:
//                the receiver reads the sender's buffer),
//   1 < j < G-1  the message is recv[q-1] at chunk c, stored there by rank
//                q-1 in step j-1 (RedCopy: reduce and forward in one store),
//   j = G-1      c = q: the store is rank q's reduced chunk (Reduce).
// AllGather step t = 1..G-1: rank q copies chunk q-t from recv[q-1] into
// recv[q] (RecvCopy; the copy is also the message rank q+1 reads next).
//
// Recursive halving-doubling (Section 2.2), G a power of two.  Halving step
// at distance d = G/2, ..., 1: rank q keeps the aligned group of d blocks that
// contains block q, and folds its partner q^d's partial of that group into
// its own (both read from the send buffers at the first step, from the recv
// buffers after).  Doubling step at d = 1, ..., G/2: rank q copies its
// partner's aligned group of d blocks from recv[q^d].
//
// Within a step no rank writes what another rank reads, and each rank reads
// its own elements before overwriting them, so recv[q] may be send[q].  Every
// hop computes down(up(received) (+) up(own)) with the fused kernel's tile
// code (two sources, fold order received-then-own); copies move bits.
#include "xred_dispatch.hpp"
#include "xred_internal.hpp"
#include "xred_kernels.hpp"

namespace xred {
namespace {

constexpr int kB = 256;    // threads per workgroup of the per-step kernels
constexpr int kU = 1;      // 16-byte vectors per thread per tile
// Workgroup shape of the one-launch kernel, per schedule and size: threads,
// and resident waves per CU (0: no cap).  Measured with 8 ranks x 64M bf16
// on three buffer layouts (separate allocations, allocations among freed
// holes, slices of one allocation), in microseconds against the
// traffic-only kernel with the same 8 reads and 8 writes at its best cap
// (340 / 352-355 / 344-345):
//   ring  512 threads, 8 waves (one workgroup per CU): 342-343 / 348-352 /
//         344-345; 256 threads, 12 waves: 357 / 369-375 / 383-384; 128
//         threads, 8 waves: 340-342 / 352-359 / 343-344; 512 threads, 16 or
//         24 waves: 383-395; 1024 threads, 16 waves: 386-410
//   RHD   (more partials live in registers) 64 threads, 16 waves: 347 / 345
//         / 351; 64 threads uncapped: 353-356; 128 threads uncapped:
//         363-367; 128 threads, 8 / 12 / 16 waves: 489 / 421-427 / 356-381;
//         256 threads uncapped: 380-383 / 393-394 / 410-413
// Below 8 MiB per rank the launch is a few rounds long and the smaller
// workgroups lose (8 ranks of 1M bf16: RHD 10.2 against 6.9 us, ring 6.7
// against 6.5; at 4M: ring 21.3 against 24.6, RHD 25.5 against 26.9), so
// such calls keep 256 threads, 12 waves (ring) and uncapped (RHD).
struct SimShape {
    int threads, waves;
};
constexpr SimShape kRingShape{512, 8}, kRhdShape{64, 16};
constexpr SimShape kRingSmallShape{256, 12}, kRhdSmallShape{256, 0};
constexpr uint64_t kSimLargeBytes = 8u << 20;   // bytes per rank from which the large shapes run

// One step: rank q's message, own contribution and output, already offset to
// the chunk (or group of blocks) the rank works on, and its length.
struct SimStep {
    const char *in[XRED_MAX_SRC];
    const char *own[XRED_MAX_SRC];
    char *out[XRED_MAX_SRC];
    uint64_t len[XRED_MAX_SRC];
};

template <class T>
__device__ __forceinline__ void copy_elem(const char *in, char *out, size_t i)
{
    if constexpr (T::kSize == 1)
        ((uint8_t *)out)[i] = ((const uint8_t *)in)[i];
    else if constexpr (T::kSize == 2)
        ((uint16_t *)out)[i] = ((const uint16_t *)in)[i];
    else if constexpr (T::kSize == 4)
        ((uint32_t *)out)[i] = ((const uint32_t *)in)[i];
    else
        ((uint64_t *)out)[i] = ((const uint64_t *)in)[i];
}

// Work item w of a step: rank w % G, tile w / G of that rank's range.  Vector
// tiles cover the 16-byte part; one extra tile per rank does the last
// (len % kVec) elements.  COPY: out = in bit for bit; otherwise out =
// down(up(in) (+) up(own)).
template <class T, class Op, bool COPY>
__global__ __launch_bounds__(kB) void sim_step_vec_kernel(SimStep a, int G, uint64_t tiles)
{
    constexpr uint32_t kTileBytes = (uint32_t)kB * kU * 16u;
    const uint64_t work = tiles * (uint64_t)G;
    for (uint64_t w = blockIdx.x; w < work; w += gridDim.x) {
        const int q = (int)(w % (uint64_t)G);
        const uint64_t t = w / (uint64_t)G;
        const uint64_t len = a.len[q];
        const uint64_t nvec = len / T::kVec;
        const size_t vbytes = nvec * 16;
        const uint64_t vtiles = (vbytes + kTileBytes - 1) / kTileBytes;
        if (t < vtiles) {
            const size_t off = t * kTileBytes;
            const Tile tl{off, tile_nrec(vbytes, off, kTileBytes)};
            if constexpr (COPY) {
                const rsrc_t r = make_rsrc(a.in[q] + off, tl.nrec);
                const rsrc_t o = make_rsrc(a.out[q] + off, tl.nrec);
#pragma unroll
                for (int u = 0; u < kU; ++u) {
                    const uint32_t b = (uint32_t)(u * kB + threadIdx.x) * 16u;
                    bstore<kStoreOut>(bload<kLoadStream>(r, b), o, b);
                }
            } else {
                KernargSrc<2> src;
                src.p[0] = a.in[q];
                src.p[1] = a.own[q];
                reduce_tile<T, Op, 2, kU, kB>(src, 2, a.out[q], tl);
            }
        } else if (t == vtiles && threadIdx.x < len - nvec * T::kVec) {
            const size_t i = nvec * T::kVec + threadIdx.x;
            if constexpr (COPY) {
                copy_elem<T>(a.in[q], a.out[q], i);
            } else {
                KernargSrc<2> src;
                src.p[0] = a.in[q];
                src.p[1] = a.own[q];
                reduce_elem<T, Op>(src, 2, a.out[q], i);
            }
        }
    }
}

// Element-aligned buffers: one element per thread, tiles of kB elements.
template <class T, class Op, bool COPY>
__global__ __launch_bounds__(kB) void sim_step_scalar_kernel(SimStep a, int G, uint64_t tiles)
{
    const uint64_t work = tiles * (uint64_t)G;
    for (uint64_t w = blockIdx.x; w < work; w += gridDim.x) {
        const int q = (int)(w % (uint64_t)G);
        const size_t i = (size_t)(w / (uint64_t)G) * kB + threadIdx.x;
        if (i >= a.len[q]) continue;
        if constexpr (COPY) {
            copy_elem<T>(a.in[q], a.out[q], i);
        } else {
            KernargSrc<2> src;
            src.p[0] = a.in[q];
            src.p[1] = a.own[q];
            reduce_elem<T, Op>(src, 2, a.out[q], i);
        }
    }
}

template <class T, class Op, bool COPY>
hipError_t launch_sim_step(const SimStep &a, int G, bool vec, hipStream_t s)
{
    uint64_t maxlen = 0;
    for (int q = 0; q < G; ++q) maxlen = a.len[q] > maxlen ? a.len[q] : maxlen;
    if (maxlen == 0) return hipSuccess;
    uint64_t tiles;
    if (vec) {
        constexpr uint64_t kTileElems = (uint64_t)kB * kU * T::kVec;
        tiles = (maxlen / T::kVec * T::kVec + kTileElems - 1) / kTileElems + 1;   // + tail tile
        return launch_kernel(sim_step_vec_kernel<T, Op, COPY>, dim3(grid_for(tiles * G)),
                             dim3(kB), 0, s, a, G, tiles);
    }
    tiles = (maxlen + kB - 1) / kB;
    return launch_kernel(sim_step_scalar_kernel<T, Op, COPY>, dim3(grid_for(tiles * G)), dim3(kB),
                         0, s, a, G, tiles);
}

// ------------------------------------------------------------ one launch --
// Every step in one launch.  Whatever the schedule, the bits every recv
// buffer ends with at element i of chunk (block) c are one fold of the G
// ranks' send values at i, in an order the schedule fixes, with the partial
// rounded to the I/O type at every hop; every message stored during the
// ReduceScatter phase is overwritten during the AllGather phase.  So one
// thread folds element vector v of chunk c in that order, hands each message
// to the next hop in registers (rounded exactly as when it is sent), and
// stores only the final bits, once per rank: the intermediate forwarding
// stores that ReduceCopy avoids (Section 5) are not made at all, and the call
// moves 2 G N elements instead of the per-step schedule's 5 (G-1) N.
//
// Leaf k = 0..G-1 of chunk c is the send buffer of rank
//   ring  (c+1+k) mod G, folded left to right: m = hop(m, leaf k), the
//         message first and the receiving rank's own value second;
//   RHD   c ^ bitrev(k), over log2 G bits.  The halving step at distance d
//         makes, on rank c ^ y (y < d), hop(partial of rank c^(y+d), own
//         partial): a pairwise tree over the leaves in bit-reversed order,
//         the later subtree received, the earlier one own.  A binary counter
//         evaluates it with one pending partial per tree level.
// Leaves are loaded 8 at a time, all before the first store, so recv[r] may
// be send[r].
struct SimAll {
    const char *send[XRED_MAX_SRC];
    char *recv[XRED_MAX_SRC];
};

constexpr int kLeafBatch = 8;
constexpr int kMaxLevels = 7;   // log2(XRED_MAX_SRC) + 1

template <class T>
__device__ __forceinline__ uint64_t load_bits(const char *base, size_t i)
{
    if constexpr (T::kSize == 1) return ((const uint8_t *)base)[i];
    else if constexpr (T::kSize == 2) return ((const uint16_t *)base)[i];
    else if constexpr (T::kSize == 4) return ((const uint32_t *)base)[i];
    else return ((const uint64_t *)base)[i];
}

template <class T>
__device__ __forceinline__ void store_bits(char *base, size_t i, uint64_t v)
{
    if constexpr (T::kSize == 1) ((uint8_t *)base)[i] = (uint8_t)v;
    else if constexpr (T::kSize == 2) ((uint16_t *)base)[i] = (uint16_t)v;
    else if constexpr (T::kSize == 4) ((uint32_t *)base)[i] = (uint32_t)v;
    else ((uint64_t *)base)[i] = v;
}

// One lane's share of a work item: a 16-byte vector (VEC) or one element.
template <class T, bool VEC>
struct Lane;

template <class T>
struct Lane<T, true> {
    using R = u32x4;
    size_t off;      // byte offset of the tile in every buffer
    uint32_t nrec;   // bytes of the tile in range
    __device__ R load(const char *base, bool present) const
    {
        // an absent leaf reads through an empty descriptor: zeros, no access
        return bload<kLoadStream>(make_rsrc(base + off, present ? nrec : 0u), threadIdx.x * 16u);
    }
    __device__ void store(R v, char *base) const
    {
        bstore<kStoreOut>(v, make_rsrc(base + off, nrec), threadIdx.x * 16u);
    }
    template <class Op>
    __device__ static R hop(R in, R own)
    {
        typename T::Acc x[T::kVec];
        up_vec<T>(in, x);
        fold_vec<T, Op>(x, own);
        return down_vec<T, Op>(x);
    }
};

template <class T>
struct Lane<T, false> {
    using R = uint64_t;
    size_t i;        // element index in every buffer
    __device__ R load(const char *base, bool present) const
    {
        return present ? load_bits<T>(base, i) : 0;
    }
    __device__ void store(R v, char *base) const { store_bits<T>(base, i, v); }
    template <class Op>
    __device__ static R hop(R in, R own)
    {
        const typename T::Acc x =
            combine<T, Op>(up1<T>((const char *)&in, 0), up1<T>((const char *)&own, 0));
        R out = 0;
        down1<T, Op>((char *)&out, 0, x);
        return out;
    }
};

template <class T, class Op, bool RHD, class L>
__device__ __forceinline__ void fold_chunk(const SimAll &a, int G, int lg, int c, const L &lane)
{
    using R = typename L::R;
    R m{};
    R pending[kMaxLevels];
    for (int k0 = 0; k0 < G; k0 += kLeafBatch) {
        R v[kLeafBatch];
#pragma unroll
        for (int u = 0; u < kLeafBatch; ++u) {
            const int k = k0 + u;
            int rank = 0;
            if (k < G)
                rank = RHD ? c ^ (int)(__builtin_bitreverse32((uint32_t)k) >> (32 - lg))
                           : (c + 1 + k) % G;
            v[u] = lane.load(a.send[rank], k < G);
        }
#pragma unroll
        for (int u = 0; u < kLeafBatch; ++u) {
            const int k = k0 + u;
            if (k >= G) break;
            if constexpr (!RHD) {
                m = k == 0 ? v[u] : L::template hop<Op>(m, v[u]);
            } else {
                R x = v[u];
#pragma unroll
                for (int l = 0; l < kMaxLevels; ++l) {
                    if (((k >> l) & 1) == 0) {
                        pending[l] = x;
                        break;
                    }
                    x = L::template hop<Op>(x, pending[l]);
                }
            }
        }
    }
    if constexpr (RHD) {
#pragma unroll
        for (int l = 0; l < kMaxLevels; ++l)
            if (l == lg) m = pending[l];
    }
    for (int r = 0; r < G; ++r) lane.store(m, a.recv[r]);
}

// Work item w: chunk w / tiles, tile w % tiles of it (the last tile of each
// chunk takes the elements after its last full vector): chunk-major, so the
// workgroups in flight read and write one contiguous stretch of every rank's
// buffers (items dealt chunk by chunk in turn spread them over G places in
// each: 8 ranks x 64M bf16, ring, 12 waves per CU, 355 against 374 us).
// VEC: 16-byte aligned buffers; otherwise one element per thread.
template <class T, class Op, bool RHD, bool VEC, int BT>
__global__ __launch_bounds__(BT) void sim_all_kernel(SimAll a, int G, int lg, uint64_t M,
                                                     uint64_t count, uint64_t tiles)
{
    constexpr uint32_t kTileBytes = (uint32_t)BT * 16u;
    const uint64_t work = tiles * (uint64_t)G;
    for (uint64_t w = blockIdx.x; w < work; w += gridDim.x) {
        const int c = (int)(w / tiles);
        const uint64_t t = w % tiles;
        const uint64_t lo = (uint64_t)c * M < count ? (uint64_t)c * M : count;
        const uint64_t hi = (uint64_t)(c + 1) * M < count ? (uint64_t)(c + 1) * M : count;
        const uint64_t len = hi - lo;
        if constexpr (VEC) {
            const uint64_t nvec = len / T::kVec;
            const size_t vbytes = nvec * 16;
            const uint64_t vtiles = (vbytes + kTileBytes - 1) / kTileBytes;
            if (t < vtiles) {
                const size_t toff = t * kTileBytes;
                fold_chunk<T, Op, RHD>(a, G, lg, c,
                                       Lane<T, true>{lo * T::kSize + toff,
                                                     tile_nrec(vbytes, toff, kTileBytes)});
            } else if (t == vtiles && threadIdx.x < len - nvec * T::kVec) {
                fold_chunk<T, Op, RHD>(a, G, lg, c,
                                       Lane<T, false>{lo + nvec * T::kVec + threadIdx.x});
            }
        } else {
            const uint64_t e = t * BT + threadIdx.x;
            if (e < len) fold_chunk<T, Op, RHD>(a, G, lg, c, Lane<T, false>{lo + e});
        }
    }
}

// One launch of sim_all_kernel with BT threads per workgroup, at most
// `waves` resident waves per CU (0: no cap) through an LDS reservation no
// thread touches.
template <class T, class Op, bool RHD, int BT>
hipError_t launch_all_shape(const SimAll &a, int G, int lg, uint64_t M, size_t count, bool vec,
                            int waves, hipStream_t s)
{
    const uint64_t tiles = vec ? (M * T::kSize + BT * 16u - 1) / (BT * 16u) + 1 : (M + BT - 1) / BT;
    const dim3 grid(grid_for(tiles * (uint64_t)G));
    const int wgs = waves / (BT / 64) > 0 ? waves / (BT / 64) : 1;
    const size_t lds = waves > 0 ? (size_t)(lds_per_cu() / wgs) / 512 * 512 : 0;
    if (vec)
        return launch_kernel(sim_all_kernel<T, Op, RHD, true, BT>, grid, dim3(BT), lds, s, a, G,
                             lg, M, (uint64_t)count, tiles);
    return launch_kernel(sim_all_kernel<T, Op, RHD, false, BT>, grid, dim3(BT), lds, s, a, G, lg,
                         M, (uint64_t)count, tiles);
}

template <class T, class Op>
hipError_t launch_all(const char *const *send, char *const *recv, int G, size_t count, bool rhd,
                      bool vec, hipStream_t s)
{
    SimAll a;
    for (int q = 0; q < XRED_MAX_SRC; ++q) {
        a.send[q] = q < G ? send[q] : nullptr;
        a.recv[q] = q < G ? recv[q] : nullptr;
    }
    int lg = 0;
    while ((1 << lg) < G) ++lg;
    const uint64_t M = sim_chunk(count, G);
    const bool large = (uint64_t)count * T::kSize >= kSimLargeBytes;
    if (rhd && large)
        return launch_all_shape<T, Op, true, kRhdShape.threads>(a, G, lg, M, count, vec,
                                                                kRhdShape.waves, s);
    if (rhd)
        return launch_all_shape<T, Op, true, kRhdSmallShape.threads>(a, G, lg, M, count, vec,
                                                                     kRhdSmallShape.waves, s);
    if (large)
        return launch_all_shape<T, Op, false, kRingShape.threads>(a, G, lg, M, count, vec,
                                                                  kRingShape.waves, s);
    return launch_all_shape<T, Op, false, kRingSmallShape.threads>(a, G, lg, M, count, vec,
                                                                   kRingSmallShape.waves, s);
}

int rank_mod(int r, int G) { return ((r % G) + G) % G; }

template <class T, class Op>
hipError_t run(const char *const *send, char *const *recv, int G, size_t count,
               xred_schedule sched, hipStream_t s)
{
    constexpr size_t es = T::kSize;
    const uint64_t M = sim_chunk(count, G);
    uintptr_t bits = 0;
    for (int q = 0; q < G; ++q) bits |= (uintptr_t)send[q] | (uintptr_t)recv[q];
    const bool vec = (bits & 15u) == 0;
    auto el = [&](uint64_t blk) { return blk * M < count ? blk * M : (uint64_t)count; };
    SimStep a;
    hipError_t e = hipSuccess;
    if (G == 1) {
        if (send[0] == recv[0]) return hipSuccess;
        a.in[0] = send[0];
        a.own[0] = nullptr;
        a.out[0] = recv[0];
        a.len[0] = count;
        return launch_sim_step<T, Op, true>(a, 1, vec, s);
    }
    if (sched == XRED_SCHEDULE_RING_ONE_LAUNCH || sched == XRED_SCHEDULE_RHD_ONE_LAUNCH)
        return launch_all<T, Op>(send, recv, G, count, sched == XRED_SCHEDULE_RHD_ONE_LAUNCH, vec,
                                 s);
    if (sched == XRED_SCHEDULE_RING) {
        for (int j = 1; j <= G - 1 && e == hipSuccess; ++j) {
            for (int q = 0; q < G; ++q) {
                const int c = rank_mod(q - 1 - j, G);
                const uint64_t lo = el(c), len = el(c + 1) - lo;
                const int p = rank_mod(q - 1, G);
                a.in[q] = (j == 1 ? send[p] : recv[p]) + lo * es;
                a.own[q] = send[q] + lo * es;
                a.out[q] = recv[q] + lo * es;
                a.len[q] = len;
            }
            e = launch_sim_step<T, Op, false>(a, G, vec, s);
        }
        for (int t = 1; t <= G - 1 && e == hipSuccess; ++t) {
            for (int q = 0; q < G; ++q) {
                const int c = rank_mod(q - t, G);
                const uint64_t lo = el(c), len = el(c + 1) - lo;
                a.in[q] = recv[rank_mod(q - 1, G)] + lo * es;
                a.own[q] = nullptr;
                a.out[q] = recv[q] + lo * es;
                a.len[q] = len;
            }
            e = launch_sim_step<T, Op, true>(a, G, vec, s);
        }
        return e;
    }
    // recursive halving, then recursive doubling
    for (int d = G / 2; d >= 1 && e == hipSuccess; d /= 2) {
        const bool first = d == G / 2;
        for (int q = 0; q < G; ++q) {
            const int p = q ^ d;
            const uint64_t b0 = (uint64_t)(q & ~(d - 1));
            const uint64_t lo = el(b0), len = el(b0 + d) - lo;
            a.in[q] = (first ? send[p] : recv[p]) + lo * es;
            a.own[q] = (first ? send[q] : recv[q]) + lo * es;
            a.out[q] = recv[q] + lo * es;
            a.len[q] = len;
        }
        e = launch_sim_step<T, Op, false>(a, G, vec, s);
    }
    for (int d = 1; d < G && e == hipSuccess; d *= 2) {
        for (int q = 0; q < G; ++q) {
            const int p = q ^ d;
            const uint64_t b0 = (uint64_t)(p & ~(d - 1));
            const uint64_t lo = el(b0), len = el(b0 + d) - lo;
            a.in[q] = recv[p] + lo * es;
            a.own[q] = nullptr;
            a.out[q] = recv[q] + lo * es;
            a.len[q] = len;
        }
        e = launch_sim_step<T, Op, true>(a, G, vec, s);
    }
    return e;
}

}  // namespace

uint64_t sim_chunk(uint64_t count, int nranks)
{
    if (nranks < 1) return 0;
    const uint64_t m = (count + (uint64_t)nranks - 1) / (uint64_t)nranks;
    return (m + 63) / 64 * 64;
}

hipError_t launch_sim(xred_dtype dtype, xred_op op, const char *const *send, char *const *recv,
                      int nranks, size_t count, xred_schedule schedule, hipStream_t stream)
{
    return with_dtype(dtype, [&](auto t) {
        using T = decltype(t);
        return with_op<T, false>(op, [&](auto o) {
            return run<T, decltype(o)>(send, recv, nranks, count, schedule, stream);
        });
    });
}

}  // namespace xred
