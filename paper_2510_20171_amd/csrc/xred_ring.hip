// xred_ring.hip -- all steps of a ring's ReduceCopy in one persistent launch.
//
// In the FTAR pipeline (Section 5) the kernel reduces each chunk as soon as
// the network has delivered it, and kernel and host thread hand chunks over
// through producer/consumer flags in host-pinned memory (the host-kernel
// coordinated mode of Section 4).  Here one launch folds nchunks chunks, in
// order, into an accumulator that never leaves the chip: each workgroup owns
// up to kMaxTilesPerWg tiles whose binary32 / uint32 accumulators live in
// LDS between steps, so the only HBM traffic is the chunks read once and the
// result written once (the per-step launches of xred_reduce_copy_step move
// the accumulator to memory and back on every step).
//
// Chunk s is read only after ready[s] has reached `epoch` (serial-number
// comparison, so a producer may run ahead).  The first wave of each
// workgroup polls the next kDepth flags at once, one lane per flag, with
// relaxed system-scope loads; once chunk `next` is ready, the run of
// consecutive ready chunks after it is folded in one round, after a single
// acquire fence (an acquire per poll would invalidate L2 on every poll).
// Every wait is bounded: after `timeout` device-clock ticks the workgroup
// records 1 in *status (if given) and stops; dst is then unspecified.
#include "xred_dispatch.hpp"
#include "xred_internal.hpp"
#include "xred_kernels.hpp"

namespace xred {
namespace {

constexpr int kB = 512;
constexpr int kDepth = 8;            // chunks in flight per round
constexpr int kMaxTilesPerWg = 4;    // tiles whose accumulators one workgroup holds
constexpr uint64_t kFlagPollers = 128;   // workgroups of a launch with ready flags
// LDS bytes of one tile's accumulators for element type T.
template <class T>
constexpr size_t lds_tile_bytes() { return (size_t)kB * acc_vecs<T>() * 16; }

// Accumulator slot of thread `tid`, tile j, 16-byte accumulator vector h:
// [j][h][tid], so consecutive lanes touch consecutive LDS addresses.
template <class T>
__device__ __forceinline__ u32x4 *acc_slot(u32x4 *s_acc, int j, int h)
{
    return s_acc + ((size_t)j * acc_vecs<T>() + h) * kB + threadIdx.x;
}

template <class T, class Op>
__global__ __launch_bounds__(kB) void ring_kernel(KernargSrc<XRED_MAX_SRC> chunks, int nchunks,
                                                  char *dst, size_t nvec, uint32_t tail,
                                                  int tiles_per_wg, const uint32_t *ready,
                                                  uint32_t epoch, uint64_t timeout,
                                                  uint32_t *status)
{
    extern __shared__ u32x4 s_acc[];
    __shared__ int s_upto;
    constexpr uint32_t kTileBytes = (uint32_t)kB * 16u;
    constexpr int H = acc_vecs<T>();
    constexpr int PV = acc_per_vec<T>();
    const size_t vbytes = nvec * 16;
    const size_t ntiles = (nvec + kB - 1) / kB;
    int next = 0;
    while (next < nchunks) {
        if (threadIdx.x < 64) {
            // Wave 0 polls: lane q watches chunk next+q (q < kDepth) with
            // relaxed system-scope loads (no cache invalidation per poll);
            // a ballot gives the run of consecutive ready chunks from `next`.
            const int last = next + kDepth < nchunks ? next + kDepth : nchunks;
            int upto = last;
            if (ready != nullptr) {
                const int idx = next + (int)threadIdx.x;
                const bool mine = idx < last;
                const uint64_t t0 = wall_clock64();
                uint64_t got = 0;
                for (;;) {
                    const bool r = mine && (int32_t)(__hip_atomic_load(ready + (mine ? idx : 0),
                                                                       __ATOMIC_RELAXED,
                                                                       __HIP_MEMORY_SCOPE_SYSTEM) -
                                                     epoch) >= 0;
                    got = __ballot(r);
                    if (got & 1u) break;
                    if (wall_clock64() - t0 > timeout) break;
                    __builtin_amdgcn_s_sleep(2);
                }
                if (got & 1u) {
                    // acquire once for the whole run: data written before the
                    // flags is visible to the loads that follow
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
                    upto = next + (int)__builtin_ctzll(~got);
                } else {
                    if (threadIdx.x == 0 && status)
                        __hip_atomic_store(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
                    upto = -1;
                }
            }
            if (threadIdx.x == 0) s_upto = upto;
        }
        __syncthreads();
        const int upto = s_upto;
        if (upto < 0) return;   // timed out: the whole workgroup stops
        for (int j = 0; j < tiles_per_wg; ++j) {
            const size_t t = blockIdx.x + (size_t)j * gridDim.x;
            if (t >= ntiles) break;
            const size_t off = t * kTileBytes;
            const uint32_t nrec = tile_nrec(vbytes, off, kTileBytes);
            u32x4 in[kDepth];
#pragma unroll
            for (int q = 0; q < kDepth; ++q) {
                const bool on = next + q < upto;
                in[q] = bload<kLoadStream>(
                    make_rsrc((on ? chunks.p[next + q] : dst) + off, on ? nrec : 0u),
                    (uint32_t)threadIdx.x * 16u);
            }
            typename T::Acc a[T::kVec];
            if (next == 0) {
                up_vec<T>(in[0], a);
            } else {
#pragma unroll
                for (int h = 0; h < H; ++h) unpack_acc<T>(*acc_slot<T>(s_acc, j, h), &a[PV * h]);
            }
#pragma unroll
            for (int q = 0; q < kDepth; ++q) {
                const bool on = next + q < upto && !(next == 0 && q == 0);
                typename T::Acc b[T::kVec];
                up_vec<T>(in[q], b);
#pragma unroll
                for (int e = 0; e < T::kVec; ++e) {
                    const typename T::Acc c = combine<T, Op>(a[e], b[e]);
                    a[e] = on ? c : a[e];
                }
            }
            if (upto == nchunks) {
                bstore<kStoreOut>(down_vec<T, Op>(a), make_rsrc(dst + off, nrec),
                                  (uint32_t)threadIdx.x * 16u);
            } else {
#pragma unroll
                for (int h = 0; h < H; ++h) *acc_slot<T>(s_acc, j, h) = pack_acc<T>(&a[PV * h]);
            }
        }
        next = upto;
        __syncthreads();   // s_upto is rewritten by the next round
    }
    // Elements after the last full vector: one workgroup, after all chunks
    // were seen ready.
    if (tail != 0 && blockIdx.x == ntiles % gridDim.x && threadIdx.x < tail)
        reduce_elem<T, Op>(chunks, nchunks, dst, nvec * T::kVec + threadIdx.x);
}

template <class T, class Op>
hipError_t go(const char *const *chunks, int nchunks, char *dst, size_t count,
              const uint32_t *ready, uint32_t epoch, uint64_t timeout, uint32_t *status,
              hipStream_t s)
{
    KernargSrc<XRED_MAX_SRC> ks;
    for (int p = 0; p < XRED_MAX_SRC; ++p) ks.p[p] = p < nchunks ? chunks[p] : nullptr;
    const size_t nvec = count / T::kVec;
    const uint32_t tail = (uint32_t)(count % T::kVec);
    const size_t ntiles = (nvec + kB - 1) / kB;
    const size_t lds_tile = lds_tile_bytes<T>();
    int per_cu = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &per_cu, (const void *)ring_kernel<T, Op>, kB, lds_tile * kMaxTilesPerWg);
    if (e != hipSuccess) return e;
    const uint64_t fit = (uint64_t)device_cus() * (uint64_t)(per_cu > 0 ? per_cu : 1);
    uint64_t grid = ntiles < fit ? ntiles : fit;
    // a CU budget shrinks the grid down to what kMaxTilesPerWg tiles per
    // workgroup allow (fewer workgroups also mean fewer pollers of the flags)
    const uint64_t least = (ntiles + kMaxTilesPerWg - 1) / kMaxTilesPerWg;
    grid = grid_for(grid);
    // With flags every workgroup polls them; host-memory polls from hundreds of
    // workgroups cost more than the bandwidth the extra workgroups add
    // (16 x 2^20 bf16 chunks, flags preset: 31.8 us with 256 workgroups, 19.4
    // us with 128, 5.4 us without flags), so flagged launches use at most
    // kFlagPollers workgroups.
    if (ready != nullptr && grid > kFlagPollers) grid = kFlagPollers;
    if (grid < least) grid = least;
    if (grid == 0) grid = 1;
    const int tpw = (int)((ntiles + grid - 1) / grid);
    if (tpw > kMaxTilesPerWg) return hipErrorInvalidValue;   // the caller checks ring_max_count
    hipLaunchKernelGGL((ring_kernel<T, Op>), dim3((unsigned)grid), dim3(kB),
                       lds_tile * (tpw > 0 ? tpw : 1), s, ks, nchunks, dst, nvec, tail, tpw,
                       ready, epoch, timeout, status);
    return hipGetLastError();
}

template <class T>
uint64_t max_count()
{
    // the grid never exceeds what fits on the chip; each workgroup holds at
    // most kMaxTilesPerWg tiles
    int per_cu = 0;
    (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &per_cu, (const void *)ring_kernel<T, OpSum>, kB, lds_tile_bytes<T>() * kMaxTilesPerWg);
    if (per_cu <= 0) per_cu = 1;
    return (uint64_t)device_cus() * per_cu * kMaxTilesPerWg * kB * T::kVec;
}

}  // namespace

uint64_t ring_max_count(xred_dtype dtype)
{
    uint64_t n = 0;
    (void)with_dtype(dtype, [&](auto t) {
        n = max_count<decltype(t)>();
        return hipSuccess;
    });
    return n;
}

hipError_t launch_ring(xred_dtype dtype, xred_op op, const char *const *chunks, int nchunks,
                       char *dst, size_t count, const uint32_t *ready, uint32_t epoch,
                       uint64_t timeout_ticks, uint32_t *status, hipStream_t stream)
{
    return with_dtype(dtype, [&](auto t) {
        using T = decltype(t);
        return with_op<T, false>(op, [&](auto o) {
            return go<T, decltype(o)>(chunks, nchunks, dst, count, ready, epoch, timeout_ticks,
                                      status, stream);
        });
    });
}

}  // namespace xred
