// xred_ring.hip -- all steps of a ring's ReduceCopy in one persistent launch.
//
// In the FTAR pipeline (Section 5) the kernel reduces each chunk as soon as
// the network has delivered it, and kernel and host thread hand chunks over
// through producer/consumer flags in host-pinned memory (the host-kernel
// coordinated mode of Section 4).  Here one launch folds nchunks chunks, in
// order, into an accumulator that never leaves the chip: each tile workgroup
// owns up to kMaxTilesPerWg tiles whose binary32 / uint32 accumulators live in
// LDS between rounds, so the only HBM traffic is the chunks read once and the
// result written once (the per-step launches of xred_reduce_copy_step move
// the accumulator to memory and back on every step).
//
// Chunk s is read only after ready[s] has reached `epoch` (serial-number
// comparison, so a producer may run ahead).  Reading host memory is what
// costs: every wave polling pinned host flags from hundreds of workgroups at
// once took 8-15 us per poll on MI355X, against 0.8-1.1 us for one lane
// alone (a flag the host writes reaches such a lane 0.8-0.9 us later).  So a
// flagged launch has one extra workgroup (blockIdx 0) whose first wave alone
// polls the flags, 64 at a time (one lane per flag), and publishes the number
// of consecutive ready chunks in a relay word in device memory; the tile
// workgroups wait on that word (agent-scope loads, served on chip).  Chunks of
// a flagged launch are read with system-coherent loads (sc0 sc1): they are
// issued only after the wave has seen the flag, and are served at the point
// of coherence rather than from a cache that could hold stale lines -- what
// an acquire fence's cache invalidation would otherwise provide, without an
// L2 invalidation per workgroup.
//
// The relay word belongs to a slot bound to the caller's stream (see
// StreamSlot): launches on one stream run in order, so they share it, and each
// launch's values carry its ticket, so a value an earlier launch left is
// never taken for this one's.  Nothing has to be reset or tracked on the GPU.
// Under graph capture (a replay would repeat the captured ticket), on the
// per-thread default stream, or once every slot is bound, there is no relay:
// each tile workgroup polls the flags itself (and the grid is capped at
// kFlagPollers).
//
// Every wait is bounded: after `timeout` device-clock ticks without progress
// the waiting workgroup records 1 in *status (if given) and stops; the poller
// also marks the relay word as failed, which stops the tile workgroups at
// once; dst is then unspecified.
#include <algorithm>

#include "xred_dispatch.hpp"
#include "xred_internal.hpp"
#include "xred_kernels.hpp"

namespace xred {
namespace {

constexpr int kB = 512;
constexpr int kGroup = 8;                // chunks loaded together before folding
constexpr int kMaxTilesPerWg = 4;        // tiles whose accumulators one workgroup holds
constexpr uint64_t kFlagPollers = 128;   // tile workgroups when each polls the flags
constexpr int kMaxDevices = 64;
// Relay value: bits 0-6 chunks known ready (at most 64), bit 7 a failed
// wait, bits 8-31 the low bits of the launch's ticket.
constexpr uint32_t kRelayCount = 0x7Fu;
constexpr uint32_t kRelayFailed = 0x80u;
// Cache policy of the chunk loads of a flagged launch: system-coherent
// (sc0 | sc1) and nontemporal.
constexpr int kLoadCoherent = 1 | 2 | 16;

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

// One flagged launch's relay.  word == NULL: no relay.
struct Relay {
    uint32_t *word;         // the relay value (device memory)
    uint32_t ticket;        // this launch's number on the slot (from 1)
};

__device__ __forceinline__ uint32_t relay_tag(const Relay &r) { return r.ticket << 8; }

// Run of consecutive ready chunks from `base` in a ballot (bit q: chunk base+q).
__device__ __forceinline__ int ready_run(uint64_t got)
{
    return ~got == 0 ? 64 : (int)__builtin_ctzll(~got);
}

__device__ __forceinline__ bool flag_set(const uint32_t *ready, int idx, bool mine, uint32_t epoch)
{
    const uint32_t v =
        __hip_atomic_load(ready + (mine ? idx : 0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    return mine && (int32_t)(v - epoch) >= 0;
}

__device__ __forceinline__ void report_timeout(uint32_t *status)
{
    if (status) __hip_atomic_store(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// The poller (first wave of workgroup 0): publish the ready prefix of the
// flags as it grows, until every chunk is published or a wait times out.
__device__ void poll_and_publish(const uint32_t *ready, uint32_t epoch, int nchunks,
                                 uint64_t timeout, uint32_t *status, const Relay &r)
{
    uint32_t *word = r.word;
    const uint32_t tag = relay_tag(r);
    const int lane = (int)threadIdx.x;
    int published = 0;
    uint64_t t0 = wall_clock64();
    while (published < nchunks) {
        const int idx = published + lane;
        const uint64_t got = __ballot(flag_set(ready, idx, idx < nchunks, epoch));
        const int run = ready_run(got);
        if (run > 0) {
            published += run;
            if (lane == 0)
                __hip_atomic_store(word, tag | (uint32_t)published, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            t0 = wall_clock64();
            continue;
        }
        if (wall_clock64() - t0 > timeout) {
            if (lane == 0) {
                report_timeout(status);
                __hip_atomic_store(word, tag | kRelayFailed | (uint32_t)published,
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            return;
        }
        __builtin_amdgcn_s_sleep(2);
    }
}

// A tile workgroup's wait on the relay (thread 0): chunks ready beyond
// `next`, or -1 after a failure or a timeout.  Values without this launch's
// tag are an earlier launch's.
__device__ int wait_relay(const Relay &r, int next, uint64_t timeout, uint32_t *status)
{
    const uint32_t tag = relay_tag(r);
    const uint64_t t0 = wall_clock64();
    for (;;) {
        const uint32_t v = __hip_atomic_load(r.word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if ((v & ~(kRelayCount | kRelayFailed)) == tag) {
            if (v & kRelayFailed) return -1;
            if ((int)(v & kRelayCount) > next) return (int)(v & kRelayCount);
        }
        if (wall_clock64() - t0 > timeout) {
            report_timeout(status);
            return -1;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// A tile workgroup polling the flags itself (first wave, all lanes): chunks
// ready from `next` on, or -1 after a timeout.
__device__ int poll_own(const uint32_t *ready, uint32_t epoch, int next, int nchunks,
                        uint64_t timeout, uint32_t *status)
{
    const int idx = next + (int)threadIdx.x;
    const uint64_t t0 = wall_clock64();
    for (;;) {
        const uint64_t got = __ballot(flag_set(ready, idx, idx < nchunks, epoch));
        if (got & 1u) return next + ready_run(got);
        if (wall_clock64() - t0 > timeout) {
            if (threadIdx.x == 0) report_timeout(status);
            return -1;
        }
        __builtin_amdgcn_s_sleep(2);
    }
}

// Chunks [next, upto) of tile j (byte offset off, nrec bytes exist), in groups
// of kGroup loaded before folding; the accumulator comes from the first chunk
// or LDS and goes to dst (last round) or LDS.  SPLIT: dst + off sits c bytes
// past a 16-byte boundary (0 < c < 16) and the results are stored realigned.
template <class T, class Op, int POL, bool SPLIT>
__device__ __forceinline__ void fold_round(const KernargSrc<XRED_MAX_SRC> &chunks, int nchunks,
                                           char *dst, u32x4 *s_acc, int j, size_t off,
                                           uint32_t nrec, int next, int upto, uint32_t c)
{
    constexpr int H = acc_vecs<T>();
    constexpr int PV = acc_per_vec<T>();
    typename T::Acc a[T::kVec];
    if (next > 0) {
#pragma unroll
        for (int h = 0; h < H; ++h) unpack_acc<T>(*acc_slot<T>(s_acc, j, h), &a[PV * h]);
    }
    for (int g0 = next; g0 < upto; g0 += kGroup) {
        u32x4 in[kGroup];
#pragma unroll
        for (int q = 0; q < kGroup; ++q) {
            const bool on = g0 + q < upto;
            in[q] = __builtin_amdgcn_raw_buffer_load_b128(
                make_rsrc((on ? chunks.p[g0 + q] : dst) + off, on ? nrec : 0u),
                (uint32_t)threadIdx.x * 16u, 0, POL);
        }
        if (g0 == 0) up_vec<T>(in[0], a);
#pragma unroll
        for (int q = 0; q < kGroup; ++q) {
            const bool on = g0 + q < upto && g0 + q > 0;
            typename T::Acc b[T::kVec];
            up_vec<T>(in[q], b);
#pragma unroll
            for (int e = 0; e < T::kVec; ++e) {
                const typename T::Acc c = combine<T, Op>(a[e], b[e]);
                a[e] = on ? c : a[e];
            }
        }
    }
    if (upto == nchunks) {
        if constexpr (SPLIT)
            split_store(down_vec<T, Op>(a), dst + off, nrec, c);
        else
            bstore<kStoreOut>(down_vec<T, Op>(a), make_rsrc(dst + off, nrec),
                              (uint32_t)threadIdx.x * 16u);
    } else {
#pragma unroll
        for (int h = 0; h < H; ++h) *acc_slot<T>(s_acc, j, h) = pack_acc<T>(&a[PV * h]);
    }
}

// Chunks at one offset within 16 bytes: the first `lead` elements (fewer
// than a vector) bring them to a 16-byte boundary and are folded one by one
// with the `tail` after the last full vector; SPLIT: dst sits c bytes off
// that grid (a separate instantiation, so the aligned kernel carries none of
// the realignment).
template <class T, class Op, bool SPLIT>
__global__ __launch_bounds__(kB) void ring_kernel(KernargSrc<XRED_MAX_SRC> chunks, int nchunks,
                                                  char *dst, size_t nvec, uint32_t tail,
                                                  uint32_t lead, uint32_t c,
                                                  int tiles_per_wg, const uint32_t *ready,
                                                  uint32_t epoch, uint64_t timeout,
                                                  uint32_t *status, Relay relay)
{
    extern __shared__ u32x4 s_acc[];
    __shared__ int s_upto;
    constexpr uint32_t kTileBytes = (uint32_t)kB * 16u;
    const bool flagged = ready != nullptr;
    const bool relayed = flagged && relay.word != nullptr;
    if (relayed && blockIdx.x == 0) {
        // the poller: one wave; the others end at once
        if (threadIdx.x < 64) poll_and_publish(ready, epoch, nchunks, timeout, status, relay);
        return;
    }
    const size_t wg = blockIdx.x - (relayed ? 1u : 0u);
    const size_t nwg = gridDim.x - (relayed ? 1u : 0u);
    const size_t vbytes = nvec * 16;
    const size_t lb = (size_t)lead * T::kSize;
    const size_t ntiles = (nvec + kB - 1) / kB;
    int next = 0;
    while (next < nchunks) {
        if (relayed) {
            if (threadIdx.x == 0) s_upto = wait_relay(relay, next, timeout, status);
        } else if (flagged) {
            if (threadIdx.x < 64) {
                const int upto = poll_own(ready, epoch, next, nchunks, timeout, status);
                if (threadIdx.x == 0) s_upto = upto;
            }
        } else if (threadIdx.x == 0) {
            s_upto = nchunks;
        }
        __syncthreads();
        const int upto = s_upto;
        if (upto < 0) break;   // failed or timed out: the whole workgroup stops
        for (int j = 0; j < tiles_per_wg; ++j) {
            const size_t t = wg + (size_t)j * nwg;
            if (t >= ntiles) break;
            const size_t toff = t * kTileBytes;
            const uint32_t nrec = tile_nrec(vbytes, toff, kTileBytes);
            if (flagged)
                fold_round<T, Op, kLoadCoherent, SPLIT>(chunks, nchunks, dst, s_acc, j,
                                                        lb + toff, nrec, next, upto, c);
            else
                fold_round<T, Op, kLoadStream, SPLIT>(chunks, nchunks, dst, s_acc, j, lb + toff,
                                                      nrec, next, upto, c);
        }
        next = upto;
        __syncthreads();   // s_upto is rewritten by the next round
    }
    // Elements before the first and after the last full vector: one
    // workgroup, once every chunk was seen ready (its plain loads need the
    // acquire the vector loads avoid).
    if (next == nchunks && (tail | lead) != 0 && wg == ntiles % nwg &&
        threadIdx.x < tail + lead) {
        if (flagged) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
        reduce_ends<T, Op>(chunks, nchunks, dst, lead, tail, lead + nvec * T::kVec);
    }
}

// Resident workgroups per CU of both ring_kernel<T, Op, *> variants with
// the LDS of kMaxTilesPerWg tiles (cached per device: the host path stays
// free of runtime queries after the first launch).
template <class T, class Op>
int ring_per_cu()
{
    static int cache[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) dev = 0;
    int v = __atomic_load_n(&cache[dev], __ATOMIC_RELAXED);
    if (v <= 0) {
        const size_t lds = lds_tile_bytes<T>() * kMaxTilesPerWg;
        int w = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &v, (const void *)ring_kernel<T, Op, false>, kB, lds) != hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &w, (const void *)ring_kernel<T, Op, true>, kB, lds) != hipSuccess)
            v = 1;
        v = std::max(1, std::min(v, w));
        __atomic_store_n(&cache[dev], v, __ATOMIC_RELAXED);
    }
    return v;
}

// Workgroups that fit on the chip at once for every operator of T.
template <class T>
uint64_t ring_fit()
{
    int v = ring_per_cu<T, OpSum>();
    v = std::min(v, ring_per_cu<T, OpProd>());
    v = std::min(v, ring_per_cu<T, OpMax>());
    v = std::min(v, ring_per_cu<T, OpMin>());
    return (uint64_t)device_cus() * (uint64_t)v;
}

template <class T, class Op>
hipError_t go(const char *const *chunks, int nchunks, char *dst, size_t count,
              const uint32_t *ready, uint32_t epoch, uint64_t timeout, uint32_t *status,
              hipStream_t s)
{
    KernargSrc<XRED_MAX_SRC> ks;
    for (int p = 0; p < XRED_MAX_SRC; ++p) ks.p[p] = p < nchunks ? chunks[p] : nullptr;
    // the chunks share one offset m within 16 bytes (checked by the caller)
    const uintptr_t m = (uintptr_t)chunks[0] & 15u;
    const uint32_t lead = (uint32_t)std::min<size_t>(m == 0 ? 0 : (16 - m) / T::kSize, count);
    const size_t nvec = (count - lead) / T::kVec;
    const uint32_t tail = (uint32_t)((count - lead) % T::kVec);
    const uint32_t c = (uint32_t)(((uintptr_t)dst + (size_t)lead * T::kSize) & 15u);
    const size_t ntiles = (nvec + kB - 1) / kB;
    // The relay word of the stream (tickets follow the order of the launches:
    // the slot stays locked until the launch is committed).
    StreamSlot slot;
    const bool relayed = ready != nullptr && slot.acquire(kSlotRing, s);
    // one workgroup per tile while they fit on the chip (a relayed launch
    // keeps one place for its poller); a CU budget shrinks the grid down to
    // what kMaxTilesPerWg tiles per workgroup allow
    const uint64_t fit = std::max<uint64_t>(ring_fit<T>(), 2) - 1;
    const uint64_t least = (ntiles + kMaxTilesPerWg - 1) / kMaxTilesPerWg;
    uint64_t grid = ntiles < fit ? ntiles : fit;
    grid = relayed ? grid_for(grid + 1) - 1 : grid_for(grid);   // the budget counts the poller
    // Without a relay every tile workgroup polls the flags: host-memory polls
    // from hundreds of workgroups cost more than the bandwidth they add.
    if (ready != nullptr && !relayed && grid > kFlagPollers) grid = kFlagPollers;
    if (grid < least) grid = least;
    if (grid == 0) grid = 1;
    const int tpw = (int)((ntiles + grid - 1) / grid);
    if (tpw > kMaxTilesPerWg) return hipErrorInvalidValue;   // the caller checks ring_max_count
    // tickets run 1 .. 2^24-1 (the tag's width), so no tag is 0, the value
    // of a fresh slot
    const Relay relay = relayed ? Relay{slot.words, (uint32_t)(slot.launches % 0xFFFFFFu) + 1}
                                : Relay{nullptr, 0};
    const dim3 g((unsigned)(grid + (relayed ? 1 : 0)));
    const size_t lds = lds_tile_bytes<T>() * (tpw > 0 ? tpw : 1);
    const hipError_t e =
        c == 0 ? launch_kernel(ring_kernel<T, Op, false>, g, dim3(kB), lds, s, ks, nchunks, dst,
                               nvec, tail, lead, c, tpw, ready, epoch, timeout, status, relay)
               : launch_kernel(ring_kernel<T, Op, true>, g, dim3(kB), lds, s, ks, nchunks, dst,
                               nvec, tail, lead, c, tpw, ready, epoch, timeout, status, relay);
    if (relayed && e == hipSuccess) slot.commit();
    return e;
}

template <class T>
uint64_t max_count()
{
    // the tile workgroups never exceed what fits on the chip beside a poller;
    // each holds at most kMaxTilesPerWg tiles
    return (std::max<uint64_t>(ring_fit<T>(), 2) - 1) * kMaxTilesPerWg * kB * T::kVec;
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
