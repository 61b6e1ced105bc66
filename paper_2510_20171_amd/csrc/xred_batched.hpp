// xred_batched.hpp -- many independent reductions in one launch: kernels and
// launch templates, instantiated per group of element types by
// xred_batched_{float,fp8,int}.hip so the groups compile in parallel.
//
// Small messages are dominated by per-call overhead (the T_c term of the
// LogP model in Section 6.2), so a batch of K reductions is run as one
// kernel.  Work is cut into tiles of 16-byte vectors of one item, in the
// global order item 0's tiles, then item 1's, ...  Four kernels:
//   table        (host descriptors, the usual case): the host stages the
//                item of every tile and one workgroup runs each tile, so the
//                hardware dispatches tiles in order, as for the fused kernel;
//   grouped      (device descriptors, more than one run of items): runs of
//                consecutive items, each dealt tile by tile to its own set of
//                workgroups, which plan their tiles from the descriptors in the
//                kernel (metadata by reference, Section 6.1); the sets are
//                dispatched in order, so the runs balance over the chip;
//   round-robin  (device descriptors of one run, or host batches past the
//                table's size): a persistent grid, tile g on workgroup g mod G,
//                the tile-start prefix in LDS (staged, or scanned from the
//                descriptors in the kernel);
//   range        (host batches past the round-robin plan's items): contiguous
//                tile ranges per workgroup, planned on the host.
// Device-descriptor kernels keep no state between calls, so they can be
// captured in a graph.

#pragma once

#include "xred_dispatch.hpp"
#include "xred_internal.hpp"
#include "xred_kernels.hpp"

namespace xred {
namespace {

constexpr int kU = 1;     // vectors per thread in one pass over a sub-tile
constexpr int kB = 512;
// Sub-tiles of kB*kU vectors per tile: two halve the per-tile descriptor
// work (measured +5-6 % on batches of large or equal items, neutral on the
// log-uniform 4096-item batch); four were no better.
constexpr int kSub = 2;

template <class T>
constexpr uint64_t tile_vecs() { return (uint64_t)kB * kU * kSub; }
template <class T>
constexpr uint64_t tile_elems() { return tile_vecs<T>() * T::kVec; }
constexpr uint32_t kTileBytes = (uint32_t)kB * kU * kSub * 16u;
constexpr uint32_t kSubBytes = (uint32_t)kB * kU * 16u;

__device__ __forceinline__ bool item_runnable(const xred_item &it)
{
    return it.nsrc >= 1 && it.nsrc <= XRED_MAX_SRC && it.reserved == 0 && it.srcs != nullptr &&
           it.dst != nullptr;
}

template <class T, bool CHECK>
__device__ __forceinline__ uint64_t item_tiles(const xred_item &it)
{
    if (CHECK && !item_runnable(it)) return 0;
    return (it.count + tile_elems<T>() - 1) / tile_elems<T>();
}

// Descriptor of item k, loaded field by field with scalar loads.
__device__ __forceinline__ xred_item load_item(const xred_item *items, uint64_t k)
{
    const xred_item *p = items + k;
    xred_item it;
    it.srcs = sload(&p->srcs);
    it.dst = sload(&p->dst);
    it.count = sload(&p->count);
    it.nsrc = sload(&p->nsrc);
    it.reserved = sload(&p->reserved);
    return it;
}

__device__ __forceinline__ uint64_t uniform64(uint64_t x)
{
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// Inclusive prefix sum over the workgroup; s[kB-1] holds the total until the
// next call.
__device__ uint64_t block_inclusive_scan(uint64_t v, uint64_t *s)
{
    __syncthreads();
    s[threadIdx.x] = v;
    __syncthreads();
    for (int off = 1; off < kB; off <<= 1) {
        const uint64_t t = threadIdx.x >= (unsigned)off ? s[threadIdx.x - off] : 0;
        __syncthreads();
        s[threadIdx.x] += t;
        __syncthreads();
    }
    return s[threadIdx.x];
}

// Exclusive prefix sum over the workgroup (kB threads); *total gets the sum.
__device__ __forceinline__ uint64_t block_exclusive_scan(uint64_t v, uint64_t *s_wave,
                                                         uint64_t *total)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint64_t incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint64_t t = __shfl_up(incl, (unsigned)off, 64);
        if (lane >= off) incl += t;
    }
    if (lane == 63) s_wave[wave] = incl;
    __syncthreads();
    uint64_t before = 0, sum = 0;
#pragma unroll
    for (int w = 0; w < kB / 64; ++w) {
        const uint64_t x = s_wave[w];
        before += w < wave ? x : 0;
        sum += x;
    }
    *total = sum;
    return before + incl - v;
}

// An item's buffers take the vector path when every pointer sits at the same
// offset m within 16 bytes (diff: the bits in which some source's address
// differs from dst's) and m is a whole number of elements: the first
// (16 - m) / size elements, fewer than a vector, are folded one by one and
// the rest is 16-byte aligned.  Returns that element count (at most count),
// or kNoVector.
constexpr uint64_t kNoVector = ~0ull;
template <class T>
__device__ __forceinline__ uint64_t item_lead(uintptr_t diff, uintptr_t dst, uint64_t count)
{
    const uintptr_t m = dst & 15u;
    if ((diff & 15u) != 0 || m % T::kSize != 0) return kNoVector;
    const uint64_t lead = m == 0 ? 0 : (16 - m) / T::kSize;
    return lead < count ? lead : count;
}

// When item_lead finds no vector path but every source sits at one offset m
// within 16 bytes (sdiff: the bits in which some source's address differs
// from the first one's, s0) and m is a whole number of elements, the sources
// still read in vectors after the first (16 - m) / size elements and the
// output is realigned (split_tile).  Returns that element count, or kNoVector
// (sources at different offsets, or an item no longer than the lead).
template <class T>
__device__ __forceinline__ uint64_t sources_lead(uintptr_t sdiff, uintptr_t s0, uint64_t count)
{
    const uintptr_t m = s0 & 15u;
    if ((sdiff & 15u) != 0 || m % T::kSize != 0) return kNoVector;
    const uint64_t lead = m == 0 ? 0 : (16 - m) / T::kSize;
    return lead < count ? lead : kNoVector;
}

// Tile lt (of SUB sub-tiles of kB*kU vectors) of one item.
template <class T, class Op, int SUB = kSub>
__device__ void batched_tile(const xred_item &it, uint64_t lt)
{
    constexpr uint32_t kTileBytes = (uint32_t)kB * kU * SUB * 16u;
    constexpr uint64_t kTileElems = (uint64_t)kB * kU * SUB * T::kVec;
    const char *const *sp = (const char *const *)it.srcs;
    const int nsrc = (int)it.nsrc;
    uintptr_t diff = 0;   // bits in which some source's address differs from dst's
    uintptr_t sdiff = 0;  // ... from the first source's
    const uintptr_t s0 = (uintptr_t)sload(sp);
    bool null_src = false;
    for (int p = 0; p < nsrc; ++p) {
        const uintptr_t q = (uintptr_t)sload(sp + p);
        diff |= q ^ (uintptr_t)it.dst;
        sdiff |= q ^ s0;
        null_src |= q == 0;
    }
    if (null_src) return;
    char *dst = (char *)it.dst;
    const GlobalSrc src{sp};
    const uint64_t count = it.count;
    uint64_t lead = item_lead<T>(diff, (uintptr_t)dst, count);
    // the output at another offset than the sources: realigned stores (c > 0)
    uint32_t c = 0;
    if (lead == kNoVector) {
        lead = sources_lead<T>(sdiff, s0, count);
        if (lead != kNoVector) c = (uint32_t)(((uintptr_t)dst + lead * T::kSize) & 15u);
        if (c == 0) lead = kNoVector;
    }
    if (lead != kNoVector) {
        const size_t lb = (size_t)lead * T::kSize;   // bytes before the first vector
        const size_t nvec = (count - lead) / T::kVec;
        const size_t vbytes = nvec * 16;
        for (int h = 0; h < SUB; ++h) {
            const size_t off = lt * kTileBytes + (size_t)h * kSubBytes;
            if (off >= vbytes) break;
            const Tile tl{lb + off, tile_nrec(vbytes, off, kSubBytes)};
            if (c != 0) {
                split_tile<T, Op, 1, kB>(src, nsrc, dst, tl, c);
                continue;
            }
            switch (nsrc) {
            case 1: reduce_tile<T, Op, 1, kU, kB>(src, nsrc, dst, tl); break;
            case 2: reduce_tile<T, Op, 2, kU, kB>(src, nsrc, dst, tl); break;
            case 3: reduce_tile<T, Op, 3, kU, kB>(src, nsrc, dst, tl); break;
            case 4: reduce_tile<T, Op, 4, kU, kB>(src, nsrc, dst, tl); break;
            case 5: reduce_tile<T, Op, 5, kU, kB>(src, nsrc, dst, tl); break;
            case 6: reduce_tile<T, Op, 6, kU, kB>(src, nsrc, dst, tl); break;
            case 7: reduce_tile<T, Op, 7, kU, kB>(src, nsrc, dst, tl); break;
            case 8: reduce_tile<T, Op, 8, kU, kB>(src, nsrc, dst, tl); break;
            // more than 8 sources: the compact group loop (the pipelined
            // 16/32/64 bodies would raise every batched kernel's register
            // count and cut its occupancy)
            default: reduce_tile<T, Op, 0, kU, kB>(src, nsrc, dst, tl); break;
            }
        }
        // the item's first tile also takes the elements before its first
        // vector, its last tile those after its last full vector
        reduce_ends<T, Op>(src, nsrc, dst, lt == 0 ? (uint32_t)lead : 0u,
                           (lt + 1) * kTileElems >= count ? (uint32_t)((count - lead) % T::kVec)
                                                          : 0u,
                           lead + nvec * T::kVec);
    } else if (const uint32_t sl = shift_lead<T>((uintptr_t)dst, count * T::kSize)) {
        // sources at different offsets: vectors realigned to dst's grid
        const size_t lb = (size_t)sl * T::kSize;
        const size_t nvec = (count * T::kSize - lb - 16) / 16, vbytes = nvec * 16;
        for (int h = 0; h < SUB; ++h) {
            const size_t off = lt * kTileBytes + (size_t)h * kSubBytes;
            if (off >= vbytes) break;
            shift_tile<T, Op, kB>(src, nsrc, dst, lb, off, tile_nrec(vbytes, off, kSubBytes));
        }
        reduce_ends<T, Op>(src, nsrc, dst, lt == 0 ? sl : 0u,
                           (lt + 1) * kTileElems >= count
                               ? (uint32_t)(count - sl - nvec * T::kVec)
                               : 0u,
                           sl + nvec * T::kVec);
    } else {
        const uint64_t e0 = lt * kTileElems;
        const uint64_t e1 = count < e0 + kTileElems ? count : e0 + kTileElems;
        for (uint64_t i = e0 + threadIdx.x; i < e1; i += kB) reduce_elem<T, Op>(src, nsrc, dst, i);
    }
}

template <class T, class Op>
__global__ __launch_bounds__(kB) void batched_kernel(const xred_item *items, int nitems,
                                                     const WgStart *wg)
{
    const WgStart *w = wg + blockIdx.x;
    uint64_t k = sload(&w->item);
    uint64_t lt = sload(&w->local_tile);
    uint64_t left = sload(&w->ntiles);
    k = uniform64(k);
    lt = uniform64(lt);
    left = uniform64(left);
    while (left > 0 && k < (uint64_t)nitems) {
        k = uniform64(k);
        const xred_item it = load_item(items, k);
        const uint64_t nt = item_tiles<T, false>(it);
        if (lt >= nt) {
            ++k;
            lt = 0;
            continue;
        }
        batched_tile<T, Op>(it, lt);
        ++lt;
        --left;
    }
}

// ------------------------------------------------------ round-robin variant --
// Global tile g is processed by workgroup g mod G (G = the workgroups that fit
// on the chip at once), so the tiles in flight form one moving window over
// the batch, as in the fused kernel, instead of G scattered ranges.  Each
// workgroup keeps the batch's tile-start prefix in LDS (copied from the host
// plan, or computed by a block scan over device-resident descriptors), finds
// the (item, tile) of each of its tiles by binary search in parallel, and
// while one tile's loads are in flight fetches the next tile's descriptor and
// source pointers with scalar loads.
constexpr int kListMax = 1024;     // tiles a workgroup plans per pass
constexpr int kRrMaxItems = 8192;  // items whose prefix fits the LDS budget

struct TileDesc {
    const char *p[8];         // sources 0..7 (valid below nsrc)
    const char *const *srcs;  // the item's source array
    char *dst;
    uint64_t count;
    uint64_t lt;              // tile within the item
    uint32_t k;               // item
    int nsrc;
    uint32_t lead;            // elements before the first vector (0 unless fast)
    uint32_t c;               // > 0: the output sits c bytes off the sources' vector grid
    bool fast;                // nsrc <= 8, no NULL source, the sources at one offset in 16 B
};

template <class T>
__device__ __forceinline__ void fetch_desc(TileDesc &d, const xred_item *items, uint32_t k,
                                           uint64_t lt)
{
    const xred_item *it = items + k;
    d.k = k;
    d.lt = lt;
    d.srcs = (const char *const *)sload(&it->srcs);
    d.dst = (char *)sload(&it->dst);
    d.count = sload(&it->count);
    d.nsrc = (int)sload(&it->nsrc);
    uintptr_t diff = 0, sdiff = 0;
    bool null_src = false;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        d.p[q] = q < d.nsrc ? sload(d.srcs + q) : nullptr;
        diff |= q < d.nsrc ? (uintptr_t)d.p[q] ^ (uintptr_t)d.dst : 0;
        sdiff |= q < d.nsrc ? (uintptr_t)d.p[q] ^ (uintptr_t)d.p[0] : 0;
        null_src |= q < d.nsrc && d.p[q] == nullptr;
    }
    uint64_t lead = item_lead<T>(diff, (uintptr_t)d.dst, d.count);
    d.c = 0;
    if (lead == kNoVector) {
        // the sources at one offset, the output at another: realigned stores
        const uint64_t sl = sources_lead<T>(sdiff, (uintptr_t)d.p[0], d.count);
        const uint32_t c =
            sl != kNoVector ? (uint32_t)(((uintptr_t)d.dst + sl * T::kSize) & 15u) : 0u;
        if (c != 0) {
            lead = sl;
            d.c = c;
        }
    }
    d.fast = d.nsrc <= 8 && !null_src && lead != kNoVector;
    d.lead = d.fast ? (uint32_t)lead : 0u;
}

// Sub-tile h of a straight-line tile whose vectors start at byte `off` of
// d's output (nrec bytes of the tile exist): one aligned vector per thread,
// or realigned stores when the output sits d.c bytes off the sources' grid.
__device__ __forceinline__ void tile_store(u32x4 v, rsrc_t w, const TileDesc &d, size_t off,
                                           uint32_t nrec, int h)
{
    if (d.c == 0) {
        bstore<kStoreOut>(v, w, (uint32_t)(h * kB + threadIdx.x) * 16u);
        return;
    }
    const uint32_t start = (uint32_t)h * kSubBytes;
    if (start >= nrec) return;
    const uint32_t left = nrec - start;
    split_store(v, d.dst + off + start, left < kSubBytes ? left : kSubBytes, d.c);
}

template <class T, class Op, bool PLANNED>
__global__ __launch_bounds__(kB) void batched_rr_kernel(const xred_item *items, int nitems,
                                                        const uint32_t *tile_start)
{
    extern __shared__ uint2 s_dyn[];
    __shared__ uint64_t s_scan[kB];
    uint2 *s_list = s_dyn;                             // kListMax entries
    uint32_t *s_pre = (uint32_t *)(s_dyn + kListMax);  // nitems + 1 entries
    if constexpr (PLANNED) {
        for (int i = threadIdx.x; i <= nitems; i += kB) s_pre[i] = tile_start[i];
    } else {
        uint64_t base = 0;
        for (int w0 = 0; w0 < nitems; w0 += kB) {
            const int i = w0 + (int)threadIdx.x;
            const uint64_t c = i < nitems ? item_tiles<T, true>(items[i]) : 0;
            const uint64_t incl = block_inclusive_scan(c, s_scan);
            if (i < nitems) s_pre[i] = (uint32_t)(base + incl - c);
            base += s_scan[kB - 1];
        }
        if (base >= 0xFFFFFFFFull) return;   // more tiles than the plan can index: run nothing
        if (threadIdx.x == 0) s_pre[nitems] = (uint32_t)base;
    }
    __syncthreads();
    const uint64_t total = s_pre[nitems];
    const uint64_t G = gridDim.x;
    for (uint64_t g0 = blockIdx.x; g0 < total; g0 += (uint64_t)kListMax * G) {
        const uint64_t left = (total - g0 + G - 1) / G;
        const int n = left < (uint64_t)kListMax ? (int)left : kListMax;
        for (int j = threadIdx.x; j < n; j += kB) {
            const uint64_t g = g0 + (uint64_t)j * G;
            int lo = 0, hi = nitems;   // s_pre[lo] <= g < s_pre[hi]
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (s_pre[mid] <= g) lo = mid;
                else hi = mid;
            }
            s_list[j] = uint2{(uint32_t)lo, (uint32_t)(g - s_pre[lo])};
        }
        __syncthreads();
        TileDesc cur, nxt;
        fetch_desc<T>(cur, items, __builtin_amdgcn_readfirstlane(s_list[0].x),
                   __builtin_amdgcn_readfirstlane(s_list[0].y));
        for (int j = 0; j < n; ++j) {
            // Issue the current tile's loads.  Straight-line code: sources
            // beyond nsrc, and tiles not on the fast path, get a zero-length
            // buffer range, so their loads return 0 without touching memory
            // and their store is dropped.
            const size_t lb = (size_t)cur.lead * T::kSize;
            const size_t nvec = (cur.count - cur.lead) / T::kVec;
            const size_t vbytes = nvec * 16, toff = cur.lt * kTileBytes;
            const uint32_t nrec = cur.fast && toff < vbytes ? tile_nrec(vbytes, toff, kTileBytes) : 0u;
            u32x4 in[8][kSub];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const bool on = q < cur.nsrc;
                const rsrc_t r = make_rsrc((on ? cur.p[q] : cur.dst) + lb + toff, on ? nrec : 0u);
#pragma unroll
                for (int h = 0; h < kSub; ++h)
                    in[q][h] = bload<kLoadStream>(r, (uint32_t)(h * kB + threadIdx.x) * 16u);
            }
            // fetch the next tile's descriptor while those loads are in flight
            if (j + 1 < n)
                fetch_desc<T>(nxt, items, __builtin_amdgcn_readfirstlane(s_list[j + 1].x),
                           __builtin_amdgcn_readfirstlane(s_list[j + 1].y));
            // fold (unused sources skipped by a uniform select) and store
            const rsrc_t w = make_rsrc(cur.dst + lb + toff, nrec);
#pragma unroll
            for (int h = 0; h < kSub; ++h) {
                typename T::Acc acc[T::kVec];
                up_vec<T>(in[0][h], acc);
#pragma unroll
                for (int q = 1; q < 8; ++q) {
                    const bool on = q < cur.nsrc;
                    typename T::Acc b[T::kVec];
                    up_vec<T>(in[q][h], b);
#pragma unroll
                    for (int e = 0; e < T::kVec; ++e) {
                        const typename T::Acc c = combine<T, Op>(acc[e], b[e]);
                        acc[e] = on ? c : acc[e];
                    }
                }
                if constexpr (__is_same(Op, OpAvg)) {
#pragma unroll
                    for (int e = 0; e < T::kVec; ++e) acc[e] = avg_scale<T, Op>(acc[e], cur.nsrc);
                }
                tile_store(down_vec<T, Op>(acc), w, cur, lb + toff, nrec, h);
            }
            if (cur.fast) {
                reduce_ends<T, Op>(GlobalSrc{cur.srcs}, cur.nsrc, cur.dst,
                                   cur.lt == 0 ? cur.lead : 0u,
                                   (cur.lt + 1) * tile_elems<T>() >= cur.count
                                       ? (uint32_t)((cur.count - cur.lead) % T::kVec)
                                       : 0u,
                                   cur.lead + nvec * T::kVec);
            } else {
                batched_tile<T, Op>(load_item(items, cur.k), cur.lt);
            }
            cur = nxt;
            // the waves start every tile together (8 items of 32M bf16 per
            // source: 5.18 against 4.99 TB/s; 64 items of 4M: 4.90 against 4.98)
            __syncthreads();
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------ queue variant --
// Device descriptors (the host never sees the sizes): a persistent grid takes
// the batch's tiles in order from a counter in device memory, one tile per
// claim, so the tiles in flight stay one compact window over the batch, as
// when the hardware dispatches one workgroup per tile of a host-built table,
// and no workgroup keeps a fixed share of the batch.  Each workgroup first
// scans the tile counts of all items into an LDS tile-start prefix (its first
// claim in flight meanwhile).  Per tile it claims the next tile and issues
// this tile's loads; while they are in flight, the claim's answer is handed
// to all waves through LDS and every wave finds the next tile's item (a
// 64-ary search of the prefix) and fetches its descriptor and source
// pointers, so the next tile's loads follow this tile's stores at once.
//
// What was measured on the 4096-item log-uniform batch (MI355X, same box):
// one workgroup of 512 threads per CU and tiles of two 512-vector sub-tiles
// (16 KiB per source) 1237-1240 us, against 1267 us with the next tile's
// descriptor fetched after this tile's stores.  With the fetch overlapped:
// 8 KiB tiles 1611 us (one or two workgroups per CU: the one counter then
// answers twice as many claims), 24 KiB 1281 us, 32 KiB 1322 us, two
// workgroups per CU 1393 us; the loads issued sub-tile by sub-tile instead
// of source by source 1248 us; the first sub-tile folded and stored before
// the claim is handed over 1314 us.  Before it: claiming two tiles ahead 1445 us
// and double-buffered loads 1262 us (a tile claimed or loaded ahead widens
// the window of tiles being read, which costs more than the latency it
// hides); eight interleaved counters 1339 us.
//
// The counter: *next is zero when the launch starts.  clear (if set) is
// another counter the launch zeroes for the next launch on the stream;
// finished (if set) counts workgroups out, and the last one returns *next and
// *finished to zero, so the counters are zero again when the launch ends.
struct QueueCtl {
    uint64_t *next;
    uint64_t *clear;
    uint64_t *finished;
};
constexpr int kQMaxItems = 16384;   // items whose 32-bit tile-start prefix fits in LDS
constexpr int kQSub = 2;            // 512-vector sub-tiles per claimed tile

// The item k < n holding tile g: the last k with pre[k] <= g (pre[0] = 0 <= g,
// pre non-decreasing).  Each level reads one prefix entry per lane and keeps
// the run of lanes at or below g: 64^levels entries in `levels` LDS reads.
__device__ __forceinline__ int find_item(const uint32_t *pre, int n, uint32_t g)
{
    const int lane = (int)(threadIdx.x & 63);
    int step = 1;
    while (step * 64 < n) step *= 64;
    int lo = 0;
    for (;;) {
        const int i = lo + lane * step;
        const bool ok = i < n && pre[i] <= g;
        lo += (__popcll(__ballot(ok)) - 1) * step;
        if (step == 1) break;
        step /= 64;
    }
    return __builtin_amdgcn_readfirstlane(lo);
}

// A workgroup barrier that orders LDS only: __syncthreads() also waits for
// every outstanding global store and atomic of the wave (its release fence
// covers global memory), which would drain each tile's stores before the
// next tile's loads could be issued.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <class T, class Op, int SUB>
__global__ __launch_bounds__(kB) void batched_queue_kernel(const xred_item *items, int nitems,
                                                           QueueCtl q)
{
    constexpr uint32_t kTileBytes = (uint32_t)kB * SUB * 16u;
    constexpr uint64_t kTileElems = (uint64_t)kB * SUB * T::kVec;
    auto tiles_of = [](const xred_item &it) -> uint64_t {
        return item_runnable(it) ? (it.count + kTileElems - 1) / kTileElems : 0;
    };
    auto claim = [&q]() -> uint64_t {
        return __hip_atomic_fetch_add(q.next, (uint64_t)1, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT);
    };
    extern __shared__ uint32_t s_pre[];   // nitems + 1 tile starts, in the occupancy reservation
    __shared__ uint64_t s_wave[kB / 64];
    // The claim made during tile b is written to s_claim[b % 2] at the
    // tile's end and read after its barrier; the slot's previous claim was
    // read before the barrier that precedes the write.
    __shared__ uint64_t s_claim[2];
    if (q.clear != nullptr && blockIdx.x == 0 && threadIdx.x == 0)
        __hip_atomic_store(q.clear, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    uint64_t c0 = 0;
    if (threadIdx.x == 0) c0 = claim();   // in flight while the workgroup scans
    // tile counts of this thread's consecutive items (four descriptor loads
    // in flight at a time), kept in the prefix's place; then the
    // workgroup's exclusive scan turns them into tile starts
    const int per = (nitems + kB - 1) / kB;
    const int i0 = min(nitems, (int)threadIdx.x * per), i1 = min(nitems, i0 + per);
    uint64_t mine = 0;
    for (int j = i0; j < i1; j += 4) {
        xred_item it[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (j + u < i1) it[u] = items[j + u];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (j + u < i1) {
                const uint64_t t = tiles_of(it[u]);
                mine += t;
                s_pre[j + u] = t < 0xFFFFFFFFull ? (uint32_t)t : 0xFFFFFFFFu;
            }
        }
    }
    uint64_t total = 0;
    uint64_t run = block_exclusive_scan(mine, s_wave, &total);
    for (int i = i0; i < i1; ++i) {
        const uint32_t t = s_pre[i];
        s_pre[i] = (uint32_t)run;
        run += t;
    }
    total = uniform64(total);
    if (total > 0xFFFFFFFFull) total = 0;   // more tiles than the prefix indexes: run nothing
    if (threadIdx.x == 0) {
        s_pre[nitems] = (uint32_t)total;
        s_claim[1] = c0;
    }
    __syncthreads();
    uint64_t g = uniform64(s_claim[1]);
    TileDesc cur{};
    if (g < total) {
        const int k = find_item(s_pre, nitems, (uint32_t)g);
        fetch_desc<T>(cur, items, (uint32_t)k, uniform64(g - s_pre[k]));
    }
    for (int b = 0; g < total; ++b) {
        uint64_t c = 0;
        if (threadIdx.x == 0) c = claim();   // answered while this tile streams
        // straight-line tile: sources beyond nsrc, and tiles off the fast
        // path, get a zero-length buffer range
        const size_t lb = (size_t)cur.lead * T::kSize;
        const size_t nvec = (cur.count - cur.lead) / T::kVec;
        const size_t vbytes = nvec * 16, toff = cur.lt * kTileBytes;
        const uint32_t nrec = cur.fast && toff < vbytes ? tile_nrec(vbytes, toff, kTileBytes) : 0u;
        u32x4 in[8][SUB];
#pragma unroll
        for (int p = 0; p < 8; ++p) {
            const bool on = p < cur.nsrc;
            const rsrc_t r = make_rsrc((on ? cur.p[p] : cur.dst) + lb + toff, on ? nrec : 0u);
#pragma unroll
            for (int h = 0; h < SUB; ++h)
                in[p][h] = bload<kLoadStream>(r, (uint32_t)(h * kB + threadIdx.x) * 16u);
        }
        // With this tile's loads in flight, hand the claim to every wave
        // and fetch the next tile's descriptor and source pointers, so the
        // next tile's loads can be issued as soon as this tile is stored.
        if (threadIdx.x == 0) s_claim[b & 1] = c;
        lds_barrier();
        const uint64_t gn = uniform64(s_claim[b & 1]);
        TileDesc nxt{};
        if (gn < total) {
            const int k = find_item(s_pre, nitems, (uint32_t)gn);
            fetch_desc<T>(nxt, items, (uint32_t)k, uniform64(gn - s_pre[k]));
        }
        const rsrc_t w = make_rsrc(cur.dst + lb + toff, nrec);
#pragma unroll
        for (int h = 0; h < SUB; ++h) {
            typename T::Acc acc[T::kVec];
            up_vec<T>(in[0][h], acc);
#pragma unroll
            for (int p = 1; p < 8; ++p) {
                const bool on = p < cur.nsrc;
                typename T::Acc x[T::kVec];
                up_vec<T>(in[p][h], x);
#pragma unroll
                for (int e = 0; e < T::kVec; ++e) {
                    const typename T::Acc cmb = combine<T, Op>(acc[e], x[e]);
                    acc[e] = on ? cmb : acc[e];
                }
            }
            if constexpr (__is_same(Op, OpAvg)) {
#pragma unroll
                for (int e = 0; e < T::kVec; ++e) acc[e] = avg_scale<T, Op>(acc[e], cur.nsrc);
            }
            tile_store(down_vec<T, Op>(acc), w, cur, lb + toff, nrec, h);
        }
        if (cur.fast) {
            reduce_ends<T, Op>(GlobalSrc{cur.srcs}, cur.nsrc, cur.dst,
                               cur.lt == 0 ? cur.lead : 0u,
                               (cur.lt + 1) * kTileElems >= cur.count
                                   ? (uint32_t)((cur.count - cur.lead) % T::kVec)
                                   : 0u,
                               cur.lead + nvec * T::kVec);
        } else {
            batched_tile<T, Op, SUB>(load_item(items, cur.k), cur.lt);
        }
        cur = nxt;
        g = gn;
    }
    // every claim of this workgroup has been answered (each was read back
    // above), so the last workgroup's reset is the counter's last write
    if (q.finished != nullptr && threadIdx.x == 0) {
        const uint64_t n = __hip_atomic_fetch_add(q.finished, (uint64_t)1, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
        if (n + 1 == gridDim.x) {
            __hip_atomic_store(q.next, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(q.finished, (uint64_t)0, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// ------------------------------------------------------- tile-table variant --
// Host descriptors: the host lists the item of every tile, and stages each
// item with the index of its first tile in the descriptor's reserved field;
// workgroup w takes tile w.  One workgroup per tile, dispatched in
// order, keeps the tiles in flight one compact window over the batch, as in
// the fused kernel; persistent workgroups each walking their own tiles drift
// apart and spread the loads in flight over the batch (c4: 5.3 against
// 6.9 TB/s for the same data).  Tiles are one 16-byte vector per thread and
// source, two workgroups per CU (16 waves: 6.9 TB/s against 5.9 uncapped).
// Other shapes on the 4096-item log-uniform batch (same box): 512 threads and
// 8 KiB per source, two per CU, 1199 us; one or three per CU 1462 / 1472 us;
// 16 KiB tiles one / two per CU 1321 / 1488 us; 1024 threads one per CU
// 1314 us; 256 threads four per CU, 4 / 8 KiB tiles 1367 / 1489 us.  The
// three dependent scalar loads before a tile's loads (table entry, then the
// descriptor, then the source pointers) also pace the workgroups: staging
// eight pointer slots per item so that the descriptor and the pointers load
// together made c4 slower (1241-1254 against 1204 us), like more resident
// workgroups per CU.
// Under a CU budget the grid is smaller and each workgroup strides over the
// table.
constexpr int kTB = 512;
constexpr int kTableSub = 1;          // 16-byte vectors per thread and source
constexpr int kTableWgsPerCu = 2;

template <class T>
constexpr uint64_t table_tile_elems() { return (uint64_t)kTB * kTableSub * T::kVec; }

// The fields of a descriptor a tile needs, loaded with scalar loads.
struct ItemHead {
    const char *const *srcs;
    char *dst;
    uint64_t count;
    int nsrc;
};

__device__ __forceinline__ ItemHead load_head(const xred_item *it)
{
    return ItemHead{(const char *const *)sload(&it->srcs), (char *)sload(&it->dst),
                    sload(&it->count), (int)sload(&it->nsrc)};
}

// Tile lt (of kTB * kTableSub vectors) of the item with header h.  CHECK: the descriptor is the
// caller's device memory, so an item with a NULL source pointer is skipped
// (the host validates its own descriptors before staging them).
template <class T, class Op, bool CHECK>
__device__ __forceinline__ void table_tile(const ItemHead &h, uint64_t lt)
{
    constexpr int U = kTableSub;
    constexpr uint32_t kBytes = (uint32_t)kTB * U * 16u;
    const char *const *srcs = h.srcs;
    char *dst = h.dst;
    const uint64_t count = h.count;
    const int nsrc = h.nsrc;
    const GlobalSrc src{srcs};
    const size_t toff = lt * kBytes;
    const char *p[8];
    uintptr_t diff = 0;   // bits in which some source's address differs from dst's
    bool null_src = false;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        p[q] = q < nsrc ? sload(srcs + q) : nullptr;
        diff |= q < nsrc ? (uintptr_t)p[q] ^ (uintptr_t)dst : 0;
        null_src |= q < nsrc && p[q] == nullptr;
    }
    uint64_t lead = item_lead<T>(diff, (uintptr_t)dst, count);
    if (nsrc > 8 || lead == kNoVector) {
        // the general tile: any source count, element-aligned buffers
        uintptr_t all = 0, sdiff = 0;
        const uintptr_t s0 = (uintptr_t)p[0];
        for (int q = 0; q < nsrc; ++q) {
            const uintptr_t x = (uintptr_t)sload(srcs + q);
            all |= x ^ (uintptr_t)dst;
            sdiff |= x ^ s0;
            null_src |= x == 0;
        }
        if (CHECK && null_src) return;
        lead = item_lead<T>(all, (uintptr_t)dst, count);
        uint32_t c = 0;   // > 0: the output at another offset than the sources
        if (lead == kNoVector) {
            lead = sources_lead<T>(sdiff, s0, count);
            if (lead != kNoVector) c = (uint32_t)(((uintptr_t)dst + lead * T::kSize) & 15u);
            if (c == 0) lead = kNoVector;
        }
        if (lead != kNoVector) {
            const size_t nvec = (count - lead) / T::kVec, vbytes = nvec * 16;
            const Tile tl{(size_t)lead * T::kSize + toff, tile_nrec(vbytes, toff, kBytes)};
            if (toff < vbytes) {
                if (c != 0) split_tile<T, Op, 1, kTB>(src, nsrc, dst, tl, c);
                else reduce_tile<T, Op, 0, U, kTB>(src, nsrc, dst, tl);
            }
        } else if (const uint32_t sl = shift_lead<T>((uintptr_t)dst, count * T::kSize)) {
            // sources at different offsets: vectors realigned to dst's grid
            const size_t lb = (size_t)sl * T::kSize;
            const size_t nvec = (count * T::kSize - lb - 16) / 16, vbytes = nvec * 16;
            if (toff < vbytes)
                shift_tile<T, Op, kTB>(src, nsrc, dst, lb, toff, tile_nrec(vbytes, toff, kBytes));
            reduce_ends<T, Op>(src, nsrc, dst, lt == 0 ? sl : 0u,
                               (lt + 1) * table_tile_elems<T>() >= count
                                   ? (uint32_t)(count - sl - nvec * T::kVec)
                                   : 0u,
                               sl + nvec * T::kVec);
            return;
        } else {
            const uint64_t e0 = lt * table_tile_elems<T>();
            const uint64_t e1 =
                count < e0 + table_tile_elems<T>() ? count : e0 + table_tile_elems<T>();
            for (uint64_t i = e0 + threadIdx.x; i < e1; i += kTB)
                reduce_elem<T, Op>(src, nsrc, dst, i);
            return;
        }
    } else {
        if (CHECK && null_src) return;
        // straight-line tile: sources beyond nsrc get a zero-length range
        const size_t lb = (size_t)lead * T::kSize;
        const size_t vbytes = (count - lead) / T::kVec * 16;
        const uint32_t nrec = toff < vbytes ? tile_nrec(vbytes, toff, kBytes) : 0u;
        u32x4 in[8][U];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const bool on = q < nsrc;
            const rsrc_t r = make_rsrc((on ? p[q] : dst) + lb + toff, on ? nrec : 0u);
#pragma unroll
            for (int u = 0; u < U; ++u)
                in[q][u] = bload<kLoadStream>(r, (uint32_t)(u * kTB + threadIdx.x) * 16u);
        }
        const rsrc_t w = make_rsrc(dst + lb + toff, nrec);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            typename T::Acc acc[T::kVec];
            up_vec<T>(in[0][u], acc);
#pragma unroll
            for (int q = 1; q < 8; ++q) {
                const bool on = q < nsrc;
                typename T::Acc b[T::kVec];
                up_vec<T>(in[q][u], b);
#pragma unroll
                for (int e = 0; e < T::kVec; ++e) {
                    const typename T::Acc c = combine<T, Op>(acc[e], b[e]);
                    acc[e] = on ? c : acc[e];
                }
            }
            if constexpr (__is_same(Op, OpAvg)) {
#pragma unroll
                for (int e = 0; e < T::kVec; ++e) acc[e] = avg_scale<T, Op>(acc[e], nsrc);
            }
            bstore<kStoreOut>(down_vec<T, Op>(acc), w, (uint32_t)(u * kTB + threadIdx.x) * 16u);
        }
    }
    // the item's first tile also takes the elements before its first vector,
    // its last tile those after its last full vector
    reduce_ends<T, Op>(src, nsrc, dst, lt == 0 ? (uint32_t)lead : 0u,
                       (lt + 1) * table_tile_elems<T>() >= count
                           ? (uint32_t)((count - lead) % T::kVec)
                           : 0u,
                       lead + (count - lead) / T::kVec * T::kVec);
}

// NARROW: the table holds 16-bit item indices (batches of at most 65536
// items), two per 32-bit word, little-endian; the word is loaded whole (the
// table is padded to 8 bytes) so every scalar load stays dword-aligned.
template <class T, class Op, bool NARROW>
__global__ __launch_bounds__(kTB) void batched_table_kernel(const xred_item *items,
                                                            const uint32_t *table,
                                                            uint64_t ntiles)
{
    extern __shared__ char occupancy_reservation[];
    (void)occupancy_reservation;
    for (uint64_t g = blockIdx.x; g < ntiles; g += gridDim.x) {
        uint32_t k;
        if constexpr (NARROW) {
            const uint32_t pair = sload(&table[g >> 1]);
            k = (g & 1) ? pair >> 16 : pair & 0xFFFFu;
        } else {
            k = sload(&table[g]);
        }
        const xred_item *it = items + k;
        table_tile<T, Op, false>(load_head(it), g - sload(&it->reserved));
    }
}

template <class T, class Op>
hipError_t go_table(const xred_item *d_items, const uint32_t *d_table, bool narrow,
                    uint64_t ntiles, hipStream_t s)
{
    const size_t lds = (size_t)(lds_per_cu() / kTableWgsPerCu) / 512 * 512 - 512;
    if (narrow)
        return launch_kernel(batched_table_kernel<T, Op, true>, dim3(grid_for(ntiles)), dim3(kTB),
                             lds, s, d_items, d_table, ntiles);
    return launch_kernel(batched_table_kernel<T, Op, false>, dim3(grid_for(ntiles)), dim3(kTB),
                         lds, s, d_items, d_table, ntiles);
}

// Tile-table launcher for the element types Ts.
template <class... Ts>
hipError_t batched_table_group(xred_dtype dtype, xred_op op, const xred_item *d_items,
                               const uint32_t *d_table, bool narrow, uint64_t ntiles,
                               hipStream_t s)
{
    return with_dtype_among<Ts...>(dtype, [&](auto t) {
        using T = decltype(t);
        return with_op<T, true>(op, [&](auto o) {
            return go_table<T, decltype(o)>(d_items, d_table, narrow, ntiles, s);
        });
    });
}

// ---------------------------------------------------------- grouped variant --
// Device descriptors (the host cannot see the sizes, so it cannot list the
// tiles): the batch is cut into `ngroups` runs of consecutive items, run q
// gets its own `m` workgroups (blockIdx m*q .. m*q+m-1), and tile j of the
// run goes to the run's workgroup j mod m.  The m workgroups of a run walk
// its tiles side by side, so the tiles in flight stay one compact window, as
// in the tile-table kernel; and since the workgroups of later runs are
// dispatched in order as earlier ones retire, no workgroup keeps a fixed
// share of the whole batch (a persistent grid ends with its slowest
// workgroup).  Each workgroup scans its run's descriptors into an LDS
// tile-start prefix, lists its own tiles (item, tile) by binary search, and
// runs the tile-table kernel's tile on each, with a barrier after every tile
// so the workgroup's waves read one tile together (c4: 5.7 against 5.45 TB/s
// with the waves left to drift apart).  No state is kept between calls,
// so the launch can be captured in a graph.  With fewer workgroups than
// m * ngroups (a CU budget), each set of m workgroups strides over the runs.
constexpr int kGrpMaxItems = 2048;          // items per run (LDS prefix)
constexpr int kGrpPerThread = kGrpMaxItems / kTB;
constexpr size_t kGrpLdsBytes =
    sizeof(uint64_t) * (kGrpMaxItems + 1 + kTB + kTB / 64) + sizeof(uint32_t) * kTB;

template <class T>
__device__ __forceinline__ uint64_t table_item_tiles(const xred_item &it)
{
    if (!item_runnable(it)) return 0;
    return (it.count + table_tile_elems<T>() - 1) / table_tile_elems<T>();
}

template <class T, class Op>
__global__ __launch_bounds__(kTB) void batched_grouped_kernel(const xred_item *items, int nitems,
                                                              uint32_t ngroups, uint32_t m)
{
    extern __shared__ uint64_t s_grp[];          // the occupancy reservation, partly used
    uint64_t *s_pre = s_grp;                     // kGrpMaxItems + 1 tile starts
    uint64_t *s_lt = s_pre + kGrpMaxItems + 1;   // kTB tiles within their item
    uint64_t *s_wave = s_lt + kTB;               // kTB / 64 wave sums
    uint32_t *s_item = (uint32_t *)(s_wave + kTB / 64);   // kTB items within the run
    const uint32_t w = blockIdx.x % m;
    const uint32_t sets = gridDim.x / m;
    for (uint32_t q = blockIdx.x / m; q < ngroups; q += sets) {
        const int i0 = (int)((uint64_t)nitems * q / ngroups);
        const int n = (int)((uint64_t)nitems * (q + 1) / ngroups) - i0;   // <= kGrpMaxItems
        // tile counts of the run's items, kGrpPerThread consecutive items per thread
        uint64_t c[kGrpPerThread], mine = 0;
#pragma unroll
        for (int j = 0; j < kGrpPerThread; ++j) {
            const int i = (int)threadIdx.x * kGrpPerThread + j;
            c[j] = i < n ? table_item_tiles<T>(items[i0 + i]) : 0;
            mine += c[j];
        }
        uint64_t total = 0;
        uint64_t run = block_exclusive_scan(mine, s_wave, &total);
#pragma unroll
        for (int j = 0; j < kGrpPerThread; ++j) {
            const int i = (int)threadIdx.x * kGrpPerThread + j;
            if (i < n) s_pre[i] = run;
            run += c[j];
        }
        if (threadIdx.x == 0) s_pre[n] = total;
        __syncthreads();
        // this workgroup's tiles are w, w + m, w + 2m, ... below total
        for (uint64_t g0 = w; g0 < total; g0 += (uint64_t)kTB * m) {
            const uint64_t left = (total - g0 + m - 1) / m;
            const int cnt = left < (uint64_t)kTB ? (int)left : kTB;
            if ((int)threadIdx.x < cnt) {
                const uint64_t g = g0 + (uint64_t)threadIdx.x * m;
                int lo = 0, hi = n;   // s_pre[lo] <= g < s_pre[hi]
                while (hi - lo > 1) {
                    const int mid = (lo + hi) >> 1;
                    if (s_pre[mid] <= g) lo = mid;
                    else hi = mid;
                }
                s_item[threadIdx.x] = (uint32_t)lo;
                s_lt[threadIdx.x] = g - s_pre[lo];
            }
            __syncthreads();
            for (int j = 0; j < cnt; ++j) {
                const uint32_t k = __builtin_amdgcn_readfirstlane(s_item[j]);
                table_tile<T, Op, true>(load_head(items + i0 + k), uniform64(s_lt[j]));
                __syncthreads();   // the waves start every tile together
            }
            __syncthreads();   // the list is rewritten next
        }
        __syncthreads();       // the prefix is rewritten next
    }
}

template <class T, class Op>
hipError_t go_grouped(const xred_item *d_items, int nitems, uint32_t ngroups, uint32_t m,
                      unsigned grid, int wgs_per_cu, hipStream_t s)
{
    size_t lds = (size_t)(lds_per_cu() / wgs_per_cu) / 512 * 512 - 512;
    if (lds < kGrpLdsBytes) lds = kGrpLdsBytes;
    return launch_kernel(batched_grouped_kernel<T, Op>, dim3(grid), dim3(kTB), lds, s, d_items,
                         nitems, ngroups, m);
}

// Grouped launcher for the element types Ts.
template <class... Ts>
hipError_t batched_grouped_group(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                 int nitems, uint32_t ngroups, uint32_t m, unsigned grid,
                                 int wgs_per_cu, hipStream_t s)
{
    return with_dtype_among<Ts...>(dtype, [&](auto t) {
        using T = decltype(t);
        return with_op<T, true>(op, [&](auto o) {
            return go_grouped<T, decltype(o)>(d_items, nitems, ngroups, m, grid, wgs_per_cu, s);
        });
    });
}

template <class T, class Op>
hipError_t go_queue(const xred_item *d_items, int nitems, QueueCtl q, unsigned grid,
                    int wgs_per_cu, hipStream_t s)
{
    size_t lds = (size_t)(lds_per_cu() / wgs_per_cu) / 512 * 512 - 512;
    const size_t need = sizeof(uint32_t) * ((size_t)nitems + 1);
    if (lds < need) lds = need;
    return launch_kernel(batched_queue_kernel<T, Op, kQSub>, dim3(grid), dim3(kB), lds, s,
                         d_items, nitems, q);
}

// Queue launcher for the element types Ts.
template <class... Ts>
hipError_t batched_queue_group(xred_dtype dtype, xred_op op, const xred_item *d_items,
                               int nitems, QueueCtl q, unsigned grid, int wgs_per_cu,
                               hipStream_t s)
{
    return with_dtype_among<Ts...>(dtype, [&](auto t) {
        using T = decltype(t);
        return with_op<T, true>(op, [&](auto o) {
            return go_queue<T, decltype(o)>(d_items, nitems, q, grid, wgs_per_cu, s);
        });
    });
}

constexpr size_t rr_lds_bytes(int nitems)
{
    return sizeof(uint2) * kListMax + sizeof(uint32_t) * ((size_t)nitems + 1);
}

// The round-robin kernel's LDS is rounded up to whole kRrLdsStep blocks, so
// its occupancy is known per block count and cached per device.
constexpr size_t kRrLdsStep = 4096;
constexpr int kRrLdsSteps = (int)((rr_lds_bytes(kRrMaxItems) + kRrLdsStep - 1) / kRrLdsStep);

template <class T, class Op, bool PLANNED>
int rr_per_cu(int steps)
{
    static int cache[kMaxDevicesCached][kRrLdsSteps + 1];
    const int dev = current_device_index();
    int v = __atomic_load_n(&cache[dev][steps], __ATOMIC_RELAXED);
    if (v <= 0) {
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &v, (const void *)batched_rr_kernel<T, Op, PLANNED>, kB,
                (size_t)steps * kRrLdsStep) != hipSuccess ||
            v <= 0)
            v = 1;
        __atomic_store_n(&cache[dev][steps], v, __ATOMIC_RELAXED);
    }
    return v;
}

template <class T, class Op>
hipError_t go_rr(bool planned, const xred_item *d_items, int nitems, const uint32_t *d_tile_start,
                 hipStream_t s)
{
    const int steps = (int)((rr_lds_bytes(nitems) + kRrLdsStep - 1) / kRrLdsStep);
    const size_t lds = (size_t)steps * kRrLdsStep;
    const int per_cu = planned ? rr_per_cu<T, Op, true>(steps) : rr_per_cu<T, Op, false>(steps);
    const unsigned grid = batched_rr_grid(per_cu);
    if (planned)
        return launch_kernel(batched_rr_kernel<T, Op, true>, dim3(grid), dim3(kB), lds, s,
                             d_items, nitems, d_tile_start);
    return launch_kernel(batched_rr_kernel<T, Op, false>, dim3(grid), dim3(kB), lds, s, d_items,
                         nitems, d_tile_start);
}

template <class T, class Op>
hipError_t go(const xred_item *d_items, int nitems, const WgStart *d_wg, unsigned grid,
              hipStream_t s)
{
    return launch_kernel(batched_kernel<T, Op>, dim3(grid), dim3(kB), 0, s, d_items, nitems, d_wg);
}

// Range-walking launcher for the element types Ts.
template <class... Ts>
hipError_t batched_group(xred_dtype dtype, xred_op op, const xred_item *d_items, int nitems,
                         const WgStart *d_wg, unsigned grid, hipStream_t s)
{
    return with_dtype_among<Ts...>(dtype, [&](auto t) {
        using T = decltype(t);
        return with_op<T, true>(op, [&](auto o) {
            return go<T, decltype(o)>(d_items, nitems, d_wg, grid, s);
        });
    });
}

// Round-robin launcher for the element types Ts.
template <class... Ts>
hipError_t batched_rr_group(xred_dtype dtype, xred_op op, const xred_item *d_items, int nitems,
                            const uint32_t *d_tile_start, hipStream_t s)
{
    const bool planned = d_tile_start != nullptr;
    return with_dtype_among<Ts...>(dtype, [&](auto t) {
        using T = decltype(t);
        return with_op<T, true>(op, [&](auto o) {
            return go_rr<T, decltype(o)>(planned, d_items, nitems, d_tile_start, s);
        });
    });
}

}  // namespace
}  // namespace xred
