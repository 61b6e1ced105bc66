// xred_batched.hip -- many independent reductions in one launch.
//
// Small messages are dominated by per-call overhead (the T_c term of the
// LogP model in Section 6.2), so a batch of K reductions is run as one
// kernel.  Work is cut into tiles of kB*kU 16-byte vectors of one item;
// the global tile sequence (item 0's tiles, then item 1's, ...) is split
// into one contiguous range per workgroup, so each workgroup walks forward
// through consecutive items and reads each descriptor once.
//
// Two ways to find a workgroup's range:
//   planned  (host descriptors): the host computes each workgroup's first
//            item, first tile and tile count and stages them with the items;
//   device   (XRED_ITEMS_ON_DEVICE): descriptors are read only when the
//            kernel runs (metadata by reference, Section 6.1), so every
//            workgroup sums the tile counts itself (an LDS scan over the
//            descriptors), then locates its first tile.  No state is kept
//            between calls, so the kernel can be captured in a graph.

#include "xred_internal.hpp"
#include "xred_kernels.hpp"

namespace xred {
namespace {

constexpr int kU = 1;
constexpr int kB = 512;

template <class T>
constexpr uint64_t tile_vecs() { return (uint64_t)kB * kU; }
template <class T>
constexpr uint64_t tile_elems() { return tile_vecs<T>() * T::kVec; }
constexpr uint32_t kTileBytes = (uint32_t)kB * kU * 16u;

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

// Tile lt of one item.
template <class T, class Op>
__device__ void batched_tile(const xred_item &it, uint64_t lt)
{
    const char *const *sp = (const char *const *)it.srcs;
    const int nsrc = (int)it.nsrc;
    uintptr_t bits = (uintptr_t)it.dst;
    bool null_src = false;
    for (int p = 0; p < nsrc; ++p) {
        const uintptr_t q = (uintptr_t)sload(sp + p);
        bits |= q;
        null_src |= q == 0;
    }
    if (null_src) return;
    char *dst = (char *)it.dst;
    const GlobalSrc src{sp};
    const uint64_t count = it.count;
    if ((bits & 15u) == 0) {
        const size_t nvec = count / T::kVec;
        const size_t vbytes = nvec * 16;
        const size_t off = lt * kTileBytes;
        if (off < vbytes) {
            const Tile tl{off, tile_nrec(vbytes, off, kTileBytes)};
            switch (nsrc) {
            case 1: reduce_tile<T, Op, 1, kU, kB>(src, nsrc, dst, tl); break;
            case 2: reduce_tile<T, Op, 2, kU, kB>(src, nsrc, dst, tl); break;
            case 3: reduce_tile<T, Op, 3, kU, kB>(src, nsrc, dst, tl); break;
            case 4: reduce_tile<T, Op, 4, kU, kB>(src, nsrc, dst, tl); break;
            case 5: reduce_tile<T, Op, 5, kU, kB>(src, nsrc, dst, tl); break;
            case 6: reduce_tile<T, Op, 6, kU, kB>(src, nsrc, dst, tl); break;
            case 7: reduce_tile<T, Op, 7, kU, kB>(src, nsrc, dst, tl); break;
            case 8: reduce_tile<T, Op, 8, kU, kB>(src, nsrc, dst, tl); break;
            case 16: reduce_tile<T, Op, 16, kU, kB>(src, nsrc, dst, tl); break;
            case 32: reduce_tile<T, Op, 32, kU, kB>(src, nsrc, dst, tl); break;
            case 64: reduce_tile<T, Op, 64, kU, kB>(src, nsrc, dst, tl); break;
            default: reduce_tile<T, Op, 0, kU, kB>(src, nsrc, dst, tl); break;
            }
        }
        // the item's last tile also takes the elements after its last full vector
        if ((lt + 1) * tile_elems<T>() >= count) {
            const uint32_t tail = (uint32_t)(count % T::kVec);
            if (threadIdx.x < tail) reduce_elem<T, Op>(src, nsrc, dst, nvec * T::kVec + threadIdx.x);
        }
    } else {
        const uint64_t e0 = lt * tile_elems<T>();
        const uint64_t e1 = count < e0 + tile_elems<T>() ? count : e0 + tile_elems<T>();
        for (uint64_t i = e0 + threadIdx.x; i < e1; i += kB) reduce_elem<T, Op>(src, nsrc, dst, i);
    }
}

template <class T, class Op, bool PLANNED>
__global__ __launch_bounds__(kB) void batched_kernel(const xred_item *items, int nitems,
                                                         const WgStart *wg)
{
    __shared__ uint64_t s_scan[kB];
    __shared__ uint64_t s_start[2];
    uint64_t k, lt, left;
    if constexpr (PLANNED) {
        const WgStart *w = wg + blockIdx.x;
        k = sload(&w->item);
        lt = sload(&w->local_tile);
        left = sload(&w->ntiles);
    } else {
        uint64_t mine = 0;
        for (int i = threadIdx.x; i < nitems; i += kB) mine += item_tiles<T, true>(items[i]);
        block_inclusive_scan(mine, s_scan);
        const uint64_t total = s_scan[kB - 1];
        const uint64_t g0 = total * blockIdx.x / gridDim.x;
        const uint64_t g1 = total * (blockIdx.x + 1) / gridDim.x;
        if (g0 == g1) return;
        left = g1 - g0;
        // find the item holding global tile g0 (if none is found the walk
        // below starts past the last item and does nothing)
        if (threadIdx.x == 0) {
            s_start[0] = (uint64_t)nitems;
            s_start[1] = 0;
        }
        uint64_t base = 0;
        for (int w0 = 0; w0 < nitems; w0 += kB) {
            const int i = w0 + (int)threadIdx.x;
            const uint64_t c = i < nitems ? item_tiles<T, true>(items[i]) : 0;
            const uint64_t incl = block_inclusive_scan(c, s_scan);
            const uint64_t excl = incl - c;
            if (c > 0 && base + excl <= g0 && g0 < base + incl) {
                s_start[0] = (uint64_t)i;
                s_start[1] = g0 - base - excl;
            }
            const uint64_t wtot = s_scan[kB - 1];
            __syncthreads();
            if (base + wtot > g0) break;
            base += wtot;
        }
        k = s_start[0];
        lt = s_start[1];
    }
    k = uniform64(k);
    lt = uniform64(lt);
    left = uniform64(left);
    while (left > 0 && k < (uint64_t)nitems) {
        k = uniform64(k);
        const xred_item it = load_item(items, k);
        const uint64_t nt = item_tiles<T, !PLANNED>(it);
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

template <class T, class Op>
hipError_t go(bool planned, const xred_item *d_items, int nitems, const WgStart *d_wg,
              unsigned grid, hipStream_t s)
{
    if (planned)
        hipLaunchKernelGGL((batched_kernel<T, Op, true>), dim3(grid), dim3(kB), 0, s, d_items,
                           nitems, d_wg);
    else
        hipLaunchKernelGGL((batched_kernel<T, Op, false>), dim3(grid), dim3(kB), 0, s,
                           d_items, nitems, d_wg);
    return hipGetLastError();
}

template <class T>
hipError_t go_op(xred_op op, bool planned, const xred_item *d_items, int nitems,
                 const WgStart *d_wg, unsigned grid, hipStream_t s)
{
    switch (op) {
    case XRED_SUM: return go<T, OpSum>(planned, d_items, nitems, d_wg, grid, s);
    case XRED_PROD: return go<T, OpProd>(planned, d_items, nitems, d_wg, grid, s);
    case XRED_MAX: return go<T, OpMax>(planned, d_items, nitems, d_wg, grid, s);
    case XRED_MIN: return go<T, OpMin>(planned, d_items, nitems, d_wg, grid, s);
    }
    return hipErrorInvalidValue;
}

hipError_t dispatch(xred_dtype dtype, xred_op op, bool planned, const xred_item *d_items,
                    int nitems, const WgStart *d_wg, unsigned grid, hipStream_t s)
{
    switch (dtype) {
    case XRED_FLOAT32: return go_op<TF32>(op, planned, d_items, nitems, d_wg, grid, s);
    case XRED_BFLOAT16: return go_op<TBF16>(op, planned, d_items, nitems, d_wg, grid, s);
    case XRED_INT32: return go_op<TI32>(op, planned, d_items, nitems, d_wg, grid, s);
    case XRED_UINT32: return go_op<TU32>(op, planned, d_items, nitems, d_wg, grid, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

uint64_t batched_tile_elems(xred_dtype dtype)
{
    switch (dtype) {
    case XRED_BFLOAT16: return tile_elems<TBF16>();
    case XRED_FLOAT32: return tile_elems<TF32>();
    case XRED_INT32: return tile_elems<TI32>();
    case XRED_UINT32: return tile_elems<TU32>();
    default: return 0;
    }
}

hipError_t launch_batched_planned(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                  int nitems, const WgStart *d_wg, unsigned grid,
                                  hipStream_t stream)
{
    return dispatch(dtype, op, true, d_items, nitems, d_wg, grid, stream);
}

hipError_t launch_batched_device(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                 int nitems, unsigned grid, hipStream_t stream)
{
    return dispatch(dtype, op, false, d_items, nitems, nullptr, grid, stream);
}

}  // namespace xred
