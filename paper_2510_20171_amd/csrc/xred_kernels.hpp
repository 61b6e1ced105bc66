// xred_kernels.hpp -- reduce-step kernels for gfx950.
//
// All kernels stream 16-byte vectors: one wavefront covers 64 lanes x 16 B =
// 1 KiB of every source per vector step, and each thread keeps U vectors of
// every source in flight before folding (the fold order over sources is the
// fixed left fold 0..P-1 whatever the load order).  Sources are read with
// nontemporal loads (each byte is used once), outputs written with
// nontemporal stores; the step-wise accumulator uses ordinary accesses so it
// stays in L2 / MALL between launches.
//
// Work is split into tiles of kBlock*U vectors.  Tile t is processed by
// workgroup t mod gridDim.x, so with a fixed grid a tile always lands on the
// same XCD (workgroups are dispatched to the 8 XCDs round-robin).
#pragma once

#include "xred_device.hpp"
#include "../../include/xred.h"

namespace xred {

// Source pointers passed by value in the kernel arguments (<= MAXP sources).
template <int MAXP>
struct KernargSrc {
    const char *p[MAXP];
    __device__ __forceinline__ const char *operator()(int i) const { return p[i]; }
};

// Source pointers read from a device array (batched descriptors).
struct GlobalSrc {
    const char *const *p;
    __device__ __forceinline__ const char *operator()(int i) const { return p[i]; }
};

// Fold G consecutive sources starting at p0 into acc (G known at compile time).
// FIRST: the first source initialises the accumulator instead of being folded.
template <class T, class Op, int G, int U, bool FIRST, bool NTL, bool CHECKED, class Src>
__device__ __forceinline__ void fold_group(typename T::Acc (&acc)[U][T::kVec], const Src &src,
                                           int p0, size_t v0, size_t nvec)
{
    u32x4 in[G][U];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const char *base = src(p0 + g);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const size_t v = v0 + (size_t)u * kBlock;
            if (!CHECKED || v < nvec) in[g][u] = load16<NTL>(base + v * 16);
            else in[g][u] = u32x4{0u, 0u, 0u, 0u};
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            if (FIRST && g == 0) up_vec<T>(in[0][u], acc[u]);
            else fold_vec<T, Op>(acc[u], in[g][u]);
        }
    }
}

// One tile of U vectors per thread: vectors v0 + u*kBlock, u < U.
// NP > 0: exactly NP sources (compile time); NP == 0: nsrc > 8 sources,
// folded in groups of 8 plus a remainder group, in source order.
template <class T, class Op, int NP, int U, bool NTL, bool NTS, bool CHECKED, class Src>
__device__ __forceinline__ void reduce_vec_tile(const Src &src, int nsrc, char *dst, size_t v0,
                                                size_t nvec)
{
    typename T::Acc acc[U][T::kVec];
    if constexpr (NP > 0) {
        fold_group<T, Op, NP, U, true, NTL, CHECKED>(acc, src, 0, v0, nvec);
    } else {
        fold_group<T, Op, 8, U, true, NTL, CHECKED>(acc, src, 0, v0, nvec);
        int p = 8;
        for (; p + 8 <= nsrc; p += 8)
            fold_group<T, Op, 8, U, false, NTL, CHECKED>(acc, src, p, v0, nvec);
        switch (nsrc - p) {
        case 1: fold_group<T, Op, 1, U, false, NTL, CHECKED>(acc, src, p, v0, nvec); break;
        case 2: fold_group<T, Op, 2, U, false, NTL, CHECKED>(acc, src, p, v0, nvec); break;
        case 3: fold_group<T, Op, 3, U, false, NTL, CHECKED>(acc, src, p, v0, nvec); break;
        case 4: fold_group<T, Op, 4, U, false, NTL, CHECKED>(acc, src, p, v0, nvec); break;
        case 5: fold_group<T, Op, 5, U, false, NTL, CHECKED>(acc, src, p, v0, nvec); break;
        case 6: fold_group<T, Op, 6, U, false, NTL, CHECKED>(acc, src, p, v0, nvec); break;
        case 7: fold_group<T, Op, 7, U, false, NTL, CHECKED>(acc, src, p, v0, nvec); break;
        default: break;
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const size_t v = v0 + (size_t)u * kBlock;
        if (!CHECKED || v < nvec) store16<NTS>(dst + v * 16, down_vec<T, Op>(acc[u]));
    }
}

// Element i (scalar path): used for tails shorter than a vector and for
// buffers that are not all 16-byte aligned.
template <class T, class Op, class Src>
__device__ __forceinline__ void reduce_elem(const Src &src, int nsrc, char *dst, size_t i)
{
    typename T::Acc a = up1<T>(src(0), i);
    for (int p = 1; p < nsrc; ++p) a = combine<T, Op>(a, up1<T>(src(p), i));
    down1<T, Op>(dst, i, a);
}

// ------------------------------------------------------ fused P-source --
// dst[i] = fold_p src_p[i] for nvec*kVec + tail elements, all pointers 16 B
// aligned.  Tiles of kBlock*U vectors; the ragged last tile is bounds
// checked; the tail (< kVec elements) is done by one workgroup, scalar.
template <class T, class Op, int NP, int MAXP, int U, bool NTL, bool NTS>
__global__ __launch_bounds__(kBlock) void reduce_vec_kernel(KernargSrc<MAXP> src, int nsrc,
                                                            char *dst, size_t nvec,
                                                            uint32_t tail)
{
    constexpr size_t kTile = (size_t)kBlock * U;
    const size_t nfull = nvec / kTile;
    for (size_t t = blockIdx.x; t < nfull; t += gridDim.x)
        reduce_vec_tile<T, Op, NP, U, NTL, NTS, false>(src, nsrc, dst, t * kTile + threadIdx.x,
                                                       nvec);
    if (nfull * kTile < nvec && blockIdx.x == nfull % gridDim.x)
        reduce_vec_tile<T, Op, NP, U, NTL, NTS, true>(src, nsrc, dst,
                                                      nfull * kTile + threadIdx.x, nvec);
    if (tail != 0 && blockIdx.x == (nfull + 1) % gridDim.x && threadIdx.x < tail)
        reduce_elem<T, Op>(src, nsrc, dst, nvec * T::kVec + threadIdx.x);
}

// Any alignment: one element per thread per step.
template <class T, class Op>
__global__ __launch_bounds__(kBlock) void reduce_scalar_kernel(KernargSrc<XRED_MAX_SRC> src,
                                                               int nsrc, char *dst,
                                                               size_t count)
{
    const size_t stride = (size_t)gridDim.x * kBlock;
    for (size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x; i < count; i += stride)
        reduce_elem<T, Op>(src, nsrc, dst, i);
}

// ------------------------------------------------------------ step-wise --
// acc holds kVec 4-byte accumulators per 16-byte input vector, i.e. kVec/4
// 16-byte accumulator vectors.
template <class T>
__device__ __forceinline__ void load_acc(const char *acc, size_t v, typename T::Acc (&a)[T::kVec])
{
#pragma unroll
    for (int h = 0; h < T::kVec / 4; ++h) {
        u32x4 x = load16<false>(acc + (v * T::kVec + 4 * h) * 4);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if constexpr (T::kFloat) a[4 * h + j] = __uint_as_float(x[j]);
            else a[4 * h + j] = x[j];
        }
    }
}

template <class T, class Op>
__device__ __forceinline__ void store_acc(char *acc, size_t v, const typename T::Acc (&a)[T::kVec])
{
#pragma unroll
    for (int h = 0; h < T::kVec / 4; ++h) {
        u32x4 x;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if constexpr (T::kFloat) x[j] = __float_as_uint(finalize<T, Op>(a[4 * h + j]));
            else x[j] = a[4 * h + j];
        }
        store16<false>(acc + (v * T::kVec + 4 * h) * 4, x);
    }
}

template <class T, class Op, unsigned FLAGS>
__device__ __forceinline__ void step_vec(const char *in, char *acc, char *dst, size_t v)
{
    constexpr bool kInit = (FLAGS & XRED_STEP_INIT) != 0, kFinal = (FLAGS & XRED_STEP_FINAL) != 0;
    u32x4 x = load16<true>(in + v * 16);
    typename T::Acc a[T::kVec];
    if constexpr (kInit) {
        up_vec<T>(x, a);
    } else {
        load_acc<T>(acc, v, a);
        fold_vec<T, Op>(a, x);
    }
    if constexpr (kFinal) store16<true>(dst + v * 16, down_vec<T, Op>(a));
    else store_acc<T, Op>(acc, v, a);
}

template <class T, class Op, unsigned FLAGS>
__device__ __forceinline__ void step_elem(const char *in, char *acc, char *dst, size_t i)
{
    constexpr bool kInit = (FLAGS & XRED_STEP_INIT) != 0, kFinal = (FLAGS & XRED_STEP_FINAL) != 0;
    typename T::Acc x = up1<T>(in, i);
    typename T::Acc a;
    if constexpr (kInit) {
        a = x;
    } else {
        if constexpr (T::kFloat) a = ((const float *)acc)[i];
        else a = ((const uint32_t *)acc)[i];
        a = combine<T, Op>(a, x);
    }
    if constexpr (kFinal) {
        down1<T, Op>(dst, i, a);
    } else {
        if constexpr (T::kFloat) ((float *)acc)[i] = finalize<T, Op>(a);
        else ((uint32_t *)acc)[i] = a;
    }
}

// One ReduceCopy step over nvec vectors + tail elements (16 B aligned) or,
// with VEC = false, over count = tail elements of any alignment.
template <class T, class Op, unsigned FLAGS, int U, bool VEC>
__global__ __launch_bounds__(kBlock) void step_kernel(const char *in, char *acc, char *dst,
                                                      size_t nvec, size_t tail)
{
    if constexpr (VEC) {
        constexpr size_t kTile = (size_t)kBlock * U;
        const size_t ntiles = (nvec + kTile - 1) / kTile;
        for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t v = t * kTile + (size_t)u * kBlock + threadIdx.x;
                if (v < nvec) step_vec<T, Op, FLAGS>(in, acc, dst, v);
            }
        }
        if (tail != 0 && blockIdx.x == ntiles % gridDim.x && threadIdx.x < tail)
            step_elem<T, Op, FLAGS>(in, acc, dst, nvec * T::kVec + threadIdx.x);
    } else {
        const size_t stride = (size_t)gridDim.x * kBlock;
        for (size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x; i < tail; i += stride)
            step_elem<T, Op, FLAGS>(in, acc, dst, i);
    }
}

// dst = down(acc): the closing cast of a step-wise sequence.
template <class T, int U, bool VEC>
__global__ __launch_bounds__(kBlock) void acc_cast_kernel(const char *acc, char *dst, size_t nvec,
                                                          size_t tail)
{
    if constexpr (VEC) {
        constexpr size_t kTile = (size_t)kBlock * U;
        const size_t ntiles = (nvec + kTile - 1) / kTile;
        for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t v = t * kTile + (size_t)u * kBlock + threadIdx.x;
                if (v < nvec) {
                    typename T::Acc a[T::kVec];
                    load_acc<T>(acc, v, a);
                    store16<true>(dst + v * 16, down_vec<T, OpSum>(a));
                }
            }
        }
        if (tail != 0 && blockIdx.x == ntiles % gridDim.x && threadIdx.x < tail) {
            const size_t i = nvec * T::kVec + threadIdx.x;
            typename T::Acc a;
            if constexpr (T::kFloat) a = ((const float *)acc)[i];
            else a = ((const uint32_t *)acc)[i];
            down1<T, OpSum>(dst, i, a);
        }
    } else {
        const size_t stride = (size_t)gridDim.x * kBlock;
        for (size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x; i < tail; i += stride) {
            typename T::Acc a;
            if constexpr (T::kFloat) a = ((const float *)acc)[i];
            else a = ((const uint32_t *)acc)[i];
            down1<T, OpSum>(dst, i, a);
        }
    }
}

}  // namespace xred
