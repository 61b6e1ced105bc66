// xred_kernels.hpp -- reduce-step kernels for gfx950.
//
// All kernels stream 16-byte vectors: one wavefront covers 64 lanes x 16 B =
// 1 KiB of every source per vector step, and each thread keeps U vectors of
// every source in flight before folding (the fold order over sources is the
// fixed left fold 0..P-1 whatever the load order).
//
// Memory is accessed through buffer resource descriptors built per tile
// (base = stream + tile offset, num_records = bytes of the tile that exist).
// The hardware range check then replaces per-lane bounds tests: loads past
// num_records return 0 and stores past it are dropped, so the ragged last
// tile runs the same straight-line code as every other tile.  Buffer
// instructions also always address global memory (no flat accesses when
// pointers come from device-side descriptors) and carry the cache policy:
// sources are read nontemporally (each byte is used once); outputs are
// written with device-scope (sc1) stores, which measured 2-5 % faster on
// MI355X for this 8:1 read/write mix than ordinary write-back stores and
// faster still than nontemporal stores; the step-wise accumulator uses
// ordinary loads and stores, which may leave it in the MALL between
// launches (not in L2: a launch starts with its L2 lines invalidated).
//
// Work is split into tiles of B*U vectors.  Tile t is processed by workgroup
// t mod gridDim.x, so with a fixed grid a tile always lands on the same XCD
// (workgroups are dispatched to the 8 XCDs round-robin).
#pragma once

#include "xred_device.hpp"
#include "../../include/xred.h"

namespace xred {

// Fourth dword of a raw (stride 0) buffer descriptor on gfx9-family parts:
// 32-bit data format, no swizzle.
constexpr int kRsrcWord3 = 0x00020000;
// Cache-policy bits of buffer instructions (gfx940 family): sc0 = 1, nt = 2, sc1 = 16.
constexpr int kLoadStream = 2;   // nontemporal
constexpr int kLoadKeep = 0;     // ordinary
constexpr int kStoreOut = 16;    // sc1: device scope
constexpr int kStoreKeep = 0;    // ordinary write-back

typedef __amdgpu_buffer_rsrc_t rsrc_t;

__device__ __forceinline__ rsrc_t make_rsrc(const char *base, uint32_t nbytes)
{
    return __builtin_amdgcn_make_buffer_rsrc((void *)base, (short)0, (int)nbytes, kRsrcWord3);
}

template <int POL>
__device__ __forceinline__ u32x4 bload(rsrc_t r, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, POL);
}

template <int POL>
__device__ __forceinline__ void bstore(u32x4 v, rsrc_t r, uint32_t off)
{
    __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, POL);
}

// Bytes of a tile that exist: min(tile, total - off).
__device__ __forceinline__ uint32_t tile_nrec(size_t total, size_t off, uint32_t tile)
{
    const size_t left = total - off;
    return left < tile ? (uint32_t)left : tile;
}

// Source pointers passed by value in the kernel arguments (<= MAXP sources).
template <int MAXP>
struct KernargSrc {
    const char *p[MAXP];
    __device__ __forceinline__ const char *operator()(int i) const { return p[i]; }
};

// Scalar load of a value every lane of the wavefront reads at the same
// address: going through the constant address space makes the compiler use
// s_load into SGPRs, so buffer descriptors built from the value are uniform
// (a vector load would force a readfirstlane loop around every buffer access).
template <class V>
__device__ __forceinline__ V sload(const V *p)
{
    return *(const __attribute__((address_space(4))) V *)p;
}

// Source pointers read from a device array (batched descriptors).
struct GlobalSrc {
    const char *const *p;
    __device__ __forceinline__ const char *operator()(int i) const { return sload(p + i); }
};

// Geometry of one tile of one 16-byte-vector stream: the byte offset of the
// tile and how many of its bytes exist.
struct Tile {
    size_t off;     // byte offset of the tile in every stream
    uint32_t nrec;  // bytes of the tile inside the streams' vector part
};

// Fold G consecutive sources starting at p0 into acc (G known at compile time).
// FIRST: the first source initialises the accumulator instead of being folded.
template <class T, class Op, int G, int U, int B, bool FIRST, class Src>
__device__ __forceinline__ void fold_group(typename T::Acc (&acc)[U][T::kVec], const Src &src,
                                           int p0, Tile tl)
{
    u32x4 in[G][U];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const rsrc_t r = make_rsrc(src(p0 + g) + tl.off, tl.nrec);
#pragma unroll
        for (int u = 0; u < U; ++u)
            in[g][u] = bload<kLoadStream>(r, (uint32_t)(u * B + threadIdx.x) * 16u);
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

// NG full groups of 8 sources (compile time), software pipelined: the loads of
// group g+1 are issued before group g is folded, so a wave always has the next
// group's bytes in flight while it folds.  Fold order is still 0..8*NG-1.
template <class T, class Op, int NG, int U, int B, class Src>
__device__ __forceinline__ void fold_groups_pipelined(typename T::Acc (&acc)[U][T::kVec],
                                                      const Src &src, Tile tl)
{
    u32x4 buf[2][8][U];
#pragma unroll
    for (int g = 0; g <= NG; ++g) {
        if (g < NG) {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const rsrc_t r = make_rsrc(src(8 * g + j) + tl.off, tl.nrec);
#pragma unroll
                for (int u = 0; u < U; ++u)
                    buf[g & 1][j][u] =
                        bload<kLoadStream>(r, (uint32_t)(u * B + threadIdx.x) * 16u);
            }
        }
        if (g > 0) {
            const int h = (g - 1) & 1;
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    if (g == 1 && j == 0) up_vec<T>(buf[h][0][u], acc[u]);
                    else fold_vec<T, Op>(acc[u], buf[h][j][u]);
                }
            }
        }
    }
}

// One tile: U vectors per thread at tile-relative vector u*B + threadIdx.x.
// 0 < NP <= 8: exactly NP sources, all loads issued before folding;
// NP = 16, 32, 64: whole groups of 8, software pipelined;
// NP == 0: any nsrc > 8, folded in groups of 8 plus a remainder group.
// Every variant folds in source order 0..P-1.
template <class T, class Op, int NP, int U, int B, class Src>
__device__ __forceinline__ void reduce_tile(const Src &src, int nsrc, char *dst, Tile tl)
{
    typename T::Acc acc[U][T::kVec];
    if constexpr (NP > 8) {
        static_assert(NP % 8 == 0, "compile-time source counts above 8 are whole groups");
        fold_groups_pipelined<T, Op, NP / 8, U, B>(acc, src, tl);
    } else if constexpr (NP > 0) {
        fold_group<T, Op, NP, U, B, true>(acc, src, 0, tl);
    } else {
        fold_group<T, Op, 8, U, B, true>(acc, src, 0, tl);
        int p = 8;
        for (; p + 8 <= nsrc; p += 8) fold_group<T, Op, 8, U, B, false>(acc, src, p, tl);
        switch (nsrc - p) {
        case 1: fold_group<T, Op, 1, U, B, false>(acc, src, p, tl); break;
        case 2: fold_group<T, Op, 2, U, B, false>(acc, src, p, tl); break;
        case 3: fold_group<T, Op, 3, U, B, false>(acc, src, p, tl); break;
        case 4: fold_group<T, Op, 4, U, B, false>(acc, src, p, tl); break;
        case 5: fold_group<T, Op, 5, U, B, false>(acc, src, p, tl); break;
        case 6: fold_group<T, Op, 6, U, B, false>(acc, src, p, tl); break;
        case 7: fold_group<T, Op, 7, U, B, false>(acc, src, p, tl); break;
        default: break;
        }
    }
    if constexpr (__is_same(Op, OpAvg)) {
        const int n = NP > 0 ? NP : nsrc;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < T::kVec; ++j) acc[u][j] = avg_scale<T, Op>(acc[u][j], n);
    }
    const rsrc_t w = make_rsrc(dst + tl.off, tl.nrec);
#pragma unroll
    for (int u = 0; u < U; ++u)
        bstore<kStoreOut>(down_vec<T, Op>(acc[u]), w, (uint32_t)(u * B + threadIdx.x) * 16u);
}

// Element i (scalar path): used for leads and tails shorter than a vector
// and for buffers at different offsets within 16 bytes.  The loads of up to
// 8 sources are issued before they are folded, in source order.
template <class T, class Op, class Src>
__device__ __forceinline__ void reduce_elem(const Src &src, int nsrc, char *dst, size_t i)
{
    typename T::Acc a{};
    for (int p = 0; p < nsrc; p += 8) {
        typename T::Acc x[8];
#pragma unroll
        for (int q = 0; q < 8; ++q)
            if (p + q < nsrc) x[q] = up1<T>(src(p + q), i);
#pragma unroll
        for (int q = 0; q < 8; ++q)
            if (p + q < nsrc) a = p + q == 0 ? x[q] : combine<T, Op>(a, x[q]);
    }
    down1<T, Op>(dst, i, avg_scale<T, Op>(a, nsrc));
}

// The elements of one reduction outside its vectors: the first nl (its lead,
// or 0) and the nt from element tail_at on (its tail, or 0), one per thread
// of the first wavefront, so both are folded by one chain of loads.
template <class T, class Op, class Src>
__device__ __forceinline__ void reduce_ends(const Src &src, int nsrc, char *dst, uint32_t nl,
                                            uint32_t nt, size_t tail_at)
{
    const uint32_t t = threadIdx.x;
    if (t < nl + nt) reduce_elem<T, Op>(src, nsrc, dst, t < nl ? (size_t)t : tail_at + (t - nl));
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Any number of sources at one 16-byte-aligned tile: the first group takes
// up to 8 sources, then groups of 8 and a remainder, all loads of a group in
// flight; fold order 0..nsrc-1.
template <class T, class Op, int U, int B, class Src>
__device__ __forceinline__ void fold_any(typename T::Acc (&acc)[U][T::kVec], const Src &src,
                                         int nsrc, Tile tl)
{
    const int g0 = nsrc < 8 ? nsrc : 8;
    switch (g0) {
    case 1: fold_group<T, Op, 1, U, B, true>(acc, src, 0, tl); break;
    case 2: fold_group<T, Op, 2, U, B, true>(acc, src, 0, tl); break;
    case 3: fold_group<T, Op, 3, U, B, true>(acc, src, 0, tl); break;
    case 4: fold_group<T, Op, 4, U, B, true>(acc, src, 0, tl); break;
    case 5: fold_group<T, Op, 5, U, B, true>(acc, src, 0, tl); break;
    case 6: fold_group<T, Op, 6, U, B, true>(acc, src, 0, tl); break;
    case 7: fold_group<T, Op, 7, U, B, true>(acc, src, 0, tl); break;
    default: fold_group<T, Op, 8, U, B, true>(acc, src, 0, tl); break;
    }
    int p = g0;
    for (; p + 8 <= nsrc; p += 8) fold_group<T, Op, 8, U, B, false>(acc, src, p, tl);
    switch (nsrc - p) {
    case 1: fold_group<T, Op, 1, U, B, false>(acc, src, p, tl); break;
    case 2: fold_group<T, Op, 2, U, B, false>(acc, src, p, tl); break;
    case 3: fold_group<T, Op, 3, U, B, false>(acc, src, p, tl); break;
    case 4: fold_group<T, Op, 4, U, B, false>(acc, src, p, tl); break;
    case 5: fold_group<T, Op, 5, U, B, false>(acc, src, p, tl); break;
    case 6: fold_group<T, Op, 6, U, B, false>(acc, src, p, tl); break;
    case 7: fold_group<T, Op, 7, U, B, false>(acc, src, p, tl); break;
    default: break;
    }
}

// Bytes [s, s+16) of the 32 bytes lo:hi (lo at the lower address), 0 < s < 16.
__device__ __forceinline__ u32x4 bytes_from(u32x4 lo, u32x4 hi, uint32_t s)
{
    const uint32_t w[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    const uint32_t b = s & 3u;
    u32x4 o;
    switch (s >> 2) {
    case 0:
        for (int i = 0; i < 4; ++i) o[i] = __builtin_amdgcn_alignbyte(w[i + 1], w[i], b);
        break;
    case 1:
        for (int i = 0; i < 4; ++i) o[i] = __builtin_amdgcn_alignbyte(w[i + 2], w[i + 1], b);
        break;
    case 2:
        for (int i = 0; i < 4; ++i) o[i] = __builtin_amdgcn_alignbyte(w[i + 3], w[i + 2], b);
        break;
    default:
        for (int i = 0; i < 4; ++i) o[i] = __builtin_amdgcn_alignbyte(w[i + 4], w[i + 3], b);
        break;
    }
    return o;
}

// The 16-byte results of B lanes, lane q's for output bytes [16q, 16q + 16)
// of `base`, where base sits c bytes past a 16-byte boundary (0 < c < 16, a
// multiple of the element size) and `nrec` of the B*16 bytes exist.  Output
// bytes [16q - c, 16q + 16 - c) are lane q-1's last c result bytes and lane
// q's first 16 - c, so every lane but the first of its wavefront takes its
// neighbour's result (a lane shuffle) and stores one aligned 16-byte vector.
// The two chunks cut by a wavefront's ends (16 - c bytes at its first lane,
// c at its last lane with a vector) go out in aligned pieces of the largest
// power of two dividing c, 16 bytes in all, from up to 16 lanes in one store
// instruction.  Every lane of the workgroup must be active.
__device__ __forceinline__ void split_store(u32x4 mine, char *base, uint32_t nrec, uint32_t c)
{
    const uint32_t q = threadIdx.x, l = q & 63u;
    u32x4 prev;
#pragma unroll
    for (int i = 0; i < 4; ++i) prev[i] = __shfl_up(mine[i], 1u, 64);
    if (l != 0)
        bstore<kStoreOut>(bytes_from(prev, mine, 16u - c), make_rsrc(base - c, nrec), 16u * q);
    const uint32_t w0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)(q >> 6)) * 64u;
    const uint32_t nl = nrec / 16u;   // lanes with a vector
    if (w0 >= nl) return;
    const uint32_t last = nl - 1u - w0 < 63u ? nl - 1u - w0 : 63u;
    u32x4 r0, rl;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        r0[i] = (uint32_t)__builtin_amdgcn_readlane((int)mine[i], 0);
        rl[i] = (uint32_t)__builtin_amdgcn_readlane((int)mine[i], (int)last);
    }
    const uint32_t piece = c & (~c + 1u);
    const uint32_t hp = (16u - c) / piece;
    if (l >= 16u / piece) return;
    const bool head = l < hp;
    const uint32_t o = head ? l * piece : 16u - c + (l - hp) * piece;   // byte of the vector
    const uint32_t at = 16u * (w0 + (head ? 0u : last)) + o;             // byte of `base`
    const u32x4 v = head ? r0 : rl;
    const uint32_t d = o >> 2;
    const uint32_t x = d == 0 ? v[0] : d == 1 ? v[1] : d == 2 ? v[2] : v[3];
    const rsrc_t w = make_rsrc(base, nrec);
    switch (piece) {
    case 8: {
        const u32x2 x2 = {x, d == 0 ? v[1] : v[3]};
        __builtin_amdgcn_raw_buffer_store_b64(x2, w, at, 0, kStoreOut);
        break;
    }
    case 4: __builtin_amdgcn_raw_buffer_store_b32(x, w, at, 0, kStoreOut); break;
    case 2:
        __builtin_amdgcn_raw_buffer_store_b16((unsigned short)(x >> (8u * (o & 3u))), w, at, 0,
                                              kStoreOut);
        break;
    default:
        __builtin_amdgcn_raw_buffer_store_b8((unsigned char)(x >> (8u * (o & 3u))), w, at, 0,
                                             kStoreOut);
        break;
    }
}

// One tile of B output vectors when the sources sit at different offsets
// within 16 bytes: the output grid is dst's, output vector q of the tile
// starts at byte lb + off + 16q of dst, which is 16-byte aligned, and of
// every source, where source p's bytes sit s_p into its aligned vectors
// A_p[q], A_p[q+1] (A_p counted from src_p + lb - s_p, which must not lie
// before src_p, and A_p one past the tile must lie inside the source).
// Lane q loads A_p[q] and takes A_p[q+1] from the next lane (a lane
// shuffle; the wavefront's last lane loads it), joining the two with byte
// funnel shifts; sources on the grid skip both.  The loads of up to 8
// sources are in flight before they are folded in source order.  nrec bytes
// of the tile exist.  Every lane of the workgroup must be active.
template <class T, class Op, int B, class Src>
__device__ __forceinline__ void shift_tile(const Src &src, int nsrc, char *dst, size_t lb,
                                           size_t off, uint32_t nrec)
{
    const uint32_t q = threadIdx.x;
    typename T::Acc acc[T::kVec];
    for (int p0 = 0; p0 < nsrc; p0 += 8) {
        u32x4 lo[8], hi[8];
        uint32_t sh[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (p0 + j < nsrc) {
                const char *a = src(p0 + j) + lb;
                sh[j] = (uint32_t)((uintptr_t)a & 15u);
                // vectors q and q+1 of the tile; the range covers one vector
                // past the tile, which exists in every source
                const rsrc_t r = make_rsrc(a - sh[j] + off, nrec + 16u);
                lo[j] = bload<kLoadStream>(r, 16u * q);
                if (sh[j] != 0 && (q & 63u) == 63u) hi[j] = bload<kLoadStream>(r, 16u * q + 16u);
            }
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (p0 + j < nsrc) {
                u32x4 v = lo[j];
                if (sh[j] != 0) {
                    u32x4 nx;
#pragma unroll
                    for (int i = 0; i < 4; ++i) nx[i] = __shfl_down(lo[j][i], 1u, 64);
                    if ((q & 63u) == 63u) nx = hi[j];
                    v = bytes_from(lo[j], nx, sh[j]);
                }
                if (p0 + j == 0) up_vec<T>(v, acc);
                else fold_vec<T, Op>(acc, v);
            }
        }
    }
    if constexpr (__is_same(Op, OpAvg)) {
#pragma unroll
        for (int e = 0; e < T::kVec; ++e) acc[e] = avg_scale<T, Op>(acc[e], nsrc);
    }
    bstore<kStoreOut>(down_vec<T, Op>(acc), make_rsrc(dst + lb + off, nrec), 16u * q);
}

// The lead shift_tile needs for a reduction of `bytes` bytes into dst: dst's
// next 16-byte boundary and one vector more, in elements; 0 when the
// reduction is too short for one vector with a vector after it, or dst is
// not element-aligned (a device descriptor's), which is then folded element
// by element.
template <class T>
__host__ __device__ __forceinline__ uint32_t shift_lead(uintptr_t dst, size_t bytes)
{
    if (dst % T::kSize != 0) return 0u;
    const uint32_t lb = (uint32_t)(((16u - (dst & 15u)) & 15u) + 16u);
    return bytes >= (size_t)lb + 32 ? lb / (uint32_t)T::kSize : 0u;
}

// A tile whose sources sit on 16-byte boundaries (tl.off past each source
// pointer) and whose output dst + tl.off sits c bytes past one: U vectors
// per thread folded as reduce_tile does, then each block of B vectors
// stored realigned (split_store).
template <class T, class Op, int U, int B, class Src>
__device__ __forceinline__ void split_tile(const Src &src, int nsrc, char *dst, Tile tl,
                                           uint32_t c)
{
    typename T::Acc acc[U][T::kVec];
    fold_any<T, Op, U, B>(acc, src, nsrc, tl);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if constexpr (__is_same(Op, OpAvg)) {
#pragma unroll
            for (int j = 0; j < T::kVec; ++j) acc[u][j] = avg_scale<T, Op>(acc[u][j], nsrc);
        }
        const uint32_t start = (uint32_t)u * B * 16u;
        if (start >= tl.nrec) break;
        const uint32_t left = tl.nrec - start;
        split_store(down_vec<T, Op>(acc[u]), dst + tl.off + start,
                    left < (uint32_t)B * 16u ? left : (uint32_t)B * 16u, c);
    }
}

// ------------------------------------------------------ fused P-source --
// dst[i] = fold_p src_p[i] for lead + nvec*kVec + tail elements, every
// pointer at the same offset within 16 bytes: the first `lead` elements
// (fewer than a vector) bring them all to a 16-byte boundary and, like the
// last `tail` ones, are done by one workgroup, scalar; the nvec vectors
// between go in tiles of B*U vectors (the last one ragged, cut by the buffer
// range check).  `head` (a multiple of 16 below 128, at most nvec*16) is the
// byte length of a first, short tile that ends where the first source
// reaches a 128-byte line: the other tiles then start on line boundaries, so
// no line is split between two tiles (whose workgroups, on different XCDs,
// would each fetch it).
template <class T, class Op, int NP, int MAXP, int U, int B>
__global__ __launch_bounds__(B) void reduce_vec_kernel(KernargSrc<MAXP> src, int nsrc, char *dst,
                                                       size_t nvec, uint32_t tail, uint32_t head,
                                                       uint32_t lead)
{
    constexpr uint32_t kTileBytes = (uint32_t)B * U * 16u;
    const size_t vbytes = nvec * 16;
    const size_t lb = (size_t)lead * T::kSize;   // bytes before the first vector
    const uint32_t first = head != 0 ? 1u : 0u;
    const size_t ntiles = first + (vbytes - head + kTileBytes - 1) / kTileBytes;
    for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const bool h = t < first;
        const size_t off = h ? 0 : head + (t - first) * kTileBytes;
        reduce_tile<T, Op, NP, U, B>(src, nsrc, dst,
                                     Tile{lb + off, h ? head : tile_nrec(vbytes, off, kTileBytes)});
    }
    if ((tail | lead) != 0 && blockIdx.x == ntiles % gridDim.x)
        reduce_ends<T, Op>(src, nsrc, dst, lead, tail, lead + nvec * T::kVec);
}

// Any alignment: one element per thread per step.
template <class T, class Op, int B>
__global__ __launch_bounds__(B) void reduce_scalar_kernel(KernargSrc<XRED_MAX_SRC> src, int nsrc,
                                                          char *dst, size_t count)
{
    const size_t stride = (size_t)gridDim.x * B;
    for (size_t i = (size_t)blockIdx.x * B + threadIdx.x; i < count; i += stride)
        reduce_elem<T, Op>(src, nsrc, dst, i);
}

// ------------------------------------------------------------ step-wise --
// The accumulator holds kVec values of T::Acc (4 or 8 bytes) per 16-byte
// input vector, i.e. acc_vecs<T>() 16-byte accumulator vectors, contiguous.
template <class T, class Op, unsigned FLAGS, int U, int B>
__device__ __forceinline__ void step_tile(const char *in, char *acc, char *dst, size_t t,
                                          size_t nvec)
{
    constexpr bool kInit = (FLAGS & XRED_STEP_INIT) != 0, kFinal = (FLAGS & XRED_STEP_FINAL) != 0;
    constexpr int H = acc_vecs<T>();               // accumulator vectors per input vector
    constexpr int PV = acc_per_vec<T>();           // accumulator values per vector
    constexpr uint32_t kTileBytes = (uint32_t)B * U * 16u;
    const size_t off = t * kTileBytes;
    const uint32_t nrec = tile_nrec(nvec * 16, off, kTileBytes);
    const rsrc_t rin = make_rsrc(in + off, nrec);
    const rsrc_t racc = make_rsrc(acc + off * H, nrec * H);
    u32x4 x[U];
    typename T::Acc a[U][T::kVec];
#pragma unroll
    for (int u = 0; u < U; ++u) x[u] = bload<kLoadStream>(rin, (uint32_t)(u * B + threadIdx.x) * 16u);
    if constexpr (!kInit) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int h = 0; h < H; ++h)
                unpack_acc<T>(bload<kLoadKeep>(racc, (uint32_t)((u * B + threadIdx.x) * H + h) * 16u),
                              &a[u][PV * h]);
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if constexpr (kInit) up_vec<T>(x[u], a[u]);
        else fold_vec<T, Op>(a[u], x[u]);
    }
    if constexpr (kFinal) {
        const rsrc_t rdst = make_rsrc(dst + off, nrec);
#pragma unroll
        for (int u = 0; u < U; ++u)
            bstore<kStoreOut>(down_vec<T, Op>(a[u]), rdst, (uint32_t)(u * B + threadIdx.x) * 16u);
    } else {
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int h = 0; h < H; ++h) {
                typename T::Acc f[PV];
#pragma unroll
                for (int j = 0; j < PV; ++j) f[j] = finalize<T, Op>(a[u][PV * h + j]);
                bstore<kStoreKeep>(pack_acc<T>(f), racc,
                                   (uint32_t)((u * B + threadIdx.x) * H + h) * 16u);
            }
        }
    }
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
        a = combine<T, Op>(((const typename T::Acc *)acc)[i], x);
    }
    if constexpr (kFinal)
        down1<T, Op>(dst, i, a);
    else
        ((typename T::Acc *)acc)[i] = finalize<T, Op>(a);
}

// One ReduceCopy step over nvec vectors + tail elements (16 B aligned) or,
// with VEC = false, over count = tail elements of any alignment.
template <class T, class Op, unsigned FLAGS, int U, int B, bool VEC>
__global__ __launch_bounds__(B) void step_kernel(const char *in, char *acc, char *dst, size_t nvec,
                                                 size_t tail)
{
    if constexpr (VEC) {
        constexpr size_t kTile = (size_t)B * U;
        const size_t ntiles = (nvec + kTile - 1) / kTile;
        for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x)
            step_tile<T, Op, FLAGS, U, B>(in, acc, dst, t, nvec);
        if (tail != 0 && blockIdx.x == ntiles % gridDim.x && threadIdx.x < tail)
            step_elem<T, Op, FLAGS>(in, acc, dst, nvec * T::kVec + threadIdx.x);
    } else {
        const size_t stride = (size_t)gridDim.x * B;
        for (size_t i = (size_t)blockIdx.x * B + threadIdx.x; i < tail; i += stride)
            step_elem<T, Op, FLAGS>(in, acc, dst, i);
    }
}

// dst = down(acc): the closing cast of a step-wise sequence.
template <class T, int U, int B, bool VEC>
__global__ __launch_bounds__(B) void acc_cast_kernel(const char *acc, char *dst, size_t nvec,
                                                     size_t tail)
{
    if constexpr (VEC) {
        constexpr int H = acc_vecs<T>();
        constexpr int PV = acc_per_vec<T>();
        constexpr uint32_t kTileBytes = (uint32_t)B * U * 16u;
        const size_t vbytes = nvec * 16;
        const size_t ntiles = (vbytes + kTileBytes - 1) / kTileBytes;
        for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
            const size_t off = t * kTileBytes;
            const uint32_t nrec = tile_nrec(vbytes, off, kTileBytes);
            const rsrc_t racc = make_rsrc(acc + off * H, nrec * H);
            const rsrc_t rdst = make_rsrc(dst + off, nrec);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                typename T::Acc a[T::kVec];
#pragma unroll
                for (int h = 0; h < H; ++h)
                    unpack_acc<T>(
                        bload<kLoadStream>(racc, (uint32_t)((u * B + threadIdx.x) * H + h) * 16u),
                        &a[PV * h]);
                bstore<kStoreOut>(down_vec<T, OpSum>(a), rdst, (uint32_t)(u * B + threadIdx.x) * 16u);
            }
        }
        if (tail != 0 && blockIdx.x == ntiles % gridDim.x && threadIdx.x < tail) {
            const size_t i = nvec * T::kVec + threadIdx.x;
            down1<T, OpSum>(dst, i, ((const typename T::Acc *)acc)[i]);
        }
    } else {
        const size_t stride = (size_t)gridDim.x * B;
        for (size_t i = (size_t)blockIdx.x * B + threadIdx.x; i < tail; i += stride)
            down1<T, OpSum>(dst, i, ((const typename T::Acc *)acc)[i]);
    }
}

}  // namespace xred
