// xred_reduce.hpp -- launch templates of the fused P-source reduce
// (xred_allreduce_local and xred_reduce_scatter_local), instantiated per
// group of element types by xred_reduce_{float,fp8,int}.hip so the groups
// compile in parallel.
#pragma once

#include <stdlib.h>

#include <algorithm>

#include "xred_dispatch.hpp"
#include "xred_internal.hpp"
#include "xred_kernels.hpp"

namespace xred {
namespace {

// Three tile shapes:
//
// * Launches that fit on the chip in one round (every tile resident at
//   once) are latency-bound: they use 512-thread workgroups of one 16-byte
//   vector per thread, uncapped, so the whole message is in flight after the
//   fewest workgroup dispatches (8 MiB per source at P=8 bf16: 10.1 us
//   against 10.8 us with 128-thread workgroups, same process and buffers).
// * Up to 8 sources, launches that fit in one round with two vectors per
//   thread (bf16: 8-16 MiB per source) use that shape too, still uncapped:
//   one round of dispatches instead of several rounds of 128-thread
//   workgroups (P=8 bf16, back to back / cold: 12 MiB 15.6 / 21.1 us against
//   17.4 / 22.4; 16 MiB 21.9 / 27.2 against 25.1 / 30.2; P=4 fp32 16 MiB
//   11.1 against 12.1 us; from 20 MiB on the 128-thread shape is as fast).
//   Three, four, six or eight vectors per thread at 20-64 MiB gained at most
//   a few percent and lost 6 % on P=8 fp32 at 32 MiB, so they are not used.
// * Larger launches are bandwidth-bound: 128-thread workgroups with a
//   bounded number of waves per CU.  HBM3E on MI355X delivers the most when
//   a CU keeps a moderate number of loads in flight; more waves than that
//   lower the rate (P=8 bf16, 2^26 elements per source: 168.6 us against
//   190.7 us with uncapped 512-thread workgroups).  Waves per CU -> TB/s on
//   32 MiB per source: P=4 is flat from 16 waves up; P=8 is flat between 8
//   and 16 and falls at full occupancy; P=12 (runtime source count) wants
//   ~16; P=16 ~10; P=32 ~6; P=64 ~4.  The cap is applied by giving each
//   workgroup an LDS reservation it never touches, sized so that only the
//   wanted number of workgroups fit on a CU.
// * Five to eight sources want more loads in flight when each holds several
//   hundred MiB, and when a launch is only a few rounds long (P=8 bf16, one
//   process per setting, best cap and time against the 12-wave cap: 16 MiB
//   per source 24, 25.5 us against 27.4 us back to back and 30.0 against
//   32.0 us cold; 32 MiB 12 (24: +4 % cold); 128 MiB 12; 256 MiB 16, 360 us
//   against 374 us; 512 MiB 24, 830 us against 963 us; 768 MiB 20-24, 1232 us
//   against 1346 us).  16 and 32 sources keep their caps up to 4.4 GB.
constexpr int kU = 1;          // 16-byte vectors per thread per tile
constexpr int kB = 128;        // threads per workgroup, bandwidth-bound launches
constexpr int kBWide = 512;    // threads per workgroup, one-round launches
constexpr int kWideWgsPerCu = 4;   // resident 512-thread workgroups per CU
constexpr int kUWide2 = 2;         // vectors per thread of the second one-round shape (NP <= 8)

// Waves per CU for a compile-time source count (NP = 0, a runtime count: see
// waves_for); 0 = no cap.
// Five and six sources stream best with more waves than seven or eight (bf16
// at 128 MiB per source on two boxes, 12 / 16 / 20 waves: P=5 6.39-6.61 /
// 6.85-7.10 / 6.92-7.08 TB/s, P=6 6.69-6.82 / 6.91-6.98 / 6.90-6.91); two to
// four sources are within noise of uncapped at 16-28 waves.
template <int NP>
constexpr int waves_per_cu()
{
    return NP == 0 ? 12 : NP <= 4 ? 0 : NP == 5 ? 20 : NP == 6 ? 16 : NP <= 8 ? 12
         : NP <= 16 ? 10 : NP <= 32 ? 6 : 4;
}

// The cap of a bandwidth-bound launch with `bytes` per source.  A runtime
// source count takes fewer waves the more sources each thread reads (bf16 at
// 32 MiB per source, 8 / 10 / 12 / 16 waves: 9 sources 6.23-6.26 / 6.22-6.26 /
// 6.37-6.44 / 6.28-6.30 TB/s, 24 sources 6.28-6.29 / 6.29 / 6.26-6.30 /
// 6.06, 48 sources 6.52-6.54 / 6.54 / 6.38-6.40 / 6.10-6.12).
// Eight-bit integers (sixteen 32-bit accumulators per vector) want 16 waves
// for 5-8 sources (P=8 at 128 MiB per source, 12 / 16 waves: uint8 max 6.64-6.66
// / 6.84 TB/s, int8 sum 6.80-6.86 / 6.90-6.91; the other types are best at 12).
template <class T, int NP>
int waves_for(size_t bytes, int nsrc)
{
    if (NP == 0) return nsrc <= 12 ? 12 : nsrc <= 48 ? 10 : 6;
    constexpr bool kByteInt = !T::kFloat && T::kSize == 1;
    if (kByteInt && NP >= 5 && NP <= 8 && bytes > ((size_t)24 << 20) &&
        bytes <= ((size_t)192 << 20))
        return waves_per_cu<NP>() > 16 ? waves_per_cu<NP>() : 16;
    if (NP >= 5 && NP <= 8) {
        if (bytes > ((size_t)384 << 20)) return 24;
        if (bytes > ((size_t)192 << 20)) return waves_per_cu<NP>() > 16 ? waves_per_cu<NP>() : 16;
        if (bytes <= ((size_t)24 << 20)) return 24;
    }
    return waves_per_cu<NP>();
}

// Dynamic LDS that leaves room for `waves` wavefronts per CU (0: no cap).
size_t lds_for_waves(int waves)
{
    static const long force = [] {
        const char *e = getenv("XRED_FUSED_WAVES_PER_CU");
        return e && *e ? strtol(e, nullptr, 10) : 0L;
    }();
    if (force > 0) waves = (int)force;
    if (waves <= 0) return 0;
    const int wgs = waves / (kB / 64);
    if (wgs <= 0 || wgs >= 16) return 0;     // at or beyond the natural occupancy
    return (size_t)(lds_per_cu() / wgs) / 512 * 512;
}

// ------------------------------------------------- split destination --
// Sources at one offset m within 16 bytes, the destination at another (a
// reduce-scatter shard of odd length leaves every rank's shard but some in
// this case): after `lead` elements every source is on a 16-byte boundary
// and is read in vectors as in reduce_vec_kernel, and each tile's results are
// realigned to dst's 16-byte grid and stored in aligned vectors (split_tile).
// P=8 bf16, 16 MiB per source: 51 us element by element, 32 us storing every
// result in 2-byte pieces, 24 us realigned (23.3 us with every buffer
// aligned).  Any source count; the vector path's three shapes: launches
// that fit on the chip in one round take 512-thread workgroups of one vector
// per thread, or (up to 8 sources) two, the others 128-thread workgroups
// under the vector path's occupancy cap.
// reduce_vec_kernel's tiles (U = 1) through split_tile; tail and lead as
// there.
template <class T, class Op, int U, int B>
__global__ __launch_bounds__(B) void reduce_split_kernel(KernargSrc<XRED_MAX_SRC> src, int nsrc,
                                                         char *dst, size_t nvec, uint32_t tail,
                                                         uint32_t head, uint32_t lead, uint32_t c)
{
    constexpr uint32_t kTileBytes = (uint32_t)B * U * 16u;
    const size_t vbytes = nvec * 16;
    const size_t lb = (size_t)lead * T::kSize;
    const uint32_t first = head != 0 ? 1u : 0u;
    const size_t ntiles = first + (vbytes - head + kTileBytes - 1) / kTileBytes;
    for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const bool h = t < first;
        const size_t off = h ? 0 : head + (t - first) * kTileBytes;
        split_tile<T, Op, U, B>(src, nsrc, dst,
                             Tile{lb + off, h ? head : tile_nrec(vbytes, off, kTileBytes)}, c);
    }
    if ((tail | lead) != 0 && blockIdx.x == ntiles % gridDim.x)
        reduce_ends<T, Op>(src, nsrc, dst, lead, tail, lead + nvec * T::kVec);
}

// --------------------------------------------------- shifted sources --
// Sources at different offsets within 16 bytes: the output grid is dst's.
// The first `lead` elements reach dst's next 16-byte boundary and one vector
// more, so every source's aligned base lies inside it, and nvec stops a
// vector short of every source's end; the tiles between are shift_tile's,
// the lead and the tail are folded element by element.  (P=8 x 64M bf16
// with the sources at alternating offsets: 574 us element by element.)
template <class T, class Op, int B>
__global__ __launch_bounds__(B) void reduce_shift_kernel(KernargSrc<XRED_MAX_SRC> src, int nsrc,
                                                         char *dst, size_t nvec, uint32_t tail,
                                                         uint32_t lead)
{
    constexpr uint32_t kTileBytes = (uint32_t)B * 16u;
    const size_t vbytes = nvec * 16;
    const size_t lb = (size_t)lead * T::kSize;
    const size_t ntiles = (vbytes + kTileBytes - 1) / kTileBytes;
    for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const size_t off = t * kTileBytes;
        shift_tile<T, Op, B>(src, nsrc, dst, lb, off, tile_nrec(vbytes, off, kTileBytes));
    }
    if (blockIdx.x == ntiles % gridDim.x)
        reduce_ends<T, Op>(src, nsrc, dst, lead, tail, lead + nvec * T::kVec);
}

// waves_for with the compile-time counts the vector path would pick.
template <class T>
int waves_split(size_t bytes, int nsrc)
{
    switch (nsrc) {
    case 1: return waves_for<T, 1>(bytes, nsrc);
    case 2: return waves_for<T, 2>(bytes, nsrc);
    case 3: return waves_for<T, 3>(bytes, nsrc);
    case 4: return waves_for<T, 4>(bytes, nsrc);
    case 5: return waves_for<T, 5>(bytes, nsrc);
    case 6: return waves_for<T, 6>(bytes, nsrc);
    case 7: return waves_for<T, 7>(bytes, nsrc);
    case 8: return waves_for<T, 8>(bytes, nsrc);
    case 16: return waves_for<T, 16>(bytes, nsrc);
    case 32: return waves_for<T, 32>(bytes, nsrc);
    case 64: return waves_for<T, 64>(bytes, nsrc);
    default: return waves_for<T, 0>(bytes, nsrc);
    }
}

template <class T, class Op>
hipError_t go_split(const char *const *srcs, int nsrc, char *dst, size_t count, uint32_t lead,
                    hipStream_t s)
{
    KernargSrc<XRED_MAX_SRC> ks;
    for (int p = 0; p < nsrc; ++p) ks.p[p] = srcs[p];
    for (int p = nsrc; p < XRED_MAX_SRC; ++p) ks.p[p] = nullptr;
    const size_t nvec = (count - lead) / T::kVec;
    const uint32_t tail = (uint32_t)((count - lead) % T::kVec);
    const size_t mis = ((uintptr_t)srcs[0] + (size_t)lead * T::kSize) & 127u;
    const uint32_t head = (uint32_t)(mis == 0 ? 0 : std::min<size_t>(128 - mis, nvec * 16));
    const size_t hv = head / 16, first = head != 0 ? 1 : 0;
    const uint32_t c = (uint32_t)(((uintptr_t)dst + (size_t)lead * T::kSize) & 15u);
    const uint64_t extra = (tail | lead) ? 1 : 0;
    const uint64_t one_round = (uint64_t)device_cus() * kWideWgsPerCu;
    const uint64_t tiles_wide = first + (nvec - hv + kBWide - 1) / kBWide + extra;
    if (tiles_wide <= one_round)
        return launch_kernel(reduce_split_kernel<T, Op, 1, kBWide>, dim3(grid_for(tiles_wide)),
                             dim3(kBWide), 0, s, ks, nsrc, dst, nvec, tail, head, lead, c);
    constexpr size_t kTileWide2 = (size_t)kBWide * kUWide2;
    const uint64_t tiles_wide2 = first + (nvec - hv + kTileWide2 - 1) / kTileWide2 + extra;
    if (nsrc <= 8 && tiles_wide2 <= one_round)
        return launch_kernel(reduce_split_kernel<T, Op, kUWide2, kBWide>,
                             dim3(grid_for(tiles_wide2)), dim3(kBWide), 0, s, ks, nsrc, dst, nvec,
                             tail, head, lead, c);
    const uint64_t tiles = first + (nvec - hv + kB - 1) / kB + extra;
    return launch_kernel(reduce_split_kernel<T, Op, 1, kB>, dim3(grid_for(tiles)), dim3(kB),
                         lds_for_waves(waves_split<T>(count * T::kSize, nsrc)), s, ks, nsrc, dst,
                         nvec, tail, head, lead, c);
}

template <class T, class Op, int NP, int MAXP>
hipError_t go_vec(const char *const *srcs, int nsrc, char *dst, size_t count, uint32_t lead,
                  hipStream_t s)
{
    KernargSrc<MAXP> ks;
    for (int p = 0; p < nsrc; ++p) ks.p[p] = srcs[p];
    for (int p = nsrc; p < MAXP; ++p) ks.p[p] = nullptr;
    const size_t nvec = (count - lead) / T::kVec;
    const uint32_t tail = (uint32_t)((count - lead) % T::kVec);
    // a short first tile up to the first source's next 128-byte line
    const size_t mis = ((uintptr_t)srcs[0] + (size_t)lead * T::kSize) & 127u;
    const uint32_t head = (uint32_t)(mis == 0 ? 0 : std::min<size_t>(128 - mis, nvec * 16));
    const size_t hv = head / 16, first = head != 0 ? 1 : 0;
    constexpr size_t kTileWide = (size_t)kBWide * kU;
    const uint64_t tiles_wide = first + (nvec - hv + kTileWide - 1) / kTileWide + ((tail | lead) ? 1 : 0);
    const uint64_t one_round = (uint64_t)device_cus() * kWideWgsPerCu;
    if (tiles_wide <= one_round)
        return launch_kernel(reduce_vec_kernel<T, Op, NP, MAXP, kU, kBWide>,
                             dim3(grid_for(tiles_wide)), dim3(kBWide), 0, s, ks, nsrc, dst, nvec,
                             tail, head, lead);
    if constexpr (NP >= 1 && NP <= 8) {
        constexpr size_t kTileWide2 = (size_t)kBWide * kUWide2;
        const uint64_t tiles_wide2 =
            first + (nvec - hv + kTileWide2 - 1) / kTileWide2 + ((tail | lead) ? 1 : 0);
        if (tiles_wide2 <= one_round)
            return launch_kernel(reduce_vec_kernel<T, Op, NP, MAXP, kUWide2, kBWide>,
                                 dim3(grid_for(tiles_wide2)), dim3(kBWide), 0, s, ks, nsrc, dst,
                                 nvec, tail, head, lead);
    }
    constexpr size_t kTile = (size_t)kB * kU;
    const uint64_t tiles = first + (nvec - hv + kTile - 1) / kTile + ((tail | lead) ? 1 : 0);
    return launch_kernel(reduce_vec_kernel<T, Op, NP, MAXP, kU, kB>, dim3(grid_for(tiles)),
                         dim3(kB), lds_for_waves(waves_for<T, NP>(count * T::kSize, nsrc)), s, ks, nsrc,
                         dst, nvec, tail, head, lead);
}

template <class T, class Op>
hipError_t go(const char *const *srcs, int nsrc, char *dst, size_t count, hipStream_t s)
{
    // Pointers all at one offset m within 16 bytes (views at one element
    // offset, a reduce-scatter shard) take the vector path after `lead`
    // elements that bring them to a 16-byte boundary; sources at different
    // offsets read realigned vectors (reduce_shift_kernel) unless the call
    // is too short, which is scalar.
    // Sources at one offset and dst at another take the vector loads with
    // split stores.
    const uintptr_t m = (uintptr_t)srcs[0] & 15u;
    bool common = true;
    for (int p = 1; p < nsrc; ++p) common = common && ((uintptr_t)srcs[p] & 15u) == m;
    const uint32_t lead = m == 0 ? 0u : (uint32_t)((16 - m) / T::kSize);
    if (common && lead < count && ((uintptr_t)dst & 15u) != m)
        return go_split<T, Op>(srcs, nsrc, dst, count, lead, s);
    if (!common) {
        // dst's next 16-byte boundary and one vector more, then vectors up to
        // a vector short of the end (see reduce_shift_kernel)
        const size_t bytes = count * T::kSize;
        const uint32_t slead = shift_lead<T>((uintptr_t)dst, bytes);
        const size_t slb = (size_t)slead * T::kSize;
        if (slead != 0) {
            KernargSrc<XRED_MAX_SRC> ks;
            for (int p = 0; p < nsrc; ++p) ks.p[p] = srcs[p];
            for (int p = nsrc; p < XRED_MAX_SRC; ++p) ks.p[p] = nullptr;
            const size_t nvec = (bytes - slb - 16) / 16;
            const uint32_t tail = (uint32_t)(count - slead - nvec * T::kVec);
            const uint64_t tiles = (nvec + kB - 1) / kB + 1;
            return launch_kernel(reduce_shift_kernel<T, Op, kB>, dim3(grid_for(tiles)), dim3(kB),
                                 lds_for_waves(waves_split<T>(bytes, nsrc)), s, ks, nsrc, dst,
                                 nvec, tail, slead);
        }
    }
    if (!common || lead >= count) {
        KernargSrc<XRED_MAX_SRC> ks;
        for (int p = 0; p < nsrc; ++p) ks.p[p] = srcs[p];
        for (int p = nsrc; p < XRED_MAX_SRC; ++p) ks.p[p] = nullptr;
        return launch_kernel(reduce_scalar_kernel<T, Op, kB>,
                             dim3(grid_for((count + kB - 1) / kB)), dim3(kB), 0, s, ks, nsrc, dst,
                             count);
    }
    constexpr bool kWide = is_core_type<T>() && !__is_same(Op, OpAvg);
    switch (nsrc) {
    case 1: return go_vec<T, Op, 1, 8>(srcs, nsrc, dst, count, lead, s);
    case 2: return go_vec<T, Op, 2, 8>(srcs, nsrc, dst, count, lead, s);
    case 3: return go_vec<T, Op, 3, 8>(srcs, nsrc, dst, count, lead, s);
    case 4: return go_vec<T, Op, 4, 8>(srcs, nsrc, dst, count, lead, s);
    case 5: return go_vec<T, Op, 5, 8>(srcs, nsrc, dst, count, lead, s);
    case 6: return go_vec<T, Op, 6, 8>(srcs, nsrc, dst, count, lead, s);
    case 7: return go_vec<T, Op, 7, 8>(srcs, nsrc, dst, count, lead, s);
    case 8: return go_vec<T, Op, 8, 8>(srcs, nsrc, dst, count, lead, s);
    case 16:
        if constexpr (kWide) return go_vec<T, Op, 16, 16>(srcs, nsrc, dst, count, lead, s);
        break;
    case 32:
        if constexpr (kWide) return go_vec<T, Op, 32, 32>(srcs, nsrc, dst, count, lead, s);
        break;
    case 64:
        if constexpr (kWide) return go_vec<T, Op, 64, 64>(srcs, nsrc, dst, count, lead, s);
        break;
    default: break;
    }
    return go_vec<T, Op, 0, XRED_MAX_SRC>(srcs, nsrc, dst, count, lead, s);
}


// The fused launcher for the element types Ts (one translation unit each).
template <class... Ts>
hipError_t reduce_group(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                        char *dst, size_t count, hipStream_t stream)
{
    return with_dtype_among<Ts...>(dtype, [&](auto t) {
        using T = decltype(t);
        return with_op<T, true>(op, [&](auto o) {
            return go<T, decltype(o)>(srcs, nsrc, dst, count, stream);
        });
    });
}

}  // namespace
}  // namespace xred
