// xred_ceiling.hip -- the traffic-only ceiling of the reduce kernels' stream
// mixes: a measuring tool for bench.py, built as its own library
// (libxred_ceiling.so), not part of libxred's interface.
//
// It reads nsrc streams and writes ndst streams of the same length with the
// fused kernel's bandwidth-bound tiles (128-thread workgroups, one 16-byte
// vector per thread and stream, one tile per workgroup, loads issued in
// groups of eight, the next group's in flight while one is combined when
// the source count is 8, 16, 32 or 64, nontemporal loads and device-scope
// stores) and no
// arithmetic beyond an XOR that keeps every load live, with the resident
// waves per CU capped the way the fused launcher caps them (an LDS
// reservation no thread touches).  Swept over caps, the best rate is what
// the memory system gives that mix of streams: the ceiling against which a
// reduce kernel with the same mix is judged (P reads and one write for the
// fused reduce, G reads and G writes for a simulated AllReduce in one
// launch).
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../csrc/xred_kernels.hpp"

namespace {

constexpr int kMaxStreams = 64;
constexpr int kB = 128;
constexpr uint32_t kTileBytes = kB * 16u;

struct Streams {
    const char *p[kMaxStreams];
};

// XOR of NG groups of eight sources (compile time), software pipelined like
// the fused kernel's 16/32/64-source bodies: group g+1's loads are issued
// before group g is combined.  NG == 0: any nsrc, one group at a time.
template <int NG>
__device__ __forceinline__ xred::u32x4 read_all(const Streams &src, int nsrc, size_t off,
                                                uint32_t nrec)
{
    xred::u32x4 x = {0u, 0u, 0u, 0u};
    if constexpr (NG > 0) {
        xred::u32x4 v[2][8];
#pragma unroll
        for (int g = 0; g <= NG; ++g) {
            if (g < NG) {
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    v[g & 1][q] = xred::bload<xred::kLoadStream>(
                        xred::make_rsrc(src.p[8 * g + q] + off, nrec), threadIdx.x * 16u);
            }
            if (g > 0) {
#pragma unroll
                for (int q = 0; q < 8; ++q) x ^= v[(g - 1) & 1][q];
            }
        }
    } else {
        for (int p0 = 0; p0 < nsrc; p0 += 8) {
            xred::u32x4 v[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const bool on = p0 + q < nsrc;
                v[q] = xred::bload<xred::kLoadStream>(
                    xred::make_rsrc((on ? src.p[p0 + q] : src.p[0]) + off, on ? nrec : 0u),
                    threadIdx.x * 16u);
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) x ^= v[q];
        }
    }
    return x;
}

template <int NG>
__global__ __launch_bounds__(kB) void mix_kernel(Streams src, int nsrc, Streams dst, int ndst,
                                                 size_t bytes)
{
    extern __shared__ char occupancy_reservation[];
    (void)occupancy_reservation;
    const size_t ntiles = (bytes + kTileBytes - 1) / kTileBytes;
    for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const size_t off = t * kTileBytes;
        const uint32_t nrec = xred::tile_nrec(bytes, off, kTileBytes);
        const xred::u32x4 x = read_all<NG>(src, nsrc, off, nrec);
        for (int d = 0; d < ndst; ++d)
            xred::bstore<xred::kStoreOut>(x, xred::make_rsrc(dst.p[d] + off, nrec),
                                          threadIdx.x * 16u);
    }
}

template <int NG>
void launch_mix(unsigned grid, size_t reserve, hipStream_t s, const Streams &src, int nsrc,
                const Streams &dst, int ndst, size_t bytes)
{
    hipLaunchKernelGGL(mix_kernel<NG>, dim3(grid), dim3(kB), reserve, s, src, nsrc, dst, ndst,
                       bytes);
}

}  // namespace

// Reads nsrc and writes ndst device buffers of `bytes` each (a multiple of
// 16, all 16-byte aligned), one workgroup per 2 KiB tile, at most
// `waves_per_cu` resident waves per CU (0: no cap).  Stream-ordered on
// `stream`; returns the hipError_t of the launch.
extern "C" __attribute__((visibility("default"))) int
xred_ceiling_mix(const void *const *srcs, int nsrc, void *const *dsts, int ndst, size_t bytes,
                 int waves_per_cu, void *stream)
{
    if (nsrc < 1 || nsrc > kMaxStreams || ndst < 0 || ndst > kMaxStreams || bytes % 16 != 0)
        return (int)hipErrorInvalidValue;
    Streams s{}, d{};
    for (int i = 0; i < nsrc; ++i) s.p[i] = (const char *)srcs[i];
    for (int i = 0; i < ndst; ++i) d.p[i] = (const char *)dsts[i];
    int dev = 0, lds = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev);
    if (e != hipSuccess) return (int)e;
    size_t reserve = 0;
    const int wgs = waves_per_cu / (kB / 64);
    if (wgs > 0 && wgs < 16) reserve = (size_t)(lds / wgs) / 512 * 512;
    const size_t ntiles = (bytes + kTileBytes - 1) / kTileBytes;
    const unsigned grid = (unsigned)(ntiles < 0x7FFFFFFFu ? ntiles : 0x7FFFFFFFu);
    if (grid == 0) return (int)hipSuccess;
    const hipStream_t st = (hipStream_t)stream;
    switch (nsrc % 8 == 0 ? nsrc / 8 : 0) {
    case 1: launch_mix<1>(grid, reserve, st, s, nsrc, d, ndst, bytes); break;
    case 2: launch_mix<2>(grid, reserve, st, s, nsrc, d, ndst, bytes); break;
    case 4: launch_mix<4>(grid, reserve, st, s, nsrc, d, ndst, bytes); break;
    case 8: launch_mix<8>(grid, reserve, st, s, nsrc, d, ndst, bytes); break;
    default: launch_mix<0>(grid, reserve, st, s, nsrc, d, ndst, bytes); break;
    }
    return (int)hipGetLastError();
}
