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
// launch).  It also measures the host-to-kernel handoff of a flag in pinned
// host memory (a ping-pong, below).
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#include <chrono>
#include <vector>

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

// ------------------------------------------------------------- handoff --
// The host-to-kernel handoff of a flag in pinned host memory, as a ping-pong:
// the host writes round number r to *ping; a polling lane that sees it
// answers by writing r to *pong, which the host is spinning on.  The host's
// round trip is one host-to-device and one device-to-host handoff.  With
// `relay` set the polling lane (workgroup 0) passes r through a word in
// device memory to a lane of workgroup 1, which answers: the hop the ring
// kernel's poller adds between a flag and the workgroups that wait for it.
// Every wait on both sides ends after `limit` device-clock ticks (device) or
// the same time on the host clock.
namespace {

struct PingPong {
    const uint32_t *ping;   // host pinned, written by the host
    uint32_t *pong;         // host pinned, written by the device
    uint32_t *relay;        // device memory (relay mode)
    uint32_t *failed;       // host pinned: the round a device wait gave up on
    uint32_t *polls;        // device memory: loads of the polled word per round
    uint64_t *seen;         // device memory: ticks from round start to seeing r
};

__device__ __forceinline__ bool wait_word(const uint32_t *w, uint32_t r, bool system,
                                          uint64_t limit, uint32_t *npolls, uint64_t *ticks)
{
    const uint64_t t0 = wall_clock64();
    uint32_t n = 0;
    for (;;) {
        ++n;
        const uint32_t v = system
            ? __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM)
            : __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t t = wall_clock64();
        if (v == r) {
            *npolls = n;
            *ticks = t - t0;
            return true;
        }
        if (t - t0 > limit) return false;
    }
}

__global__ __launch_bounds__(64) void pingpong_kernel(PingPong q, uint32_t rounds, int relay,
                                                      uint64_t limit)
{
    if (threadIdx.x != 0) return;
    for (uint32_t r = 1; r <= rounds; ++r) {
        uint32_t n = 0;
        uint64_t dt = 0;
        if (blockIdx.x == 0) {
            if (!wait_word(q.ping, r, true, limit, &n, &dt)) {
                __hip_atomic_store(q.failed, r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
                return;
            }
            q.polls[r - 1] = n;
            q.seen[r - 1] = dt;
            if (relay)
                __hip_atomic_store(q.relay, r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            else
                __hip_atomic_store(q.pong, r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        } else {
            if (!wait_word(q.relay, r, false, limit, &n, &dt)) return;
            __hip_atomic_store(q.pong, r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
    }
}

}  // namespace

// `rounds` ping-pong rounds (see above) on `stream`; relay: 0 = the polling
// lane answers, 1 = it relays through device memory to a second workgroup.
// Outputs per round (arrays of `rounds`): the host's round trip in us, the
// polling lane's loads of the flag and its device time from the start of the
// round to seeing the flag, in us.  The first round includes the launch.  Returns 0,
// a hipError_t, or -1 if a wait on either side gave up (every wait is
// bounded by limit_ms, so the kernel has always ended when this returns).
extern "C" __attribute__((visibility("default"))) int
xred_ceiling_handoff(int rounds, int relay, int limit_ms, double *rtt_us, uint32_t *polls,
                     double *seen_us, void *stream)
{
    if (rounds < 1 || rounds > (1 << 20) || limit_ms < 1 || !rtt_us || !polls || !seen_us)
        return (int)hipErrorInvalidValue;
    int dev = 0, khz = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
    if (e != hipSuccess) return (int)e;
    if (khz <= 0) return (int)hipErrorInvalidValue;
    char *host = nullptr;
    char *devmem = nullptr;
    const size_t dbytes = 256 + (size_t)rounds * (4 + 8);
    e = hipHostMalloc((void **)&host, 256, hipHostMallocCoherent);
    if (e != hipSuccess) return (int)e;
    e = hipMalloc((void **)&devmem, dbytes);
    if (e != hipSuccess) {
        (void)hipHostFree(host);
        return (int)e;
    }
    memset(host, 0, 256);
    PingPong q;
    q.ping = (const uint32_t *)host;
    q.pong = (uint32_t *)(host + 64);
    q.failed = (uint32_t *)(host + 128);
    q.relay = (uint32_t *)devmem;
    q.seen = (uint64_t *)(devmem + 256);
    q.polls = (uint32_t *)(devmem + 256 + (size_t)rounds * 8);
    const hipStream_t st = (hipStream_t)stream;
    int rc = 0;
    e = hipMemsetAsync(devmem, 0, dbytes, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e == hipSuccess) {
        const uint64_t limit = (uint64_t)khz * (uint64_t)limit_ms;   // kHz * ms = ticks
        hipLaunchKernelGGL(pingpong_kernel, dim3(relay ? 2 : 1), dim3(64), 0, st, q,
                           (uint32_t)rounds, relay, limit);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        volatile uint32_t *ping = (volatile uint32_t *)host;
        const volatile uint32_t *pong = (const volatile uint32_t *)(host + 64);
        const auto give_up = std::chrono::milliseconds(limit_ms);
        for (int r = 1; r <= rounds && rc == 0; ++r) {
            const auto t0 = std::chrono::steady_clock::now();
            __atomic_store_n(ping, (uint32_t)r, __ATOMIC_RELEASE);
            for (uint32_t spins = 0;; ++spins) {
                if (__atomic_load_n(pong, __ATOMIC_ACQUIRE) == (uint32_t)r) break;
                if ((spins & 255u) == 0 && std::chrono::steady_clock::now() - t0 > give_up) {
                    rc = -1;
                    break;
                }
            }
            rtt_us[r - 1] =
                std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0)
                    .count();
        }
        e = hipStreamSynchronize(st);   // every device wait is bounded
    }
    if (e == hipSuccess && __atomic_load_n((uint32_t *)(host + 128), __ATOMIC_ACQUIRE) != 0)
        rc = -1;
    if (e == hipSuccess) {
        std::vector<uint64_t> ticks((size_t)rounds);
        e = hipMemcpy(ticks.data(), q.seen, (size_t)rounds * 8, hipMemcpyDeviceToHost);
        if (e == hipSuccess)
            e = hipMemcpy(polls, q.polls, (size_t)rounds * 4, hipMemcpyDeviceToHost);
        for (int r = 0; r < rounds && e == hipSuccess; ++r)
            seen_us[r] = (double)ticks[(size_t)r] * 1000.0 / (double)khz;
    }
    (void)hipFree(devmem);
    (void)hipHostFree(host);
    return e != hipSuccess ? (int)e : rc;
}

// ------------------------------------------------------------ placement --
// Where the workgroups of a launch on `stream` ran: one word per workgroup,
// xcd << 16 | se << 8 | sh << 4 | cu, from the hardware's XCC_ID register
// and the shader-engine, shader-array and CU fields of its HW_ID register (a
// CU's address within its XCD).  Every workgroup of 1024 threads (at most
// two fit on a CU) sleeps about 10 us before it records, so later
// workgroups find the CUs they could use busy and spread over all of them.
namespace {

constexpr int kPlaceThreads = 1024;

__global__ __launch_bounds__(kPlaceThreads) void placement_kernel(uint32_t *out, unsigned n)
{
#pragma unroll
    for (int i = 0; i < 3; ++i) __builtin_amdgcn_s_sleep(127);
    if (threadIdx.x != 0 || blockIdx.x >= n) return;
    // s_getreg operand: register id | first bit << 6 | (bits - 1) << 11
    const uint32_t hw = __builtin_amdgcn_s_getreg(4 | (0 << 6) | (31 << 11));    // HW_ID
    const uint32_t xcc = __builtin_amdgcn_s_getreg(20 | (0 << 6) | (31 << 11));  // XCC_ID
    const uint32_t cu = (hw >> 8) & 0xF, sh = (hw >> 12) & 1, se = (hw >> 13) & 7;
    out[blockIdx.x] = (xcc & 0xF) << 16 | se << 8 | sh << 4 | cu;
}

}  // namespace

// Runs `grid` workgroups of the placement kernel on `stream` and writes each
// one's XCD and CU to out[0..grid) (device memory).  Stream-ordered; returns
// the hipError_t of the launch.
extern "C" __attribute__((visibility("default"))) int
xred_ceiling_placement(uint32_t *out, unsigned grid, void *stream)
{
    if (out == nullptr || grid == 0) return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(placement_kernel, dim3(grid), dim3(kPlaceThreads), 0,
                       (hipStream_t)stream, out, grid);
    return (int)hipGetLastError();
}
