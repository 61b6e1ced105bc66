// xred_step.hip -- launchers for the step-wise ring ReduceCopy
// (xred_reduce_copy_step) and the closing accumulator cast (xred_acc_cast).
//
// A step moves little data (a 1M-element bf16 chunk step reads 6 MiB and
// writes 4 MiB), so launch cost dominates; the launch path is one template
// lookup and one kernel.  The accumulator does not stay in L2 from one step
// to the next: on this multi-XCD part each launch starts with its L2 lines
// invalidated, and the counters show every read of a plain step missing L2
// (6 MiB of misses per launch: the chunk and the whole accumulator), only the
// accumulator's writes hitting the lines the same launch just read.  What can
// carry it between launches is the 256 MB MALL, which sits beyond L2.
#include "xred_dispatch.hpp"
#include "xred_internal.hpp"
#include "xred_kernels.hpp"

namespace xred {
namespace {

constexpr int kU = 2;
constexpr int kB = 256;

template <class T, class Op, unsigned FLAGS>
hipError_t go(const char *in, char *acc, char *dst, size_t count, hipStream_t s)
{
    // acc is touched unless INIT|FINAL; dst only with FINAL.
    constexpr bool kUsesAcc = FLAGS != (XRED_STEP_INIT | XRED_STEP_FINAL);
    constexpr bool kUsesDst = (FLAGS & XRED_STEP_FINAL) != 0;
    uintptr_t bits = (uintptr_t)in;
    if (kUsesAcc) bits |= (uintptr_t)acc;
    if (kUsesDst) bits |= (uintptr_t)dst;
    const bool vec = (bits & 15u) == 0;
    if (vec) {
        const size_t nvec = count / T::kVec;
        const size_t tail = count % T::kVec;
        constexpr size_t kTile = (size_t)kB * kU;
        const uint64_t tiles = (nvec + kTile - 1) / kTile + (tail ? 1 : 0);
        return launch_kernel(step_kernel<T, Op, FLAGS, kU, kB, true>, dim3(grid_for(tiles)),
                             dim3(kB), 0, s, in, acc, dst, nvec, tail);
    }
    return launch_kernel(step_kernel<T, Op, FLAGS, kU, kB, false>,
                         dim3(grid_for((count + kB - 1) / kB)), dim3(kB), 0, s, in, acc, dst,
                         (size_t)0, count);
}

template <class T, class Op>
hipError_t go_flags(unsigned flags, const char *in, char *acc, char *dst, size_t count,
                    hipStream_t s)
{
    switch (flags) {
    case 0: return go<T, Op, 0u>(in, acc, dst, count, s);
    case XRED_STEP_INIT: return go<T, Op, XRED_STEP_INIT>(in, acc, dst, count, s);
    case XRED_STEP_FINAL: return go<T, Op, XRED_STEP_FINAL>(in, acc, dst, count, s);
    default: return go<T, Op, XRED_STEP_INIT | XRED_STEP_FINAL>(in, acc, dst, count, s);
    }
}

template <class T>
hipError_t go_cast(const char *acc, char *dst, size_t count, hipStream_t s)
{
    if ((((uintptr_t)acc | (uintptr_t)dst) & 15u) == 0) {
        const size_t nvec = count / T::kVec;
        const size_t tail = count % T::kVec;
        constexpr size_t kTile = (size_t)kB * kU;
        const uint64_t tiles = (nvec + kTile - 1) / kTile + (tail ? 1 : 0);
        return launch_kernel(acc_cast_kernel<T, kU, kB, true>, dim3(grid_for(tiles)), dim3(kB),
                             0, s, acc, dst, nvec, tail);
    }
    return launch_kernel(acc_cast_kernel<T, kU, kB, false>, dim3(grid_for((count + kB - 1) / kB)),
                         dim3(kB), 0, s, acc, dst, (size_t)0, count);
}

}  // namespace

hipError_t launch_step(xred_dtype dtype, xred_op op, unsigned flags, const char *in, char *acc,
                       char *dst, size_t count, hipStream_t stream)
{
    return with_dtype(dtype, [&](auto t) {
        using T = decltype(t);
        return with_op<T, false>(op, [&](auto o) {
            return go_flags<T, decltype(o)>(flags, in, acc, dst, count, stream);
        });
    });
}

hipError_t launch_acc_cast(xred_dtype dtype, const char *acc, char *dst, size_t count,
                           hipStream_t stream)
{
    return with_dtype(dtype, [&](auto t) { return go_cast<decltype(t)>(acc, dst, count, stream); });
}

}  // namespace xred
