// xred_reduce.hip -- launchers for the fused P-source reduce
// (xred_allreduce_local and xred_reduce_scatter_local).
#include "xred_internal.hpp"
#include "xred_kernels.hpp"

namespace xred {
namespace {

// One 16-byte vector per thread, 512-thread workgroups: 8 KiB tiles of every
// source.  Measured on MI355X against 2 and 4 vectors per thread and 256 or
// 1024 threads; this shape was fastest or within noise of it for P = 8 and
// P = 32, and has the most workgroups for mid-size messages.
constexpr int kU = 1;    // 16-byte vectors per thread per tile
constexpr int kB = 512;  // threads per workgroup

template <class T, class Op, int NP, int MAXP>
hipError_t go_vec(const char *const *srcs, int nsrc, char *dst, size_t count, hipStream_t s)
{
    KernargSrc<MAXP> ks;
    for (int p = 0; p < nsrc; ++p) ks.p[p] = srcs[p];
    for (int p = nsrc; p < MAXP; ++p) ks.p[p] = nullptr;
    const size_t nvec = count / T::kVec;
    const uint32_t tail = (uint32_t)(count % T::kVec);
    constexpr size_t kTile = (size_t)kB * kU;
    const uint64_t tiles = (nvec + kTile - 1) / kTile + (tail ? 1 : 0);
    hipLaunchKernelGGL((reduce_vec_kernel<T, Op, NP, MAXP, kU, kB>), dim3(grid_for(tiles)),
                       dim3(kB), 0, s, ks, nsrc, dst, nvec, tail);
    return hipGetLastError();
}

template <class T, class Op>
hipError_t go(const char *const *srcs, int nsrc, char *dst, size_t count, hipStream_t s)
{
    uintptr_t bits = (uintptr_t)dst;
    for (int p = 0; p < nsrc; ++p) bits |= (uintptr_t)srcs[p];
    if (bits & 15u) {
        KernargSrc<XRED_MAX_SRC> ks;
        for (int p = 0; p < nsrc; ++p) ks.p[p] = srcs[p];
        for (int p = nsrc; p < XRED_MAX_SRC; ++p) ks.p[p] = nullptr;
        hipLaunchKernelGGL((reduce_scalar_kernel<T, Op, kB>), dim3(grid_for((count + kB - 1) / kB)),
                           dim3(kB), 0, s, ks, nsrc, dst, count);
        return hipGetLastError();
    }
    switch (nsrc) {
    case 1: return go_vec<T, Op, 1, 8>(srcs, nsrc, dst, count, s);
    case 2: return go_vec<T, Op, 2, 8>(srcs, nsrc, dst, count, s);
    case 3: return go_vec<T, Op, 3, 8>(srcs, nsrc, dst, count, s);
    case 4: return go_vec<T, Op, 4, 8>(srcs, nsrc, dst, count, s);
    case 5: return go_vec<T, Op, 5, 8>(srcs, nsrc, dst, count, s);
    case 6: return go_vec<T, Op, 6, 8>(srcs, nsrc, dst, count, s);
    case 7: return go_vec<T, Op, 7, 8>(srcs, nsrc, dst, count, s);
    case 8: return go_vec<T, Op, 8, 8>(srcs, nsrc, dst, count, s);
    case 16: return go_vec<T, Op, 16, 16>(srcs, nsrc, dst, count, s);
    case 32: return go_vec<T, Op, 32, 32>(srcs, nsrc, dst, count, s);
    case 64: return go_vec<T, Op, 64, 64>(srcs, nsrc, dst, count, s);
    default: return go_vec<T, Op, 0, XRED_MAX_SRC>(srcs, nsrc, dst, count, s);
    }
}

template <class T>
hipError_t go_op(xred_op op, const char *const *srcs, int nsrc, char *dst, size_t count,
                 hipStream_t s)
{
    switch (op) {
    case XRED_SUM: return go<T, OpSum>(srcs, nsrc, dst, count, s);
    case XRED_PROD: return go<T, OpProd>(srcs, nsrc, dst, count, s);
    case XRED_MAX: return go<T, OpMax>(srcs, nsrc, dst, count, s);
    case XRED_MIN: return go<T, OpMin>(srcs, nsrc, dst, count, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_reduce(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                         char *dst, size_t count, hipStream_t stream)
{
    switch (dtype) {
    case XRED_FLOAT32: return go_op<TF32>(op, srcs, nsrc, dst, count, stream);
    case XRED_BFLOAT16: return go_op<TBF16>(op, srcs, nsrc, dst, count, stream);
    case XRED_INT32: return go_op<TI32>(op, srcs, nsrc, dst, count, stream);
    case XRED_UINT32: return go_op<TU32>(op, srcs, nsrc, dst, count, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace xred
