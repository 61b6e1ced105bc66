// xred_reduce_fp8.hip -- fused-reduce kernels for fp8 e4m3 and e5m2.
#include "xred_reduce.hpp"

namespace xred {

hipError_t launch_reduce_fp8(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                             char *dst, size_t count, hipStream_t stream)
{
    return reduce_group<TE4M3, TE5M2>(dtype, op, srcs, nsrc, dst, count, stream);
}

}  // namespace xred
