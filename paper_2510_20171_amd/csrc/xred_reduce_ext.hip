// xred_reduce_ext.hip -- fused-reduce kernels for fp64, int8 and uint8.
#include "xred_reduce.hpp"

namespace xred {

hipError_t launch_reduce_ext(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                            char *dst, size_t count, hipStream_t stream)
{
    return reduce_group<TF64, TI8, TU8>(dtype, op, srcs, nsrc, dst, count, stream);
}

}  // namespace xred
