// xred_reduce_float.hip -- fused-reduce kernels for fp32, bf16 and fp16.
#include "xred_reduce.hpp"

namespace xred {

hipError_t launch_reduce_float(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                              char *dst, size_t count, hipStream_t stream)
{
    return reduce_group<TF32, TBF16, TF16>(dtype, op, srcs, nsrc, dst, count, stream);
}

}  // namespace xred
