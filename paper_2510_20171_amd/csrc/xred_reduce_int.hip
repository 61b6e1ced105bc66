// xred_reduce_int.hip -- fused-reduce kernels for int32, uint32, int64 and uint64.
#include "xred_reduce.hpp"

namespace xred {

hipError_t launch_reduce_int(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                            char *dst, size_t count, hipStream_t stream)
{
    return reduce_group<TI32, TU32, TI64, TU64>(dtype, op, srcs, nsrc, dst, count, stream);
}

}  // namespace xred
