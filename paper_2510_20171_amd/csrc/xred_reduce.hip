// xred_reduce.hip -- the fused P-source reduce (xred_allreduce_local and
// xred_reduce_scatter_local): dispatch to the kernels of the element type's
// group (xred_reduce_float.hip, xred_reduce_fp8.hip, xred_reduce_int.hip,
// xred_reduce_ext.hip).
#include "xred_dispatch.hpp"
#include "xred_internal.hpp"

namespace xred {

hipError_t launch_reduce(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                         char *dst, size_t count, hipStream_t stream)
{
    switch (group_of(dtype)) {
    case TypeGroup::kFloat: return launch_reduce_float(dtype, op, srcs, nsrc, dst, count, stream);
    case TypeGroup::kFp8: return launch_reduce_fp8(dtype, op, srcs, nsrc, dst, count, stream);
    case TypeGroup::kExt: return launch_reduce_ext(dtype, op, srcs, nsrc, dst, count, stream);
    default: return launch_reduce_int(dtype, op, srcs, nsrc, dst, count, stream);
    }
}

}  // namespace xred
