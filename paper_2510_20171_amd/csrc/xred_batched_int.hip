// xred_batched_int.hip -- batched-reduce kernels for int32, uint32, int64 and uint64.
#include "xred_batched.hpp"

namespace xred {

hipError_t launch_batched_range_int(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                    int nitems, const WgStart *d_wg, unsigned grid, hipStream_t stream)
{
    return batched_group<TI32, TU32, TI64, TU64>(dtype, op, d_items, nitems, d_wg, grid, stream);
}

hipError_t launch_batched_rr_int(xred_dtype dtype, xred_op op, const xred_item *d_items,
                              int nitems, const uint32_t *d_tile_start, hipStream_t stream)
{
    return batched_rr_group<TI32, TU32, TI64, TU64>(dtype, op, d_items, nitems, d_tile_start, stream);
}

hipError_t launch_batched_table_int(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                    const uint32_t *d_table, bool narrow, uint64_t ntiles,
                                    hipStream_t stream)
{
    return batched_table_group<TI32, TU32, TI64, TU64>(dtype, op, d_items, d_table, narrow,
                                                  ntiles, stream);
}

hipError_t launch_batched_grouped_int(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                 int nitems, uint32_t ngroups, uint32_t m, unsigned grid,
                                 int wgs_per_cu, hipStream_t stream)
{
    return batched_grouped_group<TI32, TU32, TI64, TU64>(dtype, op, d_items, nitems, ngroups, m, grid,
                                          wgs_per_cu, stream);
}

hipError_t launch_batched_queue_int(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                  int nitems, uint64_t *next, uint64_t *clear, uint64_t *finished,
                                  unsigned grid, int wgs_per_cu, hipStream_t stream)
{
    return batched_queue_group<TI32, TU32, TI64, TU64>(dtype, op, d_items, nitems,
                                        QueueCtl{next, clear, finished}, grid, wgs_per_cu,
                                        stream);
}

}  // namespace xred
