// xred_batched_ext.hip -- batched-reduce kernels for fp64, int8 and uint8.
#include "xred_batched.hpp"

namespace xred {

hipError_t launch_batched_range_ext(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                    int nitems, const WgStart *d_wg, unsigned grid, hipStream_t stream)
{
    return batched_group<TF64, TI8, TU8>(dtype, op, d_items, nitems, d_wg, grid, stream);
}

hipError_t launch_batched_rr_ext(xred_dtype dtype, xred_op op, const xred_item *d_items,
                              int nitems, const uint32_t *d_tile_start, hipStream_t stream)
{
    return batched_rr_group<TF64, TI8, TU8>(dtype, op, d_items, nitems, d_tile_start, stream);
}

hipError_t launch_batched_table_ext(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                    const uint32_t *d_table, bool narrow, uint64_t ntiles,
                                    hipStream_t stream)
{
    return batched_table_group<TF64, TI8, TU8>(dtype, op, d_items, d_table, narrow,
                                                  ntiles, stream);
}

hipError_t launch_batched_grouped_ext(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                 int nitems, uint32_t ngroups, uint32_t m, unsigned grid,
                                 int wgs_per_cu, hipStream_t stream)
{
    return batched_grouped_group<TF64, TI8, TU8>(dtype, op, d_items, nitems, ngroups, m, grid,
                                          wgs_per_cu, stream);
}

hipError_t launch_batched_queue_ext(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                  int nitems, uint64_t *next, uint64_t *clear, uint64_t *finished,
                                  unsigned grid, int wgs_per_cu, hipStream_t stream)
{
    return batched_queue_group<TF64, TI8, TU8>(dtype, op, d_items, nitems,
                                        QueueCtl{next, clear, finished}, grid, wgs_per_cu,
                                        stream);
}

}  // namespace xred
