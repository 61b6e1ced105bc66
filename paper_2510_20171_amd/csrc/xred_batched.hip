// xred_batched.hip -- many independent reductions in one launch: the entry
// points used by the C ABI, dispatching to the kernels of the element type's
// group (xred_batched_float.hip, xred_batched_fp8.hip, xred_batched_int.hip,
// xred_batched_ext.hip).
#include "xred_batched.hpp"

namespace xred {

uint64_t batched_tile_elems(xred_dtype dtype)
{
    uint64_t n = 0;
    (void)with_dtype(dtype, [&](auto t) {
        n = tile_elems<decltype(t)>();
        return hipSuccess;
    });
    return n;
}

hipError_t launch_batched_planned(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                  int nitems, const WgStart *d_wg, unsigned grid,
                                  hipStream_t stream)
{
    switch (group_of(dtype)) {
    case TypeGroup::kFloat:
        return launch_batched_range_float(dtype, op, d_items, nitems, d_wg, grid, stream);
    case TypeGroup::kFp8:
        return launch_batched_range_fp8(dtype, op, d_items, nitems, d_wg, grid, stream);
    case TypeGroup::kExt:
        return launch_batched_range_ext(dtype, op, d_items, nitems, d_wg, grid, stream);
    default:
        return launch_batched_range_int(dtype, op, d_items, nitems, d_wg, grid, stream);
    }
}

uint64_t batched_table_tile_elems(xred_dtype dtype)
{
    uint64_t n = 0;
    (void)with_dtype(dtype, [&](auto t) {
        n = table_tile_elems<decltype(t)>();
        return hipSuccess;
    });
    return n;
}

hipError_t launch_batched_table(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                const uint32_t *d_table, bool narrow, uint64_t ntiles,
                                hipStream_t stream)
{
    switch (group_of(dtype)) {
    case TypeGroup::kFloat:
        return launch_batched_table_float(dtype, op, d_items, d_table, narrow, ntiles, stream);
    case TypeGroup::kFp8:
        return launch_batched_table_fp8(dtype, op, d_items, d_table, narrow, ntiles, stream);
    case TypeGroup::kExt:
        return launch_batched_table_ext(dtype, op, d_items, d_table, narrow, ntiles, stream);
    default:
        return launch_batched_table_int(dtype, op, d_items, d_table, narrow, ntiles, stream);
    }
}

int batched_rr_max_items() { return kRrMaxItems; }

int batched_grouped_max_items() { return kGrpMaxItems; }

hipError_t launch_batched_grouped(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                  int nitems, uint32_t ngroups, uint32_t m, unsigned grid,
                                  int wgs_per_cu, hipStream_t stream)
{
    switch (group_of(dtype)) {
    case TypeGroup::kFloat:
        return launch_batched_grouped_float(dtype, op, d_items, nitems, ngroups, m, grid,
                                            wgs_per_cu, stream);
    case TypeGroup::kFp8:
        return launch_batched_grouped_fp8(dtype, op, d_items, nitems, ngroups, m, grid,
                                          wgs_per_cu, stream);
    case TypeGroup::kExt:
        return launch_batched_grouped_ext(dtype, op, d_items, nitems, ngroups, m, grid,
                                          wgs_per_cu, stream);
    default:
        return launch_batched_grouped_int(dtype, op, d_items, nitems, ngroups, m, grid,
                                          wgs_per_cu, stream);
    }
}

int batched_queue_max_items() { return kQMaxItems; }

hipError_t launch_batched_queue(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                int nitems, uint64_t *next, uint64_t *clear, uint64_t *finished,
                                unsigned grid, int wgs_per_cu, hipStream_t stream)
{
    switch (group_of(dtype)) {
    case TypeGroup::kFloat:
        return launch_batched_queue_float(dtype, op, d_items, nitems, next, clear, finished, grid,
                                          wgs_per_cu, stream);
    case TypeGroup::kFp8:
        return launch_batched_queue_fp8(dtype, op, d_items, nitems, next, clear, finished, grid,
                                        wgs_per_cu, stream);
    case TypeGroup::kExt:
        return launch_batched_queue_ext(dtype, op, d_items, nitems, next, clear, finished, grid,
                                        wgs_per_cu, stream);
    default:
        return launch_batched_queue_int(dtype, op, d_items, nitems, next, clear, finished, grid,
                                        wgs_per_cu, stream);
    }
}

hipError_t launch_batched_rr(xred_dtype dtype, xred_op op, const xred_item *d_items, int nitems,
                             const uint32_t *d_tile_start, hipStream_t stream)
{
    switch (group_of(dtype)) {
    case TypeGroup::kFloat:
        return launch_batched_rr_float(dtype, op, d_items, nitems, d_tile_start, stream);
    case TypeGroup::kFp8:
        return launch_batched_rr_fp8(dtype, op, d_items, nitems, d_tile_start, stream);
    case TypeGroup::kExt:
        return launch_batched_rr_ext(dtype, op, d_items, nitems, d_tile_start, stream);
    default:
        return launch_batched_rr_int(dtype, op, d_items, nitems, d_tile_start, stream);
    }
}

}  // namespace xred
