// xred_internal.hpp -- host-side interfaces between the C ABI layer and the
// kernel launchers.  Every launcher assumes arguments were validated by the
// caller (xred_api.hip) and only sizes the grid and enqueues kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <tuple>
#include <utility>

#include "../../include/xred.h"

namespace xred {

// Launch trace: with XRED_TRACE set to anything but "0" in the environment
// (read once per process) every entry point logs its arguments, every kernel
// launch its kernel, grid, block, LDS bytes, stream and status, and every
// failed call its message, one line each on stderr.  Off, a call costs one
// predictable branch per launch.
bool trace_enabled();
void trace_printf(const char *fmt, ...) __attribute__((format(printf, 1, 2)));
void trace_launch(const void *kernel, dim3 grid, dim3 block, size_t lds, hipStream_t stream,
                  hipError_t status);

// Enqueue kernel<<<grid, block, lds, stream>>>(args...) and return the launch
// status.  hipLaunchKernel takes one pointer per argument; each argument is
// first converted to the kernel's own parameter type.  (The <<<>>> form makes
// two more runtime calls per launch and needs hipGetLastError afterwards,
// about 0.15 us of host time on a launch-bound small call.)
template <class... P, class... A, size_t... I>
hipError_t launch_kernel_impl(void (*kernel)(P...), dim3 grid, dim3 block, size_t lds,
                              hipStream_t stream, std::index_sequence<I...>, A &&...args)
{
    std::tuple<P...> packed(std::forward<A>(args)...);
    void *ptrs[sizeof...(P) > 0 ? sizeof...(P) : 1] = {(void *)&std::get<I>(packed)...};
    const hipError_t e = hipLaunchKernel((const void *)kernel, grid, block, ptrs, lds, stream);
    if (trace_enabled()) trace_launch((const void *)kernel, grid, block, lds, stream, e);
    return e;
}

template <class... P, class... A>
hipError_t launch_kernel(void (*kernel)(P...), dim3 grid, dim3 block, size_t lds,
                         hipStream_t stream, A &&...args)
{
    static_assert(sizeof...(P) == sizeof...(A), "argument count differs from the kernel's");
    return launch_kernel_impl(kernel, grid, block, lds, stream,
                              std::index_sequence_for<P...>{}, std::forward<A>(args)...);
}

// Workgroup budget for one launch on the current device: the number of tiles,
// capped by XRED_MAX_WORKGROUPS when set (a CU-budget knob: it never changes
// results, only how many workgroups share the work).
unsigned grid_for(uint64_t tiles);

// Compute units and LDS bytes per CU of the current device (cached per device).
int device_cus();
int lds_per_cu();

// Index of the current device for per-device caches of kMaxDevicesCached
// entries (0 if the query fails or the index is out of range).
constexpr int kMaxDevicesCached = 64;
int current_device_index();

bool supported(xred_dtype dtype, xred_op op);
size_t elem_size(xred_dtype dtype);

// dst[i] = fold_p srcs[p][i], i < count.  srcs already include any shard offset.
hipError_t launch_reduce(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                         char *dst, size_t count, hipStream_t stream);
// The same per group of element types (each in its own translation unit).
hipError_t launch_reduce_float(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                               char *dst, size_t count, hipStream_t stream);
hipError_t launch_reduce_fp8(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                             char *dst, size_t count, hipStream_t stream);
hipError_t launch_reduce_int(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                             char *dst, size_t count, hipStream_t stream);
hipError_t launch_reduce_ext(xred_dtype dtype, xred_op op, const char *const *srcs, int nsrc,
                             char *dst, size_t count, hipStream_t stream);

hipError_t launch_step(xred_dtype dtype, xred_op op, unsigned flags, const char *in, char *acc,
                       char *dst, size_t count, hipStream_t stream);

hipError_t launch_acc_cast(xred_dtype dtype, const char *acc, char *dst, size_t count,
                           hipStream_t stream);

// Batched reduce.  A tile is batched_tile_elems(dtype) elements of one item.
struct WgStart {
    uint32_t item;        // first item this workgroup works on
    uint32_t ntiles;      // tiles this workgroup processes (over consecutive items)
    uint64_t local_tile;  // first tile within that item
};
static_assert(sizeof(WgStart) == 16, "WgStart layout");
static_assert(sizeof(xred_item) == 32, "xred_item layout");

uint64_t batched_tile_elems(xred_dtype dtype);

// Host descriptors, one workgroup per tile: tile w of the batch (of
// batched_table_tile_elems(dtype) elements) belongs to item table[w], whose
// staged descriptor holds the index of its first tile in `reserved`.  narrow:
// the entries are 16-bit (two per 32-bit word, little-endian; the table is
// padded to 8 bytes), for batches of at most 65536 items.
uint64_t batched_table_tile_elems(xred_dtype dtype);
hipError_t launch_batched_table(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                const uint32_t *d_table, bool narrow, uint64_t ntiles,
                                hipStream_t stream);

// Host-planned: d_items (device copy, srcs pointing to device arrays) and one
// WgStart per workgroup.
hipError_t launch_batched_planned(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                  int nitems, const WgStart *d_wg, unsigned grid,
                                  hipStream_t stream);

// Grid of the host-planned range layout.
unsigned batched_device_grid();

// Round-robin batched kernel (batches of at most batched_rr_max_items()
// items).  d_tile_start: the host plan (nitems + 1 exclusive tile-start
// prefix values), or NULL to have every workgroup compute it from the
// device-resident descriptors.
int batched_rr_max_items();
hipError_t launch_batched_rr(xred_dtype dtype, xred_op op, const xred_item *d_items, int nitems,
                             const uint32_t *d_tile_start, hipStream_t stream);

// Device-resident descriptors, grouped: the batch is cut into ngroups runs of
// at most batched_grouped_max_items() consecutive items, each run is dealt to
// m workgroups tile by tile, and grid (a multiple of m, at least m) is
// m * ngroups or fewer under a CU budget.  wgs_per_cu: workgroups allowed to
// share one CU (the kernel's LDS reservation enforces it; m should be the
// device's CUs times it).
int batched_grouped_max_items();
hipError_t launch_batched_grouped(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                  int nitems, uint32_t ngroups, uint32_t m, unsigned grid,
                                  int wgs_per_cu, hipStream_t stream);

// The batched launchers per group of element types (each in its own
// translation unit).
#define XRED_BATCHED_GROUP(G)                                                                  \
    hipError_t launch_batched_range_##G(xred_dtype dtype, xred_op op,                          \
                                        const xred_item *d_items, int nitems,                  \
                                        const WgStart *d_wg, unsigned grid, hipStream_t s);    \
    hipError_t launch_batched_rr_##G(xred_dtype dtype, xred_op op, const xred_item *d_items,   \
                                     int nitems, const uint32_t *d_tile_start, hipStream_t s); \
    hipError_t launch_batched_table_##G(xred_dtype dtype, xred_op op, const xred_item *d_items, \
                                        const uint32_t *d_table, bool narrow, uint64_t ntiles, \
                                        hipStream_t s);                                        \
    hipError_t launch_batched_grouped_##G(xred_dtype dtype, xred_op op,                        \
                                          const xred_item *d_items, int nitems,                \
                                          uint32_t ngroups, uint32_t m, unsigned grid,         \
                                          int wgs_per_cu, hipStream_t s);                      \
    hipError_t launch_batched_queue_##G(xred_dtype dtype, xred_op op,                          \
                                        const xred_item *d_items, int nitems, uint64_t *next,  \
                                        uint64_t *clear, uint64_t *finished, unsigned grid,    \
                                        int wgs_per_cu, hipStream_t s);
XRED_BATCHED_GROUP(float)
XRED_BATCHED_GROUP(fp8)
XRED_BATCHED_GROUP(int)
XRED_BATCHED_GROUP(ext)
#undef XRED_BATCHED_GROUP

// Device-resident descriptors, queued: a persistent grid takes tiles in
// order from a counter in device memory (see QueueCtl in xred_batched.hpp:
// `next` must be zero at launch; the launch zeroes `clear` if set; with
// `finished` set the launch leaves both counters at zero).  At most
// batched_queue_max_items() items; wgs_per_cu workgroups share one CU (the
// kernel's LDS reservation enforces it).
int batched_queue_max_items();
hipError_t launch_batched_queue(xred_dtype dtype, xred_op op, const xred_item *d_items,
                                int nitems, uint64_t *next, uint64_t *clear, uint64_t *finished,
                                unsigned grid, int wgs_per_cu, hipStream_t stream);

// Workgroups for the round-robin kernel given how many fit on one CU.
unsigned batched_rr_grid(int fit_per_cu);

// All steps of a ring ReduceCopy in one persistent launch (xred_ring_reduce).
uint64_t ring_max_count(xred_dtype dtype);
hipError_t launch_ring(xred_dtype dtype, xred_op op, const char *const *chunks, int nchunks,
                       char *dst, size_t count, const uint32_t *ready, uint32_t epoch,
                       uint64_t timeout_ticks, uint32_t *status, hipStream_t stream);

// 64 bytes of device memory bound to a stream, for kernels whose state
// carries from one launch to the next launch on the same stream (launches on
// one stream run in order, so they may share it): the ring's relay word and
// the batched queue's tile counters.  Each user has kStreamSlots slots per
// device, bound to the first streams that ask, for good (until
// xred_release), and zeroed when first allocated.  acquire() holds the
// user's lock until the object is destroyed, so the caller launches and
// commits under it and the launch count follows the order of the launches.
constexpr int kStreamSlots = 64;
enum StreamSlotUser { kSlotRing = 0, kSlotQueue = 1, kSlotUsers = 2 };
class StreamSlot {
public:
    StreamSlot() = default;
    StreamSlot(const StreamSlot &) = delete;
    StreamSlot &operator=(const StreamSlot &) = delete;
    ~StreamSlot();
    // The slot of `stream` on the current device; false under graph capture
    // (a replay would repeat the captured launch's state), on
    // hipStreamPerThread (one handle for a different stream in every thread),
    // once all slots are bound to other streams, or if allocation failed.
    bool acquire(StreamSlotUser user, hipStream_t stream);
    uint32_t *words = nullptr;   // 16 words of device memory
    uint64_t launches = 0;       // launches committed on the slot before this one
    void commit();               // the launch was enqueued
private:
    void *pool_ = nullptr;
    int index_ = -1;
};

// Frees every user's stream slots on every device (xred_release).
void release_stream_slots();

// A whole AllReduce over nranks simulated ranks on this GPU, one launch per
// step of the ring or halving-doubling schedule (xred_allreduce_sim).
uint64_t sim_chunk(uint64_t count, int nranks);
hipError_t launch_sim(xred_dtype dtype, xred_op op, const char *const *send, char *const *recv,
                      int nranks, size_t count, xred_schedule schedule, hipStream_t stream);

// Device wall-clock ticks per microsecond of the current device.
uint64_t wall_ticks_per_us();

}  // namespace xred
