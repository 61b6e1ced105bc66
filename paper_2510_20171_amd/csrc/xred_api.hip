// xred_api.hip -- the C ABI of libxred: argument validation, dispatch to the
// kernel launchers, batch-descriptor staging, status strings.
//
// Every entry point validates all arguments before enqueueing anything, so a
// failed call leaves the stream untouched.  Validation is the only host work
// per call besides the launch itself (the per-message software overhead the
// paper's low-latency path minimises, Section 6.2: no locks, allocation or
// synchronisation on the fused and step-wise paths).
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <cxxabi.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include "xred_internal.hpp"

namespace xred {

bool trace_enabled()
{
    static const bool on = [] {
        const char *v = getenv("XRED_TRACE");
        return v != nullptr && *v != 0 && strcmp(v, "0") != 0;
    }();
    return on;
}

void trace_printf(const char *fmt, ...)
{
    char line[768];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(line, sizeof line, fmt, ap);
    va_end(ap);
    fprintf(stderr, "[xred] %s\n", line);
}

void trace_launch(const void *kernel, dim3 grid, dim3 block, size_t lds, hipStream_t stream,
                  hipError_t status)
{
    const char *raw = hipKernelNameRefByPtr(kernel, stream);
    int dm = -1;
    char *name = raw ? abi::__cxa_demangle(raw, nullptr, nullptr, &dm) : nullptr;
    trace_printf("launch %s grid=%u block=%u lds=%zu stream=%p -> %s",
                 name ? name : raw ? raw : "?", grid.x, block.x, lds, (void *)stream,
                 hipGetErrorName(status));
    free(name);
}

namespace {

constexpr int kMaxDevices = 64;
thread_local char g_err[512];

xred_status fail(xred_status s, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    if (trace_enabled()) trace_printf("failed (status %d): %s", (int)s, g_err);
    return s;
}

xred_status hip_fail(hipError_t e, const char *what)
{
    return fail(XRED_HIP_ERROR, "%s: %s", what, hipGetErrorString(e));
}

bool known_dtype(xred_dtype d) { return d >= XRED_FLOAT32 && d <= XRED_UINT8; }
bool known_op(xred_op o) { return o >= XRED_SUM && o <= XRED_AVG; }

// Entry points whose kernels see only part of the fold (one step, a chunk at
// a time, or a hop) cannot divide by P: AVG is unsupported there.
xred_status check_no_avg(xred_op op, const char *entry)
{
    if (op == XRED_AVG)
        return fail(XRED_UNSUPPORTED, "%s does not support XRED_AVG (it never sees the whole fold)",
                    entry);
    return XRED_SUCCESS;
}

// Accumulator element bytes: uint64 for 64-bit integers, else 4.
size_t acc_size(xred_dtype d)
{
    return d == XRED_INT64 || d == XRED_UINT64 || d == XRED_FLOAT64 ? 8 : 4;
}

// Checks shared by every entry point on dtype and op.
xred_status check_types(xred_dtype dtype, xred_op op)
{
    if (!known_dtype(dtype)) return fail(XRED_INVALID_ARGUMENT, "unknown dtype %d", (int)dtype);
    if (!known_op(op)) return fail(XRED_INVALID_ARGUMENT, "unknown op %d", (int)op);
    if (!supported(dtype, op))
        return fail(XRED_UNSUPPORTED, "dtype %d with op %d is not implemented", (int)dtype,
                    (int)op);
    return XRED_SUCCESS;
}

// A buffer of `bytes` at p: non-NULL, aligned to `align`, no address wrap.
// align: a power of two (an element or accumulator size)
xred_status check_buf(const void *p, size_t bytes, size_t align, const char *name, int index)
{
    const uintptr_t a = (uintptr_t)p;
    if (p == nullptr) return fail(XRED_INVALID_ARGUMENT, "%s[%d] is NULL", name, index);
    if (a & (align - 1)) return fail(XRED_INVALID_ARGUMENT, "%s[%d] is not %zu-byte aligned", name,
                                     index, align);
    if (a + bytes < a) return fail(XRED_INVALID_ARGUMENT, "%s[%d] range wraps the address space",
                                   name, index);
    return XRED_SUCCESS;
}

// Overlap of [a, a+na) and [b, b+nb), other than the identical range when
// `exact_ok`.
bool bad_overlap(const void *a, size_t na, const void *b, size_t nb, bool exact_ok)
{
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    if (exact_ok && x == y && na == nb) return false;
    return x < y + nb && y < x + na;
}

bool mul_overflows(size_t a, size_t b)
{
    size_t r;
    return __builtin_mul_overflow(a, b, &r);
}

int cached_cus[kMaxDevices];
int cached_lds[kMaxDevices];
int cached_ticks[kMaxDevices];

long env_long(const char *name, long dflt)
{
    const char *v = getenv(name);
    if (!v || !*v) return dflt;
    char *end = nullptr;
    const long x = strtol(v, &end, 10);
    return (end && *end == 0 && x > 0) ? x : dflt;
}

// ------------------------------------------------ batch descriptor staging --
// Host-side descriptors are copied into pinned memory, then into device
// memory with one asynchronous copy on the caller's stream.  A ring of slots
// per device is reused once the event recorded after the launch that read a
// slot has completed.
struct Slot {
    void *host = nullptr;
    void *dev = nullptr;
    void *host_dev = nullptr;      // the device's address of `host`
    size_t cap = 0;
    hipEvent_t done = nullptr;
    hipEvent_t copied = nullptr;   // the slot's copy on the side stream has completed
    bool pending = false;
};
constexpr int kSlots = 4;
struct Pool {
    std::mutex mu;
    Slot slot[kSlots];
    unsigned next = 0;
    hipStream_t copy = nullptr;    // side stream for the copies of large batches
    // Stream on which each slot's `done` event is recorded, after waiting for
    // the caller's stream to pass the launch that read the slot.  No event the
    // library keeps is ever recorded on a caller's stream: the caller may
    // destroy its stream at any time, and an event last recorded on a
    // destroyed stream cannot be waited for afterwards (the runtime answered
    // such a wait with a capture error).
    hipStream_t track = nullptr;
};
// Staged batches at least this large are copied on the pool's side stream, so
// the copy overlaps the kernel already running on the caller's stream; smaller
// ones stay on the caller's stream, where the cross-stream wait would cost
// more than the copy.
constexpr size_t kSideCopyBytes = 256 << 10;
// At most this much staged data is read by the kernel from pinned memory.
constexpr size_t kDirectBytes = 64 << 10;
Pool g_pool[kMaxDevices];

void free_slot(Slot &s)
{
    if (s.pending && s.done) (void)hipEventSynchronize(s.done);
    if (s.host) (void)hipHostFree(s.host);
    if (s.dev) (void)hipFree(s.dev);
    s.host = s.dev = s.host_dev = nullptr;
    s.cap = 0;
    s.pending = false;
}

xred_status batched_host(const xred_item *items, int nitems, xred_dtype dtype, xred_op op,
                         hipStream_t stream)
{
    const size_t es = elem_size(dtype);
    const uint64_t te = batched_tile_elems(dtype);
    const uint64_t tt = batched_table_tile_elems(dtype);
    // both are powers of two: tile counts by shifts, not divisions (the
    // plan of a 4096-item batch divides per item several times)
    if (te == 0 || (te & (te - 1)) != 0 || tt == 0 || (tt & (tt - 1)) != 0)
        return fail(XRED_UNSUPPORTED, "batched tile sizes %llu / %llu are not powers of two",
                    (unsigned long long)te, (unsigned long long)tt);
    const int te_log = __builtin_ctzll(te), tt_log = __builtin_ctzll(tt);
    auto tiles_te = [te_log](uint64_t n) { return (n >> te_log) + ((n & ((1ull << te_log) - 1)) != 0); };
    auto tiles_tt = [tt_log](uint64_t n) { return (n >> tt_log) + ((n & ((1ull << tt_log) - 1)) != 0); };
    uint64_t total_tiles = 0, table_tiles = 0, total_ptrs = 0;
    for (int k = 0; k < nitems; ++k) {
        const xred_item &it = items[k];
        if (it.reserved != 0) return fail(XRED_INVALID_ARGUMENT, "items[%d].reserved != 0", k);
        if (it.count == 0) continue;
        if (it.nsrc < 1 || it.nsrc > XRED_MAX_SRC)
            return fail(XRED_INVALID_ARGUMENT, "items[%d].nsrc = %u outside 1..%d", k, it.nsrc,
                        XRED_MAX_SRC);
        if (it.srcs == nullptr) return fail(XRED_INVALID_ARGUMENT, "items[%d].srcs is NULL", k);
        if (mul_overflows(it.count, es))
            return fail(XRED_INVALID_ARGUMENT, "items[%d].count * element size overflows", k);
        const size_t bytes = (size_t)it.count * es;
        xred_status st = check_buf(it.dst, bytes, es, "items.dst", k);
        if (st != XRED_SUCCESS) return st;
        for (uint32_t p = 0; p < it.nsrc; ++p) {
            st = check_buf(it.srcs[p], bytes, es, "items.srcs", k);
            if (st != XRED_SUCCESS) return st;
            if (bad_overlap(it.dst, bytes, it.srcs[p], bytes, true))
                return fail(XRED_ALIAS, "items[%d].dst partially overlaps source %u", k, p);
        }
        total_tiles += tiles_te(it.count);
        table_tiles += tiles_tt(it.count);
        total_ptrs += it.nsrc;
    }
    if (total_tiles == 0) return XRED_SUCCESS;
    if (total_tiles >= 0xFFFFFFFFull)
        return fail(XRED_INVALID_ARGUMENT, "batch has %llu tiles; at most 2^32-2 are supported",
                    (unsigned long long)total_tiles);
    // The descriptors go through staging slots that later calls reuse: a
    // captured copy would replay whatever a later call left there.
    hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
    hipError_t e = hipStreamIsCapturing(stream, &capture);
    if (e != hipSuccess) return hip_fail(e, "hipStreamIsCapturing");
    if (capture != hipStreamCaptureStatusNone)
        return fail(XRED_UNSUPPORTED, "host-side descriptors cannot be captured in a graph "
                                      "(their staging is reused); use XRED_ITEMS_ON_DEVICE");

    // Tile-table layout (one workgroup per tile; the table adds 2 or 4 bytes
    // per tile to the descriptor copy, so batches of very large items, whose
    // table would pass kMaxTableTiles entries (2 MiB), use the layouts after it):
    //     items (reserved = the item's first tile) | item of every tile (u16 up
    //     to 65536 items, else u32; padded to 8 B) | source pointers
    // Round-robin layout (up to batched_rr_max_items() items):
    //     items | tile-start prefix (nitems + 1 u32, padded to 8 B) | source pointers
    // Range layout (more items):
    //     items | per-workgroup starts | source pointers
    constexpr uint64_t kMaxTableTiles = 1u << 19;
    const bool table = table_tiles <= kMaxTableTiles;
    const bool rr = !table && nitems <= batched_rr_max_items();
    // 16-bit tile-list entries while item indices fit (halves the largest part
    // of the staged copy; c4: 830 -> 616 KB)
    const bool narrow = table && nitems <= 65536;
    const unsigned grid = table || rr
                              ? 0u
                              : (unsigned)std::min<uint64_t>(total_tiles, batched_device_grid());
    const size_t items_bytes = sizeof(xred_item) * (size_t)nitems;
    const size_t plan_bytes = table ? ((narrow ? 2 : 4) * (size_t)table_tiles + 7) / 8 * 8
                              : rr  ? (4 * ((size_t)nitems + 1) + 7) / 8 * 8
                                    : sizeof(WgStart) * (size_t)grid;
    const size_t need = items_bytes + plan_bytes + 8 * (size_t)total_ptrs;

    int dev = 0;
    e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(XRED_UNSUPPORTED, "device %d", dev);
    Pool &pool = g_pool[dev];
    std::lock_guard<std::mutex> lock(pool.mu);
    Slot &s = pool.slot[pool.next++ % kSlots];
    if (s.pending) {
        e = hipEventSynchronize(s.done);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize(staging slot)");
        s.pending = false;
    }
    if (s.cap < need) {
        free_slot(s);
        size_t cap = 64 << 10;
        while (cap < need) cap <<= 1;
        // coherent: small batches are read by the kernel straight from the
        // slot, and the host rewrites a slot once its last kernel has ended,
        // so the GPU must not serve those reads from lines it cached earlier
        // (measured no slower than the default allocation for 8-512 items)
        if (hipHostMalloc(&s.host, cap, hipHostMallocCoherent) != hipSuccess) {
            s.host = nullptr;
            return fail(XRED_OUT_OF_MEMORY, "pinned staging of %zu bytes", cap);
        }
        if (hipMalloc(&s.dev, cap) != hipSuccess) {
            (void)hipHostFree(s.host);
            s.host = s.dev = nullptr;
            return fail(XRED_OUT_OF_MEMORY, "device staging of %zu bytes", cap);
        }
        if ((e = hipHostGetDevicePointer(&s.host_dev, s.host, 0)) != hipSuccess) {
            free_slot(s);
            return hip_fail(e, "hipHostGetDevicePointer(staging)");
        }
        s.cap = cap;
    }
    if (!s.done && (e = hipEventCreateWithFlags(&s.done, hipEventDisableTiming)) != hipSuccess)
        return hip_fail(e, "hipEventCreate");
    // A batch of one round of table workgroups (two per CU) and little staged
    // data is read by the kernel straight from the pinned slot: a few host
    // reads per workgroup, paid once in parallel, instead of a copy on the
    // stream before the launch.
    const bool direct = table && table_tiles <= 2 * (uint64_t)device_cus() && need <= kDirectBytes;
    const bool side = !direct && need >= kSideCopyBytes;
    if (side && !s.copied &&
        (e = hipEventCreateWithFlags(&s.copied, hipEventDisableTiming)) != hipSuccess)
        return hip_fail(e, "hipEventCreate");
    if (side && !pool.copy &&
        (e = hipStreamCreateWithFlags(&pool.copy, hipStreamNonBlocking)) != hipSuccess) {
        pool.copy = nullptr;
        return hip_fail(e, "hipStreamCreate(copy stream)");
    }
    if (!pool.track &&
        (e = hipStreamCreateWithFlags(&pool.track, hipStreamNonBlocking)) != hipSuccess) {
        pool.track = nullptr;
        return hip_fail(e, "hipStreamCreate(tracking stream)");
    }

    char *h = (char *)s.host;
    char *d = (char *)(direct ? s.host_dev : s.dev);
    xred_item *h_items = (xred_item *)h;
    const void **h_ptrs = (const void **)(h + items_bytes + plan_bytes);
    const char *d_ptrs = d + items_bytes + plan_bytes;
    uint64_t pos = 0;
    for (int k = 0; k < nitems; ++k) {
        const xred_item &it = items[k];
        xred_item &o = h_items[k];
        o = it;
        if (it.count == 0) {
            o.count = 0;
            o.srcs = nullptr;
            continue;
        }
        o.srcs = (const void *const *)(d_ptrs + 8 * pos);
        for (uint32_t p = 0; p < it.nsrc; ++p) h_ptrs[pos + p] = it.srcs[p];
        pos += it.nsrc;
    }
    if (table && narrow) {
        uint16_t *h_tab = (uint16_t *)(h + items_bytes);
        uint32_t w = 0;
        for (int k = 0; k < nitems; ++k) {
            const uint32_t nt = (uint32_t)tiles_tt(items[k].count);
            h_items[k].reserved = w;
            for (uint32_t t = 0; t < nt; ++t) h_tab[w++] = (uint16_t)k;
        }
        if (w & 1) h_tab[w] = 0;   // the padding half of the last word
    } else if (table) {
        uint32_t *h_tab = (uint32_t *)(h + items_bytes);
        uint32_t w = 0;
        for (int k = 0; k < nitems; ++k) {
            const uint32_t nt = (uint32_t)tiles_tt(items[k].count);
            h_items[k].reserved = w;
            for (uint32_t t = 0; t < nt; ++t) h_tab[w++] = (uint32_t)k;
        }
    } else if (rr) {
        uint32_t *h_pre = (uint32_t *)(h + items_bytes);
        uint64_t acc = 0;
        for (int k = 0; k < nitems; ++k) {
            h_pre[k] = (uint32_t)acc;
            acc += tiles_te(items[k].count);
        }
        h_pre[nitems] = (uint32_t)acc;
    } else {
        // Workgroup b takes global tiles [total*b/grid, total*(b+1)/grid).
        WgStart *h_wg = (WgStart *)(h + items_bytes);
        uint64_t k = 0, k_first = 0;  // item cursor and its first global tile
        for (unsigned b = 0; b < grid; ++b) {
            const uint64_t g0 = (uint64_t)((unsigned __int128)total_tiles * b / grid);
            const uint64_t g1 = (uint64_t)((unsigned __int128)total_tiles * (b + 1) / grid);
            for (;;) {
                const uint64_t nt = tiles_te(items[k].count);
                if (g0 < k_first + nt) break;
                k_first += nt;
                ++k;
            }
            h_wg[b].item = (uint32_t)k;
            h_wg[b].ntiles = (uint32_t)(g1 - g0);
            h_wg[b].local_tile = g0 - k_first;
        }
    }
    if (side) {
        // the slot's device half is free (its last kernel completed above)
        e = hipMemcpyAsync(s.dev, s.host, need, hipMemcpyHostToDevice, pool.copy);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(descriptors)");
        if ((e = hipEventRecord(s.copied, pool.copy)) != hipSuccess ||
            (e = hipStreamWaitEvent(stream, s.copied, 0)) != hipSuccess) {
            (void)hipStreamSynchronize(pool.copy);
            return hip_fail(e, "copy-stream event");
        }
    } else if (!direct) {
        e = hipMemcpyAsync(s.dev, s.host, need, hipMemcpyHostToDevice, stream);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(descriptors)");
    }
    hipError_t le;
    if (table)
        le = launch_batched_table(dtype, op, (const xred_item *)d,
                                  (const uint32_t *)(d + items_bytes), narrow, table_tiles,
                                  stream);
    else if (rr)
        le = launch_batched_rr(dtype, op, (const xred_item *)d, nitems,
                               (const uint32_t *)(d + items_bytes), stream);
    else
        le = launch_batched_planned(dtype, op, (const xred_item *)d, nitems,
                                    (const WgStart *)(d + items_bytes), grid, stream);
    // The copy is enqueued whatever the launch did: the slot stays busy until
    // the stream has passed it.  `done` marks that point on the caller's
    // stream only long enough for the tracking stream to wait for it, and is
    // then recorded again on the tracking stream (the pending wait keeps the
    // first record), so when the call returns it belongs to the library's
    // stream and completes once the caller's stream has passed the launch.
    e = hipEventRecord(s.done, stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(pool.track, s.done, 0);
    if (e == hipSuccess) e = hipEventRecord(s.done, pool.track);
    if (e != hipSuccess) {
        (void)hipStreamSynchronize(stream);
        (void)hipStreamSynchronize(pool.track);
        return hip_fail(e, "staging slot tracking");
    }
    s.pending = true;
    if (le != hipSuccess) return hip_fail(le, "batched launch");
    return XRED_SUCCESS;
}

}  // namespace

// ------------------------------------------------ allocation-free batches --
// The queue kernel's tile counters for xred_batched_reduce_noalloc: words 0
// (next tile) and 1 (workgroups finished) of a fixed array of device memory
// that each GPU the library runs on holds until the process ends (256 bytes,
// zero when the module is loaded; every launch leaves it zero again).  In
// host code the name is only a stand-in for the array: the device address
// is looked up once per device (scratch_on_device) and only that address is
// handed to kernels.
constexpr int kScratchWords = 32;
static __device__ __align__(256) uint64_t scratch[kScratchWords];
uint64_t *g_scratch_dev[kMaxDevices];

// The device address of `scratch` on the current device, looked up on the
// first call there.
xred_status scratch_on_device(uint64_t **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(XRED_UNSUPPORTED, "device %d", dev);
    uint64_t *p = __atomic_load_n(&g_scratch_dev[dev], __ATOMIC_ACQUIRE);
    if (p == nullptr) {
        void *a = nullptr;
        e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (a == nullptr) return fail(XRED_HIP_ERROR, "hipGetSymbolAddress(scratch) gave NULL");
        p = (uint64_t *)a;
        __atomic_store_n(&g_scratch_dev[dev], p, __ATOMIC_RELEASE);
    }
    *out = p;
    return XRED_SUCCESS;
}

// ------------------------------------------------------------ stream slots --
namespace {
struct SlotPool {
    std::mutex mu;
    uint32_t *words = nullptr;                  // kStreamSlots x 64 bytes
    hipStream_t stream[kStreamSlots] = {};
    uint64_t launches[kStreamSlots] = {};
    int bound = 0;
    bool unavailable = false;                   // allocation failed on this device
};
SlotPool g_slots[kMaxDevices][kSlotUsers];
}  // namespace

bool StreamSlot::acquire(StreamSlotUser user, hipStream_t stream)
{
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    int dev = 0;
    if (stream == hipStreamPerThread || hipStreamIsCapturing(stream, &cs) != hipSuccess ||
        cs != hipStreamCaptureStatusNone || hipGetDevice(&dev) != hipSuccess || dev < 0 ||
        dev >= kMaxDevices)
        return false;
    SlotPool &p = g_slots[dev][user];
    p.mu.lock();
    int i = 0;
    while (i < p.bound && p.stream[i] != stream) ++i;
    if (i == p.bound) {
        bool ok = i < kStreamSlots && !p.unavailable;
        if (ok && !p.words) {
            // zeroed on the stream that first needs a slot, and waited for, so
            // the launches of every stream find their slot zeroed
            void *w = nullptr;
            ok = hipMalloc(&w, (size_t)kStreamSlots * 64) == hipSuccess;
            if (ok && (hipMemsetAsync(w, 0, (size_t)kStreamSlots * 64, stream) != hipSuccess ||
                       hipStreamSynchronize(stream) != hipSuccess)) {
                (void)hipFree(w);
                ok = false;
            }
            if (ok) p.words = (uint32_t *)w;
            else p.unavailable = true;
        }
        if (!ok) {
            p.mu.unlock();
            return false;
        }
        p.stream[i] = stream;
        ++p.bound;
    }
    pool_ = &p;
    index_ = i;
    words = p.words + 16 * i;
    launches = p.launches[i];
    return true;
}

void StreamSlot::commit()
{
    if (pool_) ((SlotPool *)pool_)->launches[index_] = ++launches;
}

StreamSlot::~StreamSlot()
{
    if (pool_) ((SlotPool *)pool_)->mu.unlock();
}

void release_stream_slots()
{
    int cur = 0;
    const bool have_dev = hipGetDevice(&cur) == hipSuccess;
    for (int d = 0; d < kMaxDevices; ++d) {
        for (int u = 0; u < kSlotUsers; ++u) {
            SlotPool &p = g_slots[d][u];
            std::lock_guard<std::mutex> lock(p.mu);
            if (!p.words) continue;
            (void)hipSetDevice(d);
            (void)hipDeviceSynchronize();
            (void)hipFree(p.words);
            p.words = nullptr;
            for (int i = 0; i < kStreamSlots; ++i) {
                p.stream[i] = nullptr;
                p.launches[i] = 0;
            }
            p.bound = 0;
        }
    }
    if (have_dev) (void)hipSetDevice(cur);
}

// ------------------------------------------------------- internal helpers --
int device_cus()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
    int c = __atomic_load_n(&cached_cus[dev], __ATOMIC_RELAXED);
    if (c <= 0) {
        if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            c <= 0)
            c = 256;
        __atomic_store_n(&cached_cus[dev], c, __ATOMIC_RELAXED);
    }
    return c;
}

int lds_per_cu()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 160 * 1024;
    int v = __atomic_load_n(&cached_lds[dev], __ATOMIC_RELAXED);
    if (v <= 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) !=
                hipSuccess ||
            v <= 0)
            v = 160 * 1024;
        __atomic_store_n(&cached_lds[dev], v, __ATOMIC_RELAXED);
    }
    return v;
}

int current_device_index()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevicesCached) return 0;
    return dev;
}

// Workgroup budget: 0 = none.  Set by xred_set_max_workgroups (or the
// XRED_MAX_WORKGROUPS environment variable at load); read on every launch.
std::atomic<unsigned> g_max_workgroups{(unsigned)env_long("XRED_MAX_WORKGROUPS", 0)};

// Device-descriptor batches: items per run and workgroups per CU of the
// grouped kernel (measured on the 4096-item log-uniform batch: 32 / 64 / 96 /
// 128 items per run 5.44-5.50 / 5.69-5.70 / 5.49-5.51 / 5.36-5.38 TB/s; 64
// also best on equal items), and workgroups per CU of the queue kernel (one:
// a second widens the window of tiles being read, 1265 against 1301 us).
constexpr int kGroupedRunItems = 64;
constexpr int kGroupedWgsPerCu = 2;
constexpr int kQueueWgsPerCu = 1;

unsigned grid_for(uint64_t tiles)
{
    const unsigned cap = g_max_workgroups.load(std::memory_order_relaxed);
    uint64_t g = (cap != 0 && tiles > cap) ? cap : tiles;
    if (g > 0x7FFFFFFFull) g = 0x7FFFFFFFull;
    return g == 0 ? 1u : (unsigned)g;
}

unsigned batched_device_grid()
{
    static const long per_cu = env_long("XRED_BATCH_WG_PER_CU", 16);
    return grid_for((uint64_t)device_cus() * (uint64_t)per_cu);
}

// Device-resident descriptors, more than one run of items.  Batches of one
// run keep the round-robin kernel: within a run the split is fixed, and the
// round-robin kernel's larger tiles stream large items faster (64 items of
// 8 MiB per source: 5.0 against 4.8 TB/s).  Grouped kernel: runs of
// kGroupedRunItems consecutive items, each dealt to the workgroups that fit on
// the chip at once; under a CU budget, fewer workgroups per run and fewer runs
// at a time.
hipError_t batched_device(const xred_item *items, int nitems, xred_dtype dtype, xred_op op,
                          hipStream_t stream)
{
    // The queue kernel, with the two tile counters of the stream's slot: the
    // launch takes tiles from counter (launches % 2), zeroed by the launch
    // before it on the stream (or when the slot was created), and zeroes the
    // other one for the launch after it.
    if (nitems <= batched_queue_max_items()) {
        StreamSlot slot;
        if (slot.acquire(kSlotQueue, stream)) {
            uint64_t *c = (uint64_t *)slot.words;
            const int par = (int)(slot.launches & 1);
            const unsigned grid = grid_for((uint64_t)device_cus() * kQueueWgsPerCu);
            const hipError_t e = launch_batched_queue(dtype, op, items, nitems, c + par,
                                                      c + (par ^ 1), nullptr, grid,
                                                      kQueueWgsPerCu, stream);
            if (e == hipSuccess) slot.commit();
            return e;
        }
    }
    // Under graph capture (a replay would repeat the captured counter), past
    // the queue's item limit, or without a slot: the stateless grouped kernel.
    const uint64_t per_run =
        (uint64_t)std::min(kGroupedRunItems, batched_grouped_max_items());   // LDS prefix size
    const uint64_t ngroups = ((uint64_t)nitems + per_run - 1) / per_run;
    const unsigned cap = g_max_workgroups.load(std::memory_order_relaxed);
    uint64_t m = (uint64_t)device_cus() * kGroupedWgsPerCu;
    if (cap != 0 && m > cap) m = cap;
    const uint64_t max_sets = (cap != 0 ? (uint64_t)cap : 0x7FFFFFFFull) / m;
    const uint64_t sets = ngroups < max_sets ? ngroups : max_sets;
    return launch_batched_grouped(dtype, op, items, nitems, (uint32_t)ngroups, (uint32_t)m,
                                  (unsigned)(m * sets), kGroupedWgsPerCu, stream);
}

unsigned batched_rr_grid(int fit_per_cu)
{
    static const long per_cu = env_long("XRED_RR_WG_PER_CU", 0);
    return grid_for((uint64_t)device_cus() * (uint64_t)(per_cu > 0 ? per_cu : fit_per_cu));
}

uint64_t wall_ticks_per_us()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 100;
    int t = __atomic_load_n(&cached_ticks[dev], __ATOMIC_RELAXED);
    if (t <= 0) {
        int khz = 0;
        if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
            khz < 1000)
            t = 100;   // 100 MHz, the usual device wall-clock rate
        else
            t = khz / 1000;
        __atomic_store_n(&cached_ticks[dev], t, __ATOMIC_RELAXED);
    }
    return (uint64_t)t;
}

bool supported(xred_dtype dtype, xred_op op)
{
    const bool is_float = dtype == XRED_FLOAT32 || dtype == XRED_BFLOAT16 ||
                          dtype == XRED_FLOAT16 || dtype == XRED_FP8_E4M3 ||
                          dtype == XRED_FP8_E5M2 || dtype == XRED_FLOAT64;
    return known_dtype(dtype) && known_op(op) && (op != XRED_AVG || is_float);
}

size_t elem_size(xred_dtype dtype)
{
    switch (dtype) {
    case XRED_FLOAT32: case XRED_INT32: case XRED_UINT32: return 4;
    case XRED_BFLOAT16: case XRED_FLOAT16: return 2;
    case XRED_INT64: case XRED_UINT64: case XRED_FLOAT64: return 8;
    case XRED_FP8_E4M3: case XRED_FP8_E5M2: case XRED_INT8: case XRED_UINT8: return 1;
    default: return 0;
    }
}

}  // namespace xred

using namespace xred;

extern "C" {

XRED_API xred_status xred_allreduce_local(const void *const *srcs, int nsrc, void *dst,
                                          size_t count, xred_dtype dtype, xred_op op,
                                          void *hip_stream)
{
    if (trace_enabled())
        trace_printf("xred_allreduce_local nsrc=%d count=%zu dtype=%d op=%d stream=%p", nsrc,
                     count, (int)dtype, (int)op, hip_stream);
    if (nsrc < 1 || nsrc > XRED_MAX_SRC)
        return fail(XRED_INVALID_ARGUMENT, "nsrc = %d outside 1..%d", nsrc, XRED_MAX_SRC);
    xred_status st = check_types(dtype, op);
    if (st != XRED_SUCCESS) return st;
    if (count == 0) return XRED_SUCCESS;
    if (srcs == nullptr) return fail(XRED_INVALID_ARGUMENT, "srcs is NULL");
    const size_t es = elem_size(dtype);
    if (mul_overflows(count, es)) return fail(XRED_INVALID_ARGUMENT, "count * size overflows");
    const size_t bytes = count * es;
    if ((st = check_buf(dst, bytes, es, "dst", 0)) != XRED_SUCCESS) return st;
    for (int p = 0; p < nsrc; ++p) {
        if ((st = check_buf(srcs[p], bytes, es, "srcs", p)) != XRED_SUCCESS) return st;
        if (bad_overlap(dst, bytes, srcs[p], bytes, true))
            return fail(XRED_ALIAS, "dst partially overlaps srcs[%d]", p);
    }
    const hipError_t e = launch_reduce(dtype, op, (const char *const *)srcs, nsrc, (char *)dst,
                                       count, (hipStream_t)hip_stream);
    return e == hipSuccess ? XRED_SUCCESS : hip_fail(e, "reduce launch");
}

XRED_API xred_status xred_reduce_scatter_local(const void *const *srcs, int nsrc, int rank,
                                               void *dst, size_t recvcount, xred_dtype dtype,
                                               xred_op op, void *hip_stream)
{
    if (trace_enabled())
        trace_printf("xred_reduce_scatter_local nsrc=%d rank=%d recvcount=%zu dtype=%d op=%d "
                     "stream=%p", nsrc, rank, recvcount, (int)dtype, (int)op, hip_stream);
    if (nsrc < 1 || nsrc > XRED_MAX_SRC)
        return fail(XRED_INVALID_ARGUMENT, "nsrc = %d outside 1..%d", nsrc, XRED_MAX_SRC);
    if (rank < 0 || rank >= nsrc)
        return fail(XRED_INVALID_ARGUMENT, "rank = %d outside [0, %d)", rank, nsrc);
    xred_status st = check_types(dtype, op);
    if (st != XRED_SUCCESS) return st;
    if (recvcount == 0) return XRED_SUCCESS;
    if (srcs == nullptr) return fail(XRED_INVALID_ARGUMENT, "srcs is NULL");
    const size_t es = elem_size(dtype);
    if (mul_overflows(recvcount, es) || mul_overflows(recvcount * es, (size_t)nsrc))
        return fail(XRED_INVALID_ARGUMENT, "nsrc * recvcount * size overflows");
    const size_t shard = recvcount * es;
    if ((st = check_buf(dst, shard, es, "dst", 0)) != XRED_SUCCESS) return st;
    const char *slices[XRED_MAX_SRC];
    for (int p = 0; p < nsrc; ++p) {
        if ((st = check_buf(srcs[p], shard * (size_t)nsrc, es, "srcs", p)) != XRED_SUCCESS)
            return st;
        slices[p] = (const char *)srcs[p] + shard * (size_t)rank;
        if (bad_overlap(dst, shard, slices[p], shard, true))
            return fail(XRED_ALIAS, "dst partially overlaps the slice read from srcs[%d]", p);
    }
    const hipError_t e =
        launch_reduce(dtype, op, slices, nsrc, (char *)dst, recvcount, (hipStream_t)hip_stream);
    return e == hipSuccess ? XRED_SUCCESS : hip_fail(e, "reduce launch");
}

XRED_API xred_status xred_reduce_copy_step(const void *in, void *acc, void *dst, size_t count,
                                           xred_dtype dtype, xred_op op, unsigned flags,
                                           void *hip_stream)
{
    if (trace_enabled())
        trace_printf("xred_reduce_copy_step count=%zu dtype=%d op=%d flags=%u stream=%p", count,
                     (int)dtype, (int)op, flags, hip_stream);
    if (flags & ~(unsigned)(XRED_STEP_INIT | XRED_STEP_FINAL))
        return fail(XRED_INVALID_ARGUMENT, "unknown flag bits 0x%x", flags);
    xred_status st = check_types(dtype, op);
    if (st != XRED_SUCCESS) return st;
    if ((st = check_no_avg(op, "xred_reduce_copy_step")) != XRED_SUCCESS) return st;
    if (count == 0) return XRED_SUCCESS;
    const size_t es = elem_size(dtype), as = acc_size(dtype);
    if (mul_overflows(count, as)) return fail(XRED_INVALID_ARGUMENT, "count * %zu overflows", as);
    const size_t bytes = count * es, acc_bytes = count * as;
    const bool uses_acc = flags != (XRED_STEP_INIT | XRED_STEP_FINAL);
    const bool uses_dst = (flags & XRED_STEP_FINAL) != 0;
    if ((st = check_buf(in, bytes, es, "in", 0)) != XRED_SUCCESS) return st;
    if (uses_acc) {
        if ((st = check_buf(acc, acc_bytes, as, "acc", 0)) != XRED_SUCCESS) return st;
        if (bad_overlap(acc, acc_bytes, in, bytes, false))
            return fail(XRED_ALIAS, "acc overlaps in");
    }
    if (uses_dst) {
        if ((st = check_buf(dst, bytes, es, "dst", 0)) != XRED_SUCCESS) return st;
        if (bad_overlap(dst, bytes, in, bytes, true))
            return fail(XRED_ALIAS, "dst partially overlaps in");
        if (uses_acc && bad_overlap(dst, bytes, acc, acc_bytes, false))
            return fail(XRED_ALIAS, "dst overlaps acc");
    }
    const hipError_t e = launch_step(dtype, op, flags, (const char *)in, (char *)acc, (char *)dst,
                                     count, (hipStream_t)hip_stream);
    return e == hipSuccess ? XRED_SUCCESS : hip_fail(e, "step launch");
}

XRED_API xred_status xred_acc_cast(const void *acc, void *dst, size_t count, xred_dtype dtype,
                                   void *hip_stream)
{
    if (trace_enabled())
        trace_printf("xred_acc_cast count=%zu dtype=%d stream=%p", count, (int)dtype, hip_stream);
    xred_status st = check_types(dtype, XRED_SUM);
    if (st != XRED_SUCCESS) return st;
    if (count == 0) return XRED_SUCCESS;
    const size_t es = elem_size(dtype), as = acc_size(dtype);
    if (mul_overflows(count, as)) return fail(XRED_INVALID_ARGUMENT, "count * %zu overflows", as);
    if ((st = check_buf(acc, count * as, as, "acc", 0)) != XRED_SUCCESS) return st;
    if ((st = check_buf(dst, count * es, es, "dst", 0)) != XRED_SUCCESS) return st;
    if (bad_overlap(acc, count * as, dst, count * es, false))
        return fail(XRED_ALIAS, "dst overlaps acc");
    const hipError_t e =
        launch_acc_cast(dtype, (const char *)acc, (char *)dst, count, (hipStream_t)hip_stream);
    return e == hipSuccess ? XRED_SUCCESS : hip_fail(e, "cast launch");
}

XRED_API xred_status xred_batched_reduce(const xred_item *items, int nitems, xred_dtype dtype,
                                         xred_op op, unsigned flags, void *hip_stream)
{
    if (trace_enabled())
        trace_printf("xred_batched_reduce nitems=%d dtype=%d op=%d flags=%u stream=%p", nitems,
                     (int)dtype, (int)op, flags, hip_stream);
    if (nitems < 0) return fail(XRED_INVALID_ARGUMENT, "nitems = %d", nitems);
    if (flags & ~(unsigned)XRED_ITEMS_ON_DEVICE)
        return fail(XRED_INVALID_ARGUMENT, "unknown flag bits 0x%x", flags);
    xred_status st = check_types(dtype, op);
    if (st != XRED_SUCCESS) return st;
    if (nitems == 0) return XRED_SUCCESS;
    if (items == nullptr) return fail(XRED_INVALID_ARGUMENT, "items is NULL");
    if (flags & XRED_ITEMS_ON_DEVICE) {
        if ((uintptr_t)items % alignof(xred_item))
            return fail(XRED_INVALID_ARGUMENT, "items is not %zu-byte aligned", alignof(xred_item));
        const hipError_t e =
            nitems <= kGroupedRunItems
                ? launch_batched_rr(dtype, op, items, nitems, nullptr, (hipStream_t)hip_stream)
                : batched_device(items, nitems, dtype, op, (hipStream_t)hip_stream);
        return e == hipSuccess ? XRED_SUCCESS : hip_fail(e, "batched launch");
    }
    return batched_host(items, nitems, dtype, op, (hipStream_t)hip_stream);
}

XRED_API xred_status xred_batched_reduce_noalloc(const xred_item *items, int nitems,
                                                 xred_dtype dtype, xred_op op, void *hip_stream)
{
    if (trace_enabled())
        trace_printf("xred_batched_reduce_noalloc nitems=%d dtype=%d op=%d stream=%p", nitems,
                     (int)dtype, (int)op, hip_stream);
    if (nitems < 0) return fail(XRED_INVALID_ARGUMENT, "nitems = %d", nitems);
    xred_status st = check_types(dtype, op);
    if (st != XRED_SUCCESS) return st;
    if (nitems == 0) return XRED_SUCCESS;
    if (items == nullptr) return fail(XRED_INVALID_ARGUMENT, "items is NULL");
    if ((uintptr_t)items % alignof(xred_item))
        return fail(XRED_INVALID_ARGUMENT, "items is not %zu-byte aligned", alignof(xred_item));
    if (nitems > batched_queue_max_items())
        return fail(XRED_UNSUPPORTED,
                    "nitems = %d: xred_batched_reduce_noalloc plans at most %d items on chip",
                    nitems, batched_queue_max_items());
    uint64_t *sc = nullptr;
    if ((st = scratch_on_device(&sc)) != XRED_SUCCESS) return st;
    // counters sc[0] (next tile) and sc[1] (workgroups finished): zero at
    // launch, returned to zero by the launch's last workgroup
    const unsigned grid = grid_for((uint64_t)device_cus() * kQueueWgsPerCu);
    const hipError_t e = launch_batched_queue(dtype, op, items, nitems, sc, nullptr, sc + 1, grid,
                                              kQueueWgsPerCu, (hipStream_t)hip_stream);
    return e == hipSuccess ? XRED_SUCCESS : hip_fail(e, "batched launch");
}

XRED_API xred_status xred_ring_reduce(const void *const *chunks, int nchunks, void *dst,
                                      size_t count, xred_dtype dtype, xred_op op,
                                      const uint32_t *ready, uint32_t epoch, uint64_t timeout_us,
                                      uint32_t *status, void *hip_stream)
{
    if (trace_enabled())
        trace_printf("xred_ring_reduce nchunks=%d count=%zu dtype=%d op=%d flags=%s stream=%p",
                     nchunks, count, (int)dtype, (int)op, ready ? "yes" : "no", hip_stream);
    if (nchunks < 1 || nchunks > XRED_MAX_SRC)
        return fail(XRED_INVALID_ARGUMENT, "nchunks = %d outside 1..%d", nchunks, XRED_MAX_SRC);
    xred_status st = check_types(dtype, op);
    if (st != XRED_SUCCESS) return st;
    if ((st = check_no_avg(op, "xred_ring_reduce")) != XRED_SUCCESS) return st;
    if (count == 0) return XRED_SUCCESS;
    if (chunks == nullptr) return fail(XRED_INVALID_ARGUMENT, "chunks is NULL");
    const size_t es = elem_size(dtype);
    if (mul_overflows(count, es)) return fail(XRED_INVALID_ARGUMENT, "count * size overflows");
    const size_t bytes = count * es;
    if ((st = check_buf(dst, bytes, es, "dst", 0)) != XRED_SUCCESS) return st;
    uintptr_t diff = 0;   // bits in which some chunk's address differs from the first's
    for (int p = 0; p < nchunks; ++p) {
        if ((st = check_buf(chunks[p], bytes, es, "chunks", p)) != XRED_SUCCESS) return st;
        if (bad_overlap(dst, bytes, chunks[p], bytes, true))
            return fail(XRED_ALIAS, "dst partially overlaps chunks[%d]", p);
        diff |= (uintptr_t)chunks[p] ^ (uintptr_t)chunks[0];
    }
    if (diff & 15u)
        return fail(XRED_UNSUPPORTED,
                    "xred_ring_reduce needs every chunk at one offset within 16 bytes");
    if (ready != nullptr && ((uintptr_t)ready & 3u))
        return fail(XRED_INVALID_ARGUMENT, "ready is not 4-byte aligned");
    if (status != nullptr && ((uintptr_t)status & 3u))
        return fail(XRED_INVALID_ARGUMENT, "status is not 4-byte aligned");
    if (count > ring_max_count(dtype))
        return fail(XRED_UNSUPPORTED, "count %zu exceeds the on-chip accumulator capacity %llu",
                    count, (unsigned long long)ring_max_count(dtype));
    if (timeout_us == 0) timeout_us = 1000000;
    if (timeout_us > 60000000ull) timeout_us = 60000000ull;
    const hipError_t e =
        launch_ring(dtype, op, (const char *const *)chunks, nchunks, (char *)dst, count, ready,
                    epoch, timeout_us * wall_ticks_per_us(), status, (hipStream_t)hip_stream);
    return e == hipSuccess ? XRED_SUCCESS : hip_fail(e, "ring launch");
}

XRED_API size_t xred_ring_max_count(xred_dtype dtype)
{
    return known_dtype(dtype) ? (size_t)ring_max_count(dtype) : 0;
}

XRED_API xred_status xred_allreduce_sim(const void *const *sendbufs, void *const *recvbufs,
                                        int nranks, size_t count, xred_dtype dtype, xred_op op,
                                        xred_schedule schedule, void *hip_stream)
{
    if (trace_enabled())
        trace_printf("xred_allreduce_sim nranks=%d count=%zu dtype=%d op=%d schedule=%d "
                     "stream=%p", nranks, count, (int)dtype, (int)op, (int)schedule, hip_stream);
    if (nranks < 1 || nranks > XRED_MAX_SRC)
        return fail(XRED_INVALID_ARGUMENT, "nranks = %d outside 1..%d", nranks, XRED_MAX_SRC);
    if (schedule < XRED_SCHEDULE_RING || schedule > XRED_SCHEDULE_RHD_ONE_LAUNCH)
        return fail(XRED_INVALID_ARGUMENT, "unknown schedule %d", (int)schedule);
    const bool rhd = schedule == XRED_SCHEDULE_RHD || schedule == XRED_SCHEDULE_RHD_ONE_LAUNCH;
    if (rhd && (nranks & (nranks - 1)) != 0)
        return fail(XRED_INVALID_ARGUMENT, "halving-doubling needs a power-of-two nranks, not %d",
                    nranks);
    xred_status st = check_types(dtype, op);
    if (st != XRED_SUCCESS) return st;
    if ((st = check_no_avg(op, "xred_allreduce_sim")) != XRED_SUCCESS) return st;
    if (count == 0) return XRED_SUCCESS;
    if (sendbufs == nullptr || recvbufs == nullptr)
        return fail(XRED_INVALID_ARGUMENT, "sendbufs or recvbufs is NULL");
    const size_t es = elem_size(dtype);
    if (mul_overflows(count, es)) return fail(XRED_INVALID_ARGUMENT, "count * size overflows");
    const size_t bytes = count * es;
    for (int r = 0; r < nranks; ++r) {
        if ((st = check_buf(sendbufs[r], bytes, es, "sendbufs", r)) != XRED_SUCCESS) return st;
        if ((st = check_buf(recvbufs[r], bytes, es, "recvbufs", r)) != XRED_SUCCESS) return st;
    }
    for (int r = 0; r < nranks; ++r) {
        for (int q = 0; q < nranks; ++q) {
            if (bad_overlap(recvbufs[r], bytes, sendbufs[q], bytes, q == r))
                return fail(XRED_ALIAS, "recvbufs[%d] overlaps sendbufs[%d]", r, q);
            if (q != r && bad_overlap(recvbufs[r], bytes, recvbufs[q], bytes, false))
                return fail(XRED_ALIAS, "recvbufs[%d] overlaps recvbufs[%d]", r, q);
        }
    }
    const hipError_t e = launch_sim(dtype, op, (const char *const *)sendbufs,
                                    (char *const *)recvbufs, nranks, count, schedule,
                                    (hipStream_t)hip_stream);
    return e == hipSuccess ? XRED_SUCCESS : hip_fail(e, "schedule step launch");
}

XRED_API size_t xred_sim_chunk(size_t count, int nranks)
{
    return (size_t)sim_chunk(count, nranks);
}

XRED_API unsigned xred_set_max_workgroups(unsigned max_workgroups)
{
    return g_max_workgroups.exchange(max_workgroups);
}

}  // extern "C"

namespace {
__global__ void empty_kernel() {}
}  // namespace

extern "C" {

XRED_API xred_status xred_stream_create_partition(int ncu, void **stream, void **rest)
{
    if (trace_enabled())
        trace_printf("xred_stream_create_partition ncu=%d rest=%s", ncu, rest ? "yes" : "no");
    if (stream == nullptr) return fail(XRED_INVALID_ARGUMENT, "stream is NULL");
    *stream = nullptr;
    if (rest != nullptr) *rest = nullptr;
    if (ncu < 1) return fail(XRED_INVALID_ARGUMENT, "ncu = %d", ncu);
    int dev = 0, cus = 0, xcds = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&xcds, hipDeviceAttributeNumberOfXccs, dev);
    if (e != hipSuccess) return hip_fail(e, "device query");
    if (xcds < 1) xcds = 1;
    // bit b of a queue's CU mask is CU b / xcds of XCD b % xcds, so the
    // first ncu bits give every XCD ncu / xcds CUs (and the rest the others)
    constexpr int kMaxMaskWords = 32;
    if (cus % xcds != 0 || cus > 32 * kMaxMaskWords)
        return fail(XRED_UNSUPPORTED, "%d CUs over %d XCDs", cus, xcds);
    if (ncu % xcds != 0 || ncu >= cus)
        return fail(XRED_INVALID_ARGUMENT, "ncu = %d: a multiple of the %d XCDs below %d needed",
                    ncu, xcds, cus);
    uint32_t mine[kMaxMaskWords] = {}, other[kMaxMaskWords] = {};
    const uint32_t nwords = (uint32_t)(cus + 31) / 32;
    for (int b = 0; b < cus; ++b) (b < ncu ? mine : other)[b / 32] |= 1u << (b % 32);
    hipStream_t made[2] = {nullptr, nullptr};
    const int want = rest != nullptr ? 2 : 1;
    for (int i = 0; i < want && e == hipSuccess; ++i) {
        e = hipExtStreamCreateWithCUMask(&made[i], nwords, i == 0 ? mine : other);
        // the runtime may set a queue up at its first use: an empty kernel
        // and a wait here turn a queue it cannot give into an error of this call
        if (e == hipSuccess) e = launch_kernel(empty_kernel, dim3(1), dim3(64), 0, made[i]);
        if (e == hipSuccess) e = hipStreamSynchronize(made[i]);
    }
    if (e != hipSuccess) {
        for (hipStream_t s : made)
            if (s != nullptr) (void)hipStreamDestroy(s);
        return hip_fail(e, "CU-masked stream");
    }
    *stream = made[0];
    if (rest != nullptr) *rest = made[1];
    return XRED_SUCCESS;
}

XRED_API xred_status xred_stream_destroy(void *stream)
{
    if (trace_enabled()) trace_printf("xred_stream_destroy stream=%p", stream);
    if (stream == nullptr) return fail(XRED_INVALID_ARGUMENT, "stream is NULL");
    // its work ends first, so a stream created later under the same handle
    // finds the handle's device words as this one left them
    hipError_t e = hipStreamSynchronize((hipStream_t)stream);
    if (e == hipSuccess) e = hipStreamDestroy((hipStream_t)stream);
    return e == hipSuccess ? XRED_SUCCESS : hip_fail(e, "hipStreamDestroy");
}

XRED_API size_t xred_acc_elem_size(xred_dtype dtype)
{
    return known_dtype(dtype) ? acc_size(dtype) : 0;
}

XRED_API const char *xred_status_string(xred_status s)
{
    switch (s) {
    case XRED_SUCCESS: return "success";
    case XRED_INVALID_ARGUMENT: return "invalid argument";
    case XRED_UNSUPPORTED: return "unsupported dtype/op";
    case XRED_ALIAS: return "buffers overlap";
    case XRED_HIP_ERROR: return "HIP runtime error";
    case XRED_OUT_OF_MEMORY: return "out of memory";
    }
    return "unknown status";
}

XRED_API const char *xred_last_error(void) { return g_err; }

XRED_API int xred_version(void) { return 20301; }

XRED_API void xred_release(void)
{
    release_stream_slots();
    int cur = 0;
    const bool have_dev = hipGetDevice(&cur) == hipSuccess;
    for (int d = 0; d < kMaxDevices; ++d) {
        Pool &pool = g_pool[d];
        std::lock_guard<std::mutex> lock(pool.mu);
        bool any = false;
        for (Slot &s : pool.slot) any |= s.host != nullptr || s.done != nullptr;
        any |= pool.copy != nullptr || pool.track != nullptr;
        if (!any) continue;
        (void)hipSetDevice(d);
        for (Slot &s : pool.slot) {
            free_slot(s);
            if (s.done) (void)hipEventDestroy(s.done);
            if (s.copied) (void)hipEventDestroy(s.copied);
            s.done = s.copied = nullptr;
        }
        if (pool.copy) (void)hipStreamDestroy(pool.copy);
        if (pool.track) (void)hipStreamDestroy(pool.track);
        pool.copy = pool.track = nullptr;
    }
    if (have_dev) (void)hipSetDevice(cur);
}

}  // extern "C"
