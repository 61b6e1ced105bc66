/*
 * xred.h -- C ABI of libxred: one rank's reduce step of ReduceScatter /
 * AllReduce on an AMD Instinct MI355X (gfx950).
 *
 * In a ring or one-shot ReduceScatter/AllReduce every rank, at every step,
 * reduces the chunk it received with its own chunk and forwards or keeps the
 * result (the FTAR ring pipeline and its fused ReduceCopy, Section 5 "HSDP:
 * Fault tolerant AllReduce"; collective semantics as in NCCL, Section 2.2).
 * This library performs that reduce step on one GPU, with the P peer buffers
 * already resident in local HBM.
 *
 * Definition computed by every entry point, for each element index i
 * independently:
 *
 *     out[i] = down( up(src[0][i]) (+) up(src[1][i]) (+) ... (+) up(src[P-1][i]) )
 *
 *   - a LEFT fold in source order 0..P-1 (the order is fixed, so float
 *     results are deterministic and bit-reproducible);
 *   - up(): bf16, fp16, fp8 e4m3 / e5m2 -> binary32 (exact), fp32 -> binary32,
 *     fp64 -> binary64, int8 -> uint32 (sign-extended), uint8 -> uint32
 *     (zero-extended), int32/uint32 -> uint32, int64/uint64 -> uint64; the
 *     accumulator is binary32 for float types (binary64 for fp64) and uint32
 *     / uint64 for integer types;
 *   - (+): XRED_SUM  binary32 (fp64: binary64) add, round to nearest even,
 *                    subnormals kept, or addition modulo 2^32 / 2^64;
 *          XRED_PROD binary32 (fp64: binary64) multiply, or the low 32 / 64
 *                    bits of the product;
 *          XRED_MAX / XRED_MIN  float: total order -inf < ... < -0 < +0 < ...
 *                    < +inf; a NaN among the reduced values gives the quiet
 *                    NaN 0x7FC00000 (fp64: 0x7FF8000000000000; also for P = 1
 *                    and the INIT step); int8/int32/int64 signed,
 *                    uint8/uint32/uint64 unsigned;
 *          XRED_AVG  (float types only) the XRED_SUM fold, then one division
 *                    by P in the accumulator's format, rounded to nearest even;
 *   - the accumulator starts from up(src[0][i]) (never from zero), so a column
 *     of -0.0 sums to -0.0;
 *   - down(): binary32 -> bf16 / fp16 / e5m2 round to nearest even with
 *     subnormals and overflow to +-inf; binary32 -> e4m3 (OCP "FN": no
 *     infinity, largest finite 448) round to nearest even, saturating at
 *     +-448 on overflow and for infinities; the low byte for int8 / uint8 (so
 *     their sums and products wrap modulo 2^8); identity otherwise.  NaN stays
 *     NaN; NaN payloads of SUM/PROD/AVG results are unspecified.
 *
 * Conventions shared by every call:
 *   - All functions are thread-safe and never abort; they print nothing
 *     unless XRED_TRACE is set (below).
 *   - Buffers are device pointers owned by the caller; so is the stream
 *     (a hipStream_t passed as void*, NULL = the default stream).
 *   - Every call is stream-ordered and returns once the work is enqueued.
 *     Host arrays passed in (the srcs pointer array, host-side items) are
 *     consumed before the call returns and may be reused at once.
 *   - Every argument is validated before anything is enqueued: on
 *     XRED_INVALID_ARGUMENT, XRED_UNSUPPORTED, XRED_ALIAS and
 *     XRED_OUT_OF_MEMORY nothing was enqueued.  XRED_HIP_ERROR reports a
 *     runtime failure while enqueueing; the work enqueued before it (earlier
 *     launches of a multi-launch call, a descriptor copy) stays enqueued.
 *     xred_last_error() describes the problem.  count == 0 succeeds with no
 *     launch.
 *   - Device faults (e.g. a pointer to freed memory) surface at the caller's
 *     next synchronisation of the stream, as for any HIP kernel.
 *   - Element pointers must be aligned to the element size; 16-byte aligned
 *     buffers take the fast vector path.  xred_allreduce_local,
 *     xred_reduce_scatter_local and every item of xred_batched_reduce also
 *     take it when all pointers of the call (of the item) sit at the same
 *     offset within 16 bytes (views at one element offset): the elements
 *     before the next 16-byte boundary are folded one by one.
 *     The same calls and items read in vectors too when only the sources
 *     share an offset and dst sits at another (a reduce-scatter shard of odd
 *     length): results are realigned across lanes and stored as aligned
 *     16-byte vectors.  They read in vectors even when their sources sit at
 *     different offsets: each source's vectors are realigned to dst's grid
 *     across lanes (calls and items shorter than a few vectors take a slower
 *     scalar path with the same results).
 *     xred_ring_reduce refuses chunks at different offsets (see there);
 *     xred_reduce_copy_step, xred_acc_cast and
 *     xred_allreduce_sim take the vector path only when every buffer they
 *     touch is 16-byte aligned, else the scalar one.
 *   - Device words the library binds to a stream (the ring's relay word, the
 *     batch queue's counters) are looked up by the stream's handle.  Let a
 *     stream's work finish before destroying it if a stream created later
 *     may be handed the same handle while that work would still be running:
 *     the two would share the words.
 *
 * Environment (read once, when first needed; results never depend on them):
 *   XRED_MAX_WORKGROUPS      initial CU budget (see xred_set_max_workgroups)
 *   XRED_FUSED_WAVES_PER_CU  overrides the fused kernel's resident-wave cap
 *   XRED_RR_WG_PER_CU        workgroups per CU of the round-robin batched kernel
 *   XRED_BATCH_WG_PER_CU     workgroups per CU of host-planned range batches
 *   XRED_TRACE               anything but "0": one line on stderr per entry
 *                            point call (its arguments), per kernel launch
 *                            (kernel, grid, block, LDS bytes, stream, status)
 *                            and per failed call (status and message)
 * XRED_FUSED_WAVES_PER_CU, XRED_RR_WG_PER_CU and XRED_BATCH_WG_PER_CU are
 * tuning overrides for measurement; leave them unset.
 */
#ifndef XRED_H
#define XRED_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define XRED_API __attribute__((visibility("default")))

typedef enum {
    XRED_FLOAT32 = 0,
    XRED_BFLOAT16 = 1,
    XRED_FLOAT16 = 2,   /* IEEE binary16 */
    XRED_INT32 = 3,
    XRED_UINT32 = 4,
    XRED_INT64 = 5,
    XRED_UINT64 = 6,
    XRED_FP8_E4M3 = 7,  /* OCP 8-bit E4M3 ("FN"), saturating */
    XRED_FP8_E5M2 = 8,  /* OCP 8-bit E5M2 */
    XRED_FLOAT64 = 9,   /* IEEE binary64, accumulated in binary64 */
    XRED_INT8 = 10,
    XRED_UINT8 = 11
} xred_dtype;

/* XRED_AVG: float types only, and only where the whole reduction happens in
 * one call (fused, reduce-scatter and batched); elsewhere XRED_UNSUPPORTED. */
typedef enum { XRED_SUM = 0, XRED_PROD = 1, XRED_MAX = 2, XRED_MIN = 3, XRED_AVG = 4 } xred_op;

typedef enum {
    XRED_SUCCESS = 0,
    XRED_INVALID_ARGUMENT = 1,
    XRED_UNSUPPORTED = 2,
    XRED_ALIAS = 3,
    XRED_HIP_ERROR = 4,
    XRED_OUT_OF_MEMORY = 5
} xred_status;

enum { XRED_MAX_SRC = 64 };
enum { XRED_STEP_INIT = 1u, XRED_STEP_FINAL = 2u }; /* xred_reduce_copy_step flags */
enum { XRED_ITEMS_ON_DEVICE = 1u };                 /* xred_batched_reduce flag    */

/* One reduction of a batch: dst[i] = fold over srcs[0..nsrc) of element i,
 * for i < count.  32 bytes, naturally aligned. */
typedef struct {
    const void *const *srcs; /* nsrc source pointers (host or device array, see flags) */
    void *dst;               /* count output elements                                  */
    uint64_t count;          /* elements per source and in dst                         */
    uint32_t nsrc;           /* 1..XRED_MAX_SRC                                        */
    uint32_t reserved;       /* must be 0                                              */
} xred_item;

/*
 * AllReduce's local reduce (the per-rank reduction of FTAR's ring, Section 5;
 * AllReduce semantics, Section 2.2): dst[i] = fold_{p=0..nsrc-1} srcs[p][i],
 * i < count.
 *   srcs     host array of nsrc device pointers, each to count elements of dtype
 *   nsrc     1..XRED_MAX_SRC
 *   dst      device pointer to count elements of dtype.  dst may equal any
 *            srcs[p] exactly (in place); any other overlap is XRED_ALIAS.
 * Errors: XRED_INVALID_ARGUMENT (nsrc out of range, NULL or misaligned
 * pointer with count > 0, count*size overflow), XRED_UNSUPPORTED (dtype/op),
 * XRED_ALIAS, XRED_HIP_ERROR (launch failure).
 */
XRED_API xred_status xred_allreduce_local(const void *const *srcs, int nsrc, void *dst,
                                          size_t count, xred_dtype dtype, xred_op op,
                                          void *hip_stream);

/*
 * ReduceScatter's local reduce for rank `rank` (ReduceScatter semantics,
 * Section 2.2; the ReduceScatter phase of FTAR's ring, Section 5):
 * srcs[p] is rank p's full send buffer of nsrc*recvcount elements and
 *     dst[i] = fold_{p} srcs[p][rank*recvcount + i],  i < recvcount.
 *   rank     0 <= rank < nsrc
 *   dst      recvcount elements; may equal srcs[p] + rank*recvcount exactly
 *            (in place); any other overlap with a read slice is XRED_ALIAS.
 * Errors: as xred_allreduce_local, plus rank out of range.
 */
XRED_API xred_status xred_reduce_scatter_local(const void *const *srcs, int nsrc, int rank,
                                               void *dst, size_t recvcount, xred_dtype dtype,
                                               xred_op op, void *hip_stream);

/*
 * One step of a ring's ReduceCopy (the RedCopy / Reduce kernel operations of
 * the FTAR pipeline, Section 5): fold one incoming chunk into a local
 * accumulator chunk.
 *   flags 0                  acc[i] = acc[i] (+) up(in[i])
 *   XRED_STEP_INIT           acc[i] = up(in[i])              (acc not read)
 *   XRED_STEP_FINAL          dst[i] = down(acc[i] (+) up(in[i]))   (acc not written)
 *   INIT | FINAL             dst[i] = down(up(in[i]))              (acc unused)
 *   in       count elements of dtype
 *   acc      count accumulator elements of xred_acc_elem_size(dtype) bytes
 *            (binary32 for float dtypes, binary64 for fp64, uint32 for 8- and
 *            32-bit and uint64 for 64-bit integer dtypes), aligned to that
 *            size; may be NULL only for
 *            INIT|FINAL
 *   op       not XRED_AVG (a step does not know P; use XRED_SUM and divide)
 *   dst      count elements of dtype, used only with FINAL (may be NULL otherwise)
 * Buffers must not overlap, except dst == in exactly.
 * Errors: XRED_INVALID_ARGUMENT (unknown flag bits, NULL/misaligned pointer,
 * overflow), XRED_UNSUPPORTED, XRED_ALIAS, XRED_HIP_ERROR.
 */
XRED_API xred_status xred_reduce_copy_step(const void *in, void *acc, void *dst, size_t count,
                                           xred_dtype dtype, xred_op op, unsigned flags,
                                           void *hip_stream);

/*
 * Closing cast of a step-wise sequence: dst[i] = down(acc[i]), i < count --
 * the rounding to the I/O type that ends the ring's ReduceScatter phase once
 * the last incoming chunk has been folded into the accumulator (the Reduce of
 * the FTAR pipeline, Section 5, when the last step is not run as FINAL).
 *   acc      count accumulator elements (see xred_reduce_copy_step)
 *   dst      count elements of dtype; must not overlap acc
 * Errors: XRED_INVALID_ARGUMENT (NULL or misaligned pointer, overflow),
 * XRED_UNSUPPORTED (unknown dtype), XRED_ALIAS, XRED_HIP_ERROR.
 */
XRED_API xred_status xred_acc_cast(const void *acc, void *dst, size_t count, xred_dtype dtype,
                                   void *hip_stream);

/*
 * Many independent reductions in one launch, for latency-bound small messages
 * (the per-message software overhead T_c of the LogP model in Section 6.2 is
 * paid once per batch instead of once per message).  Each item computes the
 * xred_allreduce_local definition over its own sources.
 *   items    nitems descriptors.
 *   flags 0: `items` and every items[k].srcs are HOST memory, consumed before
 *            return (metadata by value).  Every item is validated as in
 *            xred_allreduce_local; the library stages the descriptors, with
 *            a list of every tile's item, into device memory it owns (pinned
 *            staging slots reused once the launch that read them has
 *            completed) and runs one workgroup per tile.  A batch of at most
 *            two tiles per CU and 64 KiB of staged data is read by the kernel
 *            straight from the pinned slot (no copy); batches of 256 KiB
 *            of staged data or more are copied on a stream the library owns
 *            (one per device, default priority), which the caller's stream
 *            then waits for through an event, so the copy overlaps earlier
 *            work on the caller's stream.  When a slot is free again is
 *            tracked on a second stream the library owns, never by an event
 *            left on the caller's stream, so the caller may destroy its
 *            stream as soon as the call returns.  Not capturable: on a
 *            stream under graph capture the call returns XRED_UNSUPPORTED
 *            (a replay would copy whatever a later call left in the slot).
 *   XRED_ITEMS_ON_DEVICE: `items` and every items[k].srcs are DEVICE memory,
 *            read when the kernels run, so an earlier kernel on the stream may
 *            still write them (metadata by reference, after the GPU-resident
 *            collectives of Section 6.1).  No host work per item: the kernel
 *            plans the batch from the descriptors.  Batches of 65..16384
 *            items launched eagerly take tiles in order from a counter pair
 *            in device memory the library binds to the calling stream (64
 *            streams per device, allocated once, until xred_release);
 *            under graph capture, past 64 streams or past 16384 items the
 *            batch runs on a kernel that keeps no state, so the call can be
 *            captured in a HIP graph (same results).  Items that cannot be
 *            run safely (nsrc outside 1..64, a NULL pointer, reserved != 0)
 *            are skipped and their dst is left untouched; pointers are
 *            otherwise trusted.
 *   Items of one batch must not write memory another item reads or writes.
 * Errors: XRED_INVALID_ARGUMENT (nitems < 0, bad item in host mode, unknown
 * flags), XRED_UNSUPPORTED (also host mode under capture), XRED_ALIAS (host
 * mode, within an item),
 * XRED_OUT_OF_MEMORY (host mode: staging allocation), XRED_HIP_ERROR.
 */
XRED_API xred_status xred_batched_reduce(const xred_item *items, int nitems, xred_dtype dtype,
                                         xred_op op, unsigned flags, void *hip_stream);

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation: the
 * device-descriptor form of xred_batched_reduce (flags XRED_ITEMS_ON_DEVICE:
 * items and every items[k].srcs are device memory, read when the kernel runs;
 * items that cannot be run safely are skipped; same results) with the tile
 * counters of its kernel in a fixed 256-byte array of device memory that the
 * library holds on each GPU it runs on until the process ends.  The call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine).
 * The counters are zero when the library is loaded and every launch leaves
 * them zero, so the call can be captured in a graph and replayed; calls that
 * overlap on one GPU (other streams, other threads, replays running
 * concurrently) share the array and race: serialise them.  The first call on
 * a device looks up the array's device address.
 *   nitems   0..16384 (XRED_UNSUPPORTED beyond: the kernel plans the whole
 *            batch in on-chip memory)
 * Errors: XRED_INVALID_ARGUMENT (nitems < 0, NULL or misaligned items),
 * XRED_UNSUPPORTED (dtype/op, too many items), XRED_HIP_ERROR.
 */
XRED_API xred_status xred_batched_reduce_noalloc(const xred_item *items, int nitems,
                                                 xred_dtype dtype, xred_op op, void *hip_stream);

/*
 * All steps of a ring's ReduceCopy in one persistent launch: the FTAR
 * pipeline's in-kernel reduce (Section 5) gated by producer/consumer flags
 * in host-pinned or device memory (the host-kernel coordinated mode of
 * Section 4).  Computes dst[i] = down(fold_{s=0..nchunks-1} up(chunks[s][i])),
 * the same definition and fold order as xred_allreduce_local over the
 * chunks, with the accumulator kept on chip (LDS) between steps, so only
 * the chunks are read and only dst is written.
 *   chunks     host array of nchunks (1..XRED_MAX_SRC) device pointers to count
 *              elements each, all at one offset within 16 bytes (else
 *              XRED_UNSUPPORTED); the elements before their next 16-byte
 *              boundary are folded one by one with the tail.  dst may sit at
 *              any element offset (at another one than the chunks, results
 *              are realigned across lanes before the 16-byte stores).
 *   count      at most xred_ring_max_count(dtype) (else XRED_UNSUPPORTED)
 *   ready      NULL: every chunk is ready at launch.  Otherwise nchunks
 *              uint32 words the GPU can read coherently (hipHostMalloc'd or
 *              device memory); chunk s is read only once
 *              (int32_t)(ready[s] - epoch) >= 0 has been observed, and then
 *              with system-coherent loads, so data written before the flag
 *              is seen.  One wave of the launch polls the flags and relays
 *              their progress to the other workgroups through a word in
 *              device memory the library binds to the calling stream (up to
 *              64 streams per device, until xred_release); under graph
 *              capture, on hipStreamPerThread or past 64 streams, every
 *              workgroup polls the flags itself, which costs more with host
 *              flags.
 *   timeout_us bound on each wait (0: one second; capped at 60 s).  A
 *              workgroup whose wait makes no progress for that long writes 1
 *              to *status (if status is not NULL) and stops; dst is then
 *              unspecified.  The caller zeroes *status before the call if it
 *              wants to check it.
 * Errors: as xred_allreduce_local; XRED_UNSUPPORTED for chunks at different
 * offsets within 16 bytes or counts beyond the capacity.
 */
XRED_API xred_status xred_ring_reduce(const void *const *chunks, int nchunks, void *dst,
                                      size_t count, xred_dtype dtype, xred_op op,
                                      const uint32_t *ready, uint32_t epoch, uint64_t timeout_us,
                                      uint32_t *status, void *hip_stream);

/* Largest count xred_ring_reduce accepts for dtype on the current device. */
XRED_API size_t xred_ring_max_count(xred_dtype dtype);

/* Schedules of xred_allreduce_sim. */
typedef enum {
    XRED_SCHEDULE_RING = 0,  /* ring: 2(G-1) steps, one launch each */
    XRED_SCHEDULE_RHD = 1,   /* recursive halving-doubling, G a power of two: 2 log2(G)
                                steps, one launch each */
    XRED_SCHEDULE_RING_ONE_LAUNCH = 2, /* the ring, every step in one launch */
    XRED_SCHEDULE_RHD_ONE_LAUNCH = 3   /* halving-doubling, every step in one launch */
} xred_schedule;

/*
 * A whole AllReduce over nranks = G simulated ranks whose buffers all live on
 * this GPU, step by step: the ring of the FTAR pipeline (Section 5:
 * sendCopy, RedCopy, Reduce, RecvCopy, Recv) or the recursive
 * halving-doubling schedule (Section 2.2).  Each step is one launch holding
 * every rank's work of that step.
 *
 * Every hop is the two-source reduce down(up(received) (+) up(own)), so a
 * partial is rounded to the I/O dtype each time it travels.  In the ring,
 * chunk c is folded in arrival order c+1, c+2, ..., c+G-1, c (mod G); in
 * halving-doubling, at distance d = G/2, ..., 1 every rank combines its
 * partner's partial with its own.  Messages are zero-copy: the partial a
 * rank forwards is stored once, in that rank's own recvbuf at the chunk's
 * place, and the next rank reads it there; a reduced chunk is forwarded from
 * where it was written.  No staging buffer and no extra store per hop.
 *
 *   sendbufs, recvbufs  host arrays of G device pointers to count elements
 *              each, consumed before return.  recvbufs[r] may equal
 *              sendbufs[r] (in place); a recvbuf must not overlap any other
 *              buffer.  Sends may overlap each other.
 *   G          1..XRED_MAX_SRC; a power of two for XRED_SCHEDULE_RHD.  With
 *              one rank recvbufs[0] becomes a bitwise copy of sendbufs[0].
 *   chunks     xred_sim_chunk(count, G) elements each, i.e. ceil(count / G)
 *              rounded up to a multiple of 64; trailing chunks are short or
 *              empty.  (RHD blocks are the same chunks.)
 * The ONE_LAUNCH schedules run every step in a single launch and give the
 * same bits.  Each thread folds one element vector of one chunk in the
 * schedule's order, handing every message to the next hop in registers,
 * rounded to the I/O dtype exactly as when it is sent, and stores only the
 * final bits into every recvbufs[r]: the messages the per-step schedule
 * stores and then overwrites in its AllGather phase are never written (the
 * intermediate stores ReduceCopy avoids, Section 5).  The call reads G N and
 * writes G N elements instead of 5 (G-1) N, in one launch instead of
 * 2 (G-1) or 2 log2(G).
 * When the stream reaches the end of the call every recvbufs[r] holds the
 * same bits.  Buffers that are all 16-byte aligned take the vector path,
 * others (element-aligned) a scalar path with the same results.
 * Errors: XRED_INVALID_ARGUMENT (G out of range, unknown schedule, RHD with G
 * not a power of two, NULL or misaligned pointer, size overflow),
 * XRED_UNSUPPORTED, XRED_ALIAS, XRED_HIP_ERROR.
 */
XRED_API xred_status xred_allreduce_sim(const void *const *sendbufs, void *const *recvbufs,
                                        int nranks, size_t count, xred_dtype dtype, xred_op op,
                                        xred_schedule schedule, void *hip_stream);

/* Chunk length of xred_allreduce_sim's schedules (0 when nranks < 1). */
XRED_API size_t xred_sim_chunk(size_t count, int nranks);

/*
 * CU budget: at most max_workgroups workgroups per launch of the fused,
 * reduce-scatter, step-wise, cast and batched kernels (0 = no limit, the
 * default), so a reduction can run beside compute kernels on the rest of the
 * chip -- the paper's FTAR kernel uses two thread blocks and stays hidden
 * behind the network (Section 5).  Results do not depend on it.  Process-wide;
 * returns the previous value.  xred_ring_reduce applies it too, but never goes
 * below the workgroups its on-chip accumulators need (one per 4 tiles).
 * The budget bounds the workgroups a launch may have in flight; it does not
 * make a reduce run beside a kernel that fills the chip: on MI355X a bf16
 * matrix product's workgroups take whole CUs, and a reduce on another stream
 * waits for free CUs and then runs alone (measured: the two streams take the
 * sum of their times, capped or not).  xred_stream_create_partition gives the
 * reduce CUs of its own.
 */
XRED_API unsigned xred_set_max_workgroups(unsigned max_workgroups);

/*
 * Co-scheduling by a CU partition (the paper keeps its collective kernels to
 * a few thread blocks so compute keeps the rest of the GPU, Section 5).
 * Creates, on the current device, a HIP stream whose kernels run only on
 * `ncu` compute units, ncu / X of them on each of the device's X XCDs, and,
 * if `rest` is not NULL, a second stream whose kernels run only on all the
 * other CUs.  Kernels on the two streams then run at the same time, each on
 * its own CUs: a reduce launched on *stream beside a matrix product on *rest
 * (measured on MI355X: P=8 x 8 MiB bf16 reduces on 16 CUs at ~1 TB/s,
 * concurrently with the product).  A kernel sized for the whole chip runs
 * slower on a partition than the CU count alone suggests (torch's bf16
 * matrix products lost 27-37 % on any partial CU set), so the partition pays
 * off only where the compute side tolerates it.
 *   ncu     a positive multiple of X below the CU count (256 CUs, X = 8 on
 *           MI355X: 8, 16, ..., 248)
 *   stream  receives the new stream (a hipStream_t); NULL on failure
 *   rest    NULL, or receives the second stream; NULL on failure
 * Each stream is a hardware queue of its own; the runtime has few per process
 * and refuses more with XRED_HIP_ERROR (nothing is created then).  The
 * streams are ordinary HIP streams to every libxred entry point and to other
 * libraries; destroy them with xred_stream_destroy or hipStreamDestroy.
 * Errors: XRED_INVALID_ARGUMENT (stream NULL, ncu out of range),
 * XRED_UNSUPPORTED (CU count not a multiple of the XCD count),
 * XRED_HIP_ERROR.
 */
XRED_API xred_status xred_stream_create_partition(int ncu, void **stream, void **rest);

/* Waits for the work enqueued on `stream` (not NULL), then destroys it.
 * Errors: XRED_INVALID_ARGUMENT, XRED_HIP_ERROR. */
XRED_API xred_status xred_stream_destroy(void *stream);

/* Bytes per accumulator element for dtype: 4 (binary32 or uint32), 8
 * (binary64 for fp64, uint64 for int64/uint64), 0 if unknown. */
XRED_API size_t xred_acc_elem_size(xred_dtype dtype);

/* Static, human-readable name of a status code. */
XRED_API const char *xred_status_string(xred_status s);

/* Detail of the last failed call on the calling thread ("" if none). */
XRED_API const char *xred_last_error(void);

/* Library version: major*10000 + minor*100 + patch. */
XRED_API int xred_version(void);

/* Frees the library's host-mode batch staging buffers, and the ring's relay
 * words and the batch queue's counters, on every device after synchronising
 * the device work that uses them, and unbinds those from their streams.
 * Optional; later calls re-create what they need. */
XRED_API void xred_release(void);

#ifdef __cplusplus
}
#endif

#endif /* XRED_H */
