/*
 * xred_oracle.c -- plain, slow, obviously correct CPU oracle for one rank's
 * reduce step of ReduceScatter / AllReduce.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, includes
 * or calls this file; only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load it.  It shares no code, header, table or
 * constant with the HIP path.
 *
 * What it computes (the per-rank reduce of the FTAR ring, Section 5 "HSDP:
 * Fault tolerant AllReduce", and the ReduceScatter/AllReduce semantics of
 * Section 2.2 "Communication libraries"):
 *
 *     out[i] = down( fold( up(src[0][i]), up(src[1][i]), ..., up(src[P-1][i]) ) )
 *
 * for every element index i independently, where fold is a LEFT fold in
 * source order 0..P-1 (the paper never states an order; a fixed rank order is
 * the reading taken), up() converts an input element to the accumulator type
 * (binary32 for bf16/fp16/fp8/fp32, binary64 for fp64, uint32 for
 * int8/uint8/int32/uint32 -- int8 sign-extended, uint8 zero-extended --,
 * uint64 for int64/uint64: the paper names no accumulator type), and down()
 * converts back with round-to-nearest-even (for the integer types: keeps the
 * low bits).  AVG (float types) is the SUM fold followed by one division by P
 * in the accumulator's format.
 *
 * Arithmetic is carried out in binary32 (binary64 for fp64) because the
 * definition being checked is accumulation in that format; this file is
 * compiled with -ffp-contract=off and without fast-math so that every float
 * operation is one IEEE operation with round-to-nearest-even, subnormals
 * preserved.
 *
 * Readings of points the paper leaves open (each is repeated in the design
 * notes):
 *   - the accumulator starts from up(src[0][i]), never from 0, so a column of
 *     -0.0 sums to -0.0;
 *   - MAX/MIN use the total order -inf < ... < -0 < +0 < ... < +inf; a NaN
 *     among the reduced values gives the canonical quiet NaN 0x7FC00000
 *     (0x7FF8000000000000 for fp64), whatever their number (also for a single
 *     source and for the INIT step of the step-wise mode);
 *   - int8 / uint8 sum and product wrap modulo 2^8 (the uint32 accumulator's
 *     low byte: wrapping modulo 2^32 first changes nothing), max / min
 *     compare signed (int8) or unsigned (uint8);
 *   - NaN payloads of SUM/PROD/AVG are not specified ("parity unpinned" for
 *     NaN payloads: tests compare NaN-ness only);
 *   - down() of a NaN keeps the sign and gives the I/O type's quiet NaN
 *     (bf16 0x7FC0, fp16 0x7E00, e5m2 0x7E, e4m3 0x7F);
 *   - down() to fp16 or e5m2 overflows to +-inf as rounding dictates; e4m3
 *     (the OCP "FN" format, no infinity) saturates: any magnitude that rounds
 *     past 448, and an infinity, gives +-448.
 *
 * Step-wise ring mode (the ReduceCopy of the FTAR pipeline, Section 5 FTAR):
 * acc <- up(in) on INIT, acc <- acc (+) up(in) otherwise, and on FINAL the
 * result is written as down(...) to dst instead of to acc.
 *
 * Simulated schedules: a whole ring (or recursive halving-doubling)
 * AllReduce over G ranks held in this process, message by message, each hop
 * being the definition with two sources (received, own) and every message
 * kept in the I/O dtype, so the fold order of an element is the order in
 * which the schedule's messages reach it.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#include <stddef.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* The oracle's own codes; the Python loader maps dtype/op names onto them. */
enum { XO_F32 = 10, XO_BF16 = 11, XO_F16 = 12, XO_I32 = 13, XO_U32 = 14, XO_I64 = 15,
       XO_U64 = 16, XO_E4M3 = 17, XO_E5M2 = 18, XO_F64 = 30, XO_I8 = 31, XO_U8 = 32 };
enum { XO_SUM = 20, XO_PROD = 21, XO_MAX = 22, XO_MIN = 23, XO_AVG = 24 };
enum { XO_INIT = 1u, XO_FINAL = 2u };
enum { XO_OK = 0, XO_BAD = -1 };

/* ---------------------------------------------------------------- bits --- */

static uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

static int is_float_type(int dtype)
{
    return dtype == XO_F32 || dtype == XO_BF16 || dtype == XO_F16 || dtype == XO_E4M3 ||
           dtype == XO_E5M2;
}

static int is_int64_type(int dtype) { return dtype == XO_I64 || dtype == XO_U64; }

static int is_int8_type(int dtype) { return dtype == XO_I8 || dtype == XO_U8; }

static size_t elem_size(int dtype)
{
    switch (dtype) {
    case XO_F32: case XO_I32: case XO_U32: return 4;
    case XO_BF16: case XO_F16: return 2;
    case XO_E4M3: case XO_E5M2: return 1;
    case XO_I64: case XO_U64: case XO_F64: return 8;
    case XO_I8: case XO_U8: return 1;
    default: return 0;
    }
}

/* ------------------------------------------------ narrow float formats --- */
/*
 * fp16  IEEE 754 binary16: exponent 5 bits (bias 15), fraction 10 bits.
 * e5m2  OCP 8-bit E5M2: exponent 5 bits (bias 15), fraction 2 bits; infinities
 *       and NaNs as in binary16.
 * e4m3  OCP 8-bit E4M3 ("FN"): exponent 4 bits (bias 7), fraction 3 bits; no
 *       infinity; exponent field 15 with fraction 7 is NaN, so the largest
 *       finite magnitude is 1.75 * 2^8 = 448.
 */
struct small_fmt {
    int mbits, ebits, bias, has_inf;
    uint32_t max_finite;   /* magnitude bits of the largest finite value */
    uint32_t qnan;         /* magnitude bits of the quiet NaN produced */
};
static const struct small_fmt FMT_F16 = {10, 5, 15, 1, 0x7BFFu, 0x7E00u};
static const struct small_fmt FMT_E5M2 = {2, 5, 15, 1, 0x7Bu, 0x7Eu};
static const struct small_fmt FMT_E4M3 = {3, 4, 7, 0, 0x7Eu, 0x7Fu};

static const struct small_fmt *small_fmt_of(int dtype)
{
    switch (dtype) {
    case XO_F16: return &FMT_F16;
    case XO_E5M2: return &FMT_E5M2;
    case XO_E4M3: return &FMT_E4M3;
    default: return NULL;
    }
}

/* Exact widening: sign, biased exponent and fraction read from the fields. */
static float small_to_f32(uint32_t bits, const struct small_fmt *f)
{
    const uint32_t sign = (bits >> (f->mbits + f->ebits)) & 1u;
    const uint32_t e = (bits >> f->mbits) & ((1u << f->ebits) - 1u);
    const uint32_t m = bits & ((1u << f->mbits) - 1u);
    const uint32_t etop = (1u << f->ebits) - 1u;
    float mag;
    if (f->has_inf && e == etop)
        mag = m ? NAN : INFINITY;
    else if (!f->has_inf && e == etop && m == (1u << f->mbits) - 1u)
        mag = NAN;
    else if (e == 0)
        mag = ldexpf((float)m, 1 - f->bias - f->mbits);
    else
        mag = ldexpf((float)(m | (1u << f->mbits)), (int)e - f->bias - f->mbits);
    return sign ? -mag : mag;
}

/*
 * binary32 -> narrow format, round to nearest, ties to even, subnormals kept.
 * |x| = M * 2^E exactly (M < 2^24).  The result's quantum is 2^Q with
 * Q = max(floor(log2 |x|), emin) - mbits; M * 2^(E-Q) is rounded to an integer
 * n by its dropped bits, and n * 2^Q is encoded.  Past the largest finite
 * value the result is infinity for formats that have one and the largest
 * finite magnitude for e4m3 (saturation; an infinite input saturates too).
 * NaN gives the format's quiet NaN with the sign kept.
 */
static uint32_t f32_to_small(float x, const struct small_fmt *f)
{
    const uint32_t b = f2u(x);
    const uint32_t sbit = (b >> 31) << (f->mbits + f->ebits);
    const uint32_t etop = (1u << f->ebits) - 1u;
    const uint32_t overflow = f->has_inf ? (etop << f->mbits) : f->max_finite;
    if (isnan(x)) return sbit | f->qnan;
    if (isinf(x)) return sbit | overflow;
    uint32_t M = b & 0x7FFFFFu;
    const uint32_t ef = (b >> 23) & 0xFFu;
    int E;
    if (ef == 0) {
        if (M == 0) return sbit;
        E = -149;
    } else {
        M |= 0x800000u;
        E = (int)ef - 150;
    }
    int msb = 31;
    while (!(M >> msb)) --msb;
    const int k = E + msb;                     /* floor(log2 |x|) */
    const int emin = 1 - f->bias;
    int Q = (k > emin ? k : emin) - f->mbits;
    const int shift = Q - E;                   /* bits of M below the quantum */
    uint64_t n;
    if (shift <= 0) {
        n = (uint64_t)M << (-shift);
    } else if (shift > 25) {
        n = 0;                                 /* below half a quantum */
    } else {
        n = (uint64_t)M >> shift;
        const uint64_t rem = (uint64_t)M & ((1ull << shift) - 1u);
        const uint64_t half = 1ull << (shift - 1);
        if (rem > half || (rem == half && (n & 1u))) n += 1;
    }
    if (n == 0) return sbit;
    if (n >= (2ull << f->mbits)) {             /* carried into the next binade */
        n >>= 1;
        Q += 1;
    }
    if (n < (1ull << f->mbits)) return sbit | (uint32_t)n;   /* subnormal */
    const int efield = Q + f->mbits + f->bias;
    if (efield > (int)etop) return sbit | overflow;
    const uint32_t mag = ((uint32_t)efield << f->mbits) | (uint32_t)(n - (1ull << f->mbits));
    if (mag > f->max_finite) return sbit | overflow;
    return sbit | mag;
}

/* ---------------------------------------------------------------- up() --- */

/* bf16 is the top half of a binary32: widening is exact. */
static float bf16_to_f32(uint16_t h) { return u2f((uint32_t)h << 16); }

static float up_float(const void *base, uint64_t i, int dtype)
{
    if (dtype == XO_BF16) {
        uint16_t h;
        memcpy(&h, (const char *)base + 2 * i, 2);
        return bf16_to_f32(h);
    }
    if (dtype == XO_F16) {
        uint16_t h;
        memcpy(&h, (const char *)base + 2 * i, 2);
        return small_to_f32(h, &FMT_F16);
    }
    if (dtype == XO_E4M3 || dtype == XO_E5M2)
        return small_to_f32(((const uint8_t *)base)[i], small_fmt_of(dtype));
    float f;
    memcpy(&f, (const char *)base + 4 * i, 4);
    return f;
}

static uint32_t up_int(const void *base, uint64_t i)
{
    uint32_t u;
    memcpy(&u, (const char *)base + 4 * i, 4);
    return u;
}

static uint64_t up_int64(const void *base, uint64_t i)
{
    uint64_t u;
    memcpy(&u, (const char *)base + 8 * i, 8);
    return u;
}

/* -------------------------------------------------------------- down() --- */

/* binary32 -> bf16, round to nearest, ties to even.  The 16 dropped bits
 * decide: above half rounds the magnitude up, below half truncates, exactly
 * half rounds up only when the kept part is odd.  A carry out of the kept
 * mantissa moves into the exponent, which is the correct next representable
 * value (and gives +-inf past the largest finite bf16). */
static uint16_t f32_to_bf16(float f)
{
    uint32_t b = f2u(f);
    if (isnan(f))
        return (uint16_t)(((b >> 16) & 0x8000u) | 0x7FC0u);
    uint32_t kept = b >> 16;
    uint32_t dropped = b & 0xFFFFu;
    if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u)))
        kept += 1u;
    return (uint16_t)kept;
}

static void down_float(void *base, uint64_t i, int dtype, float v)
{
    if (dtype == XO_BF16) {
        uint16_t h = f32_to_bf16(v);
        memcpy((char *)base + 2 * i, &h, 2);
    } else if (dtype == XO_F16) {
        uint16_t h = (uint16_t)f32_to_small(v, &FMT_F16);
        memcpy((char *)base + 2 * i, &h, 2);
    } else if (dtype == XO_E4M3 || dtype == XO_E5M2) {
        ((uint8_t *)base)[i] = (uint8_t)f32_to_small(v, small_fmt_of(dtype));
    } else {
        memcpy((char *)base + 4 * i, &v, 4);
    }
}

static void down_int64(void *base, uint64_t i, uint64_t v)
{
    memcpy((char *)base + 8 * i, &v, 8);
}

static void down_int(void *base, uint64_t i, uint32_t v)
{
    memcpy((char *)base + 4 * i, &v, 4);
}

/* --------------------------------------------------------- the operators -- */

static float canonical_nan(void) { return u2f(0x7FC00000u); }

/* Total-order maximum: NaN anywhere -> canonical NaN; otherwise the larger
 * value, with +0 counted above -0. */
static float max_total(float a, float b)
{
    if (isnan(a) || isnan(b)) return canonical_nan();
    if (a > b) return a;
    if (b > a) return b;
    /* a == b numerically: only +-0 can differ in bits */
    return signbit(a) ? b : a;
}

static float min_total(float a, float b)
{
    if (isnan(a) || isnan(b)) return canonical_nan();
    if (a < b) return a;
    if (b < a) return b;
    return signbit(a) ? a : b;
}

static float op_float(int op, float a, float b)
{
    switch (op) {
    case XO_SUM: return a + b;
    case XO_PROD: return a * b;
    case XO_MAX: return max_total(a, b);
    default: return min_total(a, b);
    }
}

/* Integer ops on uint32 accumulators: sum and product wrap modulo 2^32;
 * max/min compare as signed int32 for XO_I32 and XO_I8 (whose values are
 * sign-extended) and as unsigned otherwise. */
static uint32_t op_int(int op, int dtype, uint32_t a, uint32_t b)
{
    const int sgn = dtype == XO_I32 || dtype == XO_I8;
    switch (op) {
    case XO_SUM: return a + b;
    case XO_PROD: return a * b;
    case XO_MAX:
        if (sgn) return ((int32_t)a > (int32_t)b) ? a : b;
        return a > b ? a : b;
    default:
        if (sgn) return ((int32_t)a < (int32_t)b) ? a : b;
        return a < b ? a : b;
    }
}

/* 64-bit integers: sum and product wrap modulo 2^64; max/min signed for XO_I64. */
static uint64_t op_int64(int op, int dtype, uint64_t a, uint64_t b)
{
    switch (op) {
    case XO_SUM: return a + b;
    case XO_PROD: return a * b;
    case XO_MAX:
        if (dtype == XO_I64) return ((int64_t)a > (int64_t)b) ? a : b;
        return a > b ? a : b;
    default:
        if (dtype == XO_I64) return ((int64_t)a < (int64_t)b) ? a : b;
        return a < b ? a : b;
    }
}

/* ------------------------------------------------------------ binary64 --- */

static double u2d(uint64_t u) { double d; memcpy(&d, &u, 8); return d; }
static double canonical_nan64(void) { return u2d(0x7FF8000000000000ull); }

static double max_total64(double a, double b)
{
    if (isnan(a) || isnan(b)) return canonical_nan64();
    if (a > b) return a;
    if (b > a) return b;
    return signbit(a) ? b : a;
}

static double min_total64(double a, double b)
{
    if (isnan(a) || isnan(b)) return canonical_nan64();
    if (a < b) return a;
    if (b < a) return b;
    return signbit(a) ? a : b;
}

static double op_f64(int op, double a, double b)
{
    switch (op) {
    case XO_SUM: return a + b;
    case XO_PROD: return a * b;
    case XO_MAX: return max_total64(a, b);
    default: return min_total64(a, b);
    }
}

static double settle64(int op, double v)
{
    if ((op == XO_MAX || op == XO_MIN) && isnan(v)) return canonical_nan64();
    return v;
}

static double up_f64(const void *base, uint64_t i)
{
    double d;
    memcpy(&d, (const char *)base + 8 * i, 8);
    return d;
}

static void down_f64(void *base, uint64_t i, double v) { memcpy((char *)base + 8 * i, &v, 8); }

/* ------------------------------------------------------- int8 / uint8 --- */

/* Widened to uint32: int8 sign-extended, uint8 zero-extended. */
static uint32_t up_int8(const void *base, uint64_t i, int dtype)
{
    const uint8_t b = ((const uint8_t *)base)[i];
    return dtype == XO_I8 ? (uint32_t)(int32_t)(int8_t)b : (uint32_t)b;
}

/* The low byte of the accumulator. */
static void down_int8(void *base, uint64_t i, uint32_t v) { ((uint8_t *)base)[i] = (uint8_t)v; }

/* MAX/MIN results: a NaN anywhere among the reduced values is reported as the
 * canonical quiet NaN, also when no binary operation was applied (P = 1). */
static float settle(int op, float v)
{
    if ((op == XO_MAX || op == XO_MIN) && isnan(v)) return canonical_nan();
    return v;
}

static int valid_dtype(int dtype) { return elem_size(dtype) != 0; }
static int valid_op(int op) { return op >= XO_SUM && op <= XO_AVG; }
/* AVG is defined for float types only. */
static int valid_pair(int dtype, int op)
{
    return valid_dtype(dtype) && valid_op(op) &&
           (op != XO_AVG || is_float_type(dtype) || dtype == XO_F64);
}

/* ------------------------------------------------------ the definition --- */

/* out[i] = down(fold_op(up(srcs[0][off+i]), ..., up(srcs[P-1][off+i])));
 * AVG is the SUM fold followed by one division by P in the accumulator's
 * format. */
static void reduce_one(const void *const *srcs, int nsrc, uint64_t off, void *dst,
                       uint64_t i, int dtype, int op)
{
    if (dtype == XO_F64) {
        const int fop = op == XO_AVG ? XO_SUM : op;
        double acc = up_f64(srcs[0], off + i);
        for (int p = 1; p < nsrc; ++p) acc = op_f64(fop, acc, up_f64(srcs[p], off + i));
        if (op == XO_AVG) acc = acc / (double)nsrc;
        down_f64(dst, i, settle64(op, acc));
    } else if (is_int8_type(dtype)) {
        uint32_t acc = up_int8(srcs[0], off + i, dtype);
        for (int p = 1; p < nsrc; ++p)
            acc = op_int(op, dtype, acc, up_int8(srcs[p], off + i, dtype));
        down_int8(dst, i, acc);
    } else if (is_float_type(dtype)) {
        const int fop = op == XO_AVG ? XO_SUM : op;
        float acc = up_float(srcs[0], off + i, dtype);
        for (int p = 1; p < nsrc; ++p)
            acc = op_float(fop, acc, up_float(srcs[p], off + i, dtype));
        if (op == XO_AVG) acc = acc / (float)nsrc;
        down_float(dst, i, dtype, settle(op, acc));
    } else if (is_int64_type(dtype)) {
        uint64_t acc = up_int64(srcs[0], off + i);
        for (int p = 1; p < nsrc; ++p)
            acc = op_int64(op, dtype, acc, up_int64(srcs[p], off + i));
        down_int64(dst, i, acc);
    } else {
        uint32_t acc = up_int(srcs[0], off + i);
        for (int p = 1; p < nsrc; ++p)
            acc = op_int(op, dtype, acc, up_int(srcs[p], off + i));
        down_int(dst, i, acc);
    }
}

static int reduce_range(const void *const *srcs, int nsrc, uint64_t off, void *dst,
                        uint64_t count, int dtype, int op, int nthreads)
{
    if (nsrc < 1 || !valid_pair(dtype, op)) return XO_BAD;
    if (count == 0) return XO_OK;
    if (nthreads < 1) nthreads = 1;
    /* Elements are independent; splitting the index range over threads does
     * not change any element's fold order. */
#ifdef _OPENMP
#pragma omp parallel for num_threads(nthreads) schedule(static)
#endif
    for (int64_t i = 0; i < (int64_t)count; ++i)
        reduce_one(srcs, nsrc, off, dst, (uint64_t)i, dtype, op);
    return XO_OK;
}

/* AllReduce's local reduce: the definition over whole buffers. */
int xo_allreduce_local(const void *const *srcs, int nsrc, void *dst, uint64_t count,
                       int dtype, int op, int nthreads)
{
    return reduce_range(srcs, nsrc, 0, dst, count, dtype, op, nthreads);
}

/* ReduceScatter's local reduce for rank r: srcs[p] is rank p's full send
 * buffer of nsrc*recvcount elements; rank r keeps shard r, i.e. the
 * definition applied to srcs[p][r*recvcount .. (r+1)*recvcount). */
int xo_reduce_scatter_local(const void *const *srcs, int nsrc, int rank, void *dst,
                            uint64_t recvcount, int dtype, int op, int nthreads)
{
    if (rank < 0 || rank >= nsrc) return XO_BAD;
    return reduce_range(srcs, nsrc, (uint64_t)rank * recvcount, dst, recvcount, dtype, op,
                        nthreads);
}

/* One ReduceCopy step of a ring (FTAR pipeline, Section 5):
 *   INIT          acc <- up(in)
 *   (no flag)     acc <- acc (+) up(in)
 *   FINAL         dst <- down(acc (+) up(in))      (acc is not written)
 *   INIT|FINAL    dst <- down(up(in))
 * acc holds binary32 for float dtypes (binary64 for fp64), uint32 for 8- and
 * 32-bit integer dtypes and uint64 for 64-bit ones. */
int xo_reduce_copy_step(const void *in, void *acc, void *dst, uint64_t count, int dtype,
                        int op, unsigned flags)
{
    if (!valid_pair(dtype, op) || op == XO_AVG) return XO_BAD;
    int init = (flags & XO_INIT) != 0, fin = (flags & XO_FINAL) != 0;
    for (uint64_t i = 0; i < count; ++i) {
        if (dtype == XO_F64) {
            double x = up_f64(in, i);
            double a = settle64(op, init ? x : op_f64(op, up_f64(acc, i), x));
            if (fin) down_f64(dst, i, a);
            else down_f64(acc, i, a);
        } else if (is_int8_type(dtype)) {
            uint32_t x = up_int8(in, i, dtype);
            uint32_t a = init ? x : op_int(op, dtype, up_int(acc, i), x);
            if (fin) down_int8(dst, i, a);
            else down_int(acc, i, a);
        } else if (is_int64_type(dtype)) {
            uint64_t x = up_int64(in, i);
            uint64_t a = init ? x : op_int64(op, dtype, up_int64(acc, i), x);
            if (fin) down_int64(dst, i, a);
            else down_int64(acc, i, a);
        } else if (is_float_type(dtype)) {
            float x = up_float(in, i, dtype);
            float a = init ? x : op_float(op, up_float(acc, i, XO_F32), x);
            a = settle(op, a);
            if (fin) down_float(dst, i, dtype, a);
            else down_float(acc, i, XO_F32, a);
        } else {
            uint32_t x = up_int(in, i);
            uint32_t a = init ? x : op_int(op, dtype, up_int(acc, i), x);
            if (fin) down_int(dst, i, a);
            else down_int(acc, i, a);
        }
    }
    return XO_OK;
}

/* dst <- down(acc): the closing cast of a step-wise sequence. */
int xo_acc_cast(const void *acc, void *dst, uint64_t count, int dtype)
{
    if (!valid_dtype(dtype)) return XO_BAD;
    for (uint64_t i = 0; i < count; ++i) {
        if (dtype == XO_F64) down_f64(dst, i, up_f64(acc, i));
        else if (is_int8_type(dtype)) down_int8(dst, i, up_int(acc, i));
        else if (is_float_type(dtype)) down_float(dst, i, dtype, up_float(acc, i, XO_F32));
        else if (is_int64_type(dtype)) down_int64(dst, i, up_int64(acc, i));
        else down_int(dst, i, up_int(acc, i));
    }
    return XO_OK;
}

/* Many independent reductions: the definition applied to each item.  Item k
 * reads item_srcs[item_src_off[k] .. item_src_off[k]+item_nsrc[k]) and
 * writes item_count[k] elements to item_dst[k]. */
int xo_batched_reduce(int nitems, const void *const *item_srcs, const uint64_t *item_src_off,
                      const int *item_nsrc, void *const *item_dst, const uint64_t *item_count,
                      int dtype, int op, int nthreads)
{
    for (int k = 0; k < nitems; ++k) {
        int rc = reduce_range(item_srcs + item_src_off[k], item_nsrc[k], 0, item_dst[k],
                              item_count[k], dtype, op, nthreads);
        if (rc != XO_OK) return rc;
    }
    return XO_OK;
}

/* ------------------------------------- simulated multi-rank schedules --- */
/*
 * A whole AllReduce over G ranks whose buffers all live in this process,
 * following a schedule step by step, with every message held in a wire
 * buffer of the I/O dtype.  Each hop's reduction is the definition above
 * with two sources, received message first:  down(up(received) (+) up(own)),
 * so a partial is rounded to the I/O dtype every time it travels.
 *
 * Chunks: M = ceil(count / G) rounded up to a multiple of 64 elements; chunk
 * c is [c*M, min(count, (c+1)*M)), so trailing chunks may be short or empty.
 */
#define XO_SIM_ALIGN 64u

uint64_t xo_sim_chunk(uint64_t count, int G)
{
    if (G < 1) return 0;
    uint64_t m = (count + (uint64_t)G - 1) / (uint64_t)G;
    return (m + XO_SIM_ALIGN - 1) / XO_SIM_ALIGN * XO_SIM_ALIGN;
}

static uint64_t clampu(uint64_t v, uint64_t hi) { return v < hi ? v : hi; }
static int mod_rank(int r, int G) { return ((r % G) + G) % G; }
static char *elem_at(const void *base, uint64_t i, int dtype)
{
    return (char *)base + i * elem_size(dtype);
}

/* dst[0..n) = down(up(received[0..n)) (+) up(own[0..n))) */
static void hop_reduce(const void *received, const void *own, void *dst, uint64_t n, int dtype,
                       int op, int nthreads)
{
    const void *two[2] = {received, own};
    reduce_range(two, 2, 0, dst, n, dtype, op, nthreads);
}

static void **alloc_bufs(int G, uint64_t bytes)
{
    void **b = (void **)calloc((size_t)G, sizeof(void *));
    if (!b) return NULL;
    for (int r = 0; r < G; ++r) {
        b[r] = malloc(bytes ? bytes : 1);
        if (!b[r]) {
            for (int q = 0; q < r; ++q) free(b[q]);
            free(b);
            return NULL;
        }
    }
    return b;
}

static void free_bufs(void **b, int G)
{
    if (!b) return;
    for (int r = 0; r < G; ++r) free(b[r]);
    free(b);
}

/*
 * Ring AllReduce (the ring of the FTAR pipeline, Section 5): rank r sends to
 * rank r+1 and receives from rank r-1.
 *   ReduceScatter phase, G-1 steps after the first send:
 *     sendCopy  rank r puts its own chunk r-1 on the wire;
 *     step s    rank r receives chunk r-1-s;
 *               RedCopy (s < G-1): forwards down(up(received) (+) up(own));
 *               Reduce  (s = G-1): the chunk is r, the result goes to recv[r].
 *   AllGather phase: rank r sends its reduced chunk r; at step t it receives
 *     chunk r-t and writes it to recv[r]; RecvCopy (t < G-1) also forwards it,
 *     Recv (t = G-1) does not.
 * So chunk c is folded in arrival order c+1, c+2, ..., c+G-1, c (mod G), and
 * every rank ends with the same bits.  With G = 1 recv[0] is a copy of
 * send[0].  recv[r] may equal send[r] (in place): inputs are copied first.
 */
int xo_ring_allreduce_sim(const void *const *send, void *const *recv, int G, uint64_t count,
                          int dtype, int op, int nthreads)
{
    /* AVG is not a hop operation (each hop would halve); it is not simulated. */
    if (G < 1 || !valid_pair(dtype, op) || op == XO_AVG) return XO_BAD;
    if (count == 0) return XO_OK;
    const size_t es = elem_size(dtype);
    const uint64_t M = xo_sim_chunk(count, G);
    void **own = alloc_bufs(G, count * es);
    void **wire = alloc_bufs(G, M * es);
    void **next = alloc_bufs(G, M * es);
    if (!own || !wire || !next) {
        free_bufs(own, G); free_bufs(wire, G); free_bufs(next, G);
        return XO_BAD;
    }
    for (int r = 0; r < G; ++r) memcpy(own[r], send[r], count * es);
    if (G == 1) {
        memcpy(recv[0], own[0], count * es);
    } else {
#define LO(c) clampu((uint64_t)(c) * M, count)
#define LEN(c) (LO((c) + 1) - LO(c))
        /* ReduceScatter */
        for (int r = 0; r < G; ++r) {                      /* sendCopy */
            const int c = mod_rank(r - 1, G);
            memcpy(wire[r], elem_at(own[r], LO(c), dtype), LEN(c) * es);
        }
        for (int s = 1; s <= G - 1; ++s) {
            for (int r = 0; r < G; ++r) {
                const int c = mod_rank(r - 1 - s, G);
                const void *in = wire[mod_rank(r - 1, G)];
                if (s < G - 1)                              /* RedCopy */
                    hop_reduce(in, elem_at(own[r], LO(c), dtype), next[r], LEN(c), dtype, op,
                               nthreads);
                else                                        /* Reduce */
                    hop_reduce(in, elem_at(own[r], LO(c), dtype), elem_at(recv[r], LO(c), dtype),
                               LEN(c), dtype, op, nthreads);
            }
            void **t = wire; wire = next; next = t;
        }
        /* AllGather */
        for (int r = 0; r < G; ++r)
            memcpy(wire[r], elem_at(recv[r], LO(r), dtype), LEN(r) * es);
        for (int t = 1; t <= G - 1; ++t) {
            for (int r = 0; r < G; ++r) {
                const int c = mod_rank(r - t, G);
                const void *in = wire[mod_rank(r - 1, G)];
                memcpy(elem_at(recv[r], LO(c), dtype), in, LEN(c) * es);   /* Recv */
                if (t < G - 1) memcpy(next[r], in, LEN(c) * es);           /* ...Copy */
            }
            void **tt = wire; wire = next; next = tt;
        }
#undef LEN
#undef LO
    }
    free_bufs(own, G); free_bufs(wire, G); free_bufs(next, G);
    return XO_OK;
}

/*
 * Recursive halving-doubling AllReduce (the RHD ReduceScatter the paper
 * lists beside the ring, Section 2.2), G a power of two.  ReduceScatter by
 * recursive halving: with distance d = G/2, G/4, ..., 1, rank r and its
 * partner r^d split their common region of blocks in two; the rank whose bit
 * d is clear keeps the lower half, the other the upper half; each sends the
 * half it gives up and reduces the received message into the half it keeps,
 * down(up(received) (+) up(own)).  Afterwards rank r holds block r.
 * AllGather by recursive doubling: with d = 1, 2, ..., G/2 each rank sends
 * its region to r^d, which stores it.  Blocks are the chunks defined above.
 */
int xo_rhd_allreduce_sim(const void *const *send, void *const *recv, int G, uint64_t count,
                         int dtype, int op, int nthreads)
{
    if (G < 1 || (G & (G - 1)) != 0 || !valid_pair(dtype, op) || op == XO_AVG) return XO_BAD;
    if (count == 0) return XO_OK;
    const size_t es = elem_size(dtype);
    const uint64_t M = xo_sim_chunk(count, G);
    void **work = alloc_bufs(G, count * es);
    void **msg = alloc_bufs(G, count * es);
    int *lo = (int *)calloc((size_t)G, sizeof(int));
    if (!work || !msg || !lo) {
        free_bufs(work, G); free_bufs(msg, G); free(lo);
        return XO_BAD;
    }
#define EL(b) clampu((uint64_t)(b) * M, count)
    for (int r = 0; r < G; ++r) memcpy(work[r], send[r], count * es);
    int nblk = G;
    for (int d = G / 2; d >= 1; d /= 2) {
        const int half = nblk / 2;
        for (int r = 0; r < G; ++r) {                       /* send the half given up */
            const int give = (r & d) ? lo[r] : lo[r] + half;
            memcpy(msg[r], elem_at(work[r], EL(give), dtype), (EL(give + half) - EL(give)) * es);
        }
        for (int r = 0; r < G; ++r) {                       /* reduce into the half kept */
            const int keep = (r & d) ? lo[r] + half : lo[r];
            void *mine = elem_at(work[r], EL(keep), dtype);
            hop_reduce(msg[r ^ d], mine, mine, EL(keep + half) - EL(keep), dtype, op, nthreads);
            lo[r] = keep;
        }
        nblk = half;
    }
    for (int d = 1; d < G; d *= 2) {
        for (int r = 0; r < G; ++r)
            memcpy(msg[r], elem_at(work[r], EL(lo[r]), dtype), (EL(lo[r] + nblk) - EL(lo[r])) * es);
        for (int r = 0; r < G; ++r) {
            const int p = r ^ d;
            memcpy(elem_at(work[r], EL(lo[p]), dtype), msg[p], (EL(lo[p] + nblk) - EL(lo[p])) * es);
        }
        for (int r = 0; r < G; ++r) lo[r] = lo[r] < lo[r ^ d] ? lo[r] : lo[r ^ d];
        nblk *= 2;
    }
#undef EL
    for (int r = 0; r < G; ++r) memcpy(recv[r], work[r], count * es);
    free_bufs(work, G); free_bufs(msg, G); free(lo);
    return XO_OK;
}

/* Bulk conversions, exposed so tests can check down()/up() on their own. */
void xo_f32_bits_to_bf16(const uint32_t *in, uint16_t *out, uint64_t n)
{
    for (uint64_t i = 0; i < n; ++i) out[i] = f32_to_bf16(u2f(in[i]));
}

void xo_bf16_to_f32_bits(const uint16_t *in, uint32_t *out, uint64_t n)
{
    for (uint64_t i = 0; i < n; ++i) out[i] = f2u(bf16_to_f32(in[i]));
}

/* Returns 0 when the floating-point environment is the one the definition
 * needs: subnormal results kept (no flush-to-zero), subnormal inputs honoured
 * (no denormals-are-zero), round-to-nearest. */
int xo_selfcheck(void)
{
    volatile float tiny = u2f(0x00000001u);   /* 2^-149 */
    volatile float two_tiny = tiny + tiny;   /* 2^-148, needs no FTZ/DAZ */
    if (f2u(two_tiny) != 0x00000002u) return 1;
    volatile float one = 1.0f, eps_half = u2f(0x33800000u); /* 2^-24 */
    volatile float r = one + eps_half;       /* tie: stays 1.0 under RNE */
    if (f2u(r) != 0x3F800000u) return 2;
    volatile float r2 = one + u2f(0x33800001u); /* just above the tie: rounds up */
    if (f2u(r2) != 0x3F800001u) return 3;
    return 0;
}

int xo_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

int xo_version(void) { return 4; }

/* Narrow float conversions on their own, for the pins. */
void xo_small_to_f32_bits(const uint8_t *in, int in_size, uint32_t *out, uint64_t n, int dtype)
{
    const struct small_fmt *f = small_fmt_of(dtype);
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t v = in_size == 2 ? (uint32_t)((const uint16_t *)in)[i] : in[i];
        out[i] = f2u(small_to_f32(v, f));
    }
}

void xo_f32_bits_to_small(const uint32_t *in, uint8_t *out, uint64_t n, int dtype)
{
    const struct small_fmt *f = small_fmt_of(dtype);
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t v = f32_to_small(u2f(in[i]), f);
        if (f->mbits + f->ebits + 1 == 16) ((uint16_t *)out)[i] = (uint16_t)v;
        else out[i] = (uint8_t)v;
    }
}
