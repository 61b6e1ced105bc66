// xred_device.hpp -- device-side element types, operators and 16-byte vector
// conversions for the reduce-step kernels (gfx950).
//
// Every kernel computes, per element, a left fold in source order of
// up-converted values followed by one down-conversion (the per-rank reduce of
// the FTAR ring's ReduceCopy, Section 5).  This header fixes what up(), the
// operators and down() are on the device:
//   bf16 -> binary32 by a 16-bit shift (exact); binary32 -> bf16 with the
//   hardware round-to-nearest-even conversion v_cvt_pk_bf16_f32;
//   fp16 <-> binary32 with v_cvt_f32_f16 / v_cvt_f16_f32 (exact widening,
//   round-to-nearest-even narrowing, subnormals kept, overflow to infinity);
//   OCP fp8 e4m3 / e5m2 <-> binary32 with v_cvt_pk_f32_fp8 / _bf8 (exact) and
//   v_cvt_pk_fp8_f32 / _bf8_f32 (round-to-nearest-even, subnormals kept;
//   e5m2 overflows to infinity; the e4m3 conversion gives NaN past 448, so
//   values are first clamped to [-448, 448] with the NaN-propagating
//   minimum/maximum: e4m3 saturates);
//   float MAX/MIN with the IEEE 754-2019 maximum/minimum operations
//   (v_maximum3_f32 / v_minimum3_f32: NaN-propagating, -0 < +0), the NaN
//   result then replaced by the quiet NaN 0x7FC00000;
//   AVG: the SUM fold, then one correctly rounded binary32 division by P;
//   fp64: binary64 throughout (up and down are the identity, MAX/MIN NaN
//   0x7FF8000000000000, AVG one binary64 division);
//   int8 / uint8 widened to uint32 (sign- / zero-extended) and narrowed by
//   keeping the low byte, so sums and products wrap modulo 2^8;
//   integer SUM/PROD on uint32 / uint64 (wrap), MAX/MIN signed for int8 /
//   int32 / int64.
// All code here is compiled without contraction and with binary32 subnormals
// enabled, so a float add or multiply is exactly one IEEE operation.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xred {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// ----------------------------------------------------------------- types --
// kVec: elements per 16-byte vector; Acc: accumulator type; kSize: bytes.
struct TF32 {
    static constexpr int kVec = 4, kSize = 4;
    static constexpr bool kFloat = true, kSigned = false;
    using Acc = float;
};
struct TBF16 {
    static constexpr int kVec = 8, kSize = 2;
    static constexpr bool kFloat = true, kSigned = false;
    using Acc = float;
};
struct TI32 {
    static constexpr int kVec = 4, kSize = 4;
    static constexpr bool kFloat = false, kSigned = true;
    using Acc = uint32_t;
};
struct TU32 {
    static constexpr int kVec = 4, kSize = 4;
    static constexpr bool kFloat = false, kSigned = false;
    using Acc = uint32_t;
};
struct TF16 {
    static constexpr int kVec = 8, kSize = 2;
    static constexpr bool kFloat = true, kSigned = false;
    using Acc = float;
};
struct TE4M3 {
    static constexpr int kVec = 16, kSize = 1;
    static constexpr bool kFloat = true, kSigned = false;
    using Acc = float;
};
struct TE5M2 {
    static constexpr int kVec = 16, kSize = 1;
    static constexpr bool kFloat = true, kSigned = false;
    using Acc = float;
};
struct TI64 {
    static constexpr int kVec = 2, kSize = 8;
    static constexpr bool kFloat = false, kSigned = true;
    using Acc = uint64_t;
};
struct TU64 {
    static constexpr int kVec = 2, kSize = 8;
    static constexpr bool kFloat = false, kSigned = false;
    using Acc = uint64_t;
};
struct TF64 {
    static constexpr int kVec = 2, kSize = 8;
    static constexpr bool kFloat = true, kSigned = false;
    using Acc = double;
};
struct TI8 {
    static constexpr int kVec = 16, kSize = 1;
    static constexpr bool kFloat = false, kSigned = true;
    using Acc = uint32_t;
};
struct TU8 {
    static constexpr int kVec = 16, kSize = 1;
    static constexpr bool kFloat = false, kSigned = false;
    using Acc = uint32_t;
};

// Accumulator values per 16-byte vector, and 16-byte accumulator vectors
// per 16-byte input vector (a step-wise accumulator holds kVec values of
// Acc per input vector, contiguous).
template <class T>
constexpr int acc_per_vec() { return 16 / (int)sizeof(typename T::Acc); }
template <class T>
constexpr int acc_vecs() { return T::kVec * (int)sizeof(typename T::Acc) / 16; }

struct OpSum {};
struct OpAvg {};
struct OpProd {};
struct OpMax {};
struct OpMin {};

// ------------------------------------------------------------- operators --
template <class T, class Op>
__device__ __forceinline__ typename T::Acc combine(typename T::Acc a, typename T::Acc b)
{
    if constexpr (T::kFloat) {
        if constexpr (__is_same(Op, OpSum) || __is_same(Op, OpAvg)) return a + b;
        else if constexpr (__is_same(Op, OpProd)) return a * b;
        else if constexpr (__is_same(Op, OpMax)) return __builtin_elementwise_maximum(a, b);
        else return __builtin_elementwise_minimum(a, b);
    } else {
        static_assert(!__is_same(Op, OpAvg), "AVG is defined for float types only");
        using A = typename T::Acc;
        if constexpr (__is_same(Op, OpSum)) return a + b;
        else if constexpr (__is_same(Op, OpProd)) return a * b;
        else if constexpr (T::kSigned && sizeof(A) == 8) {
            int64_t x = (int64_t)a, y = (int64_t)b;
            if constexpr (__is_same(Op, OpMax)) return (A)(x > y ? x : y);
            else return (A)(x < y ? x : y);
        } else if constexpr (T::kSigned) {
            int32_t x = (int32_t)a, y = (int32_t)b;
            if constexpr (__is_same(Op, OpMax)) return (uint32_t)(x > y ? x : y);
            else return (uint32_t)(x < y ? x : y);
        } else {
            if constexpr (__is_same(Op, OpMax)) return a > b ? a : b;
            else return a < b ? a : b;
        }
    }
}

// MAX/MIN give the canonical quiet NaN whenever a NaN took part.
template <class T, class Op>
__device__ __forceinline__ typename T::Acc finalize(typename T::Acc a)
{
    if constexpr (__is_same(T, TF64) && (__is_same(Op, OpMax) || __is_same(Op, OpMin)))
        return __builtin_isnan(a) ? __builtin_bit_cast(double, 0x7FF8000000000000ull) : a;
    else if constexpr (T::kFloat && (__is_same(Op, OpMax) || __is_same(Op, OpMin)))
        return __builtin_isnan(a) ? __uint_as_float(0x7FC00000u) : a;
    else
        return a;
}

// AVG: the folded sum divided once by the number of sources (binary32,
// correctly rounded); other ops unchanged.
template <class T, class Op>
__device__ __forceinline__ typename T::Acc avg_scale(typename T::Acc a, int nsrc)
{
    if constexpr (__is_same(Op, OpAvg)) return a / (typename T::Acc)nsrc;
    else return a;
}

// The binary32 value itself, hidden from the optimiser.  The fp16 narrowing
// goes through it: otherwise the last multiply or add of the fold is fused
// with the conversion into one v_fma_mix (a product rounded once to fp16,
// not to binary32 and then fp16, and fma(x, y, +0) turns a -0 product into
// +0), which is not the definition.
__device__ __forceinline__ float opaque(float x)
{
    __asm__("" : "+v"(x));
    return x;
}

// binary32 -> e4m3 input range: [-448, 448], NaN kept (IEEE minimum/maximum).
__device__ __forceinline__ float e4m3_clamp(float x)
{
    return __builtin_elementwise_minimum(__builtin_elementwise_maximum(x, -448.0f), 448.0f);
}

// A NaN narrows to the format's quiet NaN with its sign kept (0x7F / 0xFF for
// e4m3, 0x7E / 0xFE for e5m2); the hardware conversion does not keep the
// sign, so NaN lanes are rewritten.
template <class T>
__device__ __forceinline__ uint32_t fp8_nan_fix(uint32_t w, float a0, float a1, float a2,
                                                float a3)
{
    constexpr uint32_t q = __is_same(T, TE4M3) ? 0x7Fu : 0x7Eu;
    const float v[4] = {a0, a1, a2, a3};
    uint32_t m = 0, fix = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const bool nan = __builtin_isnan(v[k]);
        m |= (nan ? 0xFFu : 0u) << (8 * k);
        fix |= (nan ? (((__float_as_uint(v[k]) >> 31) << 7) | q) : 0u) << (8 * k);
    }
    return (w & ~m) | fix;
}

// Four binary32 values -> four fp8 bytes (byte j = value j).
template <class T>
__device__ __forceinline__ uint32_t pack_fp8x4(float a0, float a1, float a2, float a3)
{
    uint32_t w;
    if constexpr (__is_same(T, TE4M3)) {
        int r = __builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(a0), e4m3_clamp(a1), 0, false);
        w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(e4m3_clamp(a2), e4m3_clamp(a3), r, true);
    } else {
        int r = __builtin_amdgcn_cvt_pk_bf8_f32(a0, a1, 0, false);
        w = (uint32_t)__builtin_amdgcn_cvt_pk_bf8_f32(a2, a3, r, true);
    }
    return fp8_nan_fix<T>(w, a0, a1, a2, a3);
}

// fp8 bytes 2*HI, 2*HI+1 of w -> binary32.
template <class T, bool HI>
__device__ __forceinline__ f32x2 unpack_fp8x2(uint32_t w)
{
    if constexpr (__is_same(T, TE4M3)) return __builtin_amdgcn_cvt_pk_f32_fp8((int)w, HI);
    else return __builtin_amdgcn_cvt_pk_f32_bf8((int)w, HI);
}

// ------------------------------------------------- 16-byte vector up/down --
template <class T>
__device__ __forceinline__ void up_vec(u32x4 v, typename T::Acc (&a)[T::kVec])
{
    if constexpr (__is_same(T, TBF16)) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            a[2 * j] = __uint_as_float(v[j] << 16);
            a[2 * j + 1] = __uint_as_float(v[j] & 0xFFFF0000u);
        }
    } else if constexpr (__is_same(T, TF16)) {
        // element by element: the two-lane vector conversion was miscompiled
        // when a round trip folded away (every word took the first pair)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            a[2 * j] = (float)__builtin_bit_cast(_Float16, (uint16_t)(v[j] & 0xFFFFu));
            a[2 * j + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(v[j] >> 16));
        }
    } else if constexpr (__is_same(T, TE4M3) || __is_same(T, TE5M2)) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const f32x2 lo = unpack_fp8x2<T, false>(v[j]), hi = unpack_fp8x2<T, true>(v[j]);
            a[4 * j] = lo[0];
            a[4 * j + 1] = lo[1];
            a[4 * j + 2] = hi[0];
            a[4 * j + 3] = hi[1];
        }
    } else if constexpr (__is_same(T, TF64)) {
        a[0] = __builtin_bit_cast(double, (uint64_t)v[0] | ((uint64_t)v[1] << 32));
        a[1] = __builtin_bit_cast(double, (uint64_t)v[2] | ((uint64_t)v[3] << 32));
    } else if constexpr (__is_same(T, TI8) || __is_same(T, TU8)) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const uint32_t x = (v[j] >> (8 * b)) & 0xFFu;
                a[4 * j + b] = T::kSigned ? (uint32_t)(int32_t)(int8_t)x : x;
            }
        }
    } else if constexpr (T::kFloat) {
#pragma unroll
        for (int j = 0; j < 4; ++j) a[j] = __uint_as_float(v[j]);
    } else if constexpr (sizeof(typename T::Acc) == 8) {
        a[0] = (uint64_t)v[0] | ((uint64_t)v[1] << 32);
        a[1] = (uint64_t)v[2] | ((uint64_t)v[3] << 32);
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) a[j] = v[j];
    }
}

template <class T, class Op>
__device__ __forceinline__ void fold_vec(typename T::Acc (&a)[T::kVec], u32x4 v)
{
    typename T::Acc b[T::kVec];
    up_vec<T>(v, b);
#pragma unroll
    for (int j = 0; j < T::kVec; ++j) a[j] = combine<T, Op>(a[j], b[j]);
}

template <class T, class Op>
__device__ __forceinline__ u32x4 down_vec(const typename T::Acc (&a)[T::kVec])
{
    u32x4 r;
    if constexpr (__is_same(T, TBF16)) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            f32x2 f = {finalize<T, Op>(a[2 * j]), finalize<T, Op>(a[2 * j + 1])};
            r[j] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
        }
    } else if constexpr (__is_same(T, TF16)) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t lo =
                __builtin_bit_cast(uint16_t, (_Float16)opaque(finalize<T, Op>(a[2 * j])));
            const uint32_t hi =
                __builtin_bit_cast(uint16_t, (_Float16)opaque(finalize<T, Op>(a[2 * j + 1])));
            r[j] = lo | (hi << 16);
        }
    } else if constexpr (__is_same(T, TE4M3) || __is_same(T, TE5M2)) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            r[j] = pack_fp8x4<T>(finalize<T, Op>(a[4 * j]), finalize<T, Op>(a[4 * j + 1]),
                                 finalize<T, Op>(a[4 * j + 2]), finalize<T, Op>(a[4 * j + 3]));
    } else if constexpr (__is_same(T, TF64)) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const uint64_t b = __builtin_bit_cast(uint64_t, finalize<T, Op>(a[j]));
            r[2 * j] = (uint32_t)b;
            r[2 * j + 1] = (uint32_t)(b >> 32);
        }
    } else if constexpr (__is_same(T, TI8) || __is_same(T, TU8)) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            r[j] = (a[4 * j] & 0xFFu) | ((a[4 * j + 1] & 0xFFu) << 8) |
                   ((a[4 * j + 2] & 0xFFu) << 16) | ((a[4 * j + 3] & 0xFFu) << 24);
    } else if constexpr (T::kFloat) {
#pragma unroll
        for (int j = 0; j < 4; ++j) r[j] = __float_as_uint(finalize<T, Op>(a[j]));
    } else if constexpr (sizeof(typename T::Acc) == 8) {
        r[0] = (uint32_t)a[0];
        r[1] = (uint32_t)(a[0] >> 32);
        r[2] = (uint32_t)a[1];
        r[3] = (uint32_t)(a[1] >> 32);
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) r[j] = a[j];
    }
    return r;
}

// ------------------------------------------------------ scalar up/down --
template <class T>
__device__ __forceinline__ typename T::Acc up1(const char *base, size_t i)
{
    if constexpr (__is_same(T, TBF16))
        return __uint_as_float((uint32_t)((const uint16_t *)base)[i] << 16);
    else if constexpr (__is_same(T, TF16))
        return (float)((const _Float16 *)base)[i];
    else if constexpr (__is_same(T, TE4M3) || __is_same(T, TE5M2))
        return unpack_fp8x2<T, false>((uint32_t)((const uint8_t *)base)[i])[0];
    else if constexpr (__is_same(T, TF64))
        return ((const double *)base)[i];
    else if constexpr (__is_same(T, TI8))
        return (uint32_t)(int32_t)((const int8_t *)base)[i];
    else if constexpr (__is_same(T, TU8))
        return (uint32_t)((const uint8_t *)base)[i];
    else if constexpr (T::kFloat)
        return ((const float *)base)[i];
    else
        return ((const typename T::Acc *)base)[i];
}

template <class T, class Op>
__device__ __forceinline__ void down1(char *base, size_t i, typename T::Acc a)
{
    a = finalize<T, Op>(a);
    if constexpr (__is_same(T, TBF16)) {
        f32x2 f = {a, a};
        ((uint16_t *)base)[i] =
            (uint16_t)__builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
    } else if constexpr (__is_same(T, TF16)) {
        ((_Float16 *)base)[i] = (_Float16)opaque(a);
    } else if constexpr (__is_same(T, TE4M3) || __is_same(T, TE5M2)) {
        ((uint8_t *)base)[i] = (uint8_t)pack_fp8x4<T>(a, a, a, a);
    } else if constexpr (__is_same(T, TF64)) {
        ((double *)base)[i] = a;
    } else if constexpr (__is_same(T, TI8) || __is_same(T, TU8)) {
        ((uint8_t *)base)[i] = (uint8_t)a;
    } else if constexpr (T::kFloat) {
        ((float *)base)[i] = a;
    } else {
        ((typename T::Acc *)base)[i] = a;
    }
}

// ------------------------------------------- accumulator (un)packing --
// 16-byte vector y <-> acc_per_vec<T>() accumulator values a[0..).
template <class T>
__device__ __forceinline__ void unpack_acc(u32x4 y, typename T::Acc *a)
{
    if constexpr (__is_same(T, TF64)) {
        a[0] = __builtin_bit_cast(double, (uint64_t)y[0] | ((uint64_t)y[1] << 32));
        a[1] = __builtin_bit_cast(double, (uint64_t)y[2] | ((uint64_t)y[3] << 32));
    } else if constexpr (sizeof(typename T::Acc) == 8) {
        a[0] = (uint64_t)y[0] | ((uint64_t)y[1] << 32);
        a[1] = (uint64_t)y[2] | ((uint64_t)y[3] << 32);
    } else if constexpr (T::kFloat) {
#pragma unroll
        for (int j = 0; j < 4; ++j) a[j] = __uint_as_float(y[j]);
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) a[j] = y[j];
    }
}

template <class T>
__device__ __forceinline__ u32x4 pack_acc(const typename T::Acc *a)
{
    u32x4 y;
    if constexpr (__is_same(T, TF64)) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const uint64_t b = __builtin_bit_cast(uint64_t, a[j]);
            y[2 * j] = (uint32_t)b;
            y[2 * j + 1] = (uint32_t)(b >> 32);
        }
    } else if constexpr (sizeof(typename T::Acc) == 8) {
        y[0] = (uint32_t)a[0];
        y[1] = (uint32_t)(a[0] >> 32);
        y[2] = (uint32_t)a[1];
        y[3] = (uint32_t)(a[1] >> 32);
    } else if constexpr (T::kFloat) {
#pragma unroll
        for (int j = 0; j < 4; ++j) y[j] = __float_as_uint(a[j]);
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) y[j] = a[j];
    }
    return y;
}

}  // namespace xred
