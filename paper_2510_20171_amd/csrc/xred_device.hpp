// xred_device.hpp -- device-side element types, operators and 16-byte vector
// conversions for the reduce-step kernels (gfx950).
//
// Every kernel computes, per element, a left fold in source order of
// up-converted values followed by one down-conversion (the per-rank reduce of
// the FTAR ring's ReduceCopy, Section 5).  This header fixes what up(), the
// operators and down() are on the device:
//   bf16 -> binary32 by a 16-bit shift (exact); binary32 -> bf16 with the
//   hardware round-to-nearest-even conversion v_cvt_pk_bf16_f32;
//   float MAX/MIN with the IEEE 754-2019 maximum/minimum operations
//   (v_maximum3_f32 / v_minimum3_f32: NaN-propagating, -0 < +0), the NaN
//   result then replaced by the quiet NaN 0x7FC00000;
//   integer SUM/PROD on uint32 (wrap modulo 2^32), MAX/MIN signed for int32.
// All code here is compiled without contraction and with binary32 subnormals
// enabled, so a float add or multiply is exactly one IEEE operation.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xred {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kBlock = 256;   // threads per workgroup: 4 wavefronts of 64

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

struct OpSum {};
struct OpProd {};
struct OpMax {};
struct OpMin {};

// ------------------------------------------------------------- operators --
template <class T, class Op>
__device__ __forceinline__ typename T::Acc combine(typename T::Acc a, typename T::Acc b)
{
    if constexpr (T::kFloat) {
        if constexpr (__is_same(Op, OpSum)) return a + b;
        else if constexpr (__is_same(Op, OpProd)) return a * b;
        else if constexpr (__is_same(Op, OpMax)) return __builtin_elementwise_maximum(a, b);
        else return __builtin_elementwise_minimum(a, b);
    } else {
        if constexpr (__is_same(Op, OpSum)) return a + b;
        else if constexpr (__is_same(Op, OpProd)) return a * b;
        else if constexpr (T::kSigned) {
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
    if constexpr (T::kFloat && (__is_same(Op, OpMax) || __is_same(Op, OpMin)))
        return __builtin_isnan(a) ? __uint_as_float(0x7FC00000u) : a;
    else
        return a;
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
    } else if constexpr (T::kFloat) {
#pragma unroll
        for (int j = 0; j < 4; ++j) a[j] = __uint_as_float(v[j]);
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
    } else if constexpr (T::kFloat) {
#pragma unroll
        for (int j = 0; j < 4; ++j) r[j] = __float_as_uint(finalize<T, Op>(a[j]));
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
    else if constexpr (T::kFloat)
        return ((const float *)base)[i];
    else
        return ((const uint32_t *)base)[i];
}

template <class T, class Op>
__device__ __forceinline__ void down1(char *base, size_t i, typename T::Acc a)
{
    a = finalize<T, Op>(a);
    if constexpr (__is_same(T, TBF16)) {
        f32x2 f = {a, a};
        ((uint16_t *)base)[i] =
            (uint16_t)__builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
    } else if constexpr (T::kFloat) {
        ((float *)base)[i] = a;
    } else {
        ((uint32_t *)base)[i] = a;
    }
}

// ----------------------------------------------------------- memory ops --
template <bool NT>
__device__ __forceinline__ u32x4 load16(const char *p)
{
    if constexpr (NT) return __builtin_nontemporal_load((const u32x4 *)p);
    else return *(const u32x4 *)p;
}

template <bool NT>
__device__ __forceinline__ void store16(char *p, u32x4 v)
{
    if constexpr (NT) __builtin_nontemporal_store(v, (u32x4 *)p);
    else *(u32x4 *)p = v;
}

}  // namespace xred
