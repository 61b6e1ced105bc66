// xred_dispatch.hpp -- host-side mapping of (xred_dtype, xred_op) onto the
// element types and operators of the kernel templates.
#pragma once

#include "xred_device.hpp"
#include "../../include/xred.h"

namespace xred {

// Calls f(T{}) with dtype's element type.
template <class F>
hipError_t with_dtype(xred_dtype dtype, F &&f)
{
    switch (dtype) {
    case XRED_FLOAT32: return f(TF32{});
    case XRED_BFLOAT16: return f(TBF16{});
    case XRED_FLOAT16: return f(TF16{});
    case XRED_INT32: return f(TI32{});
    case XRED_UINT32: return f(TU32{});
    case XRED_INT64: return f(TI64{});
    case XRED_UINT64: return f(TU64{});
    case XRED_FP8_E4M3: return f(TE4M3{});
    case XRED_FP8_E5M2: return f(TE5M2{});
    case XRED_FLOAT64: return f(TF64{});
    case XRED_INT8: return f(TI8{});
    case XRED_UINT8: return f(TU8{});
    }
    return hipErrorInvalidValue;
}

template <class T> constexpr xred_dtype dtype_of();
template <> constexpr xred_dtype dtype_of<TF32>() { return XRED_FLOAT32; }
template <> constexpr xred_dtype dtype_of<TBF16>() { return XRED_BFLOAT16; }
template <> constexpr xred_dtype dtype_of<TF16>() { return XRED_FLOAT16; }
template <> constexpr xred_dtype dtype_of<TI32>() { return XRED_INT32; }
template <> constexpr xred_dtype dtype_of<TU32>() { return XRED_UINT32; }
template <> constexpr xred_dtype dtype_of<TI64>() { return XRED_INT64; }
template <> constexpr xred_dtype dtype_of<TU64>() { return XRED_UINT64; }
template <> constexpr xred_dtype dtype_of<TE4M3>() { return XRED_FP8_E4M3; }
template <> constexpr xred_dtype dtype_of<TE5M2>() { return XRED_FP8_E5M2; }
template <> constexpr xred_dtype dtype_of<TF64>() { return XRED_FLOAT64; }
template <> constexpr xred_dtype dtype_of<TI8>() { return XRED_INT8; }
template <> constexpr xred_dtype dtype_of<TU8>() { return XRED_UINT8; }

// Calls f(T{}) for the one T among Ts whose dtype is `dtype` (instantiating
// f only for Ts, so a translation unit can hold one group of types).
template <class... Ts, class F>
hipError_t with_dtype_among(xred_dtype dtype, F &&f)
{
    hipError_t r = hipErrorInvalidValue;
    (void)((dtype == dtype_of<Ts>() ? (r = f(Ts{}), true) : false) || ...);
    return r;
}

// The four groups the big launchers are compiled in.
enum class TypeGroup { kFloat, kFp8, kInt, kExt };
inline TypeGroup group_of(xred_dtype dtype)
{
    switch (dtype) {
    case XRED_FLOAT32: case XRED_BFLOAT16: case XRED_FLOAT16: return TypeGroup::kFloat;
    case XRED_FP8_E4M3: case XRED_FP8_E5M2: return TypeGroup::kFp8;
    case XRED_FLOAT64: case XRED_INT8: case XRED_UINT8: return TypeGroup::kExt;
    default: return TypeGroup::kInt;
    }
}

// Calls f(Op{}) with op's operator.  AVG exists only for float element types
// and only where WITH_AVG (launchers whose kernels see the whole fold).
template <class T, bool WITH_AVG, class F>
hipError_t with_op(xred_op op, F &&f)
{
    switch (op) {
    case XRED_SUM: return f(OpSum{});
    case XRED_PROD: return f(OpProd{});
    case XRED_MAX: return f(OpMax{});
    case XRED_MIN: return f(OpMin{});
    case XRED_AVG:
        if constexpr (WITH_AVG && T::kFloat) return f(OpAvg{});
        else return hipErrorInvalidValue;
    }
    return hipErrorInvalidValue;
}

// fp32, bf16, int32 and uint32 keep every compile-time source-count
// specialisation (1..8 and the pipelined 16/32/64); the other element types
// and AVG use 1..8 and the runtime group loop, which bounds the number of
// kernels in the library.
template <class T>
constexpr bool is_core_type()
{
    return __is_same(T, TF32) || __is_same(T, TBF16) || __is_same(T, TI32) || __is_same(T, TU32);
}

}  // namespace xred
