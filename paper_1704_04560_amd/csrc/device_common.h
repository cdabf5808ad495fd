// Device-side helpers shared by the kernel files: the bfloat16 storage type and conversions.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace mtx {

// bfloat16 is stored as its 16-bit pattern; arithmetic always happens in fp32.
typedef uint16_t bf16_t;

__device__ __forceinline__ float bf16_to_f32(bf16_t h)
{
    return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// fp32 -> bfloat16, round to nearest even (gfx950 converts in hardware: v_cvt_pk_bf16_f32);
// NaN stays a (quiet) NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f)
{
    return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f));
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf16_to_f32(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }

}  // namespace mtx
