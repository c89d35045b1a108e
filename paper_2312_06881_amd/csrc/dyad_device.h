// Device-side helpers shared by the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dyad {

// bf16 is carried as its raw 16 bits.
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// fp32 -> bf16, round to nearest even; NaN stays a (quiet) NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ float load_f32(const T *p, int64_t i);
template <> __device__ __forceinline__ float load_f32<float>(const float *p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ float load_f32<uint16_t>(const uint16_t *p, int64_t i) {
    return bf16_to_f32(p[i]);
}

template <typename T> __device__ __forceinline__ void store_f32(T *p, int64_t i, float v);
template <> __device__ __forceinline__ void store_f32<float>(float *p, int64_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void store_f32<uint16_t>(uint16_t *p, int64_t i, float v) {
    p[i] = f32_to_bf16(v);
}

// GELU(x) = x * Phi(x), Phi(x) = erfc(-x / sqrt 2) / 2.
__device__ __forceinline__ float gelu_f32(float x) { return 0.5f * x * erfcf(-x * 0.70710678118654752f); }

// GELU'(x) = Phi(x) + x * phi(x).
__device__ __forceinline__ float gelu_grad_f32(float x) {
    return 0.5f * erfcf(-x * 0.70710678118654752f) + x * 0.39894228040143268f * expf(-0.5f * x * x);
}

}  // namespace dyad
