// Device-side helpers shared by the Skip-Conv kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// bf16 values are carried as raw 16-bit patterns (the top half of an fp32).
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// fp32 -> bf16, round to nearest with ties to even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return ((u >> 16) | 0x40u) & 0xffffu;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Storage traits: element type, and a vector of 8 elements widened to fp32.
template <typename T> struct Elem;

template <> struct Elem<float> {
  static constexpr int kBytes = 4;
  __device__ __forceinline__ static float load1(const float* p, size_t i) { return p[i]; }
  __device__ __forceinline__ static void load4(const float* p, size_t i, float* v) {
    float4 a = *reinterpret_cast<const float4*>(p + i);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  }
  __device__ __forceinline__ static void load8(const float* p, size_t i, float* v) {
    load4(p, i, v);
    load4(p, i + 4, v + 4);
  }
  __device__ __forceinline__ static void store1(float* p, size_t i, float v) { p[i] = v; }
};

template <> struct Elem<uint16_t> {
  static constexpr int kBytes = 2;
  __device__ __forceinline__ static float load1(const uint16_t* p, size_t i) {
    return bf16_to_f32(p[i]);
  }
  __device__ __forceinline__ static void load8(const uint16_t* p, size_t i, float* v) {
    uint4 a = *reinterpret_cast<const uint4*>(p + i);
    uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[2 * j] = __uint_as_float(w[j] << 16);
      v[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
    }
  }
  __device__ __forceinline__ static void load4(const uint16_t* p, size_t i, float* v) {
    uint2 a = *reinterpret_cast<const uint2*>(p + i);
    v[0] = __uint_as_float(a.x << 16);
    v[1] = __uint_as_float(a.x & 0xffff0000u);
    v[2] = __uint_as_float(a.y << 16);
    v[3] = __uint_as_float(a.y & 0xffff0000u);
  }
  __device__ __forceinline__ static void store1(uint16_t* p, size_t i, float v) {
    p[i] = (uint16_t)f32_to_bf16(v);
  }
};

// ReLU of the activation output: v for v > 0 and for NaN (a NaN state stays
// visible to the next layer), +0 otherwise (also for -0).
__device__ __forceinline__ float relu_f32(float v) { return (v > 0.0f || __builtin_isnan(v)) ? v : 0.0f; }

// Exact IEEE single-precision operations with no contraction into FMA: the
// gate statistic must round once per multiply and once per add.
__device__ __forceinline__ float mul_rn(float a, float b) { return __fmul_rn(a, b); }
__device__ __forceinline__ float add_rn(float a, float b) { return __fadd_rn(a, b); }

}  // namespace sc
