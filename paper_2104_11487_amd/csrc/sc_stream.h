// Streaming helpers shared by the gate kernel and the fused gate+conv kernel:
// canonical per-pixel statistic, vector loads/copies, XCD-aware tile order.
#pragma once

#include "sc_device.h"

#pragma clang fp contract(off)

namespace sc {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kUnroll = 4;  // staging chunks whose loads are issued together

__device__ __forceinline__ float term(float r, int norm_p) {
  return norm_p == 2 ? mul_rn(r, r) : fabsf(r);
}

// Canonical order of the per-pixel statistic: channels in chunks of kChunk
// consecutive channels; within a chunk the terms are added in ascending
// order from +0; the chunk sums are then added in ascending chunk order.
constexpr int kChunk = 8;

// Ordered sum of the terms of up to kChunk consecutive channels (one chunk).
template <int N>
__device__ __forceinline__ float chunk_sum(const float* r, int norm_p) {
  float part = 0.0f;
#pragma unroll
  for (int i = 0; i < N; ++i) part = add_rn(part, term(r[i], norm_p));
  return part;
}

template <typename T, int VEC>
__device__ __forceinline__ void load_vec(const T* p, size_t off, float* v) {
  if (VEC == 8) {
    Elem<T>::load8(p, off, v);
  } else if (VEC == 4) {
    Elem<T>::load4(p, off, v);
  } else {
    v[0] = Elem<T>::load1(p, off);
  }
}

template <typename T, int VEC>
__device__ __forceinline__ void copy_vec(T* dst, const T* src, size_t off) {
  if (VEC * sizeof(T) == 16) {
    *reinterpret_cast<uint4*>(dst + off) = *reinterpret_cast<const uint4*>(src + off);
  } else if (VEC * sizeof(T) == 8) {
    *reinterpret_cast<uint2*>(dst + off) = *reinterpret_cast<const uint2*>(src + off);
  } else {
#pragma unroll
    for (int j = 0; j < VEC; ++j) dst[off + j] = src[off + j];
  }
}

// floor(n / d) for 0 <= n < 2^20 and d >= 1, given inv_d = 1 / d rounded to
// fp32 (within 2.5 ulp): (n + 1/2) / d is at least 1 / (2d) away from an
// integer, and the fp32 product lies within (n + 1/2) / d * 2^-21 < 1 / (2d)
// of it, so truncation gives the exact quotient. A few VALU operations instead
// of the long integer-division sequence.
__device__ __forceinline__ int qdiv(int n, float inv_d) {
  return (int)(((float)n + 0.5f) * inv_d);
}

// Value of lane (this lane + J) of the same 16-lane row (DPP row_shl:J).
template <int J>
__device__ __forceinline__ float row_shl(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x100 + J, 0xf, 0xf, false));
}

template <int NC, int J>
__device__ __forceinline__ float group_sum_from(float acc, float v) {
  if constexpr (J < NC) {
    return group_sum_from<NC, J + 1>(add_rn(acc, row_shl<J>(v)), v);
  } else {
    return acc;
  }
}

// Ordered sum (from +0, ascending lanes) of the NC values held by lanes
// l .. l + NC - 1 of one 16-lane row, valid in lane l (NC <= 16; the group
// must not cross a row boundary). Lane-to-lane moves only, no LDS traffic.
template <int NC>
__device__ __forceinline__ float group_sum(float v) {
  return group_sum_from<NC, 1>(add_rn(0.0f, v), v);
}

// Workgroup barrier that orders LDS accesses only: outstanding global loads
// and stores stay in flight. (A global_load_lds still in flight makes the
// compiler wait for it here.)
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Raw buffer resource over `bytes` bytes at `base`: a load at an offset at or
// beyond `bytes` returns zeros and a store there is dropped, without a memory
// access (range-checked buffer addressing of the CDNA ISA).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t frame_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
constexpr uint32_t kOutOfRange = 0x80000000u;  // byte offset past every frame resource

// Workgroup b runs tile remap(b): XCD b % 8 (workgroups go to the XCDs
// round-robin) receives a contiguous range of tiles, so neighbouring tiles
// share their halo rows through one L2.
__device__ __forceinline__ int xcd_tile(int b, int g) {
  const int per = g >> 3, rem = g & 7, x = b & 7;
  return x * per + min(x, rem) + (b >> 3);
}

}  // namespace sc
