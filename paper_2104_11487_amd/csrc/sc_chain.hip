// Residual emission for chained layers (sparse residual propagation).
//
// When layer l feeds layer l+1, layer l+1's input is dtype(act(z_l)) and its
// residual (Eq. 2) is that activation's change from the previous frame. The
// activation changes only at the sites layer l updated (Eq. 3: skipped sites
// keep z), so layer l can hand its successor the residual directly:
//   r = fl32(y_new - y_old) at the blocks layer l updated this step,
//   r = 0                   at the blocks it updated on the previous step only,
// with y = dtype(act(z)). For bf16 layers r is also stored rounded to bf16 (the
// successor's convolution operand), so the successor forms exactly the
// residual and operand that x_t - x_{t-1} would give it, and its gate can skip
// every tile whose input region holds no active upstream block.
#include "sc_device.h"
#include "sc_kernels.h"

namespace sc {

namespace {

constexpr int kEmitThreads = 256;
constexpr int kEmitSites = 64;  // output sites (whole blocks) per workgroup, at least one block
constexpr int kEmitUnroll = 4;  // 8-channel groups a thread has in flight (bf16 layers)

// Workgroup w takes blocks [w * bpw, (w + 1) * bpw) of the flattened block grid
// (bpw = max(1, kEmitSites / b^2)); each thread walks (site, channel) elements.
__global__ void __launch_bounds__(kEmitThreads)
emit_kernel(const uint8_t* block_mask, uint8_t* prev_mask, int nb, int bpw, const float* z, void* y,
            float* r32, uint16_t* rb, int hb, int wb, int block, int h_out, int w_out, int c_out, int act,
            int dtype, int clear_only) {
  __shared__ uint8_t state[kEmitSites];  // bit 0: updated now, bit 1: updated by the previous step
  const int b0 = blockIdx.x * bpw, nblk = min(bpw, nb - b0);
  int any = 0;
  for (int i = threadIdx.x; i < nblk; i += kEmitThreads) {
    const uint8_t st = (block_mask[b0 + i] ? 1 : 0) | (prev_mask[b0 + i] ? 2 : 0);
    state[i] = st;
    any |= st;
  }
  if (!__syncthreads_or(any)) return;
  const int bsz = block * block;
  // elements in groups of VEC consecutive channels: 8 (16-byte y / rb and
  // 32-byte z / r32 accesses) when c_out % 8 == 0, else 1
  const int vec = (c_out & 7) == 0 ? 8 : 1;
  const int cg = c_out / vec;
  const int total = nblk * bsz * cg;
  if (vec == 8 && dtype == 1) {
    // bf16 layers: kEmitUnroll groups per thread in flight (their z and y
    // loads issued together), then computed and stored
    constexpr int U = kEmitUnroll;
    uint16_t* yb = static_cast<uint16_t*>(y);
    for (int e0 = threadIdx.x; e0 < total; e0 += kEmitThreads * U) {
      size_t o[U];
      uint8_t stu[U];
      float4 z0[U], z1[U];
      uint4 yo[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int e = e0 + u * kEmitThreads;
        stu[u] = 0;
        o[u] = 0;
        if (e < total) {
          const int bl = e / (bsz * cg), rem0 = e - bl * bsz * cg;
          const int site = rem0 / cg, ch = (rem0 - site * cg) * 8;
          const int blk = b0 + bl;
          const int img = blk / (hb * wb), rem = blk - img * hb * wb;
          const int bi = rem / wb, bj = rem - bi * wb;
          const int oy = bi * block + site / block, ox = bj * block + site % block;
          if (oy < h_out && ox < w_out) {  // ceil-mode edge block
            // clear_only: the convolution already emitted at the updated blocks
            stu[u] = (clear_only && (state[bl] & 1)) ? 0 : state[bl];
            o[u] = ((size_t)(img * h_out + oy) * w_out + ox) * c_out + ch;
          }
        }
        if (stu[u] & 1) {
          z0[u] = *reinterpret_cast<const float4*>(z + o[u]);
          z1[u] = *reinterpret_cast<const float4*>(z + o[u] + 4);
          yo[u] = *reinterpret_cast<const uint4*>(yb + o[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (!stu[u]) continue;
        if (!(stu[u] & 1)) {
          *reinterpret_cast<float4*>(r32 + o[u]) = float4{0.f, 0.f, 0.f, 0.f};
          *reinterpret_cast<float4*>(r32 + o[u] + 4) = float4{0.f, 0.f, 0.f, 0.f};
          *reinterpret_cast<uint4*>(rb + o[u]) = uint4{0u, 0u, 0u, 0u};
          continue;
        }
        float a[8] = {z0[u].x, z0[u].y, z0[u].z, z0[u].w, z1[u].x, z1[u].y, z1[u].z, z1[u].w};
        if (act == 2)
          for (int v = 0; v < 8; ++v) a[v] = relu_f32(a[v]);
        const uint32_t wo[4] = {yo[u].x, yo[u].y, yo[u].z, yo[u].w};
        float r[8];
        uint32_t wn[4], wr[4];
        for (int v = 0; v < 4; ++v) {
          const uint32_t n0 = f32_to_bf16(a[2 * v]), n1 = f32_to_bf16(a[2 * v + 1]);
          r[2 * v] = __fsub_rn(bf16_to_f32(n0), bf16_to_f32(wo[v] & 0xffffu));
          r[2 * v + 1] = __fsub_rn(bf16_to_f32(n1), bf16_to_f32(wo[v] >> 16));
          wn[v] = n0 | (n1 << 16);
          wr[v] = f32_to_bf16(r[2 * v]) | (f32_to_bf16(r[2 * v + 1]) << 16);
        }
        *reinterpret_cast<uint4*>(yb + o[u]) = uint4{wn[0], wn[1], wn[2], wn[3]};
        *reinterpret_cast<uint4*>(rb + o[u]) = uint4{wr[0], wr[1], wr[2], wr[3]};
        *reinterpret_cast<float4*>(r32 + o[u]) = float4{r[0], r[1], r[2], r[3]};
        *reinterpret_cast<float4*>(r32 + o[u] + 4) = float4{r[4], r[5], r[6], r[7]};
      }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nblk; i += kEmitThreads) prev_mask[b0 + i] = state[i] & 1;
    return;
  }
  for (int e = threadIdx.x; e < total; e += kEmitThreads) {
    const int bl = e / (bsz * cg), rem0 = e - bl * bsz * cg;
    const uint8_t st = (clear_only && (state[bl] & 1)) ? 0 : state[bl];
    if (!st) continue;
    const int site = rem0 / cg, ch = (rem0 - site * cg) * vec;
    const int blk = b0 + bl;
    const int img = blk / (hb * wb), rem = blk - img * hb * wb;
    const int bi = rem / wb, bj = rem - bi * wb;
    const int oy = bi * block + site / block, ox = bj * block + site % block;
    if (oy >= h_out || ox >= w_out) continue;  // ceil-mode edge block
    const size_t o = ((size_t)(img * h_out + oy) * w_out + ox) * c_out + ch;
    if (vec == 8) {
      if (!(st & 1)) {
        *reinterpret_cast<float4*>(r32 + o) = float4{0.f, 0.f, 0.f, 0.f};
        *reinterpret_cast<float4*>(r32 + o + 4) = float4{0.f, 0.f, 0.f, 0.f};
        if (dtype == 1) *reinterpret_cast<uint4*>(rb + o) = uint4{0u, 0u, 0u, 0u};
        continue;
      }
      const float4 z0 = *reinterpret_cast<const float4*>(z + o), z1 = *reinterpret_cast<const float4*>(z + o + 4);
      float a[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
      if (act == 2)
        for (int v = 0; v < 8; ++v) a[v] = relu_f32(a[v]);
      float r[8];
      if (dtype == 1) {
        uint16_t* yb = static_cast<uint16_t*>(y);
        const uint4 yo = *reinterpret_cast<const uint4*>(yb + o);
        const uint32_t wo[4] = {yo.x, yo.y, yo.z, yo.w};
        uint32_t wn[4], wr[4];
        for (int v = 0; v < 4; ++v) {
          const uint32_t n0 = f32_to_bf16(a[2 * v]), n1 = f32_to_bf16(a[2 * v + 1]);
          r[2 * v] = __fsub_rn(bf16_to_f32(n0), bf16_to_f32(wo[v] & 0xffffu));
          r[2 * v + 1] = __fsub_rn(bf16_to_f32(n1), bf16_to_f32(wo[v] >> 16));
          wn[v] = n0 | (n1 << 16);
          wr[v] = f32_to_bf16(r[2 * v]) | (f32_to_bf16(r[2 * v + 1]) << 16);
        }
        *reinterpret_cast<uint4*>(yb + o) = uint4{wn[0], wn[1], wn[2], wn[3]};
        *reinterpret_cast<uint4*>(rb + o) = uint4{wr[0], wr[1], wr[2], wr[3]};
      } else {
        float* yf = static_cast<float*>(y);
        const float4 y0 = *reinterpret_cast<const float4*>(yf + o), y1 = *reinterpret_cast<const float4*>(yf + o + 4);
        const float yo[8] = {y0.x, y0.y, y0.z, y0.w, y1.x, y1.y, y1.z, y1.w};
        for (int v = 0; v < 8; ++v) r[v] = __fsub_rn(a[v], yo[v]);
        *reinterpret_cast<float4*>(yf + o) = float4{a[0], a[1], a[2], a[3]};
        *reinterpret_cast<float4*>(yf + o + 4) = float4{a[4], a[5], a[6], a[7]};
      }
      *reinterpret_cast<float4*>(r32 + o) = float4{r[0], r[1], r[2], r[3]};
      *reinterpret_cast<float4*>(r32 + o + 4) = float4{r[4], r[5], r[6], r[7]};
      continue;
    }
    if (!(st & 1)) {
      r32[o] = 0.0f;
      if (dtype == 1) rb[o] = 0;
      continue;
    }
    float a = z[o];
    if (act == 2) a = relu_f32(a);
    float r;
    if (dtype == 1) {
      uint16_t* yb = static_cast<uint16_t*>(y);
      const uint16_t yn = (uint16_t)f32_to_bf16(a);
      r = __fsub_rn(bf16_to_f32(yn), bf16_to_f32(yb[o]));
      yb[o] = yn;
      rb[o] = (uint16_t)f32_to_bf16(r);
    } else {
      float* yf = static_cast<float*>(y);
      r = __fsub_rn(a, yf[o]);
      yf[o] = a;
    }
    r32[o] = r;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nblk; i += kEmitThreads) prev_mask[b0 + i] = state[i] & 1;
}

}  // namespace

hipError_t launch_emit(const uint8_t* block_mask, uint8_t* prev_mask, int nb, const float* z, void* y,
                       float* r32, uint16_t* rb, int n, int hb, int wb, int block, int h_out, int w_out,
                       int c_out, int act, int dtype, int clear_only, hipStream_t st) {
  (void)n;
  const int bpw = max(1, kEmitSites / (block * block));
  const int grid = (nb + bpw - 1) / bpw;
  hipLaunchKernelGGL(emit_kernel, dim3(grid), dim3(kEmitThreads), 0, st, block_mask, prev_mask, nb, bpw, z, y,
                     r32, rb, hb, wb, block, h_out, w_out, c_out, act, dtype, clear_only);
  return hipGetLastError();
}

}  // namespace sc
