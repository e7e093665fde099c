// Translation-compensated step (Sec. 3.3 with the warp T a known integer
// translation d of the content): r = x_t - T(x_{t-1}), z = T~(z_{t-1}) + w * r,
// T~ the translation by d / stride on the output grid, zero fill for both.
// Convolution commutes with the translation except on "exposed" output lines
// (line_exposed); blocks holding an exposed site are recomputed from x_t.
//
//   translate_state_kernel  z_dst[o] = z_src[o - d_out] (0 outside), and the
//                           activation output refreshed from it (optionally
//                           only outside the step's active blocks, which the
//                           block-halo convolution writes itself);
//   split_list_kernel       the step's ordered active list split into the
//                           blocks that follow the translated recurrence and
//                           the exposed blocks recomputed from x_t.
#include "sc_device.h"
#include "sc_kernels.h"

namespace sc {

namespace {

constexpr int kTrThreads = 256;

// One thread per VEC consecutive channels of one site (VEC = 4: 16-byte
// loads and stores), one grid row per output row (blockIdx.y = image row):
// 32-bit index arithmetic, one division per thread.
template <int VEC>
__global__ void __launch_bounds__(kTrThreads)
translate_state_kernel(const float* z_src, float* z_dst, void* y, int row0, int h_out, int w_out, int c_out,
                       int dyo, int dxo, int act, int dtype, const uint8_t* skip_mask, int block, int hb, int wb) {
  const int cg = c_out / VEC;
  const int e = blockIdx.x * kTrThreads + threadIdx.x;
  if (e >= w_out * cg) return;
  const int row = row0 + (int)blockIdx.y;  // image * h_out + oy
  const int img = row / h_out, oy = row - img * h_out;
  const int ox = e / cg, ch = (e - ox * cg) * VEC;
  // sites of active blocks are written by the step's convolution
  if (skip_mask && skip_mask[((size_t)img * hb + oy / block) * wb + ox / block]) return;
  const int sy = oy - dyo, sx = ox - dxo;
  const bool in = sy >= 0 && sy < h_out && sx >= 0 && sx < w_out;
  const size_t o = ((size_t)row * w_out + ox) * c_out + ch;
  const size_t so = (((size_t)img * h_out + sy) * w_out + sx) * c_out + ch;
  float zv[VEC];
  if constexpr (VEC == 4) {
    const float4 v = in ? *reinterpret_cast<const float4*>(z_src + so) : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    zv[0] = v.x; zv[1] = v.y; zv[2] = v.z; zv[3] = v.w;
    *reinterpret_cast<float4*>(z_dst + o) = v;
  } else {
    zv[0] = in ? z_src[so] : 0.0f;
    z_dst[o] = zv[0];
  }
  if (act) {
    float a[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) a[v] = act == 2 ? relu_f32(zv[v]) : zv[v];
    if (dtype == 1) {
      uint16_t* yb = static_cast<uint16_t*>(y) + o;
      if constexpr (VEC == 4) {
        const uint2 pk = make_uint2((uint32_t)f32_to_bf16(a[0]) | ((uint32_t)f32_to_bf16(a[1]) << 16),
                                    (uint32_t)f32_to_bf16(a[2]) | ((uint32_t)f32_to_bf16(a[3]) << 16));
        *reinterpret_cast<uint2*>(yb) = pk;
      } else {
        yb[0] = (uint16_t)f32_to_bf16(a[0]);
      }
    } else {
      float* yf = static_cast<float*>(y) + o;
      if constexpr (VEC == 4) *reinterpret_cast<float4*>(yf) = make_float4(a[0], a[1], a[2], a[3]);
      else yf[0] = a[0];
    }
  }
}

// One workgroup: list[0..count) -> list_a (translated recurrence) and list_b
// (exposed blocks); counts at counters_a[kCtrCount], counters_b[kCtrCount].
// A block is exposed when one of its output rows or columns is: the flags of
// every block row and block column are formed first (each line tested once),
// so a listed block costs two LDS reads.
constexpr int kSplitMaxLines = 4096;
__global__ void __launch_bounds__(1024)
split_list_kernel(const uint32_t* list, const uint32_t* counters, int seg_tiles, int seg_cap, uint32_t* list_a,
                  uint32_t* counters_a, uint32_t* list_b, uint32_t* counters_b, int hb, int wb, int block,
                  int h_out, int w_out, int h, int w, int k, int stride, int pad, int sy, int sx) {
  __shared__ uint32_t na, nb_;
  __shared__ uint8_t row_ex[kSplitMaxLines], col_ex[kSplitMaxLines];
  if (threadIdx.x == 0) na = nb_ = 0;
  const bool tables = hb <= kSplitMaxLines && wb <= kSplitMaxLines;
  if (tables) {
    for (int bi = threadIdx.x; bi < hb; bi += blockDim.x) {
      bool ex = false;
      for (int r = bi * block; r < min((bi + 1) * block, h_out) && !ex; ++r)
        ex = line_exposed(r, h_out, h, k, stride, pad, sy);
      row_ex[bi] = ex ? 1 : 0;
    }
    for (int bj = threadIdx.x; bj < wb; bj += blockDim.x) {
      bool ex = false;
      for (int c = bj * block; c < min((bj + 1) * block, w_out) && !ex; ++c)
        ex = line_exposed(c, w_out, w, k, stride, pad, sx);
      col_ex[bj] = ex ? 1 : 0;
    }
  }
  __syncthreads();
  const WorkList W = work_list(counters, seg_tiles, seg_cap);
  const uint32_t count = W.total;
  for (uint32_t i = threadIdx.x; i < count; i += blockDim.x) {
    const uint32_t blk = list[work_pos(W, i)];
    const int rem = (int)(blk % (uint32_t)(hb * wb));
    const int bi = rem / wb, bj = rem - bi * wb;
    bool ex = false;
    if (tables) {
      ex = row_ex[bi] != 0 || col_ex[bj] != 0;
    } else {
      for (int r = bi * block; r < min((bi + 1) * block, h_out) && !ex; ++r)
        ex = line_exposed(r, h_out, h, k, stride, pad, sy);
      for (int c = bj * block; c < min((bj + 1) * block, w_out) && !ex; ++c)
        ex = line_exposed(c, w_out, w, k, stride, pad, sx);
    }
    if (ex)
      list_b[atomicAdd(&nb_, 1u)] = blk;
    else
      list_a[atomicAdd(&na, 1u)] = blk;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    counters_a[kCtrCount] = na;
    counters_b[kCtrCount] = nb_;
  }
}

__global__ void fill_u32_kernel(uint32_t* p, int n, uint32_t v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

}  // namespace

// A kernel rather than hipMemsetAsync, so that the step stays capturable in a graph.
hipError_t launch_fill_u32(uint32_t* p, int n, uint32_t v, hipStream_t st) {
  hipLaunchKernelGGL(fill_u32_kernel, dim3((n + 255) / 256), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

hipError_t launch_translate_state(const float* z_src, float* z_dst, void* y, int n, int h_out, int w_out,
                                  int c_out, int dyo, int dxo, int act, int dtype, const uint8_t* skip_mask,
                                  int block, int hb, int wb, hipStream_t st) {
  const bool v4 = c_out % 4 == 0;
  const long per_row = (long)w_out * (v4 ? c_out / 4 : c_out);
  const long rows = (long)n * h_out;
  if (per_row >= (1L << 30) || rows >= (1L << 31)) return hipErrorInvalidValue;
  constexpr long kRowsPerLaunch = 65535;  // grid.y limit
  for (long r0 = 0; r0 < rows; r0 += kRowsPerLaunch) {
    const dim3 grid((unsigned)((per_row + kTrThreads - 1) / kTrThreads),
                    (unsigned)std::min<long>(rows - r0, kRowsPerLaunch));
    if (v4)
      hipLaunchKernelGGL(translate_state_kernel<4>, grid, dim3(kTrThreads), 0, st, z_src, z_dst, y, (int)r0, h_out,
                         w_out, c_out, dyo, dxo, act, dtype, skip_mask, block, hb, wb);
    else
      hipLaunchKernelGGL(translate_state_kernel<1>, grid, dim3(kTrThreads), 0, st, z_src, z_dst, y, (int)r0, h_out,
                         w_out, c_out, dyo, dxo, act, dtype, skip_mask, block, hb, wb);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_split_list(const uint32_t* list, const uint32_t* counters, int seg_tiles, int seg_cap,
                             uint32_t* list_a, uint32_t* counters_a, uint32_t* list_b, uint32_t* counters_b,
                             int hb, int wb, int block, int h_out, int w_out, int h, int w, int k, int stride,
                             int pad, int sy, int sx, hipStream_t st) {
  hipLaunchKernelGGL(split_list_kernel, dim3(1), dim3(1024), 0, st, list, counters, seg_tiles, seg_cap, list_a,
                     counters_a, list_b, counters_b, hb, wb, block, h_out, w_out, h, w, k, stride, pad, sy, sx);
  return hipGetLastError();
}

}  // namespace sc
