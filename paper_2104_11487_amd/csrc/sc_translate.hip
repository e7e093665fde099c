// Translation-compensated step (Sec. 3.3 with the warp T a known integer
// translation d of the content): r = x_t - T(x_{t-1}), z = T~(z_{t-1}) + w * r,
// T~ the translation by d / stride on the output grid, zero fill for both.
// Convolution commutes with the translation except on "exposed" output lines
// (line_exposed); blocks holding an exposed site are recomputed from x_t.
//
//   translate_state_kernel  z_dst[o] = z_src[o - d_out] (0 outside), and the
//                           activation output refreshed from it;
//   split_list_kernel       the step's ordered active list split into the
//                           blocks that follow the translated recurrence and
//                           the exposed blocks recomputed from x_t.
#include "sc_device.h"
#include "sc_kernels.h"

namespace sc {

namespace {

constexpr int kTrThreads = 256;

__global__ void __launch_bounds__(kTrThreads)
translate_state_kernel(const float* z_src, float* z_dst, void* y, int n, int h_out, int w_out, int c_out,
                       int dyo, int dxo, int act, int dtype) {
  const int vec = (c_out & 3) == 0 ? 4 : 1;
  const int cg = c_out / vec;
  const long total = (long)n * h_out * w_out * cg;
  for (long e = (long)blockIdx.x * kTrThreads + threadIdx.x; e < total; e += (long)gridDim.x * kTrThreads) {
    const long site = e / cg;
    const int ch = (int)(e - site * cg) * vec;
    const int img = (int)(site / ((long)h_out * w_out));
    const int rem = (int)(site - (long)img * h_out * w_out);
    const int oy = rem / w_out, ox = rem - oy * w_out;
    const int sy = oy - dyo, sx = ox - dxo;
    const bool in = sy >= 0 && sy < h_out && sx >= 0 && sx < w_out;
    const size_t o = (size_t)site * c_out + ch;
    const size_t so = (((size_t)img * h_out + sy) * w_out + sx) * c_out + ch;
    for (int v = 0; v < vec; ++v) {
      const float zv = in ? z_src[so + v] : 0.0f;
      z_dst[o + v] = zv;
      if (act) {
        const float a = act == 2 ? relu_f32(zv) : zv;
        if (dtype == 1)
          static_cast<uint16_t*>(y)[o + v] = (uint16_t)f32_to_bf16(a);
        else
          static_cast<float*>(y)[o + v] = a;
      }
    }
  }
}

// One workgroup: list[0..count) -> list_a (translated recurrence) and list_b
// (exposed blocks); counts at counters_a[kCtrCount], counters_b[kCtrCount].
__global__ void __launch_bounds__(1024)
split_list_kernel(const uint32_t* list, const uint32_t* counters, int seg_tiles, int seg_cap, uint32_t* list_a,
                  uint32_t* counters_a, uint32_t* list_b, uint32_t* counters_b, int hb, int wb, int block,
                  int h_out, int w_out, int h, int w, int k, int stride, int pad, int sy, int sx) {
  __shared__ uint32_t na, nb_;
  if (threadIdx.x == 0) na = nb_ = 0;
  __syncthreads();
  const WorkList W = work_list(counters, seg_tiles, seg_cap);
  const uint32_t count = W.total;
  for (uint32_t i = threadIdx.x; i < count; i += blockDim.x) {
    const uint32_t blk = list[work_pos(W, i)];
    const int rem = (int)(blk % (uint32_t)(hb * wb));
    const int bi = rem / wb, bj = rem - bi * wb;
    bool ex = false;
    for (int r = bi * block; r < min((bi + 1) * block, h_out) && !ex; ++r)
      ex = line_exposed(r, h_out, h, k, stride, pad, sy);
    for (int c = bj * block; c < min((bj + 1) * block, w_out) && !ex; ++c)
      ex = line_exposed(c, w_out, w, k, stride, pad, sx);
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
                                  int c_out, int dyo, int dxo, int act, int dtype, hipStream_t st) {
  const long total = (long)n * h_out * w_out * (c_out % 4 == 0 ? c_out / 4 : c_out);
  const int grid = (int)std::min<long>((total + kTrThreads - 1) / kTrThreads, 4096);
  hipLaunchKernelGGL(translate_state_kernel, dim3(grid), dim3(kTrThreads), 0, st, z_src, z_dst, y, n, h_out, w_out,
                     c_out, dyo, dxo, act, dtype);
  return hipGetLastError();
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
