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

__global__ void __launch_bounds__(kEmitThreads)
emit_kernel(const uint8_t* block_mask, uint8_t* prev_mask, const float* z, void* y, float* r32,
            uint16_t* rb, int hb, int wb, int block, int h_out, int w_out, int c_out, int act, int dtype) {
  const int blk = blockIdx.x;
  const bool cur = block_mask[blk] != 0, was = prev_mask[blk] != 0;
  if (!cur && !was) return;
  const int img = blk / (hb * wb), rem = blk - img * hb * wb;
  const int bi = rem / wb, bj = rem - bi * wb;
  const int oy0 = bi * block, ox0 = bj * block;
  const int bh = min(block, h_out - oy0), bw = min(block, w_out - ox0);
  const int total = bh * bw * c_out;
  for (int i = threadIdx.x; i < total; i += kEmitThreads) {
    const int site = i / c_out, ch = i - site * c_out;
    const int ly = site / bw, lx = site - ly * bw;
    const size_t o = ((size_t)(img * h_out + oy0 + ly) * w_out + ox0 + lx) * c_out + ch;
    if (!cur) {
      r32[o] = 0.0f;
      if (dtype == 1) rb[o] = 0;
      continue;
    }
    float v = z[o];
    if (act == 2) v = fmaxf(v, 0.0f);
    float r;
    if (dtype == 1) {
      uint16_t* yb = static_cast<uint16_t*>(y);
      const uint16_t yn = (uint16_t)f32_to_bf16(v);
      r = __fsub_rn(bf16_to_f32(yn), bf16_to_f32(yb[o]));
      yb[o] = yn;
      rb[o] = (uint16_t)f32_to_bf16(r);
    } else {
      float* yf = static_cast<float*>(y);
      r = __fsub_rn(v, yf[o]);
      yf[o] = v;
    }
    r32[o] = r;
  }
  __syncthreads();
  if (threadIdx.x == 0) prev_mask[blk] = cur ? 1 : 0;
}

}  // namespace

hipError_t launch_emit(const uint8_t* block_mask, uint8_t* prev_mask, int nb, const float* z, void* y,
                       float* r32, uint16_t* rb, int n, int hb, int wb, int block, int h_out, int w_out,
                       int c_out, int act, int dtype, hipStream_t st) {
  (void)n;
  hipLaunchKernelGGL(emit_kernel, dim3(nb), dim3(kEmitThreads), 0, st, block_mask, prev_mask, z, y, r32, rb,
                     hb, wb, block, h_out, w_out, c_out, act, dtype);
  return hipGetLastError();
}

}  // namespace sc
