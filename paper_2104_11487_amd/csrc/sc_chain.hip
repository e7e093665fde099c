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

// Workgroup w takes blocks [w * bpw, (w + 1) * bpw) of the flattened block grid
// (bpw = max(1, kEmitSites / b^2)); each thread walks (site, channel) elements.
__global__ void __launch_bounds__(kEmitThreads)
emit_kernel(const uint8_t* block_mask, uint8_t* prev_mask, int nb, int bpw, const float* z, void* y,
            float* r32, uint16_t* rb, int hb, int wb, int block, int h_out, int w_out, int c_out, int act,
            int dtype) {
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
  // elements in groups of VEC consecutive channels (4 when c_out % 4 == 0)
  const int vec = (c_out & 3) == 0 ? 4 : 1;
  const int cg = c_out / vec;
  const int total = nblk * bsz * cg;
  for (int e = threadIdx.x; e < total; e += kEmitThreads) {
    const int bl = e / (bsz * cg), rem0 = e - bl * bsz * cg;
    const uint8_t st = state[bl];
    if (!st) continue;
    const int site = rem0 / cg, ch = (rem0 - site * cg) * vec;
    const int blk = b0 + bl;
    const int img = blk / (hb * wb), rem = blk - img * hb * wb;
    const int bi = rem / wb, bj = rem - bi * wb;
    const int oy = bi * block + site / block, ox = bj * block + site % block;
    if (oy >= h_out || ox >= w_out) continue;  // ceil-mode edge block
    const size_t o = ((size_t)(img * h_out + oy) * w_out + ox) * c_out + ch;
    for (int v = 0; v < vec; ++v) {
      if (!(st & 1)) {
        r32[o + v] = 0.0f;
        if (dtype == 1) rb[o + v] = 0;
        continue;
      }
      float a = z[o + v];
      if (act == 2) a = relu_f32(a);
      float r;
      if (dtype == 1) {
        uint16_t* yb = static_cast<uint16_t*>(y);
        const uint16_t yn = (uint16_t)f32_to_bf16(a);
        r = __fsub_rn(bf16_to_f32(yn), bf16_to_f32(yb[o + v]));
        yb[o + v] = yn;
        rb[o + v] = (uint16_t)f32_to_bf16(r);
      } else {
        float* yf = static_cast<float*>(y);
        r = __fsub_rn(a, yf[o + v]);
        yf[o + v] = a;
      }
      r32[o + v] = r;
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nblk; i += kEmitThreads) prev_mask[b0 + i] = state[i] & 1;
}

}  // namespace

hipError_t launch_emit(const uint8_t* block_mask, uint8_t* prev_mask, int nb, const float* z, void* y,
                       float* r32, uint16_t* rb, int n, int hb, int wb, int block, int h_out, int w_out,
                       int c_out, int act, int dtype, hipStream_t st) {
  (void)n;
  const int bpw = max(1, kEmitSites / (block * block));
  const int grid = (nb + bpw - 1) / bpw;
  hipLaunchKernelGGL(emit_kernel, dim3(grid), dim3(kEmitThreads), 0, st, block_mask, prev_mask, nb, bpw, z, y,
                     r32, rb, hb, wb, block, h_out, w_out, c_out, act, dtype);
  return hipGetLastError();
}

}  // namespace sc
