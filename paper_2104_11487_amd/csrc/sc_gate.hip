// Gate kernel of the Skip-Conv layer: residual, Input-Norm gate statistic,
// threshold, block pooling and ordered compaction, fused in one launch.
//
//   Eq. 2     r = x_t - x_{t-1} (x_{t-1} = 0 on a reference frame, Sec. 3.1)
//   Eq. 5     s[o] = norm of r over the kernel support of output o;
//             g[o] = s[o] > eps^2 (p = 2) or s[o] > eps (p = 1), or s NaN
//   Sec 3.2.2 block mask M[B] = OR of g over the b x b block B (ceil mode)
//   Sec 4.2   active list = ascending indices of active blocks (the
//             "non-sparse columns" of the im2col product)
//
// Statistic arithmetic is canonical so that masks are reproducible bit for
// bit: fp32 r; per pixel a[q] = sum over channels in ascending order (one
// rounding per multiply and per add, no FMA); s[o] = sum of a over the taps
// (kh, kw) in row-major order, in fp32; the threshold comparison in fp64.
//
// One workgroup owns a TS x TS tile of output sites (whole blocks). It loads
// the input halo of its tile in batches of rows with coalesced 16-byte loads
// (several in flight per thread), squares the residual into an LDS staging
// area laid out [pixel][channel] with 16-byte aligned pixel rows, and then one
// thread per halo pixel sums its channels in order, four per LDS read. Input pixels
// the tile owns are copied into the spare x_{t-1} slot on the way (ping-pong:
// the slot being read is never written in the same step). Every workgroup
// then writes its block flags. A second, one-workgroup kernel scans all
// block flags in index order and writes the active list and its length (a
// kernel boundary, rather than a device-wide counter, orders the two).
#include "sc_device.h"
#include "sc_kernels.h"
#include "sc_stream.h"

#pragma clang fp contract(off)

namespace sc {

namespace {

constexpr int kGateThreads = 256;
// Stage the per-channel terms of `rows` halo rows into LDS ([pixel][channel],
// cs floats per pixel). Loads of kUnroll chunks are issued before any is used.
template <typename T, int VEC>
__device__ void stage_rows(const GateParams& p, int n, int hb0, int rows, int iy0, int ix0, int hw,
                           int xs, int xe, int own_y0, int own_y1, int own_x0, int own_x1,
                           float* stage, int cs, bool copy_in_halo) {
  const T* xt = static_cast<const T*>(p.x_t);
  const T* xp = static_cast<const T*>(p.x_prev);
  T* keep = static_cast<T*>(p.x_keep);
  const int c = p.c;
  const int nchunk = (xe - xs) * c / VEC;
  const int total = rows * nchunk;
  for (int base = 0; base < total; base += kGateThreads * kUnroll) {
    float vt[kUnroll][VEC], vp[kUnroll][VEC];
    size_t off[kUnroll];
    int dst[kUnroll];
    bool valid[kUnroll], own[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int idx = base + u * kGateThreads + threadIdx.x;
      const int row = idx / nchunk;
      const int ch = idx - row * nchunk;
      const int y = iy0 + hb0 + row;
      valid[u] = idx < total && y >= 0 && y < p.h;
      const int e = ch * VEC;
      const int px = e / c;
      const int ci = e - px * c;
      const int x = xs + px;
      off[u] = valid[u] ? ((size_t)(n * p.h + y) * p.w + x) * c + ci : 0;
      dst[u] = (row * hw + (x - ix0)) * cs + ci;
      own[u] = copy_in_halo && y >= own_y0 && y < own_y1 && x >= own_x0 && x < own_x1;
      if (valid[u]) {
        load_vec<T, VEC>(xt, off[u], vt[u]);
        if (p.reference) {
#pragma unroll
          for (int j = 0; j < VEC; ++j) vp[u][j] = 0.0f;
        } else {
          load_vec<T, VEC>(xp, off[u], vp[u]);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (!valid[u]) continue;
      float tv[VEC];
#pragma unroll
      for (int j = 0; j < VEC; ++j) tv[j] = term(__fsub_rn(vt[u][j], vp[u][j]), p.norm_p);
      float* d = stage + dst[u];
      if (VEC % 4 == 0) {
#pragma unroll
        for (int j = 0; j < VEC; j += 4)
          *reinterpret_cast<float4*>(d + j) = make_float4(tv[j], tv[j + 1], tv[j + 2], tv[j + 3]);
      } else {
#pragma unroll
        for (int j = 0; j < VEC; ++j) d[j] = tv[j];
      }
      if (own[u]) copy_vec<T, VEC>(keep, xt, off[u]);
    }
  }
}

template <typename T, int VEC>
__global__ void __launch_bounds__(kGateThreads) gate_kernel(GateParams p) {
  extern __shared__ float lds[];
  __shared__ uint32_t blk_flag[kMaxTileBlocks];

  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int tiles_per_img = p.tiles_y * p.tiles_x;
  const int n = tile / tiles_per_img;
  const int trem = tile - n * tiles_per_img;
  const int ty = trem / p.tiles_x;
  const int tx = trem - ty * p.tiles_x;
  const int oy0 = ty * p.ts, ox0 = tx * p.ts;
  const int oh = min(p.ts, p.h_out - oy0), ow = min(p.ts, p.w_out - ox0);
  const int s = p.stride, k = p.k;
  const int iy0 = oy0 * s - p.pad, ix0 = ox0 * s - p.pad;
  const int hh = (oh - 1) * s + k, hw = (ow - 1) * s + k;
  const int xs = max(ix0, 0), xe = min(ix0 + hw, p.w);
  // input pixels this tile owns (copied to the spare x_{t-1} slot)
  const int own_y0 = oy0 * s, own_x0 = ox0 * s;
  const int own_y1 = (ty == p.tiles_y - 1) ? p.h : min(p.h, (oy0 + p.ts) * s);
  const int own_x1 = (tx == p.tiles_x - 1) ? p.w : min(p.w, (ox0 + p.ts) * s);

  float* a_halo = lds;                 // hh * hw
  float* stage = lds + p.halo_floats;  // rows_per_batch * hw * cs (16-byte aligned)
  const int cs = p.stage_stride;

  const int tb_w = p.ts / p.block;
  const int nblk_y = (oh + p.block - 1) / p.block, nblk_x = (ow + p.block - 1) / p.block;
  for (int i = threadIdx.x; i < kMaxTileBlocks; i += kGateThreads) blk_flag[i] = 0u;

  for (int hb0 = 0; hb0 < hh; hb0 += p.rows_per_batch) {
    const int rows = min(p.rows_per_batch, hh - hb0);
    if (xe > xs)
      stage_rows<T, VEC>(p, n, hb0, rows, iy0, ix0, hw, xs, xe, own_y0, own_y1, own_x0, own_x1, stage,
                         cs, p.copy_in_halo != 0);
    __syncthreads();
    for (int q = threadIdx.x; q < rows * hw; q += kGateThreads) {
      const int row = q / hw, col = q - row * hw;
      const int y = iy0 + hb0 + row, x = ix0 + col;
      float a = 0.0f;
      if (y >= 0 && y < p.h && x >= 0 && x < p.w) a = sum_channels(stage + (size_t)q * cs, p.c);
      a_halo[(hb0 + row) * hw + col] = a;
    }
    __syncthreads();
  }

  if (!p.copy_in_halo) {
    // x_{t-1} update for owned pixels no output support reaches
    const T* xt = static_cast<const T*>(p.x_t);
    T* keep = static_cast<T*>(p.x_keep);
    const int ny = own_y1 - own_y0, nx = own_x1 - own_x0;
    const int per_row = nx * p.c;
    for (int i = threadIdx.x; i < ny * per_row; i += kGateThreads) {
      const int yy = i / per_row, e = i - yy * per_row;
      const size_t off = ((size_t)(n * p.h + own_y0 + yy) * p.w + own_x0) * p.c + e;
      keep[off] = xt[off];
    }
  }

  // support statistic, threshold, block flags
  for (int q = threadIdx.x; q < oh * ow; q += kGateThreads) {
    const int ly = q / ow, lx = q - ly * ow;
    float sv;
    if (p.support == 0) {
      sv = 0.0f;
      const float* base = a_halo + (ly * s) * hw + lx * s;
      for (int kh = 0; kh < k; ++kh)
        for (int kw = 0; kw < k; ++kw) sv = add_rn(sv, base[kh * hw + kw]);
    } else {
      sv = a_halo[(ly * s + p.pad) * hw + lx * s + p.pad];
    }
    const bool on = p.reference || p.force_dense || ((double)sv > p.thr) || (sv != sv);
    if (p.keep_stats) {
      const size_t o = ((size_t)n * p.h_out + oy0 + ly) * p.w_out + ox0 + lx;
      p.stat[o] = sv;
      p.site_mask[o] = on ? 1 : 0;
    }
    if (on) blk_flag[(ly / p.block) * tb_w + lx / p.block] = 1u;
  }
  __syncthreads();

  const int bi0 = oy0 / p.block, bj0 = ox0 / p.block;
  for (int i = threadIdx.x; i < nblk_y * nblk_x; i += kGateThreads) {
    const int by = i / nblk_x, bx = i - by * nblk_x;
    p.block_mask[((size_t)n * p.hb + bi0 + by) * p.wb + bj0 + bx] = (uint8_t)blk_flag[by * tb_w + bx];
  }

}

// Ordered compaction (one workgroup of kScanThreads): each thread takes a
// contiguous run of 16-byte words of block flags (bytes 0/1, the buffer is
// zero-padded to whole words), counts them, the workgroup scans the counts,
// and every thread writes the indices of its active blocks in ascending order.
constexpr int kScanThreads = 1024;

__global__ void __launch_bounds__(kScanThreads) compact_kernel(const uint8_t* block_mask, int nb,
                                                               uint32_t* list, uint32_t* counters) {
  __shared__ uint32_t wave_sum[kScanThreads / 64];
  const int nwords = (nb + 15) >> 4;
  const int per = (nwords + kScanThreads - 1) / kScanThreads;
  const int w0 = min(nwords, (int)threadIdx.x * per), w1 = min(nwords, w0 + per);
  const uint4* bm4 = reinterpret_cast<const uint4*>(block_mask);
  uint32_t cnt = 0;
  for (int i = w0; i < w1; ++i) {
    const uint4 v = bm4[i];
    cnt += __popc(v.x) + __popc(v.y) + __popc(v.z) + __popc(v.w);
  }
  // inclusive scan: within the wave by shuffles, then over the wave totals
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t incl = cnt;
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t v = __shfl_up(incl, off, 64);
    if (lane >= off) incl += v;
  }
  if (lane == 63) wave_sum[wave] = incl;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int i = 0; i < kScanThreads / 64; ++i) {
      const uint32_t v = wave_sum[i];
      wave_sum[i] = run;
      run += v;
    }
    counters[kCtrCount] = run;
  }
  __syncthreads();
  uint32_t pos = wave_sum[wave] + incl - cnt;
  for (int i = w0; i < w1; ++i) {
    const uint4 v = bm4[i];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t bits = w[q];
      while (bits) {
        const int bit = __ffs(bits) - 1;  // flags are 0/1: set bits sit at 0, 8, 16, 24
        list[pos++] = (uint32_t)(i * 16 + q * 4 + (bit >> 3));
        bits &= bits - 1;
      }
    }
  }
}

}  // namespace

template <typename T, int VEC>
static hipError_t launch_gate_t(const GateParams& p, int grid, size_t lds_bytes, hipStream_t st) {
  hipLaunchKernelGGL((gate_kernel<T, VEC>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p);
  return hipGetLastError();
}

hipError_t launch_compact(const uint8_t* block_mask, int nb, uint32_t* list, uint32_t* counters,
                          hipStream_t st) {
  hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(kScanThreads), 0, st, block_mask, nb, list, counters);
  return hipGetLastError();
}

hipError_t launch_gate(const GateParams& p, int dtype, int vec, int grid, size_t lds_bytes,
                       hipStream_t st) {
  if (dtype == 0) {
    if (vec == 4) return launch_gate_t<float, 4>(p, grid, lds_bytes, st);
    return launch_gate_t<float, 1>(p, grid, lds_bytes, st);
  }
  if (vec == 8) return launch_gate_t<uint16_t, 8>(p, grid, lds_bytes, st);
  return launch_gate_t<uint16_t, 1>(p, grid, lds_bytes, st);
}

}  // namespace sc
