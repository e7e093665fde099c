// Fused single-pass Skip-Conv step for dense bf16 layers (groups = 1,
// C_in % 32 == 0): one workgroup per TS x TS tile of output sites made of
// whole gate blocks, doing every step of Eq. 3 for its tile in one launch:
//
//   1. weights: chunks of the packed weights are copied into LDS with
//      asynchronous global_load_lds at kernel start, so the copy overlaps the
//      halo and gate work (whose barriers wait on LDS traffic only);
//   2. halo: every thread takes 8-channel chunks of the tile's halo pixels
//      (16-byte loads of x_t and x_{t-1}, several in flight), forms
//      r = x_t - x_{t-1} in fp32 (Eq. 2) and the chunk's statistic sum in the
//      canonical order (channels ascending, one rounding per multiply and per
//      add), parks the sum in LDS, writes rho = bf16_rne(r) to an LDS halo kept
//      for the product, and copies owned pixels of x_t into the spare x_{t-1}
//      slot; then one thread per pixel adds its chunk sums in ascending order;
//   3. gate (Eq. 5): support sums over taps in row-major order, exact fp64
//      threshold, block OR (Sec. 3.2.2); block flags go to global memory;
//   4. product rows: for tiles of up to 8 x 8 sites the rows are all sites
//      of the tile (one 16-row MFMA tile per wave) and the gate only decides
//      which rows are stored; for larger tiles the active sites are compacted
//      in row-major order (wave ballot + workgroup prefix) and become the
//      rows; the old z of the stored rows is fetched before the product so
//      its latency overlaps it;
//   5. MFMA product over the rows (Sec. 4.2: im2col restricted to the
//      non-sparse columns, never materialised: A fragments are read from the
//      LDS halo at each row's pixel + tap offset; rows past the last one read
//      a zero pixel);
//   6. epilogue: z (+)= U at the active sites, activation output refreshed
//      (the product is formed transposed, weights as the MFMA A operand, so a
//      lane holds 4 consecutive output channels and z moves in 16-byte pieces).
//
// Inactive tiles stop after step 3, so the hardware dispatcher balances the
// work. The ordered global active list is not needed by this pipeline; it is
// produced on demand for introspection by the compaction kernel.
#include "sc_device.h"
#include "sc_kernels.h"
#include "sc_stream.h"

#pragma clang fp contract(off)

namespace sc {

namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// bf16 round-to-nearest-even of two floats, packed (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{a, b}, bf16x2));
}

// Issue chunk `chunk` of the packed weights (k-steps [chunk*kc, ...), all
// 16-column tiles) into LDS buffer chunk % nbuf, using waves [w0, kWaves). In
// the packed order a chunk is contiguous: unit u = one 1 KB B fragment set.
template <int NTN>
__device__ __forceinline__ void issue_b(const FusedParams& p, uint8_t* ldsb, int chunk, int wave,
                                        int lane, int w0) {
  const int ks0 = chunk * p.kc;
  const int nks = min(p.kc, p.ksteps - ks0);
  const int units = nks * NTN;
  uint8_t* dst = ldsb + (size_t)(chunk % p.nbuf) * p.kc * NTN * 1024;
  const bf16x8* src = static_cast<const bf16x8*>(p.wpack) + (size_t)ks0 * NTN * 64 + lane;
  for (int u = wave - w0; u < units; u += kWaves - w0)
    __builtin_amdgcn_global_load_lds(src + (size_t)u * 64, dst + u * 1024, 16, 0, 0);
}

// Residual emission, the part outside the epilogue: at the tile's blocks that
// the previous step updated and this one does not, r = 0; then every block's
// "updated by the previous step" flag becomes this step's. `cur` holds the
// tile's block flags (NULL: none is active). All threads of the workgroup call it.
__device__ void emit_clear(const FusedParams& p, int n, int oy0, int ox0, int oh, int ow, int tb_w,
                           const uint32_t* cur, uint8_t* clr) {
  const GateParams& g = p.g;
  const int nby = (oh + g.block - 1) / g.block, nbx = (ow + g.block - 1) / g.block;
  const int bi0 = oy0 / g.block, bj0 = ox0 / g.block;
  int any = 0;
  for (int i = threadIdx.x; i < nby * nbx; i += kThreads) {
    const int by = i / nbx, bx = i - by * nbx;
    const size_t gb = ((size_t)n * g.hb + bi0 + by) * g.wb + bj0 + bx;
    const bool now = cur && cur[by * tb_w + bx] != 0u;
    clr[i] = (p.prev_mask[gb] != 0 && !now) ? 1 : 0;
    any |= clr[i];
  }
  if (__syncthreads_or(any)) {
    const int c4 = p.c_out >> 2;
    for (int e = threadIdx.x; e < oh * ow * c4; e += kThreads) {
      const int site = e / c4, col = (e - site * c4) * 4;
      const int ly = site / ow, lx = site - ly * ow;
      if (!clr[(ly / g.block) * nbx + lx / g.block]) continue;
      const size_t o = ((size_t)(n * g.h_out + oy0 + ly) * g.w_out + ox0 + lx) * p.c_out + col;
      *reinterpret_cast<floatx4*>(p.r32 + o) = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
      *reinterpret_cast<uint2*>(p.rb + o) = uint2{0u, 0u};
    }
  }
  for (int i = threadIdx.x; i < nby * nbx; i += kThreads) {
    const int by = i / nbx, bx = i - by * nbx;
    const size_t gb = ((size_t)n * g.hb + bi0 + by) * g.wb + bj0 + bx;
    p.prev_mask[gb] = (cur && cur[by * tb_w + bx] != 0u) ? 1 : 0;
  }
}

// Workgroup barrier that orders LDS accesses only: outstanding global loads
// and stores (the weight copy, the z prefetch, the x_t copy) stay in flight.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Wave layout of the product: GM waves along M (WM 16-row tiles each) by 2
// along N (WN 16-column tiles each); waves past the first 2 * GM do no MFMA.
// MODE bit 0: emit the successor's residual; bit 1: chained input (x_t is the
// upstream layer's fp32 residual, tiles without upstream blocks exit early).
template <int WM, int WN, int GM, int MODE>
__global__ void __launch_bounds__(kThreads) fused_kernel(FusedParams p) {
  constexpr bool EMIT = (MODE & 1) != 0;
  constexpr bool CHAIN = (MODE & 2) != 0;
  constexpr int NTN = WN * 2;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  __shared__ uint32_t blk_flag[kMaxTileBlocks];
  __shared__ int rows_pix[kMaxTileBlocks];
  __shared__ int rows_site[kMaxTileBlocks];
  __shared__ uint32_t wave_cnt[kWaves];
  __shared__ uint32_t tile_on;
  __shared__ uint8_t emit_clr[kMaxTileBlocks];

  const GateParams& g = p.g;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int tiles_per_img = g.tiles_y * g.tiles_x;
  const int n = tile / tiles_per_img;
  const int trem = tile - n * tiles_per_img;
  const int ty = trem / g.tiles_x;
  const int tx = trem - ty * g.tiles_x;
  const int oy0 = ty * g.ts, ox0 = tx * g.ts;
  const int oh = min(g.ts, g.h_out - oy0), ow = min(g.ts, g.w_out - ox0);
  const int s = g.stride, k = g.k, c = g.c;
  const int iy0 = oy0 * s - g.pad, ix0 = ox0 * s - g.pad;
  const int hh = (oh - 1) * s + k, hw = (ow - 1) * s + k;
  const int own_y0 = oy0 * s, own_x0 = ox0 * s;
  const int own_y1 = (ty == g.tiles_y - 1) ? g.h : min(g.h, (oy0 + g.ts) * s);
  const int own_x1 = (tx == g.tiles_x - 1) ? g.w : min(g.w, (ox0 + g.ts) * s);

  uint8_t* ldsb = lds + p.off_b;
  uint8_t* halo = lds + p.off_halo;
  float* a_halo = reinterpret_cast<float*>(lds + p.off_a);
  const int tb_w = g.ts / g.block;
  const int npix = hh * hw;

  if (CHAIN && g.up_mask) {
    // chained input: the residual is zero outside the upstream layer's active
    // blocks; a tile whose input region meets none of them has every gate off
    // and stops here, before any load (norm gates only)
    const int y0 = max(iy0, 0), y1 = min(iy0 + hh, g.h), x0 = max(ix0, 0), x1 = min(ix0 + hw, g.w);
    const int by0 = y0 / g.up_block, by1 = (y1 - 1) / g.up_block;
    const int bx0 = x0 / g.up_block, bx1 = (x1 - 1) / g.up_block;
    const int nbx = bx1 - bx0 + 1, cnt = (by1 - by0 + 1) * nbx;
    int any = 0;
    for (int i = threadIdx.x; i < cnt; i += kThreads) {
      const int by = by0 + i / nbx, bx = bx0 + i % nbx;
      any |= g.up_mask[((size_t)n * g.up_hb + by) * g.up_wb + bx] != 0;
    }
    if (!__syncthreads_or(any)) {
      if (g.keep_stats)
        for (int q = threadIdx.x; q < oh * ow; q += kThreads) {
          const int ly = q / ow, lx = q - ly * ow;
          const size_t o = ((size_t)n * g.h_out + oy0 + ly) * g.w_out + ox0 + lx;
          g.stat[o] = 0.0f;
          g.site_mask[o] = 0;
        }
      const int nby = (oh + g.block - 1) / g.block, nbx2 = (ow + g.block - 1) / g.block;
      const int bi0 = oy0 / g.block, bj0 = ox0 / g.block;
      for (int i = threadIdx.x; i < nby * nbx2; i += kThreads) {
        const int by = i / nbx2, bx = i - by * nbx2;
        g.block_mask[((size_t)n * g.hb + bi0 + by) * g.wb + bj0 + bx] = 0;
      }
      if (EMIT) emit_clear(p, n, oy0, ox0, oh, ow, g.ts / g.block, nullptr, emit_clr);
      return;
    }
  }

  // 1. weights: the waves past the first few issue the first chunk; the
  // barriers up to the product wait on LDS traffic only
  const int bw0 = min(kWaves - 1, 2);
  if (wave >= bw0) issue_b<NTN>(p, ldsb, 0, wave, lane, bw0);
  for (int i = threadIdx.x; i < kMaxTileBlocks; i += kThreads) blk_flag[i] = 0u;
  if (threadIdx.x == 0) tile_on = 0u;
  // the zero pixel read by MFMA rows past the active count
  for (int i = threadIdx.x; i < (p.pstride >> 4); i += kThreads)
    *reinterpret_cast<u32x4*>(halo + (size_t)p.zero_pix * p.pstride + i * 16) = u32x4{0u, 0u, 0u, 0u};

  // Product rows. With one M-tile per wave (tiles of <= 8 x 8 sites) the rows
  // are all sites of the tile in row-major order, fixed before the gate, which
  // only decides which rows are stored. With larger tiles the rows are the
  // active sites, compacted after the gate (step 4).
  // The product is computed transposed (weights as the MFMA A operand): a
  // lane's accumulator holds 4 consecutive output channels of one row, so z
  // moves in 16-byte pieces.
  constexpr bool kStatic = GM * WM * 16 == 64;
  const int wm = wave % GM, wn = wave / GM;
  int abase[WM], tapmul[WM], zsite[WM];
  uint32_t blk_of[WM];
  floatx4 zold[WM][WN];
  uint2 yold[WM][WN];  // emitting layers: the activation output before this step
  if (kStatic) {
#pragma unroll
    for (int i = 0; i < WM; ++i) {
      const int row = (wm * WM + i) * 16 + r16;
      const int ly = row / g.ts, lx = row - (row / g.ts) * g.ts;
      const bool ok = wn < 2 && ly < oh && lx < ow;
      abase[i] = (ok ? (ly * s) * hw + lx * s : p.zero_pix) * p.pstride + kq * 16;
      tapmul[i] = ok ? p.pstride : 0;  // the zero pixel ignores the tap offset
      zsite[i] = ok ? (n * g.h_out + oy0 + ly) * g.w_out + ox0 + lx : -1;
      blk_of[i] = ok ? (ly / g.block) * tb_w + lx / g.block : 0u;
    }
  }

  // 2. halo: one item = one 8-channel chunk of one halo pixel (consecutive
  // items are consecutive chunks, so a wave's loads are contiguous); kItems
  // items per thread have their loads in flight together. Each item forms r
  // in fp32, its chunk sum in canonical order (channels ascending, one
  // rounding per multiply and per add) and rho = bf16_rne(r) for the product.
  const uint16_t* xt = static_cast<const uint16_t*>(g.x_t);
  const uint16_t* xp = static_cast<const uint16_t*>(g.x_prev);
  uint16_t* keep = static_cast<uint16_t*>(g.x_keep);
  float* part = reinterpret_cast<float*>(lds + p.off_part);
  const int nchk = c >> 3;  // 16-byte chunks per pixel
  const int total = npix * nchk;
  constexpr int kItems = 4;
  for (int base = 0; base < total; base += kThreads * kItems) {
    uint4 vt[kItems], vp[kItems];
    size_t off[kItems];
    int px[kItems], ch[kItems];
    bool in[kItems], own[kItems];
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
      const int idx = base + u * kThreads + threadIdx.x;
      px[u] = idx < total ? idx / nchk : -1;
      ch[u] = idx - px[u] * nchk;
      const int hy = px[u] / hw, hx = px[u] - hy * hw;
      const int y = iy0 + hy, x = ix0 + hx;
      in[u] = px[u] >= 0 && y >= 0 && y < g.h && x >= 0 && x < g.w;
      own[u] = in[u] && keep && g.copy_in_halo && y >= own_y0 && y < own_y1 && x >= own_x0 && x < own_x1;
      off[u] = in[u] ? ((size_t)(n * g.h + y) * g.w + x) * c + ch[u] * 8 : 0;
      vt[u] = uint4{0u, 0u, 0u, 0u};
      vp[u] = uint4{0u, 0u, 0u, 0u};
      if (in[u]) {
        if (CHAIN) {  // fp32 residual input: channels 0-3 in vt, 4-7 in vp
          const float* rr = static_cast<const float*>(g.x_t) + off[u];
          vt[u] = *reinterpret_cast<const uint4*>(rr);
          vp[u] = *reinterpret_cast<const uint4*>(rr + 4);
        } else {
          vt[u] = *reinterpret_cast<const uint4*>(xt + off[u]);
          if (!g.no_prev) vp[u] = *reinterpret_cast<const uint4*>(xp + off[u]);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
      if (px[u] < 0) continue;
      const uint32_t wt[4] = {vt[u].x, vt[u].y, vt[u].z, vt[u].w};
      const uint32_t wpv[4] = {vp[u].x, vp[u].y, vp[u].z, vp[u].w};
      uint32_t outw[4];
      float sum = 0.0f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        // channels 2e (low half) and 2e + 1 (high half)
        float r0, r1;
        if (CHAIN) {
          const uint32_t* src = e < 2 ? wt : wpv;
          r0 = __uint_as_float(src[(2 * e) & 3]);
          r1 = __uint_as_float(src[(2 * e + 1) & 3]);
        } else {
          r0 = __fsub_rn(__uint_as_float(wt[e] << 16), __uint_as_float(wpv[e] << 16));
          r1 = __fsub_rn(__uint_as_float(wt[e] & 0xffff0000u), __uint_as_float(wpv[e] & 0xffff0000u));
        }
        sum = add_rn(sum, term(r0, g.norm_p));
        sum = add_rn(sum, term(r1, g.norm_p));
        outw[e] = pack_bf16(r0, r1);
      }
      // out-of-frame pixels: zero operand and zero statistic (outw, sum are 0)
      *reinterpret_cast<u32x4*>(halo + (size_t)px[u] * p.pstride + ch[u] * 16) =
          u32x4{outw[0], outw[1], outw[2], outw[3]};
      part[px[u] * p.pstage + ch[u]] = sum;
      if (own[u]) *reinterpret_cast<uint4*>(keep + off[u]) = vt[u];
    }
  }
  if (!g.copy_in_halo && keep) {
    const int ny = own_y1 - own_y0, nx = own_x1 - own_x0;
    const int per_row = nx * c;
    for (int i = threadIdx.x; i < ny * per_row; i += kThreads) {
      const int yy = i / per_row, e = i - yy * per_row;
      const size_t o = ((size_t)(n * g.h + own_y0 + yy) * g.w + own_x0) * c + e;
      keep[o] = xt[o];
    }
  }
  lds_barrier();
  // pixel statistic: the chunk sums of each pixel added in ascending chunk order
  for (int q = threadIdx.x; q < npix; q += kThreads) {
    float acc = 0.0f;
    for (int j = 0; j < nchk; ++j) acc = add_rn(acc, part[q * p.pstage + j]);
    a_halo[q] = acc;
  }
  lds_barrier();

  // 3. gate
  for (int q = threadIdx.x; q < oh * ow; q += kThreads) {
    const int ly = q / ow, lx = q - ly * ow;
    float sv;
    if (g.support == 0) {
      sv = 0.0f;
      const float* base = a_halo + (ly * s) * hw + lx * s;
      for (int kh = 0; kh < k; ++kh)
        for (int kw = 0; kw < k; ++kw) sv = add_rn(sv, base[kh * hw + kw]);
    } else {
      sv = a_halo[(ly * s + g.pad) * hw + lx * s + g.pad];
    }
    const bool on = g.reference || g.force_dense || ((double)sv * g.wnorm > g.thr) || (sv != sv);
    if (g.keep_stats) {
      const size_t o = ((size_t)n * g.h_out + oy0 + ly) * g.w_out + ox0 + lx;
      g.stat[o] = sv;
      g.site_mask[o] = on ? 1 : 0;
    }
    if (on) {
      blk_flag[(ly / g.block) * tb_w + lx / g.block] = 1u;
      tile_on = 1u;
    }
  }
  lds_barrier();
  {
    const int nby = (oh + g.block - 1) / g.block, nbx = (ow + g.block - 1) / g.block;
    const int bi0 = oy0 / g.block, bj0 = ox0 / g.block;
    for (int i = threadIdx.x; i < nby * nbx; i += kThreads) {
      const int by = i / nbx, bx = i - by * nbx;
      g.block_mask[((size_t)n * g.hb + bi0 + by) * g.wb + bj0 + bx] = (uint8_t)blk_flag[by * tb_w + bx];
    }
  }

  if (!tile_on) {
    __builtin_amdgcn_s_waitcnt(0);  // no weight copy may still target this workgroup's LDS
    if (EMIT) emit_clear(p, n, oy0, ox0, oh, ow, tb_w, blk_flag, emit_clr);
    return;
  }
  __syncthreads();  // the first weight chunk has landed in LDS

  // 4. local compaction (tiles of more than 64 sites): one site per thread
  // (<= 256 sites), row-major order
  int nrows = 0;
  if (!kStatic) {
    {
      const int q = threadIdx.x;
      const int ly = q / ow, lx = q - (q / ow) * ow;
      const bool act = q < oh * ow && blk_flag[(ly / g.block) * tb_w + lx / g.block] != 0u;
      const unsigned long long m = __ballot(act);
      const uint32_t rank = __popcll(m & ((1ull << lane) - 1ull));
      if (lane == 0) wave_cnt[wave] = (uint32_t)__popcll(m);
      lds_barrier();
      uint32_t off = 0;
      for (int w = 0; w < wave; ++w) off += wave_cnt[w];
      if (act) {
        rows_pix[off + rank] = (ly * s) * hw + lx * s;
        rows_site[off + rank] = (n * g.h_out + oy0 + ly) * g.w_out + ox0 + lx;
      }
    }
    lds_barrier();
#pragma unroll
    for (int w = 0; w < kWaves; ++w) nrows += (int)wave_cnt[w];
#pragma unroll
    for (int i = 0; i < WM; ++i) {
      const int row = (wm * WM + i) * 16 + r16;
      const bool ok = row < nrows;
      abase[i] = (ok ? rows_pix[row] : p.zero_pix) * p.pstride + kq * 16;
      tapmul[i] = ok ? p.pstride : 0;
      zsite[i] = ok ? rows_site[row] : -1;
      blk_of[i] = 0u;
    }
    // old z of the active rows, fetched now so that the load overlaps the product
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j) {
        const int col = (wn * WN + j) * 16 + kq * 4;
        zold[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
        yold[i][j] = uint2{0u, 0u};
        if (zsite[i] >= 0 && !g.reference && col < p.c_out)
          zold[i][j] = *reinterpret_cast<const floatx4*>(p.z + (size_t)zsite[i] * p.c_out + col);
        if (EMIT && zsite[i] >= 0 && col < p.c_out)
          yold[i][j] = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(p.y) +
                                                       (size_t)zsite[i] * p.c_out + col);
      }
  } else {
    // rows of blocks the gate left off are computed but not stored; the old z
    // of the stored rows is fetched now so that the load overlaps the product
#pragma unroll
    for (int i = 0; i < WM; ++i) {
      if (zsite[i] >= 0 && blk_flag[blk_of[i]] == 0u) zsite[i] = -1;
#pragma unroll
      for (int j = 0; j < WN; ++j) {
        const int col = (wn * WN + j) * 16 + kq * 4;
        zold[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
        yold[i][j] = uint2{0u, 0u};
        if (zsite[i] >= 0 && !g.reference && col < p.c_out)
          zold[i][j] = *reinterpret_cast<const floatx4*>(p.z + (size_t)zsite[i] * p.c_out + col);
        if (EMIT && zsite[i] >= 0 && col < p.c_out)
          yold[i][j] = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(p.y) +
                                                       (size_t)zsite[i] * p.c_out + col);
      }
    }
  }
  const bool busy = wn < 2 && (kStatic ? wm * WM * 16 < g.ts * g.ts : wm * WM * 16 < nrows);

  // 5. MFMA over the rows: wave (wm, wn) owns M-tiles wm*WM.. and N-tiles wn*WN..
  floatx4 acc[WM][WN];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j) acc[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
  const int csteps = p.csteps;
  for (int chunk = 0; chunk < p.nchunks; ++chunk) {
    if (chunk + 1 < p.nchunks) issue_b<NTN>(p, ldsb, chunk + 1, wave, lane, 0);
    if (busy) {
      const int ks0 = chunk * p.kc;
      const int nks = min(p.kc, p.ksteps - ks0);
      const uint8_t* bbuf =
          ldsb + (size_t)(chunk % p.nbuf) * p.kc * NTN * 1024 + (wn * WN) * 1024 + lane * 16;
      // walk the k-steps (kh, kw, cc) incrementally, kU at a time: the fragment
      // reads of a group are all issued before its MFMAs, so LDS latency is
      // paid once per group rather than once per k-step
      constexpr int kU = 4;
      const int tap0 = ks0 / csteps;
      int cc = ks0 - tap0 * csteps, kh = tap0 / k, kw = tap0 - (tap0 / k) * k;
      const uint8_t* bptr = bbuf;
      int kk = 0;
      for (; kk + kU <= nks; kk += kU) {
        bf16x8 a[kU][WM], bfr[kU][WN];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
          const int off = (kh * hw + kw), coff = cc * 64;
#pragma unroll
          for (int j = 0; j < WN; ++j) bfr[u][j] = *reinterpret_cast<const bf16x8*>(bptr + (u * NTN + j) * 1024);
#pragma unroll
          for (int i = 0; i < WM; ++i)
            a[u][i] = *reinterpret_cast<const bf16x8*>(halo + abase[i] + off * tapmul[i] + coff);
          if (++cc == csteps) {
            cc = 0;
            if (++kw == k) {
              kw = 0;
              ++kh;
            }
          }
        }
#pragma unroll
        for (int u = 0; u < kU; ++u)
#pragma unroll
          for (int i = 0; i < WM; ++i)
#pragma unroll
            for (int j = 0; j < WN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[u][j], a[u][i], acc[i][j], 0, 0, 0);
        bptr += kU * NTN * 1024;
      }
      for (; kk < nks; ++kk) {
        const int off = (kh * hw + kw), coff = cc * 64;
        bf16x8 a[WM], bfr[WN];
#pragma unroll
        for (int j = 0; j < WN; ++j) bfr[j] = *reinterpret_cast<const bf16x8*>(bptr + j * 1024);
#pragma unroll
        for (int i = 0; i < WM; ++i)
          a[i] = *reinterpret_cast<const bf16x8*>(halo + abase[i] + off * tapmul[i] + coff);
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
          for (int j = 0; j < WN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[j], a[i], acc[i][j], 0, 0, 0);
        bptr += NTN * 1024;
        if (++cc == csteps) {
          cc = 0;
          if (++kw == k) {
            kw = 0;
            ++kh;
          }
        }
      }
    }
    if (chunk + 1 < p.nchunks) __syncthreads();  // next chunk landed; this buffer free
  }

  // 6. epilogue: z = z_{t-1} + U (assigned on a reference frame), activation
  // output; emitting layers also write r = y_new - y_old for their successor
  if (busy) {
#pragma unroll
    for (int i = 0; i < WM; ++i) {
      if (zsite[i] < 0) continue;
#pragma unroll
      for (int j = 0; j < WN; ++j) {
        const int col = (wn * WN + j) * 16 + kq * 4;
        if (col >= p.c_out) continue;
        floatx4 nv;
#pragma unroll
        for (int v = 0; v < 4; ++v) nv[v] = g.reference ? acc[i][j][v] : zold[i][j][v] + acc[i][j][v];
        const size_t o = (size_t)zsite[i] * p.c_out + col;
        *reinterpret_cast<floatx4*>(p.z + o) = nv;
        if (p.act) {
          uint32_t yb[4];
#pragma unroll
          for (int v = 0; v < 4; ++v) yb[v] = f32_to_bf16(p.act == 2 ? fmaxf(nv[v], 0.0f) : nv[v]);
          *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.y) + o) = uint2{yb[0] | (yb[1] << 16), yb[2] | (yb[3] << 16)};
          if (EMIT) {
            const uint32_t yo[4] = {yold[i][j].x & 0xffffu, yold[i][j].x >> 16, yold[i][j].y & 0xffffu,
                                    yold[i][j].y >> 16};
            floatx4 r;
#pragma unroll
            for (int v = 0; v < 4; ++v) r[v] = __fsub_rn(bf16_to_f32(yb[v]), bf16_to_f32(yo[v]));
            *reinterpret_cast<floatx4*>(p.r32 + o) = r;
            *reinterpret_cast<uint2*>(p.rb + o) =
                uint2{f32_to_bf16(r[0]) | (f32_to_bf16(r[1]) << 16), f32_to_bf16(r[2]) | (f32_to_bf16(r[3]) << 16)};
          }
        }
      }
    }
  }
  if (EMIT) emit_clear(p, n, oy0, ox0, oh, ow, tb_w, blk_flag, emit_clr);
}

template <int WM, int WN, int GM>
hipError_t launch_fused_t(const FusedParams& p, int grid, hipStream_t st) {
  switch ((p.emit ? 1 : 0) | (p.g.rin ? 2 : 0)) {
    case 0: hipLaunchKernelGGL((fused_kernel<WM, WN, GM, 0>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
    case 1: hipLaunchKernelGGL((fused_kernel<WM, WN, GM, 1>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
    case 2: hipLaunchKernelGGL((fused_kernel<WM, WN, GM, 2>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
    default: hipLaunchKernelGGL((fused_kernel<WM, WN, GM, 3>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
  }
  return hipGetLastError();
}

// Allow the kernel its dynamic LDS (above the 64 KB default) and report how
// many workgroups fit on one CU; done once, at create time.
template <int WM, int WN, int GM, int MODE>
int prepare_fused_e(const FusedParams& p) {
  const void* fn = reinterpret_cast<const void*>(fused_kernel<WM, WN, GM, MODE>);
  if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, p.lds_bytes) != hipSuccess) return 0;
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fused_kernel<WM, WN, GM, MODE>, kThreads,
                                                   p.lds_bytes) != hipSuccess)
    return 0;
  return blocks;
}

// Every mode a layer may launch (plain or chained steps, with or without
// emission) gets its LDS attribute; the occupancy reported is the plain one.
template <int WM, int WN, int GM>
int prepare_fused_t(const FusedParams& p) {
  const int e = p.emit ? 1 : 0;
  const int a = prepare_fused_e<WM, WN, GM, 0>(p);
  const int b = prepare_fused_e<WM, WN, GM, 2>(p);
  const int c = e ? std::min(prepare_fused_e<WM, WN, GM, 1>(p), prepare_fused_e<WM, WN, GM, 3>(p)) : a;
  return std::min(std::min(a, b), c);
}

}  // namespace

// Instantiations: tiles of <= 8 x 8 sites use 4 x 2 waves of one M-tile
// each (a 2 x 2 layout of 2 M-tiles per wave reads less LDS but measured
// slower); 16 x 16 tiles use 4 x 2 waves of 4 M-tiles each. WN = N-tiles per
// wave = ntiles_n / 2.
int prepare_fused(const FusedParams& p) {
  if (p.mw == 1) {
    switch (p.ntiles_n) {
      case 2: return prepare_fused_t<1, 1, 4>(p);
      case 4: return prepare_fused_t<1, 2, 4>(p);
      case 8: return prepare_fused_t<1, 4, 4>(p);
      case 12: return prepare_fused_t<1, 6, 4>(p);
      case 16: return prepare_fused_t<1, 8, 4>(p);
      default: return 0;
    }
  }
  if (p.mw == 4) {
    switch (p.ntiles_n) {
      case 2: return prepare_fused_t<4, 1, 4>(p);
      case 4: return prepare_fused_t<4, 2, 4>(p);
      case 8: return prepare_fused_t<4, 4, 4>(p);
      default: return 0;
    }
  }
  return 0;
}

hipError_t launch_fused(const FusedParams& p, int grid, hipStream_t st) {
  if (p.mw == 1) {
    switch (p.ntiles_n) {
      case 2: return launch_fused_t<1, 1, 4>(p, grid, st);
      case 4: return launch_fused_t<1, 2, 4>(p, grid, st);
      case 8: return launch_fused_t<1, 4, 4>(p, grid, st);
      case 12: return launch_fused_t<1, 6, 4>(p, grid, st);
      case 16: return launch_fused_t<1, 8, 4>(p, grid, st);
      default: return hipErrorInvalidValue;
    }
  }
  if (p.mw == 4) {
    switch (p.ntiles_n) {
      case 2: return launch_fused_t<4, 1, 4>(p, grid, st);
      case 4: return launch_fused_t<4, 2, 4>(p, grid, st);
      case 8: return launch_fused_t<4, 4, 4>(p, grid, st);
      default: return hipErrorInvalidValue;
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace sc
