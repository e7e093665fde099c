// Fused single-pass Skip-Conv step for dense bf16 layers (groups = 1,
// C_in % 32 == 0): one workgroup per TS x TS tile of output sites made of
// whole gate blocks, doing every step of Eq. 3 for its tile in one launch:
//
//   1. halo: every thread takes 8-channel chunks of the tile's halo pixels
//      (16-byte loads of x_t and x_{t-1}, several in flight), forms
//      r = x_t - x_{t-1} in fp32 (Eq. 2) and the chunk's statistic sum in the
//      canonical order (channels ascending, one rounding per multiply and per
//      add), writes rho = bf16_rne(r) to an LDS halo kept for the product, and
//      copies owned pixels of x_t into the spare x_{t-1} slot; the chunk sums
//      of a pixel are then added in ascending chunk order (across lanes, or
//      through LDS);
//   2. gate (Eq. 5): support sums over taps in row-major order, exact fp64
//      threshold, block OR (Sec. 3.2.2); block flags go to global memory;
//      tiles with no active block stop here, so the hardware dispatcher
//      balances the work;
//   3. MFMA product (Sec. 4.2: im2col restricted to the non-sparse columns,
//      never materialised: operand fragments are read from the LDS halo at
//      each row's pixel + tap offset; rows past the last one read a zero
//      pixel), formed transposed (weights as the MFMA A operand) so that a
//      lane holds 4 consecutive output channels of one site;
//   4. epilogue: z (+)= U at the active sites, activation output refreshed.
//
// Kernels sharing steps 1-2:
//   * fused_rb_kernel (tiles of <= 8 x 8 sites): wave (ng, kp) owns two
//     16-column tiles of the output and one part of the k-steps; its weight
//     fragments go straight from global memory into registers (issued during
//     the gate), so LDS carries only the residual operand; the k-partial sums
//     meet in LDS and all waves finish the epilogue. The old z of every site
//     is fetched with the halo, so no load waits between gate and product.
//     It also runs the learned gate (Eq. 8: per-tap chunk terms in the halo
//     phase) and translated steps (Sec. 3.3: shifted x_{t-1} and z_{t-1}
//     reads, exposed blocks recomputed from x_t in a second product).
//   * fused_kernel (16 x 16 tiles and shapes the first does not cover): the
//     packed weights are copied into LDS with global_load_lds by two loader
//     waves during the halo phase; 16 x 16 tiles compact their active sites
//     (ballot + prefix) into the product rows.
//   * fused_dw_kernel (depthwise) and fused_sc_kernel (fewer than 8 bf16 or
//     at most 16 fp32 input channels): the product on the VALU, or with the
//     weights as the MFMA A operand.
//
// The ordered global active list is not needed by this pipeline; it is
// produced on demand for introspection by the compaction kernel.
#include <type_traits>

#include "sc_device.h"
#include "sc_kernels.h"
#include "sc_stream.h"

#pragma clang fp contract(off)

namespace sc {

namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int kLoadWaves = 2;  // fused_kernel: waves that copy the weights during the halo phase
constexpr int kItems = 4;      // halo items per thread whose loads are in flight together
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
      if (p.rb) *reinterpret_cast<uint2*>(p.rb + o) = uint2{0u, 0u};  // bf16 layers
    }
  }
  for (int i = threadIdx.x; i < nby * nbx; i += kThreads) {
    const int by = i / nbx, bx = i - by * nbx;
    const size_t gb = ((size_t)n * g.hb + bi0 + by) * g.wb + bj0 + bx;
    p.prev_mask[gb] = (cur && cur[by * tb_w + bx] != 0u) ? 1 : 0;
  }
}


// Geometry of one tile of output sites and of its input halo. The halo has
// the extent of a whole tile even for edge tiles (the extra pixels are out of
// the frame or read by no site), so its layout is the same for every tile.
struct Tile {
  int n, oy0, ox0, oh, ow;          // image, first output row / column, tile extent
  int iy0, ix0, hh, hw, npix;       // halo origin (input pixels) and extent
  int own_y0, own_x0, own_y1, own_x1;  // input pixels whose x_t copy this tile writes
  int tb_w;                         // blocks per tile row
  float inv_ts, inv_blk, inv_hw;    // reciprocals for qdiv (computed on the host)
};

// The tile of this workgroup, from the table built at create time (with the
// output channels split over nsplit workgroups, workgroups nsplit * i ..
// nsplit * i + nsplit - 1 share tile i).
__device__ __forceinline__ Tile make_tile(const FusedParams& p, int tile) {
  const GateParams& g = p.g;
  Tile T;
  const uint32_t tc = p.tiles[tile];
  const int tx = (int)(tc & 1023u), ty = (int)((tc >> 10) & 1023u);
  T.n = (int)(tc >> 20);
  const int s = g.stride, k = g.k;
  T.oy0 = ty * g.ts;
  T.ox0 = tx * g.ts;
  T.oh = min(g.ts, g.h_out - T.oy0);
  T.ow = min(g.ts, g.w_out - T.ox0);
  T.iy0 = T.oy0 * s - g.pad;
  T.ix0 = T.ox0 * s - g.pad;
  T.hh = (g.ts - 1) * s + k;
  T.hw = T.hh;
  T.npix = T.hh * T.hw;
  T.own_y0 = T.oy0 * s;
  T.own_x0 = T.ox0 * s;
  T.own_y1 = (ty == g.tiles_y - 1) ? g.h : min(g.h, (T.oy0 + g.ts) * s);
  T.own_x1 = (tx == g.tiles_x - 1) ? g.w : min(g.w, (T.ox0 + g.ts) * s);
  T.tb_w = g.ts / g.block;
  T.inv_ts = p.inv_ts;
  T.inv_blk = p.inv_blk;
  T.inv_hw = p.inv_hw;
  return T;
}

__global__ void fused_tiles_kernel(uint32_t* table, int grid, int tiles_y, int tiles_x) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= grid) return;
  const int tile = xcd_tile(b, grid);
  const int per_img = tiles_y * tiles_x;
  const int n = tile / per_img, rem = tile - n * per_img;
  const int ty = rem / tiles_x, tx = rem - ty * tiles_x;
  table[b] = (uint32_t)tx | ((uint32_t)ty << 10) | ((uint32_t)n << 20);
}

// Chained input: the residual is zero outside the upstream layer's active
// blocks; a tile whose input region meets none of them has every gate off and
// stops before any load (norm gates only). Returns true when the tile stops.
template <bool EMIT>
__device__ bool chain_skip(const FusedParams& p, const Tile& T, uint8_t* emit_clr, bool lead = true) {
  const GateParams& g = p.g;
  const int thh = (T.oh - 1) * g.stride + g.k, thw = (T.ow - 1) * g.stride + g.k;  // the tile's own halo
  const int y0 = max(T.iy0, 0), y1 = min(T.iy0 + thh, g.h), x0 = max(T.ix0, 0), x1 = min(T.ix0 + thw, g.w);
  const int by0 = y0 / g.up_block, by1 = (y1 - 1) / g.up_block;
  const int bx0 = x0 / g.up_block, bx1 = (x1 - 1) / g.up_block;
  const int nbx = bx1 - bx0 + 1, cnt = (by1 - by0 + 1) * nbx;
  int any = 0;
  for (int i = threadIdx.x; i < cnt; i += kThreads) {
    const int by = by0 + i / nbx, bx = bx0 + i % nbx;
    any |= g.up_mask[((size_t)T.n * g.up_hb + by) * g.up_wb + bx] != 0;
  }
  if (__syncthreads_or(any)) return false;
  if (!lead) return true;
  if (g.keep_stats)
    for (int q = threadIdx.x; q < T.oh * T.ow; q += kThreads) {
      const int ly = q / T.ow, lx = q - ly * T.ow;
      const size_t o = ((size_t)T.n * g.h_out + T.oy0 + ly) * g.w_out + T.ox0 + lx;
      g.stat[o] = 0.0f;
      g.site_mask[o] = 0;
    }
  const int nby = (T.oh + g.block - 1) / g.block, nbx2 = (T.ow + g.block - 1) / g.block;
  const int bi0 = T.oy0 / g.block, bj0 = T.ox0 / g.block;
  for (int i = threadIdx.x; i < nby * nbx2; i += kThreads) {
    const int by = i / nbx2, bx = i - by * nbx2;
    g.block_mask[((size_t)T.n * g.hb + bi0 + by) * g.wb + bj0 + bx] = 0;
  }
  if (EMIT) emit_clear(p, T.n, T.oy0, T.ox0, T.oh, T.ow, T.tb_w, nullptr, emit_clr);
  return true;
}

// Split of a halo item index (pixel, 8-channel chunk).
struct ChunkMap {
  int nchk, total, lg;  // chunks per pixel, items in the halo, log2(nchk) or -1
  float inv;            // 1 / nchk
  bool lane_sum;        // a pixel's chunks sit in one aligned group of <= 16 lanes
};

__device__ __forceinline__ ChunkMap make_chunks(const FusedParams& p, const Tile& T) {
  ChunkMap m;
  m.nchk = p.g.c >> 3;
  m.total = T.npix * m.nchk;
  m.lg = (m.nchk & (m.nchk - 1)) == 0 ? __builtin_ctz(m.nchk) : -1;
  m.inv = p.inv_chk;
  m.lane_sum = m.nchk == 4 || m.nchk == 8 || m.nchk == 16;
  return m;
}

// Per-thread walk over the halo items (pixel, 8-channel chunk). With
// rw = hw * nchk items per halo row and rg = NTHR / rw >= 1 row groups, thread
// t keeps one column item c = t % rw (pixel column c / nchk, chunk c % nchk)
// and takes rows r0 + j * rg, r0 = t / rw, so item j costs one add (threads
// t >= rg * rw take none); consecutive threads take consecutive chunks of a
// row, so a wave's loads are contiguous and a pixel's chunks sit in one
// aligned lane group. Rows longer than the thread count use the flat order
// (item base + u * NTHR + t).
struct HaloWalk {
  bool twod;
  int r0, rg, hx, ch, rows;   // 2-D walk; rows = items per thread (ceil(hh / rg))
  bool xin, xown;             // column in the frame / in the owned range
  long off0, ostep;           // frame element offset of item 0 (if in frame), step per item
  int px0, pxstep;            // halo pixel of item 0, step per item
};

// TWOD: the caller guarantees rw <= NTHR (the 2-D walk is compiled alone).
template <int NTHR, bool TWOD>
__device__ __forceinline__ HaloWalk make_walk(const GateParams& g, const Tile& T, const ChunkMap& cm, int tid) {
  HaloWalk W;
  const int rw = T.hw * cm.nchk;
  W.rg = NTHR / rw;
  W.twod = TWOD || W.rg > 0;
  if (!W.twod) return W;
  const int c = tid - (tid / rw) * rw;  // division by a wave-uniform value, once per thread
  W.r0 = tid / rw;
  W.hx = cm.lg >= 0 ? c >> cm.lg : qdiv(c, cm.inv);
  W.ch = c - W.hx * cm.nchk;
  W.rows = W.r0 < W.rg ? (T.hh + W.rg - 1) / W.rg : 0;
  const int x = T.ix0 + W.hx;
  W.xin = x >= 0 && x < g.w;
  W.xown = W.xin && g.x_keep != nullptr && g.copy_in_halo && x >= T.own_x0 && x < T.own_x1;
  W.off0 = ((long)(T.n * g.h + T.iy0 + W.r0) * g.w + x) * g.c + W.ch * 8;
  W.ostep = (long)W.rg * g.w * g.c;
  W.px0 = W.r0 * T.hw + W.hx;
  W.pxstep = W.rg * T.hw;
  return W;
}

// One round of halo items: KI items per thread (2-D walk: items
// base + u of the thread's column; flat order: item base + u * NTHR + tid).
template <int KI = kItems>
struct HaloBatch {
  uint4 vt[KI], vp[KI];
  size_t off[KI], offp[KI];  // offp: translated steps, the x_{t-1} element offset
  int px[KI], ch[KI];
  bool in[KI], own[KI], pin[KI];  // pin: translated steps, x_{t-1} source in the frame
};

// Rounds of KI items a workgroup's halo takes.
template <int NTHR, bool TWOD, int KI = kItems>
__device__ __forceinline__ int halo_rounds(const Tile& T, const ChunkMap& cm, const HaloWalk& W) {
  const int per = (TWOD || W.twod) ? (T.hh + W.rg - 1) / W.rg : (cm.total + NTHR - 1) / NTHR;
  return (per + KI - 1) / KI;
}

// Issue the loads of round `rd`. Addresses are clamped in bounds so that every
// load is issued (the wait counts stay static); out-of-frame items are zeroed
// when used.
// TRANS (translated steps, 2-D walk): x_{t-1} is read at the pixel shifted
// back by (g.sy, g.sx), zero where that lies outside the frame.
template <bool CHAIN, int NTHR, bool TWOD, int KI = kItems, bool TRANS = false>
__device__ __forceinline__ void halo_load(const GateParams& g, const Tile& T, const ChunkMap& cm,
                                          const HaloWalk& W, int rd, int tid, HaloBatch<KI>& B) {
  static_assert(!TRANS || (TWOD && !CHAIN), "translated steps take the 2-D walk on full frames");
  const uint16_t* xt = static_cast<const uint16_t*>(g.x_t);
  const uint16_t* xp = static_cast<const uint16_t*>(g.no_prev ? g.x_t : g.x_prev);
  const bool keep = g.x_keep != nullptr && g.copy_in_halo;
#pragma unroll
  for (int u = 0; u < KI; ++u) {
    if (TWOD || W.twod) {
      const int j = rd * KI + u;
      const int hy = W.r0 + j * W.rg;
      const int y = T.iy0 + hy;
      const bool valid = j < W.rows && hy < T.hh;
      B.px[u] = valid ? W.px0 + j * W.pxstep : -1;
      B.ch[u] = W.ch;
      B.in[u] = valid && W.xin && y >= 0 && y < g.h;
      B.own[u] = B.in[u] && W.xown && y >= T.own_y0 && y < T.own_y1;
      B.off[u] = B.in[u] ? (size_t)(W.off0 + j * W.ostep) : 0;
      if constexpr (TRANS) {
        const int yq = y - g.sy, xq = T.ix0 + W.hx - g.sx;
        B.pin[u] = B.in[u] && yq >= 0 && yq < g.h && xq >= 0 && xq < g.w;
        B.offp[u] = B.pin[u] ? (size_t)((long)B.off[u] - ((long)g.sy * g.w + g.sx) * g.c) : 0;
      }
    } else {
      const int idx = rd * KI * NTHR + u * NTHR + tid;
      const int q = cm.lg >= 0 ? idx >> cm.lg : qdiv(idx, cm.inv);
      B.px[u] = idx < cm.total ? q : -1;
      B.ch[u] = idx - q * cm.nchk;
      const int hy = qdiv(q, T.inv_hw), hx = q - hy * T.hw;
      const int y = T.iy0 + hy, x = T.ix0 + hx;
      B.in[u] = B.px[u] >= 0 && y >= 0 && y < g.h && x >= 0 && x < g.w;
      B.own[u] = B.in[u] && keep && y >= T.own_y0 && y < T.own_y1 && x >= T.own_x0 && x < T.own_x1;
      B.off[u] = B.in[u] ? (size_t)((T.n * g.h + y) * g.w + x) * g.c + B.ch[u] * 8 : 0;
    }
    if (CHAIN) {  // fp32 residual input: channels 0-3 in vt, 4-7 in vp
      const float* rr = static_cast<const float*>(g.x_t) + B.off[u];
      B.vt[u] = *reinterpret_cast<const uint4*>(rr);
      B.vp[u] = *reinterpret_cast<const uint4*>(rr + 4);
    } else {
      B.vt[u] = *reinterpret_cast<const uint4*>(xt + B.off[u]);
      B.vp[u] = *reinterpret_cast<const uint4*>(xp + (TRANS ? B.offp[u] : B.off[u]));
    }
  }
}

// Learned gate terms of one halo item (a pixel's 8-channel chunk, r in fp32):
// for every tap t, the chunk's term sum_j phi[t][8 ch + j] * r[j] (ascending
// from +0, one rounding per multiply and per add), then the pixel's chunk terms
// in ascending chunk order from +0 (lane group of NC), stored by the group's
// first lane (dst: its pixel's k^2 terms, null elsewhere). ph = phi + 8 ch,
// phi [tap][c] in LDS. 3 x 3 kernels take an unrolled loop: the nine chains
// are independent, so their LDS reads and group sums overlap. (Reading a
// tap's phi once for all of a thread's items measured no faster.) A wave
// skips a row kh of three taps when none of its pixels (halo row hy) serves
// it: a site's score reads tap (kh, kw) of halo row ly * stride + kh only, so
// hy - kh must lie in [0, span], span = (oh - 1) * stride (the halo's border
// rows need one or two of the three rows).
template <int NC>
__device__ __forceinline__ void learned_taps(const float* ph, int c, int k, const float (&r)[8], float* dst,
                                             int hy, int span) {
  auto tap = [&](int t) {
    const float4 f0 = *reinterpret_cast<const float4*>(ph + t * c);
    const float4 f1 = *reinterpret_cast<const float4*>(ph + t * c + 4);
    const float f[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
    float pt = 0.0f;
#pragma unroll
    for (int j = 0; j < 8; ++j) pt = add_rn(pt, mul_rn(f[j], r[j]));
    const float acc = group_sum<NC>(pt);
    if (dst) dst[t] = acc;
  };
  if (k == 3) {
#pragma unroll
    for (int kh = 0; kh < 3; ++kh) {
      if (__ballot(dst != nullptr && hy >= kh && hy - kh <= span) == 0ull) continue;  // wave-uniform
#pragma unroll
      for (int kw = 0; kw < 3; ++kw) tap(kh * 3 + kw);
    }
  } else {
    for (int t = 0; t < k * k; ++t) tap(t);
  }
}

// Use one round: r in fp32, the chunk's statistic sum in canonical order (one
// rounding per multiply and per add) and rho = bf16_rne(r) into the LDS halo;
// the pixel's chunk sums are added in ascending order by the group's first
// lane through DPP row shifts (lane_sum), or parked in LDS for a later
// combine. `wave` is the wave's index among the NTHR threads taking items.
// LEARNED (Eq. 8, lane_sum shapes): instead of the norm statistic, every tap
// t of the pixel gets a[q][t] = sum_c phi[t][c] * r[q][c] in the canonical
// chunked order (8 channels ascending from +0, chunk sums ascending from +0),
// into a_halo[q * k^2 + t]; `part` then holds phi [tap][c] (fp32, staged).
template <bool CHAIN, int NTHR, bool TWOD, int KI = kItems, bool LEARNED = false, bool TRANS = false>
__device__ __forceinline__ void halo_use(const FusedParams& p, const Tile& T, const ChunkMap& cm,
                                         const HaloWalk& W, int rd, int wave, HaloBatch<KI>& B, uint8_t* halo,
                                         float* a_halo, float* part) {
  static_assert(!LEARNED || TWOD, "the learned gate takes the 2-D halo walk");
  const GateParams& g = p.g;
#pragma unroll
  for (int u = 0; u < KI; ++u) {
    // wave-uniform: no item left for any lane of the wave
    if ((TWOD || W.twod) ? (rd * KI + u) * W.rg >= T.hh : (rd * KI + u) * NTHR + wave * 64 >= cm.total)
      break;
    if (!B.in[u]) B.vt[u] = uint4{0u, 0u, 0u, 0u};
    if (!B.in[u] || (!CHAIN && g.no_prev) || (TRANS && !B.pin[u])) B.vp[u] = uint4{0u, 0u, 0u, 0u};
    const uint32_t wt[4] = {B.vt[u].x, B.vt[u].y, B.vt[u].z, B.vt[u].w};
    const uint32_t wpv[4] = {B.vp[u].x, B.vp[u].y, B.vp[u].z, B.vp[u].w};
    uint32_t outw[4];
    float r[8];
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
      r[2 * e] = r0;
      r[2 * e + 1] = r1;
      if constexpr (!LEARNED) {
        sum = add_rn(sum, term(r0, g.norm_p));
        sum = add_rn(sum, term(r1, g.norm_p));
      }
      outw[e] = pack_bf16(r0, r1);
    }
    // out-of-frame pixels: zero operand and zero statistic (outw, sum are 0)
    if (B.px[u] >= 0)
      *reinterpret_cast<u32x4*>(halo + (size_t)B.px[u] * p.pstride + B.ch[u] * 16) =
          u32x4{outw[0], outw[1], outw[2], outw[3]};
    if constexpr (LEARNED) {
      const float* ph = part + B.ch[u] * 8;
      float* dst = (B.px[u] >= 0 && B.ch[u] == 0) ? a_halo + B.px[u] * g.k * g.k : nullptr;
      const int hy = W.r0 + (rd * KI + u) * W.rg, span = (T.oh - 1) * g.stride;
      if (cm.nchk == 8) learned_taps<8>(ph, g.c, g.k, r, dst, hy, span);
      else if (cm.nchk == 16) learned_taps<16>(ph, g.c, g.k, r, dst, hy, span);
      else learned_taps<4>(ph, g.c, g.k, r, dst, hy, span);
    } else {
      if (cm.lane_sum) {
        float acc;
        if (cm.nchk == 8) acc = group_sum<8>(sum);
        else if (cm.nchk == 16) acc = group_sum<16>(sum);
        else acc = group_sum<4>(sum);
        if (B.px[u] >= 0 && B.ch[u] == 0) a_halo[B.px[u]] = acc;
      } else if (B.px[u] >= 0) {
        part[B.px[u] * p.pstage + B.ch[u]] = sum;
      }
    }
  }
}

// The owned pixels of a round's x_t go to the spare x_{t-1} slot.
template <int KI>
__device__ __forceinline__ void halo_keep(const GateParams& g, const HaloBatch<KI>& B) {
  uint16_t* keep = static_cast<uint16_t*>(g.x_keep);
#pragma unroll
  for (int u = 0; u < KI; ++u)
    if (B.own[u]) *reinterpret_cast<uint4*>(keep + B.off[u]) = B.vt[u];
}

// Marks a register value as needed here: the compiler completes its load
// first. Used so that no load is still counted once stores are in flight
// (loads and stores share one counter, and a wait on a load issued before a
// store would otherwise wait for the store as well).
template <typename V>
__device__ __forceinline__ void settle(const V& v) {
  asm volatile("" ::"v"(v));
}

// Layers whose halos do not cover the pixels a tile owns (strides above the
// kernel size) copy them element by element.
__device__ __forceinline__ void copy_owned(const GateParams& g, const Tile& T) {
  if (g.copy_in_halo || !g.x_keep) return;
  const uint16_t* xt = static_cast<const uint16_t*>(g.x_t);
  uint16_t* keep = static_cast<uint16_t*>(g.x_keep);
  const int ny = T.own_y1 - T.own_y0, nx = T.own_x1 - T.own_x0;
  const int per_row = nx * g.c;
  for (int i = threadIdx.x; i < ny * per_row; i += kThreads) {
    const int yy = i / per_row, e = i - yy * per_row;
    const size_t o = ((size_t)(T.n * g.h + T.own_y0 + yy) * g.w + T.own_x0) * g.c + e;
    keep[o] = xt[o];
  }
}

// Pixel statistics complete (combining parked chunk sums if needed), then the
// gate of every site of the tile (Eq. 5): support sum over in-frame taps in
// row-major order, exact fp64 threshold (times the Output-Norm weight norm),
// NaN on, block OR into blk_flag and tile_on (LDS). blk_flag and tile_on are
// final only after the next barrier. All threads call it.
__device__ void gate_sites(const FusedParams& p, const Tile& T, const ChunkMap& cm, float* a_halo,
                           const float* part, uint32_t* blk_flag, uint32_t* tile_on, bool lead = true) {
  const GateParams& g = p.g;
  const int s = g.stride, k = g.k, hw = T.hw;
  lds_barrier();
  if (!cm.lane_sum) {
    for (int q = threadIdx.x; q < T.npix; q += kThreads) {
      float acc = 0.0f;
      for (int j = 0; j < cm.nchk; ++j) acc = add_rn(acc, part[q * p.pstage + j]);
      a_halo[q] = acc;
    }
    lds_barrier();
  }
  for (int q = threadIdx.x; q < g.ts * g.ts; q += kThreads) {
    const int ly = qdiv(q, T.inv_ts), lx = q - ly * g.ts;
    if (ly >= T.oh || lx >= T.ow) continue;
    float sv;
    if (g.support == 0 && k == 3) {
      const float* base = a_halo + (ly * s) * hw + lx * s;
      float v[9];
#pragma unroll
      for (int i = 0; i < 9; ++i) v[i] = base[(i / 3) * hw + i % 3];
      sv = 0.0f;
#pragma unroll
      for (int i = 0; i < 9; ++i) sv = add_rn(sv, v[i]);
    } else if (g.support == 0) {
      sv = 0.0f;
      const float* base = a_halo + (ly * s) * hw + lx * s;
      for (int kh = 0; kh < k; ++kh)
        for (int kw = 0; kw < k; ++kw) sv = add_rn(sv, base[kh * hw + kw]);
    } else {
      sv = a_halo[(ly * s + g.pad) * hw + lx * s + g.pad];
    }
    const bool on = g.reference || g.force_dense || ((double)sv * g.wnorm > g.thr) || (sv != sv);
    if (g.keep_stats && lead) {
      const size_t o = ((size_t)T.n * g.h_out + T.oy0 + ly) * g.w_out + T.ox0 + lx;
      g.stat[o] = sv;
      g.site_mask[o] = on ? 1 : 0;
    }
    if (on) {
      blk_flag[qdiv(ly, T.inv_blk) * T.tb_w + qdiv(lx, T.inv_blk)] = 1u;
      *tile_on = 1u;
    }
  }
}

// gate_sites for the register-operand kernel's learned-gate and translated
// modes: LEARNED, the Eq. 8 score (the in-frame per-tap terms in row-major
// order, then the bias; on above zero); TRANS, exposed sites on (Sec. 3.3),
// their blocks marked in blk_exp and tile_exp. (Folding these modes into
// gate_sites changed how the compiler inlined it into the other kernels, and
// some of those then took a scratch frame.)
template <bool LEARNED, bool TRANS>
__device__ __forceinline__ void gate_sites_t(const FusedParams& p, const Tile& T, const ChunkMap& cm, float* a_halo,
                           const float* part, uint32_t* blk_flag, uint32_t* tile_on, bool lead = true,
                           uint32_t* blk_exp = nullptr, uint32_t* tile_exp = nullptr) {
  const GateParams& g = p.g;
  const int s = g.stride, k = g.k, hw = T.hw;
  lds_barrier();
  if (!cm.lane_sum) {
    for (int q = threadIdx.x; q < T.npix; q += kThreads) {
      float acc = 0.0f;
      for (int j = 0; j < cm.nchk; ++j) acc = add_rn(acc, part[q * p.pstage + j]);
      a_halo[q] = acc;
    }
    lds_barrier();
  }
  for (int q = threadIdx.x; q < g.ts * g.ts; q += kThreads) {
    const int ly = qdiv(q, T.inv_ts), lx = q - ly * g.ts;
    if (ly >= T.oh || lx >= T.ow) continue;
    float sv;
    if (LEARNED && k == 3) {
      // Eq. 8 score: the in-frame taps' terms in row-major order, then the
      // bias. An out-of-frame tap adds +0 instead of being skipped: the sum
      // starts at +0 and so is never -0, and x + (+0) = x for every other x.
      // The nine reads are issued together.
      const float* base = a_halo + ((ly * s) * hw + lx * s) * 9;
      const int y0 = T.iy0 + ly * s, x0 = T.ix0 + lx * s;
      float v[9];
#pragma unroll
      for (int i = 0; i < 9; ++i) {
        const int kh = i / 3, kw = i % 3;
        const bool in = y0 + kh >= 0 && y0 + kh < g.h && x0 + kw >= 0 && x0 + kw < g.w;
        const float a = base[(kh * hw + kw) * 9 + i];
        v[i] = in ? a : 0.0f;
      }
      sv = 0.0f;
#pragma unroll
      for (int i = 0; i < 9; ++i) sv = add_rn(sv, v[i]);
      sv = add_rn(sv, g.gate_bias);
    } else if (LEARNED) {
      // as above, any kernel size: in-frame taps only
      const int k2 = k * k;
      sv = 0.0f;
      for (int kh = 0; kh < k; ++kh) {
        const int hy = ly * s + kh, y = T.iy0 + hy;
        if (y < 0 || y >= g.h) continue;
        for (int kw = 0; kw < k; ++kw) {
          const int hx = lx * s + kw, x = T.ix0 + hx;
          if (x < 0 || x >= g.w) continue;
          sv = add_rn(sv, a_halo[(hy * hw + hx) * k2 + kh * k + kw]);
        }
      }
      sv = add_rn(sv, g.gate_bias);
    } else if (g.support == 0 && k == 3) {
      const float* base = a_halo + (ly * s) * hw + lx * s;
      float v[9];
#pragma unroll
      for (int i = 0; i < 9; ++i) v[i] = base[(i / 3) * hw + i % 3];
      sv = 0.0f;
#pragma unroll
      for (int i = 0; i < 9; ++i) sv = add_rn(sv, v[i]);
    } else if (g.support == 0) {
      sv = 0.0f;
      const float* base = a_halo + (ly * s) * hw + lx * s;
      for (int kh = 0; kh < k; ++kh)
        for (int kw = 0; kw < k; ++kw) sv = add_rn(sv, base[kh * hw + kw]);
    } else {
      sv = a_halo[(ly * s + g.pad) * hw + lx * s + g.pad];
    }
    // translated steps: exposed sites on (their blocks are recomputed from x_t)
    const bool ex = TRANS && (line_exposed(T.oy0 + ly, g.h_out, g.h, k, s, g.pad, g.sy) ||
                              line_exposed(T.ox0 + lx, g.w_out, g.w, k, s, g.pad, g.sx));
    const bool on = g.reference || g.force_dense || (LEARNED ? sv > 0.0f : (double)sv * g.wnorm > g.thr) ||
                    (sv != sv) || ex;
    if (TRANS && ex) {
      blk_exp[qdiv(ly, T.inv_blk) * T.tb_w + qdiv(lx, T.inv_blk)] = 1u;
      *tile_exp = 1u;
    }
    if (g.keep_stats && lead) {
      const size_t o = ((size_t)T.n * g.h_out + T.oy0 + ly) * g.w_out + T.ox0 + lx;
      g.stat[o] = sv;
      g.site_mask[o] = on ? 1 : 0;
    }
    if (on) {
      blk_flag[qdiv(ly, T.inv_blk) * T.tb_w + qdiv(lx, T.inv_blk)] = 1u;
      *tile_on = 1u;
    }
  }
}

// The tile's block flags to global memory (after the barrier that made
// blk_flag final).
__device__ void gate_flags(const FusedParams& p, const Tile& T, const uint32_t* blk_flag) {
  const GateParams& g = p.g;
  const int nby = (T.oh + g.block - 1) / g.block, nbx = (T.ow + g.block - 1) / g.block;
  const int bi0 = T.oy0 / g.block, bj0 = T.ox0 / g.block;
  for (int i = threadIdx.x; i < nby * nbx; i += kThreads) {
    const int by = i / nbx, bx = i - by * nbx;
    g.block_mask[((size_t)T.n * g.hb + bi0 + by) * g.wb + bj0 + bx] = (uint8_t)blk_flag[by * T.tb_w + bx];
  }
}

// Gate of the tile; ends after a barrier with blk_flag and tile_on final and
// the block flags stored. All threads call it.
__device__ void gate_tile(const FusedParams& p, const Tile& T, const ChunkMap& cm, float* a_halo,
                          const float* part, uint32_t* blk_flag, uint32_t* tile_on) {
  gate_sites(p, T, cm, a_halo, part, blk_flag, tile_on);
  lds_barrier();
  gate_flags(p, T, blk_flag);
}

// Epilogue of one output piece (4 consecutive channels of one site): z =
// z_{t-1} + U (assigned on a reference frame), activation output; emitting
// layers also write r = y_new - y_old for their successor, y_old =
// dtype(act(z_{t-1})) (the activation output always equals dtype(act(z)), so
// the old z already loaded for the update gives it).
// ASSIGN: z = U (blocks recomputed from x_t on translated steps).
template <bool EMIT, bool ASSIGN = false>
__device__ __forceinline__ void store_piece(const FusedParams& p, size_t o, const floatx4& u, const floatx4& zold) {
  floatx4 nv;
#pragma unroll
  for (int v = 0; v < 4; ++v) nv[v] = (ASSIGN || p.g.reference) ? u[v] : zold[v] + u[v];
  *reinterpret_cast<floatx4*>(p.z + o) = nv;
  if (p.act) {
    uint32_t yb[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) yb[v] = f32_to_bf16(p.act == 2 ? relu_f32(nv[v]) : nv[v]);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.y) + o) = uint2{yb[0] | (yb[1] << 16), yb[2] | (yb[3] << 16)};
    if (EMIT) {
      uint32_t yo[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) yo[v] = f32_to_bf16(p.act == 2 ? relu_f32(zold[v]) : zold[v]);
      floatx4 r;
#pragma unroll
      for (int v = 0; v < 4; ++v) r[v] = __fsub_rn(bf16_to_f32(yb[v]), bf16_to_f32(yo[v]));
      *reinterpret_cast<floatx4*>(p.r32 + o) = r;
      *reinterpret_cast<uint2*>(p.rb + o) =
          uint2{f32_to_bf16(r[0]) | (f32_to_bf16(r[1]) << 16), f32_to_bf16(r[2]) | (f32_to_bf16(r[3]) << 16)};
    }
  }
}

// Translated steps: a site whose block is off keeps the translated z_{t-1}
// (written to the new slot, with its activation output).
__device__ __forceinline__ void store_copy(const FusedParams& p, size_t o, const floatx4& zold) {
  *reinterpret_cast<floatx4*>(p.z + o) = zold;
  if (p.act) {
    uint32_t yb[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) yb[v] = f32_to_bf16(p.act == 2 ? relu_f32(zold[v]) : zold[v]);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.y) + o) = uint2{yb[0] | (yb[1] << 16), yb[2] | (yb[3] << 16)};
  }
}

// ---------------------------------------------------------------------------
// Register-operand kernel for tiles of <= 8 x 8 sites (64 product rows, 4
// M-tiles, NT 16-column N-tiles). Wave w = (kp * MG + mg) * NG + ng owns
// N-tiles ng * WN .. + WN - 1, M-tiles mg * MT .. + MT - 1 and k-steps
// [kp * ksteps / KP, (kp + 1) * ksteps / KP): KPS or KPS - 1 of them (the
// instantiation is chosen so). Per tile LDS carries the residual fragments
// (each read by the NG waves of a k-part and M-group) and the KP partial
// sums; the weights come from global memory (L2) once. Rows outside the tile
// read pixel (tap) of the halo like row 0: their columns of the product are
// discarded, and a site's outputs depend on its own column only.
// MODE bit 0: emit the successor's residual; bit 1: chained input; bit 2:
// learned gate (Eq. 8; phi staged in the chunk-sum region of LDS, the per-tap
// terms in the statistic region); bit 3: translated step (Sec. 3.3: x_{t-1}
// and z_{t-1} read shifted, every site written to the new z slot, and the
// blocks holding an exposed site recomputed from x_t in a second product over
// the same weights, with the halo rewritten to bf16(x_t)).
template <int NT, int WN, int MT, int KPS, int KI, int MODE>
__global__ void __launch_bounds__(kThreads) fused_rb_kernel(FusedParams p) {
  constexpr bool EMIT = (MODE & 1) != 0;
  constexpr bool CHAIN = (MODE & 2) != 0;
  constexpr bool LEARNED = (MODE & 4) != 0;
  constexpr bool TRANS = (MODE & 8) != 0;
  static_assert(!TRANS || !(EMIT || CHAIN), "translated steps neither emit nor chain");
  constexpr int NG = NT / WN;        // wave groups along N
  constexpr int MG = 4 / MT;         // wave groups along M
  constexpr int KP = kWaves / (NG * MG);  // k-step parts
  constexpr int EP = NT / 2;        // epilogue pieces per thread: 64 sites x 4 NT pieces / 512
  constexpr int PROW = NT * 64 + 16;  // LDS bytes per site row of one partial (padded)
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  __shared__ uint32_t blk_flag[kMaxTileBlocks];
  __shared__ uint32_t tile_on;
  __shared__ uint8_t emit_clr[kMaxTileBlocks];
  __shared__ uint32_t blk_exp[TRANS ? kMaxTileBlocks : 1];  // translated steps: blocks with an exposed site
  __shared__ uint32_t tile_exp;

  const GateParams& g = p.g;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  // output channels split over p.nsplit workgroups per tile: this one owns
  // 16-column tiles n0 .. n0 + NT - 1; the lead (split 0) alone writes what
  // every split would write alike (x_{t-1} copy, gate outputs, emitted-residual
  // clears and the previous block flags it reads)
  const int tile_i = p.nsplit > 1 ? (int)(blockIdx.x / p.nsplit) : (int)blockIdx.x;
  const int n0 = ((int)blockIdx.x - tile_i * p.nsplit) * NT;
  const bool lead = n0 == 0;
  const Tile T = make_tile(p, tile_i);
  if (CHAIN && g.up_mask && chain_skip<EMIT>(p, T, emit_clr, lead)) return;
  uint8_t* pbuf = lds + p.off_b;  // partial sums [kp][site][PROW]
  uint8_t* halo = lds + p.off_halo;
  float* a_halo = reinterpret_cast<float*>(lds + p.off_a);
  float* part = reinterpret_cast<float*>(lds + p.off_part);
  const ChunkMap cm = make_chunks(p, T);
  // learned gate: phi [tap][c] (k^2 c / 4 float4, at most kFusedPhiLoads per
  // thread), loaded before anything else so that its LDS copy waits for it alone
  float4 phv[LEARNED ? kFusedPhiLoads : 1];
  if constexpr (LEARNED) {
    const int nf4 = g.k * g.k * g.c / 4;
#pragma unroll
    for (int i = 0; i < kFusedPhiLoads; ++i) {
      const int j = i * kThreads + threadIdx.x;
      phv[i] = reinterpret_cast<const float4*>(g.phi)[j < nf4 ? j : 0];
    }
  }

  // 1. this wave's weight fragments (every load issued: a step past the
  // wave's k-range rereads its first fragment and goes unused), the halo loads
  // of the first round, then the old z (and y) of this thread's epilogue
  // pieces at every site of the tile (piece e = h * 512 + thread: site
  // e / (4 NT), channels 4 (e % (4 NT)) ..). All are in flight together, and
  // no load is left between the gate and the product.
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int ng = wv % NG, mg = (wv / NG) % MG, kp = wv / (NG * MG);
  const bool mma = kp < KP;
  const int ks_lo = mma ? kp * p.ksteps / KP : 0;
  const int nks = mma ? (kp + 1) * p.ksteps / KP - ks_lo : 0;
  bf16x8 bw[KPS][WN];
  {
    const int ntn = p.ntiles_n;  // 16-column tiles of the packed weights
    const bf16x8* src = static_cast<const bf16x8*>(p.wpack) + ((size_t)ks_lo * ntn + n0 + ng * WN) * 64 + lane;
#pragma unroll
    for (int st = 0; st < KPS; ++st)
#pragma unroll
      for (int j = 0; j < WN; ++j) bw[st][j] = src[((size_t)(st < nks ? st : 0) * ntn + j) * 64];
  }
  const HaloWalk hwk = make_walk<kThreads, true>(g, T, cm, threadIdx.x);
  HaloBatch<KI> hb;
  halo_load<CHAIN, kThreads, true, KI, TRANS>(g, T, cm, hwk, 0, threadIdx.x, hb);
  int esite[EP], eloc[EP], ecol[EP];
  floatx4 zold[EP];
  bool zin[EP];  // translated steps: the source site lies in the grid (else z_{t-1} = 0 there)
#pragma unroll
  for (int h = 0; h < EP; ++h) {
    const int e = h * kThreads + threadIdx.x;
    const int site = e / (4 * NT), col = (e - site * 4 * NT) * 4;  // column within this split
    const int ly = qdiv(site, T.inv_ts), lx = site - ly * g.ts;
    const bool ok = ly < T.oh && lx < T.ow && n0 * 16 + col < p.c_out;
    const int gs = (T.n * g.h_out + T.oy0 + ly) * g.w_out + T.ox0 + lx;
    esite[h] = ok ? gs : -1;
    eloc[h] = ok ? qdiv(ly, T.inv_blk) * T.tb_w + qdiv(lx, T.inv_blk) : 0;
    ecol[h] = col;
    if constexpr (TRANS) {
      const int sy = T.oy0 + ly - g.sy / g.stride, sx = T.ox0 + lx - g.sx / g.stride;
      zin[h] = ok && sy >= 0 && sy < g.h_out && sx >= 0 && sx < g.w_out;
      const size_t os = zin[h] ? ((size_t)(T.n * g.h_out + sy) * g.w_out + sx) * p.c_out + n0 * 16 + col : 0;
      zold[h] = *reinterpret_cast<const floatx4*>(p.zsrc + os);
    } else {
      const size_t o = ok ? (size_t)gs * p.c_out + n0 * 16 + col : 0;
      zold[h] = *reinterpret_cast<const floatx4*>(p.z + o);
    }
  }

  for (int i = threadIdx.x; i < kMaxTileBlocks; i += kThreads) blk_flag[i] = 0u;
  if (threadIdx.x == 0) tile_on = 0u;
  if constexpr (TRANS) {
    for (int i = threadIdx.x; i < kMaxTileBlocks; i += kThreads) blk_exp[i] = 0u;
    if (threadIdx.x == 0) tile_exp = 0u;
  }
  // product rows: M-tile i holds 16 sites of the tile. For 8 x 8 tiles they
  // are two tile rows rd apart, rd chosen so that rd * (halo width) = 8
  // (mod 16) when possible: a fragment read (16 lanes x 16 bytes, pixel stride
  // an odd number of 16-byte units) then touches 16 distinct bank groups.
  // Other tiles take the sites in row-major order.
  int abase[MT], msite[MT];
  {
    const int hw = T.hw;
    const int rd = (4 * hw) % 16 == 8 ? 4 : ((2 * hw) % 16 == 8 ? 2 : 1);
#pragma unroll
    for (int ii = 0; ii < MT; ++ii) {
      const int i = mg * MT + ii;
      int ly, lx;
      if (g.ts == 8) {
        const int y0 = rd == 4 ? i : (rd == 2 ? (i & 1) + 4 * (i >> 1) : 2 * i);
        ly = y0 + (r16 >> 3) * rd;
        lx = r16 & 7;
      } else {
        const int row = i * 16 + r16;
        ly = qdiv(row, T.inv_ts);
        lx = row - ly * g.ts;
      }
      msite[ii] = ly * g.ts + lx;
      const bool ok = ly < T.oh && lx < T.ow;
      abase[ii] = (ok ? (ly * g.stride) * hw + lx * g.stride : 0) * p.pstride + kq * 16;
    }
  }

  if constexpr (LEARNED) {
    const int nf4 = g.k * g.k * g.c / 4;
#pragma unroll
    for (int i = 0; i < kFusedPhiLoads; ++i) {
      const int j = i * kThreads + threadIdx.x;
      if (j < nf4) reinterpret_cast<float4*>(part)[j] = phv[i];
    }
    lds_barrier();
  }

  // 2. halo use (and further rounds for large halos)
  halo_use<CHAIN, kThreads, true, KI, LEARNED, TRANS>(p, T, cm, hwk, 0, wave, hb, halo, a_halo, part);
  // weights and old z arrived with (or just after) the halo: settle them
  // before the x_t copy stores go out, so the product and the epilogue wait
  // for nothing
#pragma unroll
  for (int st = 0; st < KPS; ++st)
#pragma unroll
    for (int j = 0; j < WN; ++j) settle(bw[st][j]);
#pragma unroll
  for (int h = 0; h < EP; ++h) settle(zold[h]);
  if (lead) {
    halo_keep(g, hb);  // the halo is one round (KI rows per thread) for this kernel
    copy_owned(g, T);
  }

  // 3. gate of every site, and 4. the product, with no barrier between them:
  // the product is computed whether or not the gate turns any block of the
  // tile on (it does not depend on the gate), so the gate's latency overlaps
  // it instead of preceding it; a tile found off then stores nothing.
  if constexpr (LEARNED || TRANS)
    gate_sites_t<LEARNED, TRANS>(p, T, cm, a_halo, part, blk_flag, &tile_on, lead, blk_exp, &tile_exp);
  else
    gate_sites(p, T, cm, a_halo, part, blk_flag, &tile_on, lead);

  // product over this wave's k-steps: the first KPS - 1 always run, the
  // last one when the wave has KPS (a wave-uniform branch); the tap and
  // channel offset of a step is wave-uniform
  auto product = [&]() {
  floatx4 acc[MT][WN];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j) acc[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
  if (mma) {
    const int csteps = p.csteps, k = g.k, hw = T.hw;
    const int tap0 = ks_lo / csteps;
    int cc = ks_lo - tap0 * csteps, kh = tap0 / k, kw = tap0 - (tap0 / k) * k;
#pragma unroll
    for (int st = 0; st < KPS; ++st) {
      if (st == KPS - 1 && nks < KPS) break;
      const int off = (kh * hw + kw) * p.pstride + cc * 64;
      bf16x8 a[MT];
#pragma unroll
      for (int i = 0; i < MT; ++i) a[i] = *reinterpret_cast<const bf16x8*>(halo + abase[i] + off);
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bw[st][j], a[i], acc[i][j], 0, 0, 0);
      if (++cc == csteps) {
        cc = 0;
        if (++kw == k) {
          kw = 0;
          ++kh;
        }
      }
    }
    // partial sums of this k-part: lane (r16, kq) holds channels
    // (ng * WN + j) * 16 + 4kq .. + 3 of site msite[i]
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j)
        *reinterpret_cast<floatx4*>(pbuf + (size_t)kp * 64 * PROW + msite[i] * PROW +
                                    ((ng * WN + j) * 16 + kq * 4) * 4) = acc[i][j];
  }
  };
  product();
  lds_barrier();
  if (lead) gate_flags(p, T, blk_flag);
  if (!TRANS && !tile_on) {
    if (EMIT && lead) emit_clear(p, T.n, T.oy0, T.ox0, T.oh, T.ow, T.tb_w, blk_flag, emit_clr);
    return;
  }

  // 5. epilogue: the k-parts added in ascending order, at the active sites
  // (translated steps: the blocks off keep the translated z_{t-1}; those with
  // an exposed site wait for the second product)
  auto sum_parts = [&](int h) {
    const int site = (h * kThreads + (int)threadIdx.x) / (4 * NT);
    const uint8_t* src = pbuf + site * PROW + ecol[h] * 4;
    floatx4 u = *reinterpret_cast<const floatx4*>(src);
#pragma unroll
    for (int q = 1; q < KP; ++q) {
      const floatx4 v = *reinterpret_cast<const floatx4*>(src + (size_t)q * 64 * PROW);
#pragma unroll
      for (int c = 0; c < 4; ++c) u[c] = u[c] + v[c];
    }
    return u;
  };
#pragma unroll
  for (int h = 0; h < EP; ++h) {
    if (esite[h] < 0) continue;
    const size_t o = (size_t)esite[h] * p.c_out + n0 * 16 + ecol[h];
    if constexpr (TRANS) {
      if (!zin[h]) zold[h] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
      if (blk_exp[eloc[h]] != 0u) continue;
      if (blk_flag[eloc[h]] == 0u) {
        store_copy(p, o, zold[h]);
        continue;
      }
    } else if (blk_flag[eloc[h]] == 0u) {
      continue;
    }
    store_piece<EMIT>(p, o, sum_parts(h), zold[h]);
  }
  if (EMIT && lead) emit_clear(p, T.n, T.oy0, T.ox0, T.oh, T.ow, T.tb_w, blk_flag, emit_clr);
  if constexpr (TRANS) {
    if (!tile_exp) return;  // block-uniform (LDS, final since the barrier above)
    // 6. blocks holding an exposed site: z = W * bf16(x_t) (assigned). The
    // halo takes the x_t words (zero outside the frame) once every wave has
    // read the partial sums of the first product.
    lds_barrier();
#pragma unroll
    for (int u = 0; u < KI; ++u)
      if (hb.px[u] >= 0)
        *reinterpret_cast<uint4*>(halo + (size_t)hb.px[u] * p.pstride + hb.ch[u] * 16) = hb.vt[u];
    lds_barrier();
    product();
    lds_barrier();
#pragma unroll
    for (int h = 0; h < EP; ++h) {
      if (esite[h] < 0 || blk_exp[eloc[h]] == 0u) continue;
      store_piece<false, true>(p, (size_t)esite[h] * p.c_out + n0 * 16 + ecol[h], sum_parts(h), zold[h]);
    }
  }
}

// ---------------------------------------------------------------------------
// LDS-operand kernel. Wave layout of the product: GM waves along M (WM
// 16-row tiles each) by 2 along N (WN 16-column tiles each); waves past the
// first 2 * GM do no MFMA. MODE as above.
template <int WM, int WN, int GM, int MODE>
__global__ void __launch_bounds__(kThreads) fused_kernel(FusedParams p) {
  constexpr bool EMIT = (MODE & 1) != 0;
  constexpr bool CHAIN = (MODE & 2) != 0;
  constexpr int NTN = WN * 2;
  constexpr int kHaloThreads = kThreads - 64 * kLoadWaves;
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
  const Tile T = make_tile(p, blockIdx.x);
  const int n = T.n, oy0 = T.oy0, ox0 = T.ox0, oh = T.oh, ow = T.ow, hw = T.hw;
  const int s = g.stride, k = g.k;
  if (CHAIN && g.up_mask && chain_skip<EMIT>(p, T, emit_clr)) return;

  uint8_t* ldsb = lds + p.off_b;
  uint8_t* halo = lds + p.off_halo;
  float* a_halo = reinterpret_cast<float*>(lds + p.off_a);
  float* part = reinterpret_cast<float*>(lds + p.off_part);
  const ChunkMap cm = make_chunks(p, T);

  // 1. weights: the last kLoadWaves waves issue the first chunk and take no
  // halo work, so the halo loads of the other waves never queue behind the
  // copy (vector memory counters retire in issue order within a wave)
  const bool loader = wave >= kWaves - kLoadWaves;
  if (loader) issue_b<NTN>(p, ldsb, 0, wave, lane, kWaves - kLoadWaves);
  for (int i = threadIdx.x; i < kMaxTileBlocks; i += kThreads) blk_flag[i] = 0u;
  if (threadIdx.x == 0) tile_on = 0u;
  // the zero pixel read by MFMA rows past the active count
  for (int i = threadIdx.x; i < (p.pstride >> 4); i += kThreads)
    *reinterpret_cast<u32x4*>(halo + (size_t)p.zero_pix * p.pstride + i * 16) = u32x4{0u, 0u, 0u, 0u};

  // Product rows. With one M-tile per wave (tiles of <= 8 x 8 sites) the rows
  // are all sites of the tile in row-major order, fixed before the gate, which
  // only decides which rows are stored. With larger tiles the rows are the
  // active sites, compacted after the gate (step 4).
  constexpr bool kStatic = GM * WM * 16 == 64;
  const int wm = wave % GM, wn = wave / GM;
  int abase[WM], tapmul[WM], zsite[WM];
  uint32_t blk_of[WM];
  floatx4 zold[WM][WN];
  if (kStatic) {
#pragma unroll
    for (int i = 0; i < WM; ++i) {
      const int row = (wm * WM + i) * 16 + r16;
      const int ly = qdiv(row, T.inv_ts), lx = row - ly * g.ts;
      const bool ok = wn < 2 && ly < oh && lx < ow;
      abase[i] = (ok ? (ly * s) * hw + lx * s : p.zero_pix) * p.pstride + kq * 16;
      tapmul[i] = ok ? p.pstride : 0;  // the zero pixel ignores the tap offset
      zsite[i] = ok ? (n * g.h_out + oy0 + ly) * g.w_out + ox0 + lx : -1;
      blk_of[i] = ok ? qdiv(ly, T.inv_blk) * T.tb_w + qdiv(lx, T.inv_blk) : 0u;
    }
  }

  // 2. halo, taken by the threads of the non-loader waves
  if (!loader) {
    const HaloWalk hwk = make_walk<kHaloThreads, false>(g, T, cm, threadIdx.x);
    const int nrounds = halo_rounds<kHaloThreads, false>(T, cm, hwk);
    for (int rd = 0; rd < nrounds; ++rd) {
      HaloBatch<> hb;
      halo_load<CHAIN, kHaloThreads, false>(g, T, cm, hwk, rd, threadIdx.x, hb);
      halo_use<CHAIN, kHaloThreads, false>(p, T, cm, hwk, rd, wave, hb, halo, a_halo, part);
      halo_keep(g, hb);
    }
  }
  copy_owned(g, T);

  // 3. gate
  gate_tile(p, T, cm, a_halo, part, blk_flag, &tile_on);
  if (!tile_on) {
    __builtin_amdgcn_s_waitcnt(0);  // no weight copy may still target this workgroup's LDS
    if (EMIT) emit_clear(p, n, oy0, ox0, oh, ow, T.tb_w, blk_flag, emit_clr);
    return;
  }
  __syncthreads();  // the first weight chunk has landed in LDS

  // 4. local compaction (tiles of more than 64 sites): one site per thread
  // (<= 256 sites), row-major order
  int nrows = 0;
  if (!kStatic) {
    {
      const int q = threadIdx.x;
      const int ly = qdiv(q, T.inv_ts), lx = q - ly * g.ts;
      const bool act = q < g.ts * g.ts && ly < oh && lx < ow &&
                       blk_flag[qdiv(ly, T.inv_blk) * T.tb_w + qdiv(lx, T.inv_blk)] != 0u;
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
  } else {
    // rows of blocks the gate left off are computed but not stored
#pragma unroll
    for (int i = 0; i < WM; ++i)
      if (zsite[i] >= 0 && blk_flag[blk_of[i]] == 0u) zsite[i] = -1;
  }
  // old z of the stored rows, fetched now so that the load overlaps the product
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j) {
      const int col = (wn * WN + j) * 16 + kq * 4;
      zold[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
      // (emitting layers also on a reference frame: z_{t-1} gives y_{t-1})
      if (zsite[i] >= 0 && (!g.reference || EMIT) && col < p.c_out)
        zold[i][j] = *reinterpret_cast<const floatx4*>(p.z + (size_t)zsite[i] * p.c_out + col);
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

  // 6. epilogue
  if (busy) {
#pragma unroll
    for (int i = 0; i < WM; ++i) {
      if (zsite[i] < 0) continue;
#pragma unroll
      for (int j = 0; j < WN; ++j) {
        const int col = (wn * WN + j) * 16 + kq * 4;
        if (col >= p.c_out) continue;
        store_piece<EMIT>(p, (size_t)zsite[i] * p.c_out + col, acc[i][j], zold[i][j]);
      }
    }
  }
  if (EMIT) emit_clear(p, n, oy0, ox0, oh, ow, T.tb_w, blk_flag, emit_clr);
}

// ---------------------------------------------------------------------------
// Depthwise layers (groups = C_in = C_out, C % 8 == 0, tiles of <= 8 x 8
// sites). Steps 1-2 are those above; the product has one input channel per
// output channel (Eq. 3 with g = C), so it is VALU work, no MFMA: a thread
// forms 4 channels of one site as fp32 FMAs over the taps in row-major order,
// rho from the LDS halo and the [tap][c] weights staged in LDS. The channels
// split over nsplit workgroups per tile (at most kDwSplitMax each, so a
// thread holds at most kDwPieces pieces); every split loads the whole halo and
// evaluates the gate, the lead alone writes what all would write alike. The
// product runs before the gate's final barrier (it does not depend on it), and
// a tile found off stores nothing. KI: halo rows per thread (one round).
// MODE as above.
template <int KI, int MODE>
__global__ void __launch_bounds__(kThreads) fused_dw_kernel(FusedParams p) {
  constexpr bool EMIT = (MODE & 1) != 0;
  constexpr bool CHAIN = (MODE & 2) != 0;
  constexpr int EP = kDwPieces;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  __shared__ uint32_t blk_flag[kMaxTileBlocks];
  __shared__ uint32_t tile_on;
  __shared__ uint8_t emit_clr[kMaxTileBlocks];

  const GateParams& g = p.g;
  const int wave = threadIdx.x >> 6;
  const int tile_i = p.nsplit > 1 ? (int)(blockIdx.x / p.nsplit) : (int)blockIdx.x;
  const int cs = g.c / p.nsplit;  // channels of this split: c0 .. c0 + cs - 1
  const int c0 = ((int)blockIdx.x - tile_i * p.nsplit) * cs;
  const bool lead = c0 == 0;
  const Tile T = make_tile(p, tile_i);
  if (CHAIN && g.up_mask && chain_skip<EMIT>(p, T, emit_clr, lead)) return;
  float* wl = reinterpret_cast<float*>(lds + p.off_b);  // [tap][cs]
  uint8_t* halo = lds + p.off_halo;
  float* a_halo = reinterpret_cast<float*>(lds + p.off_a);
  float* part = reinterpret_cast<float*>(lds + p.off_part);
  const ChunkMap cm = make_chunks(p, T);
  const int q4 = cs >> 2;  // 4-channel pieces per site
  const float inv_q4 = 1.0f / (float)q4;
  const int kk = g.k * g.k;

  // 1. this split's weights (float4 w of the k*k*cs/4: tap w / q4, channels
  // c0 + 4 (w % q4) ..), the halo loads, and the old z (and y) of this
  // thread's pieces (piece e = h * 512 + thread: site e / q4, channels
  // c0 + 4 (e % q4) ..): all in flight together
  float4 wreg[kDwWeightLoads];
#pragma unroll
  for (int j = 0; j < kDwWeightLoads; ++j) {
    const int w4 = j * kThreads + threadIdx.x;
    const int tap = qdiv(w4, inv_q4), j4 = w4 - tap * q4;
    const bool ok = tap < kk;
    wreg[j] = static_cast<const float4*>(p.wpack)[ok ? ((size_t)tap * g.c + c0) / 4 + j4 : 0];
  }
  const HaloWalk hwk = make_walk<kThreads, true>(g, T, cm, threadIdx.x);
  HaloBatch<KI> hb;
  halo_load<CHAIN, kThreads, true, KI>(g, T, cm, hwk, 0, threadIdx.x, hb);
  int esite[EP], eloc[EP], ecol[EP], epix[EP];
  floatx4 zold[EP];
#pragma unroll
  for (int h = 0; h < EP; ++h) {
    const int e = h * kThreads + threadIdx.x;
    const int site = qdiv(e, inv_q4), j4 = e - site * q4;
    const int ly = qdiv(site, T.inv_ts), lx = site - ly * g.ts;
    const bool ok = site < g.ts * g.ts && ly < T.oh && lx < T.ow;
    const int gs = (T.n * g.h_out + T.oy0 + ly) * g.w_out + T.ox0 + lx;
    esite[h] = ok ? gs : -1;
    eloc[h] = ok ? qdiv(ly, T.inv_blk) * T.tb_w + qdiv(lx, T.inv_blk) : 0;
    ecol[h] = c0 + 4 * j4;
    epix[h] = ok ? (ly * g.stride) * T.hw + lx * g.stride : 0;
    const size_t o = ok ? (size_t)gs * p.c_out + ecol[h] : 0;
    zold[h] = *reinterpret_cast<const floatx4*>(p.z + o);
  }
  for (int i = threadIdx.x; i < kMaxTileBlocks; i += kThreads) blk_flag[i] = 0u;
  if (threadIdx.x == 0) tile_on = 0u;

  // 2. halo use; the weights to LDS; then (settled) the x_t copy
  halo_use<CHAIN, kThreads, true, KI>(p, T, cm, hwk, 0, wave, hb, halo, a_halo, part);
#pragma unroll
  for (int j = 0; j < kDwWeightLoads; ++j) {
    const int w4 = j * kThreads + threadIdx.x;
    if (w4 < kk * q4) reinterpret_cast<float4*>(wl)[w4] = wreg[j];
  }
#pragma unroll
  for (int h = 0; h < EP; ++h) settle(zold[h]);
  if (lead) {
    halo_keep(g, hb);
    copy_owned(g, T);
  }

  // 3. gate (its first barrier also makes the halo and the weights visible)
  gate_sites(p, T, cm, a_halo, part, blk_flag, &tile_on, lead);

  // 4. product of every piece of the tile, before the gate's outcome is known
  floatx4 u[EP];
#pragma unroll
  for (int h = 0; h < EP; ++h) {
    u[h] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
    if (esite[h] < 0) continue;
    const uint8_t* px = halo + (size_t)epix[h] * p.pstride + ecol[h] * 2;
    const float* wt = wl + (ecol[h] - c0);
    for (int kh = 0; kh < g.k; ++kh)
      for (int kw = 0; kw < g.k; ++kw) {
        const uint2 r = *reinterpret_cast<const uint2*>(px + (kh * T.hw + kw) * p.pstride);
        const float4 w = *reinterpret_cast<const float4*>(wt + (kh * g.k + kw) * cs);
        u[h][0] = __builtin_fmaf(w.x, __uint_as_float(r.x << 16), u[h][0]);
        u[h][1] = __builtin_fmaf(w.y, __uint_as_float(r.x & 0xffff0000u), u[h][1]);
        u[h][2] = __builtin_fmaf(w.z, __uint_as_float(r.y << 16), u[h][2]);
        u[h][3] = __builtin_fmaf(w.w, __uint_as_float(r.y & 0xffff0000u), u[h][3]);
      }
  }
  lds_barrier();
  if (lead) gate_flags(p, T, blk_flag);
  if (!tile_on) {
    if (EMIT && lead) emit_clear(p, T.n, T.oy0, T.ox0, T.oh, T.ow, T.tb_w, blk_flag, emit_clr);
    return;
  }

  // 5. epilogue at the active sites
#pragma unroll
  for (int h = 0; h < EP; ++h) {
    if (esite[h] < 0 || blk_flag[eloc[h]] == 0u) continue;
    store_piece<EMIT>(p, (size_t)esite[h] * p.c_out + ecol[h], u[h], zold[h]);
  }
  if (EMIT && lead) emit_clear(p, T.n, T.oy0, T.ox0, T.oh, T.ow, T.tb_w, blk_flag, emit_clr);
}

// ---------------------------------------------------------------------------
// Layers with few input channels (fp32 with C_in <= 16, bf16 with C_in < 8):
// the shapes whose pixels are narrower than the 8-channel chunks above. The
// halo is loaded in elements, VEC at a time (x_t, x_{t-1} and the x_t copy),
// and r = x_t - x_{t-1} goes to LDS in fp32; one thread per halo pixel forms
// its canonical statistic (8-channel chunk sums, then their sum); the gate is
// gate_sites. The
// product is formed transposed, weights as the MFMA A operand straight from
// the packed buffer (fetched with the halo, held in registers), the residual
// operand (fp32, or its bf16 rounding) gathered from the LDS halo per k index:
// wave w takes the 16 sites of group w % 4 and k-part w / 4 of all output
// tiles; k-part 1 hands its sums to k-part 0 through LDS, which adds them and
// runs the epilogue. Before the gate's last barrier, as above. MODE as above
// (an emitting fp32 layer hands on r = y_new - y_old in fp32 only).
// VEC consecutive elements of a frame as raw bits (what the x_{t-1} copy
// writes back) and as fp32 values.
template <typename T, int VEC>
struct ElemVec {
  static constexpr int kBytes = (int)sizeof(T) * VEC;
  using Raw = typename std::conditional<
      kBytes == 16, uint4,
      typename std::conditional<kBytes == 8, uint2,
                                typename std::conditional<kBytes == 4, uint32_t, uint16_t>::type>::type>::type;
  __device__ __forceinline__ static Raw load(const T* p, size_t i) { return *reinterpret_cast<const Raw*>(p + i); }
  __device__ __forceinline__ static void store(T* p, size_t i, Raw r) { *reinterpret_cast<Raw*>(p + i) = r; }
  __device__ __forceinline__ static void to_f32(Raw r, float* v) {
    if constexpr (sizeof(T) == 4 && VEC == 1) {
      v[0] = __uint_as_float(r);
    } else if constexpr (sizeof(T) == 4) {
      v[0] = __uint_as_float(r.x); v[1] = __uint_as_float(r.y);
      v[2] = __uint_as_float(r.z); v[3] = __uint_as_float(r.w);
    } else if constexpr (VEC == 1) {
      v[0] = __uint_as_float((uint32_t)r << 16);
    } else {
      v[0] = __uint_as_float(r.x << 16); v[1] = __uint_as_float(r.x & 0xffff0000u);
      v[2] = __uint_as_float(r.y << 16); v[3] = __uint_as_float(r.y & 0xffff0000u);
    }
  }
};

// KS: k-steps per wave at most (the weight fragments held in registers; a
// one-step build for the smallest K keeps the kernel's registers low enough
// for four workgroups per CU).
template <typename T, int VEC, int NTN, int MODE, int KS>
__global__ void __launch_bounds__(kThreads) fused_sc_kernel(FusedParams p) {
  constexpr bool EMIT = (MODE & 1) != 0;
  constexpr bool CHAIN = (MODE & 2) != 0;
  constexpr bool BF = sizeof(T) == 2;
  constexpr int KSTEP = BF ? 32 : 4;  // k indices per MFMA step
  using WFrag = typename std::conditional<BF, bf16x8, float>::type;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  __shared__ uint32_t blk_flag[kMaxTileBlocks];
  __shared__ uint32_t tile_on;
  __shared__ uint8_t emit_clr[kMaxTileBlocks];

  const GateParams& g = p.g;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  const Tile TL = make_tile(p, blockIdx.x);
  if (CHAIN && g.up_mask && chain_skip<EMIT>(p, TL, emit_clr)) return;
  float* rh = reinterpret_cast<float*>(lds + p.off_halo);  // [pixel][c] fp32 residual
  float* a_halo = reinterpret_cast<float*>(lds + p.off_a);
  floatx4* part = reinterpret_cast<floatx4*>(lds + p.off_b);  // [group][n-tile][lane]
  const int c = g.c, kk = g.k * g.k * c;
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int sg = wv & 3, kp = wv >> 2;
  const int ks_lo = kp * p.ksteps / 2, nks = (kp + 1) * p.ksteps / 2 - ks_lo;

  // 1. this wave's weight fragments, the halo loads (rounds of kScItems per
  // thread) and the old z (and y) of the pieces k-part 0 stores: lane
  // (r16, kq) of group sg holds channels 16 i + 4 kq .. + 3 of site sg*16 + r16
  WFrag aw[KS][NTN];
#pragma unroll
  for (int st = 0; st < KS; ++st)
#pragma unroll
    for (int i = 0; i < NTN; ++i)
      aw[st][i] = static_cast<const WFrag*>(p.wpack)[((size_t)(st < nks ? ks_lo + st : 0) * NTN + i) * 64 + lane];
  const int q = sg * 16 + r16;  // site of this lane's column of the product
  const int qy = q >> 3, qx = q & 7;  // tiles are at most 8 x 8 sites, laid out 8 wide here
  const bool qok = qy < TL.oh && qx < TL.ow && qy < g.ts && qx < g.ts;
  const int gsite = (TL.n * g.h_out + TL.oy0 + qy) * g.w_out + TL.ox0 + qx;
  floatx4 zold[NTN];
#pragma unroll
  for (int i = 0; i < NTN; ++i) {
    const int col = 16 * i + 4 * kq;
    const bool ok = kp == 0 && qok && col < p.c_out;
    const size_t o = ok ? (size_t)gsite * p.c_out + col : 0;
    zold[i] = *reinterpret_cast<const floatx4*>(p.z + o);
  }
  for (int i = threadIdx.x; i < kMaxTileBlocks; i += kThreads) blk_flag[i] = 0u;
  if (threadIdx.x == 0) tile_on = 0u;

  const int cv = c / VEC;  // loads per pixel
  const int items = TL.npix * cv;
  const float inv_cv = 1.0f / (float)cv;
  const bool keep = g.x_keep != nullptr && g.copy_in_halo;
  using EV = ElemVec<T, VEC>;
  for (int base = 0; base < items; base += kThreads * kScItems) {
    typename EV::Raw rt[kScItems], rp[kScItems];
    float vc[CHAIN ? kScItems : 1][VEC];
    int ro[kScItems];
    bool in[kScItems], own[kScItems];
    size_t off[kScItems];
#pragma unroll
    for (int u = 0; u < kScItems; ++u) {
      const int it = base + u * kThreads + threadIdx.x;
      const int px = qdiv(it, inv_cv), v = it - px * cv;
      const int hy = qdiv(px, TL.inv_hw), hx = px - hy * TL.hw;
      const int y = TL.iy0 + hy, x = TL.ix0 + hx;
      in[u] = it < items && y >= 0 && y < g.h && x >= 0 && x < g.w;
      own[u] = in[u] && keep && y >= TL.own_y0 && y < TL.own_y1 && x >= TL.own_x0 && x < TL.own_x1;
      ro[u] = it < items ? px * c + v * VEC : -1;
      off[u] = in[u] ? ((size_t)(TL.n * g.h + y) * g.w + x) * c + v * VEC : 0;
      if constexpr (CHAIN) {  // fp32 residual input
#pragma unroll
        for (int j = 0; j < VEC; ++j) vc[u][j] = static_cast<const float*>(g.x_t)[off[u] + j];
      } else {
        rt[u] = EV::load(static_cast<const T*>(g.x_t), off[u]);
        rp[u] = EV::load(static_cast<const T*>(g.no_prev ? g.x_t : g.x_prev), off[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < kScItems; ++u) {
      if (ro[u] < 0) continue;
      float a[VEC], b[VEC];
      if constexpr (CHAIN) {
#pragma unroll
        for (int j = 0; j < VEC; ++j) a[j] = vc[u][j];
      } else {
        EV::to_f32(rt[u], a);
        EV::to_f32(rp[u], b);
      }
#pragma unroll
      for (int j = 0; j < VEC; ++j)
        rh[ro[u] + j] = !in[u] ? 0.0f : ((CHAIN || g.no_prev) ? a[j] : __fsub_rn(a[j], b[j]));
      if (!CHAIN && own[u]) EV::store(static_cast<T*>(g.x_keep), off[u], rt[u]);
    }
  }
  if (!CHAIN && !g.copy_in_halo && g.x_keep) {  // pixels outside every halo (strides above the kernel)
    const int ny = TL.own_y1 - TL.own_y0, nx = TL.own_x1 - TL.own_x0;
    for (int i = threadIdx.x; i < ny * nx * c; i += kThreads) {
      const int yy = i / (nx * c), e = i - yy * nx * c;
      const size_t o = ((size_t)(TL.n * g.h + TL.own_y0 + yy) * g.w + TL.own_x0) * c + e;
      static_cast<T*>(g.x_keep)[o] = static_cast<const T*>(g.x_t)[o];
    }
  }
  lds_barrier();
  // pixel statistic in the canonical order: terms of each 8-channel chunk
  // added from +0 in ascending order, then the chunk sums in ascending order
  for (int px = threadIdx.x; px < TL.npix; px += kThreads) {
    float acc = 0.0f;
    for (int j0 = 0; j0 < c; j0 += kChunk) {
      float part = 0.0f;
      for (int j = j0; j < min(c, j0 + kChunk); ++j) part = add_rn(part, term(rh[px * c + j], g.norm_p));
      acc = add_rn(acc, part);
    }
    a_halo[px] = acc;
  }
  // 2. gate (its first barrier makes a_halo visible; the chunk sums are
  // already combined)
  ChunkMap cm;
  cm.nchk = 1;
  cm.total = TL.npix;
  cm.lg = 0;
  cm.inv = 1.0f;
  cm.lane_sum = true;
  gate_sites(p, TL, cm, a_halo, nullptr, blk_flag, &tile_on);

  // 3. product over this wave's k-steps (the gate's outcome not yet needed)
  floatx4 acc[NTN];
#pragma unroll
  for (int i = 0; i < NTN; ++i) acc[i] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
  {
    const int pix0 = (qok ? qy : 0) * g.stride * TL.hw + (qok ? qx : 0) * g.stride;
    const float inv_c = 1.0f / (float)c, inv_k = 1.0f / (float)g.k;
#pragma unroll
    for (int st = 0; st < KS; ++st) {
      if (st >= nks) continue;  // wave-uniform
      const int ks = ks_lo + st;
      float bv[BF ? 8 : 1];
#pragma unroll
      for (int e = 0; e < (BF ? 8 : 1); ++e) {
        const int kidx = ks * KSTEP + (BF ? kq * 8 + e : kq);
        const int tap = qdiv(kidx, inv_c), ci = kidx - tap * c;
        const int kh = qdiv(tap, inv_k), kw = tap - kh * g.k;
        const float r = rh[(kidx < kk ? pix0 + kh * TL.hw + kw : 0) * c + (kidx < kk ? ci : 0)];
        bv[e] = kidx < kk ? r : 0.0f;
      }
      if constexpr (BF) {
        u32x4 qv;
#pragma unroll
        for (int e = 0; e < 4; ++e) qv[e] = pack_bf16(bv[2 * e], bv[2 * e + 1]);
        const bf16x8 b = __builtin_bit_cast(bf16x8, qv);
#pragma unroll
        for (int i = 0; i < NTN; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aw[st][i], b, acc[i], 0, 0, 0);
      } else {
#pragma unroll
        for (int i = 0; i < NTN; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(aw[st][i], bv[0], acc[i], 0, 0, 0);
      }
    }
  }
  if (kp == 1) {
#pragma unroll
    for (int i = 0; i < NTN; ++i) part[(sg * NTN + i) * 64 + lane] = acc[i];
  }
  lds_barrier();
  gate_flags(p, TL, blk_flag);
  if (!tile_on) {
    if (EMIT) emit_clear(p, TL.n, TL.oy0, TL.ox0, TL.oh, TL.ow, TL.tb_w, blk_flag, emit_clr);
    return;
  }

  // 4. epilogue (k-part 0): part sums in part order, z at the active sites
  if (kp == 0 && qok && blk_flag[qdiv(qy, TL.inv_blk) * TL.tb_w + qdiv(qx, TL.inv_blk)] != 0u) {
#pragma unroll
    for (int i = 0; i < NTN; ++i) {
      const int col = 16 * i + 4 * kq;
      if (col >= p.c_out) continue;
      const floatx4 v = part[(sg * NTN + i) * 64 + lane];
      floatx4 u;
#pragma unroll
      for (int j = 0; j < 4; ++j) u[j] = acc[i][j] + v[j];
      const size_t o = (size_t)gsite * p.c_out + col;
      if constexpr (BF) {
        store_piece<EMIT>(p, o, u, zold[i]);
      } else {
        floatx4 nv;
#pragma unroll
        for (int j = 0; j < 4; ++j) nv[j] = g.reference ? u[j] : zold[i][j] + u[j];
        *reinterpret_cast<floatx4*>(p.z + o) = nv;
        if (p.act) {
          floatx4 a;
#pragma unroll
          for (int j = 0; j < 4; ++j) a[j] = p.act == 2 ? relu_f32(nv[j]) : nv[j];
          *reinterpret_cast<floatx4*>(static_cast<float*>(p.y) + o) = a;
          if (EMIT) {
            floatx4 r;
#pragma unroll
            for (int j = 0; j < 4; ++j)
              r[j] = __fsub_rn(a[j], p.act == 2 ? relu_f32(zold[i][j]) : zold[i][j]);
            *reinterpret_cast<floatx4*>(p.r32 + o) = r;
          }
        }
      }
    }
  }
  if (EMIT) emit_clear(p, TL.n, TL.oy0, TL.ox0, TL.oh, TL.ow, TL.tb_w, blk_flag, emit_clr);
}

// ------------------------------------------------------------ launching --

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

template <typename T, int VEC, int NTN, int KS>
hipError_t launch_sc_t(const FusedParams& p, int grid, hipStream_t st) {
  switch ((p.emit ? 1 : 0) | (p.g.rin ? 2 : 0)) {
    case 0: hipLaunchKernelGGL((fused_sc_kernel<T, VEC, NTN, 0, KS>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
    case 2: hipLaunchKernelGGL((fused_sc_kernel<T, VEC, NTN, 2, KS>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
    case 1: hipLaunchKernelGGL((fused_sc_kernel<T, VEC, NTN, 1, KS>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
    default: hipLaunchKernelGGL((fused_sc_kernel<T, VEC, NTN, 3, KS>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
  }
  return hipGetLastError();
}

// k-steps per wave of the build: fp32 kScStepsF32; bf16 1 when the layer
// has at most two k-steps, else kScStepsBf16
template <typename T, int VEC, int NTN>
hipError_t launch_sc_k(const FusedParams& p, int grid, hipStream_t st) {
  if constexpr (sizeof(T) == 4) return launch_sc_t<T, VEC, NTN, kScStepsF32>(p, grid, st);
  else return p.ksteps <= 2 ? launch_sc_t<T, VEC, NTN, 1>(p, grid, st) : launch_sc_t<T, VEC, NTN, kScStepsBf16>(p, grid, st);
}

template <typename T, int VEC>
hipError_t launch_sc_n(const FusedParams& p, int grid, hipStream_t st) {
  switch (p.ntiles_n) {
    case 1: return launch_sc_k<T, VEC, 1>(p, grid, st);
    case 2: return launch_sc_k<T, VEC, 2>(p, grid, st);
    case 4: return launch_sc_k<T, VEC, 4>(p, grid, st);
    default: return hipErrorInvalidValue;
  }
}

template <int KI>
hipError_t launch_dw_t(const FusedParams& p, int grid, hipStream_t st) {
  switch ((p.emit ? 1 : 0) | (p.g.rin ? 2 : 0)) {
    case 0: hipLaunchKernelGGL((fused_dw_kernel<KI, 0>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
    case 1: hipLaunchKernelGGL((fused_dw_kernel<KI, 1>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
    case 2: hipLaunchKernelGGL((fused_dw_kernel<KI, 2>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
    default: hipLaunchKernelGGL((fused_dw_kernel<KI, 3>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p); break;
  }
  return hipGetLastError();
}

template <int NT, int WN, int MT, int KPS, int KI>
hipError_t launch_rb_t(const FusedParams& p, int grid, hipStream_t st) {
#define SC_RB(m) hipLaunchKernelGGL((fused_rb_kernel<NT, WN, MT, KPS, KI, m>), dim3(grid), dim3(kThreads), p.lds_bytes, st, p)
  switch ((p.emit ? 1 : 0) | (p.g.rin ? 2 : 0) | (p.g.learned ? 4 : 0) | (p.zsrc ? 8 : 0)) {
    case 0: SC_RB(0); break;
    case 1: SC_RB(1); break;
    case 2: SC_RB(2); break;
    case 3: SC_RB(3); break;
    case 4: SC_RB(4); break;
    case 5: SC_RB(5); break;
    case 6: SC_RB(6); break;
    case 7: SC_RB(7); break;
    case 8: SC_RB(8); break;
    case 12: SC_RB(12); break;
    default: return hipErrorInvalidValue;
  }
#undef SC_RB
  return hipGetLastError();
}

// Allow the kernel its dynamic LDS (above the 64 KB default) and report how
// many workgroups fit on one CU; done once, at create time.
template <typename K>
int prepare_kernel(K kernel, const FusedParams& p) {
  const void* fn = reinterpret_cast<const void*>(kernel);
  if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, p.lds_bytes) != hipSuccess) return 0;
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, kThreads, p.lds_bytes) != hipSuccess) return 0;
  return blocks;
}

// Every mode a layer may launch (plain or chained steps, with or without
// emission) gets its LDS attribute; the occupancy reported is the plain one.
template <int WM, int WN, int GM>
int prepare_fused_t(const FusedParams& p) {
  const int a = prepare_kernel(fused_kernel<WM, WN, GM, 0>, p);
  const int b = prepare_kernel(fused_kernel<WM, WN, GM, 2>, p);
  const int c = p.emit ? std::min(prepare_kernel(fused_kernel<WM, WN, GM, 1>, p),
                                  prepare_kernel(fused_kernel<WM, WN, GM, 3>, p))
                       : a;
  return std::min(std::min(a, b), c);
}

template <typename T, int VEC, int NTN, int KS>
int prepare_sc_t(const FusedParams& p) {
  const int a = prepare_kernel(fused_sc_kernel<T, VEC, NTN, 0, KS>, p);
  const int b = prepare_kernel(fused_sc_kernel<T, VEC, NTN, 2, KS>, p);
  const int c = p.emit ? std::min(prepare_kernel(fused_sc_kernel<T, VEC, NTN, 1, KS>, p),
                                  prepare_kernel(fused_sc_kernel<T, VEC, NTN, 3, KS>, p))
                       : a;
  return std::min(std::min(a, b), c);
}

template <typename T, int VEC, int NTN>
int prepare_sc_k(const FusedParams& p) {
  if constexpr (sizeof(T) == 4) return prepare_sc_t<T, VEC, NTN, kScStepsF32>(p);
  else return p.ksteps <= 2 ? prepare_sc_t<T, VEC, NTN, 1>(p) : prepare_sc_t<T, VEC, NTN, kScStepsBf16>(p);
}

template <typename T, int VEC>
int prepare_sc_n(const FusedParams& p) {
  switch (p.ntiles_n) {
    case 1: return prepare_sc_k<T, VEC, 1>(p);
    case 2: return prepare_sc_k<T, VEC, 2>(p);
    case 4: return prepare_sc_k<T, VEC, 4>(p);
    default: return 0;
  }
}

template <int KI>
int prepare_dw_t(const FusedParams& p) {
  const int a = prepare_kernel(fused_dw_kernel<KI, 0>, p);
  const int b = prepare_kernel(fused_dw_kernel<KI, 2>, p);
  const int c = p.emit ? std::min(prepare_kernel(fused_dw_kernel<KI, 1>, p),
                                  prepare_kernel(fused_dw_kernel<KI, 3>, p))
                       : a;
  return std::min(std::min(a, b), c);
}

template <int NT, int WN, int MT, int KPS, int KI, int L>
int prepare_rb_m(const FusedParams& p) {
  const int a = prepare_kernel(fused_rb_kernel<NT, WN, MT, KPS, KI, L>, p);
  const int b = prepare_kernel(fused_rb_kernel<NT, WN, MT, KPS, KI, L | 2>, p);
  const int c = p.emit ? std::min(prepare_kernel(fused_rb_kernel<NT, WN, MT, KPS, KI, L | 1>, p),
                                  prepare_kernel(fused_rb_kernel<NT, WN, MT, KPS, KI, L | 3>, p))
                       : a;
  return std::min(std::min(a, b), c);
}

template <int NT, int WN, int MT, int KPS, int KI>
int prepare_rb_t(const FusedParams& p) {
  int occ = p.g.learned ? prepare_rb_m<NT, WN, MT, KPS, KI, 4>(p) : prepare_rb_m<NT, WN, MT, KPS, KI, 0>(p);
  if (p.trans_ok)
    occ = std::min(occ, p.g.learned ? prepare_kernel(fused_rb_kernel<NT, WN, MT, KPS, KI, 12>, p)
                                    : prepare_kernel(fused_rb_kernel<NT, WN, MT, KPS, KI, 8>, p));
  return occ;
}

}  // namespace

hipError_t launch_fused_tiles(uint32_t* table, int grid, int tiles_y, int tiles_x, hipStream_t st) {
  hipLaunchKernelGGL(fused_tiles_kernel, dim3((grid + 255) / 256), dim3(256), 0, st, table, grid, tiles_y, tiles_x);
  return hipGetLastError();
}

// Register-operand builds: (16-column tiles, N-tiles per wave, M-tiles per
// wave, k-steps per wave). Waves per k-part = (NT / WN) * (4 / MT); each wave
// takes KPS or KPS - 1 k-steps. All waves hold every M-tile: with fewer, the
// waves of one k-part would each load the same weight fragments (measured
// slower for 64 -> 64 layers: the weight traffic from L2 doubles).
namespace {
struct RbBuild {
  int nt, wn, mt, kps, ki;  // ki: halo rows each thread loads (the halo is one round)
};
constexpr RbBuild kRbBuilds[] = {
    {2, 2, 4, 2, 4}, {2, 2, 4, 3, 4}, {4, 2, 4, 3, 4}, {4, 2, 4, 5, 4}, {8, 2, 4, 9, 4}, {12, 2, 4, 6, 4},
    {2, 2, 4, 5, 4},  // a quarter of 128 output channels at K = 1152 (3 x 3, C_in = 128)
    {8, 2, 4, 9, 6},  // stride 2, 64 -> 128: a 17 x 17 halo of 8 chunks a pixel
    {6, 2, 4, 3, 4},  // half of 192 output channels at K = 192 (1 x 1, C_in = 192) on small frames
    {4, 2, 4, 5, 6},  // half of 128 output channels, stride 2 (17 x 17 halo) on small frames
};
}  // namespace

int fused_rb_kps(int ntiles_n, int ksteps, int halo_w, int chunks) {
  // the kernel walks the halo in whole rows, in one round of ki rows per thread
  const int rw = halo_w * chunks;
  if (rw > kThreads) return 0;
  const int rows = (halo_w + kThreads / rw - 1) / (kThreads / rw);
  for (int i = 0; i < (int)(sizeof(kRbBuilds) / sizeof(kRbBuilds[0])); ++i) {
    const RbBuild& b = kRbBuilds[i];
    if (b.nt != ntiles_n || rows > b.ki) continue;
    const int kp = kWaves / ((b.nt / b.wn) * (4 / b.mt));
    if ((ksteps + kp - 1) / kp <= b.kps && ksteps / kp >= b.kps - 1) return i + 1;  // build index + 1
  }
  return 0;
}

// Halo rows per thread (one round) the depthwise kernel is built for: 4 or 6
// (the smallest that covers the shape), 0 if neither does.
int fused_dw_ki(int halo_w, int chunks) {
  const int rw = halo_w * chunks;
  if (rw > kThreads) return 0;
  const int rows = (halo_w + kThreads / rw - 1) / (kThreads / rw);
  return rows <= 4 ? 4 : (rows <= 6 ? 6 : 0);
}

// k-parts of the register-operand build `rb` (fused_rb_kps) for the LDS layout.
int fused_rb_kparts(int rb) {
  const RbBuild& b = kRbBuilds[rb - 1];
  return kWaves / ((b.nt / b.wn) * (4 / b.mt));
}

// LDS-operand instantiations: tiles of <= 8 x 8 sites use 4 x 2 waves of one
// M-tile each; 16 x 16 tiles use 4 x 2 waves of 4 M-tiles each. WN = N-tiles
// per wave = ntiles_n / 2.
int prepare_fused(const FusedParams& p) {
  if (p.sc == 1) return prepare_sc_n<float, 1>(p);
  if (p.sc == 4) return prepare_sc_n<float, 4>(p);
  if (p.sc == 2) return prepare_sc_n<uint16_t, 1>(p);
  if (p.sc) return 0;
  if (p.dw) return p.dw == 4 ? prepare_dw_t<4>(p) : (p.dw == 6 ? prepare_dw_t<6>(p) : 0);
  if (p.rbk) {
    switch (p.rbk) {
      case 1: return prepare_rb_t<2, 2, 4, 2, 4>(p);
      case 2: return prepare_rb_t<2, 2, 4, 3, 4>(p);
      case 3: return prepare_rb_t<4, 2, 4, 3, 4>(p);
      case 4: return prepare_rb_t<4, 2, 4, 5, 4>(p);
      case 5: return prepare_rb_t<8, 2, 4, 9, 4>(p);
      case 6: return prepare_rb_t<12, 2, 4, 6, 4>(p);
      case 7: return prepare_rb_t<2, 2, 4, 5, 4>(p);
      case 8: return prepare_rb_t<8, 2, 4, 9, 6>(p);
      case 9: return prepare_rb_t<6, 2, 4, 3, 4>(p);
      case 10: return prepare_rb_t<4, 2, 4, 5, 6>(p);
      default: return 0;
    }
  }
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
  if (p.sc == 1) return launch_sc_n<float, 1>(p, grid, st);
  if (p.sc == 4) return launch_sc_n<float, 4>(p, grid, st);
  if (p.sc == 2) return launch_sc_n<uint16_t, 1>(p, grid, st);
  if (p.sc) return hipErrorInvalidValue;
  if (p.dw) return p.dw == 4 ? launch_dw_t<4>(p, grid, st) : (p.dw == 6 ? launch_dw_t<6>(p, grid, st) : hipErrorInvalidValue);
  if (p.rbk) {
    switch (p.rbk) {
      case 1: return launch_rb_t<2, 2, 4, 2, 4>(p, grid, st);
      case 2: return launch_rb_t<2, 2, 4, 3, 4>(p, grid, st);
      case 3: return launch_rb_t<4, 2, 4, 3, 4>(p, grid, st);
      case 4: return launch_rb_t<4, 2, 4, 5, 4>(p, grid, st);
      case 5: return launch_rb_t<8, 2, 4, 9, 4>(p, grid, st);
      case 6: return launch_rb_t<12, 2, 4, 6, 4>(p, grid, st);
      case 7: return launch_rb_t<2, 2, 4, 5, 4>(p, grid, st);
      case 8: return launch_rb_t<8, 2, 4, 9, 6>(p, grid, st);
      case 9: return launch_rb_t<6, 2, 4, 3, 4>(p, grid, st);
      case 10: return launch_rb_t<4, 2, 4, 5, 6>(p, grid, st);
      default: return hipErrorInvalidValue;
    }
  }
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
