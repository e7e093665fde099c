// Block-halo MFMA convolution of one tile of output sites (Eq. 3 over the
// active sites, as the im2col product of Sec. 4.2 restricted to one block):
// the per-tile work of the split pipeline's convolution kernel, which walks
// the work list. bf16 operands, fp32 accumulation, C_in % 32 == 0.
//
// A tile is `tr` output rows x b columns of one block. Per tile:
//   1. the accumulators start from z_{t-1} of the tile's sites (0 on a
//      reference frame), loaded straight into the MFMA output layout (a lane
//      holds 4 consecutive output channels of one site: z moves in 16-byte
//      pieces);
//   2. the input halo ((tr-1)s+k rows x (b-1)s+k columns x C_in) is loaded
//      with 16-byte loads of both frames, turned into rho = bf16(x_t - x_{t-1})
//      and stored in LDS with a pixel stride of 2*C_in + 16 bytes (16
//      consecutive pixels read 16 bytes each on distinct banks);
//   3. MFMA A fragments are read straight from the halo (row m of the tile at
//      tap (kh, kw) is halo pixel (ly*s + kh, lx*s + kw): no im2col copy); B
//      fragments come from the packed weights through a buffer resource, KR - 1
//      k-steps ahead of use;
//   4. the accumulators are stored back to z (and the activation output).
// Frames and z are addressed through buffer resources over one image with
// 32-bit offsets: sites and pixels outside the frame (and x_{t-1} outside a
// translated frame) read zeros at an out-of-range offset, so no load is
// conditional and the wait counts are static.
//
// Waves are laid out WAVES_M x WAVES_N; each owns WM x WN 16x16 output tiles.
// KR: B register ring (0 picks 8 / 6 / 4 by WN). KU: halo items (two 16-byte
// loads each) in flight per thread. ADB: A fragment register sets (2: the next
// step's fragments are read before this step's MFMAs; 1: M-tile by M-tile
// after them).
#pragma once

#include "sc_device.h"
#include "sc_kernels.h"
#include "sc_stream.h"

namespace sc {

typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// bf16 round-to-nearest-even of two floats, packed (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{a, b}, bf16x2));
}

__device__ __forceinline__ float activate(float v, int act) { return act == 2 ? relu_f32(v) : v; }

struct HaloTile {
  int n, oy0, ox0, rows_ok, cols_ok, iy0, ix0;
};

template <int WAVES_M, int WAVES_N, int WM, int WN, int KR, int KU, int ADB>
struct HaloConv {
  static constexpr int kThreads = 64 * WAVES_M * WAVES_N;
  static constexpr int kR = KR ? KR : (WN <= 2 ? 8 : (WN == 3 ? 6 : 4));  // even
  typedef floatx4 Acc[WM][WN];

  const ConvParams& p;
  const HaloParams& hp;
  uint8_t* halo;
  int lane, wm, r16, kq, lb, wn0, boff, chunks_per_px, csteps, total;
  size_t ximg, zimg;
  __amdgpu_buffer_rsrc_t wrs;
  int abase[WM];  // halo byte offset of this lane's A row in each of its M-tiles, before the tap

  __device__ HaloConv(const ConvParams& p_, const HaloParams& hp_, uint8_t* halo_) : p(p_), hp(hp_), halo(halo_) {
    lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    wm = wave % WAVES_M;
    const int wn = wave / WAVES_M;
    r16 = lane & 15;
    kq = lane >> 4;
    lb = __ffs(p.block) - 1;
    // packed weights: lane offset in a VGPR, the (k-step, column tile) offset in an SGPR
    wrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p.wpack), 0, p.ksteps * p.ntiles_n * 1024, 0x00020000);
    boff = lane * 16;
    wn0 = __builtin_amdgcn_readfirstlane(wn) * WN;  // first 16-channel output tile
    chunks_per_px = p.c >> 3;
    csteps = p.c >> 5;  // k-steps per tap
    ximg = (size_t)p.h * p.w * p.c;
    zimg = (size_t)p.h_out * p.w_out * p.c_out;
    total = hp.hh * hp.hw * chunks_per_px;
#pragma unroll
    for (int i = 0; i < WM; ++i) {
      const int m = (wm * WM + i) * 16 + r16;
      const int ly = m >> lb, lx = m & (p.block - 1);
      abase[i] = (ly * p.stride * hp.hw + lx * p.stride) * hp.pstride + kq * 16;
    }
  }

  __device__ HaloTile tile(int n, int oy0, int ox0) const {
    HaloTile T;
    T.n = n;
    T.oy0 = oy0;
    T.ox0 = ox0;
    T.rows_ok = min(hp.tr, p.h_out - oy0);
    T.cols_ok = min(p.block, p.w_out - ox0);
    T.iy0 = oy0 * p.stride - p.pad;
    T.ix0 = ox0 * p.stride - p.pad;
    return T;
  }

  // z byte offset (within image T.n) of this lane's piece (M-tile i, column
  // tile jn), or out of range outside the frame / past C_out
  __device__ uint32_t zoff(const HaloTile& T, int i, int jn) const {
    int l16 = r16;  // opaque: recomputed per use rather than held per (i, jn)
    asm volatile("" : "+v"(l16));
    const int m = (wm * WM + i) * 16 + l16;
    const int ly = m >> lb, lx = m & (p.block - 1);
    const int col = (wn0 + jn) * 16 + kq * 4;
    return (ly < T.rows_ok && lx < T.cols_ok && col < p.c_out)
               ? (uint32_t)((((T.oy0 + ly) * p.w_out + T.ox0 + lx) * p.c_out + col) * 4)
               : kOutOfRange;
  }

  __device__ __amdgpu_buffer_rsrc_t zres(const HaloTile& T) const {
    return frame_rsrc(p.z + (size_t)T.n * zimg, (uint32_t)(zimg * 4));
  }

  // z_{t-1} of a tile in the transposed MFMA output layout; zeros outside the
  // frame and on a reference frame (none: every piece out of range, so the
  // registers are always written)
  // (translated steps: from zsrc at the site shifted back by (zdy, zdx))
  __device__ void load_z(Acc& dst, const HaloTile& T, bool none) const {
    const auto zrs = p.zsrc ? frame_rsrc(p.zsrc + (size_t)T.n * zimg, (uint32_t)(zimg * 4)) : zres(T);
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int jn = 0; jn < WN; ++jn)
        dst[i][jn] = __builtin_bit_cast(
            floatx4, __builtin_amdgcn_raw_buffer_load_b128(
                         zrs, p.reference || none ? kOutOfRange : (p.zsrc ? zoff_src(T, i, jn) : zoff(T, i, jn)),
                         0, 0));
  }

  // byte offset in zsrc of z_{t-1} for this lane's piece under the step's
  // translation, or out of range where the shifted site leaves the frame
  __device__ uint32_t zoff_src(const HaloTile& T, int i, int jn) const {
    int l16 = r16;
    asm volatile("" : "+v"(l16));
    const int m = (wm * WM + i) * 16 + l16;
    const int ly = m >> lb, lx = m & (p.block - 1);
    const int col = (wn0 + jn) * 16 + kq * 4;
    const int sy = T.oy0 + ly - p.zdy, sx = T.ox0 + lx - p.zdx;
    return (ly < T.rows_ok && lx < T.cols_ok && col < p.c_out && sy >= 0 && sy < p.h_out && sx >= 0 &&
            sx < p.w_out)
               ? (uint32_t)(((sy * p.w_out + sx) * p.c_out + col) * 4)
               : kOutOfRange;
  }

  // one round of halo items: rho = bf16(x_t - x_{t-1}) into LDS
  __device__ void halo_round(const HaloTile& T, int base) const {
    const uint16_t* xt = static_cast<const uint16_t*>(p.x_t);
    const uint16_t* xp = static_cast<const uint16_t*>(p.x_prev);
    const auto xrs = frame_rsrc(xt + (size_t)T.n * ximg, (uint32_t)(ximg * 2));
    const auto prs = frame_rsrc((p.no_prev ? xt : xp) + (size_t)T.n * ximg, (uint32_t)(ximg * 2));
    const int c = p.c;
    u32x4 ra[KU], rb[KU];
    // the thread index, opaque to loop-invariant code motion: the per-item
    // terms are recomputed each round instead of occupying registers through
    // the product loop
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      const int idx = base + u * kThreads + tid;
      const int px = idx / chunks_per_px, ch = idx - px * chunks_per_px;
      const int hy = px / hp.hw, hx = px - hy * hp.hw;
      const int y = T.iy0 + hy, x = T.ix0 + hx;
      const bool in = idx < total && y >= 0 && y < p.h && x >= 0 && x < p.w;
      const int yp = y - p.sy, xq = x - p.sx;
      const bool pin = in && !p.no_prev && yp >= 0 && yp < p.h && xq >= 0 && xq < p.w;
      ra[u] = __builtin_amdgcn_raw_buffer_load_b128(
          xrs, in ? (uint32_t)(((y * p.w + x) * c + ch * 8) * 2) : kOutOfRange, 0, 0);
      rb[u] = __builtin_amdgcn_raw_buffer_load_b128(
          prs, pin ? (uint32_t)(((yp * p.w + xq) * c + ch * 8) * 2) : kOutOfRange, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < KU; ++u) {
      const int idx = base + u * kThreads + tid;
      if (idx >= total) continue;
      const int px = idx / chunks_per_px, ch = idx - px * chunks_per_px;
      uint32_t q[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t wa = ra[u][e], wb = rb[u][e];
        const float r0 = __fsub_rn(__uint_as_float(wa << 16), __uint_as_float(wb << 16));
        const float r1 = __fsub_rn(__uint_as_float(wa & 0xffff0000u), __uint_as_float(wb & 0xffff0000u));
        q[e] = pack_bf16(r0, r1);
      }
      *reinterpret_cast<u32x4*>(halo + px * hp.pstride + ch * 16) = u32x4{q[0], q[1], q[2], q[3]};
    }
  }

  // the whole halo (the first round outside the loop: no loop-carried waits)
  __device__ void load_halo(const HaloTile& T) const {
    halo_round(T, 0);
    for (int base = kThreads * KU; base < total; base += kThreads * KU) halo_round(T, base);
  }

  // MFMA over K = (kh, kw, ci) from the LDS halo into acc. The main loop has
  // no data-dependent branches, so the waits count outstanding loads instead
  // of draining them; scheduling barriers keep the compiler from sinking the
  // reads back to their use.
  __device__ void product(Acc& acc) const {
    const int ksteps = p.ksteps, ntn = p.ntiles_n, k = p.k;
    bf16x8 bq[kR][WN];
    bf16x8 aq[ADB][WM];
    auto load_b = [&](bf16x8* dst, int ks) {
#pragma unroll
      for (int jn = 0; jn < WN; ++jn)
        dst[jn] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                                                 wrs, boff, (ks * ntn + wn0 + jn) * 1024, 0));
    };
    int aoff = 0, cc = 0, kw = 0, snext = 0;  // halo offset of the next A step (kh, kw, cc)
    // advance aoff to the following step without branches; stays on the last step
    auto advance = [&]() {
      const bool more = ++snext < ksteps;
      const int c1 = cc + 1;
      const bool wrap = c1 == csteps;
      const int kw1 = kw + (wrap ? 1 : 0);
      const bool wrap2 = kw1 == k;
      int a1 = aoff + 64;
      a1 += wrap ? hp.pstride - csteps * 64 : 0;
      a1 += wrap2 ? (hp.hw - k) * hp.pstride : 0;
      cc = more ? (wrap ? 0 : c1) : cc;
      kw = more ? (wrap2 ? 0 : kw1) : kw;
      aoff = more ? a1 : aoff;
    };
    auto read_a = [&](bf16x8* dst) {
#pragma unroll
      for (int i = 0; i < WM; ++i) dst[i] = *reinterpret_cast<const bf16x8*>(halo + abase[i] + aoff);
      advance();
    };
    auto mfmas = [&](const bf16x8* a, const bf16x8* bf) {
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int jn = 0; jn < WN; ++jn)
          acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bf[jn], a[i], acc[i][jn], 0, 0, 0);
    };
    // one A register set: the fragment of M-tile i for the next step is read
    // right after the MFMAs of M-tile i of this step have taken it
    auto mfmas_then_read = [&](bf16x8* a, const bf16x8* bf) {
#pragma unroll
      for (int i = 0; i < WM; ++i) {
#pragma unroll
        for (int jn = 0; jn < WN; ++jn)
          acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bf[jn], a[i], acc[i][jn], 0, 0, 0);
        a[i] = *reinterpret_cast<const bf16x8*>(halo + abase[i] + aoff);
      }
      advance();
    };
#pragma unroll
    for (int r = 0; r < kR - 1; ++r) load_b(bq[r], min(r, ksteps - 1));
    read_a(aq[0]);
    int ks = 0;
    for (; ks + kR <= ksteps; ks += kR) {
#pragma unroll
      for (int r = 0; r < kR; ++r) {
        load_b(bq[(r + kR - 1) % kR], min(ks + r + kR - 1, ksteps - 1));
        if constexpr (ADB == 2) {
          read_a(aq[(r + 1) & 1]);
          __builtin_amdgcn_sched_barrier(0);
          mfmas(aq[r & 1], bq[r]);
          __builtin_amdgcn_sched_barrier(0);
        } else {
          mfmas_then_read(aq[0], bq[r]);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < kR - 1; ++r)
      if (r < ksteps - ks) {
        if constexpr (ADB == 2) {
          read_a(aq[(r + 1) & 1]);
          mfmas(aq[r & 1], bq[r]);
        } else {
          mfmas_then_read(aq[0], bq[r]);
        }
      }
  }

  // the activation output y_old = dtype(act(z_{t-1})) of the tile's sites in
  // the same layout, 4 bf16 per piece (residual emission); zeros outside
  typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
  typedef u32x2v Yv[WM][WN];
  __device__ __amdgpu_buffer_rsrc_t yres(const HaloTile& T) const {
    return frame_rsrc(static_cast<uint16_t*>(p.y) + (size_t)T.n * zimg, (uint32_t)(zimg * 2));
  }
  __device__ void load_y(Yv& dst, const HaloTile& T, bool none) const {
    const auto yrs = yres(T);
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int jn = 0; jn < WN; ++jn) {
        const uint32_t o = zoff(T, i, jn);
        dst[i][jn] = __builtin_bit_cast(
            u32x2v, __builtin_amdgcn_raw_buffer_load_b64(yrs, none || o == kOutOfRange ? kOutOfRange : o / 2, 0, 0));
      }
  }

  // z, y_new = dtype(act(z)) and the successor's residual r = fl32(y_new -
  // y_old) in fp32 and rounded to bf16, at the tile's sites
  __device__ void store_emit(const HaloTile& T, const Acc& acc, const Yv& yo) const {
    const auto zrs = zres(T);
    const auto yrs = yres(T);
    const auto rrs = frame_rsrc(p.r32 + (size_t)T.n * zimg, (uint32_t)(zimg * 4));
    const auto brs = frame_rsrc(p.rb + (size_t)T.n * zimg, (uint32_t)(zimg * 2));
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int jn = 0; jn < WN; ++jn) {
        const uint32_t o = zoff(T, i, jn);
        const uint32_t oh = o == kOutOfRange ? kOutOfRange : o / 2;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[i][jn]), zrs, o, 0, 0);
        uint32_t yn[4];
        floatx4 r;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          yn[v] = f32_to_bf16(activate(acc[i][jn][v], p.act));
          const uint32_t ob = (v < 2 ? yo[i][jn].x : yo[i][jn].y) >> (16 * (v & 1));
          r[v] = __fsub_rn(bf16_to_f32(yn[v]), bf16_to_f32(ob & 0xffffu));
        }
        __builtin_amdgcn_raw_buffer_store_b64(u32x2v{yn[0] | (yn[1] << 16), yn[2] | (yn[3] << 16)}, yrs, oh, 0, 0);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, r), rrs, o, 0, 0);
        __builtin_amdgcn_raw_buffer_store_b64(
            u32x2v{f32_to_bf16(r[0]) | (f32_to_bf16(r[1]) << 16), f32_to_bf16(r[2]) | (f32_to_bf16(r[3]) << 16)}, brs,
            oh, 0, 0);
      }
  }

  // z (and the activation output) of the tile's sites
  __device__ void store(const HaloTile& T, const Acc& acc) const {
    const auto zrs = zres(T);
    const auto yrs = frame_rsrc(p.act ? static_cast<uint16_t*>(p.y) + (size_t)T.n * zimg : nullptr,
                                p.act ? (uint32_t)(zimg * 2) : 0u);
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int jn = 0; jn < WN; ++jn) {
        const uint32_t o = zoff(T, i, jn);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[i][jn]), zrs, o, 0, 0);
        if (p.act) {
          const uint32_t lo = f32_to_bf16(activate(acc[i][jn][0], p.act)) |
                              (f32_to_bf16(activate(acc[i][jn][1], p.act)) << 16);
          const uint32_t hi = f32_to_bf16(activate(acc[i][jn][2], p.act)) |
                              (f32_to_bf16(activate(acc[i][jn][3], p.act)) << 16);
          typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
          __builtin_amdgcn_raw_buffer_store_b64(u32x2{lo, hi}, yrs, o == kOutOfRange ? kOutOfRange : o / 2, 0, 0);
        }
      }
  }
};

}  // namespace sc
