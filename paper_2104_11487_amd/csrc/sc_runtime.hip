// Host runtime of the Skip-Conv layer: descriptor validation, workspace
// layout, weight repack, ping-pong x_{t-1} slots, the per-frame launch
// sequence, introspection and kernel timing. Implements include/skipconv.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "skipconv.h"
#include "sc_kernels.h"

namespace {

thread_local char g_create_error[256] = "";

constexpr size_t kAlign = 256;
constexpr size_t kLdsLimit = 60 * 1024;  // dynamic; the gate kernel adds 2 KB static
constexpr int kMaxCout = 256;
constexpr long kHaloLdsLimit = 160 * 1024;  // LDS of one gfx950 CU
constexpr long kFusedLdsLimit = 156 * 1024; // dynamic LDS of the fused kernel (+ ~3 KB static)
constexpr long kCuGuess = 256;              // CUs assumed when a tiling is chosen before the device is queried

// Does every tile's halo contain the input pixels the tile owns?
int halo_covers_owned(int n_in, int n_out, int ts, int tiles, int s, int pad, int k) {
  for (int t = 0; t < tiles; ++t) {
    const int o0 = t * ts, on = std::min(ts, n_out - o0);
    const int hi = (o0 + on - 1) * s - pad + k - 1;
    const int own1 = t == tiles - 1 ? n_in : std::min(n_in, (o0 + ts) * s);
    if (own1 - 1 > hi) return 0;
  }
  return 1;
}

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct Geometry {
  int pad, h_out, w_out, hb, wb, nb;
  int ts, tiles_y, tiles_x, gate_grid, split_blocks;
  int seg_cap;          // work-list entries per gate tile (blocks of a tile); 0: ordered compaction
  int lane_sum;  // gate chunk sums combined in lane groups (no LDS staging)
  int hh_max, hw_max, halo_floats, stage_stride, rows_per_batch;
  size_t gate_lds;
  int copy_in_halo;
  bool depthwise;
  int kk, ksteps, ntn;  // dense: K, k-steps, 16-wide output tiles (padded to an instantiated count)
  bool fast;
  bool halo;            // dense bf16 block-halo kernel (else the gather kernel)
  sc::HaloParams hp;
  bool dw_halo;         // depthwise bf16: residual halo of tr x b sites in LDS
  sc::HaloParams dwp;
  bool fused;           // single-pass kernel instead of gate + compaction + conv
  int f_ts, f_tiles_y, f_tiles_x, f_grid, f_copy_in_halo;
  int f_nsplit;         // workgroups per tile of the register-operand kernel (output channels split)
  int f_kc, f_nchunks, f_nbuf, f_mw, f_pstride, f_zero_pix, f_off_b, f_off_halo, f_off_a, f_lds;
  int f_rb;             // register-operand fused kernel: its build (0: LDS operand)
  int f_dw;             // depthwise fused kernel: its halo rows per thread (0: not depthwise)
  int f_sc;             // few-channel fused kernel: 1 fp32 by elements, 4 fp32 by 4, 2 bf16 (0: none)
  int f_pstage, f_off_part;
  int vec;              // gate load width (elements)
  size_t elem;
  size_t off_wpack, off_slot0, off_slot1, off_z, off_y, off_bmask, off_tflag, off_list, off_ctr,
      off_stat, off_smask, off_phi, off_r32, off_rb, off_prev, off_z2, off_list_a, off_list_b, off_wlist, off_wctr,
      off_ftiles, total;
  int learned;          // learned gate: its kernel size (the layer's k), else 0
  bool phi_in_lds;      // learned gate: phi staged in LDS (else read through the caches)
  int phi_off;          // learned gate: LDS float offset of the staged phi
  int tr_off;           // learned gate over lane groups: LDS float offset of the tap-term exchange
  size_t wpack_bytes, x_bytes, z_bytes;
  int conv_max_tiles;
};

int fail(char* buf, int code, const char* msg) {
  if (buf) snprintf(buf, 256, "%s", msg);
  return code;
}

int ntn_for(int c_out) {
  const int t = (c_out + 15) / 16;
  static const int opts[] = {1, 2, 4, 8, 12, 16};
  for (int o : opts)
    if (t <= o) return o;
  return -1;
}

// Validates the descriptor and derives every size. Host only.
int derive(const skipconv_desc* d, Geometry* g, char* err) {
  if (!d) return fail(err, SKIPCONV_E_INVALID_ARG, "descriptor is NULL");
  if (d->n < 1 || d->h < 1 || d->w < 1 || d->c_in < 1 || d->c_out < 1)
    return fail(err, SKIPCONV_E_INVALID_ARG, "n, h, w, c_in and c_out must be >= 1");
  if (d->kernel < 1 || d->kernel % 2 == 0 || d->kernel > 7)
    return fail(err, SKIPCONV_E_INVALID_ARG, "kernel must be odd, 1..7");
  if (d->stride < 1 || d->stride > 4) return fail(err, SKIPCONV_E_INVALID_ARG, "stride must be 1..4");
  const int pad = d->pad == -1 ? (d->kernel - 1) / 2 : d->pad;
  if (pad < 0 || pad > d->kernel - 1)
    return fail(err, SKIPCONV_E_INVALID_ARG, "pad must be -1 or 0..kernel-1");
  if (d->groups < 1 || d->c_in % d->groups || d->c_out % d->groups)
    return fail(err, SKIPCONV_E_INVALID_ARG, "groups must divide c_in and c_out");
  const bool depthwise = d->groups > 1;
  if (depthwise && !(d->groups == d->c_in && d->c_out == d->c_in))
    return fail(err, SKIPCONV_E_UNSUPPORTED, "only groups == 1 or groups == c_in == c_out");
  if (d->block < 1 || d->block > 64) return fail(err, SKIPCONV_E_INVALID_ARG, "block must be 1..64");
  if (d->norm_p != 1 && d->norm_p != 2) return fail(err, SKIPCONV_E_INVALID_ARG, "norm_p must be 1 or 2");
  if (d->gate != SKIPCONV_GATE_INPUT_NORM && d->gate != SKIPCONV_GATE_OUTPUT_NORM &&
      d->gate != SKIPCONV_GATE_LEARNED)
    return fail(err, SKIPCONV_E_INVALID_ARG, "gate must be a SKIPCONV_GATE_* value");
  if (d->support != SKIPCONV_SUPPORT_RF && d->support != SKIPCONV_SUPPORT_CENTRE)
    return fail(err, SKIPCONV_E_INVALID_ARG, "unknown support");
  if (d->dtype != SKIPCONV_F32 && d->dtype != SKIPCONV_BF16)
    return fail(err, SKIPCONV_E_INVALID_ARG, "unknown dtype");
  if (d->act_out < SKIPCONV_ACT_NONE || d->act_out > SKIPCONV_ACT_RELU)
    return fail(err, SKIPCONV_E_INVALID_ARG, "unknown act_out");
  if ((d->flags & SKIPCONV_FLAG_EMIT_RESIDUAL) && d->act_out == SKIPCONV_ACT_NONE)
    return fail(err, SKIPCONV_E_INVALID_ARG, "EMIT_RESIDUAL needs an activation output");
  if ((d->flags & SKIPCONV_FLAG_EMIT_RESIDUAL) && (d->flags & SKIPCONV_FLAG_TRANSLATE))
    return fail(err, SKIPCONV_E_UNSUPPORTED, "EMIT_RESIDUAL and TRANSLATE cannot be combined");
  if (d->flags & ~(uint32_t)(SKIPCONV_FLAG_KEEP_STATS | SKIPCONV_FLAG_FORCE_DENSE | SKIPCONV_FLAG_SPLIT_PIPELINE |
                             SKIPCONV_FLAG_EMIT_RESIDUAL | SKIPCONV_FLAG_TRANSLATE |
                             SKIPCONV_FLAG_LARGE_GATE_TILES | SKIPCONV_FLAG_CALLER_RETAINS))
    return fail(err, SKIPCONV_E_INVALID_ARG, "unknown flag bits");
  if (std::isnan(d->eps) || d->eps < 0.0f) return fail(err, SKIPCONV_E_INVALID_ARG, "eps must be >= 0");
  if (!depthwise && d->c_out > kMaxCout) return fail(err, SKIPCONV_E_UNSUPPORTED, "c_out > 256");

  Geometry& G = *g;
  G = Geometry{};
  G.pad = pad;
  const int k = d->kernel, s = d->stride;
  G.h_out = (d->h + 2 * pad - k) / s + 1;
  G.w_out = (d->w + 2 * pad - k) / s + 1;
  if (d->h + 2 * pad < k || d->w + 2 * pad < k || G.h_out < 1 || G.w_out < 1)
    return fail(err, SKIPCONV_E_INVALID_ARG, "frame smaller than the kernel");
  const int b = d->block;
  G.hb = (G.h_out + b - 1) / b;
  G.wb = (G.w_out + b - 1) / b;
  const long nb = (long)d->n * G.hb * G.wb;
  const long sites = (long)d->n * G.h_out * G.w_out;
  const long xel = (long)d->n * d->h * d->w * d->c_in;
  if (nb > (1L << 30) || sites * d->c_out > (1L << 40) || xel > (1L << 40) ||
      (long)d->n * d->h * d->w > (1L << 31) - 1 || sites > (1L << 31) - 1)
    return fail(err, SKIPCONV_E_UNSUPPORTED, "tensor too large");
  G.nb = (int)nb;
  G.depthwise = depthwise;
  G.elem = d->dtype == SKIPCONV_BF16 ? 2 : 4;

  // gate tiling: ts x ts output sites made of whole blocks, about 16 x 16
  // sites, or 8 x 8 when 16 x 16 tiles would not give every CU two tiles or
  // their chunk sums would not fit in LDS. LDS: the a[] halo plus one fp32
  // chunk sum per (halo pixel, 8-channel chunk), odd row stride.
  const int nchk = (d->c_in + 7) / 8;
  G.stage_stride = nchk | 1;
  G.learned = d->gate == SKIPCONV_GATE_LEARNED ? k : 0;
  // norm gates with 2, 4, 8 or 16 chunks per pixel add a pixel's chunk sums
  // in registers (lane groups), and those with fewer than 8 channels sum a
  // pixel in one thread, without per-chunk staging in LDS; the kernel
  // addresses one image with 32-bit byte offsets (fp32 frames of chained
  // steps included)
  const bool lane_sum = !G.learned && (long)d->h * d->w * d->c_in * 4 < (1L << 31) &&
                        ((d->c_in % 8 == 0 && (nchk == 2 || nchk == 4 || nchk == 8 || nchk == 16)) || d->c_in < 8);
  // the learned gate takes the same lane groups (per-tap chunk terms) when
  // the channels come in 2, 4, 8 or 16 whole chunks
  const bool learned_lanes = G.learned && (long)d->h * d->w * d->c_in * 4 < (1L << 31) && d->c_in % 8 == 0 &&
                             (nchk == 2 || nchk == 4 || nchk == 8 || nchk == 16);
  G.lane_sum = (lane_sum || learned_lanes) ? 1 : 0;
  // learned gate: phi is staged in LDS unless that alone would not fit
  const long phi_floats = (long)k * k * d->c_in;
  G.phi_in_lds = G.learned && phi_floats * 4 <= (long)kLdsLimit / 2;
  auto gate_lds_for = [&](int ts) {
    const long eh = (long)(std::min(ts, G.h_out) - 1) * s + k;  // largest halo actually used
    const long ew = (long)(std::min(ts, G.w_out) - 1) * s + k;
    if (G.learned)  // per-pixel, per-tap gate terms (+ the staged phi, + the lane groups' tap-term exchange)
      return ((eh * ew * k * k + 3) / 4 * 4 + (G.phi_in_lds ? (phi_floats + 3) / 4 * 4 : 0) +
              (learned_lanes ? (long)sc::kGateThreads * std::min(k * k, sc::kLearnTapGroup) : 0)) * 4;
    const long halo = (eh * ew + 3) / 4 * 4;
    return (halo + (lane_sum ? 0 : eh * ew * G.stage_stride)) * 4;
  };
  {
    const int t32 = b <= 32 ? b * (32 / b) : b;
    const int t16 = b <= 16 ? b * (16 / b) : b;
    const int t8 = b <= 8 ? b * (8 / b) : b;
    auto tiles_for = [&](int t) { return (long)d->n * ((G.h_out + t - 1) / t) * ((G.w_out + t - 1) / t); };
    G.ts = (tiles_for(t16) < 512 && b <= 8) ? t8 : t16;
    // on request, 32 x 32 tiles when the chunk sums combine in registers: a
    // smaller share of re-read halo, but four times fewer workgroups (on
    // 4 x 512 x 512 x 128 frames 16 x 16 tiles are faster)
    if ((d->flags & SKIPCONV_FLAG_LARGE_GATE_TILES) && lane_sum && b <= 32 &&
        (t32 / b) * (t32 / b) <= sc::kMaxTileBlocks && gate_lds_for(t32) <= (long)kLdsLimit)
      G.ts = t32;
    if (G.learned && b <= 8) G.ts = t8;  // the per-tap learned gate is VALU-heavy: more, smaller tiles
    if (gate_lds_for(G.ts) > (long)kLdsLimit && b <= 8) G.ts = t8;
    // blocks larger than a tile that fits: 16 x 16 (or 8 x 8) tiles, one flag
    // per tile, OR-ed per block by the compaction kernel
    G.split_blocks = 0;
    if (gate_lds_for(G.ts) > (long)kLdsLimit && b > 16) {
      for (int t : {16, 8})
        if (b % t == 0 && gate_lds_for(t) <= (long)kLdsLimit) {
          G.ts = t;
          G.split_blocks = 1;
          break;
        }
    }
  }
  G.tiles_y = (G.h_out + G.ts - 1) / G.ts;
  G.tiles_x = (G.w_out + G.ts - 1) / G.ts;
  G.gate_grid = d->n * G.tiles_y * G.tiles_x;
  G.hh_max = (std::min(G.ts, G.h_out) - 1) * s + k;
  G.hw_max = (std::min(G.ts, G.w_out) - 1) * s + k;
  G.halo_floats = (G.hh_max * G.hw_max + 3) / 4 * 4;
  G.phi_off = (G.hh_max * G.hw_max * k * k + 3) / 4 * 4;
  G.tr_off = G.phi_off + (G.phi_in_lds ? (int)((phi_floats + 3) / 4 * 4) : 0);
  G.rows_per_batch = G.hh_max;
  G.gate_lds = gate_lds_for(G.ts);
  if (G.gate_lds > kLdsLimit)
    return fail(err, SKIPCONV_E_UNSUPPORTED, "gate tile does not fit in LDS (too many channels)");
  if (d->dtype == SKIPCONV_BF16)
    G.vec = (d->c_in % 8 == 0) ? 8 : 1;
  else
    G.vec = (d->c_in % 8 == 0) ? 8 : 1;

  // does every tile's halo cover the input pixels it owns?
  G.copy_in_halo = 1;
  for (int ty = 0; ty < G.tiles_y && G.copy_in_halo; ++ty) {
    const int oy0 = ty * G.ts, oh = std::min(G.ts, G.h_out - oy0);
    const int lo = oy0 * s - pad, hi = (oy0 + oh - 1) * s - pad + k - 1;
    const int own1 = ty == G.tiles_y - 1 ? d->h : std::min(d->h, (oy0 + G.ts) * s);
    if (oy0 * s < lo || own1 - 1 > hi) G.copy_in_halo = 0;
  }
  for (int tx = 0; tx < G.tiles_x && G.copy_in_halo; ++tx) {
    const int ox0 = tx * G.ts, ow = std::min(G.ts, G.w_out - ox0);
    const int lo = ox0 * s - pad, hi = (ox0 + ow - 1) * s - pad + k - 1;
    const int own1 = tx == G.tiles_x - 1 ? d->w : std::min(d->w, (ox0 + G.ts) * s);
    if (ox0 * s < lo || own1 - 1 > hi) G.copy_in_halo = 0;
  }

  // convolution geometry
  G.kk = k * k * (d->c_in / d->groups);
  if (!depthwise) {
    const int kstep = d->dtype == SKIPCONV_BF16 ? 32 : 4;
    G.ksteps = (G.kk + kstep - 1) / kstep;
    G.ntn = ntn_for(d->c_out);
    G.fast = d->dtype == SKIPCONV_BF16 && d->c_in % 32 == 0;
    G.wpack_bytes = (size_t)G.ksteps * G.ntn * 64 * (d->dtype == SKIPCONV_BF16 ? 16 : 4);
  } else {
    G.wpack_bytes = (size_t)k * k * d->c_in * 4;
  }
  const int conv_rows = (!depthwise && d->dtype == SKIPCONV_F32) ? sc::kConvF32Rows : 64;
  G.conv_max_tiles = (int)(((long)G.nb * b * b + conv_rows - 1) / conv_rows);

  // depthwise halo kernel: tiles of tr rows x b columns of an active block, tr
  // the largest row count (halving from b) whose halo and [tap][c] weights
  // fit in 64 KB of LDS; one image of x and z within 2^31 bytes
  G.dw_halo = false;
  if (depthwise && d->dtype == SKIPCONV_BF16 && d->c_in % 8 == 0 &&
      (long)d->h * d->w * d->c_in * 2 < (1L << 31) && (long)G.h_out * G.w_out * d->c_in * 4 < (1L << 31)) {
    sc::HaloParams& H = G.dwp;
    H.config = 0;
    H.pstride = 2 * d->c_in + 16;
    H.hw = (b - 1) * s + k;
    const long wbytes = (long)k * k * d->c_in * 4;
    for (int tr = b; tr >= 1; tr = tr > 1 ? (tr + 1) / 2 : 0) {
      const long hh = (long)(tr - 1) * s + k;
      if (hh * H.hw * H.pstride + wbytes <= 64 * 1024) {
        H.tr = tr;
        H.hh = (int)hh;
        H.tiles_per_block = (b + tr - 1) / tr;
        H.lds_bytes = (int)(hh * H.hw * H.pstride);
        H.threads = 256;
        G.dw_halo = true;
        G.conv_max_tiles = G.nb * H.tiles_per_block;
        break;
      }
      if (tr == 1) break;
    }
  }

  // block-halo kernel: tile = tr rows x b columns of a block, chosen per wave layout
  G.halo = false;
  // (one image of x and of z within 2^31 bytes: the kernel addresses them
  // through buffer resources with 32-bit offsets)
  if (!depthwise && d->dtype == SKIPCONV_BF16 && d->c_in % 32 == 0 &&
      d->c_out % 4 == 0 && (b == 4 || b == 8 || b == 16 || b == 32 || b == 64) &&
      (long)d->h * d->w * d->c_in * 2 < (1L << 31) && (long)G.h_out * G.w_out * d->c_out * 4 < (1L << 31)) {
    static const int ntns[] = {1, 2, 4, 8, 12, 16};
    int ni = 0;
    while (ntns[ni] != G.ntn) ++ni;
    sc::HaloParams& H = G.hp;
    // waves: 1 along M x WAVES_N along N; each wave owns all rows of the tile
    if (b >= 16) {
      if (G.ntn <= 8) {  // 128-site tiles, WM = 8
        H.tr = 128 / b;
        H.config = G.ntn == 1 ? 0 : (G.ntn == 2 ? 1 : (G.ntn == 4 ? 2 : 3));
      } else {           // 64-site tiles, WM = 4
        H.tr = 64 / b;
        H.config = G.ntn == 12 ? 14 : 15;
      }
    } else if (b == 8) {  // the whole block: 64 sites, WM = 4
      H.tr = 8;
      H.config = 10 + ni;
    } else {              // b = 4: 16 sites, WM = 1
      H.tr = 4;
      H.config = 20 + ni;
    }
    H.threads = 64 * (G.ntn == 1 ? 1 : (G.ntn == 2 ? 2 : 4));
    // emitting layers: the epilogue writes the successor's residual (16-byte
    // r32 pieces of 4 channels, whole 8-channel groups for the clears)
    H.emit = (d->flags & SKIPCONV_FLAG_EMIT_RESIDUAL) && d->c_out % 8 == 0 ? 1 : 0;
    H.tiles_per_block = b / H.tr;
    H.hh = (H.tr - 1) * s + k;
    H.hw = (b - 1) * s + k;
    H.pstride = 2 * d->c_in + 16;
    const long lds = (long)H.hh * H.hw * H.pstride;
    if (lds <= kHaloLdsLimit) {
      H.lds_bytes = (int)lds;
      G.halo = true;
      G.conv_max_tiles = G.nb * H.tiles_per_block;
    }
  }

  // fused single-pass kernel: dense bf16, C_in % 32 == 0, tiles of <= 16 x 16
  // sites, output tiles split over two wave groups (ntn >= 2)
  G.fused = false;
  G.f_dw = 0;
  G.f_sc = 0;
  // the learned gate runs in the register-operand build when a pixel's chunks
  // form one lane group (C_in 32, 64 or 128) and phi fits its staging loads
  const bool learned_fused = !G.learned || ((d->c_in == 32 || d->c_in == 64 || d->c_in == 128) &&
                                            (long)k * k * d->c_in <= (long)sc::kFusedPhiLoads * 512 * 4);
  if (!depthwise && d->dtype == SKIPCONV_BF16 && d->c_in % 32 == 0 && d->c_out % 4 == 0 && b <= 16 &&
      G.ntn >= 2 && learned_fused && !(d->flags & SKIPCONV_FLAG_SPLIT_PIPELINE)) {
    const int ts = b <= 8 ? b * (8 / b) : b;
    const int mw = ts <= 8 ? 1 : 4;
    if (!(mw == 4 && G.ntn > 8)) {
      const int hh = (ts - 1) * s + k;
      const long pstride = 2L * d->c_in + 16;
      const long halo_b = ((long)hh * hh + 1) * pstride;  // + the zero pixel
      // pixel statistics (learned gate: per-tap terms) and parked chunk sums
      // (learned gate: the staged phi)
      const long a_b = ((long)hh * hh * (G.learned ? k * k : 1) * 4 + 15) / 16 * 16;
      const int pstage = (d->c_in / 8) | 1;
      const long part_b = std::max(((long)hh * hh * pstage * 4 + 15) / 16 * 16,
                                   G.learned ? (long)k * k * d->c_in * 4 : 0L);
      const long whole = (long)G.ksteps * G.ntn * 1024;
      long b_bytes = whole;
      int kc = G.ksteps, nbuf = 1;
      // tiles of <= 8 x 8 sites: register-operand kernel when instantiated for
      // the shape; LDS holds the partial sums of its k-parts instead of weights
      int rb = mw == 1 ? sc::fused_rb_kps(G.ntn, G.ksteps, hh, d->c_in / 8) : 0;
      // no build for the whole width, or a wide layer with few tiles (>= 192
      // output channels and fewer tiles than half the CUs, or >= 128 and
      // fewer than a quarter; narrower layers and more tiles measured slower
      // split, e.g. 64 -> 64 on 192 tiles: 7.1 -> 10.5 us): the output
      // channels split over 2, 4 or 8 workgroups per tile, each a build for
      // its share (fewer k-steps per wave, so the weight fragments still fit
      // in registers; fewer epilogue pieces per thread)
      const long tiles = (long)d->n * ((G.h_out + ts - 1) / ts) * ((G.w_out + ts - 1) / ts);
      const bool wide_few = (G.ntn >= 12 && tiles * 2 < kCuGuess) || (G.ntn >= 8 && tiles * 4 < kCuGuess);
      int nsplit = 1;
      for (int sp = 2; mw == 1 && (!rb || wide_few) && sp <= 8; sp *= 2) {
        const int r = G.ntn % sp == 0 ? sc::fused_rb_kps(G.ntn / sp, G.ksteps, hh, d->c_in / 8) : 0;
        if (r) {
          rb = r;
          nsplit = sp;
          break;
        }
      }
      G.f_nsplit = nsplit;
      if (rb) {
        const long kparts = sc::fused_rb_kparts(rb);
        b_bytes = kparts * 64 * ((long)(G.ntn / nsplit) * 64 + 16);
      } else if (G.learned) {
        b_bytes = kFusedLdsLimit + 1;  // the learned gate has the register-operand build only
      } else if (whole + halo_b + a_b + part_b > kFusedLdsLimit) {
        kc = std::max(1, 16 / G.ntn);
        nbuf = 2;
        b_bytes = (long)nbuf * kc * G.ntn * 1024;
      }
      if (b_bytes + halo_b + a_b + part_b <= kFusedLdsLimit) {
        G.fused = true;
        G.f_ts = ts;
        G.f_mw = mw;
        G.f_rb = rb;
        G.f_kc = kc;
        G.f_nbuf = nbuf;
        G.f_nchunks = (G.ksteps + kc - 1) / kc;
        G.f_pstride = (int)pstride;
        G.f_zero_pix = hh * hh;
        G.f_off_b = 0;
        G.f_off_halo = (int)b_bytes;
        G.f_off_a = (int)(b_bytes + halo_b);
        G.f_off_part = (int)(b_bytes + halo_b + a_b);
        G.f_pstage = pstage;
        G.f_lds = (int)(b_bytes + halo_b + a_b + part_b);
        G.f_tiles_y = (G.h_out + ts - 1) / ts;
        G.f_tiles_x = (G.w_out + ts - 1) / ts;
        G.f_grid = d->n * G.f_tiles_y * G.f_tiles_x;
        if (G.f_tiles_x > 1024 || G.f_tiles_y > 1024 || d->n > 4096) G.fused = false;
        G.f_copy_in_halo = halo_covers_owned(d->h, G.h_out, ts, G.f_tiles_y, s, pad, k) &&
                           halo_covers_owned(d->w, G.w_out, ts, G.f_tiles_x, s, pad, k);
      }
    }
  }
  // fused single-pass kernel for few input channels (fp32 C_in <= 16, bf16
  // C_in < 8): tiles of <= 8 x 8 sites, C_out <= 64, two k-parts of at most
  // kScStepsF32 (kScStepsBf16) k-steps
  const bool few = d->dtype == SKIPCONV_F32 ? d->c_in <= 16 : d->c_in < 8;
  if (!depthwise && few && d->c_out % 4 == 0 && G.ntn >= 1 && G.ntn <= 4 && G.ntn != 3 && b <= 8 &&
      !G.learned && !(d->flags & SKIPCONV_FLAG_SPLIT_PIPELINE) &&
      (G.ksteps + 1) / 2 <= (d->dtype == SKIPCONV_F32 ? sc::kScStepsF32 : sc::kScStepsBf16)) {
    const int ts = b * (8 / b);
    const int hh = (ts - 1) * s + k;
    const long rh_b = ((long)hh * hh * d->c_in * 4 + 15) / 16 * 16;
    const long a_b = ((long)hh * hh * 4 + 15) / 16 * 16;
    const long part_b = 4L * G.ntn * 64 * 16;
    if (rh_b + a_b + part_b <= kFusedLdsLimit) {
      G.fused = true;
      G.f_sc = d->dtype == SKIPCONV_BF16 ? 2 : (d->c_in % 4 == 0 ? 4 : 1);
      G.f_nsplit = 1;
      G.f_ts = ts;
      G.f_mw = 1;
      G.f_rb = 0;
      G.f_kc = G.f_nchunks = G.f_nbuf = 0;
      G.f_pstride = 0;
      G.f_zero_pix = hh * hh;
      G.f_off_b = 0;
      G.f_off_halo = (int)part_b;
      G.f_off_a = (int)(part_b + rh_b);
      G.f_off_part = G.f_off_a;
      G.f_pstage = 1;
      G.f_lds = (int)(part_b + rh_b + a_b);
      G.f_tiles_y = (G.h_out + ts - 1) / ts;
      G.f_tiles_x = (G.w_out + ts - 1) / ts;
      G.f_grid = d->n * G.f_tiles_y * G.f_tiles_x;
      if (G.f_tiles_x > 1024 || G.f_tiles_y > 1024 || d->n > 4096) G.fused = false;
      G.f_copy_in_halo = halo_covers_owned(d->h, G.h_out, ts, G.f_tiles_y, s, pad, k) &&
                         halo_covers_owned(d->w, G.w_out, ts, G.f_tiles_x, s, pad, k);
    }
  }
  // fused single-pass depthwise kernel: bf16, C % 8 == 0, tiles of <= 8 x 8
  // sites; the channels split over 2, 4 or 8 workgroups per tile until each
  // owns at most kDwSplitMax; the halo taken in one round
  if (depthwise && d->dtype == SKIPCONV_BF16 && d->c_in % 8 == 0 && b <= 8 && !G.learned &&
      !(d->flags & SKIPCONV_FLAG_SPLIT_PIPELINE)) {
    const int ts = b * (8 / b);
    const int hh = (ts - 1) * s + k;
    const int nchk = d->c_in / 8;
    int nsplit = 1;
    while (d->c_in / nsplit > sc::kDwSplitMax && nsplit < 8 && nchk % (2 * nsplit) == 0) nsplit *= 2;
    const int ki = sc::fused_dw_ki(hh, nchk);
    if (d->c_in / nsplit <= sc::kDwSplitMax && ki) {
      const long pstride = 2L * d->c_in + 16;
      const long w_b = ((long)k * k * (d->c_in / nsplit) * 4 + 15) / 16 * 16;
      const long halo_b = ((long)hh * hh + 1) * pstride;
      const long a_b = ((long)hh * hh * 4 + 15) / 16 * 16;
      const int pstage = nchk | 1;
      const long part_b = ((long)hh * hh * pstage * 4 + 15) / 16 * 16;
      if (w_b + halo_b + a_b + part_b <= kFusedLdsLimit) {
        G.fused = true;
        G.f_dw = ki;
        G.f_nsplit = nsplit;
        G.f_ts = ts;
        G.f_mw = 1;
        G.f_rb = 0;
        G.f_kc = G.f_nchunks = G.f_nbuf = 0;
        G.f_pstride = (int)pstride;
        G.f_zero_pix = hh * hh;
        G.f_off_b = 0;
        G.f_off_halo = (int)w_b;
        G.f_off_a = (int)(w_b + halo_b);
        G.f_off_part = (int)(w_b + halo_b + a_b);
        G.f_pstage = pstage;
        G.f_lds = (int)(w_b + halo_b + a_b + part_b);
        G.f_tiles_y = (G.h_out + ts - 1) / ts;
        G.f_tiles_x = (G.w_out + ts - 1) / ts;
        G.f_grid = d->n * G.f_tiles_y * G.f_tiles_x;
        if (G.f_tiles_x > 1024 || G.f_tiles_y > 1024 || d->n > 4096) G.fused = false;
        G.f_copy_in_halo = halo_covers_owned(d->h, G.h_out, ts, G.f_tiles_y, s, pad, k) &&
                           halo_covers_owned(d->w, G.w_out, ts, G.f_tiles_x, s, pad, k);
      }
    }
  }

  G.x_bytes = (size_t)xel * G.elem;
  G.z_bytes = (size_t)sites * d->c_out * 4;
  size_t off = 0;
  G.off_wpack = off; off = align_up(off + G.wpack_bytes);
  // the x_{t-1} ping-pong slots (none when the caller retains its frames)
  const size_t slot_bytes = (d->flags & SKIPCONV_FLAG_CALLER_RETAINS) ? 0 : G.x_bytes;
  G.off_slot0 = off; off = align_up(off + slot_bytes);
  G.off_slot1 = off; off = align_up(off + slot_bytes);
  G.off_z = off; off = align_up(off + G.z_bytes);
  G.off_y = off;
  if (d->act_out != SKIPCONV_ACT_NONE) off = align_up(off + (size_t)sites * d->c_out * G.elem);
  G.off_bmask = off; off = align_up(off + (size_t)nb + 16);  // zero padding to whole 16-byte words
  G.off_tflag = off; off = align_up(off + (size_t)G.gate_grid);
  G.off_list = off; off = align_up(off + (size_t)nb * 4);
  // unordered work list of the split pipeline: seg_cap entries per gate tile
  // (its blocks), in kSegs segments with their counters in two alternating slots
  G.seg_cap = G.split_blocks ? 0 : (G.ts / b) * (G.ts / b);
  G.off_wlist = off; off = align_up(off + (size_t)std::max<long>(nb, (long)G.gate_grid * G.seg_cap) * 4);
  G.off_ctr = off; off = align_up(off + sc::kNumCounters * 4);
  G.off_wctr = off; off = align_up(off + 2 * sc::kSegs * sc::kSegStride * 4);
  G.off_ftiles = off;
  if (G.fused) off = align_up(off + (size_t)G.f_grid * 4);  // tile table of the fused kernel
  G.off_stat = off;
  G.off_smask = off;
  if (d->flags & SKIPCONV_FLAG_KEEP_STATS) {
    off = align_up(off + (size_t)sites * 4);
    G.off_smask = off;
    off = align_up(off + (size_t)sites);
  }
  G.off_phi = off;
  if (G.learned) off = align_up(off + (size_t)k * k * d->c_in * 4);
  G.off_r32 = G.off_rb = G.off_prev = off;
  if (d->flags & SKIPCONV_FLAG_EMIT_RESIDUAL) {  // residual handed to a chained successor
    off = align_up(off + (size_t)sites * d->c_out * 4);
    G.off_rb = off;
    if (d->dtype == SKIPCONV_BF16) off = align_up(off + (size_t)sites * d->c_out * 2);
    G.off_prev = off;
    off = align_up(off + (size_t)nb + 16);
  }
  G.off_z2 = G.off_list_a = G.off_list_b = off;
  if (d->flags & SKIPCONV_FLAG_TRANSLATE) {  // second z slot and the two block lists
    off = align_up(off + G.z_bytes);
    G.off_list_a = off;
    off = align_up(off + (size_t)nb * 4);
    G.off_list_b = off;
    off = align_up(off + (size_t)nb * 4);
  }
  G.total = off;
  return SKIPCONV_OK;
}

}  // namespace

struct skipconv_layer {
  skipconv_desc d;
  Geometry g;
  int device = 0;
  int num_cu = 256;
  int conv_occ = 4;          // resident conv workgroups per CU
  double wnorm = 1.0;        // gate weight factor: 1 (Input-Norm) or the weight norm (Output-Norm)
  bool list_valid = false;   // active list/count match the last step (fused steps skip them)
  char* ws = nullptr;
  bool owns_ws = false;
  int cur = 0;               // slot holding x_{t-1}
  const void* last_x = nullptr;  // CALLER_RETAINS: the previous step's x_t (NULL after create/reset)
  bool ref_pending = true;
  long long frames = 0;
  char last_error[256] = "";
  // timing
  std::vector<hipEvent_t> ev;
  std::vector<int32_t> ev_step;
  int timing_frames = 0, timing_done = 0, timing_every = 1, timing_seen = 0;

  void* wpack() { return ws + g.off_wpack; }
  void* slot(int i) { return ws + (i ? g.off_slot1 : g.off_slot0); }
  bool retains() const { return (d.flags & SKIPCONV_FLAG_CALLER_RETAINS) != 0; }
  // x_{t-1} as the kernels read it (x_t stands in on a reference frame, which
  // reads no x_{t-1}), and where the gate copies x_t (NULL: no copy)
  const void* prev_input(const void* x_t) { return retains() ? (last_x ? last_x : x_t) : slot(cur); }
  void* keep_slot() { return retains() ? nullptr : slot(cur ^ 1); }
  // the state update of Eq. 2 once the step's work is enqueued
  void advance_input(const void* x_t) {
    if (retains()) last_x = x_t;
    else cur ^= 1;
  }
  int zslot = 0;             // translated steps alternate z between two slots
  float* z() { return reinterpret_cast<float*>(ws + (zslot ? g.off_z2 : g.off_z)); }
  float* z_other() { return reinterpret_cast<float*>(ws + (zslot ? g.off_z : g.off_z2)); }
  void* y() { return d.act_out ? (void*)(ws + g.off_y) : nullptr; }
  uint8_t* bmask() { return reinterpret_cast<uint8_t*>(ws + g.off_bmask); }
  uint8_t* tflags() { return reinterpret_cast<uint8_t*>(ws + g.off_tflag); }
  uint32_t* list() { return reinterpret_cast<uint32_t*>(ws + g.off_list); }
  uint32_t* ctr() { return reinterpret_cast<uint32_t*>(ws + g.off_ctr); }
  float* stat() { return reinterpret_cast<float*>(ws + g.off_stat); }
  uint8_t* smask() { return reinterpret_cast<uint8_t*>(ws + g.off_smask); }
  float* phi() { return reinterpret_cast<float*>(ws + g.off_phi); }
  bool emits() const { return (d.flags & SKIPCONV_FLAG_EMIT_RESIDUAL) != 0; }
  float* r32() { return reinterpret_cast<float*>(ws + g.off_r32); }
  uint16_t* rb() { return reinterpret_cast<uint16_t*>(ws + g.off_rb); }
  uint8_t* prev_mask() { return reinterpret_cast<uint8_t*>(ws + g.off_prev); }
  bool phi_set = false;      // learned gate: skipconv_set_gate_weights was called
  // split pipeline work list: the gate appends active blocks (unordered) and
  // counts them in the kSegs segment counters of slot wslot; the convolution
  // clears the other slot's counters for the next step. wclean: a slot's
  // counters are known to be zero.
  int wslot = 0;
  bool wclean[2] = {true, true};
  // the list the last step's convolution walked: 0 none (one-pass kernel),
  // 1 the ordered list, 2 the segmented work list of slot work_slot
  int work_kind = 0, work_slot = 0;
  uint32_t* wlist() { return reinterpret_cast<uint32_t*>(ws + g.off_wlist); }
  uint32_t* wctr() { return reinterpret_cast<uint32_t*>(ws + g.off_wctr); }
  float gate_bias = 0.0f;
};

namespace {

sc::GateParams gate_params(skipconv_layer* h, const void* x_t, bool ref);

// Kernel parameters of the fused single-pass kernel (x_t / reference set per step).
sc::FusedParams fused_params(skipconv_layer* h, const void* x_t, bool ref) {
  const skipconv_desc& d = h->d;
  const Geometry& g = h->g;
  sc::FusedParams fp{};
  fp.g = gate_params(h, x_t, ref);
  fp.g.ts = g.f_ts;
  fp.g.tiles_y = g.f_tiles_y;
  fp.g.tiles_x = g.f_tiles_x;
  fp.g.copy_in_halo = g.f_copy_in_halo;
  fp.wpack = h->wpack();
  fp.z = h->z();
  fp.y = h->y();
  fp.c_out = d.c_out;
  fp.ntiles_n = g.ntn;
  fp.ksteps = g.ksteps;
  fp.csteps = d.c_in / 32;
  fp.act = d.act_out;
  fp.emit = h->emits() ? 1 : 0;  // the epilogue also writes the successor's residual
  fp.r32 = h->r32();
  fp.rb = d.dtype == SKIPCONV_BF16 ? h->rb() : nullptr;  // the bf16 rounding of r: bf16 layers only
  fp.prev_mask = h->prev_mask();
  fp.kc = g.f_kc;
  fp.nchunks = g.f_nchunks;
  fp.nbuf = g.f_nbuf;
  fp.mw = g.f_mw;
  fp.rbk = g.f_rb;
  fp.nsplit = (g.f_rb || g.f_dw) ? g.f_nsplit : 1;
  fp.dw = g.f_dw;
  fp.sc = g.f_sc;
  fp.trans_ok = (d.flags & SKIPCONV_FLAG_TRANSLATE) ? 1 : 0;
  fp.tiles = reinterpret_cast<const uint32_t*>(h->ws + g.off_ftiles);
  fp.inv_ts = 1.0f / (float)g.f_ts;
  fp.inv_blk = 1.0f / (float)d.block;
  fp.inv_hw = 1.0f / (float)((g.f_ts - 1) * d.stride + d.kernel);
  fp.inv_chk = 1.0f / (float)(d.c_in / 8);
  fp.pstride = g.f_pstride;
  fp.zero_pix = g.f_zero_pix;
  fp.off_b = g.f_off_b;
  fp.off_halo = g.f_off_halo;
  fp.off_a = g.f_off_a;
  fp.off_part = g.f_off_part;
  fp.pstage = g.f_pstage;
  fp.lds_bytes = g.f_lds;
  return fp;
}

// Output-Norm gate (Eq. 7): the norm of the whole weight tensor, in the power
// of the statistic (sum |w| for p = 1, sum w^2 for p = 2), summed in fp64 in
// ascending OIHW order. |w| and w^2 of fp32 / bf16 values are exact in fp64,
// so the only roundings are the additions, in that order. The weights are
// read back once, at create (a host synchronisation on `st`).
hipError_t weight_norm(skipconv_layer* h, const void* weights, hipStream_t st) {
  const skipconv_desc& d = h->d;
  const size_t numel = (size_t)d.c_out * (d.c_in / d.groups) * d.kernel * d.kernel;
  const size_t esz = d.dtype == SKIPCONV_BF16 ? 2 : 4;
  std::vector<uint8_t> host(numel * esz);
  hipError_t e = hipMemcpyAsync(host.data(), weights, host.size(), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return e;
  double acc = 0.0;
  for (size_t i = 0; i < numel; ++i) {
    float f;
    if (esz == 2) {
      uint16_t b;
      std::memcpy(&b, host.data() + 2 * i, 2);
      const uint32_t u = (uint32_t)b << 16;
      std::memcpy(&f, &u, 4);
    } else {
      std::memcpy(&f, host.data() + 4 * i, 4);
    }
    const double v = (double)f;
    const double term = d.norm_p == 1 ? std::fabs(v) : v * v;
    acc = acc + term;
  }
  h->wnorm = acc;
  return hipSuccess;
}

// The split pipeline's convolution writes the emitted residual itself (the
// block-halo kernel's emitting build) instead of the emission kernel.
bool conv_emits(const Geometry& g) { return g.halo && !g.depthwise && g.hp.emit; }

// After a split-pipeline step of an emitting layer: the residual at the blocks
// it updated (unless its block-halo convolution emitted them in its
// epilogue) and zeros at the blocks only the previous step updated.
hipError_t launch_emit(skipconv_layer* h, hipStream_t st) {
  const Geometry& g = h->g;
  return sc::launch_emit(h->bmask(), h->prev_mask(), g.nb, h->z(), h->y(), h->r32(), h->rb(), h->d.n, g.hb,
                         g.wb, h->d.block, g.h_out, g.w_out, h->d.c_out, h->d.act_out,
                         h->d.dtype == SKIPCONV_BF16 ? 1 : 0, conv_emits(g) ? 1 : 0, st);
}

int hip_fail(skipconv_t h, hipError_t e, const char* what) {
  if (h) snprintf(h->last_error, sizeof(h->last_error), "%s: %s", what, hipGetErrorString(e));
  return SKIPCONV_E_HIP;
}

double threshold(const skipconv_desc& d) {
  const double e = (double)d.eps;  // fp32 -> fp64 is exact; e * e is exact in fp64
  return d.norm_p == 2 ? e * e : e;
}

// Gate parameters that follow from the descriptor and geometry alone (no buffers).
sc::GateParams gate_geometry(const skipconv_desc& d, const Geometry& g, bool ref) {
  sc::GateParams gp{};
  gp.n = d.n; gp.h = d.h; gp.w = d.w; gp.c = d.c_in;
  gp.h_out = g.h_out; gp.w_out = g.w_out; gp.k = d.kernel; gp.stride = d.stride; gp.pad = g.pad;
  gp.block = d.block; gp.hb = g.hb; gp.wb = g.wb;
  gp.ts = g.ts; gp.tiles_y = g.tiles_y; gp.tiles_x = g.tiles_x;
  gp.halo_floats = g.halo_floats; gp.stage_stride = g.stage_stride; gp.lane_sum = g.lane_sum;
  gp.rows_per_batch = g.rows_per_batch; gp.copy_in_halo = g.copy_in_halo;
  gp.norm_p = d.norm_p; gp.support = d.support; gp.reference = ref ? 1 : 0; gp.no_prev = ref ? 1 : 0;
  gp.force_dense = (d.flags & SKIPCONV_FLAG_FORCE_DENSE) ? 1 : 0;
  gp.keep_stats = (d.flags & SKIPCONV_FLAG_KEEP_STATS) ? 1 : 0;
  gp.thr = threshold(d);
  gp.wnorm = 1.0;
  gp.learned = g.learned;
  gp.phi_off = g.phi_in_lds ? g.phi_off : -1;
  gp.tr_off = g.tr_off;
  gp.split_blocks = g.split_blocks;
  return gp;
}

sc::GateParams gate_params(skipconv_layer* h, const void* x_t, bool ref) {
  sc::GateParams gp = gate_geometry(h->d, h->g, ref);
  gp.x_t = x_t;
  gp.x_prev = h->prev_input(x_t);
  gp.x_keep = h->keep_slot();
  gp.wnorm = h->wnorm;
  gp.phi = h->phi();
  gp.gate_bias = h->gate_bias;
  gp.block_mask = h->bmask(); gp.list = h->list(); gp.counters = h->ctr();
  gp.tile_flags = h->tflags();
  gp.stat = h->stat(); gp.site_mask = h->smask();
  return gp;
}

// Convolution parameters that follow from the descriptor and geometry alone.
sc::ConvParams conv_geometry(const skipconv_desc& d, const Geometry& g, bool ref) {
  sc::ConvParams cp{};
  cp.n = d.n; cp.h = d.h; cp.w = d.w; cp.c = d.c_in; cp.c_out = d.c_out;
  cp.h_out = g.h_out; cp.w_out = g.w_out; cp.k = d.kernel; cp.stride = d.stride; cp.pad = g.pad;
  cp.block = d.block; cp.hb = g.hb; cp.wb = g.wb;
  cp.ksteps = g.ksteps; cp.ntiles_n = g.ntn;
  cp.reference = ref ? 1 : 0;
  cp.no_prev = ref ? 1 : 0;
  cp.act = ((d.flags & SKIPCONV_FLAG_EMIT_RESIDUAL) && !conv_emits(g)) ? 0 : d.act_out;
  return cp;
}

// The split pipeline's convolution kernel for this geometry.
hipError_t launch_split_conv(const Geometry& g, const skipconv_desc& d, const sc::ConvParams& cp, int grid,
                             hipStream_t st) {
  if (g.depthwise)
    return g.dw_halo ? sc::launch_depthwise_halo(cp, g.dwp, grid, st) : sc::launch_depthwise(cp, d.dtype, grid, st);
  if (g.halo) return sc::launch_conv_halo(cp, g.hp, grid, st);
  return sc::launch_conv(cp, d.dtype, g.fast, grid, st);
}

// Check that the split pipeline's convolution kernel fits the device (else
// fall back to the per-site kernels) and return its resident workgroups per CU.
int conv_setup(Geometry& g, const skipconv_desc* d, int device) {
  int occ_out = 4;
  if (g.dw_halo) {
    const int occ = sc::depthwise_halo_occupancy(g.dwp, d->kernel, d->c_in);
    if (occ < 1) {
      g.dw_halo = false;  // cannot hold the halo: per-site depthwise kernel
      g.conv_max_tiles = (int)(((long)g.nb * d->block * d->block + 63) / 64);
    } else {
      occ_out = std::min(8, occ);
    }
  }
  if (g.halo) {
    int max_lds = 0;
    if (hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, device) != hipSuccess ||
        max_lds < g.hp.lds_bytes) {
      g.halo = false;  // this device cannot hold the halo: gather kernel
      g.conv_max_tiles = (int)(((long)g.nb * d->block * d->block + 63) / 64);
    } else {
      occ_out = std::max(1, std::min(8, sc::conv_halo_occupancy(g.hp)));
    }
  }
  return occ_out;
}

// Two rounds of resident workgroups: the tiles of a step rarely divide into
// one round evenly, and queued workgroups fill the CUs the first round leaves
// idle (4 x 512 x 512 x 128 at 25 %: 283-284 -> 281 us per step; four rounds
// 286-287 us).
int conv_grid_of(const Geometry& g, int num_cu, int occ) {
  int grid = std::min(g.conv_max_tiles, num_cu * occ * 2);
  if (grid >= 8) grid = (grid + 7) / 8 * 8;
  return std::max(grid, 1);
}

hipError_t launch_compaction(skipconv_layer* h, hipStream_t st) {
  const Geometry& g = h->g;
  return sc::launch_compact(h->bmask(), g.nb, h->list(), h->ctr(), g.split_blocks ? h->tflags() : nullptr,
                            h->d.n, g.hb, g.wb, g.split_blocks ? h->d.block / g.ts : 0, g.tiles_y, g.tiles_x,
                            st);
}

// The list the split pipeline's convolution walks this step. Layers whose
// blocks are larger than the gate tiles need the ordered compaction (block
// flags are OR-ed over tiles first); every other layer takes the work list
// the gate kernel appends to, with no compaction launch.
struct StepList {
  const uint32_t* list;
  uint32_t* counters;  // counters[kCtrCount] = number of blocks in `list`, or kSegs segment counters
  uint32_t* zero;      // counters the convolution clears for the next step
  int seg_tiles, seg_cap;  // segmented work list (0: plain)
};

hipError_t begin_list(skipconv_layer* h, sc::GateParams& gp, hipStream_t st, StepList* out) {
  if (h->g.split_blocks) {
    *out = StepList{h->list(), h->ctr(), nullptr, 0, 0};
    h->work_kind = 1;
    return hipSuccess;
  }
  const int slot = h->wslot;
  h->work_kind = 2;
  h->work_slot = slot;
  constexpr int kSlot = sc::kSegs * sc::kSegStride;
  uint32_t* c = h->wctr() + slot * kSlot;
  hipError_t e = hipSuccess;
  if (!h->wclean[slot]) e = sc::launch_fill_u32(c, kSlot, 0u, st);
  gp.wlist = h->wlist();
  gp.wctr = c;
  gp.seg_cap = h->g.seg_cap;
  *out = StepList{h->wlist(), c, h->wctr() + (slot ^ 1) * kSlot, h->g.gate_grid, h->g.seg_cap};
  return e;
}

// After the gate: the ordered compaction when needed; called once per step.
hipError_t gate_done(skipconv_layer* h, hipStream_t st) {
  if (h->g.split_blocks) {
    h->list_valid = true;
    return launch_compaction(h, st);
  }
  h->list_valid = false;  // the ordered list is built on demand for introspection
  return hipSuccess;
}

// After the convolution that cleared the other counter.
void end_list(skipconv_layer* h) {
  if (h->g.split_blocks) return;
  h->wclean[h->wslot ^ 1] = true;
  h->wclean[h->wslot] = false;
  h->wslot ^= 1;
}

int conv_grid(const skipconv_layer* h) { return conv_grid_of(h->g, h->num_cu, h->conv_occ); }

// ---- scratch of skipconv_step_static ----
// The work list, its counters, the block flags and the packed weights of a
// step made by skipconv_step_static live in one file-scope device array of
// fixed size. Each device holds its own copy, at its own address, until the
// process ends; host code reaches it only through the address that
// hipGetSymbolAddress returns on that device (the array's name is a host-side
// stand-in, not a device address).
constexpr size_t kStaticScratchBytes = (size_t)4 << 20;
constexpr int kMaxStaticDevices = 64;
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];
std::mutex g_static_mu;
void* g_static_ptr[kMaxStaticDevices];
int g_static_cu[kMaxStaticDevices];

// Once per device, with that device current: the scratch array's device
// address and the device's CU count.
int static_scratch(void** ptr, int* device, int* num_cu) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(g_create_error, SKIPCONV_E_HIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxStaticDevices) return fail(g_create_error, SKIPCONV_E_UNSUPPORTED, "device index too large");
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (!g_static_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      snprintf(g_create_error, sizeof(g_create_error), "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
      return SKIPCONV_E_HIP;
    }
    int cu = 0;
    e = hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess || cu < 1) return fail(g_create_error, SKIPCONV_E_HIP, "CU count query failed");
    g_static_cu[dev] = cu;
    g_static_ptr[dev] = p;
  }
  *ptr = g_static_ptr[dev];
  *device = dev;
  *num_cu = g_static_cu[dev];
  return SKIPCONV_OK;
}


void destroy_events(skipconv_layer* h) {
  for (hipEvent_t e : h->ev) (void)hipEventDestroy(e);
  h->ev.clear();
  h->ev_step.clear();
  h->timing_frames = h->timing_done = h->timing_seen = 0;
  h->timing_every = 1;
}

}  // namespace

extern "C" {

int skipconv_desc_init(skipconv_desc* d) {
  if (!d) return SKIPCONV_E_INVALID_ARG;
  std::memset(d, 0, sizeof(*d));
  d->n = d->h = d->w = d->c_in = d->c_out = 1;
  d->kernel = 3;
  d->stride = 1;
  d->pad = -1;
  d->groups = 1;
  d->block = 1;
  d->norm_p = 2;
  d->support = SKIPCONV_SUPPORT_RF;
  d->dtype = SKIPCONV_F32;
  d->act_out = SKIPCONV_ACT_NONE;
  d->flags = 0;
  d->eps = 0.0f;
  d->gate = SKIPCONV_GATE_INPUT_NORM;
  return SKIPCONV_OK;
}

int skipconv_validate(const skipconv_desc* d) {
  Geometry g;
  return derive(d, &g, g_create_error);
}

int skipconv_out_shape(const skipconv_desc* d, int32_t* h_out, int32_t* w_out, int32_t* hb,
                       int32_t* wb) {
  Geometry g;
  const int rc = derive(d, &g, g_create_error);
  if (rc) return rc;
  if (h_out) *h_out = g.h_out;
  if (w_out) *w_out = g.w_out;
  if (hb) *hb = g.hb;
  if (wb) *wb = g.wb;
  return SKIPCONV_OK;
}

int skipconv_workspace_size(const skipconv_desc* d, size_t* bytes) {
  if (!bytes) return SKIPCONV_E_INVALID_ARG;
  Geometry g;
  const int rc = derive(d, &g, g_create_error);
  if (rc) return rc;
  *bytes = g.total;
  return SKIPCONV_OK;
}

int skipconv_create(const skipconv_desc* d, const void* weights, void* workspace,
                    size_t workspace_bytes, void* stream, skipconv_t* out) {
  if (!out) return fail(g_create_error, SKIPCONV_E_INVALID_ARG, "out is NULL");
  *out = nullptr;
  Geometry g;
  int rc = derive(d, &g, g_create_error);
  if (rc) return rc;
  if (!weights) return fail(g_create_error, SKIPCONV_E_INVALID_ARG, "weights is NULL");
  if (workspace && workspace_bytes < g.total)
    return fail(g_create_error, SKIPCONV_E_SMALL_BUFFER, "workspace smaller than skipconv_workspace_size");
  if (workspace && (reinterpret_cast<uintptr_t>(workspace) % kAlign))
    return fail(g_create_error, SKIPCONV_E_INVALID_ARG, "workspace must be 256-byte aligned");

  skipconv_layer* h = new (std::nothrow) skipconv_layer();
  if (!h) return fail(g_create_error, SKIPCONV_E_OOM, "host allocation failed");
  h->d = *d;
  h->d.pad = g.pad;
  h->g = g;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = hipGetDevice(&h->device);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&h->num_cu, hipDeviceAttributeMultiprocessorCount, h->device);
  if (e != hipSuccess) {
    snprintf(g_create_error, sizeof(g_create_error), "no HIP device: %s", hipGetErrorString(e));
    delete h;
    return SKIPCONV_E_HIP;
  }
  // The single-pass kernel serialises load, gate and product inside each
  // workgroup; it wins while the frame has few tiles (latency regime) and the
  // split pipeline wins on large frames, where each kernel streams at its own
  // roofline. Threshold: four tiles per CU.
  if (h->g.fused && (h->g.f_grid * ((h->g.f_rb || h->g.f_dw) ? h->g.f_nsplit : 1) > 4 * h->num_cu ||
                     sc::prepare_fused(fused_params(h, nullptr, true)) < 1))
    h->g.fused = false;
  // 16 x 16 tiles with the weights staged in LDS restage the whole weight
  // tensor per tile: they beat the split pipeline only for narrow layers on
  // few tiles (measured, 3 x 3 and 1 x 1, n = 1: 32 -> 32 up to ~3 tiles per
  // CU, 64 -> 64 up to one; 128 input or output channels lose at every size,
  // e.g. one 512 x 512 128 -> 128 frame 147 us against 78.5 us split).
  if (h->g.fused && !h->g.f_rb && !h->g.f_dw && !h->g.f_sc && h->g.f_mw == 4) {
    const long cap = (long)(d->c_in * d->c_out <= 32 * 32 ? 3 : 1) * h->num_cu;
    if (d->c_in > 64 || d->c_out > 64 || h->g.f_grid > cap) h->g.fused = false;
  }
  h->conv_occ = conv_setup(h->g, d, h->device);
  if (workspace) {
    h->ws = static_cast<char*>(workspace);
  } else {
    void* p = nullptr;
    e = hipMalloc(&p, g.total);
    if (e != hipSuccess) {
      snprintf(g_create_error, sizeof(g_create_error), "hipMalloc(%zu): %s", g.total, hipGetErrorString(e));
      delete h;
      return SKIPCONV_E_OOM;
    }
    h->ws = static_cast<char*>(p);
    h->owns_ws = true;
  }
  e = hipMemsetAsync(h->ctr(), 0, sc::kNumCounters * 4, st);
  if (e == hipSuccess) e = hipMemsetAsync(h->wctr(), 0, 2 * sc::kSegs * sc::kSegStride * 4, st);
  if (e == hipSuccess) e = hipMemsetAsync(h->bmask(), 0, g.off_list - g.off_bmask, st);
  if (e == hipSuccess) e = hipMemsetAsync(h->list(), 0, (size_t)g.nb * 4, st);
  if (e == hipSuccess && d->act_out != SKIPCONV_ACT_NONE)
    e = hipMemsetAsync(h->y(), 0, (size_t)d->n * g.h_out * g.w_out * d->c_out * g.elem, st);
  if (e == hipSuccess && h->emits()) e = hipMemsetAsync(h->r32(), 0, g.total - g.off_r32, st);
  // z starts at 0, so the activation output (0) is dtype(act(z)) from the start:
  // emitting kernels take the previous activation from the old z
  if (e == hipSuccess && h->emits()) e = hipMemsetAsync(h->z(), 0, g.z_bytes, st);
  if (e == hipSuccess) {
    if (g.depthwise)
      e = sc::launch_pack_depthwise(weights, static_cast<float*>(h->wpack()), d->dtype, d->c_in,
                                    d->kernel, st);
    else
      e = sc::launch_pack_mfma(weights, h->wpack(), d->dtype, d->c_out, d->c_in, d->kernel,
                               g.ksteps, g.ntn, st);
  }
  if (e == hipSuccess && g.fused)
    e = sc::launch_fused_tiles(reinterpret_cast<uint32_t*>(h->ws + g.off_ftiles), g.f_grid, g.f_tiles_y,
                               g.f_tiles_x, st);
  if (e == hipSuccess && d->gate == SKIPCONV_GATE_OUTPUT_NORM) e = weight_norm(h, weights, st);
  if (e != hipSuccess) {
    snprintf(g_create_error, sizeof(g_create_error), "create: %s", hipGetErrorString(e));
    if (h->owns_ws) (void)hipFree(h->ws);
    delete h;
    return SKIPCONV_E_HIP;
  }
  *out = h;
  return SKIPCONV_OK;
}

int skipconv_step(skipconv_t h, const void* x_t, void* stream, const float** z_t) {
  if (!h) return SKIPCONV_E_STATE;
  if (!x_t) return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "x_t is NULL");
  if (reinterpret_cast<uintptr_t>(x_t) % 16)
    return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "x_t must be 16-byte aligned");
  if (h->retains() && !h->ref_pending && x_t == h->last_x)
    return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "CALLER_RETAINS: x_t is the previous step's buffer");
  if (h->g.learned && !h->phi_set)
    return fail(h->last_error, SKIPCONV_E_STATE, "learned gate: call skipconv_set_gate_weights first");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const skipconv_desc& d = h->d;
  const Geometry& g = h->g;
  const bool ref = h->ref_pending;

  sc::GateParams gp = gate_params(h, x_t, ref);

  sc::ConvParams cp{};
  cp.x_t = x_t;
  cp.x_prev = h->prev_input(x_t);
  cp.wpack = h->wpack();
  cp.z = h->z();
  cp.y = h->y();
  cp.n = d.n; cp.h = d.h; cp.w = d.w; cp.c = d.c_in; cp.c_out = d.c_out;
  cp.h_out = g.h_out; cp.w_out = g.w_out; cp.k = d.kernel; cp.stride = d.stride; cp.pad = g.pad;
  cp.block = d.block; cp.hb = g.hb; cp.wb = g.wb;
  cp.ksteps = g.ksteps; cp.ntiles_n = g.ntn;
  cp.reference = ref ? 1 : 0;
  cp.no_prev = ref ? 1 : 0;
  cp.act = (h->emits() && !conv_emits(g)) ? 0 : d.act_out;
  cp.r32 = h->r32();
  cp.rb = h->rb();

  const bool timing = h->timing_done < h->timing_frames && h->timing_seen % h->timing_every == 0;
  if (h->timing_frames) ++h->timing_seen;
  if (timing) h->ev_step[h->timing_done] = h->timing_seen - 1;

  hipError_t e = hipSuccess;
  if (timing) e = hipEventRecord(h->ev[3 * h->timing_done], st);
  if (g.fused) {
    const sc::FusedParams fp = fused_params(h, x_t, ref);
    if (e == hipSuccess) e = sc::launch_fused(fp, g.f_grid * fp.nsplit, st);
    if (e != hipSuccess) return hip_fail(h, e, "fused launch");
    if (timing) e = hipEventRecord(h->ev[3 * h->timing_done + 1], st);
    h->list_valid = false;
    h->work_kind = 0;
  } else {
    StepList sl{};
    if (e == hipSuccess) e = begin_list(h, gp, st, &sl);
    if (e == hipSuccess) e = sc::launch_gate(gp, d.dtype, g.vec, g.gate_grid, g.gate_lds, st);
    if (e == hipSuccess) e = gate_done(h, st);
    if (e != hipSuccess) return hip_fail(h, e, "gate launch");
    if (timing) e = hipEventRecord(h->ev[3 * h->timing_done + 1], st);
    cp.list = sl.list;
    cp.counters = sl.counters;
    cp.zero_ctr = sl.zero;
    cp.seg_tiles = sl.seg_tiles;
    cp.seg_cap = sl.seg_cap;
    if (e == hipSuccess) e = launch_split_conv(g, d, cp, conv_grid(h), st);
    if (e != hipSuccess) return hip_fail(h, e, "conv launch");
    end_list(h);
  }
  if (h->emits() && !g.fused) {  // the fused kernel emits in its epilogue
    e = launch_emit(h, st);
    if (e != hipSuccess) return hip_fail(h, e, "emit launch");
  }
  if (timing) {
    e = hipEventRecord(h->ev[3 * h->timing_done + 2], st);
    if (e != hipSuccess) return hip_fail(h, e, "event record");
    ++h->timing_done;
  }
  h->advance_input(x_t);
  h->ref_pending = false;
  ++h->frames;
  if (z_t) *z_t = h->z();
  return SKIPCONV_OK;
}

int skipconv_step_translated(skipconv_t h, const void* x_t, int32_t dy, int32_t dx, void* stream,
                             const float** z_t) {
  if (!h) return SKIPCONV_E_STATE;
  if (!(h->d.flags & SKIPCONV_FLAG_TRANSLATE))
    return fail(h->last_error, SKIPCONV_E_STATE, "the layer was created without SKIPCONV_FLAG_TRANSLATE");
  const skipconv_desc& d = h->d;
  if (dy % d.stride || dx % d.stride)
    return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "the translation must be a multiple of the stride");
  if (dy <= -d.h || dy >= d.h || dx <= -d.w || dx >= d.w)
    return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "the translation must be smaller than the frame");
  if ((dy == 0 && dx == 0) || h->ref_pending) return skipconv_step(h, x_t, stream, z_t);
  if (!x_t) return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "x_t is NULL");
  if (reinterpret_cast<uintptr_t>(x_t) % 16)
    return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "x_t must be 16-byte aligned");
  if (h->retains() && !h->ref_pending && x_t == h->last_x)
    return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "CALLER_RETAINS: x_t is the previous step's buffer");
  if (h->g.learned && !h->phi_set)
    return fail(h->last_error, SKIPCONV_E_STATE, "learned gate: call skipconv_set_gate_weights first");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const Geometry& g = h->g;
  if (g.fused && g.f_rb) {
    // one pass of the register-operand kernel: x_{t-1} and z_{t-1} read
    // shifted, every site written to the other z slot, blocks holding an
    // exposed site recomputed from x_t
    sc::FusedParams fp = fused_params(h, x_t, false);
    fp.z = h->z_other();
    fp.zsrc = h->z();
    fp.g.sy = dy;
    fp.g.sx = dx;
    const hipError_t e = sc::launch_fused(fp, g.f_grid * fp.nsplit, st);
    if (e != hipSuccess) return hip_fail(h, e, "translated fused launch");
    h->zslot ^= 1;
    h->list_valid = false;
    h->work_kind = 0;
    h->advance_input(x_t);
    h->ref_pending = false;
    ++h->frames;
    if (z_t) *z_t = h->z();
    return SKIPCONV_OK;
  }
  // 1. z <- T~(z) into the other slot (activation output refreshed). The
  // block-halo convolution reads z_{t-1} from the old slot at the shifted site
  // itself, so there the shift runs after the gate and skips active blocks.
  const float* z_old = h->z();
  const bool zshift = g.halo && !g.depthwise;
  hipError_t e = hipSuccess;
  if (!zshift)
    e = sc::launch_translate_state(z_old, h->z_other(), h->y(), d.n, g.h_out, g.w_out, d.c_out, dy / d.stride,
                                   dx / d.stride, d.act_out, d.dtype, nullptr, d.block, g.hb, g.wb, st);
  if (e != hipSuccess) return hip_fail(h, e, "translate launch");
  h->zslot ^= 1;
  // 2. gate on r = x_t - T(x_{t-1}); exposed sites on
  sc::GateParams gp = gate_params(h, x_t, false);
  gp.sy = dy;
  gp.sx = dx;
  StepList sl{};
  e = begin_list(h, gp, st, &sl);
  if (e == hipSuccess) e = sc::launch_gate(gp, d.dtype, g.vec, g.gate_grid, g.gate_lds, st);
  if (e == hipSuccess) e = gate_done(h, st);
  if (e == hipSuccess && zshift)
    e = sc::launch_translate_state(z_old, h->z(), h->y(), d.n, g.h_out, g.w_out, d.c_out, dy / d.stride,
                                   dx / d.stride, d.act_out, d.dtype, h->bmask(), d.block, g.hb, g.wb, st);
  // 3. active blocks: translated recurrence (list a) or recomputed from x_t (list b)
  uint32_t* ctr = h->ctr();
  uint32_t* list_a = reinterpret_cast<uint32_t*>(h->ws + g.off_list_a);
  uint32_t* list_b = reinterpret_cast<uint32_t*>(h->ws + g.off_list_b);
  if (e == hipSuccess)
    e = sc::launch_split_list(sl.list, sl.counters, sl.seg_tiles, sl.seg_cap, list_a, ctr + 2, list_b, ctr + 3, g.hb,
                              g.wb, d.block, g.h_out,
                              g.w_out, d.h, d.w, d.kernel, d.stride, g.pad, dy, dx, st);
  if (e != hipSuccess) return hip_fail(h, e, "translated gate launch");
  sc::ConvParams cp{};
  cp.x_t = x_t;
  cp.x_prev = h->prev_input(x_t);
  cp.wpack = h->wpack();
  cp.z = h->z();
  cp.y = h->y();
  cp.n = d.n; cp.h = d.h; cp.w = d.w; cp.c = d.c_in; cp.c_out = d.c_out;
  cp.h_out = g.h_out; cp.w_out = g.w_out; cp.k = d.kernel; cp.stride = d.stride; cp.pad = g.pad;
  cp.block = d.block; cp.hb = g.hb; cp.wb = g.wb;
  cp.ksteps = g.ksteps; cp.ntiles_n = g.ntn;
  cp.act = d.act_out;
  for (int pass = 0; pass < 2 && e == hipSuccess; ++pass) {
    cp.list = pass ? list_b : list_a;
    cp.counters = ctr + 2 + pass;
    cp.zero_ctr = pass ? nullptr : sl.zero;
    cp.reference = pass;  // exposed blocks: assigned from x_t
    cp.no_prev = pass;
    cp.sy = pass ? 0 : dy;
    cp.sx = pass ? 0 : dx;
    cp.zsrc = (zshift && !pass) ? z_old : nullptr;
    cp.zdy = dy / d.stride;
    cp.zdx = dx / d.stride;
    e = launch_split_conv(g, d, cp, conv_grid(h), st);
  }
  if (e != hipSuccess) return hip_fail(h, e, "translated conv launch");
  end_list(h);
  h->advance_input(x_t);
  h->ref_pending = false;
  ++h->frames;
  if (z_t) *z_t = h->z();
  return SKIPCONV_OK;
}

int skipconv_step_chained(skipconv_t h, skipconv_t up, void* stream, const float** z_t) {
  if (!h) return SKIPCONV_E_STATE;
  if (!up || up == h) return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "upstream handle is NULL or the layer itself");
  if (!up->emits()) return fail(h->last_error, SKIPCONV_E_STATE, "the upstream layer does not emit its residual");
  if (up->d.n != h->d.n || up->g.h_out != h->d.h || up->g.w_out != h->d.w || up->d.c_out != h->d.c_in ||
      up->d.dtype != h->d.dtype)
    return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "upstream output does not match this layer's input");
  if (up->frames == 0) return fail(h->last_error, SKIPCONV_E_STATE, "the upstream layer has not stepped yet");
  if (h->g.learned && !h->phi_set)
    return fail(h->last_error, SKIPCONV_E_STATE, "learned gate: call skipconv_set_gate_weights first");
  // a reference frame reads the whole input: the upstream activation buffer
  if (h->ref_pending) return skipconv_step(h, up->y(), stream, z_t);

  hipStream_t st = static_cast<hipStream_t>(stream);
  const skipconv_desc& d = h->d;
  const Geometry& g = h->g;
  const bool bf16 = d.dtype == SKIPCONV_BF16;
  if (g.fused) {
    // one-pass kernel on the fp32 residual (it rounds the operand itself)
    sc::FusedParams fp = fused_params(h, up->r32(), false);
    fp.g.x_prev = nullptr;
    fp.g.x_keep = nullptr;
    fp.g.no_prev = 1;
    fp.g.rin = 1;
    if (!g.learned) {
      fp.g.up_mask = up->bmask();
      fp.g.up_block = up->d.block;
      fp.g.up_hb = up->g.hb;
      fp.g.up_wb = up->g.wb;
    }
    const hipError_t e = sc::launch_fused(fp, g.f_grid * fp.nsplit, st);
    if (e != hipSuccess) return hip_fail(h, e, "chained fused launch");
    h->list_valid = false;
    h->ref_pending = false;
    ++h->frames;
    if (z_t) *z_t = h->z();
    return SKIPCONV_OK;
  }
  // gate on the upstream residual (fp32); no x_{t-1} slot is read or written
  sc::GateParams gp = gate_params(h, up->r32(), false);
  gp.x_prev = nullptr;
  gp.x_keep = nullptr;
  gp.no_prev = 1;
  if (!g.learned) {  // a zero residual leaves a norm gate off: tiles without upstream blocks skip
    gp.up_mask = up->bmask();
    gp.up_block = up->d.block;
    gp.up_hb = up->g.hb;
    gp.up_wb = up->g.wb;
  }
  StepList sl{};
  hipError_t e = begin_list(h, gp, st, &sl);
  if (e == hipSuccess) e = sc::launch_gate(gp, SKIPCONV_F32, d.c_in % 8 == 0 ? 8 : 1, g.gate_grid, g.gate_lds, st);
  if (e == hipSuccess) e = gate_done(h, st);
  if (e != hipSuccess) return hip_fail(h, e, "chained gate launch");
  // convolution of the residual operand (bf16-rounded for bf16 layers), accumulated into z
  sc::ConvParams cp{};
  cp.x_t = bf16 ? (const void*)up->rb() : (const void*)up->r32();
  cp.x_prev = nullptr;
  cp.wpack = h->wpack();
  cp.z = h->z();
  cp.y = h->y();
  cp.list = sl.list;
  cp.counters = sl.counters;
  cp.zero_ctr = sl.zero;
  cp.seg_tiles = sl.seg_tiles;
  cp.seg_cap = sl.seg_cap;
  cp.n = d.n; cp.h = d.h; cp.w = d.w; cp.c = d.c_in; cp.c_out = d.c_out;
  cp.h_out = g.h_out; cp.w_out = g.w_out; cp.k = d.kernel; cp.stride = d.stride; cp.pad = g.pad;
  cp.block = d.block; cp.hb = g.hb; cp.wb = g.wb;
  cp.ksteps = g.ksteps; cp.ntiles_n = g.ntn;
  cp.reference = 0;
  cp.no_prev = 1;
  cp.act = (h->emits() && !conv_emits(g)) ? 0 : d.act_out;
  cp.r32 = h->r32();
  cp.rb = h->rb();
  e = launch_split_conv(g, d, cp, conv_grid(h), st);
  if (e != hipSuccess) return hip_fail(h, e, "chained conv launch");
  if (h->emits()) {
    e = launch_emit(h, st);
    if (e != hipSuccess) return hip_fail(h, e, "emit launch");
  }
  end_list(h);
  h->ref_pending = false;
  ++h->frames;
  if (z_t) *z_t = h->z();
  return SKIPCONV_OK;
}

int skipconv_reset(skipconv_t h) {
  if (!h) return SKIPCONV_E_STATE;
  h->ref_pending = true;
  h->last_x = nullptr;
  return SKIPCONV_OK;
}

int skipconv_set_eps(skipconv_t h, float eps) {
  if (!h) return SKIPCONV_E_STATE;
  if (std::isnan(eps) || eps < 0.0f) return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "eps must be >= 0");
  h->d.eps = eps;
  return SKIPCONV_OK;
}

int skipconv_set_gate_weights(skipconv_t h, const float* phi, float bias, void* stream) {
  if (!h) return SKIPCONV_E_STATE;
  if (!h->g.learned) return fail(h->last_error, SKIPCONV_E_STATE, "the layer's gate is not SKIPCONV_GATE_LEARNED");
  if (!phi) return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "phi is NULL");
  if (std::isnan(bias)) return fail(h->last_error, SKIPCONV_E_INVALID_ARG, "bias is NaN");
  const hipError_t e = sc::launch_pack_phi(phi, h->phi(), h->d.c_in, h->d.kernel, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(h, e, "set_gate_weights");
  h->gate_bias = bias;
  h->phi_set = true;
  return SKIPCONV_OK;
}

int skipconv_destroy(skipconv_t h) {
  if (!h) return SKIPCONV_OK;
  destroy_events(h);
  if (h->owns_ws) (void)hipFree(h->ws);
  delete h;
  return SKIPCONV_OK;
}

int skipconv_activation(skipconv_t h, const void** y) {
  if (!h) return SKIPCONV_E_STATE;
  if (!y) return SKIPCONV_E_INVALID_ARG;
  if (h->d.act_out == SKIPCONV_ACT_NONE) return fail(h->last_error, SKIPCONV_E_STATE, "no activation output");
  *y = h->y();
  return SKIPCONV_OK;
}

int skipconv_pipeline(skipconv_t h, int32_t* fused) {
  if (!h) return SKIPCONV_E_STATE;
  if (!fused) return SKIPCONV_E_INVALID_ARG;
  *fused = h->g.fused ? (h->g.f_sc ? 5 : (h->g.f_dw ? 4 : (h->g.f_rb ? (h->g.f_nsplit > 1 ? 3 : 2) : 1))) : 0;
  return SKIPCONV_OK;
}

int skipconv_gate_tile(skipconv_t h, int32_t* ts, int32_t* lane_sum) {
  if (!h) return SKIPCONV_E_STATE;
  if (!ts || !lane_sum) return SKIPCONV_E_INVALID_ARG;
  *ts = h->g.ts;
  *lane_sum = h->g.lane_sum;
  return SKIPCONV_OK;
}

int skipconv_conv_kernel(skipconv_t h, int32_t* kind) {
  if (!h) return SKIPCONV_E_STATE;
  if (!kind) return SKIPCONV_E_INVALID_ARG;
  *kind = h->g.depthwise ? (h->g.dw_halo ? 3 : 2) : (h->g.halo ? 1 : 0);
  return SKIPCONV_OK;
}

int skipconv_get_desc(skipconv_t h, skipconv_desc* d) {
  if (!h) return SKIPCONV_E_STATE;
  if (!d) return SKIPCONV_E_INVALID_ARG;
  *d = h->d;
  return SKIPCONV_OK;
}

static int copy_back(skipconv_t h, void* stream, void* host, const void* dev, size_t bytes) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(host, dev, bytes, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(h, e, "copy to host");
  return SKIPCONV_OK;
}

// The fused pipeline does not build the ordered list; build it on demand.
static int ensure_list(skipconv_t h, void* stream) {
  if (h->list_valid) return SKIPCONV_OK;
  const hipError_t e = sc::launch_compact(h->bmask(), h->g.nb, h->list(), h->ctr(), nullptr, 0, 0, 0, 0, 0, 0,
                                          static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(h, e, "compaction launch");
  h->list_valid = true;
  return SKIPCONV_OK;
}

int skipconv_active_count(skipconv_t h, void* stream, int64_t* blocks, int64_t* sites) {
  if (!h) return SKIPCONV_E_STATE;
  if (h->frames == 0) return fail(h->last_error, SKIPCONV_E_STATE, "no step yet");
  int rc0 = ensure_list(h, stream);
  if (rc0) return rc0;
  uint32_t cnt = 0;
  int rc = copy_back(h, stream, &cnt, h->ctr() + sc::kCtrCount, 4);
  if (rc) return rc;
  if (blocks) *blocks = cnt;
  if (sites) {
    std::vector<uint8_t> m(h->g.nb);
    rc = copy_back(h, stream, m.data(), h->bmask(), m.size());
    if (rc) return rc;
    const int b = h->d.block;
    int64_t tot = 0;
    for (int i = 0; i < h->g.nb; ++i) {
      if (!m[i]) continue;
      const int rem = i % (h->g.hb * h->g.wb);
      const int bi = rem / h->g.wb, bj = rem % h->g.wb;
      const int ny = std::min(b, h->g.h_out - bi * b), nx = std::min(b, h->g.w_out - bj * b);
      tot += (int64_t)ny * nx;
    }
    *sites = tot;
  }
  return SKIPCONV_OK;
}

int skipconv_copy_block_mask(skipconv_t h, void* stream, uint8_t* host, size_t bytes) {
  if (!h) return SKIPCONV_E_STATE;
  if (!host) return SKIPCONV_E_INVALID_ARG;
  if (bytes < (size_t)h->g.nb) return fail(h->last_error, SKIPCONV_E_SMALL_BUFFER, "block mask buffer too small");
  return copy_back(h, stream, host, h->bmask(), h->g.nb);
}

int skipconv_copy_active_list(skipconv_t h, void* stream, uint32_t* host, size_t capacity,
                              int64_t* count) {
  if (!h) return SKIPCONV_E_STATE;
  if (!host || !count) return SKIPCONV_E_INVALID_ARG;
  int rc = ensure_list(h, stream);
  if (rc) return rc;
  uint32_t cnt = 0;
  rc = copy_back(h, stream, &cnt, h->ctr() + sc::kCtrCount, 4);
  if (rc) return rc;
  *count = cnt;
  if (capacity < cnt) return fail(h->last_error, SKIPCONV_E_SMALL_BUFFER, "list buffer too small");
  if (cnt == 0) return SKIPCONV_OK;
  return copy_back(h, stream, host, h->list(), (size_t)cnt * 4);
}

int skipconv_copy_work_list(skipconv_t h, void* stream, uint32_t* host, size_t capacity, int64_t* count) {
  if (!h) return SKIPCONV_E_STATE;
  if (!host || !count) return SKIPCONV_E_INVALID_ARG;
  if (h->frames == 0) return fail(h->last_error, SKIPCONV_E_STATE, "no step yet");
  if (h->work_kind == 0)
    return fail(h->last_error, SKIPCONV_E_UNSUPPORTED, "one-pass kernel: no work list (its block flags are the block mask)");
  if (h->work_kind == 1) {  // the ordered list the compaction wrote for the convolution
    uint32_t cnt = 0;
    int rc = copy_back(h, stream, &cnt, h->ctr() + sc::kCtrCount, 4);
    if (rc) return rc;
    *count = cnt;
    if (capacity < cnt) return fail(h->last_error, SKIPCONV_E_SMALL_BUFFER, "list buffer too small");
    return cnt ? copy_back(h, stream, host, h->list(), (size_t)cnt * 4) : SKIPCONV_OK;
  }
  // segment x of the work list starts at entry (first gate tile of x) * seg_cap
  constexpr int kSlot = sc::kSegs * sc::kSegStride;
  std::vector<uint32_t> ctr(kSlot);
  int rc = copy_back(h, stream, ctr.data(), h->wctr() + h->work_slot * kSlot, kSlot * 4);
  if (rc) return rc;
  const int per = h->g.gate_grid / sc::kSegs, rem = h->g.gate_grid % sc::kSegs;
  int64_t tot = 0;
  for (int x = 0; x < sc::kSegs; ++x) tot += ctr[x * sc::kSegStride];
  *count = tot;
  if ((int64_t)capacity < tot) return fail(h->last_error, SKIPCONV_E_SMALL_BUFFER, "list buffer too small");
  size_t at = 0;
  for (int x = 0; x < sc::kSegs; ++x) {
    const uint32_t n = ctr[x * sc::kSegStride];
    const size_t base = (size_t)(x * per + std::min(x, rem)) * h->g.seg_cap;
    if (n > (size_t)(x < sc::kSegs - 1 ? (x + 1) * per + std::min(x + 1, rem) : h->g.gate_grid) * h->g.seg_cap - base)
      return fail(h->last_error, SKIPCONV_E_HIP, "work list segment overflows its range");
    if (n) {
      rc = copy_back(h, stream, host + at, h->wlist() + base, (size_t)n * 4);
      if (rc) return rc;
    }
    at += n;
  }
  return SKIPCONV_OK;
}

int skipconv_copy_site_mask(skipconv_t h, void* stream, uint8_t* host, size_t bytes) {
  if (!h) return SKIPCONV_E_STATE;
  if (!(h->d.flags & SKIPCONV_FLAG_KEEP_STATS)) return fail(h->last_error, SKIPCONV_E_STATE, "KEEP_STATS not set");
  const size_t need = (size_t)h->d.n * h->g.h_out * h->g.w_out;
  if (!host) return SKIPCONV_E_INVALID_ARG;
  if (bytes < need) return fail(h->last_error, SKIPCONV_E_SMALL_BUFFER, "site mask buffer too small");
  return copy_back(h, stream, host, h->smask(), need);
}

int skipconv_copy_stat(skipconv_t h, void* stream, float* host, size_t bytes) {
  if (!h) return SKIPCONV_E_STATE;
  if (!(h->d.flags & SKIPCONV_FLAG_KEEP_STATS)) return fail(h->last_error, SKIPCONV_E_STATE, "KEEP_STATS not set");
  const size_t need = (size_t)h->d.n * h->g.h_out * h->g.w_out * 4;
  if (!host) return SKIPCONV_E_INVALID_ARG;
  if (bytes < need) return fail(h->last_error, SKIPCONV_E_SMALL_BUFFER, "stat buffer too small");
  return copy_back(h, stream, host, h->stat(), need);
}

int skipconv_frame_macs(skipconv_t h, void* stream, uint64_t* dense, uint64_t* active) {
  if (!h) return SKIPCONV_E_STATE;
  const uint64_t per_site = (uint64_t)h->d.c_out * (h->d.c_in / h->d.groups) * h->d.kernel * h->d.kernel;
  const uint64_t sites = (uint64_t)h->d.n * h->g.h_out * h->g.w_out;
  if (dense) *dense = sites * per_site;
  if (active) {
    int64_t s = 0;
    const int rc = skipconv_active_count(h, stream, nullptr, &s);
    if (rc) return rc;
    *active = (uint64_t)s * per_site;
  }
  return SKIPCONV_OK;
}

const char* skipconv_status_string(int status) {
  switch (status) {
    case SKIPCONV_OK: return "ok";
    case SKIPCONV_E_INVALID_ARG: return "invalid argument";
    case SKIPCONV_E_UNSUPPORTED: return "unsupported";
    case SKIPCONV_E_OOM: return "out of device memory";
    case SKIPCONV_E_HIP: return "HIP error";
    case SKIPCONV_E_STATE: return "invalid state";
    case SKIPCONV_E_SMALL_BUFFER: return "buffer too small";
    default: return "unknown status";
  }
}

const char* skipconv_last_error(skipconv_t h) { return h ? h->last_error : g_create_error; }

int skipconv_timing_begin(skipconv_t h, int frames, int every) {
  if (!h) return SKIPCONV_E_STATE;
  if (frames < 0 || frames > (1 << 20) || every < 1) return SKIPCONV_E_INVALID_ARG;
  destroy_events(h);
  h->ev.resize((size_t)frames * 3, nullptr);
  h->ev_step.assign((size_t)frames, -1);
  for (auto& e : h->ev) {
    const hipError_t r = hipEventCreate(&e);
    if (r != hipSuccess) {
      destroy_events(h);
      return hip_fail(h, r, "hipEventCreate");
    }
  }
  h->timing_frames = frames;
  h->timing_every = every;
  return SKIPCONV_OK;
}

int skipconv_timing_read(skipconv_t h, void* stream, double* ms, int* frames_timed,
                         int32_t* step_index, int capacity) {
  if (!h) return SKIPCONV_E_STATE;
  if (!ms) return SKIPCONV_E_INVALID_ARG;
  if (step_index && capacity < h->timing_done)
    return fail(h->last_error, SKIPCONV_E_SMALL_BUFFER, "step_index buffer too small");
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(h, e, "sync");
  ms[0] = ms[1] = 0.0;
  for (int i = 0; i < h->timing_done; ++i) {
    float a = 0.f, b = 0.f;
    e = hipEventElapsedTime(&a, h->ev[3 * i], h->ev[3 * i + 1]);
    if (e == hipSuccess) e = hipEventElapsedTime(&b, h->ev[3 * i + 1], h->ev[3 * i + 2]);
    if (e != hipSuccess) return hip_fail(h, e, "hipEventElapsedTime");
    ms[0] += a;
    ms[1] += b;
    if (step_index) step_index[i] = h->ev_step[i];
  }
  if (frames_timed) *frames_timed = h->timing_done;
  return SKIPCONV_OK;
}

int skipconv_step_static(const skipconv_desc* d, const void* weights, const void* x_t, const void* x_prev,
                         float* z, void* stream) {
  if (!d || !weights || !x_t || !z) return fail(g_create_error, SKIPCONV_E_INVALID_ARG, "NULL argument");
  if (reinterpret_cast<uintptr_t>(x_t) % 16 || reinterpret_cast<uintptr_t>(x_prev) % 16 ||
      reinterpret_cast<uintptr_t>(z) % 16)
    return fail(g_create_error, SKIPCONV_E_INVALID_ARG, "x_t, x_prev and z must be 16-byte aligned");
  if (x_prev == x_t) return fail(g_create_error, SKIPCONV_E_INVALID_ARG, "x_prev is x_t");
  if (d->flags & ~(uint32_t)SKIPCONV_FLAG_FORCE_DENSE)
    return fail(g_create_error, SKIPCONV_E_UNSUPPORTED, "skipconv_step_static takes no flags but FORCE_DENSE");
  if (d->gate != SKIPCONV_GATE_INPUT_NORM)
    return fail(g_create_error, SKIPCONV_E_UNSUPPORTED, "skipconv_step_static takes the Input-Norm gate only");
  if (d->act_out != SKIPCONV_ACT_NONE)
    return fail(g_create_error, SKIPCONV_E_UNSUPPORTED, "skipconv_step_static has no activation output");
  skipconv_desc dd = *d;
  dd.flags |= SKIPCONV_FLAG_SPLIT_PIPELINE | SKIPCONV_FLAG_CALLER_RETAINS;
  Geometry g;
  int rc = derive(&dd, &g, g_create_error);
  if (rc) return rc;
  if (g.split_blocks)
    return fail(g_create_error, SKIPCONV_E_UNSUPPORTED, "skipconv_step_static: blocks larger than the gate tile");
  // scratch layout: work-list counters, packed weights, block flags, work list
  const size_t off_wpack = align_up((size_t)sc::kSegs * sc::kSegStride * 4);
  const size_t off_bmask = align_up(off_wpack + g.wpack_bytes);
  const size_t off_wlist = align_up(off_bmask + (size_t)g.nb + 16);
  const size_t need = off_wlist + (size_t)std::max<long>(g.nb, (long)g.gate_grid * g.seg_cap) * 4;
  if (need > kStaticScratchBytes) {
    snprintf(g_create_error, sizeof(g_create_error),
             "skipconv_step_static: the layer needs %zu bytes of scratch, the static scratch holds %zu", need,
             kStaticScratchBytes);
    return SKIPCONV_E_SMALL_BUFFER;
  }
  void* base = nullptr;
  int dev = 0, num_cu = 0;
  rc = static_scratch(&base, &dev, &num_cu);
  if (rc) return rc;
  const int occ = conv_setup(g, &dd, dev);
  char* sb = static_cast<char*>(base);
  uint32_t* ctr = reinterpret_cast<uint32_t*>(sb);
  void* wpack = sb + off_wpack;
  uint8_t* bmask = reinterpret_cast<uint8_t*>(sb + off_bmask);
  uint32_t* wlist = reinterpret_cast<uint32_t*>(sb + off_wlist);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool ref = x_prev == nullptr;

  // the previous call's counters are not zero: clear them with a kernel
  hipError_t e = sc::launch_fill_u32(ctr, sc::kSegs * sc::kSegStride, 0u, st);
  if (e == hipSuccess)
    e = g.depthwise ? sc::launch_pack_depthwise(weights, static_cast<float*>(wpack), dd.dtype, dd.c_in, dd.kernel, st)
                    : sc::launch_pack_mfma(weights, wpack, dd.dtype, dd.c_out, dd.c_in, dd.kernel, g.ksteps, g.ntn, st);
  sc::GateParams gp = gate_geometry(dd, g, ref);
  gp.x_t = x_t;
  gp.x_prev = ref ? x_t : x_prev;
  gp.x_keep = nullptr;
  gp.block_mask = bmask;
  gp.counters = ctr;
  gp.wlist = wlist;
  gp.wctr = ctr;
  gp.seg_cap = g.seg_cap;
  if (e == hipSuccess) e = sc::launch_gate(gp, dd.dtype, g.vec, g.gate_grid, g.gate_lds, st);
  sc::ConvParams cp = conv_geometry(dd, g, ref);
  cp.x_t = x_t;
  cp.x_prev = ref ? x_t : x_prev;
  cp.wpack = wpack;
  cp.z = z;
  cp.list = wlist;
  cp.counters = ctr;
  cp.seg_tiles = g.gate_grid;
  cp.seg_cap = g.seg_cap;
  if (e == hipSuccess) e = launch_split_conv(g, dd, cp, conv_grid_of(g, num_cu, occ), st);
  if (e != hipSuccess) {
    snprintf(g_create_error, sizeof(g_create_error), "skipconv_step_static: %s", hipGetErrorString(e));
    return SKIPCONV_E_HIP;
  }
  return SKIPCONV_OK;
}

}  // extern "C"
