// Kernel parameter blocks and launchers of the Skip-Conv layer (host + device).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sc {

// counters[] slots in the workspace
constexpr int kCtrCount = 0;  // active blocks of the last gate pass
constexpr int kCtrSpare = 1;
constexpr int kNumCounters = 16;
// The gate appends active blocks to kSegs work-list segments, one per XCD's
// contiguous range of gate tiles, each with its own counter kSegStride
// uint32 apart (one 128-byte line each): appends to one counter serialise,
// so spreading them over eight lines removes most of that wait.
constexpr int kSegs = 8;
constexpr int kSegStride = 32;

constexpr int kConvF32Rows = 16;     // output sites per tile of the fp32 convolution
constexpr int kMaxTileBlocks = 256;  // blocks per gate tile: (ts / b)^2 <= 256

// Gate: residual, support statistic, threshold, block pooling, compaction.
struct GateParams {
  const void* x_t;      // N x H x W x C, layer dtype
  const void* x_prev;   // x_{t-1} slot being read (unused on reference frames)
  void* x_keep;         // spare slot receiving x_t
  int n, h, w, c;
  int h_out, w_out, k, stride, pad, block, hb, wb;
  int ts, tiles_y, tiles_x;     // tile side (sites) and tile grid per image
  int halo_floats;              // LDS floats reserved for the a[] halo
  int stage_stride;             // LDS floats of chunk sums per halo pixel (>= ceil(c/8), odd)
  int lane_sum;                 // 1: chunk sums combined in lane groups, no staging (c / 8 in {4, 8, 16})
  int rows_per_batch;           // unused (whole halo staged at once)
  int copy_in_halo;             // 1: every owned input pixel lies in its tile's halo
  int norm_p, support, reference, force_dense, keep_stats;
  int no_prev;                  // x_{t-1} taken as 0 (reference frames; residual inputs)
  double thr;                   // eps^2 (p = 2) or eps (p = 1), exact in fp64
  double wnorm;                 // statistic factor: 1 (Input-Norm gate) or the weight norm (Output-Norm)
  uint8_t* block_mask;          // N x HB x WB
  uint8_t* tile_flags;          // N x tiles_y x tiles_x when blocks are larger than tiles
  int split_blocks;             // 1: ts < block (b % ts == 0): flags per tile, OR-ed by the compaction
  uint32_t* list;               // N x HB x WB (first count entries valid)
  uint32_t* counters;
  float* stat;                  // N x H_out x W_out (keep_stats)
  uint8_t* site_mask;           // N x H_out x W_out (keep_stats)
  // learned gate (Eq. 8 at inference): phi [tap][c] fp32, bias; 0 = norm gates
  int learned;
  const float* phi;
  float gate_bias;
  int phi_off;                  // LDS float offset of the staged phi, or -1: read phi from memory
  int tr_off;                   // learned gate over lane groups: LDS float offset of the per-wave tap-term exchange
  // chained input (x_t is the upstream layer's residual): tiles whose input
  // region holds no upstream active block skip their loads; NULL = no skip
  const uint8_t* up_mask;
  int up_block, up_hb, up_wb;
  int rin;                      // fused kernel: x_t is an fp32 residual (no x_{t-1})
  int sy, sx;                   // translation of the content since x_{t-1} (split gate only)
  // unordered work list of the convolution (blocks appended per tile), its
  // count (zero on entry); NULL when the ordered compaction builds the list
  uint32_t* wlist;
  uint32_t* wctr;               // kSegs counters, kSegStride apart
  int seg_cap;                  // work-list entries reserved per gate tile
};

// Sparse convolution over the active sites (dense groups = 1).
struct ConvParams {
  const void* x_t;
  const void* x_prev;
  const void* wpack;            // packed MFMA B fragments
  float* z;                     // N x H_out x W_out x C_out fp32
  void* y;                      // optional activation output (layer dtype)
  const uint32_t* list;
  const uint32_t* counters;
  int n, h, w, c, c_out;
  int h_out, w_out, k, stride, pad, block, hb, wb;
  int ksteps;                   // K padded to the MFMA k-step, in steps
  int ntiles_n;                 // ceil(C_out / 16)
  int reference;                // assign z instead of accumulating
  int no_prev;                  // x_{t-1} taken as 0 (reference frames; residual inputs)
  int act;                      // 0 none, 1 identity, 2 relu
  int sy, sx;                   // translation of the content since x_{t-1} (input pixels; 0 = none)
  uint32_t* zero_ctr;           // work-list counters (kSegs, kSegStride apart) to clear for the next step, or NULL
  int seg_tiles, seg_cap;       // segmented work list: gate tiles and entries per tile; 0: plain list
  // residual emission in the block-halo kernel's epilogue (HaloParams::emit):
  // r = fl32(y_new - y_old) and its bf16 rounding at every site it updates
  float* r32;
  uint16_t* rb;
  // translated steps (block-halo convolution): z_{t-1} is read from zsrc at
  // the output site shifted back by (zdy, zdx), zero outside the frame, and
  // the sum written to z; NULL = read z itself
  const float* zsrc;
  int zdy, zdx;
};

// Work list of a convolution: a plain list with its count at
// counters[kCtrCount], or the gate's kSegs segments, segment x holding the
// blocks of gate tiles first(x) .. first(x + 1) - 1 (the XCD-contiguous tile
// ranges of the gate launch) from entry first(x) * seg_cap on, its count at
// counters[x * kSegStride]. Entries are the linear block indices.
constexpr int kGateThreads = 256;  // threads of a gate workgroup
// learned gate over lane groups: taps whose chunk terms are exchanged at once
constexpr int kLearnTapGroup = 9;

struct WorkList {
  uint32_t total;
  uint32_t pre[kSegs + 1];  // segmented: entries before segment x
  uint32_t base[kSegs];     // segmented: first list entry of segment x
  bool seg;
};

template <typename C>
__device__ __forceinline__ WorkList work_list(const C* counters, int seg_tiles, int seg_cap) {
  WorkList W;
  W.seg = seg_tiles > 0;
  if (!W.seg) {
    W.total = counters[kCtrCount];
    return W;
  }
  const int per = seg_tiles >> 3, rem = seg_tiles & 7;
  uint32_t run = 0;
#pragma unroll
  for (int x = 0; x < kSegs; ++x) {
    W.pre[x] = run;
    W.base[x] = (uint32_t)((x * per + (x < rem ? x : rem)) * seg_cap);
    run += counters[x * kSegStride];
  }
  W.pre[kSegs] = run;
  W.total = run;
  return W;
}

// List position of work item j (j < W.total).
__device__ __forceinline__ uint32_t work_pos(const WorkList& W, uint32_t j) {
  if (!W.seg) return j;
  uint32_t pos = 0;
#pragma unroll
  for (int x = 0; x < kSegs; ++x)
    if (j >= W.pre[x] && j < W.pre[x + 1]) pos = W.base[x] + (j - W.pre[x]);
  return pos;
}

// Element offset of x_{t-1} under the step's translation at input pixel
// (n, y, x), channel ch: the translated previous frame holds x_{t-1}[y - sy,
// x - sx], and zero where that lies outside the frame (returned as -1).
template <typename P>
__device__ __forceinline__ long prev_off(const P& p, int n, int y, int x, int ch) {
  const int yp = y - p.sy, xq = x - p.sx;
  if (yp < 0 || yp >= p.h || xq < 0 || xq >= p.w) return -1;
  return ((long)(n * p.h + yp) * p.w + xq) * p.c + ch;
}

// Output line i (row or column) is "exposed" under a translation d of the
// input (a multiple of the stride s) when its source line i - d/s is outside
// the output grid, or when a tap p = i*s - pad + kh leaves the frame while
// p - d lies inside it: convolution and translation do not commute there.
__device__ __forceinline__ bool line_exposed(int i, int n_out, int n_in, int k, int s, int pad, int d) {
  if (d == 0) return false;
  const int src = i - d / s;
  if (src < 0 || src >= n_out) return true;
  for (int kh = 0; kh < k; ++kh) {
    const int q = i * s - pad + kh;
    if (q - d >= 0 && q - d < n_in && (q < 0 || q >= n_in)) return true;
  }
  return false;
}

// Block-halo variant of the dense bf16 convolution (see sc_conv.hip).
struct HaloParams {
  int config;            // wave layout / tile shape instantiation
  int tr;                // output rows per tile (tile = tr x block sites)
  int tiles_per_block;   // block / tr
  int hh, hw;            // halo rows and columns: (tr-1)*s+k, (block-1)*s+k
  int pstride;           // LDS bytes per halo pixel: 2*c_in + 16
  int lds_bytes;         // hh * hw * pstride
  int threads;           // workgroup size
  int emit;              // the epilogue also writes the successor's residual (bf16, C_out % 8 == 0)
};

// Fused single-pass step for dense bf16 layers (see sc_fused.hip). `g` carries
// the gate geometry of the fused tiling (ts, tiles, staging rows).
struct FusedParams {
  GateParams g;
  const void* wpack;
  float* z;
  void* y;
  int c_out, ntiles_n, ksteps, csteps, act;
  int kc, nchunks, nbuf;   // weight chunks: k-steps per chunk, chunk count, LDS buffers
  int mw;                  // 16-row MFMA tiles per wave (1 for 8x8 tiles, 4 for 16x16)
  int pstride;             // LDS bytes per rho halo pixel: 2*c_in + 16
  int zero_pix;            // index of the all-zero pixel just past the halo
  int pstage;              // LDS floats per halo pixel of chunk sums: (c_in / 8) | 1
  int off_b, off_halo, off_a, off_part, lds_bytes;  // off_b: weights, or partial sums (rb)
  int rbk;                 // register-operand kernel: its build (fused_rb_kps), 0: LDS operand
  int nsplit;              // register-operand kernel: workgroups per tile, each owning
                           // ntiles_n / nsplit 16-column output tiles (1: no split)
  const uint32_t* tiles;   // per workgroup: its tile, tx | ty << 10 | n << 20 (XCD-aware order)
  float inv_ts, inv_blk, inv_hw, inv_chk;  // 1/ts, 1/block, 1/halo width, 1/(c_in / 8), rounded to fp32
  // residual emission for a chained successor (act must be set): r = y_new - y_old
  int emit;
  float* r32;
  uint16_t* rb;
  uint8_t* prev_mask;      // blocks updated by the previous step
  int dw;                  // depthwise kernel: its halo rows per thread (fused_dw_ki), 0: dense
  int sc;                  // few-channel kernel: 1 fp32 by elements, 4 fp32 by 4, 2 bf16; 0: none
  // translated step (Sec. 3.3): z_{t-1} in the other slot, read at the site
  // shifted back by (g.sy, g.sx) / stride (zero outside the grid); z is then
  // written at every site. Null on other steps.
  const float* zsrc;
  int trans_ok;            // the layer may take translated steps (create: prepare that mode)
};

// Learned gate in the register-operand fused kernel: phi (k^2 * C_in fp32)
// takes at most this many float4 loads per thread (512 threads).
constexpr int kFusedPhiLoads = 2;

// Few-channel fused kernel (fp32 C_in <= 16, bf16 C_in < 8): halo loads in
// flight per thread per round, and k-steps per wave at most (two k-parts).
constexpr int kScItems = 2;
constexpr int kScStepsF32 = 24;
constexpr int kScStepsBf16 = 6;

// Depthwise fused kernel: channels per workgroup (the split) at most
// kDwSplitMax, so 64 sites x kDwSplitMax / 4 pieces take kDwPieces per thread
// of 512; its weights, k*k*split/4 float4, take kDwWeightLoads loads per thread.
constexpr int kDwSplitMax = 64;
constexpr int kDwPieces = 2;
constexpr int kDwWeightLoads = 2;

hipError_t launch_fused(const FusedParams& p, int grid, hipStream_t st);
int prepare_fused(const FusedParams& p);  // create time: LDS attribute; workgroups per CU (0 on error)
// Tile table of the fused kernel: entry b = the tile workgroup b runs, packed
// tx | ty << 10 | n << 20, in the XCD-aware order (tiles_x, tiles_y <= 1024).
hipError_t launch_fused_tiles(uint32_t* table, int grid, int tiles_y, int tiles_x, hipStream_t st);
// Build of the register-operand fused kernel for this shape (ntiles_n
// 16-column tiles, ksteps k-steps, a square halo of halo_w pixels a side,
// chunks = c_in / 8): its index + 1, or 0 if none covers it; and the number of
// k-parts whose partial sums that build keeps in LDS.
int fused_rb_kps(int ntiles_n, int ksteps, int halo_w, int chunks);
int fused_rb_kparts(int rb);
// Depthwise fused kernel: halo rows per thread of the build covering a square
// halo of halo_w pixels a side with `chunks` 8-channel chunks a pixel (4 or 6),
// or 0 if none does.
int fused_dw_ki(int halo_w, int chunks);

hipError_t launch_gate(const GateParams& p, int dtype, int vec, int grid, size_t lds_bytes,
                       hipStream_t st);
hipError_t launch_pack_phi(const float* src, float* dst, int c, int k, hipStream_t st);
// Ordered compaction of the block flags into the active list and its count.
// When tile_flags is non-NULL, block flags are first formed as the OR of the
// (block / ts)^2 tile flags of each block (tiles_y x tiles_x tiles per image).
hipError_t launch_compact(uint8_t* block_mask, int nb, uint32_t* list, uint32_t* counters,
                          const uint8_t* tile_flags, int n, int hb, int wb, int bt, int tiles_y,
                          int tiles_x, hipStream_t st);
hipError_t launch_conv(const ConvParams& p, int dtype, bool fast, int grid, hipStream_t st);
hipError_t launch_conv_halo(const ConvParams& p, const HaloParams& hp, int grid, hipStream_t st);
int conv_halo_occupancy(const HaloParams& hp);  // resident workgroups per CU (0 on error)
hipError_t launch_depthwise(const ConvParams& p, int dtype, int grid, hipStream_t st);
// Depthwise over active blocks with the residual halo in LDS (bf16, C % 8 == 0):
// hp.tr rows x block columns per tile, hp.lds_bytes of halo (+ the [tap][c]
// fp32 weights, added by the launch).
hipError_t launch_depthwise_halo(const ConvParams& p, const HaloParams& hp, int grid, hipStream_t st);
int depthwise_halo_occupancy(const HaloParams& hp, int k, int c);  // resident workgroups per CU

// Residual emission of a layer that feeds a chained layer: at the blocks the
// step updated, y = dtype(act(z)) and r = y_new - y_old (fp32, and its bf16
// rounding for bf16 layers); at blocks updated by the previous step only, r = 0.
hipError_t launch_emit(const uint8_t* block_mask, uint8_t* prev_mask, int nb, const float* z, void* y,
                       float* r32, uint16_t* rb, int n, int hb, int wb, int block, int h_out, int w_out,
                       int c_out, int act, int dtype, int clear_only, hipStream_t st);

// Translation-compensated steps (Sec. 3.3): the translated state, and the
// active list split into translated-recurrence blocks and exposed blocks.
hipError_t launch_translate_state(const float* z_src, float* z_dst, void* y, int n, int h_out, int w_out,
                                  int c_out, int dyo, int dxo, int act, int dtype, const uint8_t* skip_mask,
                                  int block, int hb, int wb, hipStream_t st);
hipError_t launch_split_list(const uint32_t* list, const uint32_t* counters, int seg_tiles, int seg_cap,
                             uint32_t* list_a, uint32_t* counters_a, uint32_t* list_b, uint32_t* counters_b,
                             int hb, int wb, int block, int h_out, int w_out, int h, int w, int k, int stride,
                             int pad, int sy, int sx, hipStream_t st);

hipError_t launch_fill_u32(uint32_t* p, int n, uint32_t v, hipStream_t st);

// One-time weight repacks (create time).
hipError_t launch_pack_mfma(const void* w, void* out, int dtype, int c_out, int c_in, int k,
                            int ksteps, int ntiles_n, hipStream_t st);
hipError_t launch_pack_depthwise(const void* w, float* out, int dtype, int c, int k,
                                 hipStream_t st);

}  // namespace sc
