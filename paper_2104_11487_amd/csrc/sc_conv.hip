// Sparse convolution of the Skip-Conv layer over the active sites (Eq. 3):
//   z[o] += sum_{kh,kw,ci} w[co, ci, kh, kw] * rho[o*s - pad + (kh, kw), ci]
// for every output site o inside an active block; untouched sites keep
// z_{t-1}. rho is the residual x_t - x_{t-1} in fp32 (fp32 layers) or rounded
// to bf16 (bf16 layers); on a reference frame x_{t-1} = 0 and z is assigned.
//
// The work is the im2col matrix product restricted to the active columns
// (Sec. 4.2): rows = active sites, K = (kh, kw, ci), N = C_out. Rows are
// enumerated block by block from the ordered active list (row g belongs to
// list entry g / b^2, site g % b^2 of that block in row-major order), in
// tiles of 64 rows; a persistent grid walks the tiles, reading the active
// count from device memory, with each XCD taking one contiguous range of
// tiles so that neighbouring sites (shared halo pixels) stay in one L2.
//
// Dense layers: each wave owns 16 rows and all output channels. For every
// k-step a lane gathers its A fragment straight from the two frames
// (x_t - x_{t-1}, rounded to bf16), and reads its B fragments from the
// weights repacked at create time into the MFMA operand layout; products
// accumulate in fp32 (v_mfma_f32_16x16x32_bf16, or v_mfma_f32_16x16x4_f32 for
// fp32 layers). The epilogue adds the tile into z (each site belongs to
// exactly one row, so there are no atomics) and refreshes the activation
// output at the same sites.
//
// Depthwise layers (groups = C): no contraction to speak of, so no MFMA; one
// thread per (site, 8 channels) sums the k x k taps with fp32 FMAs.
#include "sc_device.h"
#include "sc_halo_conv.h"
#include "sc_kernels.h"
#include "sc_stream.h"

namespace sc {

namespace {

constexpr int kConvThreads = 256;
constexpr int kRowsPerTile = 64;


struct Site {
  int n, oy, ox;
  bool ok;
};

__device__ __forceinline__ Site site_of_row(const ConvParams& p, const WorkList& W, long g, long total_rows,
                                            int bb) {
  Site st{0, 0, 0, false};
  if (g < total_rows) {
    const int j = (int)(g / bb);
    const int within = (int)(g - (long)j * bb);
    const uint32_t blk = p.list[work_pos(W, (uint32_t)j)];
    const int per_img = p.hb * p.wb;
    st.n = (int)(blk / per_img);
    const int rem = (int)(blk - (uint32_t)st.n * per_img);
    const int bi = rem / p.wb, bj = rem - bi * p.wb;
    const int wy = within / p.block;
    st.oy = bi * p.block + wy;
    st.ox = bj * p.block + (within - wy * p.block);
    st.ok = st.oy < p.h_out && st.ox < p.w_out;
  }
  return st;
}

// Tile walk of a persistent grid: XCD x = blockIdx % 8 takes a contiguous
// range of tiles (workgroups are dispatched to the 8 XCDs round-robin).
struct TileWalk {
  int t, end, step;
  __device__ TileWalk(int ntiles) {
    const int g = gridDim.x, b = blockIdx.x;
    if ((g & 7) == 0) {
      const int xcd = b & 7, idx = b >> 3, per = g >> 3;
      const int chunk = (ntiles + 7) >> 3;
      const int t0 = xcd * chunk;
      t = t0 + idx;
      end = min(ntiles, t0 + chunk);
      step = per;
    } else {
      t = b;
      end = ntiles;
      step = g;
    }
  }
};


template <typename T>
__device__ __forceinline__ void store_y(void* y, size_t i, float v) {
  Elem<T>::store1(static_cast<T*>(y), i, v);
}

// ---------------------------------------------------------------- bf16 ----

template <bool FAST, int NTN>
__global__ void __launch_bounds__(kConvThreads) conv_bf16_kernel(ConvParams p) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  const int bb = p.block * p.block;
  const WorkList W = work_list(p.counters, p.seg_tiles, p.seg_cap);
  const long total_rows = (long)W.total * bb;
  if (p.zero_ctr && blockIdx.x == 0 && threadIdx.x < kSegs) p.zero_ctr[threadIdx.x * kSegStride] = 0u;  // next step's work list
  const int ntiles = (int)((total_rows + kRowsPerTile - 1) / kRowsPerTile);
  const uint16_t* xt = static_cast<const uint16_t*>(p.x_t);
  const uint16_t* xp = static_cast<const uint16_t*>(p.no_prev ? p.x_t : p.x_prev);
  const bf16x8* wp = static_cast<const bf16x8*>(p.wpack);
  // FAST (C % 32 == 0): the A fragment of a k-step is one 16-byte piece of
  // each frame; the pieces and weight fragments of kChunkSteps k-steps are
  // loaded together (clamped, unconditional loads masked after), so a chunk
  // costs one memory round trip instead of one per k-step
  constexpr int kChunkSteps = NTN <= 2 ? 8 : (NTN <= 4 ? 4 : 2);

  for (TileWalk tw(ntiles); tw.t < tw.end; tw.t += tw.step) {
    const long g = (long)tw.t * kRowsPerTile + wave * 16 + r16;
    const Site st = site_of_row(p, W, g, total_rows, bb);
    const int iy = st.oy * p.stride - p.pad, ix = st.ox * p.stride - p.pad;
    // old z of the outputs this lane stores, loaded before the product
    const int zrow_mine = st.ok ? (st.n * p.h_out + st.oy) * p.w_out + st.ox : -1;
    int zrow[4];
    float zold[4][NTN];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      zrow[v] = __shfl(zrow_mine, kq * 4 + v, 64);
#pragma unroll
      for (int i = 0; i < NTN; ++i) {
        const int col = i * 16 + r16;
        const bool ok = zrow[v] >= 0 && col < p.c_out && !p.reference;
        zold[v][i] = p.z[ok ? (size_t)zrow[v] * p.c_out + col : 0];
      }
    }
    floatx4 acc[NTN];
#pragma unroll
    for (int i = 0; i < NTN; ++i) acc[i] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

    if constexpr (FAST) {
      const int cpt = p.c >> 5;  // k-steps per tap
      for (int k0 = 0; k0 < p.ksteps; k0 += kChunkSteps) {
        uint4 ra[kChunkSteps], rb[kChunkSteps];
        bf16x8 wv[kChunkSteps][NTN];
        bool in[kChunkSteps], pin[kChunkSteps];
#pragma unroll
        for (int u = 0; u < kChunkSteps; ++u) {
          const int ks = k0 + u;
          const int tap = ks / cpt;
          const int c0 = (ks - tap * cpt) * 32 + kq * 8;
          const int kh = tap / p.k, kw = tap - kh * p.k;
          const int y = iy + kh, x = ix + kw;
          in[u] = st.ok && ks < p.ksteps && y >= 0 && y < p.h && x >= 0 && x < p.w;
          const size_t off = in[u] ? ((size_t)(st.n * p.h + y) * p.w + x) * p.c + c0 : 0;
          const long po = (in[u] && !p.no_prev) ? prev_off(p, st.n, y, x, c0) : -1;
          pin[u] = po >= 0;
          ra[u] = *reinterpret_cast<const uint4*>(xt + off);
          rb[u] = *reinterpret_cast<const uint4*>(xp + (pin[u] ? (size_t)po : 0));
          const bf16x8* wk = wp + (size_t)(ks < p.ksteps ? ks : 0) * NTN * 64 + lane;
#pragma unroll
          for (int i = 0; i < NTN; ++i) wv[u][i] = wk[i * 64];
        }
#pragma unroll
        for (int u = 0; u < kChunkSteps; ++u) {
          if (k0 + u >= p.ksteps) continue;  // wave-uniform (not a break: the loop stays unrolled)
          const uint32_t wa[4] = {ra[u].x, ra[u].y, ra[u].z, ra[u].w};
          const uint32_t wb[4] = {rb[u].x, rb[u].y, rb[u].z, rb[u].w};
          u32x4 q;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float a0 = __uint_as_float(wa[e] << 16), a1 = __uint_as_float(wa[e] & 0xffff0000u);
            const float b0 = pin[u] ? __uint_as_float(wb[e] << 16) : 0.0f;
            const float b1 = pin[u] ? __uint_as_float(wb[e] & 0xffff0000u) : 0.0f;
            const float r0 = in[u] ? __fsub_rn(a0, b0) : 0.0f, r1 = in[u] ? __fsub_rn(a1, b1) : 0.0f;
            q[e] = f32_to_bf16(r0) | (f32_to_bf16(r1) << 16);
          }
          const bf16x8 a = __builtin_bit_cast(bf16x8, q);
#pragma unroll
          for (int i = 0; i < NTN; ++i)
            acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, wv[u][i], acc[i], 0, 0, 0);
        }
      }
    } else {
      // C % 32 != 0: the 8 k indices of a lane's A piece may fall on
      // different taps, so each element is loaded on its own; the 16 element
      // loads of every k-step of a chunk and its weight fragments go out
      // together (clamped to element 0 and masked after, as above). Tap and
      // channel come from qdiv (exact for these sizes).
      constexpr int kSteps = NTN <= 4 ? 2 : 1;
      const int kk = p.k * p.k * p.c;
      const float inv_c = 1.0f / (float)p.c, inv_k = 1.0f / (float)p.k;
      for (int k0 = 0; k0 < p.ksteps; k0 += kSteps) {
        uint32_t ea[kSteps][8], eb[kSteps][8];
        bool ein[kSteps][8], epin[kSteps][8];
        bf16x8 wv[kSteps][NTN];
#pragma unroll
        for (int u = 0; u < kSteps; ++u) {
          const int ks = k0 + u;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int kidx = ks * 32 + kq * 8 + e;
            const int tap = qdiv(kidx, inv_c), ci = kidx - tap * p.c;
            const int kh = qdiv(tap, inv_k), kw = tap - kh * p.k;
            const int y = iy + kh, x = ix + kw;
            const bool in = st.ok && ks < p.ksteps && kidx < kk && y >= 0 && y < p.h && x >= 0 && x < p.w;
            const size_t off = in ? ((size_t)(st.n * p.h + y) * p.w + x) * p.c + ci : 0;
            const long po = (in && !p.no_prev) ? prev_off(p, st.n, y, x, ci) : -1;
            ein[u][e] = in;
            epin[u][e] = po >= 0;
            ea[u][e] = xt[off];
            eb[u][e] = xp[po >= 0 ? (size_t)po : 0];
          }
          const bf16x8* wk = wp + (size_t)(ks < p.ksteps ? ks : 0) * NTN * 64 + lane;
#pragma unroll
          for (int i = 0; i < NTN; ++i) wv[u][i] = wk[i * 64];
        }
#pragma unroll
        for (int u = 0; u < kSteps; ++u) {
          if (k0 + u >= p.ksteps) continue;  // wave-uniform (not a break: the loop stays unrolled)
          float v[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float xa = __uint_as_float(ea[u][e] << 16);
            const float xb = epin[u][e] ? __uint_as_float(eb[u][e] << 16) : 0.0f;
            v[e] = ein[u][e] ? __fsub_rn(xa, xb) : 0.0f;
          }
          u32x4 q;
#pragma unroll
          for (int e = 0; e < 4; ++e) q[e] = f32_to_bf16(v[2 * e]) | (f32_to_bf16(v[2 * e + 1]) << 16);
          const bf16x8 a = __builtin_bit_cast(bf16x8, q);
#pragma unroll
          for (int i = 0; i < NTN; ++i)
            acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, wv[u][i], acc[i], 0, 0, 0);
        }
      }
    }

    // epilogue: lane holds D[4*(lane/16) + v][lane % 16] of each 16x16 tile
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      if (zrow[v] < 0) continue;
#pragma unroll
      for (int i = 0; i < NTN; ++i) {
        const int col = i * 16 + r16;
        if (col >= p.c_out) continue;
        const size_t idx = (size_t)zrow[v] * p.c_out + col;
        const float nv = p.reference ? acc[i][v] : zold[v][i] + acc[i][v];
        p.z[idx] = nv;
        if (p.act) store_y<uint16_t>(p.y, idx, activate(nv, p.act));
      }
    }
  }
}

// ------------------------------------------------------- bf16, halo ----
//
// Block tiles (b in {4, 8, 16, 32, 64}, C_in % 32 == 0): a tile is `tr` output
// rows x b columns of one active block, convolved by HaloConv (sc_halo_conv.h).
// A persistent grid walks the tiles of the listed blocks; with PZ the next
// tile's z_{t-1} is issued before this tile's stores (sites of different tiles
// are disjoint), into registers that are not the stores' sources, so no wait
// on the stores precedes them; the halo loads of a tile then wait once for
// everything in flight. Without PZ a tile's z_{t-1} is loaded with its halo.
// OCC: waves per SIMD the register budget aims for.

// EMIT: the epilogue also writes y_new and the successor's residual; y_old is
// loaded with z_{t-1}.
template <int WAVES_M, int WAVES_N, int WM, int WN, int KR = 0, bool PZ = true, int OCC = 2, int KU = 12,
          int ADB = 2, bool EMIT = false>
__global__ void __launch_bounds__(64 * WAVES_M * WAVES_N) __attribute__((amdgpu_waves_per_eu(EMIT && OCC > 2 ? 2 : OCC)))
conv_halo_kernel(ConvParams p, HaloParams hp) {
  extern __shared__ __attribute__((aligned(16))) uint8_t halo[];
  typedef HaloConv<WAVES_M, WAVES_N, WM, WN, KR, KU, ADB> HC;
  const int tpb = hp.tiles_per_block;
  const WorkList W = work_list(p.counters, p.seg_tiles, p.seg_cap);
  const int ntiles = (int)W.total * tpb;
  if (p.zero_ctr && blockIdx.x == 0 && threadIdx.x < kSegs) p.zero_ctr[threadIdx.x * kSegStride] = 0u;  // next step's work list
  const HC H(p, hp, halo);

  // Tiles walked in order; the active list is read through the scalar cache
  // (written by an earlier kernel, read-only here), so decoding a tile waits
  // on no vector memory operation.
  typedef const __attribute__((address_space(4))) uint32_t const_u32;
  const const_u32* list = (const const_u32*)p.list;
  auto decode = [&](int t) {
    const int j0 = t / tpb, band = t - j0 * tpb;
    const uint32_t blk = list[work_pos(W, (uint32_t)j0)];
    const int per_img = p.hb * p.wb;
    const int n = (int)(blk / per_img);
    const int rem = (int)(blk - (uint32_t)n * per_img);
    const int bi = rem / p.wb, bj = rem - bi * p.wb;
    return H.tile(n, bi * p.block + band * hp.tr, bj * p.block);
  };

  TileWalk tw(ntiles);
  if (tw.t >= tw.end) return;
  HaloTile T = decode(tw.t);
  typename HC::Acc zn;
  typename HC::Yv yn;  // emission: y_old of the next tile (PZ)
  if constexpr (PZ) H.load_z(zn, T, false);
  if constexpr (PZ && EMIT) H.load_y(yn, T, false);
  for (; tw.t < tw.end; tw.t += tw.step) {
    typename HC::Acc acc;
    typename HC::Yv yo;
    if constexpr (!PZ) H.load_z(acc, T, false);  // in flight with the halo loads
    if constexpr (!PZ && EMIT) H.load_y(yo, T, false);
    H.load_halo(T);
    if constexpr (PZ) {
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int jn = 0; jn < WN; ++jn) {
          acc[i][jn] = zn[i][jn];
          if constexpr (EMIT) yo[i][jn] = yn[i][jn];
        }
    }
    __syncthreads();
    H.product(acc);
    // all waves are done with the halo: the next tile may overwrite it
    __syncthreads();
    const bool more = tw.t + tw.step < tw.end;
    const HaloTile Tn = more ? decode(tw.t + tw.step) : T;
    if constexpr (PZ) H.load_z(zn, Tn, !more);
    if constexpr (PZ && EMIT) H.load_y(yn, Tn, !more);
    if constexpr (EMIT) H.store_emit(T, acc, yo);
    else H.store(T, acc);
    T = Tn;
  }
}

// ---------------------------------------------------------------- fp32 ----

// Tiles of kConvF32Rows output sites; the waves of a workgroup split the
// k-steps into contiguous parts. fp32 layers are the small frames, whose few
// tiles left most of the chip idle while one wave per tile walked all of K.
// The part sums meet in LDS, where wave 0 adds them in part order and updates
// z. Tap and channel of a k index come from qdiv (exact for these sizes), not
// from integer divisions.
template <int NTN>
__global__ void __launch_bounds__(kConvThreads) conv_f32_kernel(ConvParams p) {
  // k-steps whose operand (two frames) and weight loads are issued together:
  // every load is unconditional (clamped to element 0 and masked after), so
  // a chunk costs one memory round trip instead of one per k-step
  constexpr int kChunkSteps = NTN <= 2 ? 16 : (NTN <= 4 ? 8 : 4);
  constexpr int kWaves = kConvThreads / 64;
  __shared__ floatx4 part[kWaves - 1][NTN][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kq = lane >> 4;
  const int bb = p.block * p.block;
  const WorkList W = work_list(p.counters, p.seg_tiles, p.seg_cap);
  const long total_rows = (long)W.total * bb;
  if (p.zero_ctr && blockIdx.x == 0 && threadIdx.x < kSegs) p.zero_ctr[threadIdx.x * kSegStride] = 0u;  // next step's work list
  const int ntiles = (int)((total_rows + kConvF32Rows - 1) / kConvF32Rows);
  const float* xt = static_cast<const float*>(p.x_t);
  const float* xp = static_cast<const float*>(p.no_prev ? p.x_t : p.x_prev);
  const float* wp = static_cast<const float*>(p.wpack);
  const int kk = p.k * p.k * p.c;
  const int ks0 = wave * p.ksteps / kWaves, ks1 = (wave + 1) * p.ksteps / kWaves;  // this wave's k-part
  const float inv_c = 1.0f / (float)p.c, inv_k = 1.0f / (float)p.k;

  for (TileWalk tw(ntiles); tw.t < tw.end; tw.t += tw.step) {
    const long g = (long)tw.t * kConvF32Rows + r16;
    const Site st = site_of_row(p, W, g, total_rows, bb);
    const int iy = st.oy * p.stride - p.pad, ix = st.ox * p.stride - p.pad;
    // old z of the outputs wave 0 stores (site of lane kq * 4 + v, column
    // i * 16 + r16), loaded before the product (other waves read element 0)
    const int zrow_mine = st.ok ? (st.n * p.h_out + st.oy) * p.w_out + st.ox : -1;
    int zrow[4];
    float zold[4][NTN];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      zrow[v] = __shfl(zrow_mine, kq * 4 + v, 64);
#pragma unroll
      for (int i = 0; i < NTN; ++i) {
        const int col = i * 16 + r16;
        const bool ok = wave == 0 && zrow[v] >= 0 && col < p.c_out && !p.reference;
        zold[v][i] = p.z[ok ? (size_t)zrow[v] * p.c_out + col : 0];
      }
    }
    floatx4 acc[NTN];
#pragma unroll
    for (int i = 0; i < NTN; ++i) acc[i] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

    for (int k0 = ks0; k0 < ks1; k0 += kChunkSteps) {
      float av[kChunkSteps], pv[kChunkSteps], wv[kChunkSteps][NTN];
      bool in[kChunkSteps], pin[kChunkSteps];
#pragma unroll
      for (int u = 0; u < kChunkSteps; ++u) {
        const int ks = k0 + u;
        const int kidx = ks * 4 + kq;
        const int tap = qdiv(kidx, inv_c), ci = kidx - tap * p.c;
        const int kh = qdiv(tap, inv_k), kw = tap - kh * p.k;
        const int y = iy + kh, x = ix + kw;
        in[u] = st.ok && ks < ks1 && kidx < kk && y >= 0 && y < p.h && x >= 0 && x < p.w;
        const size_t off = in[u] ? ((size_t)(st.n * p.h + y) * p.w + x) * p.c + ci : 0;
        const long po = (in[u] && !p.no_prev) ? prev_off(p, st.n, y, x, ci) : -1;
        pin[u] = po >= 0;
        av[u] = xt[off];
        pv[u] = xp[pin[u] ? (size_t)po : 0];
        const float* wk = wp + (size_t)(ks < ks1 ? ks : 0) * NTN * 64 + lane;
#pragma unroll
        for (int i = 0; i < NTN; ++i) wv[u][i] = wk[i * 64];
      }
#pragma unroll
      for (int u = 0; u < kChunkSteps; ++u) {
        if (k0 + u < ks1) {  // wave-uniform (a guard, not a break: the loop stays unrolled)
          const float a = !in[u] ? 0.0f : (pin[u] ? __fsub_rn(av[u], pv[u]) : av[u]);
#pragma unroll
          for (int i = 0; i < NTN; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, wv[u][i], acc[i], 0, 0, 0);
        }
      }
    }

    if (wave > 0) {
#pragma unroll
      for (int i = 0; i < NTN; ++i) part[wave - 1][i][lane] = acc[i];
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int q = 0; q < kWaves - 1; ++q) {
#pragma unroll
        for (int i = 0; i < NTN; ++i) {
          const floatx4 s4 = part[q][i][lane];
#pragma unroll
          for (int v = 0; v < 4; ++v) acc[i][v] = __fadd_rn(acc[i][v], s4[v]);
        }
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        if (zrow[v] < 0) continue;
#pragma unroll
        for (int i = 0; i < NTN; ++i) {
          const int col = i * 16 + r16;
          if (col >= p.c_out) continue;
          const size_t idx = (size_t)zrow[v] * p.c_out + col;
          const float nv = p.reference ? acc[i][v] : zold[v][i] + acc[i][v];
          p.z[idx] = nv;
          if (p.act) store_y<float>(p.y, idx, activate(nv, p.act));
        }
      }
    }
    __syncthreads();  // part is rewritten by the next tile
  }
}

// ----------------------------------------------------------- depthwise ----

template <typename T, int VEC>
__global__ void __launch_bounds__(kConvThreads) depthwise_kernel(ConvParams p) {
  const int bb = p.block * p.block;
  const WorkList W = work_list(p.counters, p.seg_tiles, p.seg_cap);
  const long total_rows = (long)W.total * bb;
  if (p.zero_ctr && blockIdx.x == 0 && threadIdx.x < kSegs) p.zero_ctr[threadIdx.x * kSegStride] = 0u;  // next step's work list
  const int ntiles = (int)((total_rows + kRowsPerTile - 1) / kRowsPerTile);
  const T* xt = static_cast<const T*>(p.x_t);
  const T* xp = static_cast<const T*>(p.x_prev);
  const float* wp = static_cast<const float*>(p.wpack);  // [tap][c] fp32
  const int nchunk = p.c / VEC;
  const bool bf16 = sizeof(T) == 2;

  for (TileWalk tw(ntiles); tw.t < tw.end; tw.t += tw.step) {
    for (int item = threadIdx.x; item < kRowsPerTile * nchunk; item += kConvThreads) {
      const int row = item / nchunk;
      const int c0 = (item - row * nchunk) * VEC;
      const Site st = site_of_row(p, W, (long)tw.t * kRowsPerTile + row, total_rows, bb);
      if (!st.ok) continue;
      const int iy = st.oy * p.stride - p.pad, ix = st.ox * p.stride - p.pad;
      float acc[VEC];
#pragma unroll
      for (int j = 0; j < VEC; ++j) acc[j] = 0.0f;
      for (int kh = 0; kh < p.k; ++kh) {
        const int y = iy + kh;
        if (y < 0 || y >= p.h) continue;
        for (int kw = 0; kw < p.k; ++kw) {
          const int x = ix + kw;
          if (x < 0 || x >= p.w) continue;
          const size_t off = ((size_t)(st.n * p.h + y) * p.w + x) * p.c + c0;
          float a[VEC], b[VEC];
          const long po = p.no_prev ? -1 : prev_off(p, st.n, y, x, c0);
          if (VEC == 8) {
            Elem<T>::load8(xt, off, a);
            if (po >= 0) Elem<T>::load8(xp, (size_t)po, b);
          } else if (VEC == 4) {
            Elem<T>::load4(xt, off, a);
            if (po >= 0) Elem<T>::load4(xp, (size_t)po, b);
          } else {
            a[0] = Elem<T>::load1(xt, off);
            if (po >= 0) b[0] = Elem<T>::load1(xp, (size_t)po);
          }
          const float* wt = wp + (kh * p.k + kw) * p.c + c0;
#pragma unroll
          for (int j = 0; j < VEC; ++j) {
            float r = po < 0 ? a[j] : __fsub_rn(a[j], b[j]);
            if (bf16) r = bf16_to_f32(f32_to_bf16(r));
            acc[j] = __builtin_fmaf(wt[j], r, acc[j]);
          }
        }
      }
      const size_t zb = ((size_t)(st.n * p.h_out + st.oy) * p.w_out + st.ox) * p.c_out + c0;
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        const float nv = p.reference ? acc[j] : p.z[zb + j] + acc[j];
        p.z[zb + j] = nv;
        if (p.act) store_y<T>(p.y, zb + j, activate(nv, p.act));
      }
    }
  }
}

// ------------------------------------------------ depthwise, bf16, halo ----
//
// Depthwise layers (groups = C, bf16, C % 8 == 0) over active blocks: a tile
// is tr output rows x b columns of one active block (tr * b sites). Per tile:
// the old z of this thread's outputs is loaded, then the residual halo
// ((tr-1)s+k rows x (b-1)s+k columns x C) with every load of a round in
// flight, rho = bf16(x_t - x_{t-1}) stored in LDS (zero outside the frame:
// such taps add exactly nothing); each thread then forms 8 channels of one
// site at a time, fp32 FMA over the k x k taps in row-major order with the
// [tap][c] weights staged in LDS once per workgroup, and writes z (and the
// activation). Consecutive threads take consecutive channel chunks, so z
// moves in contiguous 32-byte pieces per thread and LDS reads are
// conflict-free.
constexpr int kDwThreads = 256;
constexpr int kDwItems = 12;  // halo chunks in flight per thread (10 x 10 x 24 chunks: one round)
constexpr int kDwOut = 8;     // output chunks per thread and pass

__global__ void __launch_bounds__(kDwThreads) depthwise_halo_kernel(ConvParams p, HaloParams hp) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  uint8_t* halo = lds;
  float* wl = reinterpret_cast<float*>(lds + hp.lds_bytes);  // [tap][c]
  const int b = p.block, s = p.stride, k = p.k, c = p.c;
  const int nchunk = c >> 3;
  const int tpb = hp.tiles_per_block;
  const WorkList W = work_list(p.counters, p.seg_tiles, p.seg_cap);
  const int ntiles = (int)W.total * tpb;
  if (p.zero_ctr && blockIdx.x == 0 && threadIdx.x < kSegs) p.zero_ctr[threadIdx.x * kSegStride] = 0u;  // next step's work list
  const uint16_t* xt = static_cast<const uint16_t*>(p.x_t);
  const uint16_t* xp = static_cast<const uint16_t*>(p.x_prev);
  const size_t ximg = (size_t)p.h * p.w * c;
  const size_t zimg = (size_t)p.h_out * p.w_out * c;
  {
    // [tap][c] weights into LDS, 16 bytes per load, four loads in flight per thread
    const float4* w4 = static_cast<const float4*>(p.wpack);
    float4* l4 = reinterpret_cast<float4*>(wl);
    const int nw4 = k * k * c / 4;
    for (int base = 0; base < nw4; base += 4 * kDwThreads) {
      float4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = base + u * kDwThreads + threadIdx.x;
        v[u] = w4[i < nw4 ? i : 0];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = base + u * kDwThreads + threadIdx.x;
        if (i < nw4) l4[i] = v[u];
      }
    }
  }
  typedef const __attribute__((address_space(4))) uint32_t const_u32;
  const const_u32* list = (const const_u32*)p.list;
  const int total = hp.hh * hp.hw * nchunk;
  const int nout = hp.tr * b * nchunk;

  for (TileWalk tw(ntiles); tw.t < tw.end; tw.t += tw.step) {
    const int j0 = tw.t / tpb, band = tw.t - j0 * tpb;
    const uint32_t blk = list[work_pos(W, (uint32_t)j0)];
    const int per_img = p.hb * p.wb;
    const int n = (int)(blk / per_img);
    const int rem = (int)(blk - (uint32_t)n * per_img);
    const int bi = rem / p.wb, bj = rem - bi * p.wb;
    const int oy0 = bi * b + band * hp.tr, ox0 = bj * b;
    const int rows_ok = min(min(hp.tr, b - band * hp.tr), p.h_out - oy0), cols_ok = min(b, p.w_out - ox0);
    const int iy0 = oy0 * s - p.pad, ix0 = ox0 * s - p.pad;
    const auto xrs = frame_rsrc(xt + (size_t)n * ximg, (uint32_t)(ximg * 2));
    const auto prs = frame_rsrc((p.no_prev ? xt : xp) + (size_t)n * ximg, (uint32_t)(ximg * 2));
    const auto zrs = frame_rsrc(p.z + (size_t)n * zimg, (uint32_t)(zimg * 4));

    // old z of a pass of kDwOut (site, chunk) outputs per thread; out-of-range
    // offsets for outputs outside the tile (and for every output on a reference frame)
    floatx4 zo[kDwOut][2];
    uint32_t zoff[kDwOut];
    auto zload = [&](int base) {
#pragma unroll
      for (int u = 0; u < kDwOut; ++u) {
        const int idx = base + u * kDwThreads + threadIdx.x;
        const int site = idx / nchunk, ch = idx - site * nchunk;
        const int ly = site / b, lx = site - ly * b;
        const bool ok = idx < nout && ly < rows_ok && lx < cols_ok;
        zoff[u] = ok ? (uint32_t)((((oy0 + ly) * p.w_out + ox0 + lx) * c + ch * 8) * 4) : kOutOfRange;
#pragma unroll
        for (int hlf = 0; hlf < 2; ++hlf)
          zo[u][hlf] = __builtin_bit_cast(
              floatx4, __builtin_amdgcn_raw_buffer_load_b128(
                           zrs, p.reference || !ok ? kOutOfRange : zoff[u] + 16 * hlf, 0, 0));
      }
    };
    auto outputs = [&](int base) {
#pragma unroll
      for (int u = 0; u < kDwOut; ++u) {
        const int idx = base + u * kDwThreads + threadIdx.x;
        if (idx >= nout) continue;
        const int site = idx / nchunk, ch = idx - site * nchunk;
        const int ly = site / b, lx = site - ly * b;
        float acc[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = 0.0f;
        for (int kh = 0; kh < k; ++kh)
          for (int kw = 0; kw < k; ++kw) {
            const u32x4 r = *reinterpret_cast<const u32x4*>(
                halo + ((ly * s + kh) * hp.hw + lx * s + kw) * hp.pstride + ch * 16);
            const float* wt = wl + (kh * k + kw) * c + ch * 8;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              acc[2 * e] = __builtin_fmaf(wt[2 * e], __uint_as_float(r[e] << 16), acc[2 * e]);
              acc[2 * e + 1] = __builtin_fmaf(wt[2 * e + 1], __uint_as_float(r[e] & 0xffff0000u), acc[2 * e + 1]);
            }
          }
        floatx4 nv[2];
#pragma unroll
        for (int j = 0; j < 8; ++j) nv[j >> 2][j & 3] = p.reference ? acc[j] : zo[u][j >> 2][j & 3] + acc[j];
#pragma unroll
        for (int hlf = 0; hlf < 2; ++hlf)
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, nv[hlf]), zrs,
                                                 zoff[u] == kOutOfRange ? kOutOfRange : zoff[u] + 16 * hlf, 0, 0);
        if (p.act && zoff[u] != kOutOfRange) {
          const size_t o = (size_t)n * zimg + zoff[u] / 4;
#pragma unroll
          for (int j = 0; j < 8; ++j) store_y<uint16_t>(p.y, o + j, activate(nv[j >> 2][j & 3], p.act));
        }
      }
    };

    // the first pass's old z is in flight with the halo loads
    zload(0);
    // halo rounds: rho = bf16(x_t - x_{t-1}) into LDS
    for (int base = 0; base < total; base += kDwThreads * kDwItems) {
      u32x4 ra[kDwItems], rb[kDwItems];
#pragma unroll
      for (int u = 0; u < kDwItems; ++u) {
        const int idx = base + u * kDwThreads + threadIdx.x;
        const int px = idx / nchunk, ch = idx - px * nchunk;
        const int hy = px / hp.hw, hx = px - hy * hp.hw;
        const int y = iy0 + hy, x = ix0 + hx;
        const bool in = idx < total && y >= 0 && y < p.h && x >= 0 && x < p.w;
        const int yp = y - p.sy, xq = x - p.sx;
        const bool pin = in && !p.no_prev && yp >= 0 && yp < p.h && xq >= 0 && xq < p.w;
        ra[u] = __builtin_amdgcn_raw_buffer_load_b128(
            xrs, in ? (uint32_t)(((y * p.w + x) * c + ch * 8) * 2) : kOutOfRange, 0, 0);
        rb[u] = __builtin_amdgcn_raw_buffer_load_b128(
            prs, pin ? (uint32_t)(((yp * p.w + xq) * c + ch * 8) * 2) : kOutOfRange, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < kDwItems; ++u) {
        const int idx = base + u * kDwThreads + threadIdx.x;
        if (idx >= total) continue;
        const int px = idx / nchunk, ch = idx - px * nchunk;
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
    __syncthreads();
    outputs(0);
    for (int base = kDwThreads * kDwOut; base < nout; base += kDwThreads * kDwOut) {
      zload(base);
      outputs(base);
    }
    // all waves are done with the halo before the next tile overwrites it
    __syncthreads();
  }
}

// -------------------------------------------------------------- repack ----

// B fragment layout of v_mfma_f32_16x16x32_bf16: for k-step ks and output tile
// nt, lane l holds B[k = ks*32 + 8*(l/16) + e][n = nt*16 + l%16], e = 0..7,
// with K ordered (kh, kw, ci). For v_mfma_f32_16x16x4_f32 lane l holds
// B[k = ks*4 + l/16][n = nt*16 + l%16]. Entries beyond K or C_out are zero.
__global__ void pack_mfma_kernel(const void* w, void* out, int dtype, int c_out, int c_in, int k,
                                 int ksteps, int ntn) {
  const int per_lane = dtype == 1 ? 8 : 1;
  const int kstep = dtype == 1 ? 32 : 4;
  const long total = (long)ksteps * ntn * 64 * per_lane;
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int e = (int)(i % per_lane);
  const long q = i / per_lane;
  const int lane = (int)(q % 64);
  const long q2 = q / 64;
  const int nt = (int)(q2 % ntn);
  const int ks = (int)(q2 / ntn);
  const int kidx = ks * kstep + (lane >> 4) * per_lane + e;
  const int co = nt * 16 + (lane & 15);
  const int kk = k * k * c_in;
  float v = 0.0f;
  if (kidx < kk && co < c_out) {
    const int tap = kidx / c_in, ci = kidx - tap * c_in;
    const int kh = tap / k, kw = tap - kh * k;
    const size_t src = (((size_t)co * c_in + ci) * k + kh) * k + kw;
    v = dtype == 1 ? bf16_to_f32(static_cast<const uint16_t*>(w)[src]) : static_cast<const float*>(w)[src];
  }
  if (dtype == 1)
    static_cast<uint16_t*>(out)[i] = (uint16_t)f32_to_bf16(v);  // exact: v is a bf16 value
  else
    static_cast<float*>(out)[i] = v;
}

// Depthwise weights (C x 1 x k x k) to [tap][c] fp32.
__global__ void pack_depthwise_kernel(const void* w, float* out, int dtype, int c, int k) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= c * k * k) return;
  const int tap = i / c, ch = i - tap * c;
  const size_t src = (size_t)ch * k * k + tap;
  out[i] = dtype == 1 ? bf16_to_f32(static_cast<const uint16_t*>(w)[src]) : static_cast<const float*>(w)[src];
}

template <bool FAST>
hipError_t launch_conv_bf16(const ConvParams& p, int grid, hipStream_t st) {
  switch (p.ntiles_n) {
    case 1: hipLaunchKernelGGL((conv_bf16_kernel<FAST, 1>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    case 2: hipLaunchKernelGGL((conv_bf16_kernel<FAST, 2>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    case 4: hipLaunchKernelGGL((conv_bf16_kernel<FAST, 4>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    case 8: hipLaunchKernelGGL((conv_bf16_kernel<FAST, 8>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    case 12: hipLaunchKernelGGL((conv_bf16_kernel<FAST, 12>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    case 16: hipLaunchKernelGGL((conv_bf16_kernel<FAST, 16>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_conv_f32(const ConvParams& p, int grid, hipStream_t st) {
  switch (p.ntiles_n) {
    case 1: hipLaunchKernelGGL((conv_f32_kernel<1>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    case 2: hipLaunchKernelGGL((conv_f32_kernel<2>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    case 4: hipLaunchKernelGGL((conv_f32_kernel<4>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    case 8: hipLaunchKernelGGL((conv_f32_kernel<8>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    case 12: hipLaunchKernelGGL((conv_f32_kernel<12>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    case 16: hipLaunchKernelGGL((conv_f32_kernel<16>), dim3(grid), dim3(kConvThreads), 0, st, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int WAVES_M, int WAVES_N, int WM, int WN, int KR, bool PZ, int OCC, int KU, int ADB>
hipError_t launch_halo_t(const ConvParams& p, const HaloParams& hp, int grid, hipStream_t st) {
  if (hp.emit)
    hipLaunchKernelGGL((conv_halo_kernel<WAVES_M, WAVES_N, WM, WN, KR, PZ, OCC, KU, ADB, true>), dim3(grid),
                       dim3(64 * WAVES_M * WAVES_N), hp.lds_bytes, st, p, hp);
  else
    hipLaunchKernelGGL((conv_halo_kernel<WAVES_M, WAVES_N, WM, WN, KR, PZ, OCC, KU, ADB>), dim3(grid),
                       dim3(64 * WAVES_M * WAVES_N), hp.lds_bytes, st, p, hp);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_conv(const ConvParams& p, int dtype, bool fast, int grid, hipStream_t st) {
  if (dtype == 0) return launch_conv_f32(p, grid, st);
  return fast ? launch_conv_bf16<true>(p, grid, st) : launch_conv_bf16<false>(p, grid, st);
}

namespace {
template <int WAVES_M, int WAVES_N, int WM, int WN, int KR, bool PZ, int OCC, int KU, int ADB>
int halo_occ_t(const HaloParams& hp) {
  auto fn = hp.emit ? conv_halo_kernel<WAVES_M, WAVES_N, WM, WN, KR, PZ, OCC, KU, ADB, true>
                    : conv_halo_kernel<WAVES_M, WAVES_N, WM, WN, KR, PZ, OCC, KU, ADB>;
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                          hp.lds_bytes) != hipSuccess)
    return 0;
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fn, 64 * WAVES_M * WAVES_N, hp.lds_bytes) !=
      hipSuccess)
    return 0;
  return blocks;
}
}  // namespace

// id, WAVES_M, WAVES_N, WM, WN, KR, PZ, OCC, KU, ADB. Config 3 (128 output
// channels, 128-site tiles): one A register set and a two-deep B ring, so
// that three workgroups fit on a CU (131-145 VGPRs), z_{t-1} loaded with the
// halo; measured 134.7 / 443 us against 141 / 452 us for the two-set build at
// 4 x 512 x 512 x 128 (29 % of the blocks / all blocks).
#define SC_HALO_CONFIGS(X)                                                                                  \
  X(0, 1, 1, 8, 1, 0, true, 2, 12, 2) X(1, 1, 2, 8, 1, 0, true, 2, 12, 2) X(2, 1, 4, 8, 1, 0, true, 2, 12, 2) \
  X(3, 1, 4, 8, 2, 2, false, 3, 6, 1)                                                                      \
  X(10, 1, 1, 4, 1, 0, true, 2, 12, 2) X(11, 1, 2, 4, 1, 0, true, 2, 12, 2)                                \
  X(12, 1, 4, 4, 1, 0, true, 2, 12, 2) X(13, 1, 4, 4, 2, 0, true, 2, 12, 2)                                \
  X(14, 1, 4, 4, 3, 0, true, 2, 12, 2) X(15, 1, 4, 4, 4, 0, true, 2, 12, 2)                                \
  X(20, 1, 1, 1, 1, 0, true, 2, 12, 2) X(21, 1, 2, 1, 1, 0, true, 2, 12, 2)                                \
  X(22, 1, 4, 1, 1, 0, true, 2, 12, 2) X(23, 1, 4, 1, 2, 0, true, 2, 12, 2)                                \
  X(24, 1, 4, 1, 3, 0, true, 2, 12, 2) X(25, 1, 4, 1, 4, 0, true, 2, 12, 2)

int conv_halo_occupancy(const HaloParams& hp) {
  switch (hp.config) {
#define SC_X(id, a, b, c, d, e, f, g, u, v) \
  case id:                                  \
    return halo_occ_t<a, b, c, d, e, f, g, u, v>(hp);
    SC_HALO_CONFIGS(SC_X)
#undef SC_X
    default: return 0;
  }
}

hipError_t launch_conv_halo(const ConvParams& p, const HaloParams& hp, int grid, hipStream_t st) {
  switch (hp.config) {
#define SC_X(id, a, b, c, d, e, f, g, u, v) \
  case id:                                  \
    return launch_halo_t<a, b, c, d, e, f, g, u, v>(p, hp, grid, st);
    SC_HALO_CONFIGS(SC_X)
#undef SC_X
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_depthwise_halo(const ConvParams& p, const HaloParams& hp, int grid, hipStream_t st) {
  const int lds = hp.lds_bytes + p.k * p.k * p.c * 4;
  hipLaunchKernelGGL(depthwise_halo_kernel, dim3(grid), dim3(kDwThreads), lds, st, p, hp);
  return hipGetLastError();
}

int depthwise_halo_occupancy(const HaloParams& hp, int k, int c) {
  const int lds = hp.lds_bytes + k * k * c * 4;
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(depthwise_halo_kernel),
                          hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess)
    return 0;
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, depthwise_halo_kernel, kDwThreads, lds) != hipSuccess)
    return 0;
  return blocks;
}

hipError_t launch_depthwise(const ConvParams& p, int dtype, int grid, hipStream_t st) {
  if (dtype == 0) {
    if (p.c % 4 == 0)
      hipLaunchKernelGGL((depthwise_kernel<float, 4>), dim3(grid), dim3(kConvThreads), 0, st, p);
    else
      hipLaunchKernelGGL((depthwise_kernel<float, 1>), dim3(grid), dim3(kConvThreads), 0, st, p);
  } else {
    if (p.c % 8 == 0)
      hipLaunchKernelGGL((depthwise_kernel<uint16_t, 8>), dim3(grid), dim3(kConvThreads), 0, st, p);
    else
      hipLaunchKernelGGL((depthwise_kernel<uint16_t, 1>), dim3(grid), dim3(kConvThreads), 0, st, p);
  }
  return hipGetLastError();
}

hipError_t launch_pack_mfma(const void* w, void* out, int dtype, int c_out, int c_in, int k,
                            int ksteps, int ntiles_n, hipStream_t st) {
  const long total = (long)ksteps * ntiles_n * 64 * (dtype == 1 ? 8 : 1);
  const int grid = (int)((total + 255) / 256);
  hipLaunchKernelGGL(pack_mfma_kernel, dim3(grid), dim3(256), 0, st, w, out, dtype, c_out, c_in, k,
                     ksteps, ntiles_n);
  return hipGetLastError();
}

hipError_t launch_pack_depthwise(const void* w, float* out, int dtype, int c, int k,
                                 hipStream_t st) {
  const int total = c * k * k;
  hipLaunchKernelGGL(pack_depthwise_kernel, dim3((total + 255) / 256), dim3(256), 0, st, w, out,
                     dtype, c, k);
  return hipGetLastError();
}

}  // namespace sc
