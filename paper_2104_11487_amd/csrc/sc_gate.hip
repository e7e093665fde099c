// Gate kernel of the Skip-Conv layer's split pipeline: residual, gate
// statistic, threshold, block pooling and the convolution's work list, fused
// in one launch.
//
//   Eq. 2     r = x_t - x_{t-1} (x_{t-1} = 0 on a reference frame, Sec. 3.1)
//   Eq. 5     s[o] = norm of r over the kernel support of output o;
//             g[o] = s[o] > eps^2 (p = 2) or s[o] > eps (p = 1), or s NaN
//             (Eq. 7: s times the weight norm; Eq. 8: a learned score > 0)
//   Sec 3.2.2 block mask M[B] = OR of g over the b x b block B (ceil mode)
//   Sec 4.2   work list = the active blocks (the "non-sparse columns" of the
//             im2col product the convolution multiplies)
//
// Statistic arithmetic is canonical so that masks are reproducible bit for
// bit: fp32 r; per pixel a[q] = chunk sums of 8 consecutive channels (terms
// added in ascending order), then the chunk sums added in ascending order,
// one rounding per multiply and per add, no FMA; s[o] = sum of a over the taps
// (kh, kw) in row-major order, in fp32; the threshold comparison in fp64.
//
// One workgroup owns a TS x TS tile of output sites (whole blocks when
// b <= 16). One thread takes one 8-channel chunk of one halo pixel at a time
// (a 16-byte load of each frame for bf16; consecutive threads read
// consecutive chunks, eight chunks in flight per thread) and forms the chunk
// sum. With 4, 8 or 16 chunks per pixel the pixel's lanes add their chunk
// sums in order through DPP lane shifts; otherwise the sums are parked in LDS
// and one thread per halo pixel adds them in order. Input pixels the tile
// owns are copied into the spare x_{t-1} slot on the way (ping-pong: the slot
// being read is never written in the same step; no copy under caller-retained
// frames). Every workgroup then writes its block flags and appends its active
// blocks to the convolution's work list: a ballot and prefix count inside the
// tile, then one atomic per tile on the counter of its segment (eight
// segments, one per XCD's contiguous range of tiles, each counter on its own
// 128-byte line). The list is therefore unordered; the convolution needs no
// order. Blocks larger than a gate tile (b > 16) are the exception: the tiles
// OR per-tile flags, and compact_kernel (one workgroup, a kernel boundary
// after the gate) scans the flags in index order and writes the ordered list
// and its length. The ordered list of every other layer is built on demand,
// for introspection only.
#include "sc_device.h"
#include "sc_kernels.h"
#include "sc_stream.h"

#pragma clang fp contract(off)

namespace sc {

namespace {

// Per-chunk partial sums of the tile's halo: one item = one chunk of kChunk
// channels of one halo pixel (consecutive items = consecutive chunks, so the
// loads of a wave are contiguous). kItems items per thread have their loads in
// flight together. VEC = kChunk (vector path, c % kChunk == 0) or 1 (scalar).
template <typename T, int VEC>
__device__ void halo_partials(const GateParams& p, int n, int iy0, int ix0, int hh, int hw, int own_y0,
                              int own_y1, int own_x0, int own_x1, float* part) {
  // bf16 chunks stay packed (one uint4 per frame) until they are consumed
  constexpr bool kPacked = sizeof(T) == 2 && VEC == kChunk;
  constexpr int kItems = kPacked ? 8 : 4;
  const T* xt = static_cast<const T*>(p.x_t);
  const T* xp = static_cast<const T*>(p.x_prev);
  T* keep = static_cast<T*>(p.x_keep);
  const int c = p.c;
  const int nchk = (c + kChunk - 1) / kChunk;
  const int total = hh * hw * nchk;
  for (int base = 0; base < total; base += kGateThreads * kItems) {
    uint4 raw_t[kPacked ? kItems : 1], raw_p[kPacked ? kItems : 1];
    float vt[kPacked ? 1 : kItems][kChunk], vp[kPacked ? 1 : kItems][kChunk];
    size_t off[kItems];
    int slot[kItems], nel[kItems];
    bool in[kItems], own[kItems];
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
      const int idx = base + u * kGateThreads + threadIdx.x;
      const int px = idx / nchk, ch = idx - px * nchk;
      const int hy = px / hw, hx = px - hy * hw;
      const int y = iy0 + hy, x = ix0 + hx;
      in[u] = idx < total && y >= 0 && y < p.h && x >= 0 && x < p.w;
      slot[u] = idx < total ? px * p.stage_stride + ch : -1;
      nel[u] = min(kChunk, c - ch * kChunk);
      off[u] = in[u] ? ((size_t)(n * p.h + y) * p.w + x) * c + ch * kChunk : 0;
      own[u] = in[u] && keep && p.copy_in_halo && y >= own_y0 && y < own_y1 && x >= own_x0 && x < own_x1;
      // x_{t-1} under the step's translation (zero outside the frame)
      const long po = (in[u] && !p.no_prev) ? prev_off(p, n, y, x, ch * kChunk) : -1;
      if (kPacked) {
        raw_t[kPacked ? u : 0] = uint4{0u, 0u, 0u, 0u};
        raw_p[kPacked ? u : 0] = uint4{0u, 0u, 0u, 0u};
        if (in[u]) {
          raw_t[kPacked ? u : 0] = *reinterpret_cast<const uint4*>(xt + off[u]);
          if (po >= 0) raw_p[kPacked ? u : 0] = *reinterpret_cast<const uint4*>(xp + po);
        }
      } else if (in[u]) {
        const int uu = kPacked ? 0 : u;
        if (VEC == kChunk) {
          load_vec<T, kChunk>(xt, off[u], vt[uu]);
          if (po >= 0) load_vec<T, kChunk>(xp, (size_t)po, vp[uu]);
          else
            for (int j = 0; j < kChunk; ++j) vp[uu][j] = 0.0f;
        } else {
#pragma unroll
          for (int j = 0; j < kChunk; ++j) {
            vt[uu][j] = j < nel[u] ? Elem<T>::load1(xt, off[u] + j) : 0.0f;
            vp[uu][j] = (j < nel[u] && po >= 0) ? Elem<T>::load1(xp, (size_t)po + j) : 0.0f;
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
      if (slot[u] < 0) continue;
      float part_u = 0.0f;
      if (in[u]) {
        float r[kChunk];
        if (kPacked) {
          const uint4 a = raw_t[kPacked ? u : 0], b = raw_p[kPacked ? u : 0];
          const uint32_t wa[4] = {a.x, a.y, a.z, a.w}, wb[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            r[2 * e] = __fsub_rn(__uint_as_float(wa[e] << 16), __uint_as_float(wb[e] << 16));
            r[2 * e + 1] = __fsub_rn(__uint_as_float(wa[e] & 0xffff0000u), __uint_as_float(wb[e] & 0xffff0000u));
          }
        } else {
          const int uu = kPacked ? 0 : u;
#pragma unroll
          for (int j = 0; j < kChunk; ++j) r[j] = p.no_prev ? vt[uu][j] : __fsub_rn(vt[uu][j], vp[uu][j]);
        }
        if (VEC == kChunk) {
          part_u = chunk_sum<kChunk>(r, p.norm_p);
          if (own[u]) copy_vec<T, kChunk>(keep, xt, off[u]);
        } else {
#pragma unroll
          for (int j = 0; j < kChunk; ++j)
            if (j < nel[u]) part_u = add_rn(part_u, term(r[j], p.norm_p));
          if (own[u])
            for (int j = 0; j < nel[u]; ++j) keep[off[u] + j] = xt[off[u] + j];
        }
      }
      part[slot[u]] = part_u;
    }
  }
}

// Cache policy of the x_{t-1} copy: non-temporal (streamed past the caches),
// so that the frame being written does not evict the two frames the
// convolution reads next.
constexpr int kNonTemporal = 2;

// Halo of a norm gate with NC = 2, 4, 8 or 16 chunks per pixel (bf16 or fp32
// frames). Items are taken in flat order (consecutive threads, consecutive
// chunks), so a pixel's chunks sit in one aligned group of NC lanes: the
// group's first lane adds the chunk sums in ascending order through DPP row
// shifts and writes a[] of the pixel directly (no per-chunk staging in LDS, no
// second pass). Loads and stores go through buffer resources over image n
// (h * w * c * 4 < 2^31 bytes, checked by the host) with 32-bit byte offsets:
// items outside the frame (or, for x_{t-1}, outside the translated frame)
// load at an out-of-range offset and read zeros, and the x_t chunks of pixels
// the tile does not own are stored out of range (dropped), so every item
// issues the same loads and stores. A chunk is one 16-byte word per frame
// (bf16) or two (fp32). The non-temporal copy to the spare x_{t-1} slot
// follows the round's use.
template <typename T, int NC>
__device__ void halo_lane_sums(const GateParams& p, int n, int iy0, int ix0, int hh, int hw, int own_y0,
                               int own_y1, int own_x0, int own_x1, float* a_halo) {
  constexpr int kWords = sizeof(T) == 2 ? 1 : 2;  // 16-byte words per chunk and frame
  constexpr int kItems = 8 / kWords;
  constexpr int kLg = NC == 2 ? 1 : (NC == 4 ? 2 : (NC == 8 ? 3 : 4));
  const uint32_t img_bytes = (uint32_t)((size_t)p.h * p.w * p.c * sizeof(T));
  const size_t img = (size_t)n * p.h * p.w * p.c;
  const auto rt = frame_rsrc(static_cast<const T*>(p.x_t) + img, img_bytes);
  const auto rp = frame_rsrc(static_cast<const T*>(p.no_prev ? p.x_t : p.x_prev) + img, img_bytes);
  const bool keep_on = p.x_keep != nullptr && p.copy_in_halo;
  const auto rk = frame_rsrc(keep_on ? static_cast<T*>(p.x_keep) + img : nullptr, keep_on ? img_bytes : 0u);
  const int total = hh * hw * NC;
  const float inv_hw = 1.0f / (float)hw;
  const int wave0 = threadIdx.x & ~63;
  for (int base = 0; base < total; base += kGateThreads * kItems) {
    u32x4 vt[kItems][kWords], vp[kItems][kWords];
    uint32_t koff[kItems];
    // the thread index, opaque to loop-invariant code motion: the per-item
    // terms below are recomputed each round rather than held in registers
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
      const int idx = base + u * kGateThreads + tid;
      const int q = idx >> kLg, ch = idx & (NC - 1);
      const int hy = qdiv(q, inv_hw), hx = q - hy * hw;
      const int y = iy0 + hy, x = ix0 + hx;
      const bool in = idx < total && y >= 0 && y < p.h && x >= 0 && x < p.w;
      const bool own = in && keep_on && y >= own_y0 && y < own_y1 && x >= own_x0 && x < own_x1;
      const uint32_t off = (uint32_t)(((y * p.w + x) * p.c + ch * kChunk) * (int)sizeof(T));
      // x_{t-1} under the step's translation (zero outside the frame)
      const int yp = y - p.sy, xq = x - p.sx;
      const bool pin = in && !p.no_prev && yp >= 0 && yp < p.h && xq >= 0 && xq < p.w;
      const uint32_t po = (uint32_t)(((yp * p.w + xq) * p.c + ch * kChunk) * (int)sizeof(T));
      koff[u] = own ? off : kOutOfRange;
#pragma unroll
      for (int wd = 0; wd < kWords; ++wd) {
        vt[u][wd] = __builtin_amdgcn_raw_buffer_load_b128(rt, (in ? off : kOutOfRange) + 16 * wd, 0, 0);
        vp[u][wd] = __builtin_amdgcn_raw_buffer_load_b128(rp, (pin ? po : kOutOfRange) + 16 * wd, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
      if (base + u * kGateThreads + wave0 >= total) break;  // wave-uniform
      float sum = 0.0f;
      if constexpr (kWords == 1) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {  // channels 2e (low half) and 2e + 1 (high half)
          const uint32_t a = vt[u][0][e], b = vp[u][0][e];
          const float r0 = __fsub_rn(__uint_as_float(a << 16), __uint_as_float(b << 16));
          const float r1 = __fsub_rn(__uint_as_float(a & 0xffff0000u), __uint_as_float(b & 0xffff0000u));
          sum = add_rn(sum, term(r0, p.norm_p));
          sum = add_rn(sum, term(r1, p.norm_p));
        }
      } else {
#pragma unroll
        for (int j = 0; j < kChunk; ++j) {  // channel j: word j / 4, component j % 4
          const float r = __fsub_rn(__uint_as_float(vt[u][j >> 2][j & 3]), __uint_as_float(vp[u][j >> 2][j & 3]));
          sum = add_rn(sum, term(r, p.norm_p));
        }
      }
      const float acc = group_sum<NC>(sum);
      const int idx = base + u * kGateThreads + threadIdx.x;
      if (idx < total && (idx & (NC - 1)) == 0) a_halo[idx >> kLg] = acc;
    }
#pragma unroll
    for (int u = 0; u < kItems; ++u)
#pragma unroll
      for (int wd = 0; wd < kWords; ++wd)
        __builtin_amdgcn_raw_buffer_store_b128(vt[u][wd], rk, koff[u] + 16 * wd, 0, kNonTemporal);
  }
}

// Halo of a norm gate with fewer than 8 channels (one partial chunk per
// pixel): one item per halo pixel, its c channels loaded element by element
// through buffer resources (every load issued: channels past c and pixels
// outside the frame read zeros at an out-of-range offset), the statistic
// summed in channel order (the canonical single-chunk order) straight into
// a[]; owned pixels copied element by element the same way (other items store
// out of range).
template <typename T>
__device__ void halo_pixels(const GateParams& p, int n, int iy0, int ix0, int hh, int hw, int own_y0,
                            int own_y1, int own_x0, int own_x1, float* a_halo) {
  constexpr int kItems = 4;
  constexpr int E = (int)sizeof(T);
  const uint32_t img_bytes = (uint32_t)((size_t)p.h * p.w * p.c * E);
  const size_t img = (size_t)n * p.h * p.w * p.c;
  const auto rt = frame_rsrc(static_cast<const T*>(p.x_t) + img, img_bytes);
  const auto rp = frame_rsrc(static_cast<const T*>(p.no_prev ? p.x_t : p.x_prev) + img, img_bytes);
  const bool keep_on = p.x_keep != nullptr && p.copy_in_halo;
  const auto rk = frame_rsrc(keep_on ? static_cast<T*>(p.x_keep) + img : nullptr, keep_on ? img_bytes : 0u);
  const int total = hh * hw;
  const float inv_hw = 1.0f / (float)hw;
  for (int base = 0; base < total; base += kGateThreads * kItems) {
    uint32_t vt[kItems][kChunk], vp[kItems][kChunk];
    uint32_t off[kItems], po[kItems], ko[kItems];
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
      const int q = base + u * kGateThreads + threadIdx.x;
      const int hy = qdiv(q, inv_hw), hx = q - hy * hw;
      const int y = iy0 + hy, x = ix0 + hx;
      const bool in = q < total && y >= 0 && y < p.h && x >= 0 && x < p.w;
      const bool own = in && keep_on && y >= own_y0 && y < own_y1 && x >= own_x0 && x < own_x1;
      const int yp = y - p.sy, xq = x - p.sx;
      const bool pin = in && !p.no_prev && yp >= 0 && yp < p.h && xq >= 0 && xq < p.w;
      off[u] = in ? (uint32_t)((y * p.w + x) * p.c * E) : kOutOfRange;
      po[u] = pin ? (uint32_t)((yp * p.w + xq) * p.c * E) : kOutOfRange;
      ko[u] = own ? off[u] : kOutOfRange;
#pragma unroll
      for (int j = 0; j < kChunk; ++j) {
        const bool ch = j < p.c;
        if constexpr (E == 2) {
          vt[u][j] = __builtin_amdgcn_raw_buffer_load_b16(rt, ch ? off[u] + 2 * j : kOutOfRange, 0, 0);
          vp[u][j] = __builtin_amdgcn_raw_buffer_load_b16(rp, ch ? po[u] + 2 * j : kOutOfRange, 0, 0);
        } else {
          vt[u][j] = __builtin_amdgcn_raw_buffer_load_b32(rt, ch ? off[u] + 4 * j : kOutOfRange, 0, 0);
          vp[u][j] = __builtin_amdgcn_raw_buffer_load_b32(rp, ch ? po[u] + 4 * j : kOutOfRange, 0, 0);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
      const int q = base + u * kGateThreads + threadIdx.x;
      float sum = 0.0f;
#pragma unroll
      for (int j = 0; j < kChunk; ++j) {
        if (j >= p.c) continue;
        const float a = E == 2 ? __uint_as_float(vt[u][j] << 16) : __uint_as_float(vt[u][j]);
        const float b = E == 2 ? __uint_as_float(vp[u][j] << 16) : __uint_as_float(vp[u][j]);
        sum = add_rn(sum, term(__fsub_rn(a, b), p.norm_p));
      }
      if (q < total) a_halo[q] = sum;
    }
#pragma unroll
    for (int u = 0; u < kItems; ++u)
#pragma unroll
      for (int j = 0; j < kChunk; ++j) {
        const uint32_t o = (ko[u] == kOutOfRange || j >= p.c) ? kOutOfRange : ko[u] + E * j;
        if constexpr (E == 2) __builtin_amdgcn_raw_buffer_store_b16((uint16_t)vt[u][j], rk, o, 0, 0);
        else __builtin_amdgcn_raw_buffer_store_b32(vt[u][j], rk, o, 0, 0);
      }
  }
}

// Learned gate (Eq. 8 at inference) with NC = 2, 4, 8 or 16 chunks per pixel:
// the items of halo_lane_sums (one 8-channel chunk of one halo pixel per lane,
// consecutive lanes holding consecutive chunks of a pixel, kItems items with
// their loads in flight together), each forming the K2 per-tap chunk terms
// sum_j phi[tap][c0 + j] * r[c0 + j] in ascending order from +0. The terms of
// up to kLearnTapGroup taps go to the wave's exchange area in LDS, [pixel]
// [tap][chunk]; lane l of a pixel's group then reads the NC terms of tap
// l (l + NC, ...) and adds them in ascending chunk order from +0, the
// canonical order, and writes a[q, tap]. Every lane reduces a different tap,
// where a lane-shift chain per tap would run in all NC lanes for one result.
// For kernels of up to 3 x 3 a lane holds its phi chunk of every tap in
// registers, so the tap loop's only LDS traffic is the exchange (reading phi
// from LDS per tap as well took the blob-sized gate from 0.29 to 0.75 ms).
// Owned pixels are copied to the spare x_{t-1} slot on the way. phi: staged
// in LDS, or in memory (each call site inlines its own copy).
template <typename T, int NC, int KL>
__device__ __forceinline__ void learned_lane_sums(const GateParams& p, int n, int iy0, int ix0, int hh, int hw, int own_y0,
                                  int own_y1, int own_x0, int own_x1, float* a2, const float* phi, float* xch) {
  constexpr int K2 = KL * KL;
  constexpr int TG = K2 < kLearnTapGroup ? K2 : kLearnTapGroup;
  constexpr int kWords = sizeof(T) == 2 ? 1 : 2;  // 16-byte words per chunk and frame
  constexpr int kItems = 4 / kWords;
  constexpr int kLg = NC == 2 ? 1 : (NC == 4 ? 2 : (NC == 8 ? 3 : 4));
  const uint32_t img_bytes = (uint32_t)((size_t)p.h * p.w * p.c * sizeof(T));
  const size_t img = (size_t)n * p.h * p.w * p.c;
  const auto rt = frame_rsrc(static_cast<const T*>(p.x_t) + img, img_bytes);
  const auto rp = frame_rsrc(static_cast<const T*>(p.no_prev ? p.x_t : p.x_prev) + img, img_bytes);
  const bool keep_on = p.x_keep != nullptr && p.copy_in_halo;
  const auto rk = frame_rsrc(keep_on ? static_cast<T*>(p.x_keep) + img : nullptr, keep_on ? img_bytes : 0u);
  const int total = hh * hw * NC;
  const float inv_hw = 1.0f / (float)hw;
  const int wave0 = threadIdx.x & ~63;
  // a thread's chunk is the same for every item (NC divides the item stride)
  const int ch = threadIdx.x & (NC - 1);
  const float* ph = phi + ch * kChunk;
  // this lane's pixel group in the wave's exchange area: TG taps x NC chunks
  float* xg = xch + wave0 * TG + ((threadIdx.x & 63) >> kLg) * (TG * NC);
  // kernels of up to 3 x 3: this lane's phi chunk of every tap in registers
  // (loaded once), so that the tap loop reads LDS only for the exchange
  constexpr bool kRegPhi = K2 <= 9;
  float fr[kRegPhi ? K2 : 1][kChunk];
  if constexpr (kRegPhi) {
#pragma unroll
    for (int t = 0; t < K2; ++t) {
      const float4 f0 = *reinterpret_cast<const float4*>(ph + t * p.c);
      const float4 f1 = *reinterpret_cast<const float4*>(ph + t * p.c + 4);
      fr[t][0] = f0.x; fr[t][1] = f0.y; fr[t][2] = f0.z; fr[t][3] = f0.w;
      fr[t][4] = f1.x; fr[t][5] = f1.y; fr[t][6] = f1.z; fr[t][7] = f1.w;
    }
  }
  for (int base = 0; base < total; base += kGateThreads * kItems) {
    u32x4 vt[kItems][kWords], vp[kItems][kWords];
    uint32_t koff[kItems];
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
      const int idx = base + u * kGateThreads + threadIdx.x;
      const int q = idx >> kLg;
      const int hy = qdiv(q, inv_hw), hx = q - hy * hw;
      const int y = iy0 + hy, x = ix0 + hx;
      const bool in = idx < total && y >= 0 && y < p.h && x >= 0 && x < p.w;
      const bool own = in && keep_on && y >= own_y0 && y < own_y1 && x >= own_x0 && x < own_x1;
      const uint32_t off = (uint32_t)(((y * p.w + x) * p.c + ch * kChunk) * (int)sizeof(T));
      // x_{t-1} under the step's translation (zero outside the frame)
      const int yp = y - p.sy, xq = x - p.sx;
      const bool pin = in && !p.no_prev && yp >= 0 && yp < p.h && xq >= 0 && xq < p.w;
      const uint32_t po = (uint32_t)(((yp * p.w + xq) * p.c + ch * kChunk) * (int)sizeof(T));
      koff[u] = own ? off : kOutOfRange;
#pragma unroll
      for (int wd = 0; wd < kWords; ++wd) {
        vt[u][wd] = __builtin_amdgcn_raw_buffer_load_b128(rt, (in ? off : kOutOfRange) + 16 * wd, 0, 0);
        vp[u][wd] = __builtin_amdgcn_raw_buffer_load_b128(rp, (pin ? po : kOutOfRange) + 16 * wd, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
      if (base + u * kGateThreads + wave0 >= total) break;  // wave-uniform
      float r[kChunk];
      if constexpr (kWords == 1) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {  // channels 2e (low half) and 2e + 1 (high half)
          const uint32_t a = vt[u][0][e], b = vp[u][0][e];
          r[2 * e] = __fsub_rn(__uint_as_float(a << 16), __uint_as_float(b << 16));
          r[2 * e + 1] = __fsub_rn(__uint_as_float(a & 0xffff0000u), __uint_as_float(b & 0xffff0000u));
        }
      } else {
#pragma unroll
        for (int j = 0; j < kChunk; ++j)
          r[j] = __fsub_rn(__uint_as_float(vt[u][j >> 2][j & 3]), __uint_as_float(vp[u][j >> 2][j & 3]));
      }
      const int idx = base + u * kGateThreads + threadIdx.x;
      const int q = idx >> kLg;
      const bool pix_ok = idx < total;  // (total is a multiple of NC: the whole group agrees)
#pragma unroll
      for (int t0 = 0; t0 < K2; t0 += TG) {
        const int tg = K2 - t0 < TG ? K2 - t0 : TG;
#pragma unroll
        for (int tl = 0; tl < TG; ++tl) {
          if (tl < tg) {
            float f[kChunk];
            if constexpr (kRegPhi) {
#pragma unroll
              for (int j = 0; j < kChunk; ++j) f[j] = fr[kRegPhi ? t0 + tl : 0][j];
            } else {
              const float4 f0 = *reinterpret_cast<const float4*>(ph + (t0 + tl) * p.c);
              const float4 f1 = *reinterpret_cast<const float4*>(ph + (t0 + tl) * p.c + 4);
              f[0] = f0.x; f[1] = f0.y; f[2] = f0.z; f[3] = f0.w;
              f[4] = f1.x; f[5] = f1.y; f[6] = f1.z; f[7] = f1.w;
            }
            float part = 0.0f;
#pragma unroll
            for (int j = 0; j < kChunk; ++j) part = add_rn(part, mul_rn(f[j], r[j]));
            xg[tl * NC + ch] = part;
          }
        }
        // the group's terms are written by lanes of this wave: LDS serves a
        // wave's accesses in order, so only the compiler must keep them so
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront", "local");
#pragma unroll
        for (int rr = 0; rr < TG; rr += NC) {
          const int tl = rr + ch;
          if (tl < tg) {
            float v[NC];
            if constexpr (NC % 4 == 0) {
#pragma unroll
              for (int i4 = 0; i4 < NC; i4 += 4) {
                const float4 w4 = *reinterpret_cast<const float4*>(xg + tl * NC + i4);
                v[i4] = w4.x;
                v[i4 + 1] = w4.y;
                v[i4 + 2] = w4.z;
                v[i4 + 3] = w4.w;
              }
            } else {
              const float2 w2 = *reinterpret_cast<const float2*>(xg + tl * NC);
              v[0] = w2.x;
              v[1] = w2.y;
            }
            float acc = add_rn(0.0f, v[0]);
#pragma unroll
            for (int i = 1; i < NC; ++i) acc = add_rn(acc, v[i]);
            if (pix_ok) a2[q * K2 + t0 + tl] = acc;
          }
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront", "local");
      }
    }
#pragma unroll
    for (int u = 0; u < kItems; ++u)
#pragma unroll
      for (int wd = 0; wd < kWords; ++wd)
        __builtin_amdgcn_raw_buffer_store_b128(vt[u][wd], rk, koff[u] + 16 * wd, 0, kNonTemporal);
  }
}

// Learned gate (Eq. 8 at inference): one thread per halo pixel forms, for
// every tap (kh, kw), a[q, tap] = sum_c phi[tap][c] * r[q, c] in the canonical
// chunked order (8 channels ascending within a chunk from +0, chunk sums
// ascending from +0, one rounding per multiply and per add), and copies the
// pixel into the spare x_{t-1} slot if the tile owns it. phi is [tap][c]
// (staged in LDS when it fits). VEC = 8: channel chunks move as 16-byte
// vectors (c % 8 == 0).
template <typename T, int VEC, int KL>
__device__ void learned_halo(const GateParams& p, int n, int iy0, int ix0, int hh, int hw, int own_y0,
                             int own_y1, int own_x0, int own_x1, float* a2, const float* phi) {
  constexpr int K2 = KL * KL;
  const T* xt = static_cast<const T*>(p.x_t);
  const T* xp = static_cast<const T*>(p.x_prev);
  T* keep = static_cast<T*>(p.x_keep);
  const int c = p.c;
  for (int q = threadIdx.x; q < hh * hw; q += kGateThreads) {
    const int hy = q / hw, hx = q - hy * hw;
    const int y = iy0 + hy, x = ix0 + hx;
    const bool in = y >= 0 && y < p.h && x >= 0 && x < p.w;
    const bool own = in && keep && p.copy_in_halo && y >= own_y0 && y < own_y1 && x >= own_x0 && x < own_x1;
    float acc[K2];
#pragma unroll
    for (int t = 0; t < K2; ++t) acc[t] = 0.0f;
    if (in) {
      const size_t base = ((size_t)(n * p.h + y) * p.w + x) * c;
      const long pbase = p.no_prev ? -1 : prev_off(p, n, y, x, 0);  // translated x_{t-1}
      for (int c0 = 0; c0 < c; c0 += kChunk) {
        const int nel = min(kChunk, c - c0);
        float r[kChunk];
        if (VEC == kChunk) {
          float vt[kChunk], vp[kChunk];
          load_vec<T, kChunk>(xt, base + c0, vt);
          if (pbase >= 0) load_vec<T, kChunk>(xp, (size_t)pbase + c0, vp);
#pragma unroll
          for (int j = 0; j < kChunk; ++j) r[j] = pbase < 0 ? vt[j] : __fsub_rn(vt[j], vp[j]);
          if (own) copy_vec<T, kChunk>(keep, xt, base + c0);
        } else {
#pragma unroll
          for (int j = 0; j < kChunk; ++j) {
            const float vt = j < nel ? Elem<T>::load1(xt, base + c0 + j) : 0.0f;
            const float vp = (j < nel && pbase >= 0) ? Elem<T>::load1(xp, (size_t)pbase + c0 + j) : 0.0f;
            r[j] = __fsub_rn(vt, vp);
            if (own && j < nel) keep[base + c0 + j] = xt[base + c0 + j];
          }
        }
#pragma unroll
        for (int t = 0; t < K2; ++t) {
          const float* ph = phi + t * c + c0;
          float part = 0.0f;
          if (VEC == kChunk) {
            const float4 f0 = *reinterpret_cast<const float4*>(ph);
            const float4 f1 = *reinterpret_cast<const float4*>(ph + 4);
            const float f[kChunk] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
#pragma unroll
            for (int j = 0; j < kChunk; ++j) part = add_rn(part, mul_rn(f[j], r[j]));
          } else {
            for (int j = 0; j < nel; ++j) part = add_rn(part, mul_rn(ph[j], r[j]));
          }
          acc[t] = add_rn(acc[t], part);
        }
      }
    }
#pragma unroll
    for (int t = 0; t < K2; ++t) a2[q * K2 + t] = acc[t];
  }
}

// The gate of one tile of output sites (this workgroup's tile): residual,
// statistic, threshold, block flags (and the work-list appends when p.wlist is
// set). Returns the tile's block flags in LDS.
// KL: learned gate kernel size (0 = norm gate). NC > 1: norm gate with NC
// chunks per pixel, chunk sums combined in lane groups (halo_lane_sums); NC =
// 1: norm gate with fewer than 8 channels, one item per pixel (halo_pixels).
template <typename T, int VEC, int KL, int NC>
__device__ __forceinline__ const uint32_t* gate_tile(const GateParams& p, float* lds) {
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
  // input pixels this tile owns (copied to the spare x_{t-1} slot)
  const int own_y0 = oy0 * s, own_x0 = ox0 * s;
  const int own_y1 = (ty == p.tiles_y - 1) ? p.h : min(p.h, (oy0 + p.ts) * s);
  const int own_x1 = (tx == p.tiles_x - 1) ? p.w : min(p.w, (ox0 + p.ts) * s);

  float* a_halo = lds;                 // hh * hw
  float* part = lds + p.halo_floats;   // hh * hw * stage_stride chunk sums
  const int nchk = (p.c + kChunk - 1) / kChunk;

  const int tb_w = p.ts / p.block;
  const int nblk_y = (oh + p.block - 1) / p.block, nblk_x = (ow + p.block - 1) / p.block;
  for (int i = threadIdx.x; i < kMaxTileBlocks; i += kGateThreads) blk_flag[i] = 0u;

  if (p.up_mask) {
    // chained input: the residual is zero outside the upstream layer's active
    // blocks; a tile whose input region meets none of them has a zero statistic
    // at every site (gate off) and skips its loads
    const int y0 = max(iy0, 0), y1 = min(iy0 + hh, p.h), x0 = max(ix0, 0), x1 = min(ix0 + hw, p.w);
    const int by0 = y0 / p.up_block, by1 = (y1 - 1) / p.up_block;
    const int bx0 = x0 / p.up_block, bx1 = (x1 - 1) / p.up_block;
    const int nbx = bx1 - bx0 + 1, cnt = (by1 - by0 + 1) * nbx;
    int any = 0;
    for (int i = threadIdx.x; i < cnt; i += kGateThreads) {
      const int by = by0 + i / nbx, bx = bx0 + i % nbx;
      any |= p.up_mask[((size_t)n * p.up_hb + by) * p.up_wb + bx] != 0;
    }
    if (!__syncthreads_or(any)) {
      if (p.keep_stats)
        for (int q = threadIdx.x; q < oh * ow; q += kGateThreads) {
          const int ly = q / ow, lx = q - ly * ow;
          const size_t o = ((size_t)n * p.h_out + oy0 + ly) * p.w_out + ox0 + lx;
          p.stat[o] = 0.0f;
          p.site_mask[o] = 0;
        }
      if (p.split_blocks) {
        if (threadIdx.x == 0) p.tile_flags[tile] = 0;
        return blk_flag;
      }
      const int bi0 = oy0 / p.block, bj0 = ox0 / p.block;
      for (int i = threadIdx.x; i < nblk_y * nblk_x; i += kGateThreads) {
        const int by = i / nblk_x, bx = i - by * nblk_x;
        p.block_mask[((size_t)n * p.hb + bi0 + by) * p.wb + bj0 + bx] = 0;
      }
      return blk_flag;
    }
  }

  if constexpr (NC == 1 && KL == 0) {
    halo_pixels<T>(p, n, iy0, ix0, hh, hw, own_y0, own_y1, own_x0, own_x1, a_halo);
  } else if constexpr (NC > 0 && KL == 0) {
    halo_lane_sums<T, NC>(p, n, iy0, ix0, hh, hw, own_y0, own_y1, own_x0, own_x1, a_halo);
  } else if constexpr (KL == 0) {
    halo_partials<T, VEC>(p, n, iy0, ix0, hh, hw, own_y0, own_y1, own_x0, own_x1, part);
    __syncthreads();
    for (int q = threadIdx.x; q < hh * hw; q += kGateThreads) {
      const int hy = q / hw, hx = q - hy * hw;
      const int y = iy0 + hy, x = ix0 + hx;
      float a = 0.0f;
      if (y >= 0 && y < p.h && x >= 0 && x < p.w) {
        const float* pp = part + q * p.stage_stride;
        for (int ch = 0; ch < nchk; ++ch) a = add_rn(a, pp[ch]);
      }
      a_halo[q] = a;
    }
  } else {
    // stage phi ([tap][c]) in LDS when it fits, then the per-pixel, per-tap gate terms
    const float* phi = p.phi;
    if (p.phi_off >= 0) {
      float* staged = lds + p.phi_off;
      for (int i = threadIdx.x; i < KL * KL * p.c; i += kGateThreads) staged[i] = p.phi[i];
      __syncthreads();
      phi = staged;
    }
    if constexpr (NC > 1) {
      if (p.phi_off >= 0)
        learned_lane_sums<T, NC, KL>(p, n, iy0, ix0, hh, hw, own_y0, own_y1, own_x0, own_x1, lds,
                                     lds + p.phi_off, lds + p.tr_off);
      else
        learned_lane_sums<T, NC, KL>(p, n, iy0, ix0, hh, hw, own_y0, own_y1, own_x0, own_x1, lds, p.phi,
                                     lds + p.tr_off);
    } else
      learned_halo<T, VEC, KL>(p, n, iy0, ix0, hh, hw, own_y0, own_y1, own_x0, own_x1, lds, phi);
  }

  if (!p.copy_in_halo && p.x_keep) {
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
  __syncthreads();

  // support statistic, threshold, block flags
  for (int q = threadIdx.x; q < oh * ow; q += kGateThreads) {
    const int ly = q / ow, lx = q - ly * ow;
    float sv;
    if constexpr (KL > 0) {
      // gate score: in-frame taps in row-major order, then the bias; on when > 0
      sv = 0.0f;
      for (int kh = 0; kh < KL; ++kh) {
        const int hy = ly * s + kh, y = iy0 + hy;
        if (y < 0 || y >= p.h) continue;
        for (int kw = 0; kw < KL; ++kw) {
          const int hx = lx * s + kw, x = ix0 + hx;
          if (x < 0 || x >= p.w) continue;
          sv = add_rn(sv, lds[(hy * hw + hx) * (KL * KL) + kh * KL + kw]);
        }
      }
      sv = add_rn(sv, p.gate_bias);
      const bool on = p.reference || p.force_dense || sv > 0.0f || (sv != sv) ||
                      line_exposed(oy0 + ly, p.h_out, p.h, p.k, p.stride, p.pad, p.sy) ||
                      line_exposed(ox0 + lx, p.w_out, p.w, p.k, p.stride, p.pad, p.sx);
      if (p.keep_stats) {
        const size_t o = ((size_t)n * p.h_out + oy0 + ly) * p.w_out + ox0 + lx;
        p.stat[o] = sv;
        p.site_mask[o] = on ? 1 : 0;
      }
      if (on) blk_flag[(ly / p.block) * tb_w + lx / p.block] = 1u;
      continue;
    }
    if (p.support == 0) {
      sv = 0.0f;
      const float* base = a_halo + (ly * s) * hw + lx * s;
      for (int kh = 0; kh < k; ++kh)
        for (int kw = 0; kw < k; ++kw) sv = add_rn(sv, base[kh * hw + kw]);
    } else {
      sv = a_halo[(ly * s + p.pad) * hw + lx * s + p.pad];
    }
    const bool on = p.reference || p.force_dense || ((double)sv * p.wnorm > p.thr) || (sv != sv) ||
                    line_exposed(oy0 + ly, p.h_out, p.h, p.k, p.stride, p.pad, p.sy) ||
                    line_exposed(ox0 + lx, p.w_out, p.w, p.k, p.stride, p.pad, p.sx);
    if (p.keep_stats) {
      const size_t o = ((size_t)n * p.h_out + oy0 + ly) * p.w_out + ox0 + lx;
      p.stat[o] = sv;
      p.site_mask[o] = on ? 1 : 0;
    }
    if (on) blk_flag[(ly / p.block) * tb_w + lx / p.block] = 1u;
  }
  __syncthreads();

  if (p.split_blocks) {
    // the tile is part of one block: one flag per tile, OR-ed per block by the compaction
    if (threadIdx.x == 0) p.tile_flags[tile] = (uint8_t)(blk_flag[0] != 0u);
    return blk_flag;
  }
  const int bi0 = oy0 / p.block, bj0 = ox0 / p.block;
  for (int i = threadIdx.x; i < nblk_y * nblk_x; i += kGateThreads) {
    const int by = i / nblk_x, bx = i - by * nblk_x;
    p.block_mask[((size_t)n * p.hb + bi0 + by) * p.wb + bj0 + bx] = (uint8_t)blk_flag[by * tb_w + bx];
  }
  if (p.wlist) {
    // append the tile's active blocks to the (unordered) work list of the
    // convolution: one thread per block (<= 256), wave ballots, one atomic
    __shared__ uint32_t wave_cnt[kGateThreads / 64];
    __shared__ uint32_t wl_base;
    const int i = threadIdx.x, lane = i & 63, wv = i >> 6;
    const int by = i / nblk_x, bx = i - by * nblk_x;
    const bool act = i < nblk_y * nblk_x && blk_flag[by * tb_w + bx] != 0u;
    const unsigned long long m = __ballot(act);
    if (lane == 0) wave_cnt[wv] = (uint32_t)__popcll(m);
    __syncthreads();
    if (i == 0) {
      uint32_t tot = 0;
      for (int w = 0; w < kGateThreads / 64; ++w) tot += wave_cnt[w];
      // segment of this workgroup's XCD (xcd_tile hands XCD b % 8 a
      // contiguous tile range starting at tile `first`)
      const int x = blockIdx.x & 7, per = gridDim.x >> 3, rem = gridDim.x & 7;
      const uint32_t first = (uint32_t)(x * per + min(x, rem));
      wl_base = tot ? first * (uint32_t)p.seg_cap + atomicAdd(p.wctr + x * kSegStride, tot) : 0u;
    }
    __syncthreads();
    if (act) {
      uint32_t off = wl_base + (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
      for (int w = 0; w < wv; ++w) off += wave_cnt[w];
      p.wlist[off] = (uint32_t)(((size_t)n * p.hb + bi0 + by) * p.wb + bj0 + bx);
    }
  }
  return blk_flag;
}

template <typename T, int VEC, int KL, int NC>
__global__ void __launch_bounds__(kGateThreads) gate_kernel(GateParams p) {
  extern __shared__ float lds[];
  gate_tile<T, VEC, KL, NC>(p, lds);
}

// Ordered compaction (one workgroup of kScanThreads): each thread takes a
// contiguous run of 16-byte words of block flags (bytes 0/1, the buffer is
// zero-padded to whole words), counts them, the workgroup scans the counts,
// and every thread writes the indices of its active blocks in ascending order.
constexpr int kScanThreads = 1024;

__global__ void __launch_bounds__(kScanThreads) compact_kernel(uint8_t* block_mask, int nb,
                                                               uint32_t* list, uint32_t* counters,
                                                               const uint8_t* tile_flags, int n_img, int hb,
                                                               int wb, int bt, int tiles_y, int tiles_x) {
  __shared__ uint32_t wave_sum[kScanThreads / 64];
  if (tile_flags) {
    // blocks larger than the gate tiles: block flag = OR of its bt x bt tiles
    for (int blk = threadIdx.x; blk < nb; blk += kScanThreads) {
      const int img = blk / (hb * wb), rem = blk - img * hb * wb;
      const int bi = rem / wb, bj = rem - bi * wb;
      uint8_t f = 0;
      for (int dy = 0; dy < bt; ++dy) {
        const int ty = bi * bt + dy;
        if (ty >= tiles_y) break;
        for (int dx = 0; dx < bt; ++dx) {
          const int tx = bj * bt + dx;
          if (tx >= tiles_x) break;
          f |= tile_flags[((size_t)img * tiles_y + ty) * tiles_x + tx];
        }
      }
      block_mask[blk] = f ? 1 : 0;
    }
    __syncthreads();
  }
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
  const int nchk = (p.c + kChunk - 1) / kChunk;
  if (p.lane_sum && p.learned) {
    // learned gate over lane groups (c = 16, 32, 64 or 128, c % 8 == 0)
    if constexpr (VEC == kChunk) {
      if ((long)p.h * p.w * p.c * 4 >= (1L << 31)) return hipErrorInvalidValue;
#define SC_LG(nc)                                                                                                \
  switch (p.learned) {                                                                                           \
    case 1: hipLaunchKernelGGL((gate_kernel<T, VEC, 1, nc>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p); break; \
    case 3: hipLaunchKernelGGL((gate_kernel<T, VEC, 3, nc>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p); break; \
    case 5: hipLaunchKernelGGL((gate_kernel<T, VEC, 5, nc>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p); break; \
    case 7: hipLaunchKernelGGL((gate_kernel<T, VEC, 7, nc>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p); break; \
    default: return hipErrorInvalidValue;                                                                        \
  }
      if (nchk == 16) { SC_LG(16) }
      else if (nchk == 8) { SC_LG(8) }
      else if (nchk == 4) { SC_LG(4) }
      else if (nchk == 2) { SC_LG(2) }
      else return hipErrorInvalidValue;
#undef SC_LG
      return hipGetLastError();
    }
    return hipErrorInvalidValue;
  }
  if (p.lane_sum) {
    // the host sized the LDS without chunk-sum staging: only these shapes
    if (p.learned != 0 || (long)p.h * p.w * p.c * 4 >= (1L << 31)) return hipErrorInvalidValue;
    if constexpr (VEC == kChunk) {
      if (nchk == 16) hipLaunchKernelGGL((gate_kernel<T, VEC, 0, 16>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p);
      else if (nchk == 8) hipLaunchKernelGGL((gate_kernel<T, VEC, 0, 8>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p);
      else if (nchk == 4) hipLaunchKernelGGL((gate_kernel<T, VEC, 0, 4>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p);
      else if (nchk == 2) hipLaunchKernelGGL((gate_kernel<T, VEC, 0, 2>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p);
      else return hipErrorInvalidValue;
    } else {
      if (p.c >= kChunk) return hipErrorInvalidValue;
      hipLaunchKernelGGL((gate_kernel<T, VEC, 0, 1>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p);
    }
    return hipGetLastError();
  }
  switch (p.learned) {
    case 0: hipLaunchKernelGGL((gate_kernel<T, VEC, 0, 0>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p); break;
    case 1: hipLaunchKernelGGL((gate_kernel<T, VEC, 1, 0>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p); break;
    case 3: hipLaunchKernelGGL((gate_kernel<T, VEC, 3, 0>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p); break;
    case 5: hipLaunchKernelGGL((gate_kernel<T, VEC, 5, 0>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p); break;
    case 7: hipLaunchKernelGGL((gate_kernel<T, VEC, 7, 0>), dim3(grid), dim3(kGateThreads), lds_bytes, st, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Pack the learned gate's weights from [c][kh][kw] (a one-output-channel OIHW
// tensor) to [tap][c].
__global__ void pack_phi_kernel(const float* src, float* dst, int c, int k2) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < c * k2) {
    const int ch = i / k2, t = i - ch * k2;
    dst[t * c + ch] = src[i];
  }
}

hipError_t launch_pack_phi(const float* src, float* dst, int c, int k, hipStream_t st) {
  const int total = c * k * k;
  hipLaunchKernelGGL(pack_phi_kernel, dim3((total + 255) / 256), dim3(256), 0, st, src, dst, c, k * k);
  return hipGetLastError();
}

hipError_t launch_compact(uint8_t* block_mask, int nb, uint32_t* list, uint32_t* counters,
                          const uint8_t* tile_flags, int n, int hb, int wb, int bt, int tiles_y,
                          int tiles_x, hipStream_t st) {
  hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(kScanThreads), 0, st, block_mask, nb, list, counters,
                     tile_flags, n, hb, wb, bt, tiles_y, tiles_x);
  return hipGetLastError();
}

hipError_t launch_gate(const GateParams& p, int dtype, int vec, int grid, size_t lds_bytes,
                       hipStream_t st) {
  if (dtype == 0) {
    if (vec == kChunk) return launch_gate_t<float, kChunk>(p, grid, lds_bytes, st);
    return launch_gate_t<float, 1>(p, grid, lds_bytes, st);
  }
  if (vec == kChunk) return launch_gate_t<uint16_t, kChunk>(p, grid, lds_bytes, st);
  return launch_gate_t<uint16_t, 1>(p, grid, lds_bytes, st);
}

}  // namespace sc
