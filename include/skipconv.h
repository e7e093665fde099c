/*
 * skipconv.h -- C ABI of the MI355X (gfx950) streaming Skip-Convolution layer.
 *
 * The layer follows Habibian et al., "Skip-Convolutions for Efficient Video
 * Processing" (CVPR 2021):
 *   Eq. 2  r_t = x_t - x_{t-1}; by linearity z_t = z_{t-1} + w * r_t.
 *   Eq. 3  z~_t = z~_{t-1} + g(r_t) (.) (w * r_t): the convolution runs only at
 *          output locations where the gate is on; elsewhere z~_{t-1} is kept.
 *   Eq. 5  Input-Norm gate g = round(sigmoid(||r_t|| - eps)), the norm taken
 *          over the kernel support (all input channels x k x k) of each output.
 *   Eq. 7  Output-Norm gate g = round(sigmoid(||w|| ||r_t|| - eps)), ||w|| the
 *          norm of the whole weight tensor (Young's inequality, Eq. 6, makes
 *          the product a bound on the norm of the skipped update).
 *   Eq. 8  Gumbel gate at inference g = round(sigmoid(f(r_t; phi))), f a
 *          convolution with one output channel and the layer's geometry.
 *   Sec. 3.2.2 structured gates: max-pool the gate with kernel = stride = b,
 *          then nearest upsample, so the mask is constant on b x b blocks.
 *   Sec. 3.1 the first frame (and each reference frame after a reset, the
 *          reset period of Table 4) is computed over the whole frame.
 *
 * Conventions shared by every call:
 *   - Tensors are NHWC, densely packed. Inputs x are in the layer dtype (fp32,
 *     or bf16 as raw 16-bit patterns). The output state z is fp32.
 *   - Weights are OIHW: c_out x (c_in/groups) x k x k, in the layer dtype.
 *   - "device pointer" means memory of the current HIP device; "host pointer"
 *     means ordinary host memory. The library never takes ownership of a
 *     caller pointer.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Work is enqueued on it without host synchronisation unless a call says
 *     otherwise.
 *   - Every call returns SKIPCONV_OK (0) or a negative skipconv_status. No C++
 *     exception crosses this boundary. A failed call leaves the handle as it
 *     was, except after SKIPCONV_E_HIP from enqueued work, after which the
 *     state is undefined until skipconv_reset.
 *   - A handle is not thread-safe; distinct handles are independent.
 */
#ifndef SKIPCONV_H
#define SKIPCONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum skipconv_status {
  SKIPCONV_OK = 0,
  SKIPCONV_E_INVALID_ARG = -1,  /* bad descriptor field, NULL pointer, bad size */
  SKIPCONV_E_UNSUPPORTED = -2,  /* valid but not implemented (e.g. 1 < groups < c_in) */
  SKIPCONV_E_OOM = -3,          /* device allocation failed */
  SKIPCONV_E_HIP = -4,          /* a HIP runtime call or kernel launch failed */
  SKIPCONV_E_STATE = -5,        /* call not allowed in the handle's current state */
  SKIPCONV_E_SMALL_BUFFER = -6  /* caller buffer smaller than required */
} skipconv_status;

enum { SKIPCONV_F32 = 0, SKIPCONV_BF16 = 1 };

/* Gate support (Eq. 5): RF = norm over each output's whole kernel support
 * (c_in x k x k, zero padding contributes nothing); CENTRE = norm over the
 * single input pixel under the output (o * stride). */
enum { SKIPCONV_SUPPORT_RF = 0, SKIPCONV_SUPPORT_CENTRE = 1 };

/* Gate function (Sec. 3.2.1). Both compare in the power of the statistic:
 *   INPUT_NORM   (Eq. 5): s > eps (p = 1) or s > eps^2 (p = 2), s the support
 *                statistic of the residual;
 *   OUTPUT_NORM  (Eq. 7): s * W > eps (p = 1) or s * W > eps^2 (p = 2), with
 *                W = sum |w| (p = 1) or sum w^2 (p = 2) over the whole weight
 *                tensor, summed in fp64 in ascending OIHW order at create; the
 *                product is rounded once in fp64.
 *   LEARNED      (Eq. 8, inference): f > 0, f(r; phi) = bias + sum over the
 *                in-frame taps (row-major) of a[q, tap], a[q, tap] = sum_c
 *                phi[c, tap] * r[q, c] over chunks of 8 channels (ascending
 *                within a chunk, chunk sums ascending), all fp32 without FMA;
 *                phi and bias come from skipconv_set_gate_weights; eps and
 *                norm_p are not used. Runs on the split pipeline, and in the
 *                single-pass register-operand kernel for bf16 layers with
 *                c_in 32, 64 or 128 and k*k*c_in <= 4096.
 * A NaN statistic turns the gate on in all three; a reference frame is dense. */
enum { SKIPCONV_GATE_INPUT_NORM = 0, SKIPCONV_GATE_OUTPUT_NORM = 1, SKIPCONV_GATE_LEARNED = 2 };

/* Optional activation output kept beside z, for chaining layers: NONE = no
 * buffer; IDENTITY = dtype(z); RELU = dtype(max(z, 0)). It changes only at
 * updated sites, like z (z is pre-activation, Eq. 1). */
enum { SKIPCONV_ACT_NONE = 0, SKIPCONV_ACT_IDENTITY = 1, SKIPCONV_ACT_RELU = 2 };

/* KEEP_STATS: also store each frame's per-site gate statistic (fp32) and
 * per-site gate bit (before block pooling), for skipconv_copy_stat /
 * skipconv_copy_site_mask. FORCE_DENSE: every block is active on every frame
 * (the same kernels, run dense; used as the dense baseline). SPLIT_PIPELINE:
 * never use the fused single-pass kernel; run the gate, compaction and
 * convolution kernels separately (the choice is otherwise made at create).
 * EMIT_RESIDUAL (needs an activation output): after every step, also hand a
 * chained successor its residual: r = fl32(y_new - y_old) at the blocks this
 * step updated (fp32, plus its bf16 rounding for bf16 layers) and r = 0 at
 * the blocks only the previous step updated; see skipconv_step_chained.
 * TRANSLATE: allow skipconv_step_translated (a second z slot and two block
 * lists in the workspace); not combinable with EMIT_RESIDUAL.
 * LARGE_GATE_TILES: the split pipeline's gate kernel takes tiles of 32 x 32
 * output sites (instead of 16 x 16 or 8 x 8) when its chunk sums combine in
 * lane groups (see skipconv_gate_tile) and such a tile holds at most 256
 * blocks: fewer halo pixels read twice, four times fewer workgroups. A tuning
 * knob; the results are the same.
 * CALLER_RETAINS: x_{t-1} is read from the caller's own buffer, the x_t of the
 * previous step, instead of a copy kept by the library (the state update of
 * Eq. 2 then writes nothing): the gate stores no copy of x_t and the workspace
 * holds no x_{t-1} slots (2 |x| less). The caller keeps each frame's buffer
 * valid and unchanged until the next step's work on the stream is done, and
 * passes a different buffer on every step after the first (E_INVALID_ARG for
 * the same pointer twice in a row, which would read as a zero residual). The
 * results are the same as without the flag. */
enum {
  SKIPCONV_FLAG_KEEP_STATS = 1u,
  SKIPCONV_FLAG_FORCE_DENSE = 2u,
  SKIPCONV_FLAG_SPLIT_PIPELINE = 4u,
  SKIPCONV_FLAG_EMIT_RESIDUAL = 8u,
  SKIPCONV_FLAG_TRANSLATE = 16u,
  SKIPCONV_FLAG_LARGE_GATE_TILES = 32u,
  SKIPCONV_FLAG_CALLER_RETAINS = 64u
};

typedef struct skipconv_desc {
  int32_t n;        /* independent streams (batch), >= 1 */
  int32_t h, w;     /* input frame height, width, >= 1 */
  int32_t c_in;     /* input channels, >= 1 */
  int32_t c_out;    /* output channels, 1..256 (dense) or == c_in (depthwise) */
  int32_t kernel;   /* k: odd, 1..7 */
  int32_t stride;   /* s: 1..4 */
  int32_t pad;      /* zero padding, 0..k-1; -1 selects (k-1)/2 */
  int32_t groups;   /* 1 (dense) or c_in == c_out (depthwise) */
  int32_t block;    /* b: gate block side, 1..64 (1 = per-site gate) */
  int32_t norm_p;   /* 1: sum |r| > eps;  2: sum r^2 > eps^2 */
  int32_t support;  /* SKIPCONV_SUPPORT_* */
  int32_t dtype;    /* SKIPCONV_F32 or SKIPCONV_BF16 (inputs, weights, activation out) */
  int32_t act_out;  /* SKIPCONV_ACT_* */
  uint32_t flags;   /* SKIPCONV_FLAG_* */
  float eps;        /* threshold, >= 0 or +inf; NaN is rejected */
  int32_t gate;     /* SKIPCONV_GATE_* */
} skipconv_desc;

typedef struct skipconv_layer* skipconv_t;

/* Fill *d with defaults: n = h = w = c_in = c_out = 1, kernel 3, stride 1,
 * pad -1, groups 1, block 1, norm_p 2, RF support, fp32, no activation
 * output, no flags, eps 0, Input-Norm gate. Host only. */
int skipconv_desc_init(skipconv_desc* d);

/* Check a descriptor without touching the GPU. Returns OK, E_INVALID_ARG or
 * E_UNSUPPORTED. Host only. */
int skipconv_validate(const skipconv_desc* d);

/* Output and block-grid extents: h_out = (h + 2 pad - k) / stride + 1 (same
 * for w); hb = ceil(h_out / block), wb = ceil(w_out / block). Host only;
 * any output pointer may be NULL. */
int skipconv_out_shape(const skipconv_desc* d, int32_t* h_out, int32_t* w_out,
                       int32_t* hb, int32_t* wb);

/* Device bytes one layer needs (packed weights, two x_{t-1} slots, z, the
 * optional activation buffer, gate masks, active list, counters). Host only. */
int skipconv_workspace_size(const skipconv_desc* d, size_t* bytes);

/* Create a layer: the convolution of Eq. 1 (weights w, kernel k, stride,
 * groups) run on residual frames (Eq. 3) behind the gate of Sec. 3.2.1
 * (threshold eps, Eq. 5; Output-Norm variant Eq. 7) or Sec. 3.2.2 (learned
 * gate, Eq. 8), with b x b block structure (Sec. 3.2.2, "Structured
 * Sparsity"). The workspace argument is the bind-workspace call of the
 * interface folded into create: every buffer the layer uses lives in it.
 *   weights:   device pointer, OIHW in d->dtype; copied and repacked on
 *              `stream` (the caller may free it once that work completes).
 *   workspace: device pointer of at least skipconv_workspace_size bytes,
 *              256-byte aligned, owned by the caller and kept alive until
 *              skipconv_destroy; or NULL to let the library allocate it.
 *   *out:      the new handle, or NULL on failure.
 * The first step after create is a reference frame. */
int skipconv_create(const skipconv_desc* d, const void* weights, void* workspace,
                    size_t workspace_bytes, void* stream, skipconv_t* out);

/* Process one frame (Eq. 3).
 *   x_t: device pointer, 16-byte aligned, N x H x W x C_in in the layer
 *        dtype; read by work enqueued on `stream`, so it must stay valid
 *        until that work is done (until the next step's work is done with
 *        SKIPCONV_FLAG_CALLER_RETAINS, whose next step reads it as x_{t-1}).
 *   *z_t: (may be NULL) set to the device pointer of the persistent state,
 *        N x H_out x W_out x C_out fp32, valid until the next step, reset or
 *        destroy on this handle. Copy it to keep it.
 * Everything is enqueued on `stream`; no host synchronisation. The pipeline
 * is chosen at create (skipconv_pipeline reports it):
 *   fused: one kernel per frame; each workgroup takes one tile of output
 *          sites through residual, statistic, threshold, block flags, x_{t-1}
 *          update, product and z update. Tiles with no active block store
 *          nothing; the product of a tile is formed before its gate is known
 *          where that hides the gate's latency, so on those builds a tile's
 *          MFMA work does not shrink with density, only its stores do.
 *   split: the gate kernel (residual, statistic, threshold, block pooling,
 *          x_{t-1} update, unordered work list of active blocks), then the
 *          sparse convolution kernel, which walks only the listed blocks
 *          (residual halo in LDS, MFMA product, z accumulate).
 * fused is chosen for shapes it is built for whose frames have at most four
 * tiles per compute unit (the variant with weights staged in LDS only for
 * layers of <= 64 input and output channels on at most one tile per compute
 * unit, three for 32 -> 32); SKIPCONV_FLAG_SPLIT_PIPELINE forces split. */
int skipconv_step(skipconv_t h, const void* x_t, void* stream, const float** z_t);

/* Process one frame whose content moved by (dy, dx) input pixels since the
 * previous frame, a known global translation (Sec. 3.3 with the warp T an
 * integer translation): r = x_t - T(x_{t-1}) and z = T~(z_{t-1}) + g (.) (w * r),
 * where T(x)[y, x] = x[y - dy, x - dx] and T~ translates the output grid by
 * (dy, dx) / stride, both zero where the source lies outside. Output rows
 * (columns) where convolution and translation do not commute -- the source
 * row is outside the grid, or a tap leaves the frame while its translated
 * source is inside -- are "exposed": their sites are gated on, and every block
 * holding one is recomputed from x_t and assigned. With eps = 0 every frame's
 * z equals the dense convolution of x_t. dy and dx must be multiples of the
 * stride with |dy| < h, |dx| < w; (0, 0) or a pending reference frame is a
 * plain skipconv_step. The layer needs SKIPCONV_FLAG_TRANSLATE (E_STATE
 * otherwise). Layers on the single-pass register-operand kernel take the
 * translated step in that kernel (the exposed blocks in a second product over
 * the same weights); the others run the split pipeline. z moves to the other
 * of its two slots, so use the returned pointer. */
int skipconv_step_translated(skipconv_t h, const void* x_t, int32_t dy, int32_t dx, void* stream,
                             const float** z_t);

/* Process one frame of a layer whose input is the activation output of the
 * layer `up` (sparse residual propagation between stacked layers, Sec. 3.1:
 * the successor's input changes only where `up` updated z). `up` must have
 * been created with SKIPCONV_FLAG_EMIT_RESIDUAL, its output must match this
 * layer's input (n, h_out = h, w_out = w, c_out = c_in, same dtype), and it
 * must have stepped the same frame already on `stream` (stream order).
 * Instead of reading x_t and x_{t-1} over the whole frame, the gate reads
 * `up`'s residual, and gate tiles whose input region holds no active block of
 * `up` skip their loads (norm gates); the convolution reads the residual
 * operand. Masks, counts and z are exactly those that skipconv_step with
 * x_t = dtype(act(z_up)) would give. A reference frame of this layer reads
 * `up`'s activation output in full. This layer's own x_{t-1} slots are not
 * maintained: step it with skipconv_step only after a reset.
 * Errors: E_INVALID_ARG (NULL or mismatched `up`), E_STATE (`up` does not emit
 * its residual or has not stepped), E_HIP. */
int skipconv_step_chained(skipconv_t h, skipconv_t up, void* stream, const float** z_t);

/* One step for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation):
 * the split-pipeline step of a layer with caller-retained frames, with no
 * handle and no workspace. Allocates nothing: every buffer its kernels use
 * beyond the arguments (work list and its counters, block flags, packed
 * weights) sits in one fixed device array of 4 MiB inside the library, one
 * per device, held until the process ends.
 *   d:       descriptor as for skipconv_create; flags 0 or FORCE_DENSE only,
 *            the Input-Norm gate, no activation output, and blocks no larger
 *            than the gate tile (E_UNSUPPORTED otherwise). A layer whose
 *            weights and work list need more than 4 MiB is rejected with
 *            E_SMALL_BUFFER (skipconv_last_error(NULL) names both sizes).
 *   weights: device pointer, OIHW in d->dtype, repacked into the array on
 *            every call.
 *   x_t:     device pointer, N x H x W x C_in, 16-byte aligned.
 *   x_prev:  the previous frame (same layout), or NULL for a reference frame
 *            (x_{t-1} taken as zero, every site on, z assigned).
 *   z:       device pointer, N x H_out x W_out x C_out fp32, 16-byte aligned:
 *            z_{t-1} on entry (not read on a reference frame), z_t on exit.
 * Enqueued on `stream`; the results equal those of skipconv_step on a layer
 * created with SKIPCONV_FLAG_SPLIT_PIPELINE | SKIPCONV_FLAG_CALLER_RETAINS.
 * Every call on a device shares that device's array and leaves its contents
 * behind: calls that overlap on one device (different streams, or threads)
 * race and must be serialised by the caller. */
int skipconv_step_static(const skipconv_desc* d, const void* weights, const void* x_t, const void* x_prev,
                         float* z, void* stream);

/* Make the next step a reference frame: x_{t-1} taken as zero, every site
 * active, z assigned instead of accumulated (Sec. 3.1, Table 4). */
int skipconv_reset(skipconv_t h);

/* Change eps for later steps (same rules as the descriptor field). */
int skipconv_set_eps(skipconv_t h, float eps);

/* Parameters of a SKIPCONV_GATE_LEARNED layer's gate convolution (Eq. 8).
 *   phi:  device pointer, fp32, c_in x k x k (a one-output-channel OIHW
 *         tensor); copied and repacked on `stream`, so it may be freed once
 *         that work completes.
 *   bias: the gate convolution's bias (not NaN).
 * Required before the first step of such a layer (E_STATE otherwise); may be
 * called again between steps. E_STATE for layers with another gate. */
int skipconv_set_gate_weights(skipconv_t h, const float* phi, float bias, void* stream);

/* Release the handle and memory the library allocated. NULL is a no-op.
 * Work still enqueued on the handle's streams must be complete. */
int skipconv_destroy(skipconv_t h);

/* Device pointer of the activation output (N x H_out x W_out x C_out in the
 * layer dtype), or E_STATE when act_out is NONE. Valid like z. */
int skipconv_activation(skipconv_t h, const void** y);

/* Descriptor the handle was created with (eps as last set). Host only. */
int skipconv_get_desc(skipconv_t h, skipconv_desc* d);

/* Kernels one step launches: *fused = 0 for the gate + compaction +
 * convolution pipeline, 1 for the single-pass kernel (gate, local compaction
 * and MFMA product in one launch) with the weights staged in LDS, 2 for the
 * single-pass kernel whose waves hold their weight fragments in registers
 * (tiles of <= 8 x 8 sites, shapes it is built for), 3 for that kernel with
 * the output channels of each tile split over 2, 4 or 8 workgroups (shapes
 * built only for a share of the channels), 4 for the single-pass depthwise
 * kernel (bf16, C % 8 == 0, blocks of <= 8: per-channel products over the
 * taps, channels split over up to 8 workgroups per tile), 5 for the
 * single-pass kernel for few input channels (fp32 C_in <= 16 or bf16
 * C_in < 8, C_out <= 64, blocks of <= 8: element halo loads, MFMA product
 * with the residual operand gathered per k index). Host only. */
int skipconv_pipeline(skipconv_t h, int32_t* fused);

/* Gate tiling of the split pipeline: *ts = output sites per side of one gate
 * workgroup's tile (whole blocks, or a divisor of the block side), *lane_sum =
 * 1 when a pixel's 8-channel chunk sums are added in registers by a group of
 * 2, 4, 8 or 16 lanes (norm gates with 16, 32, 64 or 128 input channels) or a
 * pixel's statistic is formed by one thread (fewer than 8 channels), 0 when
 * the chunk sums are staged in LDS. Host only. */
int skipconv_gate_tile(skipconv_t h, int32_t* ts, int32_t* lane_sum);

/* Convolution kernel of the split pipeline: *kind = 0 gather (tiles of 64
 * active sites, operands gathered from the frames), 1 block halo (tiles of
 * rows of one active block, the residual halo staged in LDS; bf16, C_in % 32
 * = 0, b in {4, 8, 16, 32, 64}), 2 depthwise over the listed sites (fp32, or
 * C % 8 != 0), 3 depthwise with the residual halo of tiles of an active block
 * staged in LDS (bf16, C % 8 == 0). Host only. */
int skipconv_conv_kernel(skipconv_t h, int32_t* kind);

/* ---- introspection (tests and benchmarks; each synchronises `stream`) ---- */

/* Active blocks and active output sites of the last step. */
int skipconv_active_count(skipconv_t h, void* stream, int64_t* blocks, int64_t* sites);

/* Host copy of the last step's block mask, N x HB x WB bytes (0/1). */
int skipconv_copy_block_mask(skipconv_t h, void* stream, uint8_t* host, size_t bytes);

/* Host copy of the last step's active list: ascending block indices
 * n*HB*WB + bi*WB + bj. capacity in entries; *count receives the length. */
int skipconv_copy_active_list(skipconv_t h, void* stream, uint32_t* host, size_t capacity,
                              int64_t* count);

/* Host copy of the list of active blocks the last step's convolution walked
 * (split pipeline): the gate kernel's work list, whose order is that of the
 * appends (unordered; every active block once), or, for blocks larger than a
 * gate tile, the ordered list the compaction wrote. capacity in entries;
 * *count receives the length. E_UNSUPPORTED after a one-pass step (it keeps
 * no list: its block flags, skipconv_copy_block_mask, are its own output). */
int skipconv_copy_work_list(skipconv_t h, void* stream, uint32_t* host, size_t capacity,
                            int64_t* count);

/* Host copies of the last step's per-site gate bit (N x H_out x W_out bytes)
 * and gate statistic (fp32, same shape). E_STATE without KEEP_STATS. */
int skipconv_copy_site_mask(skipconv_t h, void* stream, uint8_t* host, size_t bytes);
int skipconv_copy_stat(skipconv_t h, void* stream, float* host, size_t bytes);

/* Dense-equivalent and active MACs of the last step (the per-layer cost the
 * gate loss of Eq. 9 weighs). */
int skipconv_frame_macs(skipconv_t h, void* stream, uint64_t* dense, uint64_t* active);

/* Static text for a status code. Host only. */
const char* skipconv_status_string(int status);

/* Last error message recorded on this handle (or the last failed create on
 * this thread when h is NULL); never NULL. Host only. */
const char* skipconv_last_error(skipconv_t h);

/* ---- kernel timing (benchmarks) ----
 * Time kernel by kernel, with HIP events recorded on the step's stream, every
 * `every`-th step (every >= 1) of the following steps, for up to `frames`
 * timed steps. skipconv_timing_read (synchronises `stream`) returns in ms[0]
 * the summed milliseconds of the gate and compaction kernels (of the fused
 * kernel in the single-pass pipeline) and in ms[1] of the convolution kernel
 * (0 in the single-pass pipeline) over the timed steps, and their count; `mask` (may be NULL) receives
 * for each of them its index among the steps since skipconv_timing_begin.
 * frames = 0 stops timing. */
int skipconv_timing_begin(skipconv_t h, int frames, int every);
int skipconv_timing_read(skipconv_t h, void* stream, double* ms, int* frames_timed,
                         int32_t* step_index, int capacity);

#ifdef __cplusplus
}
#endif

#endif /* SKIPCONV_H */
