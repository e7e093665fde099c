"""CPU oracle of the streaming Skip-Convolution layer.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call this module. The GPU
library never routes through it, and the two share no code: this file imports
nothing from the ``paper_2104_11487_amd`` package.

What it computes (Habibian et al., "Skip-Convolutions for Efficient Video
Processing", CVPR 2021):

* Sec. 3.1, Eq. 1-2: a convolution is linear, so the output of frame t is the
  previous output plus the convolution of the residual frame r_t = x_t - x_{t-1}.
* Sec. 3.1: the first frame (and every reference frame) is processed over the
  whole frame, with r_1 = x_1.
* Sec. 3.1, Eq. 3: z~_t = z~_{t-1} + g(r_t) (.) (w * r_t), where the gate g maps
  r_t to one bit per output location; skipped locations keep z~_{t-1}.
* Sec. 3.2.1, Eq. 5 (Input-Norm gate): g = round(sigmoid(||r_t|| - eps)), with
  the norm taken over the kernel support of each output (all input channels
  times k_h x k_w). round(sigmoid(y)) is 1 exactly when y > 0 (a tie at y = 0
  rounds half-to-even to 0), so the gate is the comparison "norm > eps".
* Sec. 3.2.1, Eq. 6-7 (Output-Norm gate): the residual norm is multiplied by the
  norm of the whole weight tensor (all four dimensions) before the comparison
  with eps. By Young's inequality (Eq. 6) that product bounds the norm of the
  skipped update at the site, so a skipped site's update has norm <= eps.
* Sec. 3.2.2, Eq. 8 (Gumbel gate at inference): a light convolution f(r; phi)
  with one output channel and the layer's kernel size, stride and padding
  scores every output location; the gate rounds sigmoid(f), i.e. it is on
  exactly when f > 0. phi is a given parameter here (training is out of scope).
* Sec. 3.3 (residuals between warped frames): with a warp T of the previous
  frame, r_t = x_t - T(x_{t-1}) and z_t = T~(z_{t-1}) + w * r_t, T~ the same warp
  on the output grid. Here T is a known global integer translation d (the
  content moves by d pixels), so T~ is the translation by d / stride.
* Sec. 3.2.2, "Structured Sparsity": max-pool the gate with kernel = stride = b,
  then nearest-neighbour upsample by b, giving b x b constant masks.
* Sec. 4.2, "Runtime speed up": the sparse convolution is an im2col matrix
  product restricted to the active columns.

Readings taken where the paper is silent (each is a decision, listed with the
rest of the design notes):

* norm order p is a parameter: p = 2 compares sum(r^2) over the support with
  eps^2; p = 1 (the paper's default) compares sum(|r|) with eps.
* canonical statistic arithmetic, so that gate masks are reproducible bit for
  bit: residual r = fl32(x_t - x_prev); per pixel, the channel terms are
  summed in chunks of 8 consecutive channels (ascending within a chunk), and
  the chunk sums added in ascending chunk order, all in float32 with one
  rounding per multiply and per add (no fused multiply-add); then the support
  sum over taps (kh, kw) in row-major order, in float32, out-of-frame taps
  contributing nothing; the comparison is done exactly in float64 (eps is a
  float32, so eps*eps is exact in float64).
* a NaN statistic turns the gate on, so a NaN input reaches z instead of being
  silently skipped.
* Gumbel gate score, canonical order: for every input pixel q and tap (kh, kw),
  a[q, kh, kw] = sum over channels of phi[c, kh, kw] * r[q, c] in chunks of 8
  (ascending within a chunk from +0, chunk sums ascending from +0); then
  f[o] = sum of a over the in-frame taps of o in row-major order, plus the
  gate bias, all in float32 with one rounding per operation. The threshold
  eps is not used by this gate.
* Translation-compensated step: T and T~ fill with zeros where the source lies
  outside the frame; d must be a multiple of the stride. Convolution commutes
  with the translation except at output rows (columns) where a tap reaches
  content that the translation moved out of the frame, or whose source row
  (column) lies outside the output grid ("exposed"); every block holding an
  exposed site is recomputed from x_t (as on a reference frame, assigned), the
  other blocks follow the gated recurrence on the translated state. With
  eps = 0 this reproduces the dense convolution of every frame exactly.
* Output-Norm gate: the weight norm is kept in the same power as the residual
  statistic (sum |w| for p = 1, sum w^2 for p = 2), summed in float64 over the
  weights in ascending flat OIHW order (|w| and w^2 of float32 or bf16 values
  are exact in float64); the gate compares statistic * weight norm with the
  threshold, the product rounded once in float64.
* blocks are anchored at output (0, 0); partial edge blocks pool the sites they
  hold (ceil mode). The active list is the ascending row-major list of active
  block indices n*HB*WB + bi*WB + bj.
* conv operand: rho = r for float32 layers, rho = bf16_rne(r) for bf16 layers;
  the update w * rho and the state z are float64 here.
* zero "same" padding P = (k - 1) / 2 unless given; the gate lives on the
  output grid, so for stride s output (i, j) reads input rows i*s - P + kh.
* x_{t-1} is the previous input, copied in full every frame; a reference frame
  treats x_{t-1} as zero, forces every site on and assigns z instead of adding.

Parity pins: every function here is checked in ``tests/test_oracle_pins.py``
against values the mathematics fixes (library conv2d / max_pool2d /
nearest interpolate / relu and casts, exact integer arithmetic, exact rational
arithmetic, brute-force loops, telescoping of Eq. 2, closed forms for an
impulse residual). Each function has a named pin: block_upsample equals the
library's nearest interpolate and a per-site brute force; dense_conv equals the
library conv2d in fp64 (exact on integers) and a brute force; activation_to_storage
equals the library relu and casts; out_size / n_blocks equal the library's
output shapes; translate equals a brute-force shift.
"""
from __future__ import annotations

import math
from typing import Optional

import numpy as np

F32 = np.float32
F64 = np.float64
CHUNK = 8  # channels per chunk in the canonical order of the gate statistic

# ----------------------------------------------------------------------------
# Storage dtypes. bf16 values travel as their raw 16-bit patterns (uint16).
# ----------------------------------------------------------------------------


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact: bf16 is the top half of fp32)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def f32_to_bf16_rne(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round to nearest, ties to even); returns bit patterns.

    Keep the top 16 bits of the fp32 pattern after adding half an ulp of bf16
    (0x7FFF) plus the lowest kept bit (ties go to the even neighbour). NaNs
    stay NaN (quiet bit set).
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    rounded = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint32)
    nan = np.isnan(x)
    quiet = ((u >> np.uint64(16)).astype(np.uint32) | np.uint32(0x0040))
    out = np.where(nan, quiet, rounded) & np.uint32(0xFFFF)
    return out.astype(np.uint16)


def storage_to_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32)
    if dtype == "bf16":
        return bf16_bits_to_f32(x)
    raise ValueError(dtype)


# ----------------------------------------------------------------------------
# Geometry
# ----------------------------------------------------------------------------


def out_size(n_in: int, k: int, stride: int, pad: int) -> int:
    """Output extent of a convolution with zero padding pad (Eq. 1)."""
    return (n_in + 2 * pad - k) // stride + 1


def n_blocks(n_out: int, b: int) -> int:
    """Block count along one axis, ceil mode (structured gates, Sec. 3.2.2)."""
    return -(-n_out // b)


# ----------------------------------------------------------------------------
# Gate (Sec. 3.2.1, Eq. 5; structured variant Sec. 3.2.2)
# ----------------------------------------------------------------------------


def residual(x_t: np.ndarray, x_prev: np.ndarray) -> np.ndarray:
    """r_t = x_t - x_{t-1} (Eq. 2), one float32 rounding per element."""
    return np.subtract(x_t.astype(np.float32), x_prev.astype(np.float32), dtype=np.float32)


def pixel_stat(r: np.ndarray, norm_p: int) -> np.ndarray:
    """Per-pixel part of the support norm (Eq. 5): sum over channels in the canonical order.

    r: (N, H, W, C) float32. Returns (N, H, W) float32 holding sum_c r^2
    (p = 2) or sum_c |r| (p = 1). Canonical order: the channels are taken in
    chunks of CHUNK consecutive channels (the last chunk may be shorter);
    within a chunk the terms are added in ascending channel order starting
    from +0, and the chunk sums are then added in ascending chunk order
    starting from +0. Every multiply and every add is rounded to float32
    separately (no fused multiply-add).
    """
    if norm_p not in (1, 2):
        raise ValueError("norm_p must be 1 or 2")
    acc = np.zeros(r.shape[:3], dtype=np.float32)
    nc = r.shape[3]
    for c0 in range(0, nc, CHUNK):
        part = np.zeros(r.shape[:3], dtype=np.float32)
        for c in range(c0, min(c0 + CHUNK, nc)):
            v = r[..., c]
            term = np.multiply(v, v, dtype=np.float32) if norm_p == 2 else np.abs(v)
            part = np.add(part, term, dtype=np.float32)
        acc = np.add(acc, part, dtype=np.float32)
    return acc


def support_stat(a: np.ndarray, k: int, stride: int, pad: int, h_out: int, w_out: int,
                 support: str = "rf") -> np.ndarray:
    """Norm statistic of each output's kernel support (Eq. 5).

    'rf': s[o] = sum over taps (kh, kw) in row-major order of a[o*stride - pad + (kh, kw)],
    skipping taps outside the frame, in float32. 'centre': s[o] = a[o*stride].
    """
    n, h, w = a.shape
    if support == "centre":
        return a[:, 0:(h_out - 1) * stride + 1:stride, 0:(w_out - 1) * stride + 1:stride].copy()
    if support != "rf":
        raise ValueError(support)
    s = np.zeros((n, h_out, w_out), dtype=np.float32)
    oi = np.arange(h_out)
    oj = np.arange(w_out)
    for kh in range(k):
        rows = oi * stride - pad + kh
        rv = (rows >= 0) & (rows < h)
        for kw in range(k):
            cols = oj * stride - pad + kw
            cv = (cols >= 0) & (cols < w)
            tap = np.zeros((n, h_out, w_out), dtype=np.float32)
            valid = rv[:, None] & cv[None, :]
            rr = np.clip(rows, 0, h - 1)
            cc = np.clip(cols, 0, w - 1)
            tap[:] = a[:, rr][:, :, cc]
            s = np.where(valid[None], np.add(s, tap, dtype=np.float32), s)
    return s


def weight_norm(weight: np.ndarray, norm_p: int) -> float:
    """Norm of the whole weight tensor for the Output-Norm gate (Eq. 7).

    Returned in the power the gate compares: sum |w| for p = 1, sum w^2 (the
    squared 2-norm) for p = 2. The terms are taken in ascending flat OIHW order
    and added one at a time in float64 (a Python float).
    """
    acc = 0.0
    for v in np.asarray(weight, dtype=np.float64).reshape(-1).tolist():
        acc += abs(v) if norm_p == 1 else v * v
    return acc


def gate(s: np.ndarray, eps: float, norm_p: int, reference: bool, wnorm: float = 1.0) -> np.ndarray:
    """g = round(sigmoid(norm - eps)) (Eq. 5, or Eq. 7 with wnorm) as an exact comparison.

    On a reference frame every site is on (Sec. 3.1). Otherwise the site is on
    when statistic * wnorm exceeds the threshold (eps^2 for p = 2, eps for
    p = 1), computed in float64, or when the statistic is NaN. wnorm is 1 for
    the Input-Norm gate (the product is then exact) and weight_norm(w, p) for
    the Output-Norm gate.
    """
    if reference:
        return np.ones(s.shape, dtype=bool)
    e = float(np.float32(eps))
    thr = e * e if norm_p == 2 else e
    sd = s.astype(np.float64)
    return (sd * wnorm > thr) | np.isnan(sd)


def learned_pixel_taps(r: np.ndarray, phi: np.ndarray) -> np.ndarray:
    """Per-pixel, per-tap terms of the gate convolution f(r; phi) (Eq. 8, inference).

    r: (N, H, W, C) float32; phi: (C, k, k), the gate's single output channel.
    Returns (N, H, W, k, k) float32 with a[q, kh, kw] = sum_c phi[c, kh, kw] * r[q, c]
    in the canonical chunked order, every multiply and add rounded to float32.
    """
    phi = np.asarray(phi, dtype=np.float32)
    nc, k, _ = phi.shape
    assert r.shape[3] == nc
    acc = np.zeros(r.shape[:3] + (k, k), dtype=np.float32)
    for c0 in range(0, nc, CHUNK):
        part = np.zeros_like(acc)
        for c in range(c0, min(c0 + CHUNK, nc)):
            term = np.multiply(r[..., c][..., None, None], phi[c][None, None, None], dtype=np.float32)
            part = np.add(part, term, dtype=np.float32)
        acc = np.add(acc, part, dtype=np.float32)
    return acc


def learned_score(a: np.ndarray, bias: float, stride: int, pad: int, h_out: int, w_out: int) -> np.ndarray:
    """f(r; phi)[o] = sum over in-frame taps (row-major) of a[o*stride - pad + tap, tap], + bias.

    Float32, one rounding per add; the bias is added last.
    """
    n, h, w, k, _ = a.shape
    s = np.zeros((n, h_out, w_out), dtype=np.float32)
    oi, oj = np.arange(h_out), np.arange(w_out)
    for kh in range(k):
        rows = oi * stride - pad + kh
        rv = (rows >= 0) & (rows < h)
        for kw in range(k):
            cols = oj * stride - pad + kw
            cv = (cols >= 0) & (cols < w)
            blk = np.zeros((n, h_out, w_out), dtype=np.float32)
            blk[:, np.ix_(rv, cv)[0], np.ix_(rv, cv)[1]] = \
                a[:, rows[rv]][:, :, cols[cv]][..., kh, kw]
            s = np.add(s, blk, dtype=np.float32)
    return np.add(s, np.float32(bias), dtype=np.float32)


def learned_gate(y: np.ndarray, reference: bool) -> np.ndarray:
    """round(sigmoid(f)) at inference (Eq. 8): on exactly when f > 0, or f is NaN, or a reference frame."""
    if reference:
        return np.ones(y.shape, dtype=bool)
    return (y > 0) | np.isnan(y)


def block_pool(g: np.ndarray, b: int) -> np.ndarray:
    """Max-pool of the site gate with kernel = stride = b, ceil mode (Sec. 3.2.2)."""
    n, ho, wo = g.shape
    hb, wb = n_blocks(ho, b), n_blocks(wo, b)
    m = np.zeros((n, hb, wb), dtype=bool)
    for bi in range(hb):
        for bj in range(wb):
            m[:, bi, bj] = g[:, bi * b:(bi + 1) * b, bj * b:(bj + 1) * b].any(axis=(1, 2))
    return m


def block_upsample(m: np.ndarray, b: int, h_out: int, w_out: int) -> np.ndarray:
    """Nearest-neighbour upsample of the block mask by b, cropped to the output grid."""
    return np.repeat(np.repeat(m, b, axis=1), b, axis=2)[:, :h_out, :w_out]


def active_list(m: np.ndarray) -> np.ndarray:
    """Ascending row-major indices of the active blocks ("non-sparse columns", Sec. 4.2)."""
    return np.flatnonzero(m.reshape(-1)).astype(np.uint32)


# ----------------------------------------------------------------------------
# Sparse update (Eq. 3, im2col over active columns as in Sec. 4.2)
# ----------------------------------------------------------------------------


def operand(r: np.ndarray, dtype: str) -> np.ndarray:
    """Convolution operand: r itself (fp32 layers) or r rounded to bf16 (bf16 layers)."""
    if dtype == "f32":
        return r.astype(np.float64)
    return bf16_bits_to_f32(f32_to_bf16_rne(r)).astype(np.float64)


def conv_at_sites(rho: np.ndarray, weight: np.ndarray, stride: int, pad: int, groups: int,
                  sn: np.ndarray, si: np.ndarray, sj: np.ndarray,
                  chunk: int = 8192) -> np.ndarray:
    """w * rho evaluated only at output sites (sn, si, sj), in float64.

    rho: (N, H, W, C_in) float64; weight: (C_out, C_in/groups, k, k).
    For each site, its im2col row holds rho at input (si*stride - pad + kh,
    sj*stride - pad + kw, ci) ordered (kh, kw, ci), zero outside the frame; the
    row times the flattened kernel of each group gives the C_out outputs.
    Sites are processed in chunks of ``chunk`` rows to bound memory only.
    """
    n, h, w, c_in = rho.shape
    c_out, cg, k, _ = weight.shape
    og = c_out // groups
    wt = weight.astype(np.float64)
    padded = np.zeros((n, h + 2 * pad + stride * 0 + k, w + 2 * pad + k, c_in), dtype=np.float64)
    padded[:, pad:pad + h, pad:pad + w, :] = rho
    # W_g[(kh, kw, ci), co] for each group
    wmats = [wt[gi * og:(gi + 1) * og].transpose(2, 3, 1, 0).reshape(k * k * cg, og)
             for gi in range(groups)]
    out = np.empty((len(sn), c_out), dtype=np.float64)
    kh = np.arange(k)
    for c0 in range(0, len(sn), chunk):
        c1 = min(c0 + chunk, len(sn))
        nn, ii, jj = sn[c0:c1], si[c0:c1], sj[c0:c1]
        rows = (ii * stride)[:, None] + kh[None, :]          # padded coordinates
        cols = (jj * stride)[:, None] + kh[None, :]
        patch = padded[nn[:, None, None], rows[:, :, None], cols[:, None, :], :]  # (S, k, k, C_in)
        for gi in range(groups):
            pg = patch[..., gi * cg:(gi + 1) * cg].reshape(c1 - c0, k * k * cg)
            out[c0:c1, gi * og:(gi + 1) * og] = pg @ wmats[gi]
    return out


# ----------------------------------------------------------------------------
# Translation-compensated residual (Sec. 3.3, warp = integer translation)
# ----------------------------------------------------------------------------


def translate(x: np.ndarray, dy: int, dx: int) -> np.ndarray:
    """T(x)[n, i, j] = x[n, i - dy, j - dx], zero where that lies outside the frame (NHWC or NHW)."""
    out = np.zeros_like(x)
    h, w = x.shape[1], x.shape[2]
    ys, yd = slice(max(0, -dy), min(h, h - dy)), slice(max(0, dy), min(h, h + dy))
    xs, xd = slice(max(0, -dx), min(w, w - dx)), slice(max(0, dx), min(w, w + dx))
    out[:, yd, xd] = x[:, ys, xs]
    return out


def exposed_lines(n_out: int, n_in: int, k: int, stride: int, pad: int, d: int) -> np.ndarray:
    """Output rows (or columns) where the translated recurrence is not exact (Sec. 3.3).

    Line i is exposed when its source line i - d/stride lies outside the output
    grid, or when one of its taps p = i*stride - pad + kh lies outside the frame
    while p - d lies inside (content the translation pushed out of the frame).
    """
    do = d // stride
    out = np.zeros(n_out, dtype=bool)
    for i in range(n_out):
        if not (0 <= i - do < n_out):
            out[i] = True
            continue
        for kh in range(k):
            p = i * stride - pad + kh
            if (0 <= p - d < n_in) and not (0 <= p < n_in):
                out[i] = True
                break
    return out


# ----------------------------------------------------------------------------
# The streaming layer
# ----------------------------------------------------------------------------


class SkipConvOracle:
    """One Skip-Conv layer processing a stream frame by frame (Eq. 3).

    weight: OIHW (C_out, C_in/groups, k, k). For dtype 'bf16' the weights are
    given either as bf16 bit patterns (uint16) or as float values, which are
    then rounded to bf16 exactly as a bf16 layer stores them.
    gate: 'input' (Input-Norm gate, Eq. 5), 'output' (Output-Norm gate, Eq. 7;
    the norm of the stored weights) or 'learned' (Gumbel gate at inference,
    Eq. 8: gate_weight (C_in, k, k) float32 and gate_bias score each output; the
    step's 'stat' is then the score f).
    """

    def __init__(self, weight: np.ndarray, *, n: int, h: int, w: int, stride: int = 1,
                 pad: Optional[int] = None, groups: int = 1, eps: float = 0.0, block: int = 1,
                 norm_p: int = 2, support: str = "rf", dtype: str = "f32",
                 exact_residual: bool = False, gate: str = "input",
                 gate_weight: Optional[np.ndarray] = None, gate_bias: float = 0.0):
        weight = np.asarray(weight)
        if dtype == "bf16":
            bits = weight if weight.dtype == np.uint16 else f32_to_bf16_rne(weight.astype(np.float32))
            self.weight = bf16_bits_to_f32(bits).astype(np.float64)
        else:
            self.weight = weight.astype(np.float32).astype(np.float64)
        self.c_out, cg, self.k, _ = self.weight.shape
        self.groups = groups
        self.c_in = cg * groups
        self.n, self.h, self.w = n, h, w
        self.stride = stride
        self.pad = (self.k - 1) // 2 if pad is None else pad
        self.h_out = out_size(h, self.k, stride, self.pad)
        self.w_out = out_size(w, self.k, stride, self.pad)
        self.eps = float(np.float32(eps))
        self.block = block
        self.norm_p = norm_p
        self.support = support
        self.dtype = dtype
        self.exact_residual = exact_residual
        assert gate in ("input", "output", "learned"), gate
        self.gate_kind = gate
        self.wnorm = weight_norm(self.weight, norm_p) if gate == "output" else 1.0
        if gate == "learned":
            self.phi = np.asarray(gate_weight, dtype=np.float32).reshape(self.c_in, self.k, self.k)
            self.gate_bias = float(np.float32(gate_bias))
        self.z = np.zeros((n, self.h_out, self.w_out, self.c_out), dtype=np.float64)
        self.x_prev = None
        self.reference_pending = True
        self.frames = 0

    def reset(self) -> None:
        """Next step is a reference frame (Sec. 3.1; reset period of Table 4)."""
        self.reference_pending = True

    def dense_macs(self) -> int:
        return self.n * self.h_out * self.w_out * self.c_out * (self.c_in // self.groups) * self.k * self.k

    def step(self, x_t: np.ndarray, shift=(0, 0)) -> dict:
        """One frame. shift = (dy, dx): the content moved by that many input pixels
        since the previous frame (Sec. 3.3 with T a translation); multiples of the stride."""
        x32 = storage_to_f32(np.asarray(x_t), self.dtype)
        assert x32.shape == (self.n, self.h, self.w, self.c_in), x32.shape
        ref = self.reference_pending
        dy, dx = int(shift[0]), int(shift[1])
        shifted = (dy, dx) != (0, 0) and not ref
        if shifted:
            assert dy % self.stride == 0 and dx % self.stride == 0, "shift must be a multiple of the stride"
            ex = (exposed_lines(self.h_out, self.h, self.k, self.stride, self.pad, dy)[:, None]
                  | exposed_lines(self.w_out, self.w, self.k, self.stride, self.pad, dx)[None, :])
            exposed = np.broadcast_to(ex, (self.n, self.h_out, self.w_out))
            self.z = translate(self.z, dy // self.stride, dx // self.stride)
        prev = np.zeros_like(x32) if (ref or self.x_prev is None) else self.x_prev
        if shifted:
            prev = translate(prev, dy, dx)
        r = residual(x32, prev)
        if self.gate_kind == "learned":
            a = learned_pixel_taps(r, self.phi)
            s = learned_score(a, self.gate_bias, self.stride, self.pad, self.h_out, self.w_out)
            g = learned_gate(s, ref)
        else:
            a = pixel_stat(r, self.norm_p)
            s = support_stat(a, self.k, self.stride, self.pad, self.h_out, self.w_out, self.support)
            g = gate(s, self.eps, self.norm_p, ref, self.wnorm)
        if shifted:
            g = g | exposed
        m_blk = block_pool(g, self.block)
        m = block_upsample(m_blk, self.block, self.h_out, self.w_out)
        lst = active_list(m_blk)
        if self.exact_residual:
            rho = x32.astype(np.float64) - prev.astype(np.float64)
        else:
            rho = operand(r, self.dtype)
        # blocks holding an exposed site are recomputed from x_t (assigned)
        xm = (block_upsample(block_pool(exposed, self.block), self.block, self.h_out, self.w_out)
              if shifted else np.zeros_like(m))
        sn, si, sj = np.nonzero(m & ~xm)
        if len(sn):
            u = conv_at_sites(rho, self.weight, self.stride, self.pad, self.groups, sn, si, sj)
            if ref:
                self.z[sn, si, sj, :] = u
            else:
                self.z[sn, si, sj, :] += u
        sn, si, sj = np.nonzero(xm)
        if len(sn):
            rho_x = (x32.astype(np.float64) if self.exact_residual
                     else operand(residual(x32, np.zeros_like(x32)), self.dtype))
            self.z[sn, si, sj, :] = conv_at_sites(rho_x, self.weight, self.stride, self.pad, self.groups,
                                                  sn, si, sj)
        self.x_prev = x32.copy()
        self.reference_pending = False
        self.frames += 1
        active_sites = int(m.sum())
        return {
            "z": self.z.copy(),
            "stat": s,
            "site_mask": g,
            "block_mask": m_blk,
            "mask": m,
            "active": lst,
            "count": int(len(lst)),
            "active_sites": active_sites,
            "active_macs": active_sites * self.c_out * (self.c_in // self.groups) * self.k * self.k,
            "reference": ref,
        }


def activation_to_storage(z: np.ndarray, act: str, dtype: str) -> np.ndarray:
    """Next layer's input from this layer's state: dtype(act(z)) (z is pre-activation, Eq. 1).

    relu gives +0 for every non-positive value (-0 included) and passes NaN through.
    """
    y = np.maximum(z, 0.0) if act == "relu" else z
    y32 = y.astype(np.float32)
    if dtype == "f32":
        return y32
    return f32_to_bf16_rne(y32)


def dense_conv(x: np.ndarray, weight: np.ndarray, stride: int, pad: int, groups: int) -> np.ndarray:
    """Eq. 1 in float64 at every output site: z = w * x."""
    n, h, w, _ = x.shape
    k = weight.shape[2]
    ho, wo = out_size(h, k, stride, pad), out_size(w, k, stride, pad)
    sn, si, sj = np.meshgrid(np.arange(n), np.arange(ho), np.arange(wo), indexing="ij")
    u = conv_at_sites(x.astype(np.float64), weight, stride, pad, groups,
                      sn.reshape(-1), si.reshape(-1), sj.reshape(-1))
    return u.reshape(n, ho, wo, -1)


def mac_weighted_density(active_macs, dense_macs) -> float:
    """sum_l m_l * density_l with m_l the normalised MAC share (the weighting of Eq. 9)."""
    tot = float(sum(dense_macs))
    return float(sum(a for a in active_macs)) / tot if tot else 0.0
