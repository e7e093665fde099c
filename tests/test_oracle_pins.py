"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks an oracle function against something other than itself:
library routines (torch conv2d / max_pool2d / bf16 cast), exact integer or
rational arithmetic, brute-force loops, the telescoping identity of Eq. 2,
the frozen output of an all-off gate (Eq. 3), and the closed-form response of
an impulse residual. They are chosen so that a dropped term, a wrong sign, a
wrong tap index or a transposed operand fails at least one of them.
"""
from fractions import Fraction
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import skipconv_oracle as O

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def torch_conv(x_nhwc, w, stride, pad, groups):
    """Library cross-check of Eq. 1 (cross-correlation, as CNN frameworks define w * x)."""
    x = torch.from_numpy(np.ascontiguousarray(x_nhwc, dtype=np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(np.asarray(w, dtype=np.float64))
    z = F.conv2d(x, wt, stride=stride, padding=pad, groups=groups)
    return z.permute(0, 2, 3, 1).numpy()


def brute_update(rho, w, stride, pad, groups, sites):
    """Seven nested loops: the convolution at the listed sites, term by term."""
    n_, h, wd, c_in = rho.shape
    c_out, cg, k, _ = w.shape
    og = c_out // groups
    out = np.zeros((len(sites), c_out))
    for si, (n, i, j) in enumerate(sites):
        for co in range(c_out):
            gi = co // og
            acc = 0.0
            for kh in range(k):
                for kw in range(k):
                    y, x = i * stride - pad + kh, j * stride - pad + kw
                    if 0 <= y < h and 0 <= x < wd:
                        for cl in range(cg):
                            acc += float(w[co, cl, kh, kw]) * float(rho[n, y, x, gi * cg + cl])
            out[si, co] = acc
    return out


# ----------------------------------------------------------------------------
# bf16 rounding
# ----------------------------------------------------------------------------

def test_bf16_rne_matches_torch_cast():
    rng = _rng(1)
    vals = [rng.normal(0, 1, 20000), rng.normal(0, 1e-38, 2000), rng.normal(0, 1e30, 2000)]
    v = np.concatenate(vals).astype(np.float32)
    # exact ties: low 16 bits = 0x8000 with an even and an odd kept bit
    ties = np.array([0x3F808000, 0x3F818000, 0xBF808000, 0x00008000, 0x7F7F8000, 0x7F7FFFFF],
                    dtype=np.uint32).view(np.float32)
    special = np.array([0.0, -0.0, np.inf, -np.inf, 3.0e38, -3.4e38, 1e-45], dtype=np.float32)
    v = np.concatenate([v, ties, special])
    ours = O.f32_to_bf16_rne(v)
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    nan = np.array([np.nan, -np.nan], dtype=np.float32)
    assert np.isnan(O.bf16_bits_to_f32(O.f32_to_bf16_rne(nan))).all()


def test_bf16_widen_exact():
    bits = np.arange(0, 65536, dtype=np.uint32).astype(np.uint16)
    f = O.bf16_bits_to_f32(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float32).numpy()
    fin = np.isfinite(ref)
    assert np.array_equal(f[fin].view(np.uint32), ref[fin].view(np.uint32))
    assert np.array_equal(np.isnan(f), np.isnan(ref))


# ----------------------------------------------------------------------------
# Gate statistic (Eq. 5)
# ----------------------------------------------------------------------------

def test_pixel_stat_canonical_order():
    """The canonical order (chunks of 8 channels, ascending within and across chunks) is
    observable in fp32: a value that cancels inside one chunk order differs from another order."""
    r = np.zeros((1, 1, 1, 16), np.float32)
    r[..., 0] = 1.0
    r[..., 1:8] = 2.0 ** -13   # each square 2^-26: lost against 1.0 one at a time
    r[..., 8:16] = 2.0 ** -13  # next chunk: 8 * 2^-26 = 2^-23 survives as a chunk sum
    a = O.pixel_stat(r, 2)[0, 0, 0]
    assert a == np.float32(1.0) + np.float32(2.0 ** -23)
    seq = np.float32(0.0)
    for v in r[0, 0, 0]:
        seq = np.float32(seq + np.float32(v * v))
    assert seq == np.float32(1.0)  # plain left-to-right order loses every small term
    assert O.CHUNK == 8


@pytest.mark.parametrize("p", [1, 2])
def test_pixel_stat_integer_exact(p):
    rng = _rng(2)
    r = rng.integers(-9, 10, size=(2, 5, 6, 13)).astype(np.float32)
    a = O.pixel_stat(r, p)
    ri = r.astype(np.int64)
    ref = (ri * ri).sum(-1) if p == 2 else np.abs(ri).sum(-1)
    assert np.array_equal(a.astype(np.int64), ref)


@pytest.mark.parametrize("k,stride", [(1, 1), (3, 1), (3, 2), (5, 1), (5, 2)])
def test_support_stat_is_box_filter(k, stride):
    """Integer-valued a: the support sum equals a library box filter with zero padding."""
    rng = _rng(3)
    a = rng.integers(0, 50, size=(2, 9, 11)).astype(np.float32)
    pad = (k - 1) // 2
    ho, wo = O.out_size(9, k, stride, pad), O.out_size(11, k, stride, pad)
    s = O.support_stat(a, k, stride, pad, ho, wo, "rf")
    box = F.conv2d(torch.from_numpy(a.astype(np.float64))[:, None], torch.ones(1, 1, k, k, dtype=torch.float64),
                   stride=stride, padding=pad)[:, 0].numpy()
    assert s.shape == box.shape
    assert np.array_equal(s.astype(np.float64), box)


def test_support_stat_centre_and_1x1():
    rng = _rng(4)
    a = rng.random((1, 8, 7), dtype=np.float32)
    s1 = O.support_stat(a, 1, 1, 0, 8, 7, "rf")
    assert np.array_equal(s1, a)
    sc = O.support_stat(a, 3, 2, 1, 4, 4, "centre")
    assert np.array_equal(sc, a[:, ::2, ::2])


def test_statistic_within_rounding_bound_of_exact_rational():
    """fp32 canonical statistic vs the exact rational sum of squares over the support."""
    rng = _rng(5)
    c, k = 6, 3
    x1 = rng.random((1, 6, 6, c), dtype=np.float32)
    x0 = (x1 + rng.normal(0, 0.05, x1.shape).astype(np.float32)).astype(np.float32)
    r = O.residual(x1, x0)
    s = O.support_stat(O.pixel_stat(r, 2), k, 1, 1, 6, 6)
    u = 2.0 ** -24
    nterms = c * k * k
    gamma = (nterms + 2) * u / (1 - (nterms + 2) * u)
    flips = 0
    for i in range(6):
        for j in range(6):
            ex = Fraction(0)
            for kh in range(k):
                for kw in range(k):
                    y, xx = i - 1 + kh, j - 1 + kw
                    if 0 <= y < 6 and 0 <= xx < 6:
                        for ch in range(c):
                            v = Fraction(float(r[0, y, xx, ch]))
                            ex += v * v
            err = abs(Fraction(float(s[0, i, j])) - ex)
            assert err <= Fraction(gamma) * ex
            # the gate decision agrees with the exact one unless the threshold lies within the bound
            for eps2 in (float(ex) * 0.999, float(ex) * 1.001, float(ex)):
                eps = float(np.float32(math.sqrt(eps2)))
                thr = Fraction(eps) * Fraction(eps)
                g = O.gate(s[:, i:i + 1, j:j + 1], eps, 2, False)[0, 0, 0]
                if abs(ex - thr) > Fraction(gamma) * ex:
                    assert bool(g) == (ex > thr)
                else:
                    flips += 0 if bool(g) == (ex > thr) else 1
    assert flips <= 36  # counted, only possible within one rounding bound of eps


def test_residual_is_ieee_subtraction():
    rng = _rng(6)
    a = rng.random(1000, dtype=np.float32)
    b = rng.random(1000, dtype=np.float32)
    r = O.residual(a, b)
    ref = (torch.from_numpy(a) - torch.from_numpy(b)).numpy()
    assert np.array_equal(r.view(np.uint32), ref.view(np.uint32))


# ----------------------------------------------------------------------------
# Gate (Eq. 5) and blocks (structured sparsity)
# ----------------------------------------------------------------------------

def _nonzero_patch(r, k, stride, pad, ho, wo):
    n, h, w, _ = r.shape
    out = np.zeros((n, ho, wo), bool)
    for b in range(n):
        for i in range(ho):
            for j in range(wo):
                for kh in range(k):
                    for kw in range(k):
                        y, x = i * stride - pad + kh, j * stride - pad + kw
                        if 0 <= y < h and 0 <= x < w and np.any(r[b, y, x] != 0):
                            out[b, i, j] = True
    return out


@pytest.mark.parametrize("stride", [1, 2])
def test_eps0_gate_is_nonzero_patch_indicator(stride):
    rng = _rng(7)
    r = rng.normal(0, 1, size=(2, 9, 8, 3)).astype(np.float32)
    r[rng.random((2, 9, 8)) < 0.8] = 0.0
    ho, wo = O.out_size(9, 3, stride, 1), O.out_size(8, 3, stride, 1)
    for p in (1, 2):
        s = O.support_stat(O.pixel_stat(r, p), 3, stride, 1, ho, wo)
        g = O.gate(s, 0.0, p, False)
        assert np.array_equal(g, _nonzero_patch(r, 3, stride, 1, ho, wo))


def test_gate_eps_inf_empty_monotone_nan_and_reference():
    rng = _rng(8)
    s = (rng.random((2, 6, 6)) * 4).astype(np.float32)
    s[0, 2, 3] = np.nan
    off = O.gate(s, np.float32(np.inf), 2, False)
    assert off.sum() == 1 and off[0, 2, 3]  # only the NaN site
    prev = None
    for eps in (0.0, 0.3, 0.7, 1.0, 1.5, 2.5):
        g = O.gate(s, eps, 2, False)
        if prev is not None:
            assert not np.any(g & ~prev)
        prev = g
    assert O.gate(s, np.float32(np.inf), 2, True).all()
    # strict comparison: a statistic equal to the threshold is off (round(sigmoid(0)) = 0)
    t = np.array([[[0.25]]], dtype=np.float32)
    assert not O.gate(t, 0.5, 2, False)[0, 0, 0]
    assert not O.gate(t, 0.25, 1, False)[0, 0, 0]


@pytest.mark.parametrize("b", [1, 2, 3, 4, 8])
def test_block_pool_is_ceil_maxpool(b):
    rng = _rng(9 + b)
    g = rng.random((3, 13, 10)) < 0.1
    m = O.block_pool(g, b)
    ref = F.max_pool2d(torch.from_numpy(g.astype(np.float32))[:, None], b, b, ceil_mode=True)[:, 0]
    assert np.array_equal(m, ref.numpy() > 0)
    up = O.block_upsample(m, b, 13, 10)
    assert not np.any(g & ~up)  # the block mask covers every gated site
    lst = O.active_list(m)
    brute = [n * m.shape[1] * m.shape[2] + i * m.shape[2] + j
             for n in range(m.shape[0]) for i in range(m.shape[1]) for j in range(m.shape[2]) if m[n, i, j]]
    assert lst.tolist() == brute


# ----------------------------------------------------------------------------
# Sparse update (Eq. 3)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("k,stride,groups", [(1, 1, 1), (3, 1, 1), (3, 2, 1), (3, 1, 4), (1, 2, 2), (5, 1, 1)])
def test_update_at_sites_bruteforce(k, stride, groups):
    rng = _rng(10 + k * 7 + stride + groups)
    c_in, c_out = 4, 8
    rho = rng.normal(0, 1, (2, 7, 6, c_in))
    w = rng.normal(0, 1, (c_out, c_in // groups, k, k))
    pad = (k - 1) // 2
    ho, wo = O.out_size(7, k, stride, pad), O.out_size(6, k, stride, pad)
    sel = rng.random((2, ho, wo)) < 0.4
    sn, si, sj = np.nonzero(sel)
    u = O.conv_at_sites(rho, w, stride, pad, groups, sn, si, sj, chunk=5)
    ref = brute_update(rho, w, stride, pad, groups, list(zip(sn, si, sj)))
    np.testing.assert_allclose(u, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("k,stride,groups", [(3, 1, 1), (3, 2, 1), (1, 1, 1), (3, 1, 6)])
def test_reference_step_is_dense_conv(k, stride, groups):
    rng = _rng(20 + k + stride + groups)
    c = 6
    x = rng.random((2, 10, 9, c), dtype=np.float32)
    w = rng.normal(0, 1, (c, c // groups, k, k)).astype(np.float32)
    lay = O.SkipConvOracle(w, n=2, h=10, w=9, stride=stride, groups=groups, eps=10.0, block=2)
    out = lay.step(x)
    ref = torch_conv(x, w, stride, (k - 1) // 2, groups)
    np.testing.assert_allclose(out["z"], ref, rtol=1e-12, atol=1e-12)
    assert out["count"] == out["block_mask"].size and out["reference"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("block", [1, 3])
def test_eps0_telescopes_to_dense_conv_integer_exact(dtype, block):
    """Eq. 2 telescoping: with eps = 0 the accumulated output is w * x_T, bit for bit on integers."""
    rng = _rng(30)
    c = 5
    w = rng.integers(-2, 3, (7, c, 3, 3)).astype(np.float32)
    lay = O.SkipConvOracle(w, n=1, h=11, w=12, eps=0.0, block=block, dtype=dtype)
    x = rng.integers(0, 8, (1, 11, 12, c)).astype(np.float32)
    for t in range(6):
        x = x.copy()
        sel = rng.random((1, 11, 12)) < 0.15
        x[sel] = rng.integers(0, 8, (int(sel.sum()), c))
        xs = x if dtype == "f32" else O.f32_to_bf16_rne(x)
        out = lay.step(xs)
        assert np.array_equal(out["z"], torch_conv(x, w, 1, 1, 1))


def test_eps0_telescopes_exact_residual_mode():
    rng = _rng(31)
    c = 4
    w = rng.normal(0, 1, (6, c, 3, 3)).astype(np.float32)
    lay = O.SkipConvOracle(w, n=1, h=9, w=10, stride=2, eps=0.0, exact_residual=True)
    for t in range(5):
        x = rng.random((1, 9, 10, c), dtype=np.float32)
        x[:, :4] = 0.5  # part of the frame static
        out = lay.step(x)
    ref = torch_conv(x, w, 2, 1, 1)
    assert np.max(np.abs(out["z"] - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))


def test_all_gates_off_freezes_output_and_prev_advances():
    rng = _rng(32)
    c = 3
    w = rng.normal(0, 1, (4, c, 3, 3)).astype(np.float32)
    lay = O.SkipConvOracle(w, n=1, h=8, w=8, eps=np.float32(np.inf))
    xs = [rng.random((1, 8, 8, c), dtype=np.float32) for _ in range(4)]
    z1 = lay.step(xs[0])["z"]
    for t in (1, 2):
        out = lay.step(xs[t])
        assert out["count"] == 0 and len(out["active"]) == 0
        assert np.array_equal(out["z"], z1)
    lay.eps = 0.0
    out = lay.step(xs[3])
    ref = z1 + torch_conv(xs[3].astype(np.float64) - xs[2].astype(np.float64), w, 1, 1, 1)
    np.testing.assert_allclose(out["z"], ref, rtol=1e-6, atol=1e-6)


def test_reset_mid_stream_gives_dense_frame():
    rng = _rng(33)
    c = 4
    w = rng.normal(0, 1, (4, c, 3, 3)).astype(np.float32)
    lay = O.SkipConvOracle(w, n=1, h=8, w=9, eps=0.5, block=2)
    for _ in range(3):
        lay.step(rng.random((1, 8, 9, c), dtype=np.float32))
    lay.reset()
    x = rng.random((1, 8, 9, c), dtype=np.float32)
    out = lay.step(x)
    assert out["reference"] and out["count"] == out["block_mask"].size
    np.testing.assert_allclose(out["z"], torch_conv(x, w, 1, 1, 1), rtol=1e-12, atol=1e-12)


def _load_golden(name):
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", name)
    rows = [ln for ln in open(path) if ln.strip() and not ln.startswith("#")]
    return np.array([[float(v) for v in ln.split()] for ln in rows])


def test_impulse_response_golden():
    """One changed pixel: Eq. 3 updates exactly the outputs whose support holds it,
    by the kernel read backwards (hand-derived fixture)."""
    w = np.arange(1, 10, dtype=np.float32).reshape(1, 1, 3, 3)
    lay = O.SkipConvOracle(w, n=1, h=5, w=5, eps=0.0)
    x0 = np.zeros((1, 5, 5, 1), np.float32)
    lay.step(x0)
    x1 = x0.copy()
    x1[0, 2, 2, 0] = 1.0
    out = lay.step(x1)
    expect = _load_golden("impulse_3x3_5x5.txt")
    assert np.array_equal(out["z"][0, :, :, 0], expect)
    assert np.array_equal(out["site_mask"][0], expect != 0)


@pytest.mark.parametrize("k,stride,b", [(3, 1, 1), (3, 1, 2), (3, 2, 1), (5, 1, 3), (1, 1, 2)])
def test_impulse_active_set_closed_form(k, stride, b):
    rng = _rng(40 + k + stride + b)
    h, w, c = 11, 10, 3
    pad = (k - 1) // 2
    wt = rng.normal(0, 1, (2, c, k, k)).astype(np.float32)
    lay = O.SkipConvOracle(wt, n=1, h=h, w=w, stride=stride, eps=0.0, block=b)
    x0 = rng.random((1, h, w, c), dtype=np.float32)
    lay.step(x0)
    qy, qx = 4, 7
    x1 = x0.copy()
    x1[0, qy, qx, 1] += np.float32(0.75)
    out = lay.step(x1)
    ho, wo = lay.h_out, lay.w_out
    exp = np.zeros((1, ho, wo), bool)
    for i in range(ho):
        for j in range(wo):
            if i * stride - pad <= qy <= i * stride - pad + k - 1 and j * stride - pad <= qx <= j * stride - pad + k - 1:
                exp[0, i, j] = True
    assert np.array_equal(out["site_mask"], exp)
    blocks = {(i // b, j // b) for i, j in zip(*np.nonzero(exp[0]))}
    hb = -(-ho // b)
    wb = -(-wo // b)
    assert sorted(out["active"].tolist()) == sorted(bi * wb + bj for bi, bj in blocks)
    assert out["block_mask"].shape == (1, hb, wb)


def test_nan_frame_gates_on_then_reset_recovers():
    rng = _rng(50)
    c = 3
    w = rng.normal(0, 1, (4, c, 3, 3)).astype(np.float32)
    lay = O.SkipConvOracle(w, n=1, h=8, w=8, eps=np.float32(1e6))
    x = rng.random((1, 8, 8, c), dtype=np.float32)
    lay.step(x)
    xn = x.copy()
    xn[0, 3, 5, 2] = np.nan
    out = lay.step(xn)
    exp = np.zeros((8, 8), bool)
    exp[2:5, 4:7] = True
    assert np.array_equal(out["site_mask"][0], exp)
    assert np.array_equal(np.isnan(out["z"][0]).any(-1), exp)
    lay.reset()
    x3 = rng.random((1, 8, 8, c), dtype=np.float32)
    out = lay.step(x3)
    assert np.isfinite(out["z"]).all()
    np.testing.assert_allclose(out["z"], torch_conv(x3, w, 1, 1, 1), rtol=1e-12, atol=1e-12)


def test_stack_residual_zero_outside_upstream_active_set():
    """Chained layers (Sec. 3.1): the next layer's input changes only where this layer updated."""
    rng = _rng(60)
    w1 = rng.normal(0, 0.5, (6, 3, 3, 3)).astype(np.float32)
    l1 = O.SkipConvOracle(w1, n=1, h=16, w=16, eps=0.3, dtype="bf16")
    y_prev = None
    x = rng.random((1, 16, 16, 3), dtype=np.float32)
    for t in range(5):
        x = x.copy()
        x[0, 3 + t:7 + t, 4:8] = rng.random((4, 4, 3), dtype=np.float32)
        out = l1.step(O.f32_to_bf16_rne(x))
        y = O.activation_to_storage(out["z"], "relu", "bf16")
        if y_prev is not None:
            changed = np.any(y != y_prev, axis=-1)
            assert not np.any(changed & ~out["mask"])
        y_prev = y


def test_bf16_operand_rounding_applied():
    """bf16 layers convolve bf16(r): an update equals the fp64 conv of the rounded residual."""
    rng = _rng(61)
    w = O.f32_to_bf16_rne(rng.normal(0, 1, (3, 2, 3, 3)).astype(np.float32))
    lay = O.SkipConvOracle(w, n=1, h=6, w=6, eps=0.0, dtype="bf16")
    x0 = O.f32_to_bf16_rne(rng.random((1, 6, 6, 2), dtype=np.float32))
    x1 = O.f32_to_bf16_rne(rng.random((1, 6, 6, 2), dtype=np.float32) * 3)
    z0 = lay.step(x0)["z"]
    z1 = lay.step(x1)["z"]
    r = O.bf16_bits_to_f32(x1) - O.bf16_bits_to_f32(x0)
    rho = torch.from_numpy(r).to(torch.bfloat16).to(torch.float64).numpy()
    wf = O.bf16_bits_to_f32(w)
    np.testing.assert_allclose(z1 - z0, torch_conv(rho, wf, 1, 1, 1), rtol=1e-12, atol=1e-12)


def test_mac_accounting():
    rng = _rng(62)
    w = rng.normal(0, 1, (8, 4, 3, 3)).astype(np.float32)
    lay = O.SkipConvOracle(w, n=1, h=10, w=10, eps=0.5, block=2)
    lay.step(rng.random((1, 10, 10, 4), dtype=np.float32))
    x = rng.random((1, 10, 10, 4), dtype=np.float32)
    out = lay.step(x)
    assert out["active_macs"] == int(out["mask"].sum()) * 8 * 4 * 9
    assert lay.dense_macs() == 100 * 8 * 4 * 9
    d = O.mac_weighted_density([out["active_macs"], 0], [lay.dense_macs(), lay.dense_macs()])
    assert d == pytest.approx(out["mask"].mean() / 2)


# ----------------------------------------------------------------------------
# Output-Norm gate (Sec. 3.2.1, Eq. 6-7)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("p", [1, 2])
def test_weight_norm_is_the_whole_tensor_norm(p):
    # integer weights: the float64 sum is exact, so it must equal the integer norm
    rng = _rng(60)
    w = rng.integers(-7, 8, (5, 3, 3, 3)).astype(np.float64)
    exact = int(np.abs(w).sum()) if p == 1 else int((w.astype(np.int64) ** 2).sum())
    assert O.weight_norm(w, p) == float(exact)
    # random weights: within the sequential-summation bound of the correctly rounded sum
    w = rng.normal(0, 0.1, (16, 8, 3, 3)).astype(np.float32)
    terms = [abs(float(v)) if p == 1 else float(v) * float(v) for v in w.reshape(-1)]
    ref = math.fsum(terms)
    assert abs(O.weight_norm(w, p) - ref) <= len(terms) * 2.0 ** -52 * ref
    # a per-output-channel norm or a max would differ from the whole-tensor norm
    assert O.weight_norm(w, p) > max(O.weight_norm(w[c], p) for c in range(w.shape[0]))


@pytest.mark.parametrize("p", [1, 2])
def test_output_norm_gate_bounds_skipped_updates(p):
    """Young's inequality (Eq. 6): at a skipped site, ||w * r||_p <= ||w||_p ||r||_p <= eps."""
    rng = _rng(61 + p)
    n, h, wd, c, co, k = 1, 12, 10, 8, 6, 3
    w = rng.normal(0, 0.3, (co, c, k, k)).astype(np.float32)
    x0 = rng.random((n, h, wd, c), dtype=np.float32)
    x1 = x0 + rng.normal(0, 0.05, x0.shape).astype(np.float32) * (rng.random(x0.shape) < 0.3)
    x1 = x1.astype(np.float32)
    wn = O.weight_norm(w, p)
    r = O.residual(x1, x0)
    s = O.support_stat(O.pixel_stat(r, p), k, 1, 1, h, wd, "rf")
    # eps at the median of the gated quantity, so both outcomes occur
    q = s.astype(np.float64) * wn
    eps = float(np.float32(np.median(q) if p == 1 else math.sqrt(float(np.median(q)))))
    lay = O.SkipConvOracle(w, n=n, h=h, w=wd, eps=eps, norm_p=p, gate="output")
    lay.step(x0)
    out = lay.step(x1)
    off = ~out["site_mask"]
    assert 0 < off.sum() < off.size
    sn, si, sj = np.nonzero(off)
    u = brute_update(r.astype(np.float64), w.astype(np.float64), 1, 1, 1, list(zip(sn, si, sj)))
    un = np.abs(u).sum(axis=1) if p == 1 else np.sqrt((u * u).sum(axis=1))
    # the statistic is a float32 sum: allow its rounding (relative K * 2^-24)
    assert np.all(un <= eps * (1.0 + 1e-4)), (un.max(), eps)
    # a tight case: one non-zero weight (the centre tap of channel 0) and isolated
    # impulses in channel 0, so ||w * r|| = ||w|| ||r|| at the impulse sites; the
    # gate must then skip exactly the impulses whose update norm is <= eps (a
    # smaller weight norm, e.g. one output channel's, would skip larger ones)
    w = np.zeros((2, c, k, k), np.float32)
    w[0, 0, 1, 1] = 1.5
    x0 = np.zeros((n, h, wd, c), np.float32)
    x1 = x0.copy()
    amps = np.array([0.25, 0.5, 1.0, 2.0, 4.0, 8.0], np.float32)
    pos = [(1, 1), (1, 6), (5, 2), (5, 7), (9, 1), (9, 6)]
    for (y, x), a in zip(pos, amps):
        x1[0, y, x, 0] = a
    eps = 1.4 if p == 1 else 1.4  # between 1.5 * 0.5 and 1.5 * 1.0
    lay = O.SkipConvOracle(w, n=n, h=h, w=wd, eps=eps, norm_p=p, gate="output")
    lay.step(x0)
    out = lay.step(x1)
    for (y, x), a in zip(pos, amps):
        assert bool(out["site_mask"][0, y, x]) == (1.5 * float(a) > eps), (y, x, a)


@pytest.mark.parametrize("p", [1, 2])
def test_output_norm_gate_equals_input_norm_at_scaled_eps(p):
    """With ||w||_p a power of two the Output-Norm gate is the Input-Norm gate at eps / ||w||_p."""
    rng = _rng(70 + p)
    n, h, wd, c, k = 2, 9, 11, 8, 3
    w = np.zeros((4, c, k, k), np.float32)
    # four entries +-0.5: sum |w| = 2, sum w^2 = 1; scaled by 4: 8 and 16
    idx = rng.choice(w.size, 4, replace=False)
    w.reshape(-1)[idx] = np.array([0.5, -0.5, 0.5, -0.5], np.float32) * 4
    wn = O.weight_norm(w, p)
    assert wn == (8.0 if p == 1 else 16.0)
    scale = 8.0 if p == 1 else 4.0  # ||w||_p itself (the 2-norm is sqrt(16))
    frames = [rng.random((n, h, wd, c), dtype=np.float32) for _ in range(4)]
    frames = [f * (rng.random(f.shape) < 0.5) for f in frames]
    eps = 0.75
    a = O.SkipConvOracle(w, n=n, h=h, w=wd, eps=eps, norm_p=p, gate="output")
    b = O.SkipConvOracle(w, n=n, h=h, w=wd, eps=eps / scale, norm_p=p, gate="input")
    for f in frames:
        ra, rb = a.step(f.astype(np.float32)), b.step(f.astype(np.float32))
        assert np.array_equal(ra["site_mask"], rb["site_mask"])
        assert np.array_equal(ra["z"], rb["z"])


# ----------------------------------------------------------------------------
# Gumbel gate at inference (Sec. 3.2.2, Eq. 8)
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("k,stride", [(1, 1), (3, 1), (3, 2), (5, 1)])
def test_learned_score_is_single_channel_conv2d(k, stride):
    rng = _rng(80 + k + stride)
    n, h, wd, c = 2, 11, 9, 19
    r = rng.normal(0, 1, (n, h, wd, c)).astype(np.float32)
    phi = rng.normal(0, 0.5, (c, k, k)).astype(np.float32)
    pad = (k - 1) // 2
    ho, wo = O.out_size(h, k, stride, pad), O.out_size(wd, k, stride, pad)
    y = O.learned_score(O.learned_pixel_taps(r, phi), -0.125, stride, pad, ho, wo)
    ref = torch_conv(r.astype(np.float64), phi[None].astype(np.float64), stride, pad, 1)[..., 0] - 0.125
    mag = torch_conv(np.abs(r).astype(np.float64), np.abs(phi)[None].astype(np.float64), stride, pad, 1)[..., 0]
    # float32 recursive summation: |error| <= (terms) * 2^-24 * sum |phi r| (+ the bias add)
    bound = (c * k * k + 2) * 2.0 ** -24 * (mag + 0.125)
    assert np.all(np.abs(y - ref) <= bound)


def test_learned_score_single_tap_is_exact_shift():
    """phi non-zero at one tap only, integer data: f[o] is exactly the channel sum at that tap's pixel."""
    rng = _rng(85)
    n, h, wd, c = 1, 7, 8, 12
    r = rng.integers(-4, 5, (n, h, wd, c)).astype(np.float32)
    phi = np.zeros((c, 3, 3), np.float32)
    phi[:, 0, 2] = rng.integers(-3, 4, c).astype(np.float32)
    y = O.learned_score(O.learned_pixel_taps(r, phi), 0.0, 1, 1, h, wd)
    exp = np.zeros((n, h, wd), np.float64)
    for i in range(h):
        for j in range(wd):
            yy, xx = i - 1 + 0, j - 1 + 2
            if 0 <= yy < h and 0 <= xx < wd:
                exp[0, i, j] = float((r[0, yy, xx].astype(np.float64) * phi[:, 0, 2]).sum())
    assert np.array_equal(y.astype(np.float64), exp)


def test_learned_gate_with_unit_phi_is_input_norm_p1_on_growing_frames():
    """phi = 1, bias = -eps and non-negative residuals: f = s - eps, so f > 0 iff s > eps (Eq. 5, p = 1)."""
    rng = _rng(86)
    n, h, wd, c, co, k = 1, 10, 12, 16, 8, 3
    w = rng.normal(0, 0.3, (co, c, k, k)).astype(np.float32)
    x = rng.random((n, h, wd, c), dtype=np.float32)
    frames = [x]
    for t in range(4):
        grow = (rng.random(x.shape[:3]) < 0.04)[..., None]
        x = (x + rng.random(x.shape, dtype=np.float32) * 0.1 * grow).astype(np.float32)
        frames.append(x)
    eps = 0.3
    a = O.SkipConvOracle(w, n=n, h=h, w=wd, eps=0.0, norm_p=2, gate="learned",
                         gate_weight=np.ones((c, k, k), np.float32), gate_bias=-eps)
    b = O.SkipConvOracle(w, n=n, h=h, w=wd, eps=eps, norm_p=1, gate="input")
    partial = 0
    for f in frames:
        ra, rb = a.step(f), b.step(f)
        assert np.array_equal(ra["site_mask"], rb["site_mask"])
        assert np.array_equal(ra["z"], rb["z"])
        partial += 0 < int(ra["site_mask"].sum()) < ra["site_mask"].size
    assert partial >= 3  # the non-reference masks are neither all on nor all off


def test_learned_gate_nan_reference_and_strictness():
    y = np.array([[[0.0, -0.0, 1e-30, -1e-30, np.nan]]], np.float32)
    assert O.learned_gate(y, False).tolist() == [[[False, False, True, False, True]]]
    assert O.learned_gate(y, True).all()


# ----------------------------------------------------------------------------
# Translation-compensated residual (Sec. 3.3 with T an integer translation)
# ----------------------------------------------------------------------------

def test_exposed_lines_closed_form():
    # H = 10, k = 3, pad 1, stride 1, content moved down by 2: rows 0-1 have no
    # source row, row 9's bottom tap leaves the frame while its source is inside
    assert np.flatnonzero(O.exposed_lines(10, 10, 3, 1, 1, 2)).tolist() == [0, 1, 9]
    assert np.flatnonzero(O.exposed_lines(10, 10, 3, 1, 1, -2)).tolist() == [0, 8, 9]
    assert not O.exposed_lines(10, 10, 3, 1, 1, 0).any()
    # 1 x 1 kernel, no padding: only the rows without a source
    assert np.flatnonzero(O.exposed_lines(8, 8, 1, 1, 0, 3)).tolist() == [0, 1, 2]


@pytest.mark.parametrize("k,stride,d", [(3, 1, (2, -1)), (3, 2, (2, -4)), (5, 1, (-3, 2)), (1, 1, (1, 1))])
def test_convolution_commutes_with_translation_off_the_exposed_lines(k, stride, d):
    """w * T(x) == T~(w * x) exactly at every site that is not exposed (integer data)."""
    rng = _rng(110 + k + stride)
    n, h, wd, c, co = 2, 13, 11, 4, 3
    pad = (k - 1) // 2
    x = rng.integers(-5, 6, (n, h, wd, c)).astype(np.float64)
    w = rng.integers(-3, 4, (co, c, k, k)).astype(np.float64)
    a = torch_conv(O.translate(x, *d), w, stride, pad, 1)
    b = O.translate(torch_conv(x, w, stride, pad, 1), d[0] // stride, d[1] // stride)
    ho, wo = a.shape[1], a.shape[2]
    ex = O.exposed_lines(ho, h, k, stride, pad, d[0])[:, None] | O.exposed_lines(wo, wd, k, stride, pad, d[1])[None, :]
    assert np.array_equal(a[:, ~ex], b[:, ~ex])
    assert ex.any() and (~ex).any()


@pytest.mark.parametrize("dtype,stride", [("f32", 1), ("bf16", 1), ("f32", 2)])
def test_translated_recurrence_eps0_is_dense_conv_integer_exact(dtype, stride):
    """eps = 0 with translation compensation: every frame's z equals conv2d(x_t) exactly."""
    rng = _rng(120 + stride)
    n, h, wd, c, co, k = 1, 14, 12, 4, 5, 3
    w = rng.integers(-2, 3, (co, c, k, k)).astype(np.float32)
    lay = O.SkipConvOracle(w, n=n, h=h, w=wd, stride=stride, eps=0.0, block=2, dtype=dtype)
    x = rng.integers(0, 8, (n, h, wd, c)).astype(np.float32)
    shifts = [(0, 0), (2, 0), (0, -2), (-2, 2), (0, 0), (4, -2)]
    for t, d in enumerate(shifts):
        if t:
            x = O.translate(x, *d)
            fresh = rng.integers(0, 8, x.shape).astype(np.float32)
            hole = O.translate(np.ones_like(x), *d) == 0        # entering content
            x = np.where(hole, fresh, x)
            x[:, 5, 3] += 1.0                                    # plus a local change
        xs = O.f32_to_bf16_rne(x) if dtype == "bf16" else x
        out = lay.step(xs, shift=d if t else (0, 0))
        dense = torch_conv(x.astype(np.float64), w.astype(np.float64), stride, 1, 1)
        assert np.array_equal(out["z"], dense), (dtype, stride, t)


def test_translation_compensation_leaves_moved_static_content_off():
    """A textured scene moving rigidly: compensated, only the entering strip and exposed
    lines update; uncompensated, the whole textured frame fires."""
    rng = _rng(130)
    n, h, wd, c, co = 1, 24, 20, 8, 4
    w = rng.normal(0, 0.3, (co, c, 3, 3)).astype(np.float32)
    x = rng.random((n, h, wd, c), dtype=np.float32)
    a = O.SkipConvOracle(w, n=n, h=h, w=wd, eps=1e-3, block=1)
    b = O.SkipConvOracle(w, n=n, h=h, w=wd, eps=1e-3, block=1)
    a.step(x)
    b.step(x)
    x1 = O.translate(x, 1, 2)
    x1 = np.where(O.translate(np.ones_like(x), 1, 2) == 0, rng.random(x.shape, dtype=np.float32), x1)
    ra, rb = a.step(x1, shift=(1, 2)), b.step(x1)
    ex = O.exposed_lines(h, h, 3, 1, 1, 1)[:, None] | O.exposed_lines(wd, wd, 3, 1, 1, 2)[None, :]
    # compensated: exactly the exposed sites and the sites whose support reaches
    # the entering content (rows < 1, columns < 2 of the new frame)
    hole = np.zeros((h, wd), bool)
    hole[:1, :] = True
    hole[:, :2] = True
    near = np.zeros((h, wd), bool)
    for i in range(h):
        for j in range(wd):
            near[i, j] = hole[max(0, i - 1):i + 2, max(0, j - 1):j + 2].any()
    assert np.array_equal(ra["site_mask"][0], ex | near)
    assert (ex | near).mean() < 0.5
    assert rb["site_mask"].mean() > 0.9
    dense = torch_conv(x1.astype(np.float64), w.astype(np.float64), 1, 1, 1)
    assert np.abs(ra["z"] - dense).max() < 1e-5


def test_zero_translation_is_the_plain_step():
    rng = _rng(131)
    w = rng.normal(0, 0.3, (4, 6, 3, 3)).astype(np.float32)
    a = O.SkipConvOracle(w, n=1, h=9, w=10, eps=0.2, block=2)
    b = O.SkipConvOracle(w, n=1, h=9, w=10, eps=0.2, block=2)
    for t in range(4):
        x = rng.random((1, 9, 10, 6), dtype=np.float32)
        ra, rb = a.step(x, shift=(0, 0)), b.step(x)
        assert np.array_equal(ra["z"], rb["z"]) and np.array_equal(ra["block_mask"], rb["block_mask"])


# ----------------------------------------------------------------------------
# Pins of the helpers used outside the recurrence: block upsample, dense
# convolution, activation output, geometry and translation
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("b,h,w", [(1, 5, 7), (2, 13, 10), (3, 13, 10), (4, 16, 16), (8, 13, 10), (16, 9, 17)])
def test_block_upsample_is_cropped_nearest_interpolate(b, h, w):
    """Sec. 3.2.2: nearest-neighbour upsampling of the pooled gate by b, cropped to the output
    grid; equal to the library routine and to site (i, j) reading block (i // b, j // b)."""
    rng = _rng(70 + b)
    m = rng.random((3, O.n_blocks(h, b), O.n_blocks(w, b))) < 0.4
    up = O.block_upsample(m, b, h, w)
    assert up.shape == (3, h, w) and up.dtype == bool
    lib = F.interpolate(torch.from_numpy(m.astype(np.float32))[:, None], scale_factor=b, mode="nearest")
    assert np.array_equal(up, lib[:, 0, :h, :w].numpy() > 0)
    brute = np.array([[[m[n, i // b, j // b] for j in range(w)] for i in range(h)] for n in range(3)])
    assert np.array_equal(up, brute)
    # exact: pooling the upsampled mask gives the block mask back (no block grows)
    assert np.array_equal(O.block_pool(up, b), m)


@pytest.mark.parametrize("k,stride,pad,groups", [(1, 1, 0, 1), (3, 1, 1, 1), (3, 2, 1, 1), (3, 1, 0, 2),
                                                 (5, 1, 2, 1), (3, 1, 1, 6), (3, 3, 2, 3)])
def test_dense_conv_is_library_conv2d(k, stride, pad, groups):
    """Eq. 1 at every output site: equal to the library conv2d in fp64 (and exact on integers)."""
    rng = _rng(80 + k + stride + pad + groups)
    c = 6
    x = rng.normal(0, 1, (2, 11, 9, c))
    w = rng.normal(0, 1, (12, c // groups, k, k))
    z = O.dense_conv(x, w, stride, pad, groups)
    np.testing.assert_allclose(z, torch_conv(x, w, stride, pad, groups), rtol=1e-12, atol=1e-12)
    xi = rng.integers(-4, 5, x.shape).astype(np.float64)
    wi = rng.integers(-3, 4, w.shape).astype(np.float64)
    assert np.array_equal(O.dense_conv(xi, wi, stride, pad, groups), torch_conv(xi, wi, stride, pad, groups))


def test_dense_conv_bruteforce_tiny():
    rng = _rng(88)
    x = rng.normal(0, 1, (1, 4, 5, 3))
    w = rng.normal(0, 1, (2, 3, 3, 3))
    z = O.dense_conv(x, w, 2, 1, 1)
    sites = [(0, i, j) for i in range(z.shape[1]) for j in range(z.shape[2])]
    ref = brute_update(x, w, 2, 1, 1, sites).reshape(z.shape)
    np.testing.assert_allclose(z, ref, rtol=1e-12, atol=1e-12)


def test_activation_to_storage_is_relu_then_cast():
    """The next layer's input dtype(act(z)): the library relu followed by the library casts
    (fp64 -> fp32 -> bf16, round to nearest even), including signed zeros, NaN, ties and overflow.
    Reading: relu returns +0 for every non-positive value, -0 included (the library keeps the
    sign of a zero; adding +0 clears it), and passes NaN through."""
    rng = _rng(90)
    z = rng.normal(0, 10, 4096)
    z[:12] = [0.0, -0.0, np.nan, -np.nan, np.inf, -np.inf, 3.0e38, -3.0e38, 1.0 + 2.0 ** -8,
              1.0 + 3 * 2.0 ** -8, 1e-40, -1e-40]
    zt = torch.from_numpy(z)
    for act in ("relu", "identity"):
        ref = (torch.relu(zt) + 0.0 if act == "relu" else zt).to(torch.float32)
        got32 = O.activation_to_storage(z, act, "f32")
        assert got32.dtype == np.float32
        assert np.array_equal(got32.view(np.uint32)[~np.isnan(got32)],
                              ref.numpy().view(np.uint32)[~np.isnan(got32)])
        assert np.array_equal(np.isnan(got32), torch.isnan(ref).numpy())
        bits = O.activation_to_storage(z, act, "bf16")
        rb = ref.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        fin = ~torch.isnan(ref).numpy()
        assert np.array_equal(bits[fin], rb[fin])
        assert np.all(np.isnan(O.bf16_bits_to_f32(bits[~fin])))
    # relu keeps no negative value; identity keeps the sign
    assert not np.any(O.bf16_bits_to_f32(O.activation_to_storage(z, "relu", "bf16")) < 0)
    assert np.any(O.bf16_bits_to_f32(O.activation_to_storage(z, "identity", "bf16")) < 0)


@pytest.mark.parametrize("n_in,k,stride,pad", [(7, 3, 1, 1), (7, 3, 2, 1), (8, 5, 3, 2), (1, 1, 1, 0), (9, 7, 2, 0)])
def test_out_size_and_blocks_match_library(n_in, k, stride, pad):
    z = F.conv2d(torch.zeros(1, 1, n_in, n_in + 1), torch.zeros(1, 1, k, k), stride=stride, padding=pad)
    assert (O.out_size(n_in, k, stride, pad), O.out_size(n_in + 1, k, stride, pad)) == tuple(z.shape[2:])
    for b in (1, 2, 3, 16):
        pooled = F.max_pool2d(torch.zeros(1, 1, z.shape[2], z.shape[3]), b, b, ceil_mode=True)
        assert (O.n_blocks(z.shape[2], b), O.n_blocks(z.shape[3], b)) == tuple(pooled.shape[2:])


def test_translate_bruteforce():
    rng = _rng(91)
    x = rng.normal(0, 1, (2, 6, 7, 3))
    for dy, dx in [(0, 0), (1, 0), (-2, 3), (5, -6), (6, 0), (0, -7)]:
        t = O.translate(x, dy, dx)
        ref = np.zeros_like(x)
        for i in range(6):
            for j in range(7):
                if 0 <= i - dy < 6 and 0 <= j - dx < 7:
                    ref[:, i, j] = x[:, i - dy, j - dx]
        assert np.array_equal(t, ref)
