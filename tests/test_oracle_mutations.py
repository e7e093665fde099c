"""Planted mistakes in the oracle, each caught by a pin.

Every case replaces one oracle function (or the stepping of the layer) with a
plausible wrong version — a dropped term, a wrong sign or index, a transposed
operand, a non-strict comparison, truncation instead of rounding — and runs a
pin from test_oracle_pins.py against it: the pin must fail. This checks that
the pins constrain the oracle, not only that the oracle passes them. CPU only.
"""
import numpy as np
import pytest

import test_oracle_pins as pins
from oracle import skipconv_oracle as O


def _upsample_spread(orig):
    def bad(m, b, h_out, w_out):
        up = orig(m, b, h_out, w_out)
        out = up.copy()
        out[..., 1:, :] |= up[..., :-1, :]  # covers one row more than its blocks
        return out
    return bad


def _gate_not_strict(orig):
    def bad(s, eps, norm_p, reference, wnorm=1.0):
        thr = float(np.float64(eps) * np.float64(eps)) if norm_p == 2 else float(eps)
        g = (s.astype(np.float64) * wnorm >= thr) | np.isnan(s)
        return g | bool(reference)
    return bad


def _pixel_stat_drop_channel(orig):
    return lambda r, norm_p: orig(r[..., :-1], norm_p)


def _conv_flipped(orig):
    def bad(rho, weight, stride, pad, groups, *sites):
        return orig(rho, np.ascontiguousarray(weight[..., ::-1, ::-1]), stride, pad, groups, *sites)
    return bad


def _conv_transposed(orig):
    def bad(rho, weight, stride, pad, groups, *sites):
        return orig(rho, np.ascontiguousarray(weight.transpose(0, 1, 3, 2)), stride, pad, groups, *sites)
    return bad


def _operand_truncated(orig):
    def bad(r, dtype):
        if dtype != "bf16":
            return orig(r, dtype)
        bits = np.ascontiguousarray(r, dtype=np.float32).view(np.uint32) & np.uint32(0xFFFF0000)
        return bits.view(np.float32)
    return bad


def _residual_sign(orig):
    return lambda x_t, x_prev: orig(x_prev, x_t)


def _pool_and(orig):
    def bad(g, b):
        n, h, w = g.shape
        hb, wb = -(-h // b), -(-w // b)
        out = np.zeros((n, hb, wb), dtype=bool)
        for i in range(hb):
            for j in range(wb):
                out[:, i, j] = g[:, i * b:(i + 1) * b, j * b:(j + 1) * b].all(axis=(1, 2))
        return out
    return bad


def _activation_no_relu(orig):
    return lambda z, act, dtype: orig(z, "identity", dtype)


def _dense_flipped(orig):
    return lambda x, weight, stride, pad, groups: orig(x, np.ascontiguousarray(weight[..., ::-1, ::-1]),
                                                       stride, pad, groups)


def _taps_drop_channel(orig):
    return lambda r, phi: orig(r[..., :-1], phi[:-1])


def _translate_sign(orig):
    return lambda x, dy, dx: orig(x, -dy, -dx)


def _exposed_source_only(orig):
    def bad(n_out, n_in, k, stride, pad, d):
        do = d // stride
        return np.array([not (0 <= i - do < n_out) for i in range(n_out)], dtype=bool)
    return bad


def _support_short(orig):
    def bad(a, k, stride, pad, h_out, w_out, support="rf"):
        if k == 1 or support != "rf":
            return orig(a, k, stride, pad, h_out, w_out, support)
        # the last tap row left out
        n, h, w = a.shape
        out = np.zeros((n, h_out, w_out), dtype=np.float32)
        ap = np.zeros((n, h + 2 * k, w + 2 * k), dtype=np.float32)
        ap[:, pad:pad + h, pad:pad + w] = a
        for i in range(h_out):
            for j in range(w_out):
                acc = np.zeros(n, dtype=np.float32)
                for kh in range(k - 1):
                    for kw in range(k):
                        acc = acc + ap[:, i * stride + kh, j * stride + kw]
                out[:, i, j] = acc
        return out
    return bad


def _learned_gate_not_strict(orig):
    return lambda y, reference: (y >= 0) | np.isnan(y) | bool(reference)


CASES = [
    ("block_upsample", _upsample_spread, pins.test_block_upsample_is_cropped_nearest_interpolate, (2, 13, 10)),
    ("gate", _gate_not_strict, pins.test_eps0_gate_is_nonzero_patch_indicator, (1,)),
    ("pixel_stat", _pixel_stat_drop_channel, pins.test_pixel_stat_integer_exact, (2,)),
    ("conv_at_sites", _conv_flipped, pins.test_reference_step_is_dense_conv, (3, 1, 1)),
    ("conv_at_sites", _conv_transposed, pins.test_reference_step_is_dense_conv, (3, 1, 1)),
    ("operand", _operand_truncated, pins.test_bf16_operand_rounding_applied, ()),
    ("residual", _residual_sign, pins.test_residual_is_ieee_subtraction, ()),
    ("block_pool", _pool_and, pins.test_block_pool_is_ceil_maxpool, (2,)),
    ("activation_to_storage", _activation_no_relu, pins.test_activation_to_storage_is_relu_then_cast, ()),
    ("dense_conv", _dense_flipped, pins.test_dense_conv_is_library_conv2d, (3, 1, 1, 1)),
    ("learned_pixel_taps", _taps_drop_channel, pins.test_learned_score_is_single_channel_conv2d, (3, 1)),
    ("translate", _translate_sign, pins.test_translate_bruteforce, ()),
    ("exposed_lines", _exposed_source_only, pins.test_exposed_lines_closed_form, ()),
    ("support_stat", _support_short, pins.test_support_stat_is_box_filter, (3, 1)),
    ("learned_gate", _learned_gate_not_strict, pins.test_learned_gate_nan_reference_and_strictness, ()),
]


@pytest.mark.parametrize("name,mutate,pin,args", CASES,
                         ids=[f"{c[0]}-{c[1].__name__.lstrip('_')}" for c in CASES])
def test_planted_mistake_fails_a_pin(monkeypatch, name, mutate, pin, args):
    pin(*args)  # the pin holds for the oracle as it is
    monkeypatch.setattr(O, name, mutate(getattr(O, name)))
    with pytest.raises((AssertionError, ValueError, IndexError)):
        pin(*args)


def test_stale_previous_frame_fails_telescoping(monkeypatch):
    """A layer that never advances x_{t-1} (the state update of Eq. 2 dropped)."""
    orig = O.SkipConvOracle.step

    def stale(self, x_t, shift=(0, 0)):
        old = None if self.x_prev is None else self.x_prev.copy()
        out = orig(self, x_t, shift)
        if old is not None:
            self.x_prev = old
        return out

    pins.test_eps0_telescopes_to_dense_conv_integer_exact("f32", 1)
    monkeypatch.setattr(O.SkipConvOracle, "step", stale)
    with pytest.raises(AssertionError):
        pins.test_eps0_telescopes_to_dense_conv_integer_exact("f32", 1)
