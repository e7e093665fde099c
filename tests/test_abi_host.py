"""Host-side checks of the C ABI: the library loads, exports every declared
symbol, validates descriptors and sizes buffers -- without launching GPU work."""
import ctypes

import pytest

from paper_2104_11487_amd import skipconv as S


@pytest.fixture(scope="module")
def lib():
    return S.lib()


def test_every_header_symbol_is_exported(lib):
    names = S.header_symbols()
    assert "skipconv_create" in names and "skipconv_step" in names and "skipconv_reset" in names
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    assert set(names) == set(S._SIGS), set(names) ^ set(S._SIGS)


def test_desc_defaults(lib):
    d = S.skipconv_desc_init()
    assert (d.n, d.h, d.w, d.c_in, d.c_out) == (1, 1, 1, 1, 1)
    assert (d.kernel, d.stride, d.pad, d.groups, d.block, d.norm_p) == (3, 1, -1, 1, 1, 2)
    assert d.eps == 0.0 and d.flags == 0 and d.gate == S.SKIPCONV_GATE_INPUT_NORM
    assert S.skipconv_validate(d) == S.SKIPCONV_OK


def good(**kw):
    base = dict(n=1, h=128, w=96, c_in=64, c_out=64, kernel=3, block=8, dtype="bf16", eps=0.1)
    base.update(kw)
    return S.make_desc(**base)


@pytest.mark.parametrize("field,value,code", [
    ("n", 0, S.SKIPCONV_E_INVALID_ARG), ("h", 0, S.SKIPCONV_E_INVALID_ARG),
    ("c_in", 0, S.SKIPCONV_E_INVALID_ARG), ("kernel", 2, S.SKIPCONV_E_INVALID_ARG),
    ("kernel", 9, S.SKIPCONV_E_INVALID_ARG), ("stride", 0, S.SKIPCONV_E_INVALID_ARG),
    ("pad", 3, S.SKIPCONV_E_INVALID_ARG), ("pad", -2, S.SKIPCONV_E_INVALID_ARG),
    ("groups", 3, S.SKIPCONV_E_INVALID_ARG), ("groups", 2, S.SKIPCONV_E_UNSUPPORTED),
    ("block", 0, S.SKIPCONV_E_INVALID_ARG), ("block", 65, S.SKIPCONV_E_INVALID_ARG),
    ("norm_p", 3, S.SKIPCONV_E_INVALID_ARG), ("support", 2, S.SKIPCONV_E_INVALID_ARG),
    ("dtype", 2, S.SKIPCONV_E_INVALID_ARG), ("act_out", 3, S.SKIPCONV_E_INVALID_ARG),
    ("flags", 128, S.SKIPCONV_E_INVALID_ARG), ("flags", 8, S.SKIPCONV_E_INVALID_ARG),
    ("eps", -1.0, S.SKIPCONV_E_INVALID_ARG),
    ("eps", float("nan"), S.SKIPCONV_E_INVALID_ARG), ("c_out", 272, S.SKIPCONV_E_UNSUPPORTED),
    ("gate", 7, S.SKIPCONV_E_INVALID_ARG), ("gate", -1, S.SKIPCONV_E_INVALID_ARG),
    ("gate", 3, S.SKIPCONV_E_INVALID_ARG),
])
def test_validation_codes(lib, field, value, code):
    d = good()
    setattr(d, field, value)
    assert S.skipconv_validate(d) == code
    assert S.skipconv_last_error()  # a message was recorded


def test_valid_variants(lib):
    assert S.skipconv_validate(good(eps=float("inf"))) == 0
    assert S.skipconv_validate(good(groups=64)) == 0           # depthwise
    assert S.skipconv_validate(good(kernel=1, block=1)) == 0
    assert S.skipconv_validate(good(dtype="f32", c_in=3)) == 0
    assert S.skipconv_validate(good(stride=2, pad=0)) == 0
    assert S.skipconv_validate(good(block=64, h=20, w=20)) == 0
    assert S.skipconv_validate(good(support="centre", norm_p=1)) == 0
    assert S.skipconv_validate(good(gate="output")) == 0
    assert S.skipconv_validate(good(gate="output", norm_p=1, dtype="f32")) == 0
    assert S.skipconv_validate(good(gate="learned")) == 0
    assert S.skipconv_validate(good(act_out="relu", emit_residual=True)) == 0
    assert S.skipconv_validate(good(translate=True)) == 0
    assert S.skipconv_validate(good(act_out="relu", emit_residual=True, translate=True)) == S.SKIPCONV_E_UNSUPPORTED
    assert S.skipconv_validate(good(gate="learned", kernel=7, dtype="f32", c_in=256)) == 0


@pytest.mark.parametrize("h,w,k,s,pad,b,exp", [
    (32, 32, 3, 1, -1, 1, (32, 32, 32, 32)),
    (128, 96, 3, 1, -1, 8, (128, 96, 16, 12)),
    (256, 192, 3, 2, -1, 1, (128, 96, 128, 96)),
    (7, 9, 3, 2, -1, 3, (4, 5, 2, 2)),
    (10, 10, 3, 1, 0, 4, (8, 8, 2, 2)),
    (512, 512, 3, 1, -1, 16, (512, 512, 32, 32)),
])
def test_out_shape(lib, h, w, k, s, pad, b, exp):
    d = good(h=h, w=w, kernel=k, stride=s, pad=pad, block=b)
    assert S.skipconv_out_shape(d) == exp


def test_workspace_size_covers_state(lib):
    d = good()
    n = S.skipconv_workspace_size(d)
    x = 128 * 96 * 64 * 2
    z = 128 * 96 * 64 * 4
    assert n >= 2 * x + z + 64 * 64 * 9 * 2
    d2 = good(act_out="relu", keep_stats=True)
    assert S.skipconv_workspace_size(d2) >= n + 128 * 96 * 64 * 2 + 128 * 96 * 5
    d3 = good(act_out="relu", emit_residual=True)  # + fp32 and bf16 residuals + previous block flags
    assert S.skipconv_workspace_size(d3) >= n + 128 * 96 * 64 * (2 + 4 + 2) + 16 * 12
    # caller-retained frames: no x_{t-1} slots
    d4 = good(caller_retains=True)
    assert S.skipconv_validate(d4) == 0
    assert n - S.skipconv_workspace_size(d4) == 2 * x


def test_null_handles_and_status_strings(lib):
    assert lib.skipconv_step(None, None, None, None) == S.SKIPCONV_E_STATE
    assert lib.skipconv_step_chained(None, None, None, None) == S.SKIPCONV_E_STATE
    assert lib.skipconv_step_translated(None, None, 0, 0, None, None) == S.SKIPCONV_E_STATE
    assert lib.skipconv_reset(None) == S.SKIPCONV_E_STATE
    assert lib.skipconv_destroy(None) == S.SKIPCONV_OK
    assert lib.skipconv_set_eps(None, ctypes.c_float(1.0)) == S.SKIPCONV_E_STATE
    out = ctypes.c_void_p(1)
    d = good()
    assert lib.skipconv_create(ctypes.byref(d), None, None, 0, None, ctypes.byref(out)) == S.SKIPCONV_E_INVALID_ARG
    assert out.value is None
    assert lib.skipconv_create(None, None, None, 0, None, None) == S.SKIPCONV_E_INVALID_ARG
    for c in range(-6, 1):
        assert S.skipconv_status_string(c) not in ("", "unknown status")
    assert lib.skipconv_workspace_size(ctypes.byref(d), None) == S.SKIPCONV_E_INVALID_ARG
