"""ctypes binding of libskipconv.so (include/skipconv.h), plus a torch-facing layer class.

The functions below carry the C names and only marshal arguments; every step
of the layer runs in the HIP kernels of the library. PyTorch provides device
memory (the workspace, inputs) and the stream. If the library is not built,
loading raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libskipconv.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "skipconv.h")

SKIPCONV_OK = 0
SKIPCONV_E_INVALID_ARG = -1
SKIPCONV_E_UNSUPPORTED = -2
SKIPCONV_E_OOM = -3
SKIPCONV_E_HIP = -4
SKIPCONV_E_STATE = -5
SKIPCONV_E_SMALL_BUFFER = -6

SKIPCONV_F32, SKIPCONV_BF16 = 0, 1
SKIPCONV_SUPPORT_RF, SKIPCONV_SUPPORT_CENTRE = 0, 1
SKIPCONV_GATE_INPUT_NORM, SKIPCONV_GATE_OUTPUT_NORM, SKIPCONV_GATE_LEARNED = 0, 1, 2
SKIPCONV_ACT_NONE, SKIPCONV_ACT_IDENTITY, SKIPCONV_ACT_RELU = 0, 1, 2
SKIPCONV_FLAG_KEEP_STATS, SKIPCONV_FLAG_FORCE_DENSE, SKIPCONV_FLAG_SPLIT_PIPELINE = 1, 2, 4
SKIPCONV_FLAG_EMIT_RESIDUAL = 8
SKIPCONV_FLAG_TRANSLATE = 16
SKIPCONV_FLAG_LARGE_GATE_TILES = 32
SKIPCONV_FLAG_CALLER_RETAINS = 64


class skipconv_desc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32),
                ("c_in", ctypes.c_int32), ("c_out", ctypes.c_int32), ("kernel", ctypes.c_int32),
                ("stride", ctypes.c_int32), ("pad", ctypes.c_int32), ("groups", ctypes.c_int32),
                ("block", ctypes.c_int32), ("norm_p", ctypes.c_int32), ("support", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("act_out", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("eps", ctypes.c_float), ("gate", ctypes.c_int32)]


class SkipConvError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"skipconv error {code}: {msg}")
        self.code = code


_lib = None
_P = ctypes.c_void_p
_D = ctypes.POINTER(skipconv_desc)
_SIGS = {
    "skipconv_desc_init": (ctypes.c_int, [_D]),
    "skipconv_validate": (ctypes.c_int, [_D]),
    "skipconv_out_shape": (ctypes.c_int, [_D] + [ctypes.POINTER(ctypes.c_int32)] * 4),
    "skipconv_workspace_size": (ctypes.c_int, [_D, ctypes.POINTER(ctypes.c_size_t)]),
    "skipconv_create": (ctypes.c_int, [_D, _P, _P, ctypes.c_size_t, _P, ctypes.POINTER(_P)]),
    "skipconv_step": (ctypes.c_int, [_P, _P, _P, ctypes.POINTER(_P)]),
    "skipconv_step_chained": (ctypes.c_int, [_P, _P, _P, ctypes.POINTER(_P)]),
    "skipconv_step_translated": (ctypes.c_int, [_P, _P, ctypes.c_int32, ctypes.c_int32, _P, ctypes.POINTER(_P)]),
    "skipconv_step_static": (ctypes.c_int, [_D, _P, _P, _P, _P, _P]),
    "skipconv_reset": (ctypes.c_int, [_P]),
    "skipconv_set_eps": (ctypes.c_int, [_P, ctypes.c_float]),
    "skipconv_set_gate_weights": (ctypes.c_int, [_P, _P, ctypes.c_float, _P]),
    "skipconv_destroy": (ctypes.c_int, [_P]),
    "skipconv_activation": (ctypes.c_int, [_P, ctypes.POINTER(_P)]),
    "skipconv_get_desc": (ctypes.c_int, [_P, _D]),
    "skipconv_pipeline": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_int32)]),
    "skipconv_gate_tile": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)]),
    "skipconv_conv_kernel": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_int32)]),
    "skipconv_active_count": (ctypes.c_int, [_P, _P, ctypes.POINTER(ctypes.c_int64),
                                             ctypes.POINTER(ctypes.c_int64)]),
    "skipconv_copy_block_mask": (ctypes.c_int, [_P, _P, _P, ctypes.c_size_t]),
    "skipconv_copy_active_list": (ctypes.c_int, [_P, _P, _P, ctypes.c_size_t,
                                                 ctypes.POINTER(ctypes.c_int64)]),
    "skipconv_copy_work_list": (ctypes.c_int, [_P, _P, _P, ctypes.c_size_t,
                                                 ctypes.POINTER(ctypes.c_int64)]),
    "skipconv_copy_site_mask": (ctypes.c_int, [_P, _P, _P, ctypes.c_size_t]),
    "skipconv_copy_stat": (ctypes.c_int, [_P, _P, _P, ctypes.c_size_t]),
    "skipconv_frame_macs": (ctypes.c_int, [_P, _P, ctypes.POINTER(ctypes.c_uint64),
                                           ctypes.POINTER(ctypes.c_uint64)]),
    "skipconv_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "skipconv_last_error": (ctypes.c_char_p, [_P]),
    "skipconv_timing_begin": (ctypes.c_int, [_P, ctypes.c_int, ctypes.c_int]),
    "skipconv_timing_read": (ctypes.c_int, [_P, _P, ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_int), _P, ctypes.c_int]),
}


def lib() -> ctypes.CDLL:
    """Load libskipconv.so (raises if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2104_11487_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def header_symbols():
    """Function names declared in include/skipconv.h."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(skipconv_[a-z_]+)\s*\(", text)))


def _check(code: int, handle=None) -> int:
    if code != SKIPCONV_OK:
        msg = lib().skipconv_last_error(handle).decode()
        raise SkipConvError(code, f"{lib().skipconv_status_string(code).decode()}: {msg}")
    return code


# ------------------------------------------------------------------ C names --

def skipconv_desc_init() -> skipconv_desc:
    d = skipconv_desc()
    _check(lib().skipconv_desc_init(ctypes.byref(d)))
    return d


def skipconv_validate(d: skipconv_desc) -> int:
    return lib().skipconv_validate(ctypes.byref(d))


def skipconv_out_shape(d: skipconv_desc) -> Tuple[int, int, int, int]:
    v = [ctypes.c_int32() for _ in range(4)]
    _check(lib().skipconv_out_shape(ctypes.byref(d), *[ctypes.byref(x) for x in v]))
    return tuple(x.value for x in v)


def skipconv_workspace_size(d: skipconv_desc) -> int:
    n = ctypes.c_size_t()
    _check(lib().skipconv_workspace_size(ctypes.byref(d), ctypes.byref(n)))
    return n.value


def skipconv_create(d: skipconv_desc, weights_ptr: int, workspace_ptr: Optional[int],
                    workspace_bytes: int, stream: int) -> int:
    h = ctypes.c_void_p()
    _check(lib().skipconv_create(ctypes.byref(d), weights_ptr, workspace_ptr, workspace_bytes, stream,
                                 ctypes.byref(h)))
    return h.value


def skipconv_step(h: int, x_ptr: int, stream: int) -> int:
    z = ctypes.c_void_p()
    _check(lib().skipconv_step(h, x_ptr, stream, ctypes.byref(z)), h)
    return z.value


def skipconv_step_static(d: skipconv_desc, weights_ptr: int, x_ptr: int, x_prev_ptr: Optional[int],
                         z_ptr: int, stream: int) -> None:
    _check(lib().skipconv_step_static(ctypes.byref(d), weights_ptr, x_ptr, x_prev_ptr, z_ptr, stream))


def skipconv_step_chained(h: int, up: int, stream: int) -> int:
    z = ctypes.c_void_p()
    _check(lib().skipconv_step_chained(h, up, stream, ctypes.byref(z)), h)
    return z.value


def skipconv_step_translated(h: int, x_ptr: int, dy: int, dx: int, stream: int) -> int:
    z = ctypes.c_void_p()
    _check(lib().skipconv_step_translated(h, x_ptr, dy, dx, stream, ctypes.byref(z)), h)
    return z.value


def skipconv_reset(h: int) -> None:
    _check(lib().skipconv_reset(h), h)


def skipconv_set_eps(h: int, eps: float) -> None:
    _check(lib().skipconv_set_eps(h, eps), h)


def skipconv_set_gate_weights(h: int, phi_ptr: int, bias: float, stream: int) -> None:
    _check(lib().skipconv_set_gate_weights(h, phi_ptr, bias, stream), h)


def skipconv_destroy(h: int) -> None:
    _check(lib().skipconv_destroy(h))


def skipconv_activation(h: int) -> int:
    y = ctypes.c_void_p()
    _check(lib().skipconv_activation(h, ctypes.byref(y)), h)
    return y.value


def skipconv_get_desc(h: int) -> skipconv_desc:
    d = skipconv_desc()
    _check(lib().skipconv_get_desc(h, ctypes.byref(d)), h)
    return d


def skipconv_pipeline(h: int) -> int:
    f = ctypes.c_int32()
    _check(lib().skipconv_pipeline(h, ctypes.byref(f)), h)
    return f.value


def skipconv_gate_tile(h: int) -> Tuple[int, int]:
    ts, ls = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().skipconv_gate_tile(h, ctypes.byref(ts), ctypes.byref(ls)), h)
    return ts.value, ls.value


def skipconv_conv_kernel(h: int) -> int:
    k = ctypes.c_int32()
    _check(lib().skipconv_conv_kernel(h, ctypes.byref(k)), h)
    return k.value


def skipconv_active_count(h: int, stream: int) -> Tuple[int, int]:
    b, s = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().skipconv_active_count(h, stream, ctypes.byref(b), ctypes.byref(s)), h)
    return b.value, s.value


def _np_buf(arr):
    return arr.ctypes.data_as(ctypes.c_void_p), arr.nbytes


def skipconv_copy_block_mask(h: int, stream: int, out) -> None:
    p, n = _np_buf(out)
    _check(lib().skipconv_copy_block_mask(h, stream, p, n), h)


def skipconv_copy_active_list(h: int, stream: int, out) -> int:
    p, _ = _np_buf(out)
    cnt = ctypes.c_int64()
    _check(lib().skipconv_copy_active_list(h, stream, p, out.size, ctypes.byref(cnt)), h)
    return cnt.value


def skipconv_copy_work_list(h: int, stream: int, out) -> int:
    p, _ = _np_buf(out)
    cnt = ctypes.c_int64()
    _check(lib().skipconv_copy_work_list(h, stream, p, out.size, ctypes.byref(cnt)), h)
    return cnt.value


def skipconv_copy_site_mask(h: int, stream: int, out) -> None:
    p, n = _np_buf(out)
    _check(lib().skipconv_copy_site_mask(h, stream, p, n), h)


def skipconv_copy_stat(h: int, stream: int, out) -> None:
    p, n = _np_buf(out)
    _check(lib().skipconv_copy_stat(h, stream, p, n), h)


def skipconv_frame_macs(h: int, stream: int) -> Tuple[int, int]:
    d, a = ctypes.c_uint64(), ctypes.c_uint64()
    _check(lib().skipconv_frame_macs(h, stream, ctypes.byref(d), ctypes.byref(a)), h)
    return d.value, a.value


def skipconv_status_string(code: int) -> str:
    return lib().skipconv_status_string(code).decode()


def skipconv_last_error(h: Optional[int] = None) -> str:
    return lib().skipconv_last_error(h).decode()


def skipconv_timing_begin(h: int, frames: int, every: int = 1) -> None:
    _check(lib().skipconv_timing_begin(h, frames, every), h)


def skipconv_timing_read(h: int, stream: int, capacity: int = 0):
    """(gate ms, conv ms, timed steps, their indices since timing_begin)."""
    import numpy as np
    ms = (ctypes.c_double * 2)()
    n = ctypes.c_int()
    idx = np.zeros(max(capacity, 1), np.int32)
    _check(lib().skipconv_timing_read(h, stream, ms, ctypes.byref(n),
                                      idx.ctypes.data_as(ctypes.c_void_p) if capacity else None,
                                      capacity), h)
    return ms[0], ms[1], n.value, idx[:n.value].copy() if capacity else None


# ----------------------------------------------------------- torch layer ----

_SUPPORT = {"rf": SKIPCONV_SUPPORT_RF, "centre": SKIPCONV_SUPPORT_CENTRE}
_ACT = {"none": SKIPCONV_ACT_NONE, "identity": SKIPCONV_ACT_IDENTITY, "relu": SKIPCONV_ACT_RELU}
_GATE = {"input": SKIPCONV_GATE_INPUT_NORM, "output": SKIPCONV_GATE_OUTPUT_NORM,
         "learned": SKIPCONV_GATE_LEARNED}


def make_desc(*, n, h, w, c_in, c_out, kernel, stride=1, pad=-1, groups=1, block=1, norm_p=2,
              support="rf", dtype="f32", act_out="none", eps=0.0, keep_stats=False,
              force_dense=False, split=False, gate="input", emit_residual=False,
              translate=False, large_gate_tiles=False, caller_retains=False) -> skipconv_desc:
    d = skipconv_desc_init()
    d.n, d.h, d.w, d.c_in, d.c_out = n, h, w, c_in, c_out
    d.kernel, d.stride, d.pad, d.groups, d.block = kernel, stride, pad, groups, block
    d.norm_p, d.support = norm_p, _SUPPORT[support]
    d.dtype = SKIPCONV_BF16 if dtype == "bf16" else SKIPCONV_F32
    d.act_out = _ACT[act_out]
    d.flags = ((SKIPCONV_FLAG_KEEP_STATS if keep_stats else 0) | (SKIPCONV_FLAG_FORCE_DENSE if force_dense else 0)
               | (SKIPCONV_FLAG_SPLIT_PIPELINE if split else 0)
               | (SKIPCONV_FLAG_EMIT_RESIDUAL if emit_residual else 0)
               | (SKIPCONV_FLAG_TRANSLATE if translate else 0)
               | (SKIPCONV_FLAG_LARGE_GATE_TILES if large_gate_tiles else 0)
               | (SKIPCONV_FLAG_CALLER_RETAINS if caller_retains else 0))
    d.eps = eps
    d.gate = _GATE[gate]
    return d


class SkipConv:
    """One streaming Skip-Conv layer on the current GPU.

    weight: CUDA tensor, OIHW, float32 or bfloat16 (the layer dtype).
    step(x) takes an N x H x W x C_in tensor of the layer dtype and returns the
    persistent fp32 state z (N x H_out x W_out x C_out), a view that the next
    step overwrites.

    caller_retains: the next step reads this step's x as x_{t-1} instead of a
    copy in the workspace (no copy is written). The object keeps a reference
    to the last frame so that its memory is not reused; the caller must not
    modify it in place before the next step, and passes a new tensor each step.
    """

    def __init__(self, weight, *, n: int, h: int, w: int, stride: int = 1, pad: int = -1,
                 groups: int = 1, eps: float = 0.0, block: int = 1, norm_p: int = 2,
                 support: str = "rf", act_out: str = "none", keep_stats: bool = False,
                 force_dense: bool = False, split: bool = False, gate: str = "input",
                 emit_residual: bool = False, translate: bool = False, large_gate_tiles: bool = False,
                 caller_retains: bool = False, stream=None):
        import torch

        if not weight.is_cuda:
            raise ValueError("weight must be a GPU tensor")
        if weight.dtype not in (torch.float32, torch.bfloat16):
            raise ValueError("weight dtype must be float32 or bfloat16")
        self.torch = torch
        self.dtype = "bf16" if weight.dtype == torch.bfloat16 else "f32"
        self.tdtype = weight.dtype
        c_out, cg, k, _ = weight.shape
        self.desc = make_desc(n=n, h=h, w=w, c_in=cg * groups, c_out=c_out, kernel=k, stride=stride,
                              pad=pad, groups=groups, block=block, norm_p=norm_p, support=support,
                              dtype=self.dtype, act_out=act_out, eps=eps, keep_stats=keep_stats, gate=gate,
                              force_dense=force_dense, split=split, emit_residual=emit_residual,
                              translate=translate, large_gate_tiles=large_gate_tiles,
                              caller_retains=caller_retains)
        self.h_out, self.w_out, self.hb, self.wb = skipconv_out_shape(self.desc)
        nbytes = skipconv_workspace_size(self.desc)
        self.device = weight.device
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=weight.device)
        self._weight = weight.contiguous()
        self.stream = stream
        self.handle = skipconv_create(self.desc, self._weight.data_ptr(), self.workspace.data_ptr(),
                                      nbytes, self._stream())
        self._z = None
        self._zp = None
        self._y = None
        self._prev_x = None  # caller_retains: the frame the next step reads as x_{t-1}

    def _stream(self) -> int:
        s = self.stream if self.stream is not None else self.torch.cuda.current_stream(self.device)
        return s.cuda_stream

    def _view(self, ptr: int, numel: int, dtype):
        off = ptr - self.workspace.data_ptr()
        esz = self.torch.tensor([], dtype=dtype).element_size()
        v = self.workspace[off:off + numel * esz].view(dtype)
        return v.view(self.desc.n, self.h_out, self.w_out, self.desc.c_out)

    @property
    def shape_in(self):
        d = self.desc
        return (d.n, d.h, d.w, d.c_in)

    def step(self, x):
        if tuple(x.shape) != self.shape_in or x.dtype != self.tdtype or not x.is_contiguous() \
                or x.device != self.device:
            raise ValueError(f"x must be a contiguous {self.tdtype} tensor of shape {self.shape_in} on {self.device}")
        z = self._z_view(skipconv_step(self.handle, x.data_ptr(), self._stream()))
        self._retain(x)
        return z

    def _retain(self, x):
        if self.desc.flags & SKIPCONV_FLAG_CALLER_RETAINS:
            self._prev_x = x

    def _z_view(self, zp: int):
        # the state pointer is fixed except across translated steps (two z slots)
        if self._z is None or zp != self._zp:
            self._z = self._view(zp, self.desc.n * self.h_out * self.w_out * self.desc.c_out,
                                 self.torch.float32)
            self._zp = zp
        return self._z

    def step_translated(self, x, dy: int, dx: int):
        """One frame whose content moved by (dy, dx) pixels since the previous one (Sec. 3.3)."""
        if tuple(x.shape) != self.shape_in or x.dtype != self.tdtype or not x.is_contiguous() \
                or x.device != self.device:
            raise ValueError(f"x must be a contiguous {self.tdtype} tensor of shape {self.shape_in} on {self.device}")
        z = self._z_view(skipconv_step_translated(self.handle, x.data_ptr(), dy, dx, self._stream()))
        self._retain(x)
        return z

    def step_chained(self, upstream: "SkipConv"):
        """One frame whose input is `upstream`'s activation output (upstream stepped first).

        `upstream` must have been created with emit_residual=True; see
        skipconv_step_chained for the contract.
        """
        return self._z_view(skipconv_step_chained(self.handle, upstream.handle, self._stream()))

    def activation(self):
        if self._y is None:
            yp = skipconv_activation(self.handle)
            self._y = self._view(yp, self.desc.n * self.h_out * self.w_out * self.desc.c_out, self.tdtype)
        return self._y

    def reset(self):
        skipconv_reset(self.handle)
        self._prev_x = None

    @property
    def fused(self) -> bool:
        return bool(skipconv_pipeline(self.handle))

    @property
    def fused_variant(self) -> int:
        """0 split pipeline, 1 single-pass kernel with LDS weights, 2 with register weights,
        3 with register weights and the output channels split over workgroups, 4 single-pass
        depthwise kernel, 5 single-pass kernel for few input channels."""
        return skipconv_pipeline(self.handle)

    @property
    def gate_tile(self) -> Tuple[int, int]:
        """(sites per side of a gate tile, 1 if chunk sums are combined in lane groups)."""
        return skipconv_gate_tile(self.handle)

    @property
    def conv_kernel(self) -> int:
        """Split-pipeline convolution kernel: 0 gather, 1 block halo, 2 depthwise per site, 3 depthwise halo."""
        return skipconv_conv_kernel(self.handle)

    def set_eps(self, eps: float):
        skipconv_set_eps(self.handle, eps)
        self.desc.eps = eps

    def set_gate_weights(self, phi, bias: float = 0.0):
        """Learned gate (Eq. 8): phi is a float32 GPU tensor of C_in x k x k (or 1 x C_in x k x k)."""
        t = self.torch
        if not phi.is_cuda or phi.dtype != t.float32 or phi.numel() != self.desc.c_in * self.desc.kernel ** 2:
            raise ValueError("phi must be a float32 GPU tensor of c_in x k x k elements")
        phi = phi.contiguous()
        skipconv_set_gate_weights(self.handle, phi.data_ptr(), bias, self._stream())
        self._phi = phi  # keep the source alive until the repack has run

    def active_count(self) -> Tuple[int, int]:
        return skipconv_active_count(self.handle, self._stream())

    def block_mask(self):
        import numpy as np
        out = np.empty((self.desc.n, self.hb, self.wb), np.uint8)
        skipconv_copy_block_mask(self.handle, self._stream(), out)
        return out

    def active_list(self):
        import numpy as np
        out = np.empty(self.desc.n * self.hb * self.wb, np.uint32)
        cnt = skipconv_copy_active_list(self.handle, self._stream(), out)
        return out[:cnt].copy()

    def work_list(self):
        """Active blocks the last split-pipeline step's convolution walked, in append order."""
        import numpy as np
        out = np.empty(self.desc.n * self.hb * self.wb, np.uint32)
        cnt = skipconv_copy_work_list(self.handle, self._stream(), out)
        return out[:cnt].copy()

    def site_mask(self):
        import numpy as np
        out = np.empty((self.desc.n, self.h_out, self.w_out), np.uint8)
        skipconv_copy_site_mask(self.handle, self._stream(), out)
        return out

    def stat(self):
        import numpy as np
        out = np.empty((self.desc.n, self.h_out, self.w_out), np.float32)
        skipconv_copy_stat(self.handle, self._stream(), out)
        return out

    def frame_macs(self) -> Tuple[int, int]:
        return skipconv_frame_macs(self.handle, self._stream())

    def close(self):
        if getattr(self, "handle", None):
            skipconv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
