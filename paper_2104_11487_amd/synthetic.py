"""Seeded synthetic video and weights for the Skip-Conv layer workloads.

The paper measures on UA-DETRAC (Sec. 4.1) and JHMDB (Sec. 4.2); neither is
available here, so every workload is a seeded synthetic stand-in with the
structure those streams have: a static (or slowly varying) background and a
few moving foreground objects, which is what makes residual frames sparse
(Sec. 3.1).

This module holds no arithmetic of the method: it only draws frames and
weights. Frames are float32 NHWC; ``to_storage`` casts them to the storage
dtype (bf16 through torch's round-to-nearest-even cast) and returns the raw
bits (uint16) for bf16, so the GPU path and the CPU oracle receive identical
bytes. Both sides import this module; neither imports the other.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Iterator, List, Optional

import numpy as np


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Cast a float32 array to the storage dtype: 'f32' -> float32, 'bf16' -> uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "f32":
        return x
    if dtype == "bf16":
        import torch

        t = torch.from_numpy(x).to(torch.bfloat16)
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    raise ValueError(f"unknown dtype {dtype!r}")


def he_weights(c_out: int, c_in_per_group: int, k: int, seed: int,
               fan_in: Optional[int] = None) -> np.ndarray:
    """He-normal OIHW float32 weights, variance 2 / fan_in (fan_in = k*k*c_in/g)."""
    fan = fan_in if fan_in is not None else k * k * c_in_per_group
    rng = _rng(seed)
    w = rng.normal(0.0, math.sqrt(2.0 / fan), size=(c_out, c_in_per_group, k, k))
    return w.astype(np.float32)


def integer_weights(c_out: int, c_in_per_group: int, k: int, seed: int, lo: int = -2,
                    hi: int = 2) -> np.ndarray:
    """Small-integer weights: every product and partial sum is exact in fp32/bf16."""
    rng = _rng(seed)
    return rng.integers(lo, hi + 1, size=(c_out, c_in_per_group, k, k)).astype(np.float32)


# ----------------------------------------------------------------------------
# 3x3 16->16 fp32 layer, 32x32 frames: static uniform texture plus one 6x6
# square of random per-channel values moving one pixel per frame to the
# right, with N(0, 0.01) noise (variance 0.01) redrawn on the square each frame.
# ----------------------------------------------------------------------------

def square_video(h: int = 32, w: int = 32, c: int = 16, frames: int = 8, seed: int = 101,
                 side: int = 6, start=(13, 4), noise_var: float = 0.01) -> np.ndarray:
    rng = _rng(seed)
    bg = rng.random((h, w, c), dtype=np.float32)
    vals = rng.random(c, dtype=np.float32)
    out = np.empty((frames, 1, h, w, c), np.float32)
    for t in range(frames):
        f = bg.copy()
        r0, c0 = start[0], start[1] + t
        noise = rng.normal(0.0, math.sqrt(noise_var), size=(side, side, c)).astype(np.float32)
        r1, c1 = min(r0 + side, h), min(c0 + side, w)
        f[r0:r1, c0:c1, :] = (vals + noise)[: r1 - r0, : c1 - c0]
        out[t, 0] = f
    return out


# ----------------------------------------------------------------------------
# Moving textured rectangles over a static noise background, with temporal
# sensor noise on every pixel and optional one-frame camera shake.
# ----------------------------------------------------------------------------

@dataclass
class _Rect:
    h: int
    w: int
    y: int
    x: int
    vy: int
    vx: int
    tex: np.ndarray


def _bounce(pos: int, vel: int, lo: int, hi: int):
    pos += vel
    if pos < lo:
        pos, vel = 2 * lo - pos, -vel
    if pos > hi:
        pos, vel = 2 * hi - pos, -vel
    return max(lo, min(hi, pos)), vel


@dataclass
class RectVideo:
    """Stream of frames (batch, H, W, C) float32; frames are drawn in order."""

    h: int
    w: int
    c: int
    frames: int
    seed: int
    batch: int = 1
    n_rect: int = 4
    side_lo: int = 8
    side_hi: int = 32
    speeds=(1, 2, 3)
    noise_std: float = 0.02
    shake_prob: float = 0.0
    shake_frames: List[int] = field(default_factory=list)

    def __iter__(self) -> Iterator[np.ndarray]:
        rng = _rng(self.seed)
        bgs, rects = [], []
        for _ in range(self.batch):
            bgs.append(rng.random((self.h, self.w, self.c), dtype=np.float32))
            rs = []
            for _ in range(self.n_rect):
                rh = int(rng.integers(self.side_lo, self.side_hi + 1))
                rw = int(rng.integers(self.side_lo, self.side_hi + 1))
                rh, rw = min(rh, self.h), min(rw, self.w)
                tex = rng.random((rh, rw, self.c), dtype=np.float32)
                y = int(rng.integers(0, self.h - rh + 1))
                x = int(rng.integers(0, self.w - rw + 1))
                vy = int(rng.choice(self.speeds)) * int(rng.choice([-1, 1]))
                vx = int(rng.choice(self.speeds)) * int(rng.choice([-1, 1]))
                rs.append(_Rect(rh, rw, y, x, vy, vx, tex))
            rects.append(rs)
        self.shake_frames = []
        self.shake_shift = {}  # frame -> (dy, dx): that frame's content moved by (dy, dx)
        for t in range(self.frames):
            out = np.empty((self.batch, self.h, self.w, self.c), np.float32)
            shake = None
            if self.shake_prob > 0.0:
                u = rng.random()
                d = rng.integers(-1, 2, size=2)
                if t > 0 and u < self.shake_prob:
                    shake = (int(d[0]), int(d[1]))
                    self.shake_frames.append(t)
                    self.shake_shift[t] = shake
            for n in range(self.batch):
                f = bgs[n] + rng.normal(0.0, self.noise_std,
                                        size=(self.h, self.w, self.c)).astype(np.float32)
                for r in rects[n]:
                    f[r.y:r.y + r.h, r.x:r.x + r.w, :] = r.tex
                if shake is not None:
                    dy, dx = shake
                    ys = np.clip(np.arange(self.h) - dy, 0, self.h - 1)
                    xs = np.clip(np.arange(self.w) - dx, 0, self.w - 1)
                    f = f[ys][:, xs]
                out[n] = f
                for r in rects[n]:
                    r.y, r.vy = _bounce(r.y, r.vy, 0, self.h - r.h)
                    r.x, r.vx = _bounce(r.x, r.vx, 0, self.w - r.w)
            yield out

    def all(self) -> np.ndarray:
        return np.stack(list(iter(self)))


# ----------------------------------------------------------------------------
# Gaussian blobs over a static texture with a drifting illumination ramp; one
# independent stream per batch entry (seed base + n).
# ----------------------------------------------------------------------------

@dataclass
class BlobVideo:
    h: int = 512
    w: int = 512
    c: int = 128
    frames: int = 64
    seed_base: int = 500
    batch: int = 4
    n_blobs: int = 16
    bg_scale: float = 0.5
    ramp_amp: float = 0.2
    ramp_drift: float = 0.002
    ramp_rot_deg: float = 0.5

    def _stream(self, n: int) -> Iterator[np.ndarray]:
        rng = _rng(self.seed_base + n)
        bg = rng.random((self.h, self.w, self.c), dtype=np.float32) * np.float32(self.bg_scale)
        theta0 = float(rng.random()) * 2.0 * math.pi
        blobs = []
        for _ in range(self.n_blobs):
            sigma = float(rng.uniform(4.0, 24.0))
            amp = rng.uniform(0.5, 1.0, size=self.c).astype(np.float32)
            py, px = float(rng.uniform(0, self.h)), float(rng.uniform(0, self.w))
            vy, vx = float(rng.uniform(-3.0, 3.0)), float(rng.uniform(-3.0, 3.0))
            blobs.append([sigma, amp, py, px, vy, vx])
        yy = np.arange(self.h, dtype=np.float32)[:, None]
        xx = np.arange(self.w, dtype=np.float32)[None, :]
        for t in range(self.frames):
            th = theta0 + math.radians(self.ramp_rot_deg) * t
            ramp = (np.float32(self.ramp_amp) * (xx * np.float32(math.cos(th)) + yy * np.float32(math.sin(th)))
                    / np.float32(max(self.h, self.w)) + np.float32(self.ramp_drift * t))
            f = bg + ramp[:, :, None]
            for b in blobs:
                sigma, amp, py, px = b[0], b[1], b[2], b[3]
                rad = int(math.ceil(3.0 * sigma))
                y0, y1 = max(0, int(py) - rad), min(self.h, int(py) + rad + 1)
                x0, x1 = max(0, int(px) - rad), min(self.w, int(px) + rad + 1)
                if y0 >= y1 or x0 >= x1:
                    continue
                dy = np.arange(y0, y1, dtype=np.float32)[:, None] - np.float32(py)
                dx = np.arange(x0, x1, dtype=np.float32)[None, :] - np.float32(px)
                prof = np.exp(-(dy * dy + dx * dx) / np.float32(2.0 * sigma * sigma)).astype(np.float32)
                f[y0:y1, x0:x1, :] += prof[:, :, None] * amp[None, None, :]
            yield f.astype(np.float32)
            for b in blobs:
                for ax, lim in ((2, self.h), (3, self.w)):
                    p, v = b[ax] + b[ax + 2], b[ax + 2]
                    if p < 0:
                        p, v = -p, -v
                    if p > lim - 1:
                        p, v = 2 * (lim - 1) - p, -v
                    b[ax], b[ax + 2] = p, v

    def __iter__(self) -> Iterator[np.ndarray]:
        streams = [self._stream(n) for n in range(self.batch)]
        for _ in range(self.frames):
            yield np.stack([next(s) for s in streams])


# ----------------------------------------------------------------------------
# Named workloads (shapes and seeds). Each entry lists the layers of the
# workload; 'video' builds the frame iterator.
# ----------------------------------------------------------------------------

@dataclass
class LayerSpec:
    c_in: int
    c_out: int
    k: int
    stride: int
    groups: int
    weight_seed: int


@dataclass
class Workload:
    name: str
    dtype: str
    n: int
    h: int
    w: int
    c: int
    frames: int
    layers: List[LayerSpec]
    block: int
    act: str  # activation between layers: 'none' or 'relu'

    def video(self, frames: Optional[int] = None):
        t = self.frames if frames is None else frames
        if self.name == "square16":
            return iter(square_video(self.h, self.w, self.c, t))
        if self.name == "rect64":
            return iter(RectVideo(self.h, self.w, self.c, t, seed=201, batch=self.n))
        if self.name == "mbconv192":
            return iter(RectVideo(self.h, self.w, self.c, t, seed=301, batch=self.n, shake_prob=0.1))
        if self.name == "stack6":
            return iter(RectVideo(self.h, self.w, self.c, t, seed=401, batch=self.n))
        if self.name == "blob128":
            return iter(BlobVideo(self.h, self.w, self.c, t, batch=self.n))
        raise KeyError(self.name)

    def weights(self) -> List[np.ndarray]:
        return [he_weights(l.c_out, l.c_in // l.groups, l.k, l.weight_seed) for l in self.layers]


def workloads() -> dict:
    """The five single-GPU workloads, by name."""
    return {
        "square16": Workload("square16", "f32", 1, 32, 32, 16, 8,
                             [LayerSpec(16, 16, 3, 1, 1, 102)], 1, "none"),
        "rect64": Workload("rect64", "bf16", 1, 128, 96, 64, 32,
                           [LayerSpec(64, 64, 3, 1, 1, 202)], 8, "none"),
        "mbconv192": Workload("mbconv192", "bf16", 1, 64, 64, 192, 32,
                              [LayerSpec(192, 192, 1, 1, 1, 302),
                               LayerSpec(192, 192, 3, 1, 192, 303)], 8, "none"),
        "stack6": Workload("stack6", "bf16", 1, 256, 192, 3, 64,
                           [LayerSpec(3, 32, 3, 1, 1, 402), LayerSpec(32, 64, 3, 2, 1, 412),
                            LayerSpec(64, 64, 3, 1, 1, 422), LayerSpec(64, 128, 3, 2, 1, 432),
                            LayerSpec(128, 128, 3, 1, 1, 442), LayerSpec(128, 128, 3, 1, 1, 452)],
                           1, "relu"),
        "blob128": Workload("blob128", "bf16", 4, 512, 512, 128, 64,
                            [LayerSpec(128, 128, 3, 1, 1, 509)], 16, "none"),
    }


def eps_schedule(n_layers: int, seed: int = 403) -> np.ndarray:
    """Per-layer multipliers 10**u, u ~ U(-0.5, 0.5), for a layer-specific threshold."""
    rng = _rng(seed)
    return (10.0 ** rng.uniform(-0.5, 0.5, size=n_layers)).astype(np.float64)
