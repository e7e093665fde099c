"""Benchmark of the streaming Skip-Conv layer on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]
                    [--workload blob128|rect64|square16|stack6|mbconv192]

One step = one call of skipconv_step on one batch (the whole hot path) over a
frame of the synthetic clip; the clip repeats with a reset (dense reference
frame) at its first frame. Inputs are resident in HBM before the timed
region. The timed region starts right after a reference frame, so K steps
up to the clip length are steady-state frames; the reference frame is timed
on its own. Prints one JSON line.

Default workload (blob128): 3x3 conv 128 -> 128, bf16 operands with fp32
accumulation, four independent 512 x 512 streams (one step = one frame of
each), a 64-frame clip of 16 moving Gaussian blobs over a static texture with
a drifting illumination ramp, 16 x 16 gate blocks, eps calibrated on the
GPU's own gate statistics to ~25 % block density. The sweep covers block
densities 5 / 10 / 25 / 50 / 75 %, eps = 0 and the same kernels forced dense,
each with the measured speed-up over forced dense printed beside the
roofline-model speed-up, plus the caller-retained-frames contract, the other
gate kinds and torch's conv2d (MIOpen) on the same shape for context.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Skip-Conv frames/s and active-site TFLOP/s (% MFMA/HBM peak) vs gate density"
PEAK_BF16_TFLOPS = 2500.0
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


# --------------------------------------------------------------- workloads --

def load_workload(name: str, frames: int | None):
    from paper_2104_11487_amd import synthetic as syn

    wl = syn.workloads()[name]
    nfr = frames or wl.frames
    t0 = time.time()
    clip = [syn.to_storage(f, wl.dtype) for f in wl.video(nfr)]
    log(f"[bench] generated {len(clip)} frames of {wl.name} in {time.time() - t0:.1f}s")
    return wl, clip


def upload(clip, dtype):
    import torch

    out = []
    for x in clip:
        if dtype == "bf16":
            out.append(torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16))
        else:
            out.append(torch.from_numpy(x).cuda())
    return out


def weight_tensor(w32, dtype):
    import torch

    t = torch.from_numpy(w32).cuda()
    return t.to(torch.bfloat16) if dtype == "bf16" else t


# ------------------------------------------------------------- calibration --

def gpu_stats(layer_kw, wt, frames_dev):
    """Per-frame gate statistics of frames 2.. from the GPU layer itself (KEEP_STATS)."""
    from paper_2104_11487_amd.skipconv import SkipConv
    import torch

    lay = SkipConv(wt, eps=0.0, block=1, keep_stats=True, **layer_kw)
    stats = []
    for t, x in enumerate(frames_dev):
        lay.step(x)
        if t > 0:
            torch.cuda.synchronize()
            stats.append(lay.stat())
    lay.close()
    return stats


def block_quantile(stats, block, h_out, w_out, target):
    """Value v such that about `target` of the blocks have a site statistic above v."""
    vals = []
    for s in stats:
        n = s.shape[0]
        hb, wb = -(-h_out // block), -(-w_out // block)
        pad = np.full((n, hb * block, wb * block), -np.inf, np.float32)
        pad[:, :h_out, :w_out] = np.nan_to_num(s, nan=np.inf)
        vals.append(pad.reshape(n, hb, block, wb, block).max(axis=(2, 4)).reshape(-1))
    v = np.concatenate(vals).astype(np.float64)
    return float(np.quantile(v, 1.0 - target))


def eps_for_density(stats, block, h_out, w_out, target):
    """Input-Norm eps (p = 2: the statistic is compared with eps^2) for about `target` block density."""
    return float(np.sqrt(max(block_quantile(stats, block, h_out, w_out, target), 0.0)))


# ------------------------------------------------------------------ timing --

def run_steps(layer, frames_dev, steps, start, *, every=0, block=None):
    """Run `steps` steps from clip position `start` (reset at each clip start).

    With every > 0, HIP events (recorded by the library on the launch stream)
    bracket both kernels of every `every`-th step. With block = (period, length),
    a HIP event pair on the launch stream brackets `length` consecutive steps
    once every `period` steps, and the kernel time is the bracketed time over the
    launches inside (for a one-kernel step: duration plus the dispatch gap).
    Returns (wall seconds, gate ms, conv ms, clip positions of the timed launches,
    next position).
    """
    import torch
    from paper_2104_11487_amd import skipconv as S

    nfr = len(frames_dev)
    ntimed = (steps + every - 1) // every if every else 0
    if every:
        S.skipconv_timing_begin(layer.handle, ntimed, every)
    pairs, timed = [], []
    stream = layer.stream if layer.stream is not None else torch.cuda.current_stream()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    pos = start
    for j in range(steps):
        if pos % nfr == 0:
            layer.reset()
        opened = block is not None and j % block[0] == 0 and j + block[1] <= steps
        if opened:
            ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            ev[0].record(stream)
        layer.step(frames_dev[pos % nfr])
        if block is not None and j % block[0] < block[1] and j - j % block[0] + block[1] <= steps:
            timed.append(pos % nfr)
            if j % block[0] == block[1] - 1:
                ev[1].record(stream)
                pairs.append(ev)
        pos += 1
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gate_ms = conv_ms = 0.0
    timed_pos = np.zeros(0, np.int64)
    if every:
        gate_ms, conv_ms, n, idx = S.skipconv_timing_read(layer.handle, layer._stream(), ntimed)
        assert n == ntimed, (n, ntimed)
        timed_pos = (start + idx.astype(np.int64)) % nfr
        S.skipconv_timing_begin(layer.handle, 0, 1)
    elif pairs:
        gate_ms = float(sum(a.elapsed_time(b) for a, b in pairs))
        timed_pos = np.array(timed, np.int64)
    return wall, gate_ms, conv_ms, timed_pos, pos


def clip_active(layer, frames_dev):
    """Active sites and blocks of every clip position (one pass, reset at frame 0)."""
    sites, blocks = [], []
    layer.reset()
    for x in frames_dev:
        layer.step(x)
        b, s = layer.active_count()
        sites.append(s)
        blocks.append(b)
    return np.array(sites, np.int64), np.array(blocks, np.int64)


def event_period(nfr: int, steps: int) -> int:
    """Sampling period of the per-kernel events of the multi-kernel pipeline.

    Coprime with the clip length, so the sampled steps walk through every clip
    position; as long as possible (up to 17 steps: the event records, marker
    packets on the stream, then add little to the timed wall clock) while the
    timed steps still give at least two samples of every clip position.
    """
    for e in (17, 13, 11, 7, 5, 3, 2):
        if np.gcd(e, nfr) == 1 and steps // e >= 2 * nfr:
            return e
    return 1


def event_blocks(nfr: int, length: int = 16):
    """(period, length) of the bracketed runs of the one-kernel pipeline.

    Consecutive runs start length/2 clip positions apart, so together they
    cover the clip; one event pair per run keeps the marker cost per step small.
    """
    return 2 * nfr + length // 2, length


def measure_point(make_layer, frames_dev, steps, warmup, geom, *, label, events=True, retains=False):
    """Warm up, then time exactly `steps` steps; per-kernel times from HIP events on sampled steps."""
    layer = make_layer()
    fused = layer.fused
    sites, blocks = clip_active(layer, frames_dev)
    nfr = len(frames_dev)
    pos = nfr
    if warmup:
        _, _, _, _, pos = run_steps(layer, frames_dev, warmup, pos)
    # the timed steps start right after an untimed reference frame (clip position 0)
    pos = (pos + nfr - 1) // nfr * nfr
    _, _, _, _, pos = run_steps(layer, frames_dev, 1, pos)
    every = event_period(nfr, steps) if events and not fused else 0
    blk = event_blocks(nfr) if events and fused else None
    wall, gate_ms, conv_ms, tpos, _ = run_steps(layer, frames_dev, steps, pos, every=every, block=blk)
    ref_us = reference_us(layer, frames_dev[0]) if events else None
    layer.close()
    idx = (pos + np.arange(steps)) % nfr
    act_sites = sites[idx].astype(np.float64)
    macs_per_site = geom["c_out"] * geom["kk"]
    flops_active = 2.0 * act_sites.sum() * macs_per_site
    flops_dense = 2.0 * geom["sites"] * macs_per_site * steps
    nt = max(len(tpos), 1)
    # algorithmic work of the timed launches
    conv_flop = 2.0 * sites[tpos].sum() * macs_per_site / nt
    xb, nb = geom["x_bytes"], geom["nb"]
    ref = (tpos == 0)
    # x_t read (and copied unless the caller retains its frames), x_{t-1} read
    # except on a reference frame
    xio = np.where(ref, xb if retains else 2 * xb, 2 * xb if retains else 3 * xb)
    gate_bytes = (xio + 2 * nb + 4 * blocks[tpos]).sum() / nt
    # fused kernel: the same x traffic, z read-modify-written at active sites
    # (written only on a reference frame), weights, block flags
    zb = 4.0 * geom["c_out"] * sites[tpos]
    fused_bytes = (xio + np.where(ref, zb, 2 * zb) + nb + geom["w_bytes"]).sum() / nt
    gate_us = 1e3 * gate_ms / nt if len(tpos) else None
    conv_us = 1e3 * conv_ms / nt if len(tpos) else None
    res = {
        "label": label,
        "pipeline": "fused" if fused else "split",
        "ms_per_step": 1e3 * wall / steps,
        "frames_per_s": steps * geom["n"] / wall,
        "density": float(act_sites.sum() / (geom["sites"] * steps)),
        "density_steady": float(sites[1:].sum() / (geom["sites"] * (nfr - 1))),
        "active_tflops": flops_active / wall / 1e12,
        "dense_equiv_tflops": flops_dense / wall / 1e12,
        "gate_us": gate_us,
        "conv_us": conv_us,
        "timed_launches": int(len(tpos)),
        "event_period": every if every else None,
        "event_blocks": list(blk) if blk else None,
        "conv_flop_per_launch": conv_flop,
        "gate_bytes_per_launch": float(gate_bytes),
        "conv_active_tflops": conv_flop / (conv_us * 1e-6) / 1e12 if conv_us else None,
        "gate_gbs": gate_bytes / (gate_us * 1e-6) / 1e9 if gate_us else None,
        "fused_bytes_per_launch": float(fused_bytes) if fused else None,
        "reference_frame_us": ref_us,
        "active_sites_per_launch": float(sites[tpos].mean()) if len(tpos) else None,
    }
    if fused:
        log(f"[bench] {label}: {res['frames_per_s']:.0f} frames/s, {res['ms_per_step'] * 1e3:.1f} us/step, "
            f"density {res['density']:.3f}, fused kernel {gate_us or 0:.1f} us")
    else:
        log(f"[bench] {label}: {res['frames_per_s']:.0f} frames/s, {res['ms_per_step'] * 1e3:.1f} us/step, "
            f"density {res['density']:.3f}, gate {gate_us or 0:.1f} us, conv {conv_us or 0:.1f} us")
    return res


def reference_us(layer, frame, reps=3):
    """Median duration of a reference frame (reset, then one dense step), HIP events on the launch stream."""
    import torch

    stream = layer.stream if layer.stream is not None else torch.cuda.current_stream()
    out = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        layer.reset()
        a.record(stream)
        layer.step(frame)
        b.record(stream)
        torch.cuda.synchronize()
        out.append(1e3 * a.elapsed_time(b))
    return float(np.median(out))


def translate_np(x, dy, dx):
    """Frame content moved by (dy, dx) pixels, zero where nothing moved in (N, H, W, C)."""
    out = np.zeros_like(x)
    h, w = x.shape[1], x.shape[2]
    out[:, max(0, dy):min(h, h + dy), max(0, dx):min(w, w + dx)] = \
        x[:, max(0, -dy):min(h, h - dy), max(0, -dx):min(w, w - dx)]
    return out


def measure_translated(wt, layer_kw, clip, dtype, eps, block, steps):
    """Clip frames with a (1, 1) pixel camera jitter on every other frame: steps with the
    known translation (skipconv_step_translated) against plain steps on the same frames."""
    import torch
    from paper_2104_11487_amd.skipconv import SkipConv

    nfr = len(clip)
    jit = [(t % 2, t % 2) for t in range(nfr)]
    frames = []
    for t, x in enumerate(clip):
        xs = x.view(np.uint16) if dtype == "bf16" else x
        frames.append(translate_np(xs, *jit[t]))
    dev = upload([f.view(np.uint16) if dtype == "bf16" else f for f in frames], dtype)
    shifts = [(0, 0)] + [(jit[t][0] - jit[t - 1][0], jit[t][1] - jit[t - 1][1]) for t in range(1, nfr)]
    out = []
    for compensated in (True, False):
        lay = SkipConv(wt, eps=eps, block=block, translate=True, **layer_kw)
        sites = 0

        def run(n, count=False):
            nonlocal sites
            for j in range(n):
                t = j % nfr
                if t == 0:
                    lay.reset()
                if compensated:
                    lay.step_translated(dev[t], *shifts[t])
                else:
                    lay.step(dev[t])
                if count:
                    sites += lay.active_count()[1]

        run(nfr, count=True)
        run(nfr)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        run(steps)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        lay.close()
        total = nfr * lay.h_out * lay.w_out * layer_kw["n"]
        out.append({"label": f"camera jitter, {'translation-compensated' if compensated else 'plain'} steps",
                    "frames_per_s": steps * layer_kw["n"] / wall, "ms_per_step": 1e3 * wall / steps,
                    "density": sites / total})
        log(f"[bench] {out[-1]['label']}: {out[-1]['frames_per_s']:.0f} frames/s, density {out[-1]['density']:.3f}")
    return out


def torch_dense_us(wt, shape, stride, steps=200):
    """torch conv2d (MIOpen) of the same shape, channels-last, for context only."""
    import torch
    import torch.nn.functional as F

    n, h, w, c = shape
    x = torch.randn(n, c, h, w, device="cuda", dtype=wt.dtype).contiguous(memory_format=torch.channels_last)
    k = wt.shape[2]
    wcl = wt.contiguous(memory_format=torch.channels_last)
    for _ in range(10):
        F.conv2d(x, wcl, stride=stride, padding=(k - 1) // 2)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        F.conv2d(x, wcl, stride=stride, padding=(k - 1) // 2)
    torch.cuda.synchronize()
    return 1e6 * (time.perf_counter() - t0) / steps


# ------------------------------------------------------------ CPU baseline --

def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, w32, eps, block, streams=1, budget_s=12.0, threads=1):
    """The CPU oracle as it stands, BLAS limited to `threads`, on a bounded sample of the
    workload: the first `streams` stream(s) of the clip, the reference frame untimed, then
    consecutive steady-state frames until `budget_s` has passed (at least two)."""
    from threadpoolctl import threadpool_limits
    from oracle import skipconv_oracle as O
    from paper_2104_11487_amd import synthetic as syn

    lay_spec = wl.layers[0]
    wbits = w32 if wl.dtype == "f32" else O.f32_to_bf16_rne(w32)
    n = min(streams, wl.n)
    vid = wl.video(wl.frames)
    with threadpool_limits(limits=threads):
        orc = O.SkipConvOracle(wbits, n=n, h=wl.h, w=wl.w, stride=lay_spec.stride, eps=eps, block=block,
                               dtype=wl.dtype)
        orc.step(syn.to_storage(next(vid)[:n], wl.dtype))  # reference frame, untimed
        done, el = 0, 0.0
        for f in vid:
            x = syn.to_storage(f[:n], wl.dtype)
            t0 = time.perf_counter()
            orc.step(x)
            el += time.perf_counter() - t0
            done += 1
            if (el >= budget_s and done >= 2) or el >= 3 * budget_s:
                break
    return {"value": done * n / el, "unit": "frames/s", "cores": threads, "kind": "oracle",
            "sample": f"{done} consecutive steady-state frames (clip positions 1..{done}) of {n} of the "
                      f"{wl.n} streams of {wl.name}, eps={eps:.4g}, b={block}, {el:.1f}s timed after an untimed "
                      f"reference frame; numpy fp64, BLAS limited to {threads} thread(s)"}


# ---------------------------------------------------------------- traffic --

def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in sorted(os.listdir(os.path.join(ROOT, "paper_2104_11487_amd", "csrc"))):
        with open(os.path.join(ROOT, "paper_2104_11487_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def profiled_traffic(workload: str, kernel: str):
    """HBM bytes per launch from a committed rocprofv3 counter summary, if it is current."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else k.get("bytes_per_launch")


def summarize_pmc(fetch_db: str, write_db: str, out_json: str, *, workload: str, copy_mib: int):
    """Average FETCH_SIZE / WRITE_SIZE (KiB per dispatch) per kernel, scaled by a plain copy.

    Inputs are the SQLite databases rocprofv3 writes for one --pmc FETCH_SIZE
    run and one --pmc WRITE_SIZE run of the same command. The largest
    device-to-device copy in the run (the --copy-probe of `copy_mib` MiB, which
    reads and writes exactly that many bytes) gives the bytes per counter unit.
    """
    import sqlite3

    if copy_mib <= 0:
        raise SystemExit("--summarize-pmc needs --copy-probe MIB: the size of the copy the counted run made")

    def rows(db, counter):
        con = sqlite3.connect(db)
        out = con.execute("select kernel_name, value from counters_collection where counter_name = ?",
                          (counter,)).fetchall()
        con.close()
        return out

    fetch, write = rows(fetch_db, "FETCH_SIZE"), rows(write_db, "WRITE_SIZE")
    copy_bytes = float(copy_mib << 20)
    is_copy = lambda k: "copyBuffer" in k or ("copy" in k.lower() and "sc::" not in k)
    cf = max((v for k, v in fetch if is_copy(k)), default=0.0)
    cw = max((v for k, v in write if is_copy(k)), default=0.0)
    f_scale = copy_bytes / cf if cf > 0 else None
    w_scale = copy_bytes / cw if cw > 0 else None
    kernels = {}
    for label, pred in (("gate", lambda k: "gate_kernel" in k), ("compact", lambda k: "compact_kernel" in k),
                        ("fused", lambda k: "fused_kernel" in k or "fused_rb_kernel" in k or "fused_dw_kernel" in k),
                        ("conv", lambda k: "conv_" in k and "_kernel" in k),
                        ("depthwise", lambda k: "depthwise_kernel" in k)):
        vf = [v for k, v in fetch if pred(k)]
        vw = [v for k, v in write if pred(k)]
        names = sorted({k for k, _ in fetch if pred(k)})
        if not vf or not vw or f_scale is None or w_scale is None:
            continue
        af, aw = sum(vf) / len(vf), sum(vw) / len(vw)
        kernels[label] = {"kernel": names[0] if len(names) == 1 else names, "dispatches": len(vf),
                          "fetch_kib": af, "write_kib": aw, "fetch_bytes": af * f_scale,
                          "write_bytes": aw * w_scale, "bytes_per_launch": af * f_scale + aw * w_scale}
    rec = {"workload": workload, "source_hash": kernel_source_hash(), "copy_mib": copy_mib,
           "copy_fetch_kib": cf, "copy_write_kib": cw, "fetch_bytes_per_unit": f_scale,
           "write_bytes_per_unit": w_scale, "kernels": kernels}
    with open(out_json, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec, indent=1))


def summarize_trace(db: str, out_md: str, command: str) -> None:
    """Markdown table of per-kernel dispatch counts and durations from a rocprofv3 --kernel-trace database."""
    import sqlite3

    con = sqlite3.connect(db)
    rows = con.execute("select name, count(*), sum(duration), avg(duration), min(duration), max(duration) "
                       "from kernels group by name order by sum(duration) desc").fetchall()
    con.close()
    total = sum(r[2] for r in rows) or 1.0
    lines = [f"# rocprofv3 kernel trace: {os.path.basename(db)}", "", "Command:", "", "```", command, "```", "",
             "| kernel | calls | total us | avg us | min us | max us | share |",
             "|---|---:|---:|---:|---:|---:|---:|"]
    for name, n, tot, avg, mn, mx in rows:
        short = name.replace("(anonymous namespace)::", "").split("(sc::")[0].split("(unsigned")[0]
        lines.append(f"| `{short[:90]}` | {n} | {tot / 1e3:.1f} | {avg / 1e3:.2f} | {mn / 1e3:.2f} | "
                     f"{mx / 1e3:.2f} | {100 * tot / total:.1f}% |")
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_counters(db: str, out_md: str, command: str) -> None:
    """Markdown table of the per-dispatch average of every counter in a rocprofv3 --pmc database, per kernel."""
    import sqlite3

    con = sqlite3.connect(db)
    rows = con.execute("select kernel_name, counter_name, count(*), avg(value) from counters_collection "
                       "group by kernel_name, counter_name order by kernel_name, counter_name").fetchall()
    con.close()
    lines = [f"# rocprofv3 counters: {os.path.basename(db)}", "", "Command:", "", "```", command, "```", "",
             "| kernel | counter | dispatches | average per dispatch |", "|---|---|---:|---:|"]
    for name, counter, n, avg in rows:
        short = name.replace("(anonymous namespace)::", "").split("(sc::")[0].split("(unsigned")[0]
        lines.append(f"| `{short[:90]}` | {counter} | {n} | {avg:.6g} |")
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


# ----------------------------------------------------------------- stacks --

def bench_stack(args):
    """Six stacked 3x3 layers (3-32-64-64-128-128-128 channels, strides 1/2, ReLU,
    per-site gates, 256 x 192 bf16 frames): one step = all six layers on one frame.

    The layer thresholds are eps0 * a fixed per-layer schedule, eps0 bisected on
    the GPU for a MAC-weighted density near --density. Two variants run the same
    frames: 'full' (each layer reads its whole input frame, x_t and x_{t-1}) and
    'chained' (layers 2..6 step on the previous layer's emitted residual).
    """
    import torch
    from paper_2104_11487_amd import synthetic as syn
    from paper_2104_11487_amd.skipconv import SkipConv

    wl, clip = load_workload("stack6", args.frames)
    frames_dev = upload(clip, wl.dtype)
    wts = [weight_tensor(w, wl.dtype) for w in wl.weights()]
    sched = syn.eps_schedule(len(wl.layers))

    def build(eps0, chained):
        lays, h, w = [], wl.h, wl.w
        for i, sp in enumerate(wl.layers):
            last = i == len(wl.layers) - 1
            lay = SkipConv(wts[i], n=wl.n, h=h, w=w, stride=sp.stride, groups=sp.groups,
                           eps=float(eps0 * sched[i]), block=wl.block, act_out="none" if last else "relu",
                           emit_residual=chained and not last)
            lays.append(lay)
            h, w = lay.h_out, lay.w_out
        return lays

    def step(lays, x, chained):
        lays[0].step(x)
        for i in range(1, len(lays)):
            if chained:
                lays[i].step_chained(lays[i - 1])
            else:
                lays[i].step(lays[i - 1].activation())

    def density(eps0):
        lays = build(eps0, False)
        act = dense = 0
        for t, x in enumerate(frames_dev):
            if t == 0:
                for l in lays:
                    l.reset()
            step(lays, x, False)
            if t > 0:
                for l in lays:
                    a, d = S_frame_macs(l)
                    act += a
                    dense += d
        for l in lays:
            l.close()
        return act / max(dense, 1)

    def S_frame_macs(l):
        from paper_2104_11487_amd import skipconv as S
        dense, active = S.skipconv_frame_macs(l.handle, l._stream())
        return active, dense

    lo, hi = 0.0, 8.0
    for _ in range(14):
        mid = 0.5 * (lo + hi)
        if density(mid) > args.density:
            lo = mid
        else:
            hi = mid
    eps0 = 0.5 * (lo + hi)
    d_mac = density(eps0)
    log(f"[bench] stack6: eps0 {eps0:.4g}, MAC-weighted density {d_mac:.3f}")

    nfr = len(frames_dev)

    def timed(frames, chained):
        lays = build(eps0, chained)
        for _ in range(max(1, args.warmup // nfr)):
            for t, x in enumerate(frames):
                if t == 0:
                    for l in lays:
                        l.reset()
                step(lays, x, chained)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for j in range(args.steps):
            if j % nfr == 0:
                for l in lays:
                    l.reset()
            step(lays, frames[j % nfr], chained)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        for l in lays:
            l.close()
        return wall

    res = {}
    for chained in (False, True):
        res["chained" if chained else "full"] = wall = timed(frames_dev, chained)
        log(f"[bench] stack6 {'chained' if chained else 'full'}: {args.steps / wall:.0f} frames/s, "
            f"{1e6 * wall / args.steps:.1f} us/step")
    # the same stack and thresholds on the same rectangles over a noise-free
    # static background: activity stays with the moving objects
    clean = [syn.to_storage(f, wl.dtype) for f in
             syn.RectVideo(wl.h, wl.w, wl.c, nfr, seed=401, batch=wl.n, noise_std=0.0)]
    clean_dev = upload(clean, wl.dtype)
    sweep = []
    for chained in (False, True):
        wall_c = timed(clean_dev, chained)
        sweep.append({"label": f"clean background, {'chained' if chained else 'full'}",
                      "frames_per_s": args.steps / wall_c, "ms_per_step": 1e3 * wall_c / args.steps})
        log(f"[bench] stack6 clean background {'chained' if chained else 'full'}: {args.steps / wall_c:.0f} "
            f"frames/s, {1e6 * wall_c / args.steps:.1f} us/step")
    # algorithmic bytes of the full-frame formulation: per layer 3|x| (x_t, x_{t-1}
    # read, x_t kept) + 2 d |z| + activation writes; reported against the chained step
    wall = res["chained"]
    out = {
        "metric": METRIC, "value": args.steps / wall, "unit": "frames/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": 1e3 * wall / args.steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": "stack6: six 3x3 layers 3-32-64-64-128-128-128, strides 1,2,1,2,1,1, ReLU, "
                               f"256x192 frames, batch 1, {nfr}-frame clip (reset at frame 1), per-site gates, "
                               "layers 2-6 chained on emitted residuals",
                   "eps0": eps0, "mac_density": d_mac,
                   "full_frames_per_s": args.steps / res["full"], "chained_frames_per_s": args.steps / wall,
                   "speedup_chained": res["full"] / wall},
        "roofline": None, "cpu_baseline": None, "sweep": sweep,
    }
    print(json.dumps(out), flush=True)


# ------------------------------------------- two large layers, chained --

def bench_blob_pair(args):
    """Two stacked 3x3 128 -> 128 bf16 layers with ReLU between on the 4 x 512 x 512
    blob clip, 16 x 16 blocks, each layer's threshold for ~--density block density on
    its own input. 'full': layer 2 steps on layer 1's activation (x_t and x_{t-1} over
    the whole frame); 'chained': layer 2 steps on the residual layer 1 emits at the
    blocks it updated (Sec. 3.1: residuals at intermediate feature maps), its gate
    skipping tiles with no upstream block."""
    import torch
    from paper_2104_11487_amd import skipconv as S
    from paper_2104_11487_amd import synthetic as syn
    from paper_2104_11487_amd.skipconv import SkipConv

    wl, clip = load_workload("blob128", args.frames)
    frames_dev = upload(clip, wl.dtype)
    nfr = len(frames_dev)
    w1 = weight_tensor(wl.weights()[0], wl.dtype)
    w2 = weight_tensor(syn.he_weights(128, 128, 3, seed=519), wl.dtype)
    kw = dict(n=wl.n, h=wl.h, w=wl.w, stride=1, groups=1)
    b = wl.block
    e1 = eps_for_density(gpu_stats(kw, w1, frames_dev), b, wl.h, wl.w, args.density)
    # layer 2's statistics on layer 1's activations at e1
    l1 = SkipConv(w1, eps=e1, block=b, act_out="relu", **kw)
    probe = SkipConv(w2, eps=0.0, block=1, keep_stats=True, **kw)
    stats2 = []
    for t, x in enumerate(frames_dev):
        l1.step(x)
        probe.step(l1.activation())
        if t > 0:
            torch.cuda.synchronize()
            stats2.append(probe.stat())
    l1.close()
    probe.close()
    e2 = eps_for_density(stats2, b, wl.h, wl.w, args.density)
    log(f"[bench] blob pair: eps {e1:.4g} / {e2:.4g}")

    def run(chained, steps, count=False):
        a = SkipConv(w1, eps=e1, block=b, act_out="relu", emit_residual=chained, **kw)
        c = SkipConv(w2, eps=e2, block=b, **kw)
        dens = [0, 0]

        def one(j, counted):
            t = j % nfr
            if t == 0:
                a.reset()
                c.reset()
            a.step(frames_dev[t])
            if chained:
                c.step_chained(a)
            else:
                c.step(a.activation())
            if counted:
                dens[0] += a.active_count()[1]
                dens[1] += c.active_count()[1]

        for j in range(nfr + 1):  # warm-up: one clip and the next reference frame
            one(j, False)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for j in range(1, steps + 1):  # steady-state frames after the reference
            one(j, count)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        a.close()
        c.close()
        return wall, dens

    res = {}
    for chained in (False, True):
        wall, _ = run(chained, args.steps)
        res["chained" if chained else "full"] = wall
        log(f"[bench] blob pair {'chained' if chained else 'full'}: {args.steps * wl.n / wall:.0f} frames/s, "
            f"{1e6 * wall / args.steps:.1f} us/step")
    _, dens = run(False, nfr - 1, count=True)
    sites = wl.n * wl.h * wl.w * (nfr - 1)
    out = {
        "metric": METRIC, "value": args.steps * wl.n / res["chained"], "unit": "frames/s", "n_gpus": 1,
        "steps": args.steps, "warmup": nfr + 1, "ms_per_step": 1e3 * res["chained"] / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": "blob pair: two 3x3 conv 128->128 layers with ReLU between on 4 x 512 x 512 "
                               f"frames, {nfr}-frame blob clip (reset at frame 1), 16x16 blocks, layer 2 chained on "
                               "layer 1's emitted residual; steady-state steps",
                   "eps": [e1, e2], "density": [dens[0] / sites, dens[1] / sites],
                   "full_frames_per_s": args.steps * wl.n / res["full"],
                   "chained_frames_per_s": args.steps * wl.n / res["chained"],
                   "speedup_chained": res["full"] / res["chained"]},
        "roofline": None, "cpu_baseline": None, "sweep": [],
    }
    print(json.dumps(out), flush=True)


# ------------------------------------------------------- pointwise + dw --

def bench_mbconv(args):
    """Pointwise 1x1 192->192, then depthwise 3x3 (groups 192), 64 x 64 bf16 frames,
    8 x 8 blocks, identity between (an MBConv-style pair); 10 % of the frames carry a
    one-frame camera shake. One step = both layers on one frame. Per-layer thresholds
    are calibrated for each target density on the GPU (layer 2 on layer 1's outputs).
    Variants: 'full' (layer 2 steps on layer 1's activation output) and 'chained'
    (layer 2 steps on layer 1's emitted residual); per-kernel times from the library's
    events; shake frames: layer-1 density with and without the known-shift step."""
    import torch
    from paper_2104_11487_amd import skipconv as S
    from paper_2104_11487_amd import synthetic as syn
    from paper_2104_11487_amd.skipconv import SkipConv

    wl, clip = load_workload("mbconv192", args.frames)
    nfr = len(clip)
    vid = syn.RectVideo(wl.h, wl.w, wl.c, nfr, seed=301, batch=wl.n, shake_prob=0.1)
    for _ in vid:
        pass
    shake = set(vid.shake_frames)
    frames_dev = upload(clip, wl.dtype)
    w1, w2 = [weight_tensor(w, wl.dtype) for w in wl.weights()]
    b = args.block or wl.block
    kw1 = dict(n=wl.n, h=wl.h, w=wl.w, stride=1, groups=1)
    kw2 = dict(n=wl.n, h=wl.h, w=wl.w, stride=1, groups=wl.c)
    x_bytes = wl.n * wl.h * wl.w * wl.c * 2
    sites = wl.n * wl.h * wl.w

    def build(e1, e2, chained):
        l1 = SkipConv(w1, eps=e1, block=b, act_out="identity", emit_residual=chained, **kw1)
        l2 = SkipConv(w2, eps=e2, block=b, **kw2)
        return l1, l2

    def step(l1, l2, x, chained):
        l1.step(x)
        if chained:
            l2.step_chained(l1)
        else:
            l2.step(l1.activation())

    stats1 = gpu_stats(kw1, w1, frames_dev)

    def calibrate(d):
        e1 = eps_for_density(stats1, b, wl.h, wl.w, d)
        l1 = SkipConv(w1, eps=e1, block=b, act_out="identity", **kw1)
        ys = []
        for x in frames_dev:
            l1.step(x)
            ys.append(l1.activation().clone().view(wl.n, wl.h, wl.w, wl.c))
        l1.close()
        e2 = eps_for_density(gpu_stats(kw2, w2, ys), b, wl.h, wl.w, d)
        return e1, e2

    def run(e1, e2, chained, steps, timing):
        l1, l2 = build(e1, e2, chained)
        for t in range(nfr):  # warm-up pass over the clip
            if t == 0:
                l1.reset()
                l2.reset()
            step(l1, l2, frames_dev[t], chained)
        if timing:
            S.skipconv_timing_begin(l1.handle, steps, 1)
            S.skipconv_timing_begin(l2.handle, steps, 1)
        act = [0, 0]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for j in range(steps):
            if j % nfr == 0:
                l1.reset()
                l2.reset()
            step(l1, l2, frames_dev[j % nfr], chained)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        res = {"frames_per_s": steps * wl.n / wall, "us_per_step": 1e6 * wall / steps}
        if timing:
            g1, c1, n1, _ = S.skipconv_timing_read(l1.handle, l1._stream(), steps)
            g2, c2, n2, _ = S.skipconv_timing_read(l2.handle, l2._stream(), steps)
            n1, n2 = max(n1, 1), max(n2, 1)
            res.update({"pw_gate_us": 1e3 * g1 / n1, "pw_conv_us": 1e3 * c1 / n1,
                        "dw_gate_us": 1e3 * g2 / n2, "dw_conv_us": 1e3 * c2 / n2, "timed_steps": [n1, n2]})
            # active sites of both layers over one clip pass (same schedule)
            for t in range(nfr):
                if t == 0:
                    l1.reset()
                    l2.reset()
                step(l1, l2, frames_dev[t], chained)
                act[0] += l1.active_count()[1]
                act[1] += l2.active_count()[1]
            res["density_pw"] = act[0] / (sites * nfr)
            res["density_dw"] = act[1] / (sites * nfr)
            # depthwise convolution kernel: residual at the active sites (x_t and
            # x_{t-1}) and z read-modify-written there, per launch
            dw_bytes = act[1] / nfr * wl.c * (2 + 2 + 8)
            res["dw_conv_bytes_per_launch"] = dw_bytes
            res["dw_conv_gbs"] = dw_bytes / (res["dw_conv_us"] * 1e-6) / 1e9
        l1.close()
        l2.close()
        return res

    points = []
    for d in (0.1, 0.25, 0.5):
        e1, e2 = calibrate(d)
        for chained in (False, True):
            r = run(e1, e2, chained, args.steps, False)
            r.update(run(e1, e2, chained, max(2 * nfr, 64), True) | {"frames_per_s": r["frames_per_s"],
                                                                      "us_per_step": r["us_per_step"]})
            r.update({"target_density": d, "eps": [e1, e2], "variant": "chained" if chained else "full"})
            log(f"[bench] mbconv192 d={d} {r['variant']}: {r['frames_per_s']:.0f} frames/s, "
                f"{r['us_per_step']:.1f} us/step; pw gate {r['pw_gate_us']:.1f} conv {r['pw_conv_us']:.1f}, "
                f"dw gate {r['dw_gate_us']:.1f} conv {r['dw_conv_us']:.1f} us; density pw {r['density_pw']:.3f} "
                f"dw {r['density_dw']:.3f}")
            points.append(r)

    # shake frames: layer-1 active sites per clip position, plain steps vs steps
    # with the known shift (Sec. 3.3) at the 25 % threshold
    e1, _ = calibrate(0.25)
    shift = [(0, 0)] * nfr
    prev = (0, 0)
    for t in range(1, nfr):
        cur = vid.shake_shift.get(t, (0, 0))
        shift[t] = (cur[0] - prev[0], cur[1] - prev[1])
        prev = cur
    dens = {}
    for comp in (False, True):
        lay = SkipConv(w1, eps=e1, block=b, translate=True, **kw1)
        per = []
        for t in range(nfr):
            if comp:
                lay.step_translated(frames_dev[t], *shift[t])
            else:
                lay.step(frames_dev[t])
            per.append(lay.active_count()[1] / sites)
        lay.close()
        sh = [per[t] for t in range(1, nfr) if shift[t] != (0, 0)]
        ot = [per[t] for t in range(1, nfr) if shift[t] == (0, 0)]
        dens["compensated" if comp else "plain"] = {"shake": float(np.mean(sh)) if sh else None,
                                                    "other": float(np.mean(ot)) if ot else None}
    log(f"[bench] mbconv192 shake frames {sorted(shake)}: layer-1 density {dens}")

    head = next(p for p in points if p["target_density"] == args.density and p["variant"] == "chained") \
        if any(p["target_density"] == args.density for p in points) else points[3]
    a = head["dw_conv_gbs"]
    out = {
        "metric": METRIC, "value": head["frames_per_s"], "unit": "frames/s", "n_gpus": 1, "steps": args.steps,
        "warmup": nfr, "ms_per_step": head["us_per_step"] * 1e-3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": "mbconv192: 1x1 conv 192->192 then depthwise 3x3 (groups 192), identity between, "
                               f"64x64 frames, batch 1, {nfr}-frame clip (reset at frame 1), 8x8 blocks, "
                               "10% camera-shake frames, layer 2 chained on layer 1's emitted residual",
                   "target_density": head["target_density"], "eps": head["eps"],
                   "shake_frames": sorted(shake), "shake_density_layer1": dens},
        "roofline": {"kernel": "depthwise conv (VALU, active blocks)", "bound": "hbm", "achieved": a,
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": a / PEAK_HBM_GBS, "traffic": None,
                     "bytes_per_launch": head["dw_conv_bytes_per_launch"], "us_per_launch": head["dw_conv_us"]},
        "cpu_baseline": None, "sweep": points,
    }
    print(json.dumps(out), flush=True)


# -------------------------------------------------------------------- main --

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="blob128",
                    choices=["rect64", "blob128", "square16", "stack6", "mbconv192", "blobpair"])
    ap.add_argument("--block", type=int, default=None)
    ap.add_argument("--density", type=float, default=0.25)
    ap.add_argument("--frames", type=int, default=None)
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-events", action="store_true", help="time without per-kernel events")
    ap.add_argument("--no-peaks", action="store_true", help="skip the measured copy / GEMM peaks")
    ap.add_argument("--split", action="store_true",
                    help="force the gate + compaction + conv pipeline instead of the fused kernel")
    ap.add_argument("--caller-retains", action="store_true",
                    help="headline layer reads x_{t-1} from the previous frame's buffer (no copy)")
    ap.add_argument("--eps", type=float, default=None,
                    help="fixed gate threshold (skips calibration; used for counter runs)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="also run one device-to-device copy of MIB MiB (counter calibration)")
    ap.add_argument("--summarize-trace", nargs=3, metavar=("TRACE_DB", "OUT_MD", "COMMAND"),
                    help="write a markdown summary of a rocprofv3 --kernel-trace database")
    ap.add_argument("--summarize-pmc", nargs=3, metavar=("FETCH_DB", "WRITE_DB", "OUT_JSON"),
                    help="turn the databases of two rocprofv3 --pmc runs into a traffic summary")
    ap.add_argument("--summarize-counters", nargs=3, metavar=("PMC_DB", "OUT_MD", "COMMAND"),
                    help="write a markdown summary of any rocprofv3 --pmc database")
    args = ap.parse_args()
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace)
        return
    if args.summarize_counters:
        summarize_counters(*args.summarize_counters)
        return
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, workload=args.workload, copy_mib=args.copy_probe)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the layer runs on a single "
              "MI355X; independent streams would shard across GPUs with no communication.",
              file=sys.stderr, flush=True)
        sys.exit(2)

    import torch
    from paper_2104_11487_amd import skipconv as S
    from paper_2104_11487_amd.skipconv import SkipConv

    S.lib()  # fail loudly if the HIP library is missing
    torch.cuda.set_device(0)
    if args.workload == "stack6":
        bench_stack(args)
        return
    if args.workload == "mbconv192":
        bench_mbconv(args)
        return
    if args.workload == "blobpair":
        bench_blob_pair(args)
        return
    wl, clip = load_workload(args.workload, args.frames)
    frames_dev = upload(clip, wl.dtype)
    w32 = wl.weights()[0]
    wt = weight_tensor(w32, wl.dtype)
    spec = wl.layers[0]
    block = args.block or wl.block
    layer_kw = dict(n=wl.n, h=wl.h, w=wl.w, stride=spec.stride, groups=spec.groups)
    probe = SkipConv(wt, eps=0.0, block=block, **layer_kw)
    h_out, w_out = probe.h_out, probe.w_out
    probe.close()
    kk = spec.k * spec.k * spec.c_in // spec.groups
    esz = 2 if wl.dtype == "bf16" else 4
    x_bytes = wl.n * wl.h * wl.w * wl.c * esz
    geom = {"n": wl.n, "sites": wl.n * h_out * w_out, "c_out": spec.c_out, "kk": kk, "x_bytes": x_bytes,
            "nb": wl.n * (-(-h_out // block)) * (-(-w_out // block)),
            "w_bytes": kk * spec.c_out * esz}
    big = args.workload == "blob128"

    if args.copy_probe:
        src = torch.empty(args.copy_probe << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    stats = None if args.eps is not None else gpu_stats(layer_kw, wt, frames_dev)

    def mk(b, eps, dense=False, split=args.split, gate="input", retains=args.caller_retains):
        return lambda: SkipConv(wt, eps=eps, block=b, force_dense=dense, split=split, gate=gate,
                                caller_retains=retains, **layer_kw)

    eps_head = args.eps if args.eps is not None else eps_for_density(stats, block, h_out, w_out, args.density)
    head = measure_point(mk(block, eps_head), frames_dev, args.steps, args.warmup, geom,
                         label=f"b={block} d={args.density}", events=not args.no_events,
                         retains=args.caller_retains)

    # roofline model of one step (memory-bound at both ends of the sweep): the
    # fixed bytes (x_t and x_{t-1} read, x_t kept unless the caller retains its
    # frames, weights) plus the z read-modify-write at the active sites
    z_bytes = geom["sites"] * spec.c_out * 4

    def model_us(d, retains):
        fixed = (2 if retains else 3) * x_bytes + geom["w_bytes"]
        return 1e6 * (fixed + 2 * d * z_bytes) / (PEAK_HBM_GBS * 1e9)

    dense_flop = 2.0 * geom["sites"] * spec.c_out * kk
    peak_mfma = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    ideal_dense_us = 1e6 * max(dense_flop / (peak_mfma * 1e12), (2 * x_bytes + z_bytes + geom["w_bytes"])
                               / (PEAK_HBM_GBS * 1e9))

    sweep = []
    if not args.no_sweep and stats is not None:
        sweep_steps = min(args.steps, len(clip) - 1) if big else max(len(clip) * 2, min(args.steps, 256))
        sweep_steps = max(sweep_steps, 8)
        warm = 2 if big else len(clip)
        blocks_sweep = [block] if big else [1, 4, 8]
        dens_sweep = (0.05, 0.10, 0.25, 0.50, 0.75) if big else (0.10, 0.25, 0.50)
        r = measure_point(mk(block, 0.0, dense=True), frames_dev, sweep_steps, warm, geom,
                          label=f"forced dense b={block}")
        r.update({"block": block, "target_density": 1.0, "forced_dense": True})
        dense_ms = r["ms_per_step"]
        sweep.append(r)
        for b in blocks_sweep:
            for d in dens_sweep + ((0.0,) if big else ()):
                e = eps_for_density(stats, b, h_out, w_out, d) if d > 0 else 0.0
                g2 = dict(geom, nb=wl.n * (-(-h_out // b)) * (-(-w_out // b)))
                lab = f"b={b} d={d}" if d > 0 else f"b={b} eps=0"
                r = measure_point(mk(b, e), frames_dev, sweep_steps, warm, g2, label=lab)
                r.update({"block": b, "target_density": d if d > 0 else 1.0, "eps": e})
                if b == block:
                    ds = r["density"]
                    r["speedup_vs_forced_dense"] = dense_ms / r["ms_per_step"]
                    r["model_speedup_vs_forced_dense"] = model_us(1.0, False) / model_us(ds, False)
                    r["model_us_per_step"] = model_us(ds, False)
                    r["model_speedup_vs_ideal_dense"] = ideal_dense_us / model_us(ds, False)
                    log(f"[bench] {lab}: speed-up over forced dense {r['speedup_vs_forced_dense']:.2f}x "
                        f"(roofline model {r['model_speedup_vs_forced_dense']:.2f}x at density {ds:.3f})")
                sweep.append(r)
                if big and d > 0:
                    # the same point with caller-retained frames (no x_t copy)
                    r2 = measure_point(mk(b, e, retains=True), frames_dev, sweep_steps, warm, g2,
                                       label=f"{lab} caller-retained frames", retains=True)
                    r2.update({"block": b, "target_density": d, "eps": e, "caller_retains": True,
                               "speedup_vs_forced_dense": dense_ms / r2["ms_per_step"],
                               "model_us_per_step": model_us(r2["density"], True),
                               "model_speedup_vs_forced_dense": model_us(1.0, False) / model_us(r2["density"], True)})
                    sweep.append(r2)
        if not big:  # (the large workload runs the split pipeline either way)
            r = measure_point(mk(block, eps_head, split=not args.split), frames_dev, sweep_steps, warm, geom,
                              label=f"b={block} d={args.density} other pipeline")
            r.update({"block": block, "target_density": args.density})
            sweep.append(r)
            other = not args.caller_retains
            r = measure_point(mk(block, eps_head, retains=other), frames_dev, sweep_steps, warm, geom,
                              label=f"b={block} d={args.density} " + ("caller-retained frames" if other
                                                                      else "library x_(t-1) copy"),
                              retains=other)
            r.update({"block": block, "target_density": args.density, "caller_retains": other})
            sweep.append(r)
        # Output-Norm gate (Eq. 7) at the same density: with p = 2 it compares
        # s * sum(w^2) with eps^2, so eps scales by the weight 2-norm
        wq = wt.float().cpu().numpy().astype(np.float64)
        e_out = eps_head * float(np.sqrt(np.sum(wq * wq)))
        r = measure_point(mk(block, e_out, gate="output"), frames_dev, sweep_steps, warm, geom,
                          label=f"output-norm gate b={block} d={args.density}")
        r.update({"block": block, "target_density": args.density, "gate": "output-norm", "eps": e_out})
        sweep.append(r)
        # learned gate (Eq. 8 at inference; the layer's own pipeline): seeded random phi,
        # bias from the GPU's own scores for the same block density (a 16-frame
        # clip on the large workload)
        short = frames_dev[:16] if big else frames_dev
        rng = np.random.Generator(np.random.PCG64(7))
        phi = torch.from_numpy(rng.normal(0, 0.05, (spec.c_in, spec.k, spec.k)).astype(np.float32)).cuda()
        probe = SkipConv(wt, eps=0.0, block=1, keep_stats=True, gate="learned", **layer_kw)
        probe.set_gate_weights(phi, 0.0)
        scores = []
        for t, x in enumerate(short):
            probe.step(x)
            if t > 0:
                torch.cuda.synchronize()
                scores.append(probe.stat())
        probe.close()
        bias = -block_quantile(scores, block, h_out, w_out, args.density)

        def mk_learned():
            lay = SkipConv(wt, eps=0.0, block=block, gate="learned", **layer_kw)
            lay.set_gate_weights(phi, bias)
            return lay
        r = measure_point(mk_learned, short, min(sweep_steps, len(short) - 1) if big else sweep_steps,
                          warm, geom, label=f"learned gate b={block} d={args.density}")
        r.update({"block": block, "target_density": args.density, "gate": "learned", "bias": bias})
        sweep.append(r)
        # translation-compensated steps (Sec. 3.3): the clip with a one-pixel
        # camera jitter on every other frame, stepped with the known shift vs. plainly
        r1, r2 = measure_translated(wt, layer_kw, clip[:16] if big else clip, wl.dtype, eps_head, block,
                                    32 if big else sweep_steps)
        sweep += [r1, r2]
        tus = torch_dense_us(wt, (wl.n, wl.h, wl.w, wl.c), spec.stride, steps=20 if big else 200)
        sweep.append({"label": "torch conv2d (MIOpen), dense, same shape", "us_per_frame_batch": tus,
                      "dense_tflops": dense_flop / (tus * 1e-6) / 1e12})
        log(f"[bench] torch conv2d dense: {tus:.1f} us")

    # roofline of the dominant kernel, from the events of the timed region;
    # the committed counter summaries are of the library-copy contract
    def traffic(kernel):
        return None if args.caller_retains else profiled_traffic(args.workload, kernel)

    meas = measured_peaks() if not args.no_peaks else None
    roof, kernels = None, {}
    if head["gate_us"] is not None and head["pipeline"] == "fused":
        fb, ff, fus = head["fused_bytes_per_launch"], head["conv_flop_per_launch"], head["gate_us"]
        hbm_bound = fb / (PEAK_HBM_GBS * 1e9) >= ff / (peak_mfma * 1e12)
        if hbm_bound:
            a = fb / (fus * 1e-6) / 1e9
            roof = {"kernel": "fused (residual, gate, local compaction, MFMA conv, z update)", "bound": "hbm",
                    "achieved": a, "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": a / PEAK_HBM_GBS,
                    "traffic": traffic("fused"), "bytes_per_launch": fb,
                    "flop_per_launch": ff, "us_per_launch": fus}
        else:
            a = ff / (fus * 1e-6) / 1e12
            roof = {"kernel": "fused (residual, gate, local compaction, MFMA conv, z update)", "bound": "mfma",
                    "achieved": a, "peak": peak_mfma, "unit": "TFLOP/s", "frac": a / peak_mfma,
                    "traffic": traffic("fused"), "bytes_per_launch": fb,
                    "flop_per_launch": ff, "us_per_launch": fus}
    elif head["conv_us"] is not None:
        # convolution: algorithmic bytes = the residual operand at the active sites
        # (x_t and x_{t-1}) + z read-modify-written there (written on a reference frame)
        act_sites = head["active_sites_per_launch"]
        conv_bytes = act_sites * (2 * spec.c_in * esz + 8 * spec.c_out) + geom["w_bytes"]
        cf, cus = head["conv_flop_per_launch"], head["conv_us"]
        gb, gus = head["gate_bytes_per_launch"], head["gate_us"]
        kernels = {
            "gate": {"us_per_launch": gus, "bytes_per_launch": gb, "gbs": gb / (gus * 1e-6) / 1e9,
                     "frac_hbm": gb / (gus * 1e-6) / 1e9 / PEAK_HBM_GBS, "traffic": traffic("gate")},
            "conv": {"us_per_launch": cus, "flop_per_launch": cf, "bytes_per_launch": conv_bytes,
                     "tflops": cf / (cus * 1e-6) / 1e12, "frac_mfma": cf / (cus * 1e-6) / 1e12 / peak_mfma,
                     "gbs": conv_bytes / (cus * 1e-6) / 1e9,
                     "frac_hbm": conv_bytes / (cus * 1e-6) / 1e9 / PEAK_HBM_GBS,
                     "arith_intensity": cf / conv_bytes, "traffic": traffic("conv")},
        }
        if meas:
            kernels["gate"]["frac_measured_hbm"] = kernels["gate"]["gbs"] / meas["hbm_measured_gbs"]
            kernels["conv"]["frac_measured_mfma"] = kernels["conv"]["tflops"] / meas["bf16_gemm_tflops"]
            kernels["conv"]["frac_measured_hbm"] = kernels["conv"]["gbs"] / meas["hbm_measured_gbs"]
        if cus >= gus:
            k = kernels["conv"]
            mfma_bound = cf / (peak_mfma * 1e12) >= conv_bytes / (PEAK_HBM_GBS * 1e9)
            roof = {"kernel": "conv (sparse halo-gather MFMA over active blocks)",
                    "bound": "mfma" if mfma_bound else "hbm",
                    "achieved": k["tflops"] if mfma_bound else k["gbs"],
                    "peak": peak_mfma if mfma_bound else PEAK_HBM_GBS,
                    "unit": "TFLOP/s" if mfma_bound else "GB/s",
                    "frac": k["frac_mfma"] if mfma_bound else k["frac_hbm"], "traffic": k["traffic"],
                    "flop_per_launch": cf, "bytes_per_launch": conv_bytes, "us_per_launch": cus}
        else:
            k = kernels["gate"]
            roof = {"kernel": "gate (residual, statistic, threshold, blocks, work list, x_t copy)",
                    "bound": "hbm", "achieved": k["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": k["frac_hbm"], "traffic": k["traffic"], "bytes_per_launch": gb,
                    "us_per_launch": gus}
    if roof is not None and meas:
        roof["measured_peak"] = meas["hbm_measured_gbs"] if roof["unit"] == "GB/s" else meas["bf16_gemm_tflops"]
        roof["frac_of_measured_peak"] = roof["achieved"] / roof["measured_peak"]

    cpu = None
    if not args.no_cpu:
        e_cpu = eps_head
        cpu = cpu_baseline(wl, w32, e_cpu, block, streams=1 if big else wl.n, threads=1)
        log(f"[bench] cpu oracle, 1 core: {cpu['value']:.3f} frames/s")
        ncores = len(os.sched_getaffinity(0))
        allc = cpu_baseline(wl, w32, e_cpu, block, streams=1 if big else wl.n, threads=ncores)
        log(f"[bench] cpu oracle, {ncores} cores: {allc['value']:.3f} frames/s")
        cpu["all_cores"] = {"value": allc["value"], "cores": ncores, "sample": allc["sample"]}
        cpu["cpu_model"] = cpu_model()

    d_head = head["density"]
    out = {
        "metric": METRIC,
        "value": head["frames_per_s"],
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: {spec.k}x{spec.k} conv {spec.c_in}->{spec.c_out} stride {spec.stride}, "
                        f"{wl.h}x{wl.w} frames, batch {wl.n} independent streams (one step = one frame of each), "
                        f"{len(clip)}-frame clip (reset at frame 1), gate block {block}, "
                        f"eps for ~{args.density:.0%} block density; steady-state steps after a reference frame",
            "eps": eps_head, "block": block, "density": d_head,
            "density_steady": head["density_steady"],
            "active_tflops": head["active_tflops"], "dense_equiv_tflops": head["dense_equiv_tflops"],
            "pipeline": head["pipeline"], "caller_retains": bool(args.caller_retains),
            "kernel_us": head["gate_us"] if head["pipeline"] == "fused" else None,
            "gate_us": head["gate_us"] if head["pipeline"] == "split" else None,
            "conv_us": head["conv_us"] if head["pipeline"] == "split" else None,
            "reference_frame_us": head["reference_frame_us"],
            "model_us_per_step": model_us(d_head, args.caller_retains),
            "model_frac": model_us(d_head, args.caller_retains) / (1e3 * head["ms_per_step"]),
            "kernels": kernels or None,
            "measured_peaks": meas,
        },
        "roofline": roof,
        "cpu_baseline": cpu,
        "sweep": sweep,
    }
    print(json.dumps(out), flush=True)


def measured_peaks():
    """Achievable peaks on this device, measured with torch next to the datasheet figures:
    a 2 GiB device-to-device copy (bytes read + written per second) and a large bf16 GEMM
    (hipBLASLt through torch.matmul)."""
    import torch

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e-3 / reps

    n = 2 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    t = timed(lambda: dst.copy_(src), 20)
    copy_gbs = 2 * n / t / 1e9
    del src, dst
    # two streams read, one written (the gate's pattern: x_t, x_(t-1) in, x_t kept)
    k = 256 << 20
    xa = torch.zeros(k // 4, dtype=torch.int32, device="cuda")
    xb = torch.ones_like(xa)
    xc = torch.empty_like(xa)
    t = timed(lambda: torch.bitwise_xor(xa, xb, out=xc), 20)
    stream_gbs = 3 * k / t / 1e9
    del xa, xb, xc
    m = 8192
    a = torch.randn(m, m, device="cuda", dtype=torch.bfloat16)
    bm = torch.randn(m, m, device="cuda", dtype=torch.bfloat16)
    t = timed(lambda: torch.matmul(a, bm), 20)
    gemm = 2.0 * m ** 3 / t / 1e12
    del a, bm
    hbm = max(copy_gbs, stream_gbs)
    log(f"[bench] measured peaks: device copy {copy_gbs:.0f} GB/s, 2-read 1-write stream {stream_gbs:.0f} GB/s, "
        f"bf16 GEMM {gemm:.0f} TFLOP/s")
    return {"hbm_copy_gbs": copy_gbs, "hbm_stream_gbs": stream_gbs, "hbm_measured_gbs": hbm,
            "bf16_gemm_tflops": gemm, "hbm_spec_gbs": PEAK_HBM_GBS, "bf16_spec_tflops": PEAK_BF16_TFLOPS,
            "how": "torch: 2 GiB device copy (read + write bytes); 3 x 256 MiB int32 xor (2 reads, 1 write); "
                   "8192^3 bf16 matmul; hbm_measured_gbs = the larger of the two streams"}


if __name__ == "__main__":
    main()
