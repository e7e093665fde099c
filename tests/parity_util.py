"""Shared helpers of the GPU parity tests: drive the HIP layer and the CPU
oracle on the same seeded frames and compare them frame by frame."""
from __future__ import annotations

import numpy as np

from oracle import skipconv_oracle as O

TOL = {"f32": 1e-4, "bf16": 2e-2}  # normwise relative bound on z after every frame (the contract)
ORDER_TOL = 1e-4   # normwise, both dtypes: accumulation order only (measured <= 1.8e-6)
ELEM_TOL = 1e-2    # per element, relative to |z| + 1e-3 max|z| (measured <= 4.4e-4)


def say(msg: str) -> None:
    print(msg, flush=True)


def to_device(x_storage: np.ndarray, dtype: str):
    """Upload a storage array (float32, or bf16 bit patterns) as a CUDA tensor of the layer dtype."""
    import torch

    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(x_storage, np.float32)).cuda()
    t = torch.from_numpy(np.ascontiguousarray(x_storage).view(np.int16)).cuda()
    return t.view(torch.bfloat16)


def to_host_storage(t, dtype: str) -> np.ndarray:
    import torch

    if dtype == "f32":
        return t.detach().float().cpu().numpy()
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def weight_storage(w_f32: np.ndarray, dtype: str) -> np.ndarray:
    return w_f32.astype(np.float32) if dtype == "f32" else O.f32_to_bf16_rne(w_f32)


def rel_err(z_gpu: np.ndarray, z_ref: np.ndarray) -> float:
    """max |z_gpu - z_ref| / max |z_ref| over finite entries; NaN layout must agree."""
    ng, nr = np.isnan(z_gpu), np.isnan(z_ref)
    assert np.array_equal(ng, nr), f"NaN layout differs at {int((ng ^ nr).sum())} entries"
    fin = ~nr
    if not fin.any():
        return 0.0
    den = max(float(np.max(np.abs(z_ref[fin]))), 1e-30)
    return float(np.max(np.abs(z_gpu[fin].astype(np.float64) - z_ref[fin]))) / den


def compare_frame(layer, ref: dict, dtype: str, *, t: int, tag: str, keep_stats: bool,
                  exact_z: bool = False, z_gpu=None) -> float:
    """Bit-exact gate outputs, z within the tolerance (or bit-exact)."""
    import torch

    torch.cuda.synchronize()
    bm = layer.block_mask()
    assert np.array_equal(bm.astype(bool), ref["block_mask"]), f"{tag} t={t}: block mask differs"
    lst = layer.active_list()
    assert np.array_equal(lst, ref["active"]), f"{tag} t={t}: active list differs"
    if not layer.fused:
        check_work_list(layer, ref["active"], tag=tag, t=t)
    blocks, sites = layer.active_count()
    assert blocks == ref["count"] and sites == ref["active_sites"], f"{tag} t={t}: counts differ"
    if keep_stats:
        st = layer.stat()
        rs = ref["stat"]
        assert np.array_equal(np.isnan(st), np.isnan(rs)), f"{tag} t={t}: stat NaN layout"
        fin = ~np.isnan(rs)
        assert np.array_equal(st[fin].view(np.uint32), rs[fin].view(np.uint32)), \
            f"{tag} t={t}: gate statistic not bit-exact"
        assert np.array_equal(layer.site_mask().astype(bool), ref["site_mask"]), f"{tag} t={t}: site mask"
    zg = (z_gpu if z_gpu is not None else layer._z).cpu().numpy()
    if exact_z:
        assert np.array_equal(zg.astype(np.float64), ref["z"]), f"{tag} t={t}: z not bit-exact"
        return 0.0
    e = rel_err(zg, ref["z"])
    assert e <= TOL[dtype], f"{tag} t={t}: z rel err {e:.3e} > {TOL[dtype]}"
    # tighter than the contract: both sides apply the same operand rounding,
    # so what remains is the fp32 accumulation order of one frame's K <= 1152
    # products (K * 2^-24 < 1e-4 normwise) carried over the frames
    assert e <= ORDER_TOL, f"{tag} t={t}: z rel err {e:.3e} > {ORDER_TOL} (accumulation-order bound)"
    pe = elementwise_err(zg, ref["z"])
    assert pe <= ELEM_TOL, f"{tag} t={t}: per-element z error {pe:.3e} > {ELEM_TOL}"
    return e


def elementwise_err(z_gpu: np.ndarray, z_ref: np.ndarray) -> float:
    """max |z_gpu - z_ref| / (|z_ref| + 1e-3 max |z_ref|) over finite entries: an
    update missing at a few sites shows here even when the normwise error is small."""
    fin = ~np.isnan(z_ref)
    if not fin.any():
        return 0.0
    scale = max(float(np.max(np.abs(z_ref[fin]))), 1e-30)
    d = np.abs(z_gpu[fin].astype(np.float64) - z_ref[fin])
    return float(np.max(d / (np.abs(z_ref[fin]) + 1e-3 * scale)))


def check_work_list(layer, active, *, tag: str, t: int) -> None:
    """The list the split pipeline's convolution walked (the gate's own appends, unordered):
    every active block exactly once, nothing else."""
    wl = layer.work_list()
    assert len(np.unique(wl)) == len(wl), f"{tag} t={t}: work list holds a block twice"
    assert np.array_equal(np.sort(wl), active), f"{tag} t={t}: work list is not the active set"


def eps_for_density(stat_frames, block: int, h_out: int, w_out: int, target: float,
                    norm_p: int = 2) -> float:
    """eps giving about `target` mean block density over the given oracle statistics."""
    vals = []
    for s in stat_frames:
        n = s.shape[0]
        hb, wb = -(-h_out // block), -(-w_out // block)
        pad = np.full((n, hb * block, wb * block), -np.inf, np.float32)
        pad[:, :h_out, :w_out] = np.nan_to_num(s, nan=np.inf)
        bmax = pad.reshape(n, hb, block, wb, block).max(axis=(2, 4))
        vals.append(bmax.reshape(-1))
    v = np.concatenate(vals).astype(np.float64)
    q = float(np.quantile(v, 1.0 - target))
    return float(np.sqrt(max(q, 0.0))) if norm_p == 2 else q
