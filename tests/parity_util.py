"""Helpers for comparing GPU arenas with the oracle's (test-only)."""
from __future__ import annotations

import numpy as np

from paper_2608_14635_amd import workloads as W

TOL = {W.F32: 1e-4, W.BF16: 2e-2}


def to_float(bits: np.ndarray, dt: int) -> np.ndarray:
    if dt == W.BF16:
        return W.bf16_bits_to_f32(bits)
    return bits.view(np.float32)


def written_mask(wl: W.Workload) -> np.ndarray:
    s = wl.shape
    m = np.zeros((s.num_layers, 2, wl.num_blocks, wl.block_size), bool)
    for r in range(wl.num_requests):
        p = np.arange(int(wl.lens[r]))
        m[:, :, wl.block_tables[r, p // wl.block_size], p % wl.block_size] = True
    return m


def compare(wl: W.Workload, gpu_bits: np.ndarray, ora_bits: np.ndarray, before_bits: np.ndarray):
    """Returns (worst normwise error per layer [L, 2], report dict).

    Error metric per (layer, K|V, kv head) tensor over written slots:
    max|g - o| / max|o|.  Unwritten slots must keep their pre-fill bits
    exactly and written slots must hold finite values."""
    s = wl.shape
    dt = s.dtype
    shp = (s.num_layers, 2, wl.num_blocks, wl.block_size, s.num_kv_heads, s.head_dim)
    g = gpu_bits.reshape(shp)
    o = ora_bits.reshape(shp)
    b = before_bits.reshape(shp)
    m = written_mask(wl)
    report = {}
    report["unwritten_changed"] = int(np.sum(g[~m] != b[~m]))
    gf = to_float(g[m], dt)  # [n_written, nkv, d] across all layers/planes
    report["written_nonfinite"] = int(np.sum(~np.isfinite(gf)))
    worst = np.zeros((s.num_layers, 2))
    for l in range(s.num_layers):
        for kv in range(2):
            mm = m[l, kv]
            if not mm.any():
                continue
            gv = to_float(g[l, kv][mm], dt).astype(np.float64)
            ov = to_float(o[l, kv][mm], dt).astype(np.float64)
            for h in range(s.num_kv_heads):
                den = np.max(np.abs(ov[:, h]))
                err = np.max(np.abs(gv[:, h] - ov[:, h])) / (den if den > 0 else 1.0)
                if not np.isfinite(err):
                    err = np.inf  # a NaN would otherwise vanish in max() below
                worst[l, kv] = max(worst[l, kv], err)
    report["worst"] = float(worst.max()) if worst.size else 0.0
    return worst, report
