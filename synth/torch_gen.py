"""Device-side generator of the same recipe, for full-size workloads.

Per-channel scales (and the outlier channels) come from the same numpy cell
streams as ``workloads``; the Gaussian draws come from a torch generator on the
target device seeded per (workload, layer, tensor), and RoPE angles are formed
in fp32.  Values therefore differ from the numpy path, but each run is
reproducible, and a consumer that checks a cell reads that cell's stored values
back from these tensors.
"""
from __future__ import annotations

import numpy as np
import torch

from .workloads import Workload, cell_rng, channel_scales, _TENSOR_ID

_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def _seed(wl: Workload, *key: int) -> int:
    return int(cell_rng(wl.wid, *key, 1 << 23).integers(0, 2**62))


def _scales(wl: Workload, layer: int, tensor: str, n_heads: int, device) -> torch.Tensor:
    tid = _TENSOR_ID[tensor]
    sig = np.stack([channel_scales(cell_rng(wl.wid, layer, h, tid, 1 << 20), wl.d, wl.n_outliers,
                                   wl.outlier_mult) for h in range(n_heads)])
    return torch.from_numpy(sig).to(device, torch.float32)


def rope_torch(x: torch.Tensor, positions: torch.Tensor, base: float, layout: str) -> torch.Tensor:
    """x [..., n, H, d] float32 rotated at positions [n]."""
    d = x.shape[-1]
    half = d // 2
    j = torch.arange(half, device=x.device, dtype=torch.float64)
    theta = (base ** (-2.0 * j / d))
    ang = (positions.to(torch.float64)[:, None] * theta[None, :]).to(torch.float32)
    cos = torch.cos(ang)[:, None, :]
    sin = torch.sin(ang)[:, None, :]
    if layout == "half":
        a, b = x[..., :half], x[..., half:]
        return torch.cat([a * cos - b * sin, b * cos + a * sin], dim=-1)
    a, b = x[..., 0::2], x[..., 1::2]
    out = torch.empty_like(x)
    out[..., 0::2] = a * cos - b * sin
    out[..., 1::2] = b * cos + a * sin
    return out


def gen_kv_layer(wl: Workload, layer: int, seq: int, positions: torch.Tensor, step: int = -1,
                 device="cuda"):
    """Stored (k, v) of one sequence and layer: [n, n_kv, d] in the workload dtype."""
    n = positions.numel()
    out = []
    for tensor in ("k", "v"):
        g = torch.Generator(device=device)
        g.manual_seed(_seed(wl, layer, _TENSOR_ID[tensor], seq, step + 1))
        x = torch.randn((n, wl.n_kv, wl.d), generator=g, device=device, dtype=torch.float32)
        x *= _scales(wl, layer, tensor, wl.n_kv, device)[None]
        if tensor == "k":
            x = rope_torch(x, positions, wl.rope_base, wl.rope_layout)
        out.append(x.to(_DT[wl.dtype]))
    return out[0], out[1]


def gen_q_batch(wl: Workload, layer: int, step: int, positions: torch.Tensor, device="cuda"):
    """Stored queries [batch, n_q, d] of every sequence at one decode step."""
    g = torch.Generator(device=device)
    g.manual_seed(_seed(wl, layer, _TENSOR_ID["q"], step + 1))
    bsz = positions.numel()
    x = torch.randn((bsz, wl.n_q, wl.d), generator=g, device=device, dtype=torch.float32)
    x *= _scales(wl, layer, "q", wl.n_q, device)[None] * wl.q_scale
    x = torch.stack([rope_torch(x[b:b + 1], positions[b:b + 1], wl.rope_base, wl.rope_layout)[0]
                     for b in range(bsz)])
    return x.to(_DT[wl.dtype])
