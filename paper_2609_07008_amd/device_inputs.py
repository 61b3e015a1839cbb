"""Upload a seeded workload's inputs to the GPU as bfloat16 tensors (bit patterns
from the workload generator; no arithmetic of the method)."""
from __future__ import annotations

import numpy as np
import torch

from workloads import f32_to_bf16_bits


def to_bf16(x: np.ndarray, device="cuda") -> torch.Tensor:
    bits = f32_to_bf16_bits(np.ascontiguousarray(x, dtype=np.float32))
    return torch.from_numpy(bits.view(np.int16)).to(device).view(torch.bfloat16)


def upload(wl, z_off=None, device="cuda", threads=None):
    """kv [N, D], q_glob [N, G, D], q_loc [P, G, hpg-1, D], w_o, z_off [N, d_model] (bf16)."""
    g = wl.geom
    out = {}
    out["kv"] = to_bf16(wl.kv(threads=threads), device)
    out["q_glob"] = to_bf16(wl.q_glob(threads=threads), device)
    if wl.n_prot > 0 and g.heads_per_group > 1:
        out["q_loc"] = to_bf16(wl.q_loc(threads=threads), device)
    else:
        out["q_loc"] = None
    out["w_o"] = to_bf16(wl.w_o(), device)
    if z_off is None:
        z_off = wl.z_off(threads=threads)
    out["z_off"] = to_bf16(z_off, device)
    return out
