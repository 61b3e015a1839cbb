"""Seeded synthetic inputs of the MoE fanout and of the shared W_b projection
(input generation only).

Router weights:

Each row is a softmax over the experts of N(0, 1) logits scaled by a per-row
temperature drawn from U(0.3, 4), so the batch mixes concentrated rows (a few
experts hold most of the weight) with ambiguous ones (weight spread over many).
Rows are drawn in chunks of ROW_CHUNK from PCG64(SeedSequence([seed, chunk])),
so any row subset can be regenerated.
"""
from __future__ import annotations

import numpy as np

from .configs import ROW_CHUNK


def router_weights(n_rows: int, n_experts: int, seed: int = 70080, rows=None) -> np.ndarray:
    """float32 [len(rows), n_experts] router weights (all rows when rows is None)."""
    rows = np.arange(n_rows) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.empty((rows.shape[0], n_experts), dtype=np.float32)
    chunks = np.unique(rows // ROW_CHUNK)
    for c in chunks:
        lo = int(c) * ROW_CHUNK
        m = min(ROW_CHUNK, n_rows - lo)
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, int(c)])))
        temp = rng.uniform(0.3, 4.0, size=(m, 1))
        logits = rng.standard_normal((m, n_experts)) * temp
        e = np.exp(logits - logits.max(axis=1, keepdims=True))
        w = (e / e.sum(axis=1, keepdims=True)).astype(np.float32)
        sel = (rows // ROW_CHUNK) == c
        out[sel] = w[rows[sel] - lo]
    return out


def wb_inputs(n_rows: int, d_in: int, d_out: int, seed: int = 70080, rows=None, z_std: float = 0.05,
              w_std: float = 0.02):
    """bf16-representable float32 inputs of y = W_b z: z rows [len(rows), d_in]
    ~ N(0, z_std^2) drawn per ROW_CHUNK chunk (any row subset regenerates), and
    W_b [d_out, d_in] ~ N(0, w_std^2) (the std of the paper's W_o stand-in)."""
    from .configs import round_bf16
    rows = np.arange(n_rows) if rows is None else np.asarray(rows, dtype=np.int64)
    z = np.empty((rows.shape[0], d_in), dtype=np.float32)
    for c in np.unique(rows // ROW_CHUNK):
        lo = int(c) * ROW_CHUNK
        m = min(ROW_CHUNK, n_rows - lo)
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 1, int(c)])))
        block = rng.standard_normal((m, d_in), dtype=np.float32) * np.float32(z_std)
        sel = (rows // ROW_CHUNK) == c
        z[sel] = block[rows[sel] - lo]
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 2])))
    w = rng.standard_normal((d_out, d_in), dtype=np.float32) * np.float32(w_std)
    return round_bf16(z), round_bf16(w)
