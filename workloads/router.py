"""Seeded synthetic router weights for the MoE fanout (input generation only).

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
