"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics,
independent of the oracle's own formulas (CPU only).

Each check is a plain function so that the mutation tests at the bottom can
plant a plausible mistake in the oracle and confirm that some pin catches it.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.linalg
import torch

from oracle import mla_oracle as M
from workloads import make_custom, make_workload

HERE = os.path.dirname(os.path.abspath(__file__))


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return np.abs(a - b).max() / max(np.abs(b).max(), 1e-300)


# ----------------------------------------------------------------------------
# RoPE: eq:rope, the rotation group, and an independent complex-number form
# ----------------------------------------------------------------------------
def complex_rope(x, angle, base):
    """Half-split RoPE written as complex multiplication: pair j is the complex
    number x_j + i x_{j+h}, multiplied by exp(i * angle * base^(-2j/d))."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    h = d // 2
    z = x[..., :h] + 1j * x[..., h:]
    th = np.array([base ** (-2.0 * j / d) for j in range(h)])
    z = z * np.exp(1j * np.asarray(angle, dtype=np.float64)[..., None] * th)
    return np.concatenate([z.real, z.imag], axis=-1)


def check_rope_complex():
    rng = np.random.default_rng(1)
    for d in (4, 16, 64):
        x = rng.standard_normal((7, d))
        a = rng.integers(-300000, 300000, size=7)
        assert rel(M.rope(x, a, 10000.0), complex_rope(x, a, 10000.0)) < 1e-9


def check_rope_theta_closed_form():
    # base 10000, d = 16: theta_j = 10^(-j/2); d = 64: theta_j = 10^(-j/8)
    assert rel(M.rope_theta(16, 10000.0), 10.0 ** (-np.arange(8) / 2.0)) < 1e-14
    assert rel(M.rope_theta(64, 10000.0), 10.0 ** (-np.arange(32) / 8.0)) < 1e-14
    # d = 2 is the textbook 2x2 rotation by the angle itself
    a = 0.7
    x = np.array([1.3, -0.4])
    rot = np.array([[math.cos(a), -math.sin(a)], [math.sin(a), math.cos(a)]]) @ x
    assert rel(M.rope(x, a, 10000.0), rot) < 1e-15


def check_rope_relative_identity():
    """eq:rope: <R(p_q) q, R(p_k + D) k> = <R(p_q - D) q, R(p_k) k>."""
    rng = np.random.default_rng(2)
    for d in (16, 64):
        for _ in range(20):
            q, k = rng.standard_normal(d), rng.standard_normal(d)
            pq, pk, dd = rng.integers(0, 270000, size=3)
            lhs = M.rope(q, pq, 1e4) @ M.rope(k, pk + dd, 1e4)
            rhs = M.rope(q, pq - dd, 1e4) @ M.rope(k, pk, 1e4)
            assert abs(lhs - rhs) < 1e-9 * (1 + abs(lhs))
            ab = M.rope(M.rope(q, pq, 1e4), pk, 1e4)
            assert rel(ab, M.rope(q, pq + pk, 1e4)) < 1e-9
            assert abs(np.linalg.norm(M.rope(q, pq, 1e4)) - np.linalg.norm(q)) < 1e-12


def test_rope_complex_form():
    check_rope_complex()


def test_rope_theta_closed_form():
    check_rope_theta_closed_form()


def test_rope_relative_identity():
    check_rope_relative_identity()


# ----------------------------------------------------------------------------
# E1: relocated, segment-wise, merged attention == direct attention
# ----------------------------------------------------------------------------
def _family(seed):
    rng = np.random.default_rng(seed)
    nd = int(rng.integers(1, 7))
    lens = [int(x) for x in rng.integers(1, 41, size=nd)]
    perm = [int(x) for x in rng.permutation(nd)]
    G = int(rng.integers(1, 4))
    hpg = int(rng.integers(1, 4))
    d_c = int(rng.choice([16, 64]))
    d_r = int(rng.choice([4, 16]))
    tq = int(rng.integers(0, 9))
    if sum(lens) + tq == 0:
        tq = 1
    return make_custom(lens, req_perm=perm, tq=tq, H=G * hpg, G=G, d_c=d_c, d_r=d_r,
                       d_model=8 * G, prot_frac=0.3, seed=seed)


def check_factorized_equals_direct(wl):
    g = wl.geom
    kv = wl.kv(exact=True)
    q = wl.q_full(exact=True)
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    _, _, pos = M.row_geometry(wl.segs)
    worst = 0.0
    for r in range(wl.n_rows):
        od, ld = M.attend_direct(keys, q[r], int(pos[r]), g.softmax_scale)
        of, lf = M.attend_factorized(kv, wl.segs, q[r], int(pos[r]), g.softmax_scale,
                                     g.d_latent, g.rope_base)
        worst = max(worst, rel(of, od), np.abs(lf - ld).max() / (1 + np.abs(ld).max()))
    assert worst < 1e-11, worst


def test_factorized_equals_direct_tiny_workload():
    check_factorized_equals_direct(make_workload(1))


@pytest.mark.parametrize("seed", range(12))
def test_factorized_equals_direct_random_family(seed):
    check_factorized_equals_direct(_family(seed))


# ----------------------------------------------------------------------------
# E2: the merge
# ----------------------------------------------------------------------------
def check_merge():
    rng = np.random.default_rng(3)
    o = rng.standard_normal((6, 5, 32))
    lse = rng.standard_normal((6, 5)) * 30
    a, la = M.lse_merge(o, lse)
    p = rng.permutation(6)
    b, lb = M.lse_merge(o[p], lse[p])
    assert rel(a, b) < 1e-13 and rel(la, lb) < 1e-13
    one, l1 = M.lse_merge(o[:1], lse[:1])
    assert rel(one, o[0]) < 1e-15 and rel(l1, lse[0]) < 1e-15
    eq, le = M.lse_merge(o[:2], np.stack([lse[0], lse[0]]))
    assert rel(eq, 0.5 * (o[0] + o[1])) < 1e-14
    assert rel(le, lse[0] + math.log(2.0)) < 1e-14
    # merging the softmax statistics of two halves of a score vector equals the
    # softmax over the whole vector (brute force)
    s = rng.standard_normal(50) * 4
    v = rng.standard_normal((50, 8))
    w = np.exp(s - s.max())
    full = (w / w.sum()) @ v
    lfull = s.max() + math.log(w.sum())
    parts = []
    for lo, hi in ((0, 17), (17, 50)):
        ww = np.exp(s[lo:hi] - s[lo:hi].max())
        parts.append(((ww / ww.sum()) @ v[lo:hi], s[lo:hi].max() + math.log(ww.sum())))
    mo, ml = M.lse_merge(np.stack([p_[0] for p_ in parts]), np.array([p_[1] for p_ in parts]))
    assert rel(mo, full) < 1e-13 and abs(ml - lfull) < 1e-12


def test_merge():
    check_merge()


# ----------------------------------------------------------------------------
# E3: protected everywhere => z = W_o^T O_full (block-diagonal W_o built by scipy)
# E8: every head Global => no artifact, z = full recompute
# ----------------------------------------------------------------------------
def _w_matrix(wl, w_o):
    """The full first projection as one [H*d_c, d_model] matrix: block-diagonal
    over projection groups (scipy's block_diag), the plain W_o when n_pg = 1."""
    return scipy.linalg.block_diag(*[np.asarray(w, dtype=np.float64) for w in w_o])


def check_full_projection(wl):
    g = wl.geom
    w_o = wl.w_o(exact=True)
    nan = np.full((wl.n_rows, g.d_model), np.nan)
    res = M.reference_rows(wl, np.arange(wl.n_rows), z_off=nan, exact=True)
    o_full, _ = M.full_recompute_rows(wl, np.arange(wl.n_rows), exact=True)
    z_ref = o_full.reshape(wl.n_rows, -1) @ _w_matrix(wl, w_o)
    assert np.isfinite(res.z).all()
    assert rel(res.z, z_ref) < 1e-12
    # Global + Local contributions equal the full projection
    _, z_full = M.full_recompute_rows(wl, np.arange(wl.n_rows), exact=True)
    assert rel(z_full, z_ref) < 1e-12


def test_all_protected_is_full_projection_grouped():
    wl = make_custom([9, 14, 5], req_perm=[2, 0, 1], tq=4, H=6, G=3, d_c=16, d_r=4, d_model=12,
                     seed=5, prot_rows=np.arange(32))
    check_full_projection(wl)


def test_all_protected_is_full_projection_dense():
    wl = make_custom([9, 14], req_perm=[1, 0], tq=4, H=4, G=2, d_c=16, d_r=4, d_model=10,
                     n_pg=1, seed=6, prot_rows=np.arange(27))
    check_full_projection(wl)


def check_all_global(wl):
    z_off = M.artifact(wl, exact=True)
    assert np.all(z_off == 0.0)
    res = M.reference_rows(wl, np.arange(wl.n_rows), z_off=z_off, exact=True)
    _, z_full = M.full_recompute_rows(wl, np.arange(wl.n_rows), exact=True)
    assert rel(res.z, z_full) < 1e-12


def test_all_global_heads_is_full_recompute():
    wl = make_custom([12, 7, 9], req_perm=[1, 2, 0], tq=3, H=3, G=3, d_c=16, d_r=4, d_model=9,
                     seed=7, prot_frac=0.2)
    check_all_global(wl)


# ----------------------------------------------------------------------------
# E4: the first document of a request is a prefix (offset 0): its artifact is exact
# ----------------------------------------------------------------------------
def check_prefix_document(wl):
    z_off = M.artifact(wl, exact=True)
    seg0 = wl.segs[np.argmin(wl.segs[:, 2])]
    assert seg0[2] == 0
    rows = [r for r in range(seg0[0], seg0[0] + seg0[1]) if r not in set(wl.prot_rows.tolist())]
    assert rows
    res = M.reference_rows(wl, rows, z_off=z_off, exact=True)
    _, z_full = M.full_recompute_rows(wl, rows, exact=True)
    assert rel(res.z, z_full) < 1e-12
    # a relocated document's artifact is NOT exact (Local heads see only their document)
    seg1 = wl.segs[np.argsort(wl.segs[:, 2])[1]]
    rows1 = [r for r in range(seg1[0], seg1[0] + seg1[1]) if r not in set(wl.prot_rows.tolist())]
    res1 = M.reference_rows(wl, rows1, z_off=z_off, exact=True)
    _, z_full1 = M.full_recompute_rows(wl, rows1, exact=True)
    assert rel(res1.z, z_full1) > 1e-6


def test_prefix_document_artifact_is_exact():
    wl = make_custom([10, 13, 8], req_perm=[1, 0, 2], tq=4, H=4, G=2, d_c=16, d_r=4, d_model=8,
                     seed=8, prot_frac=0.25)
    check_prefix_document(wl)


def test_tiny_workload_prefix_document():
    check_prefix_document(make_workload(1))


# ----------------------------------------------------------------------------
# E5: protected rows replace the artifact (never read, never added)
# ----------------------------------------------------------------------------
def test_protected_rows_never_read_artifact():
    wl = make_workload(1)
    z_off = M.artifact(wl, exact=True)
    rows = np.arange(wl.n_rows)
    a = M.reference_rows(wl, rows, z_off=z_off, exact=True)
    poisoned = z_off.copy()
    poisoned[wl.prot_rows] = np.nan
    b = M.reference_rows(wl, rows, z_off=poisoned, exact=True)
    assert np.isfinite(b.z).all()
    assert np.array_equal(a.z, b.z)
    # unprotected rows do add it
    un = np.setdiff1d(rows, wl.prot_rows)
    assert rel(a.z[un] - a.z_online[un], z_off[un]) < 1e-15


# ----------------------------------------------------------------------------
# E7: closed forms of softmax attention
# ----------------------------------------------------------------------------
def test_closed_forms():
    wl = make_custom([6, 9], req_perm=[1, 0], tq=3, H=2, G=1, d_c=16, d_r=4, d_model=4, seed=9)
    g = wl.geom
    kv = wl.kv(exact=True).astype(np.float64)
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    _, _, pos = M.row_geometry(wl.segs)
    order = np.argsort(pos)
    for r in range(wl.n_rows):
        t = int(pos[r])
        o, lse = M.attend_direct(keys, np.zeros((1, g.d_qk)), t, g.softmax_scale)
        vis = kv[order[: t + 1], : g.d_latent]
        assert rel(o[0], vis.mean(axis=0)) < 1e-13
        assert abs(lse[0] - math.log(t + 1)) < 1e-13
    # the row at request position 0 sees exactly one key: itself
    r0 = int(order[0])
    q = wl.q_full(exact=True)[r0]
    o, lse = M.attend_direct(keys, q, 0, g.softmax_scale)
    assert rel(o, np.broadcast_to(kv[r0, : g.d_latent], o.shape)) < 1e-15
    s = g.softmax_scale * (q[:, : g.d_latent] @ kv[r0, : g.d_latent]
                           + M.rope(q[:, g.d_latent:], 0, g.rope_base) @ kv[r0, g.d_latent:])
    assert rel(lse, s) < 1e-13


# ----------------------------------------------------------------------------
# E9: one document at offset 0 with every row protected is textbook causal
# attention: compare with torch's scaled_dot_product_attention (fp64, CPU)
# ----------------------------------------------------------------------------
def check_textbook_sdpa():
    wl = make_custom([37], tq=0, H=3, G=1, d_c=64, d_r=16, d_model=8, seed=10,
                     prot_rows=np.arange(37))
    g = wl.geom
    kv = wl.kv(exact=True)
    q = wl.q_full(exact=True)                           # [T, H, D]
    t = np.arange(wl.n_rows)
    # true-position queries via the complex form; canonical keys at offset 0 are true keys
    qt = np.concatenate([q[..., : g.d_latent],
                         complex_rope(q[..., g.d_latent:], np.repeat(t[:, None], g.n_heads, 1), 1e4)], -1)
    Q = torch.from_numpy(qt.transpose(1, 0, 2).copy())              # [H, T, D]
    K = torch.from_numpy(kv.astype(np.float64))[None].expand(g.n_heads, -1, -1)
    V = torch.from_numpy(kv[:, : g.d_latent].astype(np.float64))[None].expand(g.n_heads, -1, -1)
    ref = torch.nn.functional.scaled_dot_product_attention(Q, K, V, is_causal=True,
                                                           scale=g.softmax_scale).numpy()
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    for r in range(wl.n_rows):
        o, _ = M.attend_direct(keys, q[r], r, g.softmax_scale)
        assert rel(o, ref[:, r, :]) < 1e-12


def test_textbook_sdpa():
    check_textbook_sdpa()


# ----------------------------------------------------------------------------
# needles: a planted key dominates exactly the rows that can see it
# ----------------------------------------------------------------------------
def test_needle_visibility():
    wl = make_custom([20, 16, 24], req_perm=[2, 0, 1], tq=6, H=2, G=1, d_c=16, d_r=16, d_model=4,
                     seed=11)
    g = wl.geom
    kv = wl.kv(exact=True).astype(np.float64)
    q = wl.q_full(exact=True)
    seg, u, pos = M.row_geometry(wl.segs)
    r = wl.n_rows - 1                       # last query row
    t = int(pos[r])
    s = int(np.argsort(wl.segs[:, 2])[1])   # second document in request order
    ks, ln, ps = wl.segs[s]
    j = int(ks + 5)
    qr = q[r, 0, g.d_latent:]
    # canonical-frame key aligned with the relocated query: score ~ +40
    kv[j, g.d_latent:] = 40.0 / g.softmax_scale * M.rope(qr, t - ps, g.rope_base) / (qr @ qr)
    kv[j, : g.d_latent] = 0.0
    kv[j, 0] = 5.0
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    o, lse = M.attend_direct(keys, q[r], t, g.softmax_scale)
    assert abs(o[0, 0] - 5.0) < 1e-6 and np.abs(o[0, 1:]).max() < 1e-6
    of, _ = M.attend_factorized(kv, wl.segs, q[r], t, g.softmax_scale, g.d_latent, g.rope_base)
    assert rel(of, o) < 1e-11
    # a row placed just before the needle cannot see it
    rb = int(np.nonzero(pos == pos[j] - 1)[0][0])
    kv2 = kv.copy()
    kv2[j] = wl.kv(exact=True)[j]
    a, _ = M.attend_direct(keys, q[rb], int(pos[rb]), g.softmax_scale)
    b, _ = M.attend_direct(M.TrueKeys(kv2, wl.segs, g.d_latent, g.rope_base), q[rb], int(pos[rb]),
                           g.softmax_scale)
    assert np.array_equal(a, b)


# ----------------------------------------------------------------------------
# bookkeeping: brute-force visibility and the chunk rule
# ----------------------------------------------------------------------------
def check_bookkeeping(wl, split_keys):
    G, hpg = wl.geom.n_groups, wl.geom.heads_per_group
    row_src, ptr, pseg = M.enumerate_plan(wl.segs, G, hpg, wl.prot_rows, split_keys)
    seg, _, pos = M.row_geometry(wl.segs)
    n = wl.n_rows
    hl = hpg - 1
    n_slots = n * G + wl.n_prot * G * hl
    assert ptr.shape == (n_slots + 1,) and ptr[0] == 0 and np.all(np.diff(ptr) >= 1)
    assert pseg.shape == (ptr[-1], 2)
    assert np.array_equal(np.nonzero(row_src)[0], np.asarray(wl.prot_rows))
    req_rank = np.argsort(np.argsort(wl.segs[:, 2]))
    # brute force: segment s is visible to row r iff some key of s sits at a
    # true position <= pos[r]
    vis = {}
    for r in range(n):
        vis[r] = sorted({int(seg[j]) for j in range(n) if pos[j] <= pos[r]}, key=lambda s: req_rank[s])

    def slot_row(i):
        return i // G if i < n * G else int(wl.prot_rows[(i - n * G) // (G * hl)])

    for i in range(n_slots):
        parts = pseg[ptr[i]:ptr[i + 1]]
        covered = []
        for a, b in parts:
            ra, rb = req_rank[a], req_rank[b]
            assert ra <= rb
            block = [int(s) for s in np.argsort(wl.segs[:, 2])[ra:rb + 1]]
            if split_keys > 0 and len(block) > 1:
                assert wl.segs[block, 1].sum() <= split_keys
            covered += block
        assert covered == vis[slot_row(i)]
        if split_keys == 0:
            assert all(a == b for a, b in parts)
        elif len(parts) > 1:
            # greedy: each chunk could not take the next chunk's first segment
            for (a, b), (c, _) in zip(parts[:-1], parts[1:]):
                blk = np.argsort(wl.segs[:, 2])[req_rank[a]:req_rank[b] + 1]
                assert wl.segs[blk, 1].sum() + wl.segs[c, 1] > split_keys


@pytest.mark.parametrize("split_keys", [0, 1, 25, 60, 10 ** 9])
def test_bookkeeping_brute_force(split_keys):
    wl = make_custom([7, 19, 3, 11], req_perm=[2, 0, 3, 1], tq=5, H=6, G=2, d_c=16, d_r=4,
                     d_model=8, seed=12, prot_frac=0.3)
    check_bookkeeping(wl, split_keys)


def test_bookkeeping_tiny_workload():
    check_bookkeeping(make_workload(1), 0)


def test_per_segment_partial_counts_large():
    """Per-segment mode at the 32K shape: a row of the k-th document in request
    order has exactly k+1 partials per slot (closed form)."""
    wl = make_workload(3)
    G, hpg = wl.geom.n_groups, wl.geom.heads_per_group
    row_src, ptr, pseg = M.enumerate_plan(wl.segs, G, hpg, wl.prot_rows, 0)
    seg, _, _ = M.row_geometry(wl.segs)
    rank = np.argsort(np.argsort(wl.segs[:, 2]))
    cnt = np.diff(ptr)
    n = wl.n_rows
    assert np.array_equal(cnt[: n * G], np.repeat(rank[seg] + 1, G))
    assert np.array_equal(cnt[n * G:], np.repeat(rank[seg[wl.prot_rows]] + 1, G * (hpg - 1)))


# ----------------------------------------------------------------------------
# head partition: the paper's printed structural ceilings (eq:ceiling)
# ----------------------------------------------------------------------------
def test_head_partition_printed_ceiling():
    gold = json.load(open(os.path.join(HERE, "golden", "paper_profiles.json")))["profiles"]
    for name, p in gold.items():
        H = p["local_heads"] + p["global_heads"]
        wl = make_custom([4], tq=0, H=H, G=H // p["heads_per_group"], d_c=16, d_r=4, d_model=8)
        n_local = wl.local_head_ids().size
        assert n_local == p["local_heads"]
        assert len(set(wl.local_head_ids().ravel()) | set(wl.global_head_ids())) == H
        n_layers = p["fence_front"] + p["reusable"] + p["fence_back"]
        ceiling = p["reusable"] / n_layers * n_local / H
        assert round(100 * ceiling, 2) == p["printed_ceiling_percent"], (name, ceiling)


# ----------------------------------------------------------------------------
# mutation tests: a plausible mistake planted in the oracle fails a pin
# ----------------------------------------------------------------------------
def _rope_wrong_sign(x, angle, base):
    return _ORIG["rope"](x, -np.asarray(angle), base)


def _rope_wrong_pairs(x, angle, base):
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    # adjacent pairs (x_0, x_1), (x_2, x_3), ... instead of half-split pairs
    perm = np.concatenate([np.arange(0, d, 2), np.arange(1, d, 2)])
    inv = np.argsort(perm)
    return _ORIG["rope"](x[..., perm], angle, base)[..., inv]


def _theta_off_by_one(d_r, base):
    j = np.arange(1, d_r // 2 + 1, dtype=np.float64)
    return np.power(base, -2.0 * j / d_r)


def _merge_no_weights(o, lse):
    o = np.asarray(o, dtype=np.float64)
    return o.mean(axis=0), np.asarray(lse).max(axis=0)


def _blocks_wrong_offset(w_o, n_heads, d_latent, d_model):
    out = _ORIG["dense_blocks"](w_o, n_heads, d_latent, d_model)
    return np.roll(out, 1, axis=0) if w_o.shape[0] > 1 else out.transpose(0, 1, 2)[::-1]


def _rope_identity(x, angle, base):
    return np.asarray(x, dtype=np.float64).copy()


_ORIG = {k: getattr(M, k) for k in ("rope", "rope_theta", "lse_merge", "dense_blocks", "row_geometry",
                                    "softmax_stats")}


def _softmax_no_max_shift_wrong_lse(scores, values):
    o, lse = _ORIG["softmax_stats"](scores, values)
    return o, lse - scores.max(axis=-1)


MUTATIONS = {
    "rope_sign": ("rope", _rope_wrong_sign),
    "rope_pairs": ("rope", _rope_wrong_pairs),
    "rope_dropped": ("rope", _rope_identity),
    "theta_index": ("rope_theta", _theta_off_by_one),
    "merge_weights": ("lse_merge", _merge_no_weights),
    "oproj_blocks": ("dense_blocks", _blocks_wrong_offset),
    "lse_term": ("softmax_stats", _softmax_no_max_shift_wrong_lse),
}


def _all_checks():
    check_rope_complex()
    check_rope_theta_closed_form()
    check_rope_relative_identity()
    check_merge()
    check_textbook_sdpa()
    check_full_projection(make_custom([9, 14, 5], req_perm=[2, 0, 1], tq=4, H=6, G=3, d_c=16, d_r=4,
                                      d_model=12, seed=5, prot_rows=np.arange(32)))
    check_factorized_equals_direct(_family(3))
    test_closed_forms()


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, bad = MUTATIONS[name]
    monkeypatch.setattr(M, attr, bad)
    with pytest.raises(AssertionError):
        _all_checks()


def test_unmutated_checks_pass():
    _all_checks()


# ----------------------------------------------------------------------------
# protected token-row set (Sec. 2.3, eq:protected)
# ----------------------------------------------------------------------------
def _protect_case(seed=0, n_docs=5, qlen=7, edge=3, tail=9, budget=0.3, ties=False):
    rng = np.random.default_rng(seed)
    lens = rng.integers(2, 14, size=n_docs).tolist()
    perm = rng.permutation(n_docs).tolist()
    wl = make_custom(lens, req_perm=perm, tq=qlen, H=4, G=2, seed=seed)
    segs = np.asarray(wl.segs, dtype=np.int64)
    n = int(segs[:, 1].sum())
    flags = np.zeros(n, dtype=np.uint8)
    flags[rng.choice(n, size=3, replace=False)] |= 1
    flags[rng.choice(n, size=3, replace=False)] |= 2
    scores = rng.standard_normal(n).astype(np.float32)
    if ties:
        scores = np.round(scores).astype(np.float32)
    return segs, n_docs, flags, scores, edge, tail, budget


def _fixed_sets_by_rows(segs, qseg, flags, edge, tail):
    """The fixed sets of eq:protected, row by row from the segment table."""
    n = int(segs[:, 1].sum())
    base, cand = set(), set()
    for s, (ks, ln, ro) in enumerate(segs):
        for u in range(int(ln)):
            r = int(ks) + u
            t = int(ro) + u
            is_q = s == qseg
            is_new = bool(flags[r] & 1)
            in_b = (not is_q) and ro != 0 and (u < edge or u >= ln - edge)
            if is_q or is_new or (flags[r] & 2) or in_b or t >= n - tail:
                base.add(r)
            if not is_q and not is_new:
                cand.add(r)
    return base, cand


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("ties", [False, True])
def test_protected_rows_definition(seed, ties):
    segs, qseg, flags, scores, edge, tail, budget = _protect_case(seed, ties=ties)
    got = M.protected_rows(segs, qseg, flags, scores, edge, tail, budget)
    assert got.dtype == np.int32 and np.all(np.diff(got) > 0)           # ascending, unique
    base, cand = _fixed_sets_by_rows(segs, qseg, flags, edge, tail)
    sel = set(got.tolist())
    assert base <= sel                                                    # Q, N, D, B, T all kept
    target = int(np.floor(budget * len(cand) + 0.5))
    assert len(sel & cand) == max(target, len(base & cand))               # the budget, exactly
    assert sel <= base | cand
    # I_top, by counting for every eligible row how many eligible rows outrank it
    key = M.total_order_key(scores).astype(np.int64)
    elig = sorted(cand - base)
    k = len(sel & cand) - len(base & cand)
    for r in elig:
        beaten_by = sum(1 for x in elig if key[x] > key[r] or (key[x] == key[r] and x < r))
        assert (r in sel) == (beaten_by < k), r


def test_protected_rows_budget_limits():
    segs, qseg, flags, scores, edge, tail, _ = _protect_case(3)
    base, cand = _fixed_sets_by_rows(segs, qseg, flags, edge, tail)
    assert set(M.protected_rows(segs, qseg, flags, scores, edge, tail, 0.0).tolist()) == base
    n = int(segs[:, 1].sum())
    assert M.protected_rows(segs, qseg, flags, scores, edge, tail, 1.0).tolist() == list(range(n))
    assert M.protected_rows(segs, qseg, flags, scores, edge, n, 0.0).tolist() == list(range(n))   # tail covers all


def test_protected_rows_edges_of_relocated_segments_only():
    # three documents: the first at request offset 0 (not relocated), a short one,
    # a long one; no query block, no tail, no budget
    segs = np.array([[0, 10, 0], [10, 4, 30], [14, 20, 10]], dtype=np.int64)
    got = set(M.protected_rows(segs, -1, np.zeros(34, np.uint8), np.zeros(34, np.float32),
                               edge=3, tail=0, budget=0.0).tolist())
    assert got == {10, 11, 12, 13} | {14, 15, 16, 31, 32, 33}


def test_protected_rows_total_order_ties():
    # one relocated-free document of 6 rows; budget 1/2 of 6 candidates -> 3 rows
    segs = np.array([[0, 6, 0]], dtype=np.int64)
    scores = np.array([-0.0, 0.0, 1.0, 1.0, np.nan, -np.inf], dtype=np.float32)
    got = M.protected_rows(segs, -1, np.zeros(6, np.uint8), scores, edge=0, tail=0, budget=0.5).tolist()
    # positive NaN ranks above every number; the two 1.0 tie -> both before +0 and -0
    assert got == [2, 3, 4]
    got = M.protected_rows(segs, -1, np.zeros(6, np.uint8), scores, edge=0, tail=0, budget=4 / 6).tolist()
    assert got == [1, 2, 3, 4]        # +0 ranks above -0


# ----------------------------------------------------------------------------
# adaptive MoE fanout (Sec. 2.4, eq:moe)
# ----------------------------------------------------------------------------
def test_moe_fanout_hand_cases():
    # six weights whose shares are 0.5, 0.2, 0.1, 0.1, 0.05, 0.05, among 8 experts;
    # scaled by 0.37 so that only the normalized shares reach tau
    base = np.array([0.05, 0.5, 0.1, 0.2, 0.05, 0.1, 0.0, 0.01], np.float32)
    p = (base * np.float32(0.37))[None, :]
    expect = {0.10: 3, 0.80: 3, 0.85: 4, 0.93: 5, 0.99: 6, 1.5: 6}
    for tau, k in expect.items():
        idx, w, kk = M.moe_fanout(p, tau)
        assert kk.tolist() == [k], tau
    assert idx.tolist() == [[1, 3, 2, 5, 0, 4]]          # equal weights: the lower expert first
    assert np.array_equal(w[0], p[0, idx[0]])             # original weights, not renormalized
    assert M.moe_fanout(p, 0.65, min_k=1)[2].tolist() == [2]   # 0.5 + 0.2 >= 0.65 > 0.5
    assert M.moe_fanout(p, 0.45, min_k=1)[2].tolist() == [1]


def _moe_rows(seed, n=300, e=64, ties=False):
    rng = np.random.default_rng(seed)
    temp = rng.uniform(0.3, 4.0, size=(n, 1))
    logits = rng.standard_normal((n, e)) * temp
    p = np.exp(logits - logits.max(axis=1, keepdims=True))
    p = (p / p.sum(axis=1, keepdims=True)).astype(np.float32)
    if ties:
        p = (np.round(p * 64) / 64).astype(np.float32)
    return p


@pytest.mark.parametrize("ties", [False, True])
def test_moe_fanout_top6_brute_force(ties):
    p = _moe_rows(1, ties=ties)
    idx, w, _ = M.moe_fanout(p, 0.9)
    for r in range(p.shape[0]):
        ranked = sorted(range(p.shape[1]), key=lambda x: (-float(p[r, x]), x))[:6]
        assert idx[r].tolist() == ranked
        assert np.array_equal(w[r], p[r, ranked])


def test_moe_fanout_matches_exact_arithmetic_away_from_tau():
    """fp64 shares decide the same K wherever no cumulative share lies within
    1e-5 of tau (the float32 decision can only differ at the threshold)."""
    p = _moe_rows(2, n=500)
    for tau in (0.5, 0.7, 0.8, 0.9, 0.95):
        _, w, k32 = M.moe_fanout(p, tau)
        w64 = w.astype(np.float64)
        cum = np.cumsum(w64 / w64.sum(axis=1, keepdims=True), axis=1)
        ok = np.all(np.abs(cum - tau) > 1e-5, axis=1)
        k64 = np.array([next((k for k in range(3, 7) if cum[r, k - 1] >= tau), 6) for r in range(p.shape[0])])
        assert ok.sum() > 400
        assert np.array_equal(k32[ok], k64[ok])
        assert np.all((k32 >= 3) & (k32 <= 6))


def test_moe_fanout_monotone_in_tau_and_extremes():
    p = _moe_rows(3)
    ks = [M.moe_fanout(p, t)[2] for t in np.linspace(0.0, 1.0, 21)]
    for a, b in zip(ks, ks[1:]):
        assert np.all(b >= a)
    assert np.all(M.moe_fanout(p, 0.0)[2] == 3)
    assert np.all(M.moe_fanout(p, 1.01)[2] == 6)
    # a row of zeros has no shares: the full top-6 is kept
    z = np.zeros((1, 16), np.float32)
    idx, w, k = M.moe_fanout(z, 0.5)
    assert k.tolist() == [6] and idx.tolist() == [[0, 1, 2, 3, 4, 5]]


# ----------------------------------------------------------------------------
# shared second projection y = W_b z (Sec. 2.1 eq:factorization, Alg. 2)
# ----------------------------------------------------------------------------
def test_shared_wb_brute_force_and_identities():
    rng = np.random.default_rng(4)
    z = rng.standard_normal((5, 7))
    w = rng.standard_normal((3, 7))           # [d_out, d_in], not square: a transposed operand fails
    y = M.shared_wb(z, w)
    assert y.shape == (5, 3)
    for r in range(5):
        for o in range(3):
            assert abs(y[r, o] - sum(w[o, i] * z[r, i] for i in range(7))) < 1e-12
    assert np.allclose(M.shared_wb(z, np.eye(7)), z, rtol=0, atol=1e-15)
    # y = W_b (z_off + z_online) = W_b z_off + W_b z_online (eq:factorization meets one W_b)
    z2 = rng.standard_normal((5, 7))
    assert np.allclose(M.shared_wb(z + z2, w), M.shared_wb(z, w) + M.shared_wb(z2, w), rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------
# rotary value: RestorePhase per segment and inverse output RoPE (Sec. 2.1
# eq:offonline, Alg. 2)
# ----------------------------------------------------------------------------
def _vrope_family(seed):
    rng = np.random.default_rng(500 + seed)
    nd = int(rng.integers(2, 5))
    lens = [int(x) for x in rng.integers(1, 30, size=nd)]
    perm = [int(x) for x in rng.permutation(nd)]
    return make_custom(lens, req_perm=perm, tq=int(rng.integers(1, 6)), H=4, G=2, d_c=16, d_r=8,
                       d_model=8, prot_frac=0.3, seed=600 + seed, value_rope=True)


@pytest.mark.parametrize("seed", range(6))
def test_value_rope_factorized_equals_direct(seed):
    """With a rotary value the factorized route equals the direct definition
    only when each partial's phase is restored (R(+p_s)) before the merge: the
    restore is what the GPU must reproduce, and dropping it is caught here."""
    wl = _vrope_family(seed)
    g = wl.geom
    kv = wl.kv(exact=True)
    q = wl.q_full(exact=True)
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    _, _, pos = M.row_geometry(wl.segs)
    worst, worst_unrestored = 0.0, 0.0
    for r in range(wl.n_rows):
        od, ld = M.attend_direct(keys, q[r], int(pos[r]), g.softmax_scale, value_rope=True)
        of, lf = M.attend_factorized(kv, wl.segs, q[r], int(pos[r]), g.softmax_scale, g.d_latent,
                                     g.rope_base, value_rope=True)
        ou, _ = M.attend_factorized(kv, wl.segs, q[r], int(pos[r]), g.softmax_scale, g.d_latent,
                                    g.rope_base, value_rope=True, restore=False)
        assert od.shape[1] == g.d_latent + g.d_rope
        assert np.allclose(od[:, :g.d_latent], M.attend_direct(keys, q[r], int(pos[r]), g.softmax_scale)[0],
                           rtol=0, atol=1e-14)                      # the latent part is unchanged
        worst = max(worst, rel(of, od), np.abs(lf - ld).max() / (1 + np.abs(ld).max()))
        worst_unrestored = max(worst_unrestored, rel(ou, od))
    assert worst < 1e-11, worst
    assert worst_unrestored > 1e-3


def test_value_rope_relative_rotation_brute_force():
    """The head output's RoPE part is sum_j softmax_j R(P_j - t) k^_j: each
    value rotated by its position relative to the query (R^{-1} R(P) = R(P - t)),
    written here key by key from the raw keys k^ = R(-u) k_r."""
    wl = _vrope_family(1)
    g = wl.geom
    kv = wl.kv(exact=True)
    q = wl.q_full(exact=True)
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    seg, u, pos = M.row_geometry(wl.segs)
    by_pos = np.argsort(pos)
    for r in range(0, wl.n_rows, 3):
        t = int(pos[r])
        od, _ = M.attend_direct(keys, q[r], t, g.softmax_scale, value_rope=True)
        qt = np.concatenate([q[r][:, :g.d_latent], M.rope(q[r][:, g.d_latent:], np.full(g.n_heads, t), g.rope_base)],
                            axis=1)
        s = g.softmax_scale * (qt @ keys.k[: t + 1].T)
        w = np.exp(s - s.max(axis=1, keepdims=True))
        w /= w.sum(axis=1, keepdims=True)
        acc = np.zeros((g.n_heads, g.d_rope))
        for p_j in range(t + 1):
            j = by_pos[p_j]
            raw = M.rope(kv[j:j + 1, g.d_latent:].astype(np.float64), np.array([-u[j]]), g.rope_base)[0]
            acc += w[:, p_j:p_j + 1] * M.rope(raw[None, :], np.array([p_j - t]), g.rope_base)[0][None, :]
        assert rel(od[:, g.d_latent:], acc) < 1e-12


def test_value_rope_prefix_document_artifact_is_exact():
    wl = make_custom([10, 13, 8], req_perm=[1, 0, 2], tq=4, H=4, G=2, d_c=16, d_r=4, d_model=8,
                     seed=8, prot_frac=0.25, value_rope=True)
    check_prefix_document(wl)
