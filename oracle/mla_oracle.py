"""fp64 CPU oracle for the MLA-Online step of RedKnot-MLA (arXiv 2609.07008).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU-baseline
leg of the benchmark may import this module.  It shares no code with the HIP
library (``paper_2609_07008_amd``) and never imports it; its only shared
dependency is the seeded input generator in ``workloads``.

What it computes, and where the paper defines it:

* ``rope`` -- the rotary map R(a) on half-split pairs (x_j, x_{j+d_r/2}) with
  frequencies base^(-2j/d_r).  The paper relies on RoPE orthogonality (Sec. 2.3,
  eq:rope) but does not print the convention; half-split pairs with base 10000
  is the reading used throughout (the tiny workload fixes base 10000).
* ``attend_direct`` -- the plain definition the method must reproduce: every
  online head of a row at true request position t attends, with one softmax,
  to every key whose true position is <= t.  Keys are rebuilt at true
  positions from the canonical-frame artifact rows; nothing is factorized per
  segment and nothing is relocated.  (Full recomputation is the paper's
  reference arm, Sec. 4.1; eq:factorization is exact when the head outputs are
  full-recomputation outputs, Sec. 2.1.)
* ``attend_factorized`` -- the method's own route (Alg. 2): per visible
  document segment, query-side relocation R(t - p_s) (eq:rope), attention to
  the canonical latent, then ``lse_merge`` (the segmented log-sum-exp merge).
  Used only by the tests that pin the identity factorized == direct.
* ``project`` / ``reference_rows`` -- the group-aligned sliced first output
  projection and the artifact restore-and-replace: z = z_online + z_off on rows
  outside the protected set, z = z_online on protected rows, whose cached
  Local values are replaced, never added (Sec. 2.1 eq:offonline and
  eq:factorization, Sec. 2.3, Alg. 2).
* ``artifact`` -- the canonical offline artifact z_off = W_{a,L} O_L with each
  document evaluated alone at positions 0..n-1 (Sec. 2.2, Alg. 1).  How well
  the artifact approximates full recomputation in a changed context depends on
  a trained model and is not a parity claim ("parity unpinned" as a quality
  statement; the function itself is pinned by the prefix-document identity).
* ``enumerate_plan`` -- the integer bookkeeping: which segments each output
  slot sees, how they are cut into partials, and the protected-row flags.
* ``protected_rows`` -- the protected token-row set of Sec. 2.3 (eq:protected):
  query rows, new and dirty rows, the first and last rows of every relocated
  segment, the recent tail, and the Indexer's top rows, which top the
  protected share of the candidate rows up to the controller's budget.
* ``shared_wb`` -- the shared second projection y = W_b z (Sec. 2.1
  eq:factorization; Alg. 2 returns W_b z), with W_b stored as a linear
  layer's weight [d_out, d_in].
* ``moe_fanout`` -- the adaptive MoE fanout of Sec. 2.4 (eq:moe): per token
  row, the router's top-6 experts, and the smallest fanout K in {3,..,6} whose
  normalized top-6 weights reach tau; executed experts keep their original
  weights.  The paper fixes no precision: the integer K is decided in float32
  (normalize by the float32 sum of the six, then accumulate in rank order),
  as the GPU kernel decides it.

Readings where the paper is silent: V is the latent itself, so the inverse
output RoPE and RestorePhase are the identity -- unless the geometry's
``value_rope`` is set: then the value is the whole latent row [c ; k_r] at the
key's true position, a head output's RoPE part is rotated back by the query's
position (R^{-1}, eq:offonline), and the factorized route restores each
canonical-frame partial's phase by R(+p_s) before the merge (RestorePhase,
Alg. 2); a key is visible to a row iff
its true position is <= the row's (the diagonal included); every request row is
an output row, Global heads run on every row and Local heads only on protected
rows (Alg. 2 writes O_G without and O_{L,A} with the protected-set subscript).
"""
from __future__ import annotations

import numpy as np

F64 = np.float64


# ----------------------------------------------------------------------------
# RoPE (Sec. 2.3, eq:rope)
# ----------------------------------------------------------------------------
def rope_theta(d_r: int, base: float) -> np.ndarray:
    """Frequencies theta_j = base^(-2j/d_r), j = 0 .. d_r/2 - 1."""
    j = np.arange(d_r // 2, dtype=F64)
    return np.power(F64(base), -2.0 * j / F64(d_r))


def rope(x: np.ndarray, angle, base: float) -> np.ndarray:
    """R(angle) applied to the last axis of x (length d_r).  Pair j is
    (x_j, x_{j+d_r/2}); it is rotated by angle*theta_j:
        x'_j       = x_j cos - x_{j+h} sin
        x'_{j+h}   = x_j sin + x_{j+h} cos
    `angle` broadcasts against x's leading axes."""
    x = np.asarray(x, dtype=F64)
    d_r = x.shape[-1]
    h = d_r // 2
    ang = np.asarray(angle, dtype=F64)[..., None] * rope_theta(d_r, base)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=-1)


# ----------------------------------------------------------------------------
# segment geometry
# ----------------------------------------------------------------------------
def row_geometry(segs: np.ndarray):
    """For every storage row: its segment, canonical offset u and true position
    P = req_offset + u.  Segments tile the rows in storage and in request space."""
    segs = np.asarray(segs, dtype=np.int64)
    n = int(segs[:, 1].sum())
    seg = np.full(n, -1, dtype=np.int64)
    u = np.zeros(n, dtype=np.int64)
    for i, (ks, ln, _ro) in enumerate(segs):
        seg[ks:ks + ln] = i
        u[ks:ks + ln] = np.arange(ln)
    pos = segs[seg, 2] + u
    return seg, u, pos


# ----------------------------------------------------------------------------
# attention
# ----------------------------------------------------------------------------
def softmax_stats(scores: np.ndarray, values: np.ndarray):
    """Plain softmax over the last axis of `scores` [..., n]: returns
    (sum_j softmax_j values_j, natural-log log-sum-exp)."""
    m = scores.max(axis=-1, keepdims=True)
    e = np.exp(scores - m)
    s = e.sum(axis=-1, keepdims=True)
    o = (e / s) @ values
    lse = (m + np.log(s))[..., 0]
    return o, lse


class TrueKeys:
    """All keys of a request rebuilt at their true positions, in request order.

    The artifact keeps k_r in each document's canonical frame (RoPE applied at
    canonical position u).  The raw key is R(-u) k_r and its true-position key
    is R(P) R(-u) k_r with P = p_s + u.  Sorting rows by P puts the keys visible
    to a row at position t in the first t+1 places."""

    def __init__(self, kv: np.ndarray, segs: np.ndarray, d_latent: int, base: float):
        kv = np.asarray(kv, dtype=F64)
        _, u, pos = row_geometry(segs)
        raw = rope(kv[:, d_latent:], -u, base)
        k_true = np.concatenate([kv[:, :d_latent], rope(raw, pos, base)], axis=1)
        order = np.argsort(pos, kind="stable")
        assert np.array_equal(pos[order], np.arange(pos.shape[0]))
        self.k = np.ascontiguousarray(k_true[order])          # [N, D] request order
        self.c = np.ascontiguousarray(kv[order, :d_latent])    # values = latent
        self.d_latent = d_latent
        self.base = base


def attend_direct(keys: TrueKeys, q: np.ndarray, t: int, scale: float, value_rope: bool = False):
    """Unfactorized attention of one row at true position t.  q [nh, d_c + d_r]
    holds absorbed queries with the RoPE part not yet rotated; it is rotated
    to position t and scored against every key at true position <= t.
    value_rope: the values are the true-position key rows [c ; R(P) k^] and the
    output's RoPE part is rotated back by R(-t) (inverse output RoPE)."""
    q = np.asarray(q, dtype=F64)
    d_c = keys.d_latent
    qt = np.concatenate([q[:, :d_c], rope(q[:, d_c:], np.full(q.shape[0], t), keys.base)], axis=1)
    vis = keys.k[: t + 1]
    scores = F64(scale) * (qt @ vis.T)
    if not value_rope:
        return softmax_stats(scores, keys.c[: t + 1])
    o, lse = softmax_stats(scores, vis)
    o[:, d_c:] = rope(o[:, d_c:], np.full(o.shape[0], -t), keys.base)
    return o, lse


def attend_segment(kv: np.ndarray, seg_row: np.ndarray, q: np.ndarray, delta: int,
                   scale: float, d_latent: int, base: float, value_rope: bool = False):
    """One segment of the factorized route: the query is relocated into the
    segment's canonical frame by R(delta) with delta = t - p_s (eq:rope), and
    scored against the canonical keys of the segment at offsets u <= delta.
    Returns (o_s, lse_s) or None when the segment is not visible.  value_rope:
    the values are the canonical latent rows [c ; k_r], so o_s is in the
    segment's canonical frame (its phase is restored by the caller)."""
    ks, ln, _ = seg_row
    lim = min(delta, ln - 1)
    if lim < 0:
        return None
    q = np.asarray(q, dtype=F64)
    kc = np.asarray(kv[ks:ks + lim + 1], dtype=F64)
    qd = np.concatenate([q[:, :d_latent], rope(q[:, d_latent:], np.full(q.shape[0], delta), base)], axis=1)
    scores = F64(scale) * (qd @ kc.T)
    return softmax_stats(scores, kc if value_rope else kc[:, :d_latent])


def lse_merge(o: np.ndarray, lse: np.ndarray):
    """Segmented log-sum-exp merge of partials o [n, ..., d] with lse [n, ...]:
    m = max lse, w = exp(lse - m), O = sum w o / sum w, lse = m + ln sum w."""
    o = np.asarray(o, dtype=F64)
    lse = np.asarray(lse, dtype=F64)
    m = lse.max(axis=0)
    w = np.exp(lse - m)
    wsum = w.sum(axis=0)
    out = (w[..., None] * o).sum(axis=0) / wsum[..., None]
    return out, m + np.log(wsum)


def attend_factorized(kv, segs, q, t, scale, d_latent, base, value_rope: bool = False, restore: bool = True):
    """Alg. 2 for one row: relocate per visible segment (request order), attend
    to the canonical latent of that segment, then merge the partials.
    value_rope: each partial's RoPE part is moved from the segment's canonical
    frame to true positions by R(+p_s) (RestorePhase; `restore=False` skips it,
    for the tests), and after the merge rotated back by R(-t) (R^{-1})."""
    segs = np.asarray(segs, dtype=np.int64)
    parts_o, parts_l = [], []
    for s in np.argsort(segs[:, 2], kind="stable"):
        delta = int(t - segs[s, 2])
        r = attend_segment(kv, segs[s], q, delta, scale, d_latent, base, value_rope)
        if r is not None:
            o_s = r[0]
            if value_rope and restore:
                o_s = o_s.copy()
                o_s[:, d_latent:] = rope(o_s[:, d_latent:], np.full(o_s.shape[0], int(segs[s, 2])), base)
            parts_o.append(o_s)
            parts_l.append(r[1])
    o, lse = lse_merge(np.stack(parts_o), np.stack(parts_l))
    if value_rope:
        o[:, d_latent:] = rope(o[:, d_latent:], np.full(o.shape[0], -int(t)), base)
    return o, lse


# ----------------------------------------------------------------------------
# first output projection (Sec. 2.1 eq:offonline, Alg. 2)
# ----------------------------------------------------------------------------
def dense_blocks(w_o: np.ndarray, n_heads: int, d_latent: int, d_model: int) -> np.ndarray:
    """Expand W_o [n_pg, (H/n_pg)*d_v, d_model/n_pg] into per-head blocks
    [H, d_v, d_model] (d_v = the head output width, passed as `d_latent`): head h
    of projection group pg = h // (H/n_pg) maps its d_v outputs to channels
    pg*d_model/n_pg .. (pg+1)*d_model/n_pg, zero elsewhere."""
    w_o = np.asarray(w_o, dtype=F64)
    npg = w_o.shape[0]
    hp = n_heads // npg
    cw = d_model // npg
    out = np.zeros((n_heads, d_latent, d_model), dtype=F64)
    for h in range(n_heads):
        pg, hl = divmod(h, hp)
        out[h, :, pg * cw:(pg + 1) * cw] = w_o[pg, hl * d_latent:(hl + 1) * d_latent, :]
    return out


def project(o_heads: np.ndarray, head_ids, blocks: np.ndarray) -> np.ndarray:
    """sum over the listed heads of W_block(h)^T o_h; o_heads [n, d_c]."""
    o_heads = np.asarray(o_heads, dtype=F64)
    z = np.zeros(blocks.shape[2], dtype=F64)
    for o, h in zip(o_heads, head_ids):
        z += o @ blocks[h]
    return z


# ----------------------------------------------------------------------------
# whole step on a set of rows
# ----------------------------------------------------------------------------
class RowResult:
    __slots__ = ("rows", "o_glob", "lse_glob", "o_loc", "lse_loc", "z_online", "z", "prot_idx")


def reference_rows(wl, rows, z_off=None, kv=None, keys=None, w_o=None, exact=False):
    """Direct (unfactorized) reference for the storage rows `rows` of workload `wl`.

    Returns per row: O and lse of the G Global heads; for protected rows also O
    and lse of the Local heads; z_online; and z after restore-and-replace.
    `z_off` maps a storage row to its artifact vector (a full [N, d_model]
    array or a dict); it is read only for rows outside the protected set."""
    g = wl.geom
    rows = np.asarray(rows, dtype=np.int64)
    _, _, pos = row_geometry(wl.segs)
    if kv is None:
        kv = wl.kv(exact=exact)
    if keys is None:
        keys = TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    if w_o is None:
        w_o = wl.w_o(exact=exact)
    vr = bool(getattr(g, "value_rope", False))
    dv = g.d_latent + (g.d_rope if vr else 0)
    blocks = dense_blocks(w_o, g.n_heads, dv, g.d_model)
    glob_ids = wl.global_head_ids()
    loc_ids = wl.local_head_ids()
    prot = np.asarray(wl.prot_rows, dtype=np.int64)
    prot_index = {int(r): i for i, r in enumerate(prot)}
    qg = wl.q_glob(rows=rows, exact=exact)
    pidx = [prot_index[int(r)] for r in rows if int(r) in prot_index]
    ql = wl.q_loc(idx=pidx, exact=exact) if pidx else None
    res = RowResult()
    res.rows = rows
    res.o_glob = np.zeros((rows.shape[0], g.n_groups, dv))
    res.lse_glob = np.zeros((rows.shape[0], g.n_groups))
    res.o_loc, res.lse_loc, res.prot_idx = {}, {}, {}
    res.z_online = np.zeros((rows.shape[0], g.d_model))
    res.z = np.zeros((rows.shape[0], g.d_model))
    k = 0
    for i, r in enumerate(rows):
        t = int(pos[r])
        o, lse = attend_direct(keys, qg[i], t, g.softmax_scale, vr)
        res.o_glob[i], res.lse_glob[i] = o, lse
        zon = project(o, glob_ids, blocks)
        if int(r) in prot_index:
            q = ql[k].reshape(-1, g.d_qk)
            k += 1
            ol, ll = attend_direct(keys, q, t, g.softmax_scale, vr)
            hl = g.heads_per_group - 1
            res.o_loc[i] = ol.reshape(g.n_groups, hl, dv)
            res.lse_loc[i] = ll.reshape(g.n_groups, hl)
            res.prot_idx[i] = prot_index[int(r)]
            zon = zon + project(ol, loc_ids.reshape(-1), blocks)
            res.z[i] = zon                       # replaced: the artifact row is not read
        else:
            res.z[i] = zon + np.asarray(z_off[int(r)], dtype=F64)
        res.z_online[i] = zon
    return res


def full_recompute_rows(wl, rows, kv=None, w_o=None, exact=True, q_all=None):
    """Every head online on every listed row, no artifact: the paper's
    recomputed arm, z = sum_h W_block(h)^T O_h.  q_all [N, H, D] defaults to
    the workload's all-head queries."""
    g = wl.geom
    rows = np.asarray(rows, dtype=np.int64)
    _, _, pos = row_geometry(wl.segs)
    if kv is None:
        kv = wl.kv(exact=exact)
    keys = TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    if w_o is None:
        w_o = wl.w_o(exact=exact)
    vr = bool(getattr(g, "value_rope", False))
    dv = g.d_latent + (g.d_rope if vr else 0)
    blocks = dense_blocks(w_o, g.n_heads, dv, g.d_model)
    if q_all is None:
        q_all = wl.q_full(exact=exact)
    out_o = np.zeros((rows.shape[0], g.n_heads, dv))
    z = np.zeros((rows.shape[0], g.d_model))
    for i, r in enumerate(rows):
        o, _ = attend_direct(keys, q_all[r], int(pos[r]), g.softmax_scale, vr)
        out_o[i] = o
        z[i] = project(o, range(g.n_heads), blocks)
    return out_o, z


def artifact_row(g, kc: np.ndarray, q_loc: np.ndarray, u: int, blocks: np.ndarray, loc) -> np.ndarray:
    """z_off of the row at canonical position u of its segment (Alg. 1): every
    Local head (queries q_loc [L_h, D], in the order of `loc`) attends to the
    segment's keys u' <= u (kc: the segment's rows) with its query rotated to u,
    and the outputs are projected by their W_o blocks."""
    vr = bool(getattr(g, "value_rope", False))
    dv = g.d_latent + (g.d_rope if vr else 0)
    q = np.asarray(q_loc, dtype=F64)
    qc = np.concatenate([q[:, :g.d_latent], rope(q[:, g.d_latent:], np.full(q.shape[0], u), g.rope_base)], axis=1)
    scores = F64(g.softmax_scale) * (qc @ kc[: u + 1].T)
    o, _ = softmax_stats(scores, kc[: u + 1, :dv])
    if vr:   # canonical values carry R(u'); R^{-1} at the row's canonical position u
        o[:, g.d_latent:] = rope(o[:, g.d_latent:], np.full(o.shape[0], -u), g.rope_base)
    return project(o, loc, blocks)


def artifact(wl, kv=None, q_all=None, w_o=None, exact=False) -> np.ndarray:
    """Canonical MLA-Off artifact (Alg. 1): each segment is evaluated alone with
    its first row at position 0; for each row u of a segment, every Local head
    attends to the segment's keys u' <= u with the query rotated to u, and the
    Local outputs are projected: z_off[r] = sum_{h in L} W_block(h)^T O_h^can."""
    g = wl.geom
    if kv is None:
        kv = wl.kv(exact=exact)
    kv = np.asarray(kv, dtype=F64)
    if q_all is None:
        q_all = wl.q_full(exact=exact)
    if w_o is None:
        w_o = wl.w_o(exact=exact)
    vr = bool(getattr(g, "value_rope", False))
    dv = g.d_latent + (g.d_rope if vr else 0)
    blocks = dense_blocks(w_o, g.n_heads, dv, g.d_model)
    loc = wl.local_head_ids().reshape(-1)
    z_off = np.zeros((wl.n_rows, g.d_model))
    for ks, ln, _ in np.asarray(wl.segs):
        kc = kv[ks:ks + ln]
        for u in range(ln):
            z_off[ks + u] = artifact_row(g, kc, q_all[ks + u][loc], u, blocks, loc)
    return z_off


# ----------------------------------------------------------------------------
# integer bookkeeping (segment visibility, partial index, protected flags)
# ----------------------------------------------------------------------------
def segment_chunks(segs: np.ndarray, split_keys: int):
    """For every segment s: the segments visible to rows of s (all segments
    whose request offset is <= p_s, in request order), cut into chunks.
    split_keys == 0: one chunk per segment.  split_keys > 0: greedy, a chunk is
    closed before a segment that would push its summed length past split_keys
    (a chunk always holds at least one segment).  Chunks are (first, last)
    segment indices into `segs`."""
    segs = np.asarray(segs, dtype=np.int64)
    order = np.argsort(segs[:, 2], kind="stable")
    out = []
    for s in range(segs.shape[0]):
        vis = [int(i) for i in order if segs[i, 2] <= segs[s, 2]]
        chunks = []
        if split_keys == 0:
            chunks = [(i, i) for i in vis]
        else:
            cur, keys = [], 0
            for i in vis:
                if cur and keys + segs[i, 1] > split_keys:
                    chunks.append((cur[0], cur[-1]))
                    cur, keys = [], 0
                cur.append(i)
                keys += int(segs[i, 1])
            chunks.append((cur[0], cur[-1]))
        out.append(chunks)
    return out


def enumerate_plan(segs, n_groups: int, heads_per_group: int, prot_rows, split_keys: int):
    """Output slots and their partials.

    Slots: Global slot (r, g) = r*G + g for every row r; Local slot (a, g, j) =
    N*G + (a*G + g)*(hpg-1) + j for protected row prot_rows[a] and the j-th
    Local head of group g.  Each slot gets one partial per chunk of its row's
    visible segments, in request order.  Returns row_src [N] u8 (1 = protected,
    recomputed online), part_ptr [n_slots+1] i64 (CSR offsets) and part_seg
    [n_parts, 2] i32 (first, last segment of each partial)."""
    segs = np.asarray(segs, dtype=np.int64)
    prot = np.asarray(prot_rows, dtype=np.int64)
    seg_of, _, _ = row_geometry(segs)
    n = seg_of.shape[0]
    chunks = segment_chunks(segs, split_keys)
    nch = np.array([len(c) for c in chunks], dtype=np.int64)
    flat = np.array([x for c in chunks for x in c], dtype=np.int32).reshape(-1, 2)
    choff = np.concatenate([[0], np.cumsum(nch)])
    hl = heads_per_group - 1
    slot_seg = np.concatenate([np.repeat(seg_of, n_groups), np.repeat(seg_of[prot], n_groups * hl)])
    counts = nch[slot_seg]
    part_ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    within = np.arange(part_ptr[-1]) - np.repeat(part_ptr[:-1], counts)
    part_seg = flat[np.repeat(choff[slot_seg], counts) + within]
    row_src = np.zeros(n, dtype=np.uint8)
    row_src[prot] = 1
    return row_src, part_ptr, part_seg


# ----------------------------------------------------------------------------
# protected token-row set (Sec. 2.3, eq:protected)
# ----------------------------------------------------------------------------
def total_order_key(scores) -> np.ndarray:
    """uint32 keys that sort float32 values by the IEEE-754 totalOrder predicate
    (-0 below +0): the sign-magnitude bit pattern mapped to an unsigned order."""
    u = np.ascontiguousarray(scores, dtype=np.float32).view(np.uint32)
    neg = (u >> np.uint32(31)) != 0
    return np.where(neg, ~u, u | np.uint32(0x80000000)).astype(np.uint32)


def protected_rows(segs, query_seg: int, row_flags, scores, edge: int = 128, tail: int = 32768,
                   budget: float = 0.10) -> np.ndarray:
    """A = Q u N u D u B_edge u I_top u T_tail (eq:protected), as sorted storage rows.

    Q: rows of the query segment.  N, D: rows flagged new (bit 0 of row_flags) or
    dirty (bit 1).  B_edge: the first and last `edge` rows of every relocated
    segment (a non-query segment whose request offset is not 0).  T_tail: rows
    whose true request position is among the last `tail` of the request.
    Candidates are the rows that have an artifact: neither query nor new rows.
    The controller's budget is a share of the candidates: I_top adds the
    highest-scoring candidates outside the other sets until
    round(budget * |candidates|) candidates are protected (nothing when the
    other sets already reach it).  Scores rank by IEEE-754 totalOrder,
    descending; equal scores go to the lower row.  Rounding is half up."""
    segs = np.asarray(segs, dtype=np.int64)
    seg, u, pos = row_geometry(segs)
    n = seg.shape[0]
    flags = np.asarray(row_flags, dtype=np.uint8)
    new = (flags & 1) != 0
    dirty = (flags & 2) != 0
    q = seg == int(query_seg)
    length = segs[seg, 1]
    relocated = (segs[seg, 2] != 0) & ~q
    edge_rows = relocated & ((u < edge) | (u >= length - edge))
    recent = pos >= n - tail
    base = q | new | dirty | edge_rows | recent
    cand = ~q & ~new
    target = int(np.floor(budget * int(cand.sum()) + 0.5))
    k = max(0, target - int((base & cand).sum()))
    elig = np.flatnonzero(cand & ~base)
    key = total_order_key(np.asarray(scores, dtype=np.float32)[elig])
    order = np.lexsort((elig, -key.astype(np.int64)))   # key descending, then row ascending
    sel = base.copy()
    sel[elig[order[:k]]] = True
    return np.flatnonzero(sel).astype(np.int32)



# ----------------------------------------------------------------------------
# adaptive MoE fanout (Sec. 2.4, eq:moe)
# ----------------------------------------------------------------------------
def moe_fanout(router, tau: float, top_k: int = 6, min_k: int = 3):
    """Per row of router weights p [N, E]: the top_k experts ranked by weight
    (IEEE-754 totalOrder, descending; equal weights go to the lower expert),
    their original weights, and the fanout
        K = min{k in [min_k, top_k] : sum_{j<=k} p_(j) / sum_{r<=top_k} p_(r) >= tau},
    or top_k when no k qualifies (eq:moe, with top_k = 6 and min_k = 3 in the
    paper).  float32 throughout, in rank order: S = p_(1) + ... + p_(top_k)
    summed left to right, p^_j = p_(j) / S, and the running sum of the p^_j is
    compared with float32(tau).  Returns (idx [N, top_k] int32, w [N, top_k]
    float32, K [N] int32)."""
    p = np.ascontiguousarray(router, dtype=np.float32)
    n, e = p.shape
    key = total_order_key(p).astype(np.int64)
    expert = np.broadcast_to(np.arange(e, dtype=np.int64), (n, e))
    order = np.lexsort((expert, -key), axis=-1)           # weight descending, then expert ascending
    idx = order[:, :top_k].astype(np.int32)
    w = np.take_along_axis(p, order[:, :top_k], axis=1)
    s = w[:, 0].copy()
    for j in range(1, top_k):
        s = (s + w[:, j]).astype(np.float32)
    cum = np.zeros(n, dtype=np.float32)
    k_out = np.full(n, top_k, dtype=np.int32)
    decided = np.zeros(n, dtype=bool)
    t = np.float32(tau)
    with np.errstate(invalid="ignore", divide="ignore"):
        for j in range(top_k):
            cum = (cum + (w[:, j] / s).astype(np.float32)).astype(np.float32)
            if j + 1 >= min_k:
                hit = ~decided & (cum >= t)
                k_out[hit] = j + 1
                decided |= hit
    return idx, w, k_out


# ----------------------------------------------------------------------------
# shared second projection (Sec. 2.1 eq:factorization, Alg. 2)
# ----------------------------------------------------------------------------
def shared_wb(z, w_b) -> np.ndarray:
    """y = W_b z for every row: y[r, o] = sum_i w_b[o, i] z[r, i], in fp64."""
    return np.asarray(z, dtype=F64) @ np.asarray(w_b, dtype=F64).T
