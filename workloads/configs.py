"""Seeded synthetic inputs for the MLA-Online step (structure and values only).

This module is shared by the fp64 oracle, the tests, the smoke check and the
benchmark.  It holds none of the method's arithmetic: it draws segment
layouts, protected-row sets, head roles and tensor values, and rounds values to
bfloat16.  Everything else (RoPE, attention, merge, projection) lives either in
the oracle or in the HIP library, never here.

Workloads stand in for the paper's 64K-440K-token RAG prompts (Sec. 4.1 and
4.3), which are built from public QA datasets and a model checkpoint that are
not available; the shapes follow the paper's geometry instead: the packed
512+64 latent row (Sec. 1 and 2.1), the 56/8 and 112/16 Local/Global head
profiles with one Global head per output group of eight (Sec. 3.1), and
multi-document prompts whose documents sit at relocated request offsets
(Sec. 2.3).

Random values are drawn per (tensor, chunk of rows) from
``numpy.random.PCG64(SeedSequence([seed, tensor_id, chunk]))`` so any subset of
rows can be regenerated without drawing the whole tensor; the oracle uses that
to sample rows of the 256K workload.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

# tensor ids for per-chunk seeding
_T_STRUCT, _T_KV, _T_QG, _T_QL, _T_WO, _T_ZOFF, _T_QFULL = 0, 1, 2, 3, 4, 5, 6
ROW_CHUNK = 2048          # rows per independently seeded chunk
BASE_SEED = 70080         # workload k uses seed BASE_SEED + k


# ----------------------------------------------------------------------------
# bfloat16 helpers (round-to-nearest-even), pure bit manipulation
# ----------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (RNE); returns the uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_bf16(x: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(f32_to_bf16_bits(x))


# ----------------------------------------------------------------------------
# geometry
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class Geometry:
    n_heads: int          # H logical query heads
    n_groups: int         # G native output groups, one Global head each
    d_latent: int         # d_c: latent width (also the value width)
    d_rope: int           # d_r: decoupled RoPE key width
    d_model: int          # width of the projected state z
    n_proj_groups: int    # 1 = dense first projection; G = group-sliced
    softmax_scale: float
    rope_base: float = 10000.0
    value_rope: bool = False  # the value is the whole latent row (its RoPE part rotary)

    @property
    def d_v(self) -> int:
        """Width of a head output: d_c, or d_c + d_r when the value carries the RoPE part."""
        return self.d_latent + (self.d_rope if self.value_rope else 0)

    @property
    def heads_per_group(self) -> int:
        return self.n_heads // self.n_groups

    @property
    def d_qk(self) -> int:
        return self.d_latent + self.d_rope

    @property
    def n_local(self) -> int:
        """Local heads per protected row (every head except the Global ones)."""
        return self.n_heads - self.n_groups


@dataclass
class Workload:
    name: str
    seed: int
    geom: Geometry
    segs: np.ndarray            # int64 [S, 3]: kv_start, length, req_offset (storage order)
    glob_head: np.ndarray       # int32 [G]: in-group index of each group's Global head
    prot_rows: np.ndarray       # int32 [P]: sorted storage rows of the protected set
    std: dict                   # value scales per tensor part
    fp32_source: bool = False   # inputs specified in fp32 (the tiny exactness case)
    random_zoff: bool = True    # False: the artifact must be computed offline
    query_rows: int = 0         # rows of the trailing request-query segment
    meta: dict = field(default_factory=dict)

    # ---------------- shapes ----------------
    @property
    def n_rows(self) -> int:
        return int(self.segs[:, 1].sum())

    @property
    def n_prot(self) -> int:
        return int(self.prot_rows.shape[0])

    # ---------------- chunked drawing ----------------
    def _rng(self, tensor: int, chunk: int) -> np.random.Generator:
        return np.random.Generator(np.random.PCG64(np.random.SeedSequence([self.seed, tensor, chunk])))

    def _draw_rows(self, tensor: int, n_total: int, parts, rows, bf16: bool, threads: int | None):
        """Draw rows of a tensor made of `parts` = [(shape_per_row, std), ...]
        concatenated on the last axis. Returns float32 values (bf16-rounded if bf16)."""
        if rows is None:
            rows = np.arange(n_total, dtype=np.int64)
        rows = np.asarray(rows, dtype=np.int64)
        chunks = np.unique(rows // ROW_CHUNK)
        per_row_shape = parts[0][0][:-1]
        width = sum(p[0][-1] for p in parts)

        def one(c):
            lo = int(c) * ROW_CHUNK
            hi = min(n_total, lo + ROW_CHUNK)
            n = hi - lo
            g = self._rng(tensor, int(c))
            pieces = []
            for shape, sd in parts:
                x = g.standard_normal((n,) + tuple(shape), dtype=np.float32)
                x *= np.float32(sd)
                pieces.append(x)
            x = np.concatenate(pieces, axis=-1) if len(pieces) > 1 else pieces[0]
            if bf16:
                x = round_bf16(x)
            return c, x

        if threads is None:
            threads = min(16, os.cpu_count() or 1)
        out = np.empty((rows.shape[0],) + tuple(per_row_shape) + (width,), dtype=np.float32)
        full = rows.shape[0] == n_total and np.array_equal(rows, np.arange(n_total))
        with ThreadPoolExecutor(max(1, threads)) as ex:
            for c, x in ex.map(one, chunks):
                lo = int(c) * ROW_CHUNK
                if full:
                    out[lo:lo + x.shape[0]] = x
                else:
                    sel = np.nonzero(rows // ROW_CHUNK == c)[0]
                    out[sel] = x[rows[sel] - lo]
        return out

    # ---------------- tensors (float32 values; bf16-exact unless exact=True) --------
    def kv(self, rows=None, exact=False, threads=None) -> np.ndarray:
        """Packed latent rows [n, d_c + d_r]: latent c_kv then the canonical-frame RoPE key."""
        g = self.geom
        parts = [((g.d_latent,), self.std["c"]), ((g.d_rope,), self.std["kr"])]
        return self._draw_rows(_T_KV, self.n_rows, parts, rows, not exact, threads)

    def q_full(self, rows=None, exact=False, threads=None) -> np.ndarray:
        """Absorbed queries of every head [n, H, d_c + d_r] (tiny case only: the
        offline artifact needs Local-head queries of unprotected rows too)."""
        g = self.geom
        parts = [((g.n_heads, g.d_latent), self.std["qc"]), ((g.n_heads, g.d_rope), self.std["qr"])]
        return self._draw_rows(_T_QFULL, self.n_rows, parts, rows, not exact, threads)

    def local_head_ids(self) -> np.ndarray:
        """[G, hpg-1] absolute head index of each Local head, ascending within a group."""
        g = self.geom
        hpg = g.heads_per_group
        out = np.empty((g.n_groups, hpg - 1), dtype=np.int64)
        for grp in range(g.n_groups):
            js = [j for j in range(hpg) if j != int(self.glob_head[grp])]
            out[grp] = [grp * hpg + j for j in js]
        return out

    def global_head_ids(self) -> np.ndarray:
        g = self.geom
        return np.arange(g.n_groups) * g.heads_per_group + self.glob_head.astype(np.int64)

    def q_glob(self, rows=None, exact=False, threads=None) -> np.ndarray:
        """Global-head queries [n, G, d_c + d_r] for storage rows `rows`."""
        g = self.geom
        if self.fp32_source:
            return self.q_full(rows, exact, threads)[:, self.global_head_ids(), :]
        parts = [((g.n_groups, g.d_latent), self.std["qc"]), ((g.n_groups, g.d_rope), self.std["qr"])]
        return self._draw_rows(_T_QG, self.n_rows, parts, rows, not exact, threads)

    def q_loc(self, idx=None, exact=False, threads=None) -> np.ndarray:
        """Local-head queries [n, G, hpg-1, d_c + d_r] for protected-row indices `idx`."""
        g = self.geom
        if idx is None:
            idx = np.arange(self.n_prot)
        idx = np.asarray(idx, dtype=np.int64)
        if self.fp32_source:
            q = self.q_full(self.prot_rows[idx], exact, threads)
            return q[:, self.local_head_ids(), :]
        hl = g.heads_per_group - 1
        parts = [((g.n_groups, hl, g.d_latent), self.std["qc"]),
                 ((g.n_groups, hl, g.d_rope), self.std["qr"])]
        return self._draw_rows(_T_QL, self.n_prot, parts, idx, not exact, threads)

    def w_o(self, exact=False) -> np.ndarray:
        """First output projection [n_pg, (H/n_pg)*d_v, d_model/n_pg]; block pg maps the
        head outputs of heads pg*H/n_pg .. to channels pg*d_model/n_pg .."""
        g = self.geom
        npg = g.n_proj_groups
        rows = (g.n_heads // npg) * g.d_v
        cols = g.d_model // npg
        x = self._rng(_T_WO, 0).standard_normal((npg, rows, cols), dtype=np.float32)
        x *= np.float32(self.std["wo"])
        return x if exact else round_bf16(x)

    def z_off(self, rows=None, threads=None) -> np.ndarray:
        """Random stand-in for the projected Local artifact [n, d_model] (bf16 values)."""
        if not self.random_zoff:
            raise ValueError("this workload's artifact is computed offline, not drawn")
        parts = [((self.geom.d_model,), self.std["zoff"])]
        return self._draw_rows(_T_ZOFF, self.n_rows, parts, rows, True, threads)

    # ---------------- structure helpers (no method arithmetic) ----------------
    def row_segment(self) -> np.ndarray:
        """Segment index of every storage row."""
        seg = np.empty(self.n_rows, dtype=np.int64)
        for i, (ks, ln, _) in enumerate(self.segs):
            seg[ks:ks + ln] = i
        return seg

    def row_position(self) -> np.ndarray:
        """True request position of every storage row."""
        pos = np.empty(self.n_rows, dtype=np.int64)
        for ks, ln, ro in self.segs:
            pos[ks:ks + ln] = ro + np.arange(ln)
        return pos


# ----------------------------------------------------------------------------
# structure draws
# ----------------------------------------------------------------------------
def _contiguous(lengths):
    segs = []
    off = 0
    for ln in lengths:
        segs.append((off, ln, off))
        off += ln
    return segs


def _uniform_protected(rng, n_doc_rows, frac):
    k = int(round(frac * n_doc_rows))
    return np.sort(rng.choice(n_doc_rows, size=k, replace=False)).astype(np.int64)


def _clustered_protected(rng, segs_doc, frac, run):
    """Runs of `run` consecutive rows inside one document; a run that overlaps an
    existing one is rejected and drawn again."""
    t_doc = sum(s[1] for s in segs_doc)
    n_runs = int(round(frac * t_doc / run))
    taken = np.zeros(t_doc, dtype=bool)
    runs = 0
    while runs < n_runs:
        d = int(rng.integers(0, len(segs_doc)))
        ks, ln, _ = segs_doc[d]
        st = int(rng.integers(0, ln - run + 1))
        if taken[ks + st:ks + st + run].any():
            continue
        taken[ks + st:ks + st + run] = True
        runs += 1
    return np.nonzero(taken)[0].astype(np.int64)


def _lengths_summing(rng, n, lo, hi, total):
    """n-1 lengths uniform in [lo, hi]; the last closes the sum and must also be in range."""
    while True:
        head = rng.integers(lo, hi + 1, size=n - 1)
        last = total - int(head.sum())
        if lo <= last <= hi:
            return [int(x) for x in head] + [last]


def _std_bf16_cfg(peaked: bool, d_c: int, d_r: int):
    if peaked:
        return dict(c=1.0, kr=1.0, qc=1.0, qr=1.0, wo=0.02, zoff=0.05)
    return dict(c=1 / math.sqrt(d_c), kr=1 / math.sqrt(d_r), qc=1 / math.sqrt(d_c),
                qr=1 / math.sqrt(d_r), wo=0.02, zoff=0.05)


def make_workload(cfg: int, variant: str = "default", seed: int | None = None,
                  n_proj_groups: int | None = None, value_rope: bool = False) -> Workload:
    """Build workload `cfg` (1..5).  variant: "default" or "peaked" (unscaled
    queries and keys, which make the softmax far from uniform).  value_rope:
    the value is the whole latent row (cfg 2..5; W_o then has d_c + d_r rows
    per head)."""
    if seed is None:
        seed = BASE_SEED + cfg + (1000 if variant == "peaked" else 0)
    peaked = variant == "peaked"
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, _T_STRUCT, 0])))

    if cfg == 1:
        H, G, d_c, d_r, d_model = 8, 1, 64, 16, 128
        doc = [128, 128]
        tq = 32
        segs = _contiguous(doc + [tq])
        prot_doc = _uniform_protected(rng, sum(doc), 8 / 256)
        std = dict(c=1.0, kr=1.0, qc=1 / math.sqrt(d_c), qr=1 / math.sqrt(d_r), wo=0.02, zoff=0.05)
        if peaked:
            std.update(qc=1.0, qr=1.0)
        geom = Geometry(H, G, d_c, d_r, d_model, n_proj_groups or 1, 1 / math.sqrt(d_c + d_r))
        fp32, rz = True, False
    elif cfg in (2, 4, 5):
        if cfg == 2:
            H, G, d_model, doc, tq, frac = 64, 8, 4096, [4096] * 8, 256, 0.02
        elif cfg == 4:
            H, G, d_model, doc, tq, frac = 128, 16, 7168, [2048] * 32, 2048, 0.03
        else:
            H, G, d_model, doc, tq, frac = 64, 8, 4096, [4096] * 64, 2048, 0.02
        d_c, d_r = 512, 64
        segs = _contiguous(doc + [tq])
        prot_doc = _uniform_protected(rng, sum(doc), frac)
        std = _std_bf16_cfg(peaked, d_c, d_r)
        geom = Geometry(H, G, d_c, d_r, d_model, n_proj_groups or G, 1 / math.sqrt(d_c + d_r))
        fp32, rz = False, True
    elif cfg == 3:
        H, G, d_model, d_c, d_r, tq = 64, 8, 4096, 512, 64, 1024
        lens = _lengths_summing(rng, 16, 1024, 3072, 32768)
        perm = rng.permutation(16)
        req = np.zeros(16, dtype=np.int64)
        acc = 0
        for d in perm:               # documents laid out in request order perm[0], perm[1], ...
            req[d] = acc
            acc += lens[d]
        segs = []
        ks = 0
        for d in range(16):          # storage order = document id
            segs.append((ks, lens[d], int(req[d])))
            ks += lens[d]
        segs.append((ks, tq, 32768))
        prot_doc = _clustered_protected(rng, segs[:16], 0.05, 16)
        std = _std_bf16_cfg(peaked, d_c, d_r)
        geom = Geometry(H, G, d_c, d_r, d_model, n_proj_groups or G, 1 / math.sqrt(d_c + d_r))
        fp32, rz = False, True
    else:
        raise ValueError(f"unknown workload {cfg}")

    if value_rope:
        if cfg == 1:
            raise ValueError("a rotary value is built for the 512+64 latent (workloads 2..5)")
        geom = Geometry(geom.n_heads, geom.n_groups, geom.d_latent, geom.d_rope, geom.d_model,
                        geom.n_proj_groups, geom.softmax_scale, geom.rope_base, value_rope=True)
    segs = np.asarray(segs, dtype=np.int64)
    n = int(segs[:, 1].sum())
    qrows = np.arange(n - tq, n, dtype=np.int64)
    prot = np.unique(np.concatenate([prot_doc, qrows])).astype(np.int32)
    hpg = H // G
    glob_head = rng.integers(0, hpg, size=G).astype(np.int32)
    names = {1: "tiny exactness case: 2x128 docs + 32 query rows, 8 heads in 1 group, 64+16 latent",
             2: "8x4096 docs + 256 query rows, 64 heads in 8 groups, 512+64 latent",
             3: "32K context: 16 uneven docs at permuted offsets + 1024 query rows, 64/8 heads",
             4: "64K context: 32x2048 docs + 2048 query rows, 128 heads in 16 groups",
             5: "256K context: 64x4096 docs + 2048 query rows, 64 heads in 8 groups, 512+64 latent"}
    return Workload(name=names[cfg] + (" (peaked)" if peaked else "") + (", rotary value" if value_rope else ""),
                    seed=seed, geom=geom,
                    segs=segs, glob_head=glob_head, prot_rows=prot, std=std, fp32_source=fp32,
                    random_zoff=rz, query_rows=tq, meta=dict(cfg=cfg, variant=variant))


def make_custom(doc_lens, req_perm=None, tq=8, H=4, G=2, d_c=64, d_r=16, d_model=32, n_pg=None,
                prot_frac=0.2, seed=1234, glob_head=None, fp32=True, std=None, prot_rows=None,
                value_rope=False):
    """Small workload family for exactness tests: arbitrary document lengths, optional
    request-order permutation, arbitrary head partition."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, _T_STRUCT, 1])))
    nd = len(doc_lens)
    order = list(range(nd)) if req_perm is None else list(req_perm)
    req = {}
    acc = 0
    for d in order:
        req[d] = acc
        acc += doc_lens[d]
    segs = []
    ks = 0
    for d in range(nd):
        segs.append((ks, doc_lens[d], req[d]))
        ks += doc_lens[d]
    if tq > 0:
        segs.append((ks, tq, acc))
    segs = np.asarray(segs, dtype=np.int64)
    n = int(segs[:, 1].sum())
    t_doc = int(sum(doc_lens))
    if prot_rows is None:
        k = int(round(prot_frac * t_doc))
        pd = rng.choice(t_doc, size=k, replace=False) if k > 0 else np.zeros(0, dtype=np.int64)
        prot_rows = np.unique(np.concatenate([pd, np.arange(t_doc, n)]))
    prot_rows = np.asarray(prot_rows, dtype=np.int32)
    hpg = H // G
    if glob_head is None:
        glob_head = rng.integers(0, hpg, size=G)
    if std is None:
        std = dict(c=1.0, kr=1.0, qc=1 / math.sqrt(d_c), qr=1 / math.sqrt(d_r), wo=0.02, zoff=0.05)
    geom = Geometry(H, G, d_c, d_r, d_model, n_pg or G, 1 / math.sqrt(d_c + d_r), value_rope=bool(value_rope))
    return Workload(name="custom", seed=seed, geom=geom, segs=segs,
                    glob_head=np.asarray(glob_head, dtype=np.int32), prot_rows=prot_rows, std=std,
                    fp32_source=fp32, random_zoff=True, query_rows=tq, meta=dict(cfg=0))
