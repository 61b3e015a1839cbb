"""Host-side checks of the C ABI (no GPU needed): the library loads and exports
every function the header declares, the size query agrees with the oracle's
enumeration, and every validation failure is reported before any device work."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import mla_oracle as M
from workloads import make_custom, make_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h"))


@pytest.fixture(scope="module")
def mla():
    from paper_2609_07008_amd import mla as m
    return m


def header_functions():
    """every function declared by the headers under include/"""
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names.update(re.findall(r"\b(mla_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def test_exports_every_declared_symbol(mla):
    declared = header_functions()
    assert "mla_online_attend" in declared and "mla_segment_merge" in declared
    assert "mla_sliced_oproj_add" in declared and "mla_probe_mfma_bf16" in declared
    for name in declared:
        assert hasattr(mla.LIB, name), name
    assert set(declared) == set(mla.EXPORTS)
    assert mla.version().startswith("mla_online")


def test_status_strings(mla):
    for code, name in mla.STATUS.items():
        assert mla.LIB.mla_status_str(code).decode().startswith(name)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("split", [0, 4096, 10 ** 9])
def test_size_query_matches_oracle(mla, cfg, split):
    wl = make_workload(cfg)
    g = wl.geom
    if cfg >= 4 and split == 0:
        # closed form instead of a full enumeration (70M partials at 256K)
        rank = np.argsort(np.argsort(wl.segs[:, 2]))
        seg, _, _ = M.row_geometry(wl.segs)
        n_parts = int((rank[seg] + 1).sum()) * g.n_groups + int((rank[seg[wl.prot_rows]] + 1).sum()) * g.n_local
        n_slots = wl.n_rows * g.n_groups + wl.n_prot * g.n_local
    else:
        _, ptr, _ = M.enumerate_plan(wl.segs, g.n_groups, g.heads_per_group, wl.prot_rows, split)
        n_slots, n_parts = ptr.shape[0] - 1, int(ptr[-1])
    s, p, ws = mla.attend_query(g, wl.segs, wl.prot_rows, split)
    assert (s, p) == (n_slots, n_parts)
    assert ws > 0 and ws % 256 == 0


def _tiny():
    return make_custom([5, 9], req_perm=[1, 0], tq=3, H=4, G=2, d_c=64, d_r=16, d_model=64, seed=3)


class _G:
    def __init__(self, **kw):
        self.__dict__.update(kw)


def _geom(wl, **over):
    g = wl.geom
    d = dict(n_heads=g.n_heads, n_groups=g.n_groups, d_latent=g.d_latent, d_rope=g.d_rope, d_model=g.d_model,
             n_proj_groups=g.n_proj_groups, softmax_scale=g.softmax_scale, rope_base=g.rope_base)
    d.update(over)
    return _G(**d)


@pytest.mark.parametrize("case,status", [
    ("heads_not_multiple", "MLA_ERR_SHAPE"),
    ("dims_unsupported", "MLA_ERR_UNSUPPORTED"),
    ("bad_scale", "MLA_ERR_SHAPE"),
    ("gap_in_storage", "MLA_ERR_SEGMENTS"),
    ("overlap_in_request", "MLA_ERR_SEGMENTS"),
    ("zero_length", "MLA_ERR_SEGMENTS"),
    ("no_segments", "MLA_ERR_SEGMENTS"),
    ("unsorted_prot", "MLA_ERR_ROWS"),
    ("duplicate_prot", "MLA_ERR_ROWS"),
    ("prot_out_of_range", "MLA_ERR_ROWS"),
    ("negative_split", "MLA_ERR_SHAPE"),
    ("huge_length", "MLA_ERR_UNSUPPORTED"),
])
def test_size_query_rejects(mla, case, status):
    wl = _tiny()
    geom, segs, prot, split = _geom(wl), wl.segs.copy(), np.asarray(wl.prot_rows).copy(), 0
    if case == "heads_not_multiple":
        geom = _geom(wl, n_heads=5)
    elif case == "dims_unsupported":
        geom = _geom(wl, d_latent=128, d_rope=32)
    elif case == "bad_scale":
        geom = _geom(wl, softmax_scale=float("nan"))
    elif case == "gap_in_storage":
        segs[1, 0] += 1
    elif case == "overlap_in_request":
        segs[0, 2] = segs[1, 2]
    elif case == "zero_length":
        segs[0, 1] = 0
    elif case == "no_segments":
        segs = segs[:0]
    elif case == "unsorted_prot":
        prot = prot[::-1].copy()
    elif case == "duplicate_prot":
        prot = np.concatenate([prot[:1], prot])
    elif case == "prot_out_of_range":
        prot = np.concatenate([prot, [wl.n_rows]])
    elif case == "negative_split":
        split = -1
    elif case == "huge_length":                    # the row total would overflow int64 before any tiling check
        segs[1, 1] = np.iinfo(np.int64).max
    with pytest.raises(mla.MlaError) as ei:
        mla.attend_query(geom, segs, prot, split)
    assert mla.STATUS[ei.value.status] == status, ei.value


def test_attend_rejects_before_device_work(mla):
    """Validation failures of mla_online_attend need no GPU: they return before
    any HIP call (here: NULL device pointers, misaligned pointers, short workspace)."""
    wl = _tiny()
    g = mla.make_geom(wl.geom)
    sarr, ns = mla.make_segments(wl.segs)
    prot = np.ascontiguousarray(wl.prot_rows, dtype=np.int32)
    P = ctypes.c_void_p
    _, _, ws = mla.attend_query(wl.geom, wl.segs, prot, 0)

    def call(kv, qg, ql, po, pl, pp, wsp, wsb):
        return mla.LIB.mla_online_attend(ctypes.byref(g), sarr, ns, prot.ctypes.data_as(P), len(prot), 0,
                                         P(kv), P(qg), P(ql), P(po), P(pl), P(pp), None, None, P(wsp), wsb, None)
    ok = 1 << 20
    assert call(0, ok, ok, ok, ok, ok, ok, ws) == 1          # MLA_ERR_NULL
    assert call(ok, ok, 0, ok, ok, ok, ok, ws) == 1          # q_loc missing with Local heads
    assert call(ok + 8, ok, ok, ok, ok, ok, ok, ws) == 2     # misaligned kv
    assert call(ok, ok, ok, ok, ok, ok, ok + 16, ws) == 2    # workspace not 256-byte aligned
    assert call(ok, ok, ok, ok, ok, ok, ok, ws - 256) == 6   # MLA_ERR_WORKSPACE
    assert "workspace" in mla.LIB.mla_last_error_detail().decode()


def test_merge_and_oproj_reject(mla):
    P = ctypes.c_void_p
    assert mla.LIB.mla_segment_merge(4, 128, P(1 << 20), P(1 << 20), P(1 << 20), 0, P(1 << 20), None, None) == 3
    assert mla.LIB.mla_segment_merge(4, 512, None, P(1 << 20), P(1 << 20), 0, P(1 << 20), None, None) == 1
    assert mla.LIB.mla_segment_merge(4, 512, P(1 << 20), P(1 << 20), P(1 << 20), 7, P(1 << 20), None, None) == 2
    assert mla.LIB.mla_segment_merge(0, 512, None, None, None, 0, None, None, None) == 0   # nothing to do
    wl = _tiny()
    gh = np.asarray(wl.glob_head, dtype=np.int32)
    g = mla.make_geom(wl.geom)
    a = P(1 << 20)

    def call(geom, n_rows, gh_arr, n_prot, zoff):
        return mla.LIB.mla_sliced_oproj_add(ctypes.byref(geom), n_rows, a, a, gh_arr.ctypes.data_as(P), a, n_prot,
                                            a, zoff, a, None)
    assert call(g, 0, gh, 0, a) == 2                                      # no rows
    assert call(g, wl.n_rows, gh, wl.n_rows + 1, a) == 5                  # more protected rows than rows
    bad = gh.copy()
    bad[0] = wl.geom.heads_per_group
    assert call(g, wl.n_rows, bad, 2, a) == 2                             # Global head outside its group
    assert call(g, wl.n_rows, gh, 2, None) == 1                           # z_off needed
    g2 = mla.make_geom(_geom(wl, d_model=40, n_proj_groups=2))
    assert call(g2, wl.n_rows, gh, 2, a) == 3                             # 20 channels per group
    assert call(g, wl.n_rows, gh, 2, P((1 << 20) + 8)) == 2               # z_off misaligned (8-byte reads)
    assert mla.LIB.mla_sliced_oproj_add(ctypes.byref(g), wl.n_rows, a, a, gh.ctypes.data_as(P), a, 2, a, a,
                                        P((1 << 20) + 4), None) == 2      # z misaligned (16-byte writes)
    g3 = mla.make_geom(_geom(wl, d_model=1 << 26))
    assert call(g3, 2**31 - 1, gh, 2, a) == 3                             # tile count beyond one launch


def test_offline_produce_rejects(mla):
    """mla_offline_produce validates everything before its first HIP call."""
    wl = _tiny()
    g = mla.make_geom(wl.geom)
    sarr, ns = mla.make_segments(wl.segs)
    P = ctypes.c_void_p
    ws = mla.offline_produce_query(wl.geom, wl.segs)
    hl = wl.geom.heads_per_group - 1
    assert ws >= wl.n_rows * wl.geom.n_groups * hl * wl.geom.d_latent * 2   # holds the bf16 head outputs
    gh = np.asarray(wl.glob_head, dtype=np.int32)
    ok = 1 << 20

    def call(kv, q, gh_arr, w, dt, z, wsp, wsb):
        return mla.LIB.mla_offline_produce(ctypes.byref(g), sarr, ns, P(kv), P(q), gh_arr.ctypes.data_as(P), P(w),
                                           dt, P(z), P(wsp), wsb, None)
    assert call(ok, ok, gh, ok, 7, ok, ok, ws) == 2                 # out_dtype
    bad = gh.copy()
    bad[0] = wl.geom.heads_per_group
    assert call(ok, ok, bad, ok, 0, ok, ok, ws) == 2                # Global head outside its group
    assert call(ok, ok, gh, ok, 0, 0, ok, ws) == 1                  # z_off missing
    assert call(ok, ok, gh, ok, 0, ok + 8, ok, ws) == 2             # z_off misaligned
    assert call(ok, ok, gh, ok, 0, ok, ok + 16, ws) == 2            # workspace not 256-byte aligned
    assert call(ok, ok, gh, ok, 0, ok, ok, ws - 256) == 6           # workspace too small
    assert call(0, ok, gh, ok, 0, ok, ok, ws) == 1                  # kv missing


def test_protected_rows_rejects(mla):
    """mla_protected_rows validates its configuration before any HIP call, and its
    workspace holds one 8-byte key and one flag byte per row."""
    wl = _tiny()
    sarr, ns = mla.make_segments(wl.segs)
    P = ctypes.c_void_p
    ws = mla.protected_rows_query(wl.segs)
    assert ws >= 9 * wl.n_rows
    ok = 1 << 20

    def call(q, edge, tail, budget, out, wsp, wsb, cfg_null=False):
        cfg = mla.ProtectCfg(q, edge, tail, budget)
        return mla.LIB.mla_protected_rows(sarr, ns, None if cfg_null else ctypes.byref(cfg), None, None, P(out),
                                          P(out), P(wsp), wsb, None)
    nseg = int(np.asarray(wl.segs).shape[0])
    assert call(0, 4, 8, 0.1, ok, ok, ws, cfg_null=True) == 1
    assert call(nseg, 4, 8, 0.1, ok, ok, ws) == 2                   # query segment out of range
    assert call(-2, 4, 8, 0.1, ok, ok, ws) == 2
    assert call(0, -1, 8, 0.1, ok, ok, ws) == 2                     # negative edge
    assert call(0, 4, -8, 0.1, ok, ok, ws) == 2                     # negative tail
    assert call(0, 4, 8, 1.5, ok, ok, ws) == 2                      # budget above 1
    assert call(0, 4, 8, float("nan"), ok, ok, ws) == 2             # budget NaN
    assert call(0, 4, 8, 0.1, 0, ok, ws) == 1                       # outputs missing
    assert call(0, 4, 8, 0.1, ok, ok + 16, ws) == 2                 # workspace not 256-byte aligned
    assert call(0, 4, 8, 0.1, ok, ok, ws - 256) == 6                # workspace too small
    bad = np.asarray(wl.segs, dtype=np.int64).copy()
    bad[0, 1] += 1                                                  # no longer tiles the rows
    sb, nb = mla.make_segments(bad)
    cfg = mla.ProtectCfg(0, 4, 8, 0.1)
    assert mla.LIB.mla_protected_rows(sb, nb, ctypes.byref(cfg), None, None, P(ok), P(ok), P(ok), ws, None) == 4


def test_moe_fanout_rejects():
    from paper_2609_07008_amd import mla
    L = mla.LIB
    P = ctypes.c_void_p
    fake = P(4096)

    def call(n=4, e=16, router=fake, top_k=6, min_k=3, tau=0.9, idx=fake, w=fake, k=fake, cnt=None):
        return L.mla_moe_fanout(n, e, router, top_k, min_k, tau, idx, w, k, cnt, None)

    assert call(n=-1) == 2
    assert call(top_k=0) == 3 and call(top_k=9) == 3
    assert call(min_k=0) == 2 and call(min_k=7) == 2
    assert call(e=5) == 2
    assert call(e=1025) == 3
    assert call(tau=float("nan")) == 2
    assert call(router=None) == 1 and call(idx=None) == 1 and call(w=None) == 1 and call(k=None) == 1
    assert call(w=P(4098)) == 2
    assert call(n=2**62, e=16) == 2


def test_shared_wb_rejects():
    from paper_2609_07008_amd import mla
    L = mla.LIB
    P = ctypes.c_void_p
    fake = P(4096)

    def call(n=4, d_in=64, d_out=16, z=fake, w=fake, out=1, y=fake):
        return L.mla_shared_wb(n, d_in, d_out, z, w, out, y, None)

    assert call(n=-1) == 2
    assert call(d_in=0) == 2 and call(d_in=96) == 2 and call(d_in=32) == 2
    assert call(d_in=16448) == 3
    assert call(d_out=0) == 2
    assert call(out=5) == 2
    assert call(z=None) == 1 and call(w=None) == 1 and call(y=None) == 1
    assert call(z=P(4104)) == 2
    assert call(n=0, z=None) == 0
    assert call(n=2**62, d_out=4096) == 3 and call(n=2**63 - 1, d_out=2**31 - 1) == 3   # tile count, no overflow


def test_value_rope_geometry_checks():
    from paper_2609_07008_amd import mla
    segs = np.array([[0, 10, 0]], dtype=np.int64)

    class G:
        n_heads, n_groups, d_latent, d_rope, d_model, n_proj_groups = 8, 2, 64, 16, 64, 2
        softmax_scale, rope_base, value_rope = 0.1, 10000.0, True

    with pytest.raises(mla.MlaError) as e:
        mla.offline_produce_query(G, segs)
    assert e.value.status == 3                         # rotary value: built for (512, 64) only
    G.d_latent, G.d_rope = 512, 64
    big = mla.offline_produce_query(G, segs)
    G.value_rope = False
    small = mla.offline_produce_query(G, segs)
    assert big > small                                 # 576-wide head outputs and their lse
    g = mla.make_geom(G)
    g.value_rope = 2
    ws = ctypes.c_size_t()
    sarr, ns = mla.make_segments(segs)
    assert mla.LIB.mla_offline_produce_query(ctypes.byref(g), sarr, ns, ctypes.byref(ws)) == 2


# ----------------------------------------------------------------------------
# plan-once path: sizes and bounds on the host, and the checks made before any
# device work (no GPU call is reached by these cases)
# ----------------------------------------------------------------------------
def _local_items(wl, split, prot):
    """Work items the device plan lays out for the Local heads of protected set
    `prot`: per segment and chunk, ceil(|A in segment| * L_h / 128)."""
    g = wl.geom
    lh = g.n_groups * (g.heads_per_group - 1)
    if lh == 0:
        return 0
    chunks = M.segment_chunks(wl.segs, split)
    seg, _, _ = M.row_geometry(wl.segs)
    cnt = np.bincount(seg[np.asarray(prot, dtype=np.int64)], minlength=len(wl.segs))
    return sum(len(chunks[s]) * -(-int(cnt[s]) * lh // 128) for s in range(len(wl.segs)))


@pytest.mark.parametrize("cfg", [1, 2, 3, 5])
@pytest.mark.parametrize("split", [0, 4096, 10 ** 9])
def test_plan_bounds_cover_every_protected_set(mla, cfg, split):
    wl = make_workload(cfg)
    g = wl.geom
    if cfg == 5 and split == 0:
        pytest.skip("70M per-segment partials at 256K: covered by the closed form of the size query")
    split = min(split, wl.n_rows)
    rng = np.random.default_rng(cfg)
    lh = g.n_groups * (g.heads_per_group - 1)
    for cap in sorted({wl.n_prot, wl.n_rows, max(1, wl.n_prot // 3)}):
        info = mla.plan_query(g, wl.segs, split, cap)
        assert info.max_slots == wl.n_rows * g.n_groups + cap * lh
        assert info.prot_cap == cap and info.n_rows == wl.n_rows and info.split_keys == split
        assert info.plan_bytes % 256 == 0 and info.ws_bytes % 256 == 0
        assert info.one_chunk == int(split >= wl.n_rows or len(wl.segs) == 1)
        glob_items = sum(len(c) * -(-int(ln) * g.n_groups // 128)
                         for c, (_, ln, _) in zip(M.segment_chunks(wl.segs, split), wl.segs))
        # protected sets of `cap` rows: the workload's own (when it fits), the rows
        # of the segments with the most chunks, and random ones
        sets = [np.sort(rng.choice(wl.n_rows, size=cap, replace=False)) for _ in range(3)]
        if wl.n_prot <= cap:
            sets.append(np.asarray(wl.prot_rows))
        seg, _, _ = M.row_geometry(wl.segs)
        nch = np.array([len(c) for c in M.segment_chunks(wl.segs, split)])
        sets.append(np.sort(np.argsort(-nch[seg], kind="stable")[:cap]))
        for prot in sets:
            assert glob_items + _local_items(wl, split, prot) <= info.max_items
            if cfg <= 3:
                _, ptr, _ = M.enumerate_plan(wl.segs, g.n_groups, g.heads_per_group, prot, split)
                assert int(ptr[-1]) <= info.max_parts


def test_plan_query_rejects(mla):
    wl = _tiny()
    for cap in (-1, wl.n_rows + 1):
        with pytest.raises(mla.MlaError) as e:
            mla.plan_query(wl.geom, wl.segs, 0, cap)
        assert e.value.status == 2
    with pytest.raises(mla.MlaError) as e:
        mla.plan_query(_geom(wl, d_latent=128, d_rope=32), wl.segs, 0, 1)
    assert e.value.status == 3
    segs = wl.segs.copy()
    segs[1, 0] += 1
    with pytest.raises(mla.MlaError) as e:
        mla.plan_query(wl.geom, segs, 0, 1)
    assert e.value.status == 4


def test_planned_calls_check_the_plan_first(mla):
    """A changed plan description or another geometry is refused on the host,
    before any pointer is used (the device pointers here are all NULL)."""
    import ctypes
    wl = _tiny()
    info = mla.plan_query(wl.geom, wl.segs, 0, wl.n_prot)
    g = mla.make_geom(wl.geom)

    def attend(gm, inf):
        return mla.LIB.mla_online_attend_planned(ctypes.byref(gm), ctypes.byref(inf), None, None, None, None, None,
                                                 None, 0, None, None, None, None, None, None, None, 0, None)

    def oproj(gm, inf):
        gh = np.zeros(wl.geom.n_groups, dtype=np.int32)
        return mla.LIB.mla_sliced_oproj_add_planned(ctypes.byref(gm), ctypes.byref(inf), None, None,
                                                    gh.ctypes.data_as(ctypes.c_void_p), None, None, None, None, 1,
                                                    None, None)

    assert attend(g, info) == 1 and oproj(g, info) == 1          # intact: fails later, on a NULL pointer
    bad = mla.PlanInfo.from_buffer_copy(info)
    bad.max_items += 1
    assert attend(g, bad) == 2 and oproj(g, bad) == 2
    assert "mla_online_plan" in mla.LIB.mla_last_error_detail().decode()
    other = mla.make_geom(_geom(wl, softmax_scale=0.5))
    assert attend(other, info) == 2 and oproj(other, info) == 2
    assert "geometry" in mla.LIB.mla_last_error_detail().decode()


def test_noalloc_refuses_a_plan_larger_than_its_scratch(mla):
    """Checked on the host before the scratch array is looked up: the device
    pointers below are aligned placeholders that are never dereferenced."""
    import ctypes
    wl = make_workload(2)
    info = mla.plan_query(wl.geom, wl.segs, 0, wl.n_prot)      # per-segment partials: GBs of workspace
    assert info.ws_bytes > mla.NOALLOC_SCRATCH_BYTES
    g = mla.make_geom(wl.geom)
    fake = ctypes.c_void_p(1 << 20)
    st = mla.LIB.mla_online_attend_planned_noalloc(ctypes.byref(g), ctypes.byref(info), fake, fake, fake, fake, fake,
                                                   fake, 0, fake, None, None, None, None, None, None)
    assert st == 6 and "scratch" in mla.LIB.mla_last_error_detail().decode()


def test_probe_validates_before_any_device_work(mla):
    flop = ctypes.c_double(0.0)
    sink = ctypes.c_void_p(256)   # never dereferenced: every call below fails validation first
    assert mla.LIB.mla_probe_mfma_bf16(0, ctypes.byref(flop), sink, None) == 2
    assert mla.LIB.mla_probe_mfma_bf16((1 << 24) + 1, ctypes.byref(flop), sink, None) == 2
    assert mla.LIB.mla_probe_mfma_bf16(10, None, sink, None) == 1
    assert mla.LIB.mla_probe_mfma_bf16(10, ctypes.byref(flop), None, None) == 1
    assert flop.value == 0.0
