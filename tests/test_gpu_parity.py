"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Tolerances (bf16 inputs, fp32 accumulation): on each of O, lse, z_online and z,
max abs error <= 2e-2 and max abs error / max |reference| <= 1e-2.  Integer
bookkeeping (row_src, part_ptr, part_seg) must be bit-exact.
"""
import numpy as np
import pytest

from oracle import mla_oracle as M
from workloads import make_custom, make_workload, round_bf16

from parity import (artifact_bf16, boundary_sample, check, check_bookkeeping, compare_rows, run,
                    segment_edge_sample)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2609_07008_amd import mla  # noqa: F401  (fails loudly if the library is missing)
    yield


# ----------------------------------------------------------------------------
# tiny exactness workload: every row, every head, three split modes
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("variant", ["default", "peaked"])
@pytest.mark.parametrize("split", [0, 128, 10 ** 9])
def test_tiny_workload(variant, split):
    wl = make_workload(1, variant)
    z_off = artifact_bf16(wl)
    st, _ = run(wl, split, z_off=z_off)
    check_bookkeeping(wl, st, split)
    compare_rows(wl, st, np.arange(wl.n_rows), z_off)


# ----------------------------------------------------------------------------
# 512+64 latent on small custom requests: ragged segments, permuted offsets
# ----------------------------------------------------------------------------
CUSTOM = {
    "ragged": dict(doc_lens=[1, 2, 63, 64, 65, 130, 7], req_perm=[4, 0, 6, 2, 5, 1, 3], tq=37, H=16, G=2,
                   d_model=256, prot_frac=0.1),
    "dense_proj": dict(doc_lens=[70, 33, 128], req_perm=[2, 0, 1], tq=20, H=16, G=2, d_model=256, n_pg=1,
                       prot_frac=0.15),
    "wide_groups": dict(doc_lens=[96, 40], req_perm=[1, 0], tq=9, H=32, G=4, d_model=512, prot_frac=0.2),
    "single_segment": dict(doc_lens=[200], req_perm=None, tq=0, H=8, G=1, d_model=128, prot_frac=0.3),
}


@pytest.mark.parametrize("name", sorted(CUSTOM))
@pytest.mark.parametrize("split", [0, 100, 10 ** 9])
@pytest.mark.parametrize("peaked", [False, True])
def test_custom_512(name, split, peaked):
    kw = dict(CUSTOM[name])
    std = None
    if peaked:
        std = dict(c=1.0, kr=1.0, qc=1.0, qr=1.0, wo=0.02, zoff=0.05)
    wl = make_custom(d_c=512, d_r=64, seed=100 + sorted(CUSTOM).index(name), fp32=False, std=std, **kw)
    st, _ = run(wl, split)
    check_bookkeeping(wl, st, split)
    z_off = wl.z_off()
    compare_rows(wl, st, np.arange(wl.n_rows), z_off)


@pytest.mark.parametrize("case", ["no_protected", "all_protected", "all_global", "one_row", "one_row_unprotected",
                                  "one_row_and_query"])
def test_edge_cases(case):
    kw = dict(doc_lens=[65, 3, 64], req_perm=[1, 2, 0], tq=5, d_c=512, d_r=64, fp32=False, seed=21)
    one = dict(doc_lens=[1], req_perm=None, d_c=512, d_r=64, fp32=False, seed=23, H=16, G=2, d_model=256)
    if case == "one_row":                        # a one-row request: one key, every head
        wl = make_custom(tq=0, prot_rows=np.array([0]), **one)
    elif case == "one_row_unprotected":          # Global heads only, the artifact added
        wl = make_custom(tq=0, prot_rows=np.zeros(0, dtype=np.int32), **one)
    elif case == "one_row_and_query":            # a one-row document and a one-row query block
        wl = make_custom(tq=1, **one)
    elif case == "no_protected":
        wl = make_custom(H=16, G=2, d_model=256, prot_rows=np.zeros(0, dtype=np.int32), **kw)
    elif case == "all_protected":
        wl = make_custom(H=16, G=2, d_model=256, prot_rows=np.arange(137), **kw)
    else:
        wl = make_custom(H=4, G=4, d_model=128, prot_frac=0.2, **kw)   # one head per group: no Local heads
    z_off = wl.z_off()
    if case == "all_protected":
        z_off = np.full_like(z_off, np.nan)        # replaced everywhere: must never be read
    st, _ = run(wl, 0, z_off=z_off)
    check_bookkeeping(wl, st, 0)
    compare_rows(wl, st, np.arange(wl.n_rows), z_off)


# ----------------------------------------------------------------------------
# relocation and visibility: planted needles
# ----------------------------------------------------------------------------
def _needle_workload(seed=31):
    wl = make_custom([70, 90, 66], req_perm=[2, 0, 1], tq=12, H=16, G=2, d_c=512, d_r=64, d_model=256,
                     fp32=False, seed=seed, prot_frac=0.1)
    return wl


def _plant(wl, kv, row, head_g, seg_idx, u, logit, value=3.0):
    """Make key u of segment seg_idx score `logit` (natural units) above zero
    for Global head head_g of `row`, through the RoPE part only, and give it a
    distinctive latent (`value` in latent dim 0, zero elsewhere)."""
    g = wl.geom
    _, _, pos = M.row_geometry(wl.segs)
    q = wl.q_glob(rows=[row])[0, head_g]
    ks, ln, ps = wl.segs[seg_idx]
    qr = q[g.d_latent:].astype(np.float64)
    j = int(ks + u)
    kv = kv.copy()
    kv[j, : g.d_latent] = 0.0
    kv[j, 0] = value
    kv[j, g.d_latent:] = logit / g.softmax_scale * M.rope(qr, int(pos[row]) - int(ps), g.rope_base) / (qr @ qr)
    return round_bf16(kv.astype(np.float32)), j


def _run_with_kv(wl, kv_vals):
    import torch
    from paper_2609_07008_amd import device_inputs, step
    inputs = device_inputs.upload(wl)
    inputs["kv"] = device_inputs.to_bf16(kv_vals)
    st = step.OnlineStep(wl.geom, wl.segs, wl.prot_rows, wl.glob_head, 0)
    st.run(inputs["kv"], inputs["q_glob"], inputs["q_loc"], inputs["w_o"], inputs["z_off"])
    torch.cuda.synchronize()
    return st


@pytest.mark.parametrize("logit,restart,value", [(25.0, False, 3.0), (50.0, True, 3.0),
                                                 (100.0, True, 1.0), (200.0, True, 1.0)])
def test_needle_relocation(logit, restart, value):
    """A key planted in an earlier, relocated document dominates the row that
    sees it.  At +50 nats the needle's weight against the first tile's softmax
    reference passes 2^64 (44.4 nats), which exercises the kernel's restart
    path; at +100 and +200 nats it overflows float32 (88.7 nats), so the
    restarted reference must itself be raised again.  The overflow cases plant a
    latent of 1.0, keeping the outputs in the range the absolute tolerance is
    set for (bf16 outputs near 3 are 0.0156 apart)."""
    wl = _needle_workload()
    g = wl.geom
    row = wl.n_rows - 1
    seg_idx = int(np.argsort(wl.segs[:, 2])[1])        # second document in request order
    kv, j = _plant(wl, wl.kv(), row, 0, seg_idx, 41, logit, value)
    st = _run_with_kv(wl, kv)
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    # scores of the target head without the needle: the restart condition holds iff
    # the needle exceeds every other score (hence the first tile's max) by > 64 log2 units
    _, _, pos = M.row_geometry(wl.segs)
    q = wl.q_glob(rows=[row])[0, 0].astype(np.float64)
    t = int(pos[row])
    qt = np.concatenate([q[:g.d_latent], M.rope(q[g.d_latent:], t, g.rope_base)])
    sc = g.softmax_scale * (keys.k[: t + 1] @ qt)
    needle = int(np.argmax(sc))
    others = np.delete(sc, needle).max()
    assert (sc[needle] - others > 64 * np.log(2.0)) == restart
    o = st.out_o.float()[row * g.n_groups].cpu().numpy()
    assert abs(o[0] - value) < 0.05 and np.abs(o[1:]).max() < 0.05
    # the needle's score is planted through the RoPE part, parallel to the
    # relocated query, which the kernel rounds to bf16 (relative error 2^-9 per
    # element): the score, and the lse it dominates, may be off by up to
    # logit * 2^-9, more than 2e-2 once the logit passes 10
    lse_tol = max(2e-2, logit * 2.0 ** -9)
    compare_rows(wl, st, [row, row - 1, 0, int(wl.segs[seg_idx, 0]) + 41], wl.z_off(), kv=kv, keys=keys,
                 lse_abs_tol=lse_tol)


@pytest.mark.parametrize("logit,restart", [(25.0, False), (50.0, True)])
def test_needle_relocation_256k(logit, restart):
    """The same needle at the 256K geometry, in the benchmark's launch (one
    partial per slot): the last query row sees a key of the second document in
    request order, relocated by about 2.6e5 positions, so the query's RoPE part
    turns through the largest angles the workload has.  The lse bound for the
    planted score is the one derived in test_needle_relocation."""
    import torch
    from paper_2609_07008_amd import device_inputs, step
    wl = make_workload(5)
    g = wl.geom
    row = wl.n_rows - 1
    seg_idx = int(np.argsort(wl.segs[:, 2])[1])
    kv, j = _plant(wl, wl.kv(), row, 3, seg_idx, 3000, logit, 1.0)
    _, _, pos = M.row_geometry(wl.segs)
    assert int(pos[row]) - int(wl.segs[seg_idx, 2]) > 250000
    inputs = device_inputs.upload(wl)
    inputs["kv"] = device_inputs.to_bf16(kv)
    st = step.OnlineStep(g, wl.segs, wl.prot_rows, wl.glob_head, wl.n_rows, with_part_seg=False)
    st.run(inputs["kv"], inputs["q_glob"], inputs["q_loc"], inputs["w_o"], inputs["z_off"])
    torch.cuda.synchronize()
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    q = wl.q_glob(rows=[row])[0, 3].astype(np.float64)
    t = int(pos[row])
    qt = np.concatenate([q[:g.d_latent], M.rope(q[g.d_latent:], t, g.rope_base)])
    sc = g.softmax_scale * (keys.k[: t + 1] @ qt)
    pj = int(pos[j])                       # keys.k is in request order
    assert int(np.argmax(sc)) == pj
    assert (sc[pj] - np.delete(sc, pj).max() > 64 * np.log(2.0)) == restart
    o = st.out_o.float()[row * g.n_groups + 3].cpu().numpy()
    assert abs(o[0] - 1.0) < 0.05 and np.abs(o[1:]).max() < 0.05
    compare_rows(wl, st, [row, row - 1, j], None, kv=kv, keys=keys, lse_abs_tol=max(2e-2, logit * 2.0 ** -9))


def test_needle_in_the_future_is_invisible():
    """The needle sits one request position after `row`: `row` cannot see it,
    the next row (for whose query it is aimed) is dominated by it."""
    wl = _needle_workload()
    g = wl.geom
    s_last = int(np.argsort(wl.segs[:, 2])[2])
    ks, ln, ps = wl.segs[s_last]
    row = int(ks + 10)
    kv, j = _plant(wl, wl.kv(), row + 1, 0, s_last, 11, 25.0)
    st_a = _run_with_kv(wl, wl.kv())
    st_b = _run_with_kv(wl, kv)
    a = st_a.out_o.float()[row * g.n_groups: (row + 1) * g.n_groups].cpu().numpy()
    b = st_b.out_o.float()[row * g.n_groups: (row + 1) * g.n_groups].cpu().numpy()
    assert np.array_equal(a, b)
    c = st_b.out_o.float()[(row + 1) * g.n_groups].cpu().numpy()
    assert abs(c[0] - 3.0) < 0.05 and np.abs(c[1:]).max() < 0.05


# ----------------------------------------------------------------------------
# merge and o-proj entry points on their own
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("d_c", [64, 512, 576])
@pytest.mark.parametrize("out_f32", [True, False])
@pytest.mark.parametrize("max_parts", [8, 400])
def test_segment_merge(d_c, out_f32, max_parts):
    """1..max_parts partials per slot (400: more than a query row of the 256K
    workload has segments), lse spread over +-60 nats."""
    import torch
    from paper_2609_07008_amd import mla
    rng = np.random.default_rng(5 + max_parts)
    counts = rng.integers(1, max_parts + 1, size=1001 if max_parts <= 8 else 97)
    ptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    n_parts = int(ptr[-1])
    po = rng.standard_normal((n_parts, d_c)).astype(np.float32)
    pl = (rng.standard_normal(n_parts) * 20).astype(np.float32)
    out = torch.empty((len(counts), d_c), dtype=torch.float32 if out_f32 else torch.bfloat16, device="cuda")
    lse = torch.empty((len(counts),), dtype=torch.float32, device="cuda")
    mla.segment_merge(len(counts), d_c, torch.from_numpy(po).cuda(), torch.from_numpy(pl).cuda(),
                      torch.from_numpy(ptr).cuda(), mla.MLA_F32 if out_f32 else mla.MLA_BF16, out, lse)
    torch.cuda.synchronize()
    ref_o = np.zeros((len(counts), d_c))
    ref_l = np.zeros(len(counts))
    for s in range(len(counts)):
        ref_o[s], ref_l[s] = M.lse_merge(po[ptr[s]:ptr[s + 1]], pl[ptr[s]:ptr[s + 1]])
    got = out.float().cpu().numpy()
    check("merged O", got, ref_o, abs_tol=2e-2 if not out_f32 else 1e-5, rel_tol=1e-2 if not out_f32 else 1e-5,
          bf16_out=not out_f32)
    check("merged lse", lse.cpu().numpy(), ref_l, abs_tol=1e-4, rel_tol=1e-5)
    single = counts == 1
    if out_f32:
        assert np.array_equal(got[single], po[ptr[:-1][single]])


@pytest.mark.parametrize("n_pg,d_model", [(None, 256), (1, 256), (2, 320), (1, 96)],
                         ids=["sliced_128", "dense_256", "sliced_160", "dense_96"])
def test_sliced_oproj_alone(n_pg, d_model):
    """Channels per projection group of one full 128-channel tile, two, one and a
    ragged 32-channel tile, and one ragged tile; rows over two 256-row tiles."""
    import torch
    from paper_2609_07008_amd import device_inputs, mla
    wl = make_custom([300, 211], req_perm=[1, 0], tq=30, H=16, G=2, d_c=512, d_r=64, d_model=d_model,
                     n_pg=n_pg, fp32=False, seed=9, prot_frac=0.1)
    g = wl.geom
    rng = np.random.default_rng(3)
    N, P, G, hl = wl.n_rows, wl.n_prot, g.n_groups, g.heads_per_group - 1
    og = round_bf16(rng.standard_normal((N, G, g.d_latent)).astype(np.float32))
    ol = round_bf16(rng.standard_normal((P, G, hl, g.d_latent)).astype(np.float32))
    w_o = wl.w_o()
    z_off = wl.z_off()
    zpois = z_off.copy()
    zpois[wl.prot_rows] = np.nan
    z = torch.empty((N, g.d_model), dtype=torch.float32, device="cuda")
    mla.sliced_oproj_add(g, N, device_inputs.to_bf16(og), device_inputs.to_bf16(ol), wl.glob_head,
                         torch.from_numpy(np.asarray(wl.prot_rows, dtype=np.int32)).cuda(), P,
                         device_inputs.to_bf16(w_o), device_inputs.to_bf16(zpois), z)
    torch.cuda.synchronize()
    blocks = M.dense_blocks(w_o, g.n_heads, g.d_latent, g.d_model)
    gid, lid = wl.global_head_ids(), wl.local_head_ids().reshape(-1)
    prot_idx = {int(r): i for i, r in enumerate(wl.prot_rows)}
    ref = np.zeros((N, g.d_model))
    for r in range(N):
        ref[r] = M.project(og[r], gid, blocks)
        if r in prot_idx:
            ref[r] += M.project(ol[prot_idx[r]].reshape(-1, g.d_latent), lid, blocks)
        else:
            ref[r] += z_off[r]
    check("z", z.cpu().numpy(), ref, abs_tol=1e-3, rel_tol=1e-4)


def test_sliced_oproj_skips_rows_outside_z():
    """prot_rows is read on the device; an entry past the last row is skipped by
    the Local pass (its o_loc row is not written anywhere), every real row is as
    if the entry were absent."""
    import torch
    from paper_2609_07008_amd import device_inputs, mla
    wl = make_custom([96, 64], req_perm=[1, 0], tq=16, H=16, G=2, d_c=512, d_r=64, d_model=256,
                     fp32=False, seed=4, prot_frac=0.1)
    g = wl.geom
    rng = np.random.default_rng(8)
    N, G, hl = wl.n_rows, g.n_groups, g.heads_per_group - 1
    prot = np.concatenate([np.asarray(wl.prot_rows, dtype=np.int32), [N + 3]]).astype(np.int32)
    P = prot.shape[0]
    og = round_bf16(rng.standard_normal((N, G, g.d_latent)).astype(np.float32))
    ol = round_bf16(rng.standard_normal((P, G, hl, g.d_latent)).astype(np.float32))
    w_o, z_off = wl.w_o(), wl.z_off()
    # guard band after z: rows N .. N+7 of the allocation must stay untouched
    zbuf = torch.full((N + 8, g.d_model), 7.0, dtype=torch.float32, device="cuda")
    mla.sliced_oproj_add(g, N, device_inputs.to_bf16(og), device_inputs.to_bf16(ol), wl.glob_head,
                         torch.from_numpy(prot).cuda(), P, device_inputs.to_bf16(w_o), device_inputs.to_bf16(z_off),
                         zbuf[:N])
    torch.cuda.synchronize()
    assert torch.all(zbuf[N:] == 7.0)
    blocks = M.dense_blocks(w_o, g.n_heads, g.d_latent, g.d_model)
    gid, lid = wl.global_head_ids(), wl.local_head_ids().reshape(-1)
    prot_idx = {int(r): i for i, r in enumerate(prot[:-1])}
    ref = np.zeros((N, g.d_model))
    for r in range(N):
        ref[r] = M.project(og[r], gid, blocks)
        if r in prot_idx:
            ref[r] += M.project(ol[prot_idx[r]].reshape(-1, g.d_latent), lid, blocks)
        else:
            ref[r] += z_off[r]
    check("z", zbuf[:N].cpu().numpy(), ref, abs_tol=1e-3, rel_tol=1e-4)


# ----------------------------------------------------------------------------
# the five workloads at full size, in the launch configuration of the benchmark
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("cfg,split,n_pg", [(2, 0, None), (2, 10 ** 9, None), (2, 0, 1), (2, 10 ** 9, 1),
                                            (3, 8192, None), (3, 10 ** 9, None), (4, 10 ** 9, None),
                                            (5, 10 ** 9, None)])
def test_full_workload(cfg, split, n_pg):
    """Each workload at full size; n_pg = 1 is the dense first projection
    (K = 64 heads x 512 into all 4096 channels) on the 8 x 4096 + 256 workload.
    Per-segment partials are compared on the boundary sample; the other launches
    on the first and last row of every segment plus 32 protected rows."""
    wl = make_workload(cfg, n_proj_groups=n_pg)
    split = min(split, wl.n_rows) if split else 0
    st, _ = run(wl, split, with_part_seg=(cfg <= 3))
    check_bookkeeping(wl, st, split, full_part_seg=(cfg <= 3))
    g = wl.geom
    kv = wl.kv()
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    rows = boundary_sample(wl) if cfg <= 3 and split == 0 else segment_edge_sample(wl)
    compare_rows(wl, st, rows, None, kv=kv, keys=keys)


@pytest.mark.parametrize("cfg", [2, 5])
def test_full_workload_peaked(cfg):
    """Far-from-uniform softmax at full size: unscaled queries and keys."""
    wl = make_workload(cfg, "peaked")
    split = wl.n_rows
    st, _ = run(wl, split, with_part_seg=False)
    g = wl.geom
    kv = wl.kv()
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    compare_rows(wl, st, segment_edge_sample(wl, n_prot=16, seed=2), None, kv=kv, keys=keys)


def test_optional_outputs_may_be_null():
    """part_seg and row_src of the attend call and out_lse of the merge are
    optional (NULL): the required outputs are then bit-identical to a run that
    writes all of them."""
    import torch
    from paper_2609_07008_amd import mla
    wl = _needle_workload(seed=37)
    st, inp = run(wl, 0)
    g = wl.geom
    part_o = torch.full_like(st.part_o, float("nan"))
    part_lse = torch.full_like(st.part_lse, float("nan"))
    part_ptr = torch.zeros_like(st.part_ptr)
    mla.online_attend(g, wl.segs, np.asarray(wl.prot_rows, dtype=np.int32), 0, inp["kv"], inp["q_glob"],
                      inp["q_loc"], part_o, part_lse, part_ptr, None, None, st.ws)
    out_o = torch.full_like(st.out_o, float("nan"))
    mla.segment_merge(st.n_slots, g.d_latent, part_o, part_lse, part_ptr, mla.MLA_BF16, out_o, None)
    torch.cuda.synchronize()
    assert torch.equal(part_ptr, st.part_ptr)
    assert torch.equal(part_o.view(torch.int32), st.part_o.view(torch.int32))
    assert torch.equal(part_lse.view(torch.int32), st.part_lse.view(torch.int32))
    assert torch.equal(out_o.view(torch.int16), st.out_o.view(torch.int16))
