"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
compare it with the fp64 oracle on the same seeded inputs."""
from __future__ import annotations

import numpy as np

from oracle import mla_oracle as M
from workloads import round_bf16

ABS_TOL = 2e-2     # max abs error
REL_TOL = 1e-2     # max abs error / max |reference|


def check(name, got, ref, abs_tol=ABS_TOL, rel_tol=REL_TOL, bf16_out=False):
    """max |got - ref| <= abs_tol element-wise and max |got - ref| / max |ref| <= rel_tol.
    bf16_out: the output is stored in bf16, whose rounding alone moves a value by
    up to half an ulp, 2^-8 of its magnitude (more than abs_tol once |ref| > 5);
    that rounding is added to each element's absolute bound."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{name}: non-finite output"
    diff = np.abs(got - ref)
    err = float(diff.max()) if got.size else 0.0
    scale = float(np.abs(ref).max()) if ref.size else 0.0
    rel = err / scale if scale > 0 else err
    allow = abs_tol + (2.0 ** -8 * np.abs(ref) if bf16_out else 0.0)
    assert np.all(diff <= allow) and rel <= rel_tol, f"{name}: max abs err {err:.3e}, relative {rel:.3e}"
    return err, rel


def run(wl, split_keys, z_off=None, with_part_seg=True, out_dtype=None, inputs=None):
    """One step on the GPU; returns the OnlineStep (device buffers) and the uploaded inputs."""
    import torch
    from paper_2609_07008_amd import device_inputs, mla, step
    if inputs is None:
        inputs = device_inputs.upload(wl, z_off=z_off)
    st = step.OnlineStep(wl.geom, wl.segs, wl.prot_rows, wl.glob_head, split_keys,
                         with_part_seg=with_part_seg,
                         out_dtype=mla.MLA_BF16 if out_dtype is None else out_dtype)
    st.run(inputs["kv"], inputs["q_glob"], inputs["q_loc"], inputs["w_o"], inputs["z_off"])
    torch.cuda.synchronize()
    return st, inputs


def artifact_bf16(wl):
    """The tiny workload's artifact, computed by the oracle and rounded to bf16
    (the values the GPU receives)."""
    return round_bf16(M.artifact(wl).astype(np.float32)).astype(np.float64)


def compare_rows(wl, st, rows, z_off, kv=None, keys=None, lse_abs_tol=ABS_TOL, z_abs_tol=ABS_TOL):
    """Oracle vs GPU on storage rows `rows`: O and lse of every online head, z_online and z.
    `lse_abs_tol` widens the absolute bound on lse alone, for planted scores far
    above the workload's range: the kernel rounds the relocated query to bf16,
    so its score error (and the lse error) grows with the score itself.
    `z_abs_tol` (a scalar, or one bound per sorted row and channel) does the same
    for z, whose input is the bf16-rounded head outputs (see rounded_o_bound)."""
    g = wl.geom
    rows = np.asarray(sorted(set(int(r) for r in rows)), dtype=np.int64)
    if isinstance(z_off, np.ndarray):
        zmap = z_off
    else:
        zr = wl.z_off(rows=rows)
        zmap = {int(r): zr[i] for i, r in enumerate(rows)}
    ref = M.reference_rows(wl, rows, z_off=zmap, kv=kv, keys=keys)
    G, hl, d_c = g.n_groups, g.heads_per_group - 1, g.d_v
    N = wl.n_rows
    gslots = (rows[:, None] * G + np.arange(G)[None, :]).reshape(-1)
    o_bf16 = st.out_o.element_size() == 2
    out_o = st.out_o.float()
    o_g = out_o[gslots].cpu().numpy().reshape(len(rows), G, d_c)
    l_g = st.out_lse[gslots].cpu().numpy().reshape(len(rows), G)
    check("O (Global heads)", o_g, ref.o_glob, bf16_out=o_bf16)
    check("lse (Global heads)", l_g, ref.lse_glob, abs_tol=lse_abs_tol)
    if ref.prot_idx:
        idx = sorted(ref.prot_idx)
        a = np.array([ref.prot_idx[i] for i in idx])
        lslots = (N * G + (a[:, None] * G * hl) + np.arange(G * hl)[None, :]).reshape(-1)
        o_l = out_o[lslots].cpu().numpy().reshape(len(a), G, hl, d_c)
        l_l = st.out_lse[lslots].cpu().numpy().reshape(len(a), G, hl)
        check("O (Local heads)", o_l, np.stack([ref.o_loc[i] for i in idx]), bf16_out=o_bf16)
        check("lse (Local heads)", l_l, np.stack([ref.lse_loc[i] for i in idx]), abs_tol=lse_abs_tol)
    z_bf16 = st.z.element_size() == 2
    z = st.z[rows].float().cpu().numpy().astype(np.float64)
    prot = np.isin(rows, np.asarray(wl.prot_rows))
    zoff_rows = np.stack([np.zeros(g.d_model) if p else np.asarray(zmap[int(r)], dtype=np.float64)
                          for r, p in zip(rows, prot)])
    if z_bf16:
        # z stored in bf16: each element carries up to two roundings of 2^-9 |z|
        # (a protected row's Local sum, then z), which z - z_off inherits
        allow = z_abs_tol + 2.0 ** -8 * np.abs(ref.z)
        assert np.all(np.abs(z - zoff_rows - ref.z_online) <= allow), "z_online (bf16 z)"
        check("z", z, ref.z, abs_tol=z_abs_tol, bf16_out=True)
    else:
        check("z_online", z - zoff_rows, ref.z_online, abs_tol=z_abs_tol)
        check("z", z, ref.z, abs_tol=z_abs_tol)
    return ref


def rounded_o_bound(wl, rows, kv=None, keys=None):
    """Per sorted row and channel, the most that rounding the row's head outputs
    to bf16 (half an ulp, 2^-8 of each value) can move z: 2^-8 sum_h |o_h| |W_h|,
    with the oracle's o.  Added to the absolute z bound where planted scores make
    the head outputs large."""
    g = wl.geom
    rows = np.asarray(sorted(set(int(r) for r in rows)), dtype=np.int64)
    zr = wl.z_off(rows=rows)
    ref = M.reference_rows(wl, rows, z_off={int(r): zr[i] for i, r in enumerate(rows)}, kv=kv, keys=keys)
    blocks = np.abs(M.dense_blocks(wl.w_o(), g.n_heads, g.d_v, g.d_model))
    out = np.zeros((rows.shape[0], g.d_model))
    for i in range(rows.shape[0]):
        out[i] = M.project(np.abs(ref.o_glob[i]), wl.global_head_ids(), blocks)
        if i in ref.o_loc:
            out[i] += M.project(np.abs(ref.o_loc[i]).reshape(-1, g.d_v), wl.local_head_ids().reshape(-1), blocks)
    return 2.0 ** -8 * out


def check_bookkeeping(wl, st, split_keys, full_part_seg=True):
    G, hpg = wl.geom.n_groups, wl.geom.heads_per_group
    rs, ptr, pseg = M.enumerate_plan(wl.segs, G, hpg, wl.prot_rows, split_keys)
    assert np.array_equal(st.row_src.cpu().numpy(), rs), "row_src"
    # buffers sized for a capacity hold the call's entries first
    assert st.part_ptr.shape[0] >= ptr.shape[0]
    assert np.array_equal(st.part_ptr[: ptr.shape[0]].cpu().numpy(), ptr), "part_ptr"
    if st.part_seg is not None and full_part_seg:
        assert st.part_seg.shape[0] >= pseg.shape[0]
        assert np.array_equal(st.part_seg[: pseg.shape[0]].cpu().numpy(), pseg), "part_seg"


def boundary_sample(wl, n_extra=8, seed=0):
    """Rows that stress the path: first and last row of every segment, rows on
    both sides of segment boundaries in request order, protected and query rows."""
    rng = np.random.default_rng(seed)
    rows = set()
    for ks, ln, _ in wl.segs:
        rows.update([int(ks), int(ks + ln - 1), int(ks + min(1, ln - 1))])
    prot = np.asarray(wl.prot_rows)
    if prot.size:
        rows.update(int(x) for x in rng.choice(prot, size=min(n_extra, prot.size), replace=False))
    rows.update(int(x) for x in rng.integers(0, wl.n_rows, size=n_extra))
    return sorted(rows)


def produce(wl, out_dtype_name="f32"):
    """z_off of every row from the GPU producer (float64 copy on the host)."""
    import torch
    from paper_2609_07008_amd import device_inputs, mla
    g = wl.geom
    bf16 = out_dtype_name == "bf16"
    kv = device_inputs.to_bf16(wl.kv())
    if g.heads_per_group > 1:
        q = np.ascontiguousarray(wl.q_full()[:, wl.local_head_ids(), :])
        q_loc = device_inputs.to_bf16(q)
    else:
        q_loc = None
    w_o = device_inputs.to_bf16(wl.w_o())
    ws_bytes = mla.offline_produce_query(g, wl.segs)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    z = torch.full((wl.n_rows, g.d_model), float("nan"), dtype=torch.bfloat16 if bf16 else torch.float32,
                   device="cuda")
    mla.offline_produce(g, wl.segs, kv, q_loc, wl.glob_head, w_o, mla.MLA_BF16 if bf16 else mla.MLA_F32, z, ws)
    torch.cuda.synchronize()
    return z.float().cpu().numpy().astype(np.float64)


def segment_edge_sample(wl, n_prot=32, n_rand=8, seed=1):
    """Rows for the full-size comparisons: the first and last row of every
    segment (where relocation angles and chunk boundaries change), `n_prot`
    protected rows (every head online) and `n_rand` uniform rows; seeded."""
    rng = np.random.default_rng(seed)
    rows = set()
    for ks, ln, _ in wl.segs:
        rows.update([int(ks), int(ks + ln - 1)])
    prot = np.asarray(wl.prot_rows)
    if prot.size:
        rows.update(int(x) for x in rng.choice(prot, size=min(n_prot, prot.size), replace=False))
    rows.update(int(x) for x in rng.integers(0, wl.n_rows, size=n_rand))
    return sorted(rows)
