"""GPU parity of the rotary-value variant (geom.value_rope: the value is the
whole latent row, each segment's RoPE output restored by R(+p_s) and rotated
back by R(-t), eq:offonline, Alg. 2) against the fp64 oracle: the 576-wide head
outputs, lse, z_online and z of every online head, same tolerances as the
latent-value step; the offline producer's artifact in the same variant."""
import numpy as np
import pytest

from oracle import mla_oracle as M
from workloads import make_custom, make_workload, round_bf16

from parity import (ABS_TOL, boundary_sample, check, check_bookkeeping, compare_rows, produce, rounded_o_bound, run,
                    segment_edge_sample)

pytestmark = pytest.mark.gpu

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
def test_vrope_custom(name, split, peaked):
    std = dict(c=1.0, kr=1.0, qc=1.0, qr=1.0, wo=0.02, zoff=0.05) if peaked else None
    wl = make_custom(d_c=512, d_r=64, seed=700 + sorted(CUSTOM).index(name), fp32=False, std=std,
                     value_rope=True, **CUSTOM[name])
    assert wl.geom.d_v == 576
    st, _ = run(wl, split)
    check_bookkeeping(wl, st, split)
    compare_rows(wl, st, np.arange(wl.n_rows), wl.z_off())


@pytest.mark.parametrize("case", ["no_protected", "all_protected"])
def test_vrope_edge_cases(case):
    kw = dict(doc_lens=[65, 3, 64], req_perm=[1, 2, 0], tq=5, d_c=512, d_r=64, fp32=False, seed=721,
              H=8, G=2, d_model=128, value_rope=True)
    n = 65 + 3 + 64 + 5
    prot = np.zeros(0, np.int32) if case == "no_protected" else np.arange(n, dtype=np.int32)
    wl = make_custom(prot_rows=prot, **kw)
    for split in (0, 10 ** 9):
        st, _ = run(wl, split)
        compare_rows(wl, st, np.arange(wl.n_rows), wl.z_off())


@pytest.mark.parametrize("tq,prot", [(0, [0]), (0, []), (1, None)], ids=["one_row", "one_row_unprotected",
                                                                       "one_row_and_query"])
def test_vrope_one_row(tq, prot):
    """One-row requests with a rotary value: one key, so each head output is that
    key's latent row with its RoPE part rotated back by the relative angle."""
    kw = dict(doc_lens=[1], req_perm=None, tq=tq, d_c=512, d_r=64, fp32=False, seed=723, H=16, G=2,
              d_model=256, value_rope=True)
    if prot is not None:
        kw["prot_rows"] = np.asarray(prot, dtype=np.int32)
    wl = make_custom(**kw)
    for split in (0, 10 ** 9):
        st, _ = run(wl, split)
        check_bookkeeping(wl, st, split)
        compare_rows(wl, st, np.arange(wl.n_rows), wl.z_off())
    check("z_off (f32)", produce(wl, "f32"), M.artifact(wl))


@pytest.mark.parametrize("cfg,split", [(2, 0), (2, 10 ** 9), (3, 8192), (3, 10 ** 9), (4, 10 ** 9), (5, 10 ** 9)])
def test_vrope_full_workload(cfg, split):
    wl = make_workload(cfg, value_rope=True)
    split = min(split, wl.n_rows) if split else 0
    st, _ = run(wl, split, with_part_seg=False)
    g = wl.geom
    kv = wl.kv()
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    rows = boundary_sample(wl) if cfg == 2 else segment_edge_sample(wl, n_prot=32, seed=cfg)
    compare_rows(wl, st, rows, None, kv=kv, keys=keys)


OFFLINE = {
    "ragged": dict(doc_lens=[1, 2, 63, 64, 65, 130, 7], req_perm=[4, 0, 6, 2, 5, 1, 3], tq=37, H=16, G=2,
                   d_model=256),
    "dense_proj": dict(doc_lens=[70, 33, 128], req_perm=[2, 0, 1], tq=20, H=16, G=2, d_model=256, n_pg=1),
}


@pytest.mark.parametrize("name", sorted(OFFLINE))
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_vrope_offline_producer(name, out):
    std = dict(c=1.0, kr=1.0, qc=1.0, qr=1.0, wo=0.02, zoff=0.05)
    wl = make_custom(d_c=512, d_r=64, seed=740 + sorted(OFFLINE).index(name), fp32=False, std=std,
                     value_rope=True, **OFFLINE[name])
    check(f"z_off ({out})", produce(wl, out), M.artifact(wl), bf16_out=out == "bf16")


def _plant_full(wl, kv, row, seg_idx, u, logit):
    """Key u of segment seg_idx scores `logit` (natural units) for Global head 0
    of `row`: the whole key (latent and RoPE part, the rotary value) is laid
    along that head's query as the row sees it, so with large queries the
    planted value stays moderate."""
    g = wl.geom
    _, _, pos = M.row_geometry(wl.segs)
    q = wl.q_glob(rows=[row])[0, 0].astype(np.float64)
    qc, qr = q[: g.d_latent], q[g.d_latent:]
    ks, _, ps = wl.segs[seg_idx]
    j = int(ks + u)
    n2 = qc @ qc + qr @ qr
    kv = kv.copy()
    kv[j, : g.d_latent] = logit / g.softmax_scale * qc / n2
    kv[j, g.d_latent:] = logit / g.softmax_scale * M.rope(qr, int(pos[row]) - int(ps), g.rope_base) / n2
    return round_bf16(kv.astype(np.float32)), j


@pytest.mark.parametrize("logit,restart", [(25.0, False), (50.0, True), (100.0, True)])
@pytest.mark.parametrize("split", [0, 10 ** 9])
def test_vrope_needle_restart(logit, restart, split):
    """A rotary-value row whose attention restarts: a key of an earlier,
    relocated document planted `logit` nats above zero for one head, with
    queries and keys of unit scale.  Past 2^64 against the first tile's
    reference (+50 nats) the item restarts, and past the float32 range (+100)
    it restarts twice; the RoPE output sums kept in the workspace must be
    cleared with the rest of the item's state."""
    import torch
    from paper_2609_07008_amd import device_inputs, step
    std = dict(c=1.0, kr=1.0, qc=1.0, qr=1.0, wo=0.02, zoff=0.05)
    wl = make_custom([70, 90, 66], req_perm=[2, 0, 1], tq=12, H=16, G=2, d_c=512, d_r=64, d_model=256,
                     fp32=False, seed=31, prot_frac=0.1, std=std, value_rope=True)
    g = wl.geom
    row = wl.n_rows - 1
    seg_idx = int(np.argsort(wl.segs[:, 2])[1])        # second document in request order
    kv, j = _plant_full(wl, wl.kv(), row, seg_idx, 41, logit)
    keys = M.TrueKeys(kv, wl.segs, g.d_latent, g.rope_base)
    _, _, pos = M.row_geometry(wl.segs)
    q = wl.q_glob(rows=[row])[0, 0].astype(np.float64)
    t = int(pos[row])
    qt = np.concatenate([q[:g.d_latent], M.rope(q[g.d_latent:], t, g.rope_base)])
    sc = g.softmax_scale * (keys.k[: t + 1] @ qt)
    needle = int(np.argmax(sc))
    assert (sc[needle] - np.delete(sc, needle).max() > 64 * np.log(2.0)) == restart
    inputs = device_inputs.upload(wl)
    inputs["kv"] = device_inputs.to_bf16(kv)
    st = step.OnlineStep(g, wl.segs, wl.prot_rows, wl.glob_head, min(split, wl.n_rows) if split else 0)
    st.run(inputs["kv"], inputs["q_glob"], inputs["q_loc"], inputs["w_o"], inputs["z_off"])
    torch.cuda.synchronize()
    lse_tol = max(2e-2, logit * 2.0 ** -9)
    rows = [row, row - 1, 0, j]
    # the needle's value reaches the o-proj rounded to bf16: its share of z
    # carries that rounding (up to 2^-8 of each head output times |W_o|)
    z_tol = ABS_TOL + rounded_o_bound(wl, rows, kv=kv, keys=keys)
    compare_rows(wl, st, rows, wl.z_off(), kv=kv, keys=keys, lse_abs_tol=lse_tol, z_abs_tol=z_tol)
