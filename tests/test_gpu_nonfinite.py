"""Non-finite inputs on the GPU: a NaN or infinite latent row ends in bounded
time and stays confined to the rows that attend to it.

A key row j is visible to every row at request position >= P_j.  Those rows
must come out non-finite (no reference max can repair a NaN or infinite score;
IEEE arithmetic carries it into O, lse and z).  Every row that cannot see j is
unaffected, bit for bit, with one documented exception: a row of j's own
document that shares j's work item (a run of at most 128 head-rows) and its
64-key tile multiplies j's latent by a zero weight on the matrix cores, and
0 * inf and 0 * NaN are NaN; such a row's elements are either bit-identical to
the clean run or non-finite.  An infinite score makes the restart vote fire on
every pass, so it also exercises the bounded number of passes of a work item;
a restart keeps the reference max of every head-row that did not vote, so the
other head-rows of the item are recomputed bit for bit.
"""
import numpy as np
import pytest

from oracle import mla_oracle as M
from workloads import make_custom

from parity import run

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2609_07008_amd import mla  # noqa: F401
    yield


def _workload():
    return make_custom([70, 150, 66], req_perm=[2, 0, 1], tq=12, H=16, G=2, d_c=512, d_r=64, d_model=256,
                       fp32=False, seed=41, prot_frac=0.25)


def _outputs(wl, st):
    import torch
    torch.cuda.synchronize()
    G, hl = wl.geom.n_groups, wl.geom.heads_per_group - 1
    o = st.out_o.float().cpu().numpy()
    lse = st.out_lse.cpu().numpy()
    z = st.z.cpu().numpy()
    n = wl.n_rows
    per_row_o, per_row_l = {}, {}
    prot_idx = {int(r): i for i, r in enumerate(wl.prot_rows)}
    for r in range(n):
        slots = list(range(r * G, (r + 1) * G))
        if r in prot_idx:
            a = prot_idx[r]
            slots += list(range(n * G + a * G * hl, n * G + (a + 1) * G * hl))
        per_row_o[r] = o[slots]
        per_row_l[r] = lse[slots]
    return per_row_o, per_row_l, z


def _query_dim0(wl):
    """Latent dim 0 of every online head's query, per row (bf16 values): the sign
    of a score against a key whose latent dim 0 is +inf."""
    G, hl = wl.geom.n_groups, wl.geom.heads_per_group - 1
    qg = wl.q_glob()[:, :, 0]
    out = {r: list(qg[r]) for r in range(wl.n_rows)}
    if len(wl.prot_rows) and hl > 0:
        ql = wl.q_loc()[:, :, :, 0].reshape(len(wl.prot_rows), G * hl)
        for a, r in enumerate(wl.prot_rows):
            out[int(r)] += list(ql[a])
    return {r: np.asarray(v) for r, v in out.items()}


@pytest.mark.parametrize("split", [0, 10 ** 9])
@pytest.mark.parametrize("case", ["nan_row_first", "nan_row_mid", "inf_latent_mid"])
def test_nonfinite_key_row(case, split):
    """nan_row_*: a whole latent row NaN at the first (u = 0) or a middle
    (u = length/2 + 7) position of the middle document: every head of every row that sees it is
    non-finite.  inf_latent_mid: latent dim 0 of that row is +inf, so a head
    whose query dim 0 is positive scores +inf -- its weight overflows on every
    pass, the item restarts until its last permitted pass, and the head output
    is NaN (inf / inf); a head with a negative query dim 0 scores -inf (weight
    0), whose output is finite or NaN depending on whether the matrix cores
    take 0 * inf as NaN, so only the positive heads and z are asserted."""
    import torch
    from paper_2609_07008_amd import device_inputs
    wl = _workload()
    g = wl.geom
    order = np.argsort(wl.segs[:, 2])
    sidx = int(order[1])                          # the middle document in request order
    ks, ln, ps = (int(x) for x in wl.segs[sidx])
    u = 0 if case.endswith("first") else ln // 2 + 7
    assert u < ln
    j = ks + u
    kv = wl.kv().copy()
    if case.startswith("nan"):
        kv[j, :] = np.nan
    else:
        kv[j, 0] = np.inf
    split = min(split, wl.n_rows) if split else 0
    clean, inputs = run(wl, split, with_part_seg=False)
    inputs = dict(inputs)
    inputs["kv"] = device_inputs.to_bf16(kv)
    bad, _ = run(wl, split, with_part_seg=False, inputs=inputs)
    torch.cuda.synchronize()
    assert torch.equal(bad.part_ptr, clean.part_ptr)
    o0, l0, z0 = _outputs(wl, clean)
    o1, l1, z1 = _outputs(wl, bad)
    q0 = _query_dim0(wl)
    _, _, pos = M.row_geometry(wl.segs)
    sees = pos >= pos[j]
    assert sees.sum() > 0 and (~sees).sum() > 0
    for r in range(wl.n_rows):
        if sees[r]:
            bad_heads = (~np.isfinite(o1[r])).any(axis=1)
            must = np.ones_like(bad_heads) if case.startswith("nan") else q0[r] > 0
            assert bad_heads[must].all(), f"row {r} sees row {j} but a head output is finite"
            if must.any():
                assert not np.isfinite(z1[r]).any(), f"row {r} sees row {j} but z has finite elements"
            continue
        same_item_window = ks <= r < j and j - r <= 128     # j's own document, just before it
        for name, a, b in (("O", o0[r], o1[r]), ("lse", l0[r], l1[r]), ("z", z0[r], z1[r])):
            same = a.view(np.uint32) == b.view(np.uint32)
            if same_item_window:
                assert np.all(same | ~np.isfinite(b)), f"row {r}: {name} changed by a finite amount"
            else:
                assert same.all(), f"row {r} cannot see row {j} but its {name} changed"
