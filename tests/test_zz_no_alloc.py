"""The allocation-free attend entry point (mla_online_attend_planned_noalloc)
through the C ABI against mla_online_attend_planned with a caller workspace, on
two calls in a row, the second with a smaller request: the library's scratch
array keeps the first call's contents, which the second must not depend on."""
import numpy as np
import pytest

from workloads import make_custom, make_workload

pytestmark = pytest.mark.gpu


def _bits(t):
    import torch
    size = t.element_size()
    if size == 1:
        return t.contiguous().clone()
    return t.contiguous().view({2: torch.int16, 4: torch.int32, 8: torch.int64}[size]).clone()


def _both(wl, split, cap, tag):
    """One workspace call and one scratch call on the same inputs; returns both
    sets of outputs (bit patterns) after checking the scratch call's status."""
    import torch
    from paper_2609_07008_amd import device_inputs, mla, step
    print(f"no-alloc case {tag}: rows {wl.n_rows}, protected {wl.n_prot}, split {split}, cap {cap}", flush=True)
    inputs = device_inputs.upload(wl)
    ref = step.PlannedStep(wl.geom, wl.segs, wl.glob_head, split, cap)
    assert ref.info.ws_bytes <= mla.NOALLOC_SCRATCH_BYTES
    p = np.zeros(max(cap, 1), dtype=np.int32)
    p[: wl.n_prot] = wl.prot_rows
    prot_d = torch.from_numpy(p).cuda()
    n_d = torch.tensor([wl.n_prot], dtype=torch.int32, device="cuda")
    ref.attend(prot_d, n_d, inputs["kv"], inputs["q_glob"], inputs["q_loc"])
    out_o = torch.full_like(ref.out_o, float("nan"))
    out_lse = torch.full_like(ref.out_lse, float("nan"))
    part_ptr = torch.full_like(ref.part_ptr, -3)
    part_seg = torch.full_like(ref.part_seg, -3)
    row_src = torch.full_like(ref.row_src, 9)
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    mla.online_attend_planned_noalloc(wl.geom, ref.info, ref.plan, prot_d, n_d, inputs["kv"], inputs["q_glob"],
                                      inputs["q_loc"], out_o, out_lse, part_ptr, part_seg, row_src, status)
    torch.cuda.synchronize()
    assert int(ref.status.item()) == 0 and int(status.item()) == 0
    n_slots = wl.n_rows * wl.geom.n_groups + wl.n_prot * wl.geom.n_local
    n_parts = int(ref.part_ptr[n_slots].item())
    for name, a, b in (("out_o", out_o[:n_slots], ref.out_o[:n_slots]),
                       ("out_lse", out_lse[:n_slots], ref.out_lse[:n_slots]),
                       ("part_ptr", part_ptr[: n_slots + 1], ref.part_ptr[: n_slots + 1]),
                       ("part_seg", part_seg[:n_parts], ref.part_seg[:n_parts]),
                       ("row_src", row_src, ref.row_src)):
        assert torch.equal(_bits(a), _bits(b)), f"{tag}: {name} differs from the workspace call"


def test_noalloc_two_calls_second_smaller():
    # first: the 8 x 4096 + 256 workload, every row may be protected, one chunk per slot
    big = make_workload(2)
    _both(big, big.n_rows, big.n_rows, "large")
    # second, right after: a small ragged request in a chunked plan
    small = make_custom([1, 2, 63, 64, 65, 130, 7], req_perm=[4, 0, 6, 2, 5, 1, 3], tq=37, H=16, G=2, d_c=512,
                        d_r=64, d_model=256, fp32=False, seed=81, prot_frac=0.1)
    _both(small, 100, small.n_prot, "small")


def test_noalloc_refuses_plans_larger_than_its_scratch():
    """A plan whose workspace exceeds the scratch array is refused before anything
    is enqueued (a per-segment plan of the 8 x 4096 workload needs GBs of partials)."""
    import torch
    from paper_2609_07008_amd import mla, step
    wl = make_workload(2)
    st = step.PlannedStep(wl.geom, wl.segs, wl.glob_head, 0, wl.n_prot, bookkeeping=False)
    assert st.info.ws_bytes > mla.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((16,), dtype=torch.int32, device="cuda")
    with pytest.raises(mla.MlaError) as e:
        mla.online_attend_planned_noalloc(wl.geom, st.info, st.plan, x, x, x, x, x, st.out_o)
    assert e.value.status == 6 and "scratch" in e.value.detail
