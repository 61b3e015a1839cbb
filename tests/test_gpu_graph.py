"""HIP graph capture through the C ABI.

The kernel-only entry points (merge, o-proj, W_b, MoE fanout) are captured once
and replayed several times, with eager work, output poisoning and
synchronizations between the replays; every replay must reproduce the eager
call's outputs bit for bit.  The entry points that upload a plan from the
library's staging buffer (attend, producer, protected set) must refuse a
capturing stream with MLA_ERR_UNSUPPORTED and enqueue nothing."""
import numpy as np
import pytest

from parity import run
from workloads import make_custom, wb_inputs

pytestmark = pytest.mark.gpu


def _bits(t):
    import torch
    return t.contiguous().view(torch.int16 if t.element_size() == 2 else torch.int32).clone()


def _workload():
    return make_custom([70, 90, 66], req_perm=[2, 0, 1], tq=12, H=16, G=2, d_c=512, d_r=64, d_model=256,
                       fp32=False, seed=17, prot_frac=0.2)


def test_kernel_only_calls_replay():
    import torch
    from paper_2609_07008_amd import device_inputs, mla
    wl = _workload()
    st, inp = run(wl, split_keys=0)     # eager attend: several partials per slot for the merge
    # W_b and MoE fanout inputs
    z, w = wb_inputs(300, 192, 200, seed=5)
    zd, wd = device_inputs.to_bf16(z), device_inputs.to_bf16(w)
    y = torch.empty((300, 200), dtype=torch.float32, device="cuda")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(11)
    router = torch.softmax(torch.randn((777, 64), generator=gen, device="cuda") * 2.0, dim=1)
    e_idx = torch.empty((777, 6), dtype=torch.int32, device="cuda")
    e_w = torch.empty((777, 6), dtype=torch.float32, device="cuda")
    fan = torch.empty((777,), dtype=torch.int32, device="cuda")
    cnt = torch.empty((64,), dtype=torch.int32, device="cuda")

    def tail():
        st.merge()
        st.oproj(inp["w_o"], inp["z_off"])
        mla.shared_wb(zd, wd, y)
        mla.moe_fanout(router, 0.9, e_idx, e_w, fan, cnt)

    outs = [st.out_o, st.out_lse, st.z, y, e_idx, e_w, fan, cnt]
    tail()
    torch.cuda.synchronize()
    ref = [_bits(t) for t in outs]

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        tail()
    for rep in range(3):
        for t in outs:             # poison every output, eagerly, on the default stream
            t.view(torch.uint8).fill_(0xFF)
        other = torch.empty_like(y)
        mla.shared_wb(zd, wd, other)   # eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, t, r in zip(("out_o", "out_lse", "z", "y", "expert_idx", "expert_w", "fanout", "count"),
                              outs, ref):
            assert torch.equal(_bits(t), r), f"replay {rep}: {name} differs from the eager call"
        assert torch.equal(_bits(other), ref[3])


def test_plan_uploads_refuse_capture():
    import torch
    from paper_2609_07008_amd import device_inputs, mla
    wl = _workload()
    st, inp = run(wl, split_keys=0)
    part_ref = _bits(st.part_o)
    g = wl.geom
    n = wl.n_rows
    hl = g.heads_per_group - 1
    q_all = torch.zeros((n, g.n_groups, hl, g.d_latent + g.d_rope), dtype=torch.bfloat16, device="cuda")
    z_pro = torch.empty((n, g.d_model), dtype=torch.bfloat16, device="cuda")
    ws_pro = torch.empty(mla.offline_produce_query(g, wl.segs), dtype=torch.uint8, device="cuda")
    flags = torch.zeros((n,), dtype=torch.uint8, device="cuda")
    scores = torch.zeros((n,), dtype=torch.float32, device="cuda")
    prot = torch.empty((n,), dtype=torch.int32, device="cuda")
    n_prot = torch.empty((1,), dtype=torch.int32, device="cuda")
    ws_prot = torch.empty(mla.protected_rows_query(wl.segs), dtype=torch.uint8, device="cuda")
    st.part_o.view(torch.uint8).fill_(0xFF)
    marker = torch.zeros((16,), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        marker.add_(1.0)
        with pytest.raises(mla.MlaError) as e1:
            st.attend(inp["kv"], inp["q_glob"], inp["q_loc"])
        with pytest.raises(mla.MlaError) as e2:
            mla.offline_produce(g, wl.segs, inp["kv"], q_all, wl.glob_head, inp["w_o"], mla.MLA_BF16, z_pro, ws_pro)
        with pytest.raises(mla.MlaError) as e3:
            mla.protected_rows(wl.segs, len(wl.segs) - 1, 4, 8, 0.2, flags, scores, prot, n_prot, ws_prot)
    assert e1.value.status == e2.value.status == e3.value.status == 3
    assert "capturing" in e1.value.detail
    graph.replay()
    torch.cuda.synchronize()
    assert torch.equal(marker, torch.ones_like(marker))          # the graph holds the add only
    assert torch.all(_bits(st.part_o) == -1)                      # the refused attend wrote nothing
    st.attend(inp["kv"], inp["q_glob"], inp["q_loc"])             # eager again: unaffected
    torch.cuda.synchronize()
    assert torch.equal(_bits(st.part_o), part_ref)
