"""GPU parity of the MLA-Off producer (mla_offline_produce, Alg. 1 NativeProducer)
against the fp64 oracle's canonical artifact: every segment evaluated alone at
canonical positions, Local heads only, projected by their W_o blocks."""
import numpy as np
import pytest

from oracle import mla_oracle as M
from parity import check, compare_rows, run
from workloads import make_custom, make_workload, round_bf16

pytestmark = pytest.mark.gpu


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


@pytest.mark.parametrize("out", ["f32", "bf16"])
@pytest.mark.parametrize("variant", ["default", "peaked"])
def test_offline_tiny(out, variant):
    wl = make_workload(1, variant)
    check(f"z_off ({out})", produce(wl, out), M.artifact(wl))


OFFLINE = {
    "ragged": dict(doc_lens=[1, 2, 63, 64, 65, 130, 7], req_perm=[4, 0, 6, 2, 5, 1, 3], tq=37, H=16, G=2,
                   d_model=256),
    "dense_proj": dict(doc_lens=[70, 33, 128], req_perm=[2, 0, 1], tq=20, H=16, G=2, d_model=256, n_pg=1),
    "wide_groups": dict(doc_lens=[96, 40], req_perm=[1, 0], tq=9, H=32, G=4, d_model=512),
    "global_first": dict(doc_lens=[150, 17], req_perm=[1, 0], tq=6, H=16, G=2, d_model=256,
                         glob_head=np.array([0, 0])),
    "global_last": dict(doc_lens=[150, 17], req_perm=[1, 0], tq=6, H=16, G=2, d_model=256,
                        glob_head=np.array([7, 7])),
}


@pytest.mark.parametrize("name", sorted(OFFLINE))
@pytest.mark.parametrize("peaked", [False, True])
def test_offline_512(name, peaked):
    std = dict(c=1.0, kr=1.0, qc=1.0, qr=1.0, wo=0.02, zoff=0.05) if peaked else None
    wl = make_custom(d_c=512, d_r=64, seed=300 + sorted(OFFLINE).index(name), fp32=False, std=std,
                     **OFFLINE[name])
    check("z_off", produce(wl, "f32"), M.artifact(wl))


def test_offline_without_local_heads_is_zero():
    wl = make_custom(doc_lens=[65, 3], req_perm=[1, 0], tq=5, H=4, G=4, d_c=512, d_r=64, d_model=128,
                     fp32=False, seed=31)
    z = produce(wl, "bf16")
    assert np.array_equal(z, np.zeros_like(z))


def test_offline_artifact_feeds_the_online_step():
    """The producer's bf16 artifact as the online step's z_off: the step's z then
    matches the oracle run with the oracle's own artifact."""
    wl = make_workload(1)
    z_gpu = produce(wl, "bf16")
    z_ref = round_bf16(M.artifact(wl).astype(np.float32)).astype(np.float64)
    check("z_off (bf16)", z_gpu, z_ref)
    st, _ = run(wl, 0, z_off=z_gpu)
    compare_rows(wl, st, np.arange(wl.n_rows), z_ref)
