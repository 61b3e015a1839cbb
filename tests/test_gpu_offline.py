"""GPU parity of the MLA-Off producer (mla_offline_produce, Alg. 1 NativeProducer)
against the fp64 oracle's canonical artifact: every segment evaluated alone at
canonical positions, Local heads only, projected by their W_o blocks."""
import numpy as np
import pytest

from oracle import mla_oracle as M
from parity import check, compare_rows, produce, run
from workloads import make_custom, make_workload, round_bf16

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("out", ["f32", "bf16"])
@pytest.mark.parametrize("variant", ["default", "peaked"])
def test_offline_tiny(out, variant):
    wl = make_workload(1, variant)
    check(f"z_off ({out})", produce(wl, out), M.artifact(wl), bf16_out=out == "bf16")


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


@pytest.mark.parametrize("tq", [0, 1])
def test_offline_one_row_documents(tq):
    """A request of one one-row document (and a one-row query block): every head
    output is the single key's latent, projected by the Local heads' blocks."""
    wl = make_custom(doc_lens=[1], req_perm=None, tq=tq, H=16, G=2, d_c=512, d_r=64, d_model=256,
                     fp32=False, seed=33)
    for out in ("f32", "bf16"):
        check(f"z_off ({out})", produce(wl, out), M.artifact(wl), bf16_out=out == "bf16")


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
    check("z_off (bf16)", z_gpu, z_ref, bf16_out=True)
    st, _ = run(wl, 0, z_off=z_gpu)
    compare_rows(wl, st, np.arange(wl.n_rows), z_ref)


@pytest.mark.parametrize("cfg", [4, 5])
def test_offline_full_size_sampled(cfg):
    """The producer at full size: the benchmark's 256K geometry and launch (64 x
    4096-token documents + 2048 query rows, 56 Local heads, 512 channels per
    projection group) and the 128-head workload (32 x 2048-token documents, 112
    Local heads, 16 projection groups of 448 channels: a ragged last column
    tile), bf16 artifact, inputs drawn on the device as the benchmark draws them;
    sampled rows (segment starts and ends, tile edges, query rows, random rows)
    against the oracle's canonical artifact computed from the same values copied
    back."""
    import torch
    from paper_2609_07008_amd import mla
    wl = make_workload(cfg)
    g = wl.geom
    n, hl = wl.n_rows, g.heads_per_group - 1
    gen = torch.Generator(device="cuda")
    gen.manual_seed(4242)

    def draw(shape, std):
        x = torch.empty(shape, dtype=torch.float32, device="cuda").normal_(0.0, 1.0, generator=gen)
        return (x * std).to(torch.bfloat16)

    kv = torch.cat([draw((n, g.d_latent), g.d_latent ** -0.5), draw((n, g.d_rope), g.d_rope ** -0.5)], 1)
    q = torch.empty((n, g.n_groups, hl, g.d_qk), dtype=torch.bfloat16, device="cuda")
    for c0 in range(0, n, 16384):
        c1 = min(n, c0 + 16384)
        q[c0:c1, :, :, :g.d_latent] = draw((c1 - c0, g.n_groups, hl, g.d_latent), g.d_latent ** -0.5)
        q[c0:c1, :, :, g.d_latent:] = draw((c1 - c0, g.n_groups, hl, g.d_rope), g.d_rope ** -0.5)
    rows_w = (g.n_heads // g.n_proj_groups) * g.d_latent
    w_o = draw((g.n_proj_groups, rows_w, g.d_model // g.n_proj_groups), 0.02)
    z = torch.full((n, g.d_model), float("nan"), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(mla.offline_produce_query(g, wl.segs), dtype=torch.uint8, device="cuda")
    mla.offline_produce(g, wl.segs, kv, q, wl.glob_head, w_o, mla.MLA_BF16, z, ws)
    torch.cuda.synchronize()

    segs = np.asarray(wl.segs)
    rng = np.random.default_rng(11)
    picks = []                                   # (segment, canonical u)
    n_docs = len(segs) - 1
    for s in [0, 1, n_docs // 2, n_docs - 1]:
        picks += [(s, u) for u in (0, 1, 63, 64, 65, 127, 2047, 4095) if u < segs[s, 1]]
    q_seg = int(np.argmax(segs[:, 2]))           # the query block (last in request order)
    picks += [(q_seg, u) for u in (0, 1, 1000, int(segs[q_seg, 1]) - 1)]
    picks += [(int(s), int(rng.integers(0, segs[s, 1]))) for s in rng.integers(0, len(segs), size=8)]
    blocks = M.dense_blocks(w_o.float().cpu().numpy(), g.n_heads, g.d_latent, g.d_model)
    loc = wl.local_head_ids().reshape(-1)
    got, ref = [], []
    for s, u in picks:
        ks = int(segs[s, 0])
        kc = kv[ks:ks + u + 1].float().cpu().numpy().astype(np.float64)
        q_row = q[ks + u].float().cpu().numpy().reshape(-1, g.d_qk)
        ref.append(M.artifact_row(g, kc, q_row, u, blocks, loc))
        got.append(z[ks + u].float().cpu().numpy())
    assert bool(torch.isfinite(z).all())         # every row written
    check("z_off (bf16, 256K, sampled)", np.stack(got), np.stack(ref), bf16_out=True)
