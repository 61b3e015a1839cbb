"""GPU parity of the adaptive MoE fanout (mla_moe_fanout, eq:moe) against the
oracle: ranks, weights and fanouts compared bit-exactly (the fanout is decided
in float32 on both sides), expert counts against a count of the oracle's
executed experts."""
import numpy as np
import pytest

from oracle import mla_oracle as M
from workloads import router_weights

pytestmark = pytest.mark.gpu


def gpu_fanout(p, tau, top_k=6, min_k=3, counts=True):
    import torch
    from paper_2609_07008_amd import mla
    n, e = p.shape
    router = torch.from_numpy(np.ascontiguousarray(p, dtype=np.float32)).cuda()
    idx = torch.full((n, top_k), -7, dtype=torch.int32, device="cuda")
    w = torch.full((n, top_k), float("nan"), dtype=torch.float32, device="cuda")
    k = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    cnt = torch.full((e,), -7, dtype=torch.int32, device="cuda") if counts else None
    mla.moe_fanout(router, tau, idx, w, k, cnt, top_k=top_k, min_k=min_k)
    torch.cuda.synchronize()
    return (idx.cpu().numpy(), w.cpu().numpy(), k.cpu().numpy(), None if cnt is None else cnt.cpu().numpy())


def executed_counts(idx, k, e):
    taken = np.arange(idx.shape[1])[None, :] < k[:, None]
    return np.bincount(idx[taken].ravel(), minlength=e).astype(np.int32)


def check(p, tau, top_k=6, min_k=3):
    gi, gw, gk, gc = gpu_fanout(p, tau, top_k, min_k)
    oi, ow, ok = M.moe_fanout(p, tau, top_k=top_k, min_k=min_k)
    assert np.array_equal(gi, oi)
    assert np.array_equal(gw.view(np.uint32), ow.view(np.uint32))   # bit-exact copies of the inputs
    assert np.array_equal(gk, ok)
    assert np.array_equal(gc, executed_counts(oi, ok, p.shape[1]))


@pytest.mark.parametrize("e", [6, 8, 16, 20, 64, 100, 128, 200, 256, 300, 512, 1000, 1024])
@pytest.mark.parametrize("tau", [0.5, 0.8, 0.9, 0.97])
def test_moe_fanout_random(e, tau):
    check(router_weights(777, e, seed=11 + e), tau)


@pytest.mark.parametrize("top_k,min_k", [(8, 1), (6, 6), (1, 1), (4, 2), (6, 1)])
def test_moe_fanout_top_k_variants(top_k, min_k):
    check(router_weights(513, 96, seed=5), 0.85, top_k, min_k)


def test_moe_fanout_ties_and_specials():
    rng = np.random.default_rng(9)
    p = router_weights(400, 64, seed=9)
    p[:100] = np.round(p[:100] * 16) / 16                       # many equal weights
    p[100:150] = 0.0                                            # zero rows: no shares, K = top_k
    sp = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, -np.nan, -1.0, 3.0], dtype=np.float32)
    for r in range(150, 250):
        p[r, rng.choice(64, size=8, replace=False)] = sp
    p[250:300] = -p[250:300]                                    # negative weights
    for tau in (0.5, 0.9, 1.0, 1.5, -1.0):
        check(p.astype(np.float32), tau)


def test_moe_fanout_empty_clears_counts():
    import torch
    from paper_2609_07008_amd import mla
    cnt = torch.full((32,), 5, dtype=torch.int32, device="cuda")
    empty = torch.empty((0, 32), dtype=torch.float32, device="cuda")
    z32 = torch.empty((0, 6), dtype=torch.int32, device="cuda")
    mla.moe_fanout(empty, 0.9, z32, torch.empty((0, 6), dtype=torch.float32, device="cuda"),
                   torch.empty((0,), dtype=torch.int32, device="cuda"), cnt)
    torch.cuda.synchronize()
    assert cnt.cpu().numpy().tolist() == [0] * 32


def test_moe_fanout_256k_rows_sampled():
    """The 256K-row batch with 256 experts (the benchmark's launch): the oracle on
    2048 sampled rows, exact; every row's fanout in [3, 6]; the counts add up."""
    n, e = 264192, 256
    p = router_weights(n, e, seed=70080)
    gi, gw, gk, gc = gpu_fanout(p, 0.9)
    rows = np.random.default_rng(1).choice(n, size=2048, replace=False)
    oi, ow, ok = M.moe_fanout(p[rows], 0.9)
    assert np.array_equal(gi[rows], oi)
    assert np.array_equal(gw[rows].view(np.uint32), ow.view(np.uint32))
    assert np.array_equal(gk[rows], ok)
    assert gk.min() >= 3 and gk.max() <= 6
    assert int(gc.sum()) == int(gk.sum())
    assert np.array_equal(gc, executed_counts(gi, gk, e))
