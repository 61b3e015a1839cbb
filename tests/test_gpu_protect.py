"""GPU parity of the protected token-row set (mla_protected_rows, eq:protected)
against the oracle: integer output, compared bit-exactly (rows and count)."""
import numpy as np
import pytest

from oracle import mla_oracle as M
from workloads import make_custom, make_workload

pytestmark = pytest.mark.gpu


def gpu_protect(segs, qseg, flags, scores, edge, tail, budget):
    import torch
    from paper_2609_07008_amd import mla
    segs = np.asarray(segs, dtype=np.int64)
    n = int(segs[:, 1].sum())
    ws = torch.empty(mla.protected_rows_query(segs), dtype=torch.uint8, device="cuda")
    out = torch.full((n,), -1, dtype=torch.int32, device="cuda")
    cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    fl = None if flags is None else torch.from_numpy(np.ascontiguousarray(flags, dtype=np.uint8)).cuda()
    sc = None if scores is None else torch.from_numpy(np.ascontiguousarray(scores, dtype=np.float32)).cuda()
    mla.protected_rows(segs, qseg, edge, tail, budget, fl, sc, out, cnt, ws)
    torch.cuda.synchronize()
    k = int(cnt.item())
    rest = out[k:].cpu().numpy()
    assert np.all(rest == -1), "rows written past the count"
    return out[:k].cpu().numpy()


def oracle(segs, qseg, flags, scores, edge, tail, budget):
    n = int(np.asarray(segs)[:, 1].sum())
    f = np.zeros(n, np.uint8) if flags is None else flags
    s = np.zeros(n, np.float32) if scores is None else scores
    return M.protected_rows(segs, qseg, f, s, edge, tail, budget)


def case(seed, n_docs, max_len, ties=False, specials=False):
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, max_len, size=n_docs).tolist()
    wl = make_custom(lens, req_perm=rng.permutation(n_docs).tolist(), tq=int(rng.integers(1, 40)), H=4, G=2,
                     seed=seed)
    segs = np.asarray(wl.segs, dtype=np.int64)
    n = int(segs[:, 1].sum())
    flags = np.zeros(n, dtype=np.uint8)
    flags[rng.choice(n, size=max(1, n // 50), replace=False)] |= 1
    flags[rng.choice(n, size=max(1, n // 40), replace=False)] |= 2
    scores = rng.standard_normal(n).astype(np.float32)
    if ties:
        scores = np.round(scores * 2).astype(np.float32)
    if specials:
        idx = rng.choice(n, size=min(n, 24), replace=False)
        scores[idx] = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, -np.nan] * 4, dtype=np.float32)[: idx.size]
    return segs, n_docs, flags, scores


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("kind", ["plain", "ties", "specials"])
@pytest.mark.parametrize("budget", [0.10, 0.25, 0.6])
def test_protect_random(seed, kind, budget):
    segs, q, flags, scores = case(seed, n_docs=12, max_len=900, ties=kind == "ties", specials=kind == "specials")
    args = (segs, q, flags, scores, 128, 1000, budget)
    assert np.array_equal(gpu_protect(*args), oracle(*args))


@pytest.mark.parametrize("budget", [0.10, 0.20, 0.25])
def test_protect_256k_geometry(budget):
    wl = make_workload(5)
    segs = np.asarray(wl.segs, dtype=np.int64)
    q = int(np.argmax(segs[:, 2]))                       # the query block is the last segment in request order
    n = wl.n_rows
    rng = np.random.default_rng(5)
    flags = np.zeros(n, dtype=np.uint8)
    flags[rng.choice(n, size=300, replace=False)] |= 2   # dirty rows
    scores = rng.standard_normal(n).astype(np.float32)
    args = (segs, q, flags, scores, 128, 32768, budget)
    got = gpu_protect(*args)
    assert np.array_equal(got, oracle(*args))


@pytest.mark.parametrize("variant", ["no_query", "budget0", "budget1", "all_tail", "null_scores", "null_flags",
                                     "single_row", "edge_zero"])
def test_protect_edge_cases(variant):
    segs, q, flags, scores = case(11, n_docs=5, max_len=300)
    edge, tail, budget = 16, 50, 0.2
    n = int(segs[:, 1].sum())
    if variant == "no_query":
        q = -1
    elif variant == "budget0":
        budget = 0.0
    elif variant == "budget1":
        budget = 1.0
    elif variant == "all_tail":
        tail = n + 5
    elif variant == "null_scores":
        scores = None
    elif variant == "null_flags":
        flags = None
    elif variant == "single_row":
        segs = np.array([[0, 1, 0]], dtype=np.int64)
        q, flags, scores = -1, np.zeros(1, np.uint8), np.ones(1, np.float32)
        budget = 1.0
    elif variant == "edge_zero":
        edge = 0
    args = (segs, q, flags, scores, edge, tail, budget)
    assert np.array_equal(gpu_protect(*args), oracle(*args))


@pytest.mark.parametrize("budget", [0.10, 0.5])
def test_protect_many_segments(budget):
    """More segments than the classify kernel holds in LDS (it then searches the
    table in device memory), many short ones, ragged last block."""
    segs, q, flags, scores = case(21, n_docs=1500, max_len=40, ties=True)
    args = (segs, q, flags, scores, 4, 300, budget)
    assert np.array_equal(gpu_protect(*args), oracle(*args))
