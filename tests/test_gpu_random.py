"""Randomized GPU parity of the MLA-Online step (512+64 latent): seeded random
segment tables (1-8 documents of 1-300 rows at permuted offsets, 0-40 query
rows), head partitions, dense or sliced W_o, protected fractions, split modes
and value scales; every row and head against the fp64 oracle, bookkeeping
bit-exact.  The draw of each case depends only on its seed."""
import numpy as np
import pytest

from oracle import mla_oracle as M
from workloads import make_custom

from parity import check, check_bookkeeping, compare_rows, produce, run

pytestmark = pytest.mark.gpu

PARTITIONS = [(8, 1), (16, 2), (32, 4), (16, 4), (8, 8)]


def random_case(seed):
    rng = np.random.default_rng(9000 + seed)
    nd = int(rng.integers(1, 9))
    lens = [int(x) for x in rng.integers(1, 301, size=nd)]
    perm = [int(x) for x in rng.permutation(nd)]
    tq = int(rng.integers(0, 41))
    H, G = PARTITIONS[int(rng.integers(0, len(PARTITIONS)))]
    n_pg = G if rng.random() < 0.6 else 1
    d_model = int(rng.choice([128, 256])) if n_pg == 1 else 64 * G
    peaked = bool(rng.random() < 0.4)
    std = dict(c=1.0, kr=1.0, qc=1.0, qr=1.0, wo=0.02, zoff=0.05) if peaked else None
    wl = make_custom(lens, req_perm=perm, tq=tq, H=H, G=G, d_c=512, d_r=64, d_model=d_model, n_pg=n_pg,
                     prot_frac=float(rng.uniform(0.0, 0.5)), seed=9100 + seed, fp32=False, std=std)
    split = int(rng.choice([0, 50, 200, 10 ** 9]))
    return wl, split


@pytest.mark.parametrize("seed", range(16))
def test_random_step(seed):
    wl, split = random_case(seed)
    st, _ = run(wl, split)
    check_bookkeeping(wl, st, split)
    compare_rows(wl, st, np.arange(wl.n_rows), wl.z_off())


@pytest.mark.parametrize("seed", range(8))
def test_random_offline_producer(seed):
    """The producer on the same random segment tables and head partitions (its
    plan ignores the protected set and the split mode): z_off of every row
    against the oracle's canonical artifact, in f32 and bf16."""
    wl, _ = random_case(seed)
    ref = M.artifact(wl)
    out = "bf16" if seed % 2 else "f32"
    check(f"z_off ({out})", produce(wl, out), ref, bf16_out=out == "bf16")
