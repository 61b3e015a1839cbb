"""GPU parity of the shared second projection y = W_b z (mla_shared_wb) against
the fp64 oracle.  Inputs are bf16 values, so every product is exact in fp32 and
the only GPU error is fp32 accumulation (and the final bf16 rounding for bf16
output): besides the stated tolerance, each element is held to
|err| <= 3e-4 * sum_i |w_b[o,i] z[r,i]| (+ 2^-8 |y| for bf16 output)."""
import numpy as np
import pytest

from oracle import mla_oracle as M
from parity import check
from workloads import wb_inputs

pytestmark = pytest.mark.gpu


def gpu_wb(z, w, out="f32"):
    import torch
    from paper_2609_07008_amd import device_inputs, mla
    zd = device_inputs.to_bf16(z)
    wd = device_inputs.to_bf16(w)
    y = torch.full((z.shape[0], w.shape[0]), float("nan"), device="cuda",
                   dtype=torch.bfloat16 if out == "bf16" else torch.float32)
    mla.shared_wb(zd, wd, y)
    torch.cuda.synchronize()
    return y.float().cpu().numpy().astype(np.float64)


def check_wb(got, z, w, out="f32", rows=None):
    zz = z if rows is None else z[rows]
    ref = M.shared_wb(zz, w)
    check("y", got, ref)
    bound = 3e-4 * (np.abs(zz.astype(np.float64)) @ np.abs(w.astype(np.float64)).T) + 1e-30
    if out == "bf16":
        bound = bound + 2.0 ** -8 * np.abs(ref)
    assert np.all(np.abs(got - ref) <= bound)


SHAPES = {
    "one_tile_ragged": (100, 64, 40),
    "ragged_rows_and_channels": (300, 192, 200),
    "several_tiles": (1000, 512, 520),
    "single_k_step": (257, 64, 257),
    "two_k_steps": (513, 128, 300),
    "one_channel": (70, 128, 1),
    "wide": (600, 2048, 1024),
    "one_row": (1, 64, 1),
    "largest_d_in": (40, 16384, 70),
}


@pytest.mark.parametrize("name", sorted(SHAPES))
@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_wb_shapes(name, out):
    n, d_in, d_out = SHAPES[name]
    z, w = wb_inputs(n, d_in, d_out, seed=17 + sorted(SHAPES).index(name), z_std=1.0, w_std=d_in ** -0.5)
    check_wb(gpu_wb(z, w, out), z, w, out)


def test_wb_256k_geometry_sampled():
    """The benchmark's launch: 264,192 rows, 4096 -> 4096, z drawn on the device
    by torch (seeded); the oracle on 512 sampled rows (all channels) of the same
    bf16 z, copied back."""
    import torch
    from paper_2609_07008_amd import device_inputs, mla
    n, d = 264192, 4096
    g = torch.Generator(device="cuda")
    g.manual_seed(70081)
    z = (torch.randn((n, d), generator=g, device="cuda") * 0.05).to(torch.bfloat16)
    _, w = wb_inputs(1, d, d, seed=70080)
    y = torch.empty((n, d), dtype=torch.float32, device="cuda")
    mla.shared_wb(z, device_inputs.to_bf16(w), y)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(2).choice(n, size=512, replace=False))
    rows[0], rows[-1] = 0, n - 1
    idx = torch.from_numpy(rows).cuda()
    zs = z[idx].float().cpu().numpy()
    got = y[idx].cpu().numpy().astype(np.float64)
    check_wb(got, zs, w)
