"""GPU parity of the fp32 implicit-GEMM kernel (forward, forward with the
bias + leaky-ReLU epilogue and slope mask, backward-data with every stride
parity class) against the oracle, for every tile shape the kernel is built
with (CF_F32_TILE forces one), at sizes that span several tiles and end in
ragged tails."""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_04728_amd import binding as B
from tests._util import TOL, dev, maxabs_err, to_np

pytestmark = pytest.mark.gpu

# N, (D,H,W), CI, CO, k, stride, pad
CASES = [
    (1, (17, 9, 33), 16, 32, 4, 1, "same"),     # the 16 -> 32 layer, ragged in every dimension
    (2, (12, 10, 14), 32, 64, 4, 2, "same"),    # the stride-2 layer: 8 backward classes
    (1, (9, 8, 8), 64, 64, 3, 1, "same"),
    (1, (8, 8, 9), 64, 128, 2, 1, "same"),      # asymmetric SAME (0, 1)
    (1, (7, 8, 8), 128, 128, 2, 1, "valid"),
    (2, (5, 6, 7), 48, 96, 3, 2, "valid"),      # 48 = 3 k-steps of 16 channels, odd classes
]
TILES = list(range(7))


def ids(c):
    return "n%d_%dx%dx%d_c%d-%d_k%d_s%d_%s" % (c[0], *c[1], *c[2:])


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("case", CASES, ids=ids)
def test_f32_fwd_and_bwd_data(case, tile, monkeypatch):
    N, dhw, CI, CO, k, s, pad = case
    desc = B.make_desc(N, dhw, CI, CO, k, s, pad, "f32")
    monkeypatch.setenv("CF_F32_TILE", str(tile))
    rng = np.random.default_rng(31 + tile)
    x = dev(rng.standard_normal((N, *dhw, CI)), "f32")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CI), "f32")
    b = torch.as_tensor(rng.standard_normal(CO) * 0.1, dtype=torch.float32, device="cuda")
    od = B.cf_conv3d_out_shape(desc)
    z = torch.full((N, *od, CO), float("nan"), device="cuda")
    y = torch.full_like(z, float("nan"))
    mask = torch.zeros(B.cf_conv3d_mask_bytes(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_fwd(desc, x, w, z)
    assert B.cf_conv3d_fused_supported(desc, 0) & B.FUSED_FWD
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.2, 0, y, mask)
    dz = dev(rng.standard_normal((N, *od, CO)), "f32")
    dx = torch.full((N, *dhw, CI), float("nan"), device="cuda")
    B.cf_conv3d_bwd_data(desc, dz, w, dx)
    torch.cuda.synchronize()
    zr = oracle.conv3d_fwd(to_np(x), to_np(w), stride=s, pad=pad)
    assert maxabs_err(to_np(z), zr) <= TOL["f32"]
    u = zr + to_np(b)
    assert maxabs_err(to_np(y), oracle.bias_lrelu_fwd(zr, to_np(b), 0.2)) <= TOL["f32"]
    bits = np.unpackbits(mask.cpu().numpy(), bitorder="little")[:u.size].astype(bool).reshape(u.shape)
    decided = np.abs(u) > 1e-5 * np.abs(u).max()
    assert np.array_equal(bits[decided], (u > 0)[decided])
    dxr = oracle.conv3d_bwd_data(to_np(dz), to_np(w), dhw, stride=s, pad=pad)
    assert maxabs_err(to_np(dx), dxr) <= TOL["f32"]
