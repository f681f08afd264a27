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
TILES = list(range(8))


def ids(c):
    return "n%d_%dx%dx%d_c%d-%d_k%d_s%d_%s" % (c[0], *c[1], *c[2:])


@pytest.mark.parametrize("fn", ["auto", "1", "2", "4"])
@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("case", CASES, ids=ids)
def test_f32_fwd_and_bwd_data(case, tile, fn, monkeypatch):
    """Every tile shape, with the column-group width forced to 1, 2 or 4
    groups of 16 (CF_F32_FN; ignored where it does not divide the columns) or
    left to the cost model."""
    if fn != "auto" and tile not in (0, 3, 6):
        pytest.skip("column-group widths are covered on three tile shapes")
    N, dhw, CI, CO, k, s, pad = case
    desc = B.make_desc(N, dhw, CI, CO, k, s, pad, "f32")
    monkeypatch.setenv("CF_F32_TILE", str(tile))
    if fn != "auto":
        monkeypatch.setenv("CF_F32_FN", fn)
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


# N, (D,H,W), CI, CO, k, stride: the pooled layers of the stack (16 -> 32 and the
# stride-2 32 -> 64) at sizes with several bricks, ragged tails and odd extents
POOLED = [
    (1, (17, 9, 33), 16, 32, 4, 1),
    (2, (12, 10, 14), 32, 64, 4, 2),
    (1, (13, 11, 18), 32, 64, 4, 2),    # odd conv-output extents: floor pooling
    (2, (7, 8, 9), 64, 64, 3, 1),       # 64-channel units of the weight gradient
]


@pytest.mark.parametrize("ru", ["auto", "1", "2"])
@pytest.mark.parametrize("case", POOLED, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d_s%d" % (c[0], *c[1], *c[2:]))
def test_f32_pooled_layer_fused(case, ru, monkeypatch):
    """Fused forward (pooled output + slope mask) and fused backward-weights
    (dW, db and the stored dz) of a pooled fp32 layer, any stride, against the
    oracle; the unfused backward-data of the stored dz against the oracle.
    CF_F32W_RU forces one or two row units per wave in the weight gradient."""
    if ru != "auto":
        monkeypatch.setenv("CF_F32W_RU", ru)
    N, dhw, CI, CO, k, s = case
    desc = B.make_desc(N, dhw, CI, CO, k, s, "same", "f32")
    sup = B.cf_conv3d_fused_supported(desc, B.CF_FUSE_POOL2)
    assert sup & B.FUSED_FWD and sup & B.FUSED_BWD_WEIGHT and sup & B.FUSED_BWD_WEIGHT_DZ
    rng = np.random.default_rng(41)
    od = B.cf_conv3d_out_shape(desc)
    pdhw = tuple(t // 2 for t in od)
    x = dev(np.log1p(rng.poisson(np.exp(rng.standard_normal((N, *dhw, CI))))), "f32")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CI), "f32")
    bh = rng.standard_normal(CO) * 0.1
    b = torch.as_tensor(bh, dtype=torch.float32, device="cuda")
    out = torch.full((N, *pdhw, CO), float("nan"), device="cuda")
    mask = torch.zeros(B.cf_conv3d_mask_bytes(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.01, B.CF_FUSE_POOL2, out, mask)
    g = dev(rng.standard_normal((N, *pdhw, CO)), "f32")
    mask_r = torch.as_tensor(rng.integers(0, 256, mask.numel(), dtype=np.uint8), device="cuda")
    ws = torch.empty(B.cf_conv3d_bwd_weight_fused_workspace_size(desc, B.CF_FUSE_POOL2), dtype=torch.uint8,
                     device="cuda")
    dw = torch.full((k, k, k, CI, CO), float("nan"), device="cuda")
    db = torch.full((CO,), float("nan"), device="cuda")
    dz = torch.full((N, *od, CO), float("nan"), device="cuda")
    B.cf_conv3d_bwd_weight_fused_dz(desc, x, g, mask_r, 0.2, B.CF_FUSE_POOL2, dw, db, dz, ws)
    dx = torch.full((N, *dhw, CI), float("nan"), device="cuda")
    B.cf_conv3d_bwd_data(desc, dz, w, dx)
    torch.cuda.synchronize()
    zr = oracle.conv3d_fwd(to_np(x), to_np(w), stride=s)
    u = zr + bh
    pr = oracle.avgpool3d_fwd(oracle.bias_lrelu_fwd(zr, bh, 0.01))
    assert maxabs_err(to_np(out), pr) <= TOL["f32"]
    nb = u.size
    bits = np.unpackbits(mask.cpu().numpy(), bitorder="little")[:nb].astype(bool).reshape(u.shape)
    decided = np.abs(u) > 1e-5 * np.abs(u).max()
    assert np.array_equal(bits[decided], (u > 0)[decided])
    rb = np.unpackbits(mask_r.cpu().numpy(), bitorder="little")[:nb].astype(bool).reshape(u.shape)
    dzr = oracle.avgpool3d_bwd(to_np(g), od) * np.where(rb, 1.0, 0.2)
    assert maxabs_err(to_np(dz), dzr) <= TOL["f32"]
    assert maxabs_err(to_np(dw), oracle.conv3d_bwd_weight(to_np(x), dzr, k, stride=s)) <= TOL["f32"]
    assert maxabs_err(to_np(db), dzr.reshape(-1, CO).sum(0)) <= TOL["f32"]
    assert maxabs_err(to_np(dx), oracle.conv3d_bwd_data(dzr, to_np(w), dhw, stride=s)) <= TOL["f32"]


# the four-tap modes (stride-1 4-wide kernels): forward, forward + bias + lReLU
# + mask, pooled forward and backward-data,
# each with the default modes ("tk": taps in K forward, output shift backward
# where the w rows tile), with DPP lane shifts ("dpp") and with neither ("off":
# one tap per k-step), against the oracle
SHIFT = [
    (1, (9, 7, 32), 16, 32, 4),
    (2, (5, 6, 48), 16, 32, 4),
    (1, (6, 5, 32), 32, 64, 4),
    (1, (8, 6, 16), 16, 32, 4),     # one fragment per row: both edges are padding
    (2, (3, 5, 64), 16, 32, 4),     # whole 64-voxel w rows per tile (output shift)
    (2, (4, 5, 45), 16, 32, 4),     # a 64-row tile per 45-voxel w row (output shift)
    (1, (6, 5, 63), 16, 32, 4, "valid"),  # the paper's padding: 60 -> 63 backward-data
]


@pytest.mark.parametrize("mode", ["tk", "dpp", "off"])
@pytest.mark.parametrize("case", SHIFT, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d" % (c[0], *c[1], *c[2:5]) + "".join(c[5:]))
def test_f32_shift_mode(case, mode, monkeypatch):
    N, dhw, CI, CO, k = case[:5]
    pad = case[5] if len(case) > 5 else "same"
    monkeypatch.setenv("CF_F32_SHIFT", "0" if mode == "off" else "1")
    monkeypatch.setenv("CF_F32_TK", "0" if mode == "dpp" else "1")
    monkeypatch.setenv("CF_F32_OS", "0" if mode == "dpp" else "1")
    desc = B.make_desc(N, dhw, CI, CO, k, 1, pad, "f32")
    rng = np.random.default_rng(51)
    x = dev(rng.standard_normal((N, *dhw, CI)), "f32")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CI), "f32")
    bh = rng.standard_normal(CO) * 0.1
    b = torch.as_tensor(bh, dtype=torch.float32, device="cuda")
    od = B.cf_conv3d_out_shape(desc)
    z = torch.full((N, *od, CO), float("nan"), device="cuda")
    y = torch.full_like(z, float("nan"))
    B.cf_conv3d_fwd(desc, x, w, z)
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.2, 0, y, None)
    p = torch.full((N, *(t // 2 for t in od), CO), float("nan"), device="cuda")
    mask = torch.zeros(B.cf_conv3d_mask_bytes(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.2, B.CF_FUSE_POOL2, p, mask)
    dz = dev(rng.standard_normal((N, *od, CO)), "f32")
    dx = torch.full((N, *dhw, CI), float("nan"), device="cuda")
    B.cf_conv3d_bwd_data(desc, dz, w, dx)
    torch.cuda.synchronize()
    zr = oracle.conv3d_fwd(to_np(x), to_np(w), pad=pad)
    assert maxabs_err(to_np(z), zr) <= TOL["f32"]
    yr = oracle.bias_lrelu_fwd(zr, bh, 0.2)
    assert maxabs_err(to_np(y), yr) <= TOL["f32"]
    assert maxabs_err(to_np(p), oracle.avgpool3d_fwd(yr)) <= TOL["f32"]
    u = zr + bh
    bits = np.unpackbits(mask.cpu().numpy(), bitorder="little")[:u.size].astype(bool).reshape(u.shape)
    decided = np.abs(u) > 1e-5 * np.abs(u).max()
    assert np.array_equal(bits[decided], (u > 0)[decided])
    assert maxabs_err(to_np(dx), oracle.conv3d_bwd_data(to_np(dz), to_np(w), dhw, pad=pad)) <= TOL["f32"]


# unpooled fp32 layers, backward from (dy, y): N, (D,H,W), CI, CO, k, stride
DYY = [
    (1, (8, 8, 8), 64, 64, 3, 1),
    (2, (5, 6, 7), 64, 128, 2, 1),
    (1, (9, 7, 8), 128, 128, 2, 1),
    (2, (12, 10, 14), 32, 64, 4, 2),    # stride 2: every backward-data class
    (1, (6, 5, 32), 16, 32, 4, 1),      # shift-mode backward-data
]


@pytest.mark.parametrize("case", DYY, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d_s%d" % (c[0], *c[1], *c[2:]))
def test_f32_unpooled_fused_backward(case):
    """dW, db (and the stored dz) from (dy, y) and dx from (dy, y), with
    dz = dy * (y > 0 ? 1 : alpha): the activation y comes from the fused
    forward of the same layer (exact zeros included where the bias cancels)."""
    N, dhw, CI, CO, k, s = case
    desc = B.make_desc(N, dhw, CI, CO, k, s, "same", "f32")
    sup = B.cf_conv3d_fused_supported(desc, 0)
    assert sup & B.FUSED_FWD and sup & B.FUSED_BWD_WEIGHT and sup & B.FUSED_BWD_DATA and sup & B.FUSED_BWD_WEIGHT_DZ
    rng = np.random.default_rng(61)
    od = B.cf_conv3d_out_shape(desc)
    x = dev(rng.standard_normal((N, *dhw, CI)), "f32")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CI), "f32")
    b = torch.as_tensor(rng.standard_normal(CO) * 0.1, dtype=torch.float32, device="cuda")
    y = torch.full((N, *od, CO), float("nan"), device="cuda")
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.2, 0, y, None)
    y[..., 0] = 0.0  # exact zeros: the slope there is alpha
    dy = dev(rng.standard_normal((N, *od, CO)), "f32")
    ws = torch.empty(B.cf_conv3d_bwd_weight_fused_workspace_size(desc, 0), dtype=torch.uint8, device="cuda")
    dw = torch.full((k, k, k, CI, CO), float("nan"), device="cuda")
    db = torch.full((CO,), float("nan"), device="cuda")
    B.cf_conv3d_bwd_weight_fused(desc, x, dy, y, 0.2, 0, dw, db, ws)
    dw2, db2 = torch.full_like(dw, float("nan")), torch.full_like(db, float("nan"))
    dz = torch.full((N, *od, CO), float("nan"), device="cuda")
    B.cf_conv3d_bwd_weight_fused_dz(desc, x, dy, y, 0.2, 0, dw2, db2, dz, ws)
    dx = torch.full((N, *dhw, CI), float("nan"), device="cuda")
    B.cf_conv3d_bwd_data_fused(desc, dy, y, w, 0.2, 0, dx)
    torch.cuda.synchronize()
    assert torch.equal(dw, dw2) and torch.equal(db, db2)
    dzr, dbr = oracle.bias_lrelu_bwd(to_np(dy), to_np(y), 0.2)
    assert maxabs_err(to_np(dz), dzr) <= TOL["f32"]
    assert maxabs_err(to_np(db), dbr) <= TOL["f32"]
    assert maxabs_err(to_np(dw), oracle.conv3d_bwd_weight(to_np(x), dzr, k, stride=s)) <= TOL["f32"]
    assert maxabs_err(to_np(dx), oracle.conv3d_bwd_data(dzr, to_np(w), dhw, stride=s)) <= TOL["f32"]
