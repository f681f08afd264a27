"""GPU parity of the deep-layer implicit-GEMM kernels (bf16, 32 or more
channels on the contracted side) against the CPU oracle.

Every tile variant the library can choose is forced in turn through
CF_DIRECT_TILE, on shapes that span several row tiles with a ragged last one,
both strides of the stack, 2-, 3- and 4-wide kernels, column tiles of 32 and
64 and several column blocks.  Forward with the fused bias + leaky-ReLU
epilogue is checked together with its slope mask (bit-exact where the
pre-activation is decided, as in the fused-layer tests).
"""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_1808_04728_amd import binding as B
from tests._util import TOL, dev, maxabs_err, tdtype, to_np

pytestmark = pytest.mark.gpu

TILES = [None, "4,2,2", "2,2,2", "4,1,4", "2,1,4", "1,1,4"]

# N, (D, H, W), CI, CO, k, stride
CASES = [
    (2, (9, 8, 7), 64, 64, 3, 1),      # 1008 rows: several tiles, ragged tail
    (2, (10, 9, 8), 32, 64, 4, 2),     # the stride-2 layer shape; backward-data N = 32
    (1, (8, 8, 8), 64, 128, 2, 1),     # asymmetric SAME (0, 1), two column blocks
    (1, (6, 5, 7), 128, 128, 2, 1),
    (1, (5, 4, 6), 96, 64, 3, 1),      # three 32-channel k-steps per tap
    (3, (7, 6, 9), 32, 64, 4, 2),      # odd extents with stride 2: uneven parity classes
]


def ids(c):
    return "n%d_%dx%dx%d_c%d-%d_k%d_s%d" % (c[0], *c[1], *c[2:])


@pytest.fixture
def tile(request):
    t = request.param
    old = os.environ.get("CF_DIRECT_TILE")
    if t is None:
        os.environ.pop("CF_DIRECT_TILE", None)
    else:
        os.environ["CF_DIRECT_TILE"] = t
    yield t
    if old is None:
        os.environ.pop("CF_DIRECT_TILE", None)
    else:
        os.environ["CF_DIRECT_TILE"] = old


@pytest.mark.parametrize("tile", TILES, indirect=True, ids=lambda t: t or "auto")
@pytest.mark.parametrize("case", CASES, ids=ids)
def test_direct_fwd(case, tile):
    N, dhw, CI, CO, k, s = case
    rng = np.random.default_rng(31)
    x = dev(rng.standard_normal((N, *dhw, CI)), "bf16")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CI), "bf16")
    desc = B.make_desc(N, dhw, CI, CO, k, s, "same", "bf16")
    od = B.cf_conv3d_out_shape(desc)
    z = torch.full((N, *od, CO), float("nan"), dtype=tdtype("bf16"), device="cuda")
    B.cf_conv3d_fwd(desc, x, w, z)
    torch.cuda.synchronize()
    ref = oracle.conv3d_fwd(to_np(x), to_np(w), stride=s, pad="same")
    e = maxabs_err(to_np(z), ref)
    assert e <= TOL["bf16"], e


@pytest.mark.parametrize("tile", TILES, indirect=True, ids=lambda t: t or "auto")
@pytest.mark.parametrize("case", CASES, ids=ids)
def test_direct_bwd_data(case, tile):
    N, dhw, CI, CO, k, s = case
    rng = np.random.default_rng(32)
    desc = B.make_desc(N, dhw, CI, CO, k, s, "same", "bf16")
    od = B.cf_conv3d_out_shape(desc)
    dz = dev(rng.standard_normal((N, *od, CO)), "bf16")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CO), "bf16")
    dx = torch.full((N, *dhw, CI), float("nan"), dtype=tdtype("bf16"), device="cuda")
    B.cf_conv3d_bwd_data(desc, dz, w, dx)
    torch.cuda.synchronize()
    ref = oracle.conv3d_bwd_data(to_np(dz), to_np(w), dhw, stride=s, pad="same")
    e = maxabs_err(to_np(dx), ref)
    assert e <= TOL["bf16"], e


def unpack_mask(m, count):
    bits = np.unpackbits(m.detach().cpu().numpy().view(np.uint8), bitorder="little")
    return bits[:count].astype(bool)


@pytest.mark.parametrize("tile", [None, "4,2,2", "1,1,4"], indirect=True, ids=lambda t: t or "auto")
@pytest.mark.parametrize("case", [c for c in CASES if c[5] == 1], ids=ids)
def test_direct_fwd_bias_lrelu(case, tile):
    """conv + bias + leaky ReLU written once as y, with the 1-bit slope mask."""
    N, dhw, CI, CO, k, s = case
    desc = B.make_desc(N, dhw, CI, CO, k, s, "same", "bf16")
    assert B.cf_conv3d_fused_supported(desc, 0) & B.FUSED_FWD
    rng = np.random.default_rng(33)
    x = dev(rng.standard_normal((N, *dhw, CI)), "bf16")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) * np.sqrt(2.0 / (k ** 3 * CI)), "bf16")
    b = torch.as_tensor(rng.standard_normal(CO) * 0.1, dtype=torch.float32, device="cuda")
    od = B.cf_conv3d_out_shape(desc)
    y = torch.full((N, *od, CO), float("nan"), dtype=tdtype("bf16"), device="cuda")
    mask = torch.zeros(B.cf_conv3d_mask_bytes(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.01, 0, y, mask)
    y2 = torch.full_like(y, float("nan"))
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.01, 0, y2, None)
    torch.cuda.synchronize()
    z = oracle.conv3d_fwd(to_np(x), to_np(w))
    u = z + to_np(b)
    e = maxabs_err(to_np(y), oracle.bias_lrelu_fwd(z, to_np(b), 0.01))
    assert e <= TOL["bf16"], e
    assert torch.equal(y, y2)
    bits = unpack_mask(mask, u.size).reshape(u.shape)
    decided = np.abs(u) > 1e-5 * np.abs(u).max()
    assert np.array_equal(bits[decided], (u > 0)[decided])


def test_direct_delta_kernel_is_identity():
    """A delta weight at the padding tap copies x bit for bit (64 channels)."""
    C, k = 64, 3
    rng = np.random.default_rng(34)
    x = dev(rng.standard_normal((2, 9, 8, 7, C)), "bf16")
    _, pb = oracle.geometry(9, k, 1, "same")
    w = np.zeros((k, k, k, C, C))
    for c in range(C):
        w[pb, pb, pb, c, c] = 1.0
    desc = B.make_desc(2, (9, 8, 7), C, C, k, 1, "same", "bf16")
    z = torch.full_like(x, float("nan"))
    B.cf_conv3d_fwd(desc, x, dev(w, "bf16"), z)
    dx = torch.full_like(x, float("nan"))
    B.cf_conv3d_bwd_data(desc, x, dev(w, "bf16"), dx)
    torch.cuda.synchronize()
    assert torch.equal(z, x)
    assert torch.equal(dx, x)


@pytest.mark.parametrize("pf", ["1", "3"])
@pytest.mark.parametrize("tile", ["4,2,2", "1,1,4"], indirect=True)
@pytest.mark.parametrize("case", [CASES[0], CASES[1], CASES[4]], ids=ids)
def test_direct_prefetch_depths(case, tile, pf, monkeypatch):
    """The register ring at prefetch depths 1 and 3 (step counts that are not
    multiples of the ring size)."""
    monkeypatch.setenv("CF_DIRECT_PF", pf)
    N, dhw, CI, CO, k, s = case
    rng = np.random.default_rng(35)
    desc = B.make_desc(N, dhw, CI, CO, k, s, "same", "bf16")
    od = B.cf_conv3d_out_shape(desc)
    x = dev(rng.standard_normal((N, *dhw, CI)), "bf16")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CI), "bf16")
    dz = dev(rng.standard_normal((N, *od, CO)), "bf16")
    z = torch.full((N, *od, CO), float("nan"), dtype=tdtype("bf16"), device="cuda")
    dx = torch.full((N, *dhw, CI), float("nan"), dtype=tdtype("bf16"), device="cuda")
    B.cf_conv3d_fwd(desc, x, w, z)
    B.cf_conv3d_bwd_data(desc, dz, w, dx)
    torch.cuda.synchronize()
    e = maxabs_err(to_np(z), oracle.conv3d_fwd(to_np(x), to_np(w), stride=s, pad="same"))
    assert e <= TOL["bf16"], e
    e = maxabs_err(to_np(dx), oracle.conv3d_bwd_data(to_np(dz), to_np(w), dhw, stride=s, pad="same"))
    assert e <= TOL["bf16"], e


# the LDS-staged kernel: a 4- or 8-stage DMA ring run in whole rounds of
# k-steps, so step counts below one round and not a multiple of it are covered
LDS_CASES = CASES + [
    (1, (5, 6, 7), 32, 64, 1, 1),      # a single k-step (three padding steps); backward-data N = 32
    (2, (7, 9, 6), 64, 32, 3, 2),      # k = 3, stride 2: classes of 1, 2, 4 and 8 taps
    (2, (1, 6, 5), 32, 64, 3, 2),      # extent 1 along D: the odd-D classes are empty
]


@pytest.mark.parametrize("ring", ["4x1", "4x2", "8x1"])
@pytest.mark.parametrize("kern", ["lds128", "lds64"])
@pytest.mark.parametrize("case", LDS_CASES, ids=ids)
def test_lds_kernel(case, kern, ring, monkeypatch):
    """Forward, forward with the fused bias + leaky-ReLU epilogue and its mask,
    and backward-data through the LDS-staged kernel at both row tiles, both
    ring depths and one or two k-steps per stage."""
    stages, ksub = ring.split("x")
    monkeypatch.setenv("CF_DIRECT_KERNEL", kern)
    monkeypatch.setenv("CF_DIRECT_STAGES", stages)
    monkeypatch.setenv("CF_DIRECT_KSUB", ksub)
    N, dhw, CI, CO, k, s = case
    rng = np.random.default_rng(36)
    desc = B.make_desc(N, dhw, CI, CO, k, s, "same", "bf16")
    od = B.cf_conv3d_out_shape(desc)
    x = dev(rng.standard_normal((N, *dhw, CI)), "bf16")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CI), "bf16")
    dz = dev(rng.standard_normal((N, *od, CO)), "bf16")
    b = torch.as_tensor(rng.standard_normal(CO) * 0.1, dtype=torch.float32, device="cuda")
    z = torch.full((N, *od, CO), float("nan"), dtype=tdtype("bf16"), device="cuda")
    y = torch.full_like(z, float("nan"))
    dx = torch.full((N, *dhw, CI), float("nan"), dtype=tdtype("bf16"), device="cuda")
    B.cf_conv3d_fwd(desc, x, w, z)
    B.cf_conv3d_bwd_data(desc, dz, w, dx)
    fused = bool(B.cf_conv3d_fused_supported(desc, 0) & B.FUSED_FWD)
    if fused:
        mask = torch.zeros(B.cf_conv3d_mask_bytes(desc), dtype=torch.uint8, device="cuda")
        B.cf_conv3d_fwd_fused(desc, x, w, b, 0.01, 0, y, mask)
    torch.cuda.synchronize()
    zr = oracle.conv3d_fwd(to_np(x), to_np(w), stride=s, pad="same")
    e = maxabs_err(to_np(z), zr)
    assert e <= TOL["bf16"], e
    e = maxabs_err(to_np(dx), oracle.conv3d_bwd_data(to_np(dz), to_np(w), dhw, stride=s, pad="same"))
    assert e <= TOL["bf16"], e
    if fused:
        e = maxabs_err(to_np(y), oracle.bias_lrelu_fwd(zr, to_np(b), 0.01))
        assert e <= TOL["bf16"], e
        u = zr + to_np(b)
        bits = unpack_mask(mask, u.size).reshape(u.shape)
        decided = np.abs(u) > 1e-5 * np.abs(u).max()
        assert np.array_equal(bits[decided], (u > 0)[decided])


@pytest.mark.parametrize("case", [CASES[1], CASES[4], LDS_CASES[-2]], ids=ids)
def test_lds_tiles_agree_bitwise(case, monkeypatch):
    """Both row tiles of the LDS-staged kernel accumulate each output over the
    same k-steps in the same order with the same MFMA: identical bits."""
    N, dhw, CI, CO, k, s = case
    rng = np.random.default_rng(37)
    desc = B.make_desc(N, dhw, CI, CO, k, s, "same", "bf16")
    od = B.cf_conv3d_out_shape(desc)
    x = dev(rng.standard_normal((N, *dhw, CI)), "bf16")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CI), "bf16")
    dz = dev(rng.standard_normal((N, *od, CO)), "bf16")
    outs = {}
    for kk in ("lds128", "lds64"):
        monkeypatch.setenv("CF_DIRECT_KERNEL", kk)
        z = torch.empty((N, *od, CO), dtype=tdtype("bf16"), device="cuda")
        dx = torch.empty((N, *dhw, CI), dtype=tdtype("bf16"), device="cuda")
        B.cf_conv3d_fwd(desc, x, w, z)
        B.cf_conv3d_bwd_data(desc, dz, w, dx)
        outs[kk] = (z, dx)
    torch.cuda.synchronize()
    assert torch.equal(outs["lds128"][0], outs["lds64"][0])
    assert torch.equal(outs["lds128"][1], outs["lds64"][1])


# deep-layer weight gradient: N, (D, H, W), CI, CO, k, stride, pad
WG_CASES = [
    (2, (10, 9, 8), 32, 64, 4, 2, "same"),   # stride-2 layer shape: two taps per 64-row block
    (1, (7, 6, 8), 64, 64, 3, 1, "same"),    # 27 taps: ragged last row block
    (1, (6, 5, 7), 64, 128, 2, 1, "same"),   # 128-wide column blocks (two waves per dz tile)
    (1, (5, 6, 7), 40, 192, 3, 1, "same"),   # 40 channels: row blocks straddle taps; three column blocks
    (1, (3, 2, 4), 64, 64, 2, 1, "same"),    # 24 voxels: one partial k-step
    (2, (9, 8, 7), 64, 64, 3, 2, "valid"),   # VALID, stride 2
    (2, (12, 12, 12), 64, 64, 3, 1, "same"), # 3456 voxels: many K slices
]


def wg_ids(c):
    return "n%d_%dx%dx%d_c%d-%d_k%d_s%d_%s" % (c[0], *c[1], *c[2:])


@pytest.mark.parametrize("wgs", [None, "1", "100000"], ids=["auto", "one_slice", "max_slices"])
@pytest.mark.parametrize("case", WG_CASES, ids=wg_ids)
def test_direct_wgrad(case, wgs, monkeypatch):
    """dW through the LDS-staged K-split kernel (slice counts from one to the
    most the 8-step minimum allows) against the oracle; repeat calls are
    bitwise identical."""
    if wgs is not None:
        monkeypatch.setenv("CF_DWGRAD_WGS", wgs)
    N, dhw, CI, CO, k, s, pad = case
    rng = np.random.default_rng(38)
    desc = B.make_desc(N, dhw, CI, CO, k, s, pad, "bf16")
    od = B.cf_conv3d_out_shape(desc)
    x = dev(rng.standard_normal((N, *dhw, CI)), "bf16")
    dz = dev(rng.standard_normal((N, *od, CO)), "bf16")
    dw = torch.full((k, k, k, CI, CO), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(16, B.cf_conv3d_bwd_weight_workspace_size(desc)), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_bwd_weight(desc, x, dz, dw, ws)
    dw2 = torch.full_like(dw, float("nan"))
    B.cf_conv3d_bwd_weight(desc, x, dz, dw2, ws)
    torch.cuda.synchronize()
    ref = oracle.conv3d_bwd_weight(to_np(x), to_np(dz), k, stride=s, pad=pad)
    # bf16 products are exact in fp32: only the fp32 accumulation order differs
    e = maxabs_err(to_np(dw), ref)
    assert e <= 1e-4, e
    assert torch.equal(dw, dw2)


@pytest.mark.parametrize("case", [WG_CASES[0], WG_CASES[3]], ids=wg_ids)
def test_direct_wgrad_matches_generic(case, monkeypatch):
    """The deep-layer kernel and the generic tiled kernel agree to fp32
    rounding (different summation orders)."""
    N, dhw, CI, CO, k, s, pad = case
    rng = np.random.default_rng(39)
    desc = B.make_desc(N, dhw, CI, CO, k, s, pad, "bf16")
    od = B.cf_conv3d_out_shape(desc)
    x = dev(rng.standard_normal((N, *dhw, CI)), "bf16")
    dz = dev(rng.standard_normal((N, *od, CO)), "bf16")
    out = []
    for kern in (None, "igemm"):
        if kern:
            monkeypatch.setenv("CF_WGRAD_KERNEL", kern)
        dw = torch.empty((k, k, k, CI, CO), dtype=torch.float32, device="cuda")
        ws = torch.empty(max(16, B.cf_conv3d_bwd_weight_workspace_size(desc)), dtype=torch.uint8, device="cuda")
        B.cf_conv3d_bwd_weight(desc, x, dz, dw, ws)
        torch.cuda.synchronize()
        out.append(to_np(dw))
    scale = np.abs(out[1]).max()
    assert np.abs(out[0] - out[1]).max() <= 1e-5 * scale
