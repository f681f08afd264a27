"""GPU parity of the fused bf16 deep-layer entry points against the CPU oracle.

Pooled layers (the stride-2 32 -> 64 layer of the stack and its relatives):
the forward writes the 2^3-pooled activation and the slope mask; backward-
weights (dW, db) and backward-data (dx) take the pooled-output gradient and a
mask and form dz as they load it.  Unpooled layers: backward-weights and
backward-data take (dy, y).  The oracle forms dz in fp64 from the same inputs
(dz = pool_bwd(g) * (bit ? 1 : alpha), or dy * (y > 0 ? 1 : alpha)) and applies
the definitions of Section III-C; the GPU rounds dz to bf16 before its MFMAs,
which the bf16 tolerance covers.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_04728_amd import binding as B
from tests._util import TOL, dev, maxabs_err, to_np

pytestmark = pytest.mark.gpu

# N, (D,H,W), CI, CO, k, stride
POOLED = [
    (2, (12, 10, 14), 32, 64, 4, 2),     # stride 2, ragged 16-wide bricks
    (1, (13, 11, 18), 32, 64, 4, 2),     # odd conv-output extents: floor pooling
    (1, (12, 8, 80), 32, 64, 4, 2),      # 32-wide bricks, ragged last one
    (2, (7, 8, 9), 64, 64, 3, 1),        # stride 1, odd extents
    (1, (6, 6, 20), 64, 128, 2, 1),      # two column blocks
]


def ids(c):
    return "n%d_%dx%dx%d_c%d-%d_k%d_s%d" % (c[0], *c[1], *c[2:])


def _unpack(mask, count, shape):
    return np.unpackbits(mask.cpu().numpy(), bitorder="little")[:count].astype(bool).reshape(shape)


@pytest.mark.parametrize("variant", ["default", "stages8", "ksub1", "lds64", "lds128", "lds64_stages8"])
@pytest.mark.parametrize("case", POOLED, ids=ids)
def test_bf16_pooled_deep_layer_fused(case, variant, monkeypatch):
    """Fused pooled forward (pooled output + slope mask), fused backward-weights
    (dW, db) and fused backward-data (dx) from a pooled gradient and a mask;
    the variants force the LDS-staged kernel's ring shapes and, for the
    backward-data, the LDS-staged kernel instead of the register kernel."""
    if "stages8" in variant:
        monkeypatch.setenv("CF_DIRECT_STAGES", "8")
    if variant == "ksub1":
        monkeypatch.setenv("CF_DIRECT_KSUB", "1")
    if variant.startswith("lds"):
        monkeypatch.setenv("CF_DIRECT_KERNEL", variant.split("_")[0])
    N, dhw, CI, CO, k, s = case
    desc = B.make_desc(N, dhw, CI, CO, k, s, "same", "bf16")
    sup = B.cf_conv3d_fused_supported(desc, B.CF_FUSE_POOL2)
    assert sup & B.FUSED_FWD and sup & B.FUSED_BWD_WEIGHT and sup & B.FUSED_BWD_DATA
    assert not sup & B.FUSED_BWD_WEIGHT_DZ
    rng = np.random.default_rng(71)
    od = B.cf_conv3d_out_shape(desc)
    pdhw = tuple(t // 2 for t in od)
    x = dev(np.log1p(rng.poisson(np.exp(rng.standard_normal((N, *dhw, CI))))), "bf16")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CI), "bf16")
    bh = rng.standard_normal(CO) * 0.1
    b = torch.as_tensor(bh, dtype=torch.float32, device="cuda")
    out = torch.full((N, *pdhw, CO), float("nan"), dtype=torch.bfloat16, device="cuda")
    mask = torch.zeros(B.cf_conv3d_mask_bytes(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.01, B.CF_FUSE_POOL2, out, mask)
    g = dev(rng.standard_normal((N, *pdhw, CO)), "bf16")
    mask_r = torch.as_tensor(rng.integers(0, 256, mask.numel(), dtype=np.uint8), device="cuda")
    ws = torch.empty(B.cf_conv3d_bwd_weight_fused_workspace_size(desc, B.CF_FUSE_POOL2), dtype=torch.uint8,
                     device="cuda")
    dw = torch.full((k, k, k, CI, CO), float("nan"), device="cuda")
    db = torch.full((CO,), float("nan"), device="cuda")
    B.cf_conv3d_bwd_weight_fused(desc, x, g, mask_r, 0.2, B.CF_FUSE_POOL2, dw, db, ws)
    dw2, db2 = torch.full_like(dw, float("nan")), torch.full_like(db, float("nan"))
    B.cf_conv3d_bwd_weight_fused(desc, x, g, mask_r, 0.2, B.CF_FUSE_POOL2, dw2, db2, ws)
    dx = torch.full((N, *dhw, CI), float("nan"), dtype=torch.bfloat16, device="cuda")
    B.cf_conv3d_bwd_data_fused(desc, g, mask_r, w, 0.2, B.CF_FUSE_POOL2, dx)
    torch.cuda.synchronize()
    zr = oracle.conv3d_fwd(to_np(x), to_np(w), stride=s)
    u = zr + bh
    pr = oracle.avgpool3d_fwd(oracle.bias_lrelu_fwd(zr, bh, 0.01))
    assert maxabs_err(to_np(out), pr) <= TOL["bf16"]
    bits = _unpack(mask, u.size, u.shape)
    decided = np.abs(u) > 1e-5 * np.abs(u).max()
    assert np.array_equal(bits[decided], (u > 0)[decided])
    assert decided.mean() > 0.99
    # the gradient sums are fixed-order: a second call gives the same bits
    assert torch.equal(dw, dw2) and torch.equal(db, db2)
    rb = _unpack(mask_r, u.size, u.shape)
    dzr = oracle.avgpool3d_bwd(to_np(g), od) * np.where(rb, 1.0, 0.2)
    assert maxabs_err(to_np(dw), oracle.conv3d_bwd_weight(to_np(x), dzr, k, stride=s)) <= TOL["bf16"]
    assert maxabs_err(to_np(db), dzr.reshape(-1, CO).sum(0)) <= TOL["bf16"]
    assert maxabs_err(to_np(dx), oracle.conv3d_bwd_data(dzr, to_np(w), dhw, stride=s)) <= TOL["bf16"]


# unpooled bf16 layers, backward from (dy, y): N, (D,H,W), CI, CO, k, stride
DYY = [
    (1, (8, 8, 8), 64, 64, 3, 1),        # the stack's 8^3 layers
    (2, (5, 6, 7), 64, 128, 2, 1),
    (1, (9, 7, 8), 128, 128, 2, 1),
    (2, (12, 10, 14), 32, 64, 4, 2),     # stride 2: every backward-data class
    (3, (9, 10, 11), 64, 64, 3, 1),      # ragged row tiles
]


@pytest.mark.parametrize("tile", ["auto", "4,1,4", "2,2,2", "1,1,4"])
@pytest.mark.parametrize("case", DYY, ids=ids)
def test_bf16_unpooled_fused_backward(case, tile, monkeypatch):
    """dW, db and dx from (dy, y) with dz = dy * (y > 0 ? 1 : alpha): y comes
    from the fused forward of the same layer, with a channel of exact zeros
    (slope alpha there)."""
    if tile != "auto":
        monkeypatch.setenv("CF_DIRECT_TILE", tile)
    N, dhw, CI, CO, k, s = case
    desc = B.make_desc(N, dhw, CI, CO, k, s, "same", "bf16")
    sup = B.cf_conv3d_fused_supported(desc, 0)
    assert sup & B.FUSED_FWD and sup & B.FUSED_BWD_WEIGHT and sup & B.FUSED_BWD_DATA
    rng = np.random.default_rng(81)
    od = B.cf_conv3d_out_shape(desc)
    x = dev(rng.standard_normal((N, *dhw, CI)), "bf16")
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CI), "bf16")
    b = torch.as_tensor(rng.standard_normal(CO) * 0.1, dtype=torch.float32, device="cuda")
    y = torch.full((N, *od, CO), float("nan"), dtype=torch.bfloat16, device="cuda")
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.2, 0, y, None)
    y[..., 0] = 0.0  # exact zeros: the slope there is alpha
    y[..., 1] = -0.0
    dy = dev(rng.standard_normal((N, *od, CO)), "bf16")
    ws = torch.empty(B.cf_conv3d_bwd_weight_fused_workspace_size(desc, 0), dtype=torch.uint8, device="cuda")
    dw = torch.full((k, k, k, CI, CO), float("nan"), device="cuda")
    db = torch.full((CO,), float("nan"), device="cuda")
    B.cf_conv3d_bwd_weight_fused(desc, x, dy, y, 0.2, 0, dw, db, ws)
    dx = torch.full((N, *dhw, CI), float("nan"), dtype=torch.bfloat16, device="cuda")
    B.cf_conv3d_bwd_data_fused(desc, dy, y, w, 0.2, 0, dx)
    torch.cuda.synchronize()
    dzr, dbr = oracle.bias_lrelu_bwd(to_np(dy), to_np(y), 0.2)
    assert maxabs_err(to_np(db), dbr) <= TOL["bf16"]
    assert maxabs_err(to_np(dw), oracle.conv3d_bwd_weight(to_np(x), dzr, k, stride=s)) <= TOL["bf16"]
    assert maxabs_err(to_np(dx), oracle.conv3d_bwd_data(dzr, to_np(w), dhw, stride=s)) <= TOL["bf16"]


# n, (d, h, w) conv-output extent, c
POOL_DZ = [
    (2, (16, 16, 16), 64),     # the stride-2 layer's output at 128^3 / 2 samples
    (1, (7, 9, 11), 64),       # odd extents: voxels outside every window get zero
    (3, (4, 6, 8), 32),
    (1, (6, 4, 10), 128),
]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("case", POOL_DZ, ids=lambda c: "n%d_%dx%dx%d_c%d" % (c[0], *c[1], c[2]))
def test_pool_lrelu_bwd(case, dt):
    """One-pass dz and db of a pooled layer from the pooled gradient and the
    slope mask, against the oracle's pool adjoint times the slope; the deferred
    form gives the same bits."""
    n, dhw, c = case
    rng = np.random.default_rng(91)
    pd = tuple(t // 2 for t in dhw)
    g = dev(rng.standard_normal((n, *pd, c)), dt)
    nel = n * dhw[0] * dhw[1] * dhw[2] * c
    mask = torch.as_tensor(rng.integers(0, 256, (nel + 31) // 32 * 4, dtype=np.uint8), device="cuda")
    ws = torch.empty(B.cf_avgpool3d_lrelu_bwd_workspace_size(n, *dhw, c), dtype=torch.uint8, device="cuda")
    dz = torch.full((n, *dhw, c), float("nan"), dtype=g.dtype, device="cuda")
    db = torch.full((c,), float("nan"), device="cuda")
    B.cf_avgpool3d_lrelu_bwd(n, *dhw, c, dt, g, mask, 0.2, dz, db, ws)
    dz2, db2 = torch.full_like(dz, float("nan")), torch.full_like(db, float("nan"))
    pend = B.cf_avgpool3d_lrelu_bwd_deferred(n, *dhw, c, dt, g, mask, 0.2, dz2, db2, ws)
    B.cf_reduce_partials(pend)
    torch.cuda.synchronize()
    bits = _unpack(mask, nel, (n, *dhw, c))
    dzr = oracle.avgpool3d_bwd(to_np(g), dhw) * np.where(bits, 1.0, 0.2)
    assert maxabs_err(to_np(dz), dzr) <= TOL[dt]
    assert maxabs_err(to_np(db), dzr.reshape(-1, c).sum(0)) <= TOL["f32"]
    assert torch.equal(dz, dz2) and torch.equal(db, db2)


@pytest.mark.parametrize("dz_pass", [True, False])
def test_bf16_stack_pooled_backward_forms(dz_pass):
    """The 64^3 stack at batch 2 in bf16 with the stride-2 layer's backward
    through the one-pass dz (True) or the fused kernels (False): forward and
    every weight and bias gradient against the oracle chain, teacher-forced at
    the stride-2 layer (its dz from the GPU's own pooled gradient and mask)."""
    from paper_1808_04728_amd import inputs
    from paper_1808_04728_amd.stack import ConvStack
    name = "stack_64c_b1_f32"
    wl = inputs.WORKLOADS[name]
    st = ConvStack(wl["layers"], 64, 2, "bf16", inputs.ALPHA, "cuda", pooled_dz_pass=dz_pass)
    L3 = st.L[2]
    assert L3["fused"] and L3["dz_pass"] == dz_pass
    ws, bs = inputs.make_weights(name)
    rng = np.random.default_rng(93)
    bs = [rng.standard_normal(b.shape) * 0.1 for b in bs]
    st.set_params(ws, bs)
    st.set_input(np.log1p(rng.poisson(np.exp(rng.standard_normal((2, 64, 64, 64, 1))))))
    out = st.forward()
    dout = dev(rng.standard_normal(tuple(out.shape)), "bf16")
    st.backward(dout)
    torch.cuda.synchronize()
    # layer 3 teacher-forced: its input, weights, bias, the gradient of its pooled
    # output and its mask as the GPU held them
    x3 = to_np(st.layer_input(2))
    w3 = to_np(L3["w"])
    g3 = to_np(st.L[3]["dx"])
    od = L3["out_dhw"]
    bits = _unpack(L3["mask"], 2 * od[0] * od[1] * od[2] * 64, (2, *od, 64))
    dzr = oracle.avgpool3d_bwd(g3, od) * np.where(bits, 1.0, inputs.ALPHA)
    assert maxabs_err(to_np(L3["dw"]), oracle.conv3d_bwd_weight(x3, dzr, 4, stride=2)) <= TOL["bf16"]
    assert maxabs_err(to_np(L3["db"]), dzr.reshape(-1, 64).sum(0)) <= TOL["bf16"]
    assert maxabs_err(to_np(L3["dx"]), oracle.conv3d_bwd_data(dzr, w3, x3.shape[1:4], stride=2)) <= TOL["bf16"]
    # its forward: pooled output and mask from the same x, W, b
    zr = oracle.conv3d_fwd(x3, w3, stride=2)
    u = zr + to_np(L3["b"])
    assert maxabs_err(to_np(L3["p"]), oracle.avgpool3d_fwd(oracle.bias_lrelu_fwd(zr, to_np(L3["b"]),
                                                                                  inputs.ALPHA))) <= TOL["bf16"]
    decided = np.abs(u) > 1e-5 * np.abs(u).max()
    assert np.array_equal(bits[decided], (u > 0)[decided])
