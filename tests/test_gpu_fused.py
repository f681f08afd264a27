"""GPU parity of the fused layer entry points against the CPU oracle.

Forward: pooled output of conv -> bias + leaky ReLU -> 2^3 pool, and the
1-bit slope mask, from the same x, W, b the kernel saw.  The mask is compared
bit-exactly wherever the pre-activation is decided (|u| above a small
fraction of max|u| in the fp64 oracle); at |u| near 0 fp32 and fp64 may
round to different signs, and both answers are valid.

Backward-weights: teacher-forced from a random pooled-output gradient and a
random mask; the oracle forms dz = pool_bwd(g) * slope(mask) in fp64 and
applies the weight-gradient definition and db = sum dz.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_04728_amd import binding as B
from tests._util import TOL, dev, maxabs_err, tdtype, to_np

pytestmark = pytest.mark.gpu

# N, (D,H,W), CI, CO, k
FWD_CASES = [
    (1, (32, 32, 32), 1, 16, 3),     # the first CosmoFlow layer, single-sample size
    (2, (13, 12, 11), 1, 16, 3),     # odd extents: ragged tiles, floor pooling
    (1, (10, 18, 40), 4, 16, 3),     # four input channels
    (1, (9, 8, 34), 1, 32, 3),       # 32 output channels
    (1, (8, 9, 10), 2, 16, 2),       # even kernel, asymmetric SAME
    (1, (8, 8, 36), 1, 16, 4),
    (1, (16, 12, 64), 16, 32, 4),    # the second CosmoFlow layer: 16 -> 32, 4^3
    (2, (9, 7, 33), 16, 32, 4),      # ragged tiles in every dimension
    (1, (10, 10, 40), 16, 32, 3),
    (1, (10, 10, 10), 16, 32, 2),
    (2, (16, 12, 40), 1, 16, 3),     # several 32-wide tiles, overhang in w
    (1, (9, 7, 16), 1, 16, 3),       # odd extents: floor pooling, ragged tiles in d and h
    (3, (6, 10, 8), 1, 16, 3),       # rows of one 16-byte vector
    (1, (10, 6, 24), 1, 16, 2),      # 2^3 kernel, asymmetric SAME
]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("case", FWD_CASES, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d" % (c[0], *c[1], *c[2:]))
def test_fused_fwd_no_pool(case, dt):
    """conv + bias + leaky ReLU in one kernel (y written once, optional mask)."""
    N, dhw, CI, CO, k = case
    desc = B.make_desc(N, dhw, CI, CO, k, 1, "same", dt)
    if not B.cf_conv3d_fused_supported(desc, 0) & B.FUSED_FWD:
        pytest.skip("no fused forward kernel without pooling for this shape")
    rng = np.random.default_rng(14)
    x = dev(rng.standard_normal((N, *dhw, CI)), dt)
    w = dev(rng.standard_normal((k, k, k, CI, CO)) * np.sqrt(2.0 / (k ** 3 * CI)), dt)
    b = torch.as_tensor(rng.standard_normal(CO) * 0.1, dtype=torch.float32, device="cuda")
    od = B.cf_conv3d_out_shape(desc)
    y = torch.full((N, *od, CO), float("nan"), dtype=tdtype(dt), device="cuda")
    mask = torch.zeros(B.cf_conv3d_mask_bytes(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.2, 0, y, mask)
    y2 = torch.full_like(y, float("nan"))
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.2, 0, y2, None)
    torch.cuda.synchronize()
    z = oracle.conv3d_fwd(to_np(x), to_np(w))
    u = z + to_np(b)
    e = maxabs_err(to_np(y), oracle.bias_lrelu_fwd(z, to_np(b), 0.2))
    assert e <= TOL[dt], e
    assert torch.equal(y, y2)
    bits = unpack_mask(mask, u.size).reshape(u.shape)
    decided = np.abs(u) > 1e-5 * np.abs(u).max()
    assert np.array_equal(bits[decided], (u > 0)[decided])


def unpack_mask(m, count):
    bits = np.unpackbits(m.detach().cpu().numpy().view(np.uint8), bitorder="little")
    return bits[:count].astype(bool)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("case", FWD_CASES, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d" % (c[0], *c[1], *c[2:]))
def test_fused_fwd(case, dt):
    N, dhw, CI, CO, k = case
    desc = B.make_desc(N, dhw, CI, CO, k, 1, "same", dt)
    if not B.cf_conv3d_fused_supported(desc) & B.FUSED_FWD:
        pytest.skip("no fused forward kernel for this shape")
    rng = np.random.default_rng(11)
    x = dev(np.log1p(rng.poisson(np.exp(rng.standard_normal((N, *dhw, CI))))), dt)  # many exact zeros
    w = dev(rng.standard_normal((k, k, k, CI, CO)) * np.sqrt(2.0 / (k ** 3 * CI)), dt)
    b = torch.as_tensor(rng.standard_normal(CO) * 0.1, dtype=torch.float32, device="cuda")
    alpha = 0.01
    od = B.cf_conv3d_out_shape(desc)
    pshape = (N,) + tuple(t // 2 for t in od) + (CO,)
    out = torch.full(pshape, float("nan"), dtype=tdtype(dt), device="cuda")
    mask = torch.zeros(B.cf_conv3d_mask_bytes(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_fwd_fused(desc, x, w, b, alpha, B.CF_FUSE_POOL2, out, mask)
    torch.cuda.synchronize()
    z = oracle.conv3d_fwd(to_np(x), to_np(w))
    u = z + to_np(b)
    y = oracle.bias_lrelu_fwd(z, to_np(b), alpha)
    p = oracle.avgpool3d_fwd(y)
    e = maxabs_err(to_np(out), p)
    assert e <= TOL[dt], e
    bits = unpack_mask(mask, u.size).reshape(u.shape)
    decided = np.abs(u) > 1e-5 * np.abs(u).max()
    assert np.array_equal(bits[decided], (u > 0)[decided])
    assert decided.mean() > 0.99


# bf16 first layer with even output extents runs on the voxel-pair kernel:
# SAME and VALID leading pads, widths that end inside a 16-voxel segment, two
# 128-wide w tiles, partial d and h tiles, and alpha 0.2
PAIR_CASES = [
    (1, (8, 8, 128), "valid", 0.01),    # out (6, 6, 126): the paper's first-layer width
    (1, (6, 10, 136), "same", 0.2),     # out (6, 10, 136): a second w tile 8 voxels wide
    (2, (12, 6, 24), "valid", 0.01),    # out (10, 4, 22)
    (1, (4, 4, 8), "same", 0.01),       # one 8-voxel segment
    (1, (10, 18, 64), "same", 0.01),    # h tiles 8 + 8 + 2, d tiles 4 + 4 + 2
]


@pytest.mark.parametrize("case", PAIR_CASES, ids=lambda c: "n%d_%dx%dx%d_%s_a%g" % (c[0], *c[1], c[2], c[3]))
def test_fused_fwd_first_layer_pairs(case):
    N, dhw, pad, alpha = case
    dt = "bf16"
    desc = B.make_desc(N, dhw, 1, 16, 3, 1, pad, dt)
    assert B.cf_conv3d_fused_supported(desc) & B.FUSED_FWD
    rng = np.random.default_rng(17)
    x = dev(np.log1p(rng.poisson(np.exp(rng.standard_normal((N, *dhw, 1))))), dt)  # many exact zeros
    w = dev(rng.standard_normal((3, 3, 3, 1, 16)) * np.sqrt(2.0 / 27), dt)
    b = torch.as_tensor(rng.standard_normal(16) * 0.1, dtype=torch.float32, device="cuda")
    od = B.cf_conv3d_out_shape(desc)
    assert all(t % 2 == 0 for t in od)
    out = torch.full((N,) + tuple(t // 2 for t in od) + (16,), float("nan"), dtype=tdtype(dt), device="cuda")
    mask = torch.zeros(B.cf_conv3d_mask_bytes(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_fwd_fused(desc, x, w, b, alpha, B.CF_FUSE_POOL2, out, mask)
    torch.cuda.synchronize()
    z = oracle.conv3d_fwd(to_np(x), to_np(w), pad=pad)
    u = z + to_np(b)
    p = oracle.avgpool3d_fwd(oracle.bias_lrelu_fwd(z, to_np(b), alpha))
    e = maxabs_err(to_np(out), p)
    assert e <= TOL[dt], e
    bits = unpack_mask(mask, u.size).reshape(u.shape)
    decided = np.abs(u) > 1e-5 * np.abs(u).max()
    assert np.array_equal(bits[decided], (u > 0)[decided])
    assert decided.mean() > 0.99


# more tiles than the persistent kernels start workgroups: every workgroup loops
# over several tiles, the next tile's halo arriving during the current tile's MFMAs
MULTI_CASES = [
    (3, (64, 64, 48), 16, 32, 4),    # 16 -> 32, 4^3: 768 tiles, ragged last w tile
    (2, (64, 64, 64), 1, 16, 3),     # the first layer
]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("case", MULTI_CASES, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d" % (c[0], *c[1], *c[2:]))
def test_fused_fwd_multitile_sampled(case, dt):
    """Pooled values at sampled windows and the slope mask at sampled
    conv-output points, each evaluated by the oracle one by one."""
    N, dhw, CI, CO, k = case
    desc = B.make_desc(N, dhw, CI, CO, k, 1, "same", dt)
    if not B.cf_conv3d_fused_supported(desc) & B.FUSED_FWD:
        pytest.skip("no fused forward kernel for this shape")
    rng = np.random.default_rng(15)
    xs = np.log1p(rng.poisson(np.exp(rng.standard_normal((N, *dhw, CI)))))
    x = dev(xs, dt)
    w = dev(rng.standard_normal((k, k, k, CI, CO)) * np.sqrt(2.0 / (k ** 3 * CI)), dt)
    bh = rng.standard_normal(CO) * 0.1
    b = torch.as_tensor(bh, dtype=torch.float32, device="cuda")
    alpha = 0.01
    od = B.cf_conv3d_out_shape(desc)
    pshape = (N,) + tuple(t // 2 for t in od) + (CO,)
    out = torch.full(pshape, float("nan"), dtype=tdtype(dt), device="cuda")
    mask = torch.zeros(B.cf_conv3d_mask_bytes(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_fwd_fused(desc, x, w, b, alpha, B.CF_FUSE_POOL2, out, mask)
    torch.cuda.synchronize()
    xh, wh, bf = to_np(x), to_np(w), to_np(b)
    outh = to_np(out)
    pidx = np.stack([rng.integers(0, t, 256) for t in pshape], 1)
    ref, win = [], []
    for n, pd, ph, pw, c in pidx:
        pts = [(n, 2 * pd + u, 2 * ph + v, 2 * pw + t, c) for u in (0, 1) for v in (0, 1) for t in (0, 1)]
        win += pts
        u8 = oracle.conv3d_fwd_points(xh, wh, pts) + bf[c]
        ref.append(np.mean(np.where(u8 > 0, u8, alpha * u8)))
    e = maxabs_err(outh[tuple(pidx.T)], np.asarray(ref))
    assert e <= TOL[dt], e
    pts = np.concatenate([np.asarray(win), np.stack([rng.integers(0, t, 4096) for t in (N, *od, CO)], 1)])
    u = oracle.conv3d_fwd_points(xh, wh, pts) + bf[pts[:, 4]]
    bits = unpack_mask(mask, N * od[0] * od[1] * od[2] * CO).reshape((N, *od, CO))[tuple(pts.T)]
    decided = np.abs(u) > 1e-5 * np.abs(u).max()
    assert decided.mean() > 0.95
    assert np.array_equal(bits[decided], (u > 0)[decided])


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("case", FWD_CASES, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d" % (c[0], *c[1], *c[2:]))
def test_fused_bwd_weight(case, dt):
    N, dhw, CI, CO, k = case
    desc = B.make_desc(N, dhw, CI, CO, k, 1, "same", dt)
    if not B.cf_conv3d_fused_supported(desc) & B.FUSED_BWD_WEIGHT:
        pytest.skip("no fused backward-weights kernel for this shape")
    rng = np.random.default_rng(12)
    od = B.cf_conv3d_out_shape(desc)
    pdhw = tuple(t // 2 for t in od)
    x = dev(rng.standard_normal((N, *dhw, CI)), dt)
    g = dev(rng.standard_normal((N, *pdhw, CO)), dt)
    nbits = N * od[0] * od[1] * od[2] * CO
    mbytes = B.cf_conv3d_mask_bytes(desc)
    mask_np = rng.integers(0, 256, mbytes, dtype=np.uint8)
    mask = torch.as_tensor(mask_np, device="cuda")
    alpha = 0.2
    dw = torch.full((k, k, k, CI, CO), float("nan"), dtype=torch.float32, device="cuda")
    db = torch.full((CO,), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(B.cf_conv3d_bwd_weight_fused_workspace_size(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_bwd_weight_fused(desc, x, g, mask, alpha, B.CF_FUSE_POOL2, dw, db, ws)
    torch.cuda.synchronize()
    bits = np.unpackbits(mask_np, bitorder="little")[:nbits].astype(bool).reshape((N, *od, CO))
    dy = oracle.avgpool3d_bwd(to_np(g), od)
    dz = dy * np.where(bits, 1.0, alpha)
    dw_ref = oracle.conv3d_bwd_weight(to_np(x), dz, k)
    db_ref = dz.reshape(-1, CO).sum(0)
    e = maxabs_err(to_np(dw), dw_ref)
    assert e <= TOL[dt], e
    e = maxabs_err(to_np(db), db_ref)
    assert e <= TOL["f32"], e
    # bitwise reproducible
    dw2 = torch.empty_like(dw)
    db2 = torch.empty_like(db)
    B.cf_conv3d_bwd_weight_fused(desc, x, g, mask, alpha, B.CF_FUSE_POOL2, dw2, db2, ws)
    torch.cuda.synchronize()
    assert torch.equal(dw, dw2) and torch.equal(db, db2)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_fused_matches_unfused_composition(dt):
    """The fused forward + backward-weights equal the unfused ABI composition
    (conv, bias+lReLU, pool; pool bwd, lReLU bwd, wgrad) to the path tolerance."""
    N, dhw, CI, CO, k = 1, (16, 16, 32), 1, 16, 3
    desc = B.make_desc(N, dhw, CI, CO, k, 1, "same", dt)
    rng = np.random.default_rng(13)
    x = dev(rng.standard_normal((N, *dhw, CI)), dt)
    w = dev(rng.standard_normal((k, k, k, CI, CO)) * 0.3, dt)
    b = torch.as_tensor(rng.standard_normal(CO) * 0.1, dtype=torch.float32, device="cuda")
    od = B.cf_conv3d_out_shape(desc)
    nvox = N * od[0] * od[1] * od[2]
    # unfused
    z = torch.empty((N, *od, CO), dtype=tdtype(dt), device="cuda")
    B.cf_conv3d_fwd(desc, x, w, z)
    B.cf_bias_lrelu_fwd(nvox, CO, dt, z, b, 0.01, z)
    p = torch.empty((N, od[0] // 2, od[1] // 2, od[2] // 2, CO), dtype=tdtype(dt), device="cuda")
    B.cf_avgpool3d_fwd(N, *od, CO, 2, 2, dt, z, p)
    # fused
    pf = torch.empty_like(p)
    mask = torch.empty(B.cf_conv3d_mask_bytes(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_fwd_fused(desc, x, w, b, 0.01, B.CF_FUSE_POOL2, pf, mask)
    torch.cuda.synchronize()
    e = maxabs_err(to_np(pf), to_np(p))
    assert e <= TOL[dt], e
    g = dev(rng.standard_normal(p.shape), dt)
    dy = torch.empty_like(z)
    B.cf_avgpool3d_bwd(N, *od, CO, 2, 2, dt, g, dy)
    dz = torch.empty_like(z)
    db = torch.empty(CO, device="cuda")
    wsb = torch.empty(B.cf_bias_lrelu_bwd_workspace_size(nvox, CO), dtype=torch.uint8, device="cuda")
    B.cf_bias_lrelu_bwd(nvox, CO, dt, dy, z, 0.01, dz, db, wsb)
    dw = torch.empty((k, k, k, CI, CO), device="cuda")
    wsw = torch.empty(B.cf_conv3d_bwd_weight_workspace_size(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_bwd_weight(desc, x, dz, dw, wsw)
    dwf = torch.empty_like(dw)
    dbf = torch.empty_like(db)
    wsf = torch.empty(B.cf_conv3d_bwd_weight_fused_workspace_size(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_bwd_weight_fused(desc, x, g, mask, 0.01, B.CF_FUSE_POOL2, dwf, dbf, wsf)
    torch.cuda.synchronize()
    # Two valid roundings of the same layer: the unfused path decides the slope
    # from the bf16-rounded y, the fused one from the fp32 pre-activation, so a
    # pre-activation within rounding of 0 can take different slopes, moving
    # single dW entries by ~1/sqrt(voxels) of max|dW|.  Compare normwise.
    ref, got = to_np(dw), to_np(dwf)
    e = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert e <= (TOL["f32"] if dt == "f32" else 1e-2), e
    ref, got = to_np(db), to_np(dbf)
    e = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert e <= (TOL["f32"] if dt == "f32" else 1e-2), e


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("case", FWD_CASES, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d" % (c[0], *c[1], *c[2:]))
def test_fused_bwd_data(case, dt):
    """dx from the pooled-output gradient and the mask, teacher-forced."""
    N, dhw, CI, CO, k = case
    desc = B.make_desc(N, dhw, CI, CO, k, 1, "same", dt)
    if not B.cf_conv3d_fused_supported(desc) & B.FUSED_BWD_DATA:
        pytest.skip("no fused backward-data kernel for this shape")
    rng = np.random.default_rng(15)
    od = B.cf_conv3d_out_shape(desc)
    pdhw = tuple(t // 2 for t in od)
    g = dev(rng.standard_normal((N, *pdhw, CO)), dt)
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CO), dt)
    mbytes = B.cf_conv3d_mask_bytes(desc)
    mask_np = rng.integers(0, 256, mbytes, dtype=np.uint8)
    mask = torch.as_tensor(mask_np, device="cuda")
    alpha = 0.2
    dx = torch.full((N, *dhw, CI), float("nan"), dtype=tdtype(dt), device="cuda")
    B.cf_conv3d_bwd_data_fused(desc, g, mask, w, alpha, B.CF_FUSE_POOL2, dx)
    torch.cuda.synchronize()
    nbits = N * od[0] * od[1] * od[2] * CO
    bits = np.unpackbits(mask_np, bitorder="little")[:nbits].astype(bool).reshape((N, *od, CO))
    dz = oracle.avgpool3d_bwd(to_np(g), od) * np.where(bits, 1.0, alpha)
    ref = oracle.conv3d_bwd_data(dz, to_np(w), dhw)
    e = maxabs_err(to_np(dx), ref)
    assert e <= TOL[dt], e


# the one-call plain backward from a stored dz: N, (D,H,W), CI, CO, k, stride, dtype.
# The fp32 stride-2 layer of the 128^3 stack takes the combined launch
BWDP_CASES = [
    (1, (32, 32, 32), 32, 64, 4, 2, "f32"),
    (2, (14, 12, 18), 32, 64, 4, 2, "f32"),  # ragged, other tile plans
    (1, (16, 16, 16), 16, 32, 4, 1, "f32"),
    (2, (16, 16, 16), 32, 64, 4, 2, "bf16"),
]


@pytest.mark.parametrize("case", BWDP_CASES, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d_s%d_%s" % (c[0], *c[1], *c[2:]))
def test_bwd_one_call(case, monkeypatch):
    """cf_conv3d_bwd (and its deferred form) return the bits of
    cf_conv3d_bwd_weight + cf_conv3d_bwd_data, with the combined launch on and
    off, and match the oracle."""
    N, dhw, CI, CO, k, st, dt = case
    desc = B.make_desc(N, dhw, CI, CO, k, st, "same", dt)
    rng = np.random.default_rng(23)
    od = B.cf_conv3d_out_shape(desc)
    x = dev(rng.standard_normal((N, *dhw, CI)), dt)
    w = dev(rng.standard_normal((k, k, k, CI, CO)) * np.sqrt(2.0 / (k ** 3 * CI)), dt)
    dz = dev(rng.standard_normal((N, *od, CO)), dt)
    ws = torch.empty(max(16, B.cf_conv3d_bwd_weight_workspace_size(desc)), dtype=torch.uint8, device="cuda")

    def outs():
        return (torch.full((k, k, k, CI, CO), float("nan"), device="cuda"),
                torch.full((N, *dhw, CI), float("nan"), dtype=tdtype(dt), device="cuda"))

    dw0, dx0 = outs()
    B.cf_conv3d_bwd_weight(desc, x, dz, dw0, ws)
    B.cf_conv3d_bwd_data(desc, dz, w, dx0)
    got = []
    for pair in ("1", "0"):
        monkeypatch.setenv("CF_F32_PAIR", pair)
        dw1, dx1 = outs()
        B.cf_conv3d_bwd(desc, x, dz, w, dw1, dx1, ws)
        dw2, dx2 = outs()
        B.cf_reduce_partials(B.cf_conv3d_bwd_deferred(desc, x, dz, w, dw2, dx2, ws))
        got += [(dw1, dx1), (dw2, dx2)]
    torch.cuda.synchronize()
    for i, (dw1, dx1) in enumerate(got):
        what = ("one launch allowed", "one launch allowed, deferred", "two launches", "two launches, deferred")[i]
        assert torch.equal(dw1, dw0), (what, "dW", (dw1 - dw0).abs().max().item())
        assert torch.equal(dx1, dx0), (what, "dx", (dx1.float() - dx0.float()).abs().max().item())
    assert maxabs_err(to_np(dw0), oracle.conv3d_bwd_weight(to_np(x), to_np(dz), (k, k, k), stride=st)) <= TOL[dt]
    assert maxabs_err(to_np(dx0), oracle.conv3d_bwd_data(to_np(dz), to_np(w), dhw, stride=st)) <= TOL[dt]


# the one-call fused backward: N, (D,H,W), CI, CO, k, flags, dtype.  The
# stack's fp32 deep layers at 128^3 batch 1 take the combined launch; the rest
# run the two calls in sequence
BWD1_CASES = [
    (1, (8, 8, 8), 64, 64, 3, 0, "f32"),
    (1, (8, 8, 8), 64, 128, 2, 0, "f32"),
    (1, (8, 8, 8), 128, 128, 2, 0, "f32"),
    (2, (6, 5, 7), 64, 64, 3, 0, "f32"),     # ragged extents
    (1, (16, 16, 16), 64, 64, 3, 0, "f32"),  # more rows: other tile shapes
    (2, (8, 8, 8), 64, 64, 3, 0, "bf16"),
    (1, (16, 12, 64), 16, 32, 4, 1, "bf16"),  # pooled form (CF_FUSE_POOL2)
]


@pytest.mark.parametrize("case", BWD1_CASES, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d_f%d_%s" % (c[0], *c[1], *c[2:]))
def test_fused_bwd_one_call(case, monkeypatch):
    """cf_conv3d_bwd_fused (and its deferred form) return the bits of
    cf_conv3d_bwd_weight_fused + cf_conv3d_bwd_data_fused, with the combined
    launch on and off; the results also match the oracle."""
    N, dhw, CI, CO, k, flags, dt = case
    desc = B.make_desc(N, dhw, CI, CO, k, 1, "same", dt)
    sup = B.cf_conv3d_fused_supported(desc, flags)
    if not (sup & B.FUSED_BWD_WEIGHT and sup & B.FUSED_BWD_DATA):
        pytest.skip("no fused backward pair for this shape")
    rng = np.random.default_rng(21)
    od = B.cf_conv3d_out_shape(desc)
    alpha = 0.01
    x = dev(rng.standard_normal((N, *dhw, CI)), dt)
    w = dev(rng.standard_normal((k, k, k, CI, CO)) * np.sqrt(2.0 / (k ** 3 * CI)), dt)
    if flags:
        g = dev(rng.standard_normal((N,) + tuple(t // 2 for t in od) + (CO,)), dt)
        aux = torch.as_tensor(rng.integers(0, 256, B.cf_conv3d_mask_bytes(desc), dtype=np.uint8), device="cuda")
    else:
        g = dev(rng.standard_normal((N, *od, CO)), dt)
        yv = rng.standard_normal((N, *od, CO))
        yv[rng.random(yv.shape) < 0.05] = 0.0  # exact zeros take the alpha slope
        aux = dev(yv, dt)
    ws = torch.empty(B.cf_conv3d_bwd_weight_fused_workspace_size(desc, flags), dtype=torch.uint8, device="cuda")

    def outs():
        return (torch.full((k, k, k, CI, CO), float("nan"), device="cuda"), torch.full((CO,), float("nan"), device="cuda"),
                torch.full((N, *dhw, CI), float("nan"), dtype=tdtype(dt), device="cuda"))

    dw0, db0, dx0 = outs()
    B.cf_conv3d_bwd_weight_fused(desc, x, g, aux, alpha, flags, dw0, db0, ws)
    B.cf_conv3d_bwd_data_fused(desc, g, aux, w, alpha, flags, dx0)
    got = []
    for pair in ("1", "0"):
        monkeypatch.setenv("CF_F32_PAIR", pair)
        dw1, db1, dx1 = outs()
        B.cf_conv3d_bwd_fused(desc, x, g, aux, w, alpha, flags, dw1, db1, dx1, ws)
        dw2, db2, dx2 = outs()
        jobs = B.cf_conv3d_bwd_fused_deferred(desc, x, g, aux, w, alpha, flags, dw2, db2, dx2, ws)
        B.cf_reduce_partials(jobs)
        got += [(dw1, db1, dx1), (dw2, db2, dx2)]
    torch.cuda.synchronize()
    for i, (dw1, db1, dx1) in enumerate(got):
        what = ("one launch allowed", "one launch allowed, deferred", "two launches", "two launches, deferred")[i]
        assert torch.equal(dw1, dw0), (what, "dW", (dw1 - dw0).abs().max().item())
        assert torch.equal(db1, db0), (what, "db", (db1 - db0).abs().max().item())
        assert torch.equal(dx1, dx0), (what, "dx", (dx1.float() - dx0.float()).abs().max().item())
    if flags == 0:
        dz = to_np(g) * np.where(to_np(aux) > 0, 1.0, alpha)
        if dt == "bf16":
            dz = to_np(dev(dz, dt))  # the bf16 path rounds dz before the products
        assert maxabs_err(to_np(dw0), oracle.conv3d_bwd_weight(to_np(x), dz, (k, k, k))) <= TOL[dt]
        assert maxabs_err(to_np(dx0), oracle.conv3d_bwd_data(dz, to_np(w), dhw)) <= TOL[dt]
        assert maxabs_err(to_np(db0), dz.sum(axis=(0, 1, 2, 3))) <= TOL[dt]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("case", FWD_CASES, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d" % (c[0], *c[1], *c[2:]))
def test_fused_bwd_weight_dz(case, dt):
    """Backward-weights that also stores the rebuilt dz: dW, db bitwise equal to
    the plain fused call, every dz element written and equal to the oracle's
    dz within the path tolerance, and the unfused backward-data of that dz
    bitwise equal to the fused backward-data where the library has one."""
    N, dhw, CI, CO, k = case
    desc = B.make_desc(N, dhw, CI, CO, k, 1, "same", dt)
    if not B.cf_conv3d_fused_supported(desc) & B.FUSED_BWD_WEIGHT_DZ:
        pytest.skip("no dz-emitting backward-weights kernel for this shape")
    rng = np.random.default_rng(16)
    od = B.cf_conv3d_out_shape(desc)
    pdhw = tuple(t // 2 for t in od)
    x = dev(rng.standard_normal((N, *dhw, CI)), dt)
    g = dev(rng.standard_normal((N, *pdhw, CO)), dt)
    w = dev(rng.standard_normal((k, k, k, CI, CO)) / np.sqrt(k ** 3 * CO), dt)
    mbytes = B.cf_conv3d_mask_bytes(desc)
    mask_np = rng.integers(0, 256, mbytes, dtype=np.uint8)
    mask = torch.as_tensor(mask_np, device="cuda")
    alpha = 0.2
    ws = torch.empty(B.cf_conv3d_bwd_weight_fused_workspace_size(desc), dtype=torch.uint8, device="cuda")
    dw = torch.empty((k, k, k, CI, CO), dtype=torch.float32, device="cuda")
    db = torch.empty((CO,), dtype=torch.float32, device="cuda")
    dw2, db2 = torch.empty_like(dw), torch.empty_like(db)
    dz = torch.full((N, *od, CO), float("nan"), dtype=tdtype(dt), device="cuda")
    B.cf_conv3d_bwd_weight_fused(desc, x, g, mask, alpha, B.CF_FUSE_POOL2, dw, db, ws)
    B.cf_conv3d_bwd_weight_fused_dz(desc, x, g, mask, alpha, B.CF_FUSE_POOL2, dw2, db2, dz, ws)
    dx_f = torch.empty((N, *dhw, CI), dtype=tdtype(dt), device="cuda")
    dx_u = torch.full_like(dx_f, float("nan"))
    has_fused_dgrad = bool(B.cf_conv3d_fused_supported(desc) & B.FUSED_BWD_DATA)
    if has_fused_dgrad:
        B.cf_conv3d_bwd_data_fused(desc, g, mask, w, alpha, B.CF_FUSE_POOL2, dx_f)
    B.cf_conv3d_bwd_data(desc, dz, w, dx_u)
    torch.cuda.synchronize()
    assert torch.equal(dw, dw2) and torch.equal(db, db2)
    nbits = N * od[0] * od[1] * od[2] * CO
    bits = np.unpackbits(mask_np, bitorder="little")[:nbits].astype(bool).reshape((N, *od, CO))
    dz_ref = oracle.avgpool3d_bwd(to_np(g), od) * np.where(bits, 1.0, alpha)
    dz_np = to_np(dz)
    assert np.isfinite(dz_np).all()
    e = maxabs_err(dz_np, dz_ref)
    assert e <= TOL[dt], e
    if has_fused_dgrad:
        assert torch.equal(dx_f, dx_u)
    ref = oracle.conv3d_bwd_data(dz_ref, to_np(w), dhw)
    e = maxabs_err(to_np(dx_u), ref)
    assert e <= TOL[dt], e


# first layer, VALID padding: output widths that are even but not a multiple
# of 8 (the mask rows then end inside a 16-byte group), and an odd one
VALID_L1_CASES = [
    (2, (12, 10, 48), 3),    # out (10, 8, 46)
    (1, (9, 12, 128), 3),    # out (7, 10, 126): the paper's first-layer width
    (1, (10, 10, 40), 2),    # out (9, 9, 39): odd width
    (2, (12, 10, 50), 3),    # out (10, 8, 48): the fp32 register-window kernel without padding
    (1, (11, 10, 41), 2),    # out (10, 9, 40)
]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("case", VALID_L1_CASES, ids=lambda c: "n%d_%dx%dx%d_k%d" % (c[0], *c[1], c[2]))
def test_fused_bwd_weight_first_layer_valid(case, dt):
    N, dhw, k = case
    desc = B.make_desc(N, dhw, 1, 16, k, 1, "valid", dt)
    assert B.cf_conv3d_fused_supported(desc) & B.FUSED_BWD_WEIGHT
    rng = np.random.default_rng(16)
    od = B.cf_conv3d_out_shape(desc)
    pdhw = tuple(t // 2 for t in od)
    x = dev(rng.standard_normal((N, *dhw, 1)), dt)
    g = dev(rng.standard_normal((N, *pdhw, 16)), dt)
    nbits = N * od[0] * od[1] * od[2] * 16
    mbytes = B.cf_conv3d_mask_bytes(desc)
    mask_np = rng.integers(0, 256, mbytes, dtype=np.uint8)
    mask = torch.as_tensor(mask_np, device="cuda")
    dw = torch.full((k, k, k, 1, 16), float("nan"), dtype=torch.float32, device="cuda")
    db = torch.full((16,), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(B.cf_conv3d_bwd_weight_fused_workspace_size(desc), dtype=torch.uint8, device="cuda")
    B.cf_conv3d_bwd_weight_fused(desc, x, g, mask, 0.2, B.CF_FUSE_POOL2, dw, db, ws)
    torch.cuda.synchronize()
    bits = np.unpackbits(mask_np, bitorder="little")[:nbits].astype(bool).reshape((N, *od, 16))
    dz = oracle.avgpool3d_bwd(to_np(g), od) * np.where(bits, 1.0, 0.2)
    e = maxabs_err(to_np(dw), oracle.conv3d_bwd_weight(to_np(x), dz, k, pad="valid"))
    assert e <= TOL[dt], e
    e = maxabs_err(to_np(db), dz.reshape(-1, 16).sum(0))
    assert e <= TOL["f32"], e
