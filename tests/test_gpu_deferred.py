"""Deferred gradient sums: every _deferred entry point followed by one
cf_reduce_partials over the collected jobs writes exactly the bits of the
plain call (the sums' order depends only on the partials' shape), for the
unfused weight gradient, the bias gradient and the fused weight gradient with
and without the dz output, separately and batched together."""
import numpy as np
import pytest
import torch

from paper_1808_04728_amd import binding as B
from tests._util import tdtype, dev

pytestmark = pytest.mark.gpu

# N, (D,H,W), CI, CO, k, stride, dtype
WCASES = [
    (1, (9, 10, 11), 16, 32, 4, 1, "bf16"),
    (2, (7, 6, 9), 32, 64, 4, 2, "bf16"),
    (1, (13, 12, 11), 1, 16, 3, 1, "bf16"),
    (1, (6, 5, 7), 64, 128, 2, 1, "f32"),
    (2, (8, 8, 8), 64, 64, 3, 1, "bf16"),
]


@pytest.mark.parametrize("case", WCASES, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d_s%d_%s" % (c[0], *c[1], *c[2:]))
def test_deferred_wgrad_and_bias_bitwise(case):
    N, dhw, CI, CO, k, s, dt = case
    desc = B.make_desc(N, dhw, CI, CO, k, s, "same", dt)
    rng = np.random.default_rng(21)
    od = B.cf_conv3d_out_shape(desc)
    x = dev(rng.standard_normal((N, *dhw, CI)), dt)
    dz = dev(rng.standard_normal((N, *od, CO)), dt)
    y = dev(rng.standard_normal((N, *od, CO)), dt)
    ws = torch.empty(max(B.cf_conv3d_bwd_weight_workspace_size(desc), 16), dtype=torch.uint8, device="cuda")
    nvox = N * od[0] * od[1] * od[2]
    wsb = torch.empty(max(B.cf_bias_lrelu_bwd_workspace_size(nvox, CO), 16), dtype=torch.uint8, device="cuda")
    dw_ref = torch.empty((k, k, k, CI, CO), dtype=torch.float32, device="cuda")
    db_ref = torch.empty(CO, dtype=torch.float32, device="cuda")
    dz2_ref = torch.empty_like(dz)
    B.cf_conv3d_bwd_weight(desc, x, dz, dw_ref, ws)
    B.cf_bias_lrelu_bwd(nvox, CO, dt, dz, y, 0.2, dz2_ref, db_ref, wsb)
    dw = torch.full_like(dw_ref, float("nan"))
    db = torch.full_like(db_ref, float("nan"))
    dz2 = torch.empty_like(dz)
    jobs = B.cf_conv3d_bwd_weight_deferred(desc, x, dz, dw, ws)
    jobs += B.cf_bias_lrelu_bwd_deferred(nvox, CO, dt, dz, y, 0.2, dz2, db, wsb)
    assert len(jobs) == 2
    B.cf_reduce_partials(jobs)
    torch.cuda.synchronize()
    assert torch.equal(dw, dw_ref) and torch.equal(db, db_ref) and torch.equal(dz2, dz2_ref)


FCASES = [
    (1, (16, 12, 64), 16, 32, 4),
    (2, (9, 7, 33), 16, 32, 4),
    (2, (13, 12, 11), 1, 16, 3),
    (1, (32, 32, 32), 1, 16, 3),
]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("case", FCASES, ids=lambda c: "n%d_%dx%dx%d_c%d-%d_k%d" % (c[0], *c[1], *c[2:]))
def test_deferred_fused_wgrad_bitwise(case, dt):
    N, dhw, CI, CO, k = case
    desc = B.make_desc(N, dhw, CI, CO, k, 1, "same", dt)
    sup = B.cf_conv3d_fused_supported(desc)
    if not sup & B.FUSED_BWD_WEIGHT:
        pytest.skip("no fused backward-weights kernel for this shape")
    rng = np.random.default_rng(22)
    od = B.cf_conv3d_out_shape(desc)
    pdhw = tuple(t // 2 for t in od)
    x = dev(rng.standard_normal((N, *dhw, CI)), dt)
    g = dev(rng.standard_normal((N, *pdhw, CO)), dt)
    mask = torch.as_tensor(rng.integers(0, 256, B.cf_conv3d_mask_bytes(desc), dtype=np.uint8), device="cuda")
    ws = torch.empty(B.cf_conv3d_bwd_weight_fused_workspace_size(desc), dtype=torch.uint8, device="cuda")
    dw_ref = torch.empty((k, k, k, CI, CO), dtype=torch.float32, device="cuda")
    db_ref = torch.empty(CO, dtype=torch.float32, device="cuda")
    B.cf_conv3d_bwd_weight_fused(desc, x, g, mask, 0.2, B.CF_FUSE_POOL2, dw_ref, db_ref, ws)
    dw = torch.full_like(dw_ref, float("nan"))
    db = torch.full_like(db_ref, float("nan"))
    jobs = B.cf_conv3d_bwd_weight_fused_deferred(desc, x, g, mask, 0.2, B.CF_FUSE_POOL2, dw, db, None, ws)
    assert len(jobs) == 2
    B.cf_reduce_partials(jobs)
    torch.cuda.synchronize()
    assert torch.equal(dw, dw_ref) and torch.equal(db, db_ref)
    if sup & B.FUSED_BWD_WEIGHT_DZ:
        dz_ref = torch.empty((N, *od, CO), dtype=tdtype(dt), device="cuda")
        B.cf_conv3d_bwd_weight_fused_dz(desc, x, g, mask, 0.2, B.CF_FUSE_POOL2, dw_ref, db_ref, dz_ref, ws)
        dz = torch.full_like(dz_ref, float("nan"))
        dw.fill_(float("nan"))
        jobs = B.cf_conv3d_bwd_weight_fused_deferred(desc, x, g, mask, 0.2, B.CF_FUSE_POOL2, dw, db, dz, ws)
        B.cf_reduce_partials(jobs)
        torch.cuda.synchronize()
        assert torch.equal(dw, dw_ref) and torch.equal(db, db_ref) and torch.equal(dz, dz_ref)


def test_reduce_partials_batch_matches_single_jobs():
    """Many jobs of mixed shapes in one call equal each job run alone; a job
    with zero rows writes zeros."""
    rng = np.random.default_rng(23)
    shapes = [(1, 5), (3, 300), (17, 1024), (64, 33), (512, 4096), (0, 8), (7, 256), (100, 1)]
    parts = [torch.as_tensor(rng.standard_normal((r, c)), dtype=torch.float32, device="cuda") for r, c in shapes]
    outs = [torch.full((c,), float("nan"), dtype=torch.float32, device="cuda") for r, c in shapes]
    refs = [torch.full((c,), float("nan"), dtype=torch.float32, device="cuda") for r, c in shapes]
    job = lambda p, o, r, c: B.cf_reduction(p.data_ptr() if r else 0, o.data_ptr(), r, c)
    for (r, c), p, o in zip(shapes, parts, refs):
        B.cf_reduce_partials([job(p, o, r, c)])
    B.cf_reduce_partials([job(p, o, r, c) for (r, c), p, o in zip(shapes, parts, outs)])
    torch.cuda.synchronize()
    for (r, c), p, o, ref in zip(shapes, parts, outs, refs):
        assert torch.equal(o, ref)
        want = p.double().sum(0).cpu().numpy() if r else np.zeros(c)
        assert np.allclose(o.cpu().numpy(), want, rtol=1e-5, atol=1e-5 * max(1, r))
