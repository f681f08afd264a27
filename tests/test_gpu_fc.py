"""GPU parity of the fully-connected head and the loss (Section III-A: three
FC layers with leaky ReLU after the convolutions; loss read as the mean
squared error) against the CPU oracle.

Per op teacher-forced (the oracle evaluates the exact values the GPU saw),
gate max|gpu - oracle| / max|oracle| <= 1e-5 (fp32) or 2e-2 (bf16); dW is
fp32 with exact bf16 products, gated at 1e-5 in both dtypes.  Sizes cover
the vector and scalar column paths, batches above one pass of 8 rows, a
ragged last split of K, and the full first layer of the 128^3 stack
(65536 features -> 128).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_04728_amd import binding as B
from paper_1808_04728_amd.head import FCHead
from tests._util import TOL, dev, maxabs_err, tdtype, to_np

pytestmark = pytest.mark.gpu

DTYPES = ["f32", "bf16"]
# (m, k, n): scalar columns (n = 1, 5, 3), vector columns with k a multiple of
# 8 or not, more than 8 batch rows, more column groups than one row group of
# 64 lanes (n = 1040) and than one forward pass of 256 threads (n = 2056)
SHAPES = [(1, 1, 1), (3, 37, 5), (8, 1000, 128), (5, 2049, 64), (13, 300, 24), (8, 64, 3), (2, 70001, 16),
          (3, 100, 1040), (2, 40, 2056), (4, 70001, 128), (8, 65536, 128)]


def fwd(m, k, n, dt, x, w):
    z = torch.empty((m, n), dtype=tdtype(dt), device="cuda")
    ws = torch.empty(max(16, B.cf_fc_fwd_workspace_size(m, k, n)), dtype=torch.uint8, device="cuda")
    B.cf_fc_fwd(m, k, n, dt, x, w, z, ws)
    return z


@pytest.mark.parametrize("dt", DTYPES)
@pytest.mark.parametrize("shape", SHAPES)
def test_fc_ops(dt, shape):
    m, k, n = shape
    rng = np.random.default_rng(m * 1000 + n)
    x = dev(rng.standard_normal((m, k), dtype=np.float32), dt)
    w = dev(rng.standard_normal((k, n), dtype=np.float32) / np.sqrt(k), dt)
    dz = dev(rng.standard_normal((m, n), dtype=np.float32), dt)
    z = fwd(m, k, n, dt, x, w)
    dx = torch.empty((m, k), dtype=tdtype(dt), device="cuda")
    B.cf_fc_bwd_data(m, k, n, dt, dz, w, dx)
    dw = torch.full((k, n), float("nan"), dtype=torch.float32, device="cuda")
    B.cf_fc_bwd_weight(m, k, n, dt, x, dz, dw)
    torch.cuda.synchronize()
    xn, wn, dzn = to_np(x), to_np(w), to_np(dz)
    assert maxabs_err(to_np(z), oracle.fc_fwd(xn, wn)) <= TOL[dt]
    assert maxabs_err(to_np(dx), oracle.fc_bwd_data(dzn, wn)) <= TOL[dt]
    assert maxabs_err(to_np(dw), oracle.fc_bwd_weight(xn, dzn)) <= 1e-5


def test_fc_deterministic_and_empty_batch():
    rng = np.random.default_rng(3)
    m, k, n = 8, 9000, 128
    x = dev(rng.standard_normal((m, k)), "f32")
    w = dev(rng.standard_normal((k, n)), "f32")
    a = fwd(m, k, n, "f32", x, w)
    b = fwd(m, k, n, "f32", x, w)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    # m == 0: forward and backward data are no-ops, backward weights writes zeros
    dw = torch.full((k, n), float("nan"), dtype=torch.float32, device="cuda")
    z = torch.full((1, n), 7.0, device="cuda")
    B.cf_fc_fwd(0, k, n, "f32", x, w, z, None)
    B.cf_fc_bwd_weight(0, k, n, "f32", x, z, dw)
    torch.cuda.synchronize()
    assert torch.all(z == 7.0) and torch.all(dw == 0)


def test_fc_argument_errors_launch_nothing():
    x = torch.zeros((2, 8), device="cuda")
    w = torch.zeros((8, 4), device="cuda")
    z = torch.full((2, 4), 5.0, device="cuda")
    with pytest.raises(B.CfError) as e:
        B.cf_fc_fwd(2, 8, 4, "f32", x, w, z, None)
    assert e.value.status == B.CF_ERR_WORKSPACE
    with pytest.raises(B.CfError) as e:
        B.cf_fc_bwd_data(2, 8, 4, "f32", z, w, w)  # dx overlaps W
    assert e.value.status == B.CF_ERR_ALIAS
    with pytest.raises(B.CfError) as e:
        B.cf_fc_bwd_weight(2, 0, 4, "f32", x, z, w)
    assert e.value.status == B.CF_ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.all(z == 5.0)


@pytest.mark.parametrize("dt", DTYPES)
@pytest.mark.parametrize("mn", [(8, 3), (1, 1), (1000, 7)])
def test_mse_loss(dt, mn):
    m, n = mn
    rng = np.random.default_rng(m + n)
    p = dev(rng.standard_normal((m, n)), dt)
    t = torch.from_numpy(rng.standard_normal((m, n)).astype(np.float32)).cuda()
    loss = torch.empty(4, dtype=torch.float32, device="cuda")
    dp = torch.empty((m, n), dtype=tdtype(dt), device="cuda")
    B.cf_mse_loss(m, n, dt, p, t, loss, dp)
    torch.cuda.synchronize()
    ref, dref = oracle.mse_loss(to_np(p), t.cpu().double().numpy())
    assert abs(loss[0].item() - ref) <= 1e-5 * abs(ref)
    assert maxabs_err(to_np(dp), dref) <= TOL[dt]


@pytest.mark.parametrize("dt", DTYPES)
def test_head_chain(dt):
    """The whole head on the flattened 128^3 stack output (8 x 8^3 x 128
    features -> 128 -> 64 -> 3): forward chain and loss gated against the
    oracle run from the same features and weights; backward teacher-forced
    per layer from the GPU's own dz."""
    rng = np.random.default_rng(21)
    m, dims, alpha = 8, [65536, 128, 64, 3], 0.01
    feat = dev(rng.standard_normal((m, 8, 8, 8, 128), dtype=np.float32), dt)
    ws = [rng.standard_normal((dims[i], dims[i + 1])) * np.sqrt(2.0 / dims[i]) for i in range(3)]
    bs = [rng.normal(0, 0.1, dims[i + 1]) for i in range(3)]
    tgt = np.stack([rng.uniform(0.25, 0.35, m), rng.uniform(0.78, 0.95, m), rng.uniform(0.9, 1.0, m)], 1)
    h = FCHead(m, dims[0], dims[1:], dtype=dt, alpha=alpha)
    h.set_params(ws, bs, tgt)
    loss = h.forward(feat)
    torch.cuda.synchronize()
    dp = to_np(h.dz[-1])  # the loss gradient as stored (the backward pass overwrites it in place)
    dfeat = h.backward()
    torch.cuda.synchronize()
    wn = [to_np(w) for w in h.w]  # the weights the GPU used (bf16-rounded in the bf16 path)
    tn = h.target.cpu().double().numpy()
    lref, dpref, acts = oracle.head_forward(to_np(feat), wn, bs, alpha, tn)
    for i in range(3):
        assert maxabs_err(to_np(h.y[i]), acts[i]["y"]) <= TOL[dt], ("fwd", i)
    assert abs(loss[0].item() - lref) <= TOL[dt] * abs(lref)
    assert maxabs_err(dp, oracle.mse_loss(to_np(h.y[2]), tn)[1]) <= TOL[dt]
    # backward, teacher-forced from the GPU's inputs of each op
    g = dp
    for i in range(2, -1, -1):
        dz, db = oracle.bias_lrelu_bwd(g, to_np(h.y[i]), alpha)
        assert maxabs_err(to_np(h.dz[i]), dz) <= TOL[dt], ("dz", i)
        # db sums the unrounded products (bf16 path: before dz is rounded to bf16)
        assert maxabs_err(to_np(h.db[i]), db) <= 1e-5, ("db", i)
        xin = to_np(feat).reshape(m, -1) if i == 0 else to_np(h.y[i - 1])
        assert maxabs_err(to_np(h.dw[i]), oracle.fc_bwd_weight(xin, to_np(h.dz[i]))) <= 1e-5, ("dw", i)
        assert maxabs_err(to_np(h.dx[i]), oracle.fc_bwd_data(to_np(h.dz[i]), wn[i])) <= TOL[dt], ("dx", i)
        g = to_np(h.dx[i])
    assert dfeat.data_ptr() == h.dx[0].data_ptr()


def _head_setup(dt, m, dims, seed):
    rng = np.random.default_rng(seed)
    feat = dev(rng.standard_normal((m, dims[0]), dtype=np.float32), dt)
    ws = [rng.standard_normal((dims[i], dims[i + 1])) * np.sqrt(2.0 / dims[i]) for i in range(len(dims) - 1)]
    bs = [rng.normal(0, 0.1, dims[i + 1]) for i in range(len(dims) - 1)]
    tgt = rng.uniform(0.2, 1.0, (m, dims[-1]))
    h = FCHead(m, dims[0], dims[1:], dtype=dt, alpha=0.01)
    h.set_params(ws, bs, tgt)
    return h, feat, bs


def _grad_of_loss(h, dt):
    """dL/dy of the last layer as the one-call head forms it: 2 (y - t) / (m n)
    in fp32, rounded once to the dtype."""
    y = h.y[-1].float().cpu()
    inv = np.float32(1.0 / (h.m * h.dims[-1]))
    dp = (torch.tensor(2.0, dtype=torch.float32) * (y - h.target.cpu())) * torch.tensor(inv)
    return to_np(dp.to(tdtype(dt)))


HEAD_CASES = [(8, [65536, 128, 64, 3]), (1, [65536, 128, 64, 3]), (5, [4000, 64, 48, 16, 3]), (3, [1024, 256, 7])]


@pytest.mark.parametrize("dt", DTYPES)
@pytest.mark.parametrize("m,dims", HEAD_CASES)
def test_head_one_call(dt, m, dims):
    """cf_fc_head (four launches) against the oracle, teacher-forced per op
    from the GPU's own intermediate tensors, as the per-layer chain test."""
    h, feat, bs = _head_setup(dt, m, dims, 33 + m)
    assert h.fused
    dfeat = h.step(feat)
    torch.cuda.synchronize()
    L = len(dims) - 1
    wn = [to_np(w) for w in h.w]
    tn = h.target.cpu().double().numpy()
    lref, _, acts = oracle.head_forward(to_np(feat), wn, bs, 0.01, tn)
    for i in range(L):
        assert maxabs_err(to_np(h.y[i]), acts[i]["y"]) <= TOL[dt], ("fwd", i)
    assert abs(h.loss[0].item() - lref) <= TOL[dt] * abs(lref)
    # the loss gradient: against the oracle's, and as rounded by the kernel for the teacher-forced steps
    dp = _grad_of_loss(h, dt)
    assert maxabs_err(dp, oracle.mse_loss(to_np(h.y[-1]), tn)[1]) <= TOL[dt]
    g = dp
    for i in range(L - 1, -1, -1):
        dz, db = oracle.bias_lrelu_bwd(g, to_np(h.y[i]), 0.01)
        assert maxabs_err(to_np(h.dz[i]), dz) <= TOL[dt], ("dz", i)
        assert maxabs_err(to_np(h.db[i]), db) <= 1e-5, ("db", i)
        xin = to_np(feat) if i == 0 else to_np(h.y[i - 1])
        assert maxabs_err(to_np(h.dw[i]), oracle.fc_bwd_weight(xin, to_np(h.dz[i]))) <= 1e-5, ("dw", i)
        assert maxabs_err(to_np(h.dx[i]), oracle.fc_bwd_data(to_np(h.dz[i]), wn[i])) <= TOL[dt], ("dx", i)
        g = to_np(h.dx[i])
    assert dfeat.data_ptr() == h.dx[0].data_ptr()


@pytest.mark.parametrize("dt", DTYPES)
def test_head_one_call_matches_per_layer_calls(dt):
    """The first layer's y is bitwise the per-layer calls' (same split-K sums,
    bias and leaky ReLU); its dW and dx are bitwise cf_fc_bwd_weight and
    cf_fc_bwd_data on the one-call dz; the rest agrees to the dtype's
    tolerance; two calls give the same bits."""
    m, dims = 8, [65536, 128, 64, 3]
    h, feat, _ = _head_setup(dt, m, dims, 7)
    h.forward(feat)
    h.backward()
    torch.cuda.synchronize()
    ref = {k: [t.clone() for t in getattr(h, k)] for k in ("y", "dz", "dx", "dw", "db")}
    ref_loss = h.loss[0].item()
    h.step(feat)
    torch.cuda.synchronize()
    one = {k: [t.clone() for t in getattr(h, k)] for k in ("y", "dz", "dx", "dw", "db")}
    assert torch.equal(one["y"][0], ref["y"][0])
    dw0 = torch.empty_like(h.dw[0])
    dx0 = torch.empty_like(h.dx[0])
    B.cf_fc_bwd_weight(m, dims[0], dims[1], dt, feat, one["dz"][0], dw0)
    B.cf_fc_bwd_data(m, dims[0], dims[1], dt, one["dz"][0], h.w[0], dx0)
    torch.cuda.synchronize()
    assert torch.equal(one["dw"][0], dw0) and torch.equal(one["dx"][0], dx0)
    for k in ("y", "dz", "dx"):
        for i in range(3):
            assert maxabs_err(to_np(one[k][i]), to_np(ref[k][i])) <= 2 * TOL[dt], (k, i)
    for k in ("dw", "db"):
        for i in range(3):
            assert maxabs_err(to_np(one[k][i]), to_np(ref[k][i])) <= 2 * TOL[dt], (k, i)
    assert abs(h.loss[0].item() - ref_loss) <= TOL[dt] * abs(ref_loss)
    h.step(feat)
    torch.cuda.synchronize()
    for k in ("y", "dz", "dx", "dw", "db"):
        for a, b in zip(one[k], getattr(h, k)):
            assert torch.equal(a, b), k


@pytest.mark.parametrize("dt", DTYPES)
def test_head_step_outside_limits_runs_per_layer(dt):
    """Widths outside cf_fc_head's limits (40 first-layer outputs: not a power
    of two of vector lanes) make FCHead.step run the per-layer calls, with the
    same results as forward() + backward()."""
    m, dims = 3, [1000, 40, 3]
    h, feat, _ = _head_setup(dt, m, dims, 5)
    assert not h.fused
    d1 = h.step(feat).clone()
    l1 = h.loss[0].item()
    h.forward(feat)
    d2 = h.backward()
    torch.cuda.synchronize()
    assert torch.equal(d1, d2) and h.loss[0].item() == l1
