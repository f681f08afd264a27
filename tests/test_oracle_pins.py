"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test checks the oracle against a library routine computing the same
mathematical object (PyTorch's CPU fp64 convolution / pooling and autograd,
numpy matmul), a closed form, an invariant of the definitions (delta kernels,
linearity, adjoint identities, finite differences), or numbers printed in the
paper (Table I, via tests/golden/).  A dropped term, a wrong sign or index, a
flipped kernel or a transposed operand in the oracle fails at least one.
"""
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
torch.set_num_threads(4)


def rnd(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def torch_conv_same_or_valid(x, w, s, pad):
    """PyTorch fp64 CPU reference: explicit asymmetric zero padding, then conv3d."""
    N, D, H, W, CI = x.shape
    K = w.shape[:3]
    pads = []
    for i, (n_in, k) in enumerate(zip((D, H, W), K)):
        out, pb = oracle.geometry(n_in, k, s, pad)
        tot = max((out - 1) * s + k - n_in, 0) if pad == "same" else 0
        pads.append((pb, tot - pb))
    xt = torch.from_numpy(x).permute(0, 4, 1, 2, 3).contiguous().requires_grad_(True)
    wt = torch.from_numpy(w).permute(4, 3, 0, 1, 2).contiguous().requires_grad_(True)
    xp = F.pad(xt, (pads[2][0], pads[2][1], pads[1][0], pads[1][1], pads[0][0], pads[0][1]))
    zt = F.conv3d(xp, wt, stride=s)
    return xt, wt, zt


# ---------------------------------------------------------------------------
# Geometry: TensorFlow SAME / VALID rule
# ---------------------------------------------------------------------------

# (in, k, s, pad) -> (out, pad_before); TensorFlow's documented SAME rule puts
# the odd padding element after the data.
GEOMETRY_CASES = [
    (32, 3, 1, "same", 32, 1), (64, 4, 1, "same", 64, 1), (32, 4, 2, "same", 16, 1),
    (8, 3, 1, "same", 8, 1), (8, 2, 1, "same", 8, 0), (7, 4, 2, "same", 4, 1),
    (5, 1, 2, "same", 3, 0), (128, 3, 1, "valid", 126, 0), (63, 4, 1, "valid", 60, 0),
    (30, 4, 1, "valid", 27, 0), (7, 3, 2, "valid", 3, 0),
]


@pytest.mark.parametrize("n_in,k,s,pad,out,pb", GEOMETRY_CASES)
def test_geometry(n_in, k, s, pad, out, pb):
    assert oracle.geometry(n_in, k, s, pad) == (out, pb)


def test_valid_kernel_too_large_raises():
    with pytest.raises(ValueError):
        oracle.geometry(3, 4, 1, "valid")


def test_table1_flop_products():
    """Per-layer FLOPs of the paper's own VALID network (conv1..conv3) from the
    oracle's geometry agree with time x rate printed in Table I."""
    rows = []
    with open(os.path.join(GOLDEN, "table1_conv_layers.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append(line.split())
    assert len(rows) == 3
    for name, n_in, k, ci, co, *vals in rows:
        n_in, k, ci, co = int(n_in), int(k), int(ci), int(co)
        out, _ = oracle.geometry(n_in, k, 1, "valid")
        flops = 2.0 * out ** 3 * co * k ** 3 * ci
        vals = [float(v) for v in vals]
        products = [vals[i] * vals[i + 3] * 1e9 for i in range(3) if vals[i] > 0]
        for p in products:
            # ms x TF/s, each printed to 2-3 significant digits: allow 1.5 %
            assert abs(p - flops) / flops < 0.015, (name, p, flops)


# ---------------------------------------------------------------------------
# Convolution against PyTorch's fp64 CPU convolution and its autograd
# ---------------------------------------------------------------------------

CONV_CASES = [
    # N, (D,H,W), CI, CO, k, s, pad
    (1, (5, 6, 7), 1, 3, 3, 1, "same"),
    (2, (6, 5, 4), 3, 4, 4, 1, "same"),
    (1, (7, 7, 6), 4, 2, 4, 2, "same"),
    (1, (6, 6, 6), 16, 5, 2, 1, "same"),
    (2, (5, 4, 6), 3, 3, 1, 2, "same"),
    (1, (7, 6, 5), 3, 2, 3, 2, "valid"),
    (1, (6, 7, 6), 4, 3, 4, 1, "valid"),
    (1, (4, 5, 6), 5, 4, 2, 2, "same"),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_matches_torch(case):
    N, dhw, CI, CO, k, s, pad = case
    x = rnd((N, *dhw, CI), 1)
    w = rnd((k, k, k, CI, CO), 2)
    xt, wt, zt = torch_conv_same_or_valid(x, w, s, pad)
    z_ref = zt.detach().permute(0, 2, 3, 4, 1).numpy()
    z = oracle.conv3d_fwd(x, w, stride=s, pad=pad)
    assert z.shape == z_ref.shape
    np.testing.assert_allclose(z, z_ref, rtol=0, atol=1e-12 * max(1, np.abs(z_ref).max()))
    # backward through the library's autograd
    g = rnd(z.shape, 3)
    zt.backward(torch.from_numpy(g).permute(0, 4, 1, 2, 3))
    dx_ref = xt.grad.permute(0, 2, 3, 4, 1).numpy()
    dw_ref = wt.grad.permute(2, 3, 4, 1, 0).numpy()
    dx = oracle.conv3d_bwd_data(g, w, dhw, stride=s, pad=pad)
    dw = oracle.conv3d_bwd_weight(x, g, k, stride=s, pad=pad)
    np.testing.assert_allclose(dx, dx_ref, rtol=0, atol=1e-12 * max(1, np.abs(dx_ref).max()))
    np.testing.assert_allclose(dw, dw_ref, rtol=0, atol=1e-12 * max(1, np.abs(dw_ref).max()))


def test_conv_nonuniform_strides_match_torch():
    x = rnd((1, 6, 7, 8, 3), 4)
    w = rnd((3, 2, 4, 3, 2), 5)
    xt = torch.from_numpy(x).permute(0, 4, 1, 2, 3)
    wt = torch.from_numpy(w).permute(4, 3, 0, 1, 2)
    z_ref = F.conv3d(xt, wt, stride=(1, 2, 2)).permute(0, 2, 3, 4, 1).numpy()
    z = oracle.conv3d_fwd(x, w, stride=(1, 2, 2), pad="valid")
    np.testing.assert_allclose(z, z_ref, atol=1e-12)


# ---------------------------------------------------------------------------
# Delta kernels: identity, shifts (pins pad placement), subsampling
# ---------------------------------------------------------------------------

def delta_weight(k, C, tap):
    w = np.zeros((k, k, k, C, C))
    for c in range(C):
        w[tap[0], tap[1], tap[2], c, c] = 1.0
    return w


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_delta_kernel_identity_bitwise(k):
    x = rnd((2, 6, 5, 7, 3), 6)
    _, pb = oracle.geometry(6, k, 1, "same")
    z = oracle.conv3d_fwd(x, delta_weight(k, 3, (pb, pb, pb)))
    assert np.array_equal(z, x)


def test_delta_kernel_shift_pins_padding():
    # k = 4 SAME: pad (1, 2).  Tap t reads x[o + t - 1]; tap 3 reads two ahead,
    # so the last two outputs along that axis see padding (zeros).
    x = rnd((1, 6, 6, 6, 2), 7)
    z = oracle.conv3d_fwd(x, delta_weight(4, 2, (3, 1, 0)))
    ref = np.zeros_like(x)
    ref[:, 0:4, :, 1:6] = x[:, 2:6, :, 0:5]
    assert np.array_equal(z, ref)


def test_delta_stride2_subsamples():
    x = rnd((1, 8, 8, 8, 2), 8)
    _, pb = oracle.geometry(8, 4, 2, "same")
    z = oracle.conv3d_fwd(x, delta_weight(4, 2, (pb, pb, pb)), stride=2)
    assert np.array_equal(z, x[:, ::2, ::2, ::2])


# ---------------------------------------------------------------------------
# Linearity, adjoint identities, special cases
# ---------------------------------------------------------------------------

def test_linearity():
    x1, x2 = rnd((1, 5, 6, 5, 3), 9), rnd((1, 5, 6, 5, 3), 10)
    w1, w2 = rnd((3, 3, 3, 3, 4), 11), rnd((3, 3, 3, 3, 4), 12)
    a, b = 0.75, -1.5
    lhs = oracle.conv3d_fwd(a * x1 + b * x2, w1)
    rhs = a * oracle.conv3d_fwd(x1, w1) + b * oracle.conv3d_fwd(x2, w1)
    np.testing.assert_allclose(lhs, rhs, atol=1e-12)
    lhs = oracle.conv3d_fwd(x1, a * w1 + b * w2)
    rhs = a * oracle.conv3d_fwd(x1, w1) + b * oracle.conv3d_fwd(x1, w2)
    np.testing.assert_allclose(lhs, rhs, atol=1e-12)


@pytest.mark.parametrize("k,s,pad", [(3, 1, "same"), (4, 1, "same"), (4, 2, "same"),
                                     (2, 1, "same"), (3, 2, "valid")])
def test_adjoint_identities(k, s, pad):
    x = rnd((2, 7, 6, 5, 3), 13)
    w = rnd((k, k, k, 3, 4), 14)
    z = oracle.conv3d_fwd(x, w, stride=s, pad=pad)
    g = rnd(z.shape, 15)
    lhs = np.sum(z * g)
    dx = oracle.conv3d_bwd_data(g, w, x.shape[1:4], stride=s, pad=pad)
    dw = oracle.conv3d_bwd_weight(x, g, k, stride=s, pad=pad)
    assert abs(lhs - np.sum(x * dx)) < 1e-10 * abs(lhs) + 1e-10
    assert abs(lhs - np.sum(w * dw)) < 1e-10 * abs(lhs) + 1e-10


def test_pointwise_kernel_is_matmul():
    x = rnd((2, 3, 4, 5, 6), 16)
    w = rnd((1, 1, 1, 6, 7), 17)
    z = oracle.conv3d_fwd(x, w)
    np.testing.assert_allclose(z, x @ w[0, 0, 0], atol=1e-12)


def test_constant_input_interior():
    c = 1.75
    x = np.full((1, 7, 7, 7, 3), c)
    w = rnd((3, 3, 3, 3, 2), 18)
    z = oracle.conv3d_fwd(x, w)
    np.testing.assert_allclose(z[0, 1:-1, 1:-1, 1:-1], np.broadcast_to(c * w.sum(axis=(0, 1, 2, 3)), (5, 5, 5, 2)),
                               atol=1e-12)


def test_batch_independence():
    x = rnd((3, 5, 5, 5, 2), 19)
    w = rnd((3, 3, 3, 2, 3), 20)
    z = oracle.conv3d_fwd(x, w)
    for n in range(3):
        np.testing.assert_array_equal(z[n:n + 1], oracle.conv3d_fwd(x[n:n + 1], w))


def test_point_evaluators_agree_with_full():
    x = rnd((2, 7, 6, 5, 3), 21)
    w = rnd((4, 4, 4, 3, 4), 22)
    for s in (1, 2):
        z = oracle.conv3d_fwd(x, w, stride=s)
        g = rnd(z.shape, 23)
        dx = oracle.conv3d_bwd_data(g, w, (7, 6, 5), stride=s)
        dw = oracle.conv3d_bwd_weight(x, g, 4, stride=s)
        rng = np.random.default_rng(s)
        iz = np.stack([rng.integers(0, t, 20) for t in z.shape], 1)
        ix = np.stack([rng.integers(0, t, 20) for t in x.shape], 1)
        iw = np.stack([rng.integers(0, t, 20) for t in w.shape], 1)
        np.testing.assert_array_equal(oracle.conv3d_fwd_points(x, w, iz, stride=s), z[tuple(iz.T)])
        np.testing.assert_array_equal(oracle.conv3d_bwd_data_points(g, w, (7, 6, 5), ix, stride=s), dx[tuple(ix.T)])
        np.testing.assert_array_equal(oracle.conv3d_bwd_weight_points(x, g, 4, iw, stride=s), dw[tuple(iw.T)])


# ---------------------------------------------------------------------------
# Pooling
# ---------------------------------------------------------------------------

def test_pool_matches_torch():
    y = rnd((2, 6, 8, 4, 3), 24)
    p = oracle.avgpool3d_fwd(y)
    ref = F.avg_pool3d(torch.from_numpy(y).permute(0, 4, 1, 2, 3), 2, 2).permute(0, 2, 3, 4, 1).numpy()
    np.testing.assert_allclose(p, ref, atol=1e-14)


def test_pool_odd_extent_floors():
    y = rnd((1, 7, 5, 6, 2), 25)
    p = oracle.avgpool3d_fwd(y)
    assert p.shape == (1, 3, 2, 3, 2)
    ref = F.avg_pool3d(torch.from_numpy(y).permute(0, 4, 1, 2, 3), 2, 2).permute(0, 2, 3, 4, 1).numpy()
    np.testing.assert_allclose(p, ref, atol=1e-14)


def test_pool_is_constant_weight_conv():
    """Average pooling is a per-channel convolution with weights 1/KS^3."""
    y = rnd((1, 6, 6, 8, 3), 26)
    w = np.zeros((2, 2, 2, 3, 3))
    for c in range(3):
        w[:, :, :, c, c] = 1.0 / 8.0
    np.testing.assert_allclose(oracle.avgpool3d_fwd(y), oracle.conv3d_fwd(y, w, stride=2, pad="valid"), atol=1e-14)


def test_pool_adjoint():
    y = rnd((2, 7, 6, 4, 3), 27)
    p = oracle.avgpool3d_fwd(y)
    g = rnd(p.shape, 28)
    dy = oracle.avgpool3d_bwd(g, y.shape[1:4])
    assert abs(np.sum(p * g) - np.sum(y * dy)) < 1e-12
    # the trailing odd plane is not covered by any window
    assert np.all(dy[:, 6] == 0)


# ---------------------------------------------------------------------------
# Bias + leaky ReLU
# ---------------------------------------------------------------------------

def test_lrelu_special_cases():
    z = rnd((3, 4, 5, 6, 4), 29)
    b = rnd((4,), 30)
    # alpha = 0 is ReLU, alpha = 1 is the identity
    np.testing.assert_array_equal(oracle.bias_lrelu_fwd(z, b, 0.0), np.maximum(z + b, 0.0))
    np.testing.assert_array_equal(oracle.bias_lrelu_fwd(z, b, 1.0), z + b)
    np.testing.assert_allclose(oracle.bias_lrelu_fwd(z, b, 0.01),
                               torch.nn.functional.leaky_relu(torch.from_numpy(z + b), 0.01).numpy(), atol=0)


def test_lrelu_bwd_matches_autograd_and_zero_rule():
    z = rnd((2, 3, 4, 5, 3), 31)
    z[0, 0, 0, :2] = 0.0  # pre-activations exactly zero
    b = np.zeros(3)
    alpha = 0.2
    y = oracle.bias_lrelu_fwd(z, b, alpha)
    g = rnd(z.shape, 32)
    dz, db = oracle.bias_lrelu_bwd(g, y, alpha)
    zt = torch.from_numpy(z).requires_grad_(True)
    bt = torch.from_numpy(b).requires_grad_(True)
    F.leaky_relu(zt + bt, alpha).backward(torch.from_numpy(g))
    nz = z != 0
    np.testing.assert_allclose(dz[nz], zt.grad.numpy()[nz], atol=1e-15)
    # at exactly zero the slope is alpha (reading of the subgradient)
    np.testing.assert_allclose(dz[~nz], alpha * g[~nz], atol=1e-15)
    np.testing.assert_allclose(db, dz.reshape(-1, 3).sum(0), atol=1e-12)
    np.testing.assert_allclose(db[nz.reshape(-1, 3).all(0)], bt.grad.numpy()[nz.reshape(-1, 3).all(0)], atol=1e-12)


# ---------------------------------------------------------------------------
# Finite differences through conv -> bias + lReLU -> pool
# ---------------------------------------------------------------------------

def test_finite_differences_layer_chain():
    layers = [dict(k=3, stride=1, pool=True), dict(k=4, stride=2, pool=False)]
    x = rnd((1, 8, 8, 8, 2), 33)
    ws = [rnd((3, 3, 3, 2, 3), 34) * 0.5, rnd((4, 4, 4, 3, 2), 35) * 0.3]
    bs = [rnd((3,), 36) * 0.1, rnd((2,), 37) * 0.1]
    alpha = 0.2

    def loss(x_, ws_, bs_):
        acts = oracle.stack_forward(x_, layers, ws_, bs_, alpha)
        return np.sum(acts[-1]["out"] * gout), acts

    acts = oracle.stack_forward(x, layers, ws, bs, alpha)
    gout = rnd(acts[-1]["out"].shape, 38)
    grads = oracle.stack_backward(acts, layers, ws, gout, alpha, skip_first_dgrad=False)
    h = 1e-6
    rng = np.random.default_rng(39)

    def check(get, grad, n=6):
        for _ in range(n):
            arr = get()
            idx = tuple(rng.integers(0, s) for s in arr.shape)
            old = arr[idx]
            arr[idx] = old + h
            lp, _ = loss(x, ws, bs)
            arr[idx] = old - h
            lm, _ = loss(x, ws, bs)
            arr[idx] = old
            fd = (lp - lm) / (2 * h)
            assert abs(fd - grad[idx]) < 1e-6 * max(1.0, abs(fd)), (idx, fd, grad[idx])

    check(lambda: ws[0], grads[0]["dw"])
    check(lambda: ws[1], grads[1]["dw"])
    check(lambda: bs[0], grads[0]["db"], n=3)
    check(lambda: bs[1], grads[1]["db"], n=2)
    check(lambda: x, grads[0]["dx"])
