"""Pins of the oracle's fully-connected head and loss (Section III-A: three
FC layers after the convolutions, leaky ReLU on every layer, three outputs;
the loss, which the paper does not name, read as the mean squared error).

Each test checks the oracle against something it does not compute itself:
brute-force Python loops, PyTorch's CPU fp64 linear / mse_loss and autograd,
adjoint identities, closed forms, or central finite differences of the whole
head's loss.  A transposed weight, a dropped 2 or 1/(M N) factor, a wrong
slope or a swapped operand fails at least one.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def rnd(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def test_fc_fwd_brute_force_and_torch():
    x, w = rnd((3, 7), 1), rnd((7, 5), 2)
    ref = [[sum(x[m, k] * w[k, j] for k in range(7)) for j in range(5)] for m in range(3)]
    z = oracle.fc_fwd(x, w)
    assert np.abs(z - np.array(ref)).max() < 1e-13
    # torch's linear takes the weight as [out][in]
    zt = F.linear(torch.from_numpy(x), torch.from_numpy(w).T.contiguous()).numpy()
    assert np.abs(z - zt).max() < 1e-13


def test_fc_fwd_flattens_ndhwc_rows_in_memory_order():
    """A stack output [M, D, H, W, C] enters the first FC layer as rows of
    D*H*W*C features in memory order (TensorFlow's flatten of NDHWC)."""
    a = rnd((2, 2, 3, 2, 4), 3)
    w = rnd((48, 3), 4)
    z = oracle.fc_fwd(a, w)
    for m in range(2):
        ref = np.zeros(3)
        for d in range(2):
            for h in range(3):
                for ww in range(2):
                    for c in range(4):
                        ref += a[m, d, h, ww, c] * w[((d * 3 + h) * 2 + ww) * 4 + c]
        assert np.abs(z[m] - ref).max() < 1e-13


@pytest.mark.parametrize("M,K,N", [(1, 1, 1), (4, 9, 3), (8, 33, 16), (2, 5, 1)])
def test_fc_adjoint_identities(M, K, N):
    x, w, g = rnd((M, K), 5), rnd((K, N), 6), rnd((M, N), 7)
    lhs = np.sum(oracle.fc_fwd(x, w) * g)
    assert abs(lhs - np.sum(x * oracle.fc_bwd_data(g, w))) <= 1e-12 * max(1.0, abs(lhs))
    assert abs(lhs - np.sum(w * oracle.fc_bwd_weight(x, g))) <= 1e-12 * max(1.0, abs(lhs))


def test_fc_backward_matches_autograd():
    x, w, g = rnd((5, 11), 8), rnd((11, 6), 9), rnd((5, 6), 10)
    xt = torch.from_numpy(x).requires_grad_(True)
    wt = torch.from_numpy(w).requires_grad_(True)
    (xt @ wt).backward(torch.from_numpy(g))
    assert np.abs(oracle.fc_bwd_data(g, w) - xt.grad.numpy()).max() < 1e-13
    assert np.abs(oracle.fc_bwd_weight(x, g) - wt.grad.numpy()).max() < 1e-13


def test_fc_bwd_weight_single_row_is_outer_product():
    x, g = rnd((1, 9), 11), rnd((1, 4), 12)
    assert np.array_equal(oracle.fc_bwd_weight(x, g), np.outer(x[0], g[0]))


def test_mse_closed_forms_and_torch():
    t = rnd((4, 3), 13)
    loss, dp = oracle.mse_loss(t + 0.5, t)
    assert abs(loss - 0.25) < 1e-15
    assert np.allclose(dp, 2 * 0.5 / 12, rtol=0, atol=1e-16)
    loss0, dp0 = oracle.mse_loss(t, t)
    assert loss0 == 0.0 and not dp0.any()
    p = rnd((4, 3), 14)
    pt = torch.from_numpy(p).requires_grad_(True)
    lt = F.mse_loss(pt, torch.from_numpy(t))
    lt.backward()
    loss, dp = oracle.mse_loss(p, t)
    assert abs(loss - lt.item()) < 1e-14
    assert np.abs(dp - pt.grad.numpy()).max() < 1e-15


@pytest.mark.parametrize("alpha", [0.01, 0.2])
def test_head_finite_differences(alpha):
    """Central differences (h = 1e-6, fp64) of the head's loss -- three FC
    layers with bias + leaky ReLU, then the mean squared error -- against the
    oracle's backward, for entries of every weight, bias and the features."""
    rng = np.random.default_rng(15)
    M, widths = 3, [20, 8, 6, 3]
    feat = rng.standard_normal((M, widths[0]))
    ws = [rng.standard_normal((widths[i], widths[i + 1])) / np.sqrt(widths[i]) for i in range(3)]
    bs = [rng.normal(0, 0.1, widths[i + 1]) for i in range(3)]
    tgt = rng.standard_normal((M, 3))
    loss, dp, acts = oracle.head_forward(feat, ws, bs, alpha, tgt)
    # keep the finite difference away from the kink of every pre-activation
    for a in acts:
        zb = a["y"]
        assert np.abs(zb).min() > 1e-5  # every perturbation below moves z by < 4e-6
    grads, dfeat = oracle.head_backward(acts, ws, dp, alpha)
    h = 1e-6

    def f(feat_, ws_, bs_):
        return oracle.head_forward(feat_, ws_, bs_, alpha, tgt)[0]

    checks = []
    for li in range(3):
        for idx in [(0, 0), (widths[li] - 1, widths[li + 1] - 1), (widths[li] // 2, 1)]:
            wp = [w.copy() for w in ws]
            wm = [w.copy() for w in ws]
            wp[li][idx] += h
            wm[li][idx] -= h
            checks.append(((f(feat, wp, bs) - f(feat, wm, bs)) / (2 * h), grads[li]["dw"][idx]))
        for j in [0, widths[li + 1] - 1]:
            bp = [b.copy() for b in bs]
            bm = [b.copy() for b in bs]
            bp[li][j] += h
            bm[li][j] -= h
            checks.append(((f(feat, ws, bp) - f(feat, ws, bm)) / (2 * h), grads[li]["db"][j]))
    for idx in [(0, 0), (M - 1, widths[0] - 1), (1, 7)]:
        fp, fm = feat.copy(), feat.copy()
        fp[idx] += h
        fm[idx] -= h
        checks.append(((f(fp, ws, bs) - f(fm, ws, bs)) / (2 * h), dfeat[idx]))
    for fd, an in checks:
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (fd, an)


def test_head_matches_torch_autograd():
    """The same head built from torch's fp64 CPU ops (linear, leaky_relu,
    mse_loss) and differentiated by autograd."""
    rng = np.random.default_rng(16)
    M, widths, alpha = 4, [24, 10, 5, 3], 0.01
    feat = rng.standard_normal((M, widths[0]))
    ws = [rng.standard_normal((widths[i], widths[i + 1])) for i in range(3)]
    bs = [rng.normal(0, 0.1, widths[i + 1]) for i in range(3)]
    tgt = rng.standard_normal((M, 3))
    loss, dp, acts = oracle.head_forward(feat, ws, bs, alpha, tgt)
    grads, dfeat = oracle.head_backward(acts, ws, dp, alpha)
    ft = torch.from_numpy(feat).requires_grad_(True)
    wt = [torch.from_numpy(w).requires_grad_(True) for w in ws]
    bt = [torch.from_numpy(b).requires_grad_(True) for b in bs]
    h = ft
    for w, b in zip(wt, bt):
        h = F.leaky_relu(h @ w + b, alpha)
    lt = F.mse_loss(h, torch.from_numpy(tgt))
    lt.backward()
    assert abs(loss - lt.item()) <= 1e-13 * max(1.0, abs(loss))
    assert np.abs(dfeat - ft.grad.numpy()).max() < 1e-12
    for i in range(3):
        assert np.abs(grads[i]["dw"] - wt[i].grad.numpy()).max() < 1e-12
        assert np.abs(grads[i]["db"] - bt[i].grad.numpy()).max() < 1e-12
