"""Pins of the oracle's parameter update (Section III-B: Adam + LARC + linear
learning-rate decay) against what the paper and the mathematics fix: the
schedule's values at the paper's constants, Adam as implemented by
torch.optim.Adam (a different code, fp64 on the CPU), the closed forms of
Adam's first step and of a constant gradient, LARC's defining property (the
rescaled gradient's norm is coef times the weight norm), the fallback and
clip branches, invariance to the gradient's scale, and independence of the
groups.  No GPU."""
import numpy as np
import pytest
import torch

import oracle

B1, B2 = 0.9, 0.999


def _rand(n, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(n) * scale


def test_schedule_paper_values():
    td = 1000
    assert oracle.lr_schedule(0, td) == pytest.approx(2e-3, abs=1e-18)
    assert oracle.lr_schedule(td, td) == pytest.approx(1e-4, abs=1e-18)
    assert oracle.lr_schedule(td // 2, td) == pytest.approx(1.05e-3, abs=1e-18)
    assert oracle.lr_schedule(5 * td, td) == pytest.approx(1e-4, abs=1e-18)  # clamped after t_decay
    # linear: equal decrements of (eta0 - eta_min) / t_decay
    d = np.diff([oracle.lr_schedule(t, td) for t in range(0, td + 1, 50)])
    np.testing.assert_allclose(d, -1.9e-3 * 50 / td, rtol=1e-9)


def _torch_adam(v0, grads, lr, eps):
    p = torch.nn.Parameter(torch.tensor(v0, dtype=torch.float64))
    opt = torch.optim.Adam([p], lr=lr, betas=(B1, B2), eps=eps, foreach=False)
    out = []
    for g in grads:
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        st = opt.state[p]
        out.append((p.detach().numpy().copy(), st["exp_avg"].numpy().copy(), st["exp_avg_sq"].numpy().copy()))
    return out


NO_LARC = dict(larc_coef=1e300, larc_clip=1.0)  # eta* is huge, so the clip makes eta+ = 1 and g* = g


def test_pure_adam_matches_torch_over_steps():
    """LARC switched off, constant rate, eps_hat = 0: the epsilon-hat form and
    torch's form are then the same method."""
    n, lr = 37, 3e-3
    v = _rand(n, 1)
    grads = [_rand(n, 10 + k) for k in range(6)]
    ref = _torch_adam(v, grads, lr, 0.0)
    m = np.zeros(n)
    s = np.zeros(n)
    for t, g in enumerate(grads):
        v, m, s, dag = oracle.adam_larc_step([0, n], t, 10, v, g, m, s, eta0=lr, eta_min=lr, eps_hat=0.0, **NO_LARC)
        assert dag[0] == 1.0
        np.testing.assert_allclose(v, ref[t][0], rtol=1e-13, atol=1e-16)
        np.testing.assert_allclose(m, ref[t][1], rtol=1e-13, atol=1e-18)
        np.testing.assert_allclose(s, ref[t][2], rtol=1e-13, atol=1e-20)


def test_eps_hat_placement_first_step():
    """At step 1 eps_hat = eps * sqrt(1 - beta2) maps torch's epsilon (added
    to the bias-corrected root) onto the paper's epsilon-hat."""
    n, lr, eps_hat = 29, 1e-3, 1e-3
    v = _rand(n, 2)
    g = _rand(n, 3, 1e-3)  # comparable to eps so the placement matters
    ref = _torch_adam(v, [g], lr, eps_hat / np.sqrt(1 - B2))
    v1, m1, s1, _ = oracle.adam_larc_step([0, n], 0, 10, v, g, np.zeros(n), np.zeros(n),
                                          eta0=lr, eta_min=lr, eps_hat=eps_hat, **NO_LARC)
    np.testing.assert_allclose(v1, ref[0][0], rtol=1e-13, atol=1e-16)


def test_first_step_closed_form():
    """From zero moments, Adam's first step is eta0 * g* / (|g*| + eps_hat / sqrt(1 - beta2))
    element by element (paper's hyperparameters, LARC on)."""
    off = [0, 50, 130]
    v = _rand(130, 4, 0.05)
    g = _rand(130, 5, 3.0)
    v1, m1, s1, dag = oracle.adam_larc_step(off, 0, 100, v, g, np.zeros(130), np.zeros(130))
    for l in range(2):
        sl = slice(off[l], off[l + 1])
        gs = dag[l] * g[sl]
        step = 2e-3 * gs / (np.abs(gs) + 1e-8 / np.sqrt(1 - B2))
        np.testing.assert_allclose(v[sl] - v1[sl], step, rtol=1e-12, atol=1e-20)


def test_larc_rescaled_gradient_norm():
    """Unclipped: ||g*|| = coef * ||v|| per group, read back from the first
    moment after one step from zero (m = (1 - beta1) g*)."""
    off = [0, 7, 7, 100, 1000]  # includes an empty group
    v = _rand(1000, 6, 0.1)
    g = _rand(1000, 7, 50.0)
    _, m1, _, dag = oracle.adam_larc_step(off, 0, 100, v, g, np.zeros(1000), np.zeros(1000))
    for l in (0, 2, 3):
        sl = slice(off[l], off[l + 1])
        assert dag[l] < 1.0
        assert np.linalg.norm(m1[sl]) / (1 - B1) == pytest.approx(0.002 * np.linalg.norm(v[sl]), rel=1e-12)
    assert dag[1] == pytest.approx(6.25e-5)  # empty group: both norms are zero


def test_gradient_scale_invariance():
    """While the clip does not bind, the update does not depend on the
    gradient's scale (the trust ratio divides it out)."""
    off = [0, 64, 200]
    v = _rand(200, 8, 0.1)
    g = _rand(200, 9, 10.0)
    m0 = _rand(200, 10, 1e-3)
    s0 = np.abs(_rand(200, 11, 1e-6))
    a = oracle.adam_larc_step(off, 3, 100, v, g, m0, s0)
    b = oracle.adam_larc_step(off, 3, 100, v, 1000.0 * g, m0, s0)
    for x, y in zip(a[:3], b[:3]):
        np.testing.assert_allclose(x, y, rtol=1e-12, atol=1e-22)
    np.testing.assert_allclose(a[3], 1000.0 * b[3], rtol=1e-12)


def test_clip_binds_for_small_gradients():
    """coef * ||v|| / ||g|| > 1: eta+ = 1 and the update is plain Adam on g."""
    n = 40
    v = _rand(n, 12)
    g = _rand(n, 13, 1e-6)
    v1, m1, s1, dag = oracle.adam_larc_step([0, n], 0, 100, v, g, np.zeros(n), np.zeros(n))
    assert dag[0] == 1.0
    ref = _torch_adam(v, [g], 2e-3, 1e-8 / np.sqrt(1 - B2))
    np.testing.assert_allclose(v1, ref[0][0], rtol=1e-13, atol=1e-16)


def test_fallback_branches():
    n = 16
    # zero gradient: eta+ = 6.25e-5, the moments only decay
    v = _rand(n, 14)
    m0 = _rand(n, 15, 1e-3)
    s0 = np.abs(_rand(n, 16, 1e-6))
    _, m1, s1, dag = oracle.adam_larc_step([0, n], 2, 100, v, np.zeros(n), m0, s0)
    assert dag[0] == 6.25e-5
    np.testing.assert_array_equal(m1, B1 * m0)
    np.testing.assert_array_equal(s1, B2 * s0)
    # zero weights (a bias at initialisation): eta+ = 6.25e-5 scales the gradient
    g = _rand(n, 17)
    _, m1, s1, dag = oracle.adam_larc_step([0, n], 0, 100, np.zeros(n), g, np.zeros(n), np.zeros(n))
    assert dag[0] == 6.25e-5
    np.testing.assert_allclose(m1, (1 - B1) * 6.25e-5 * g, rtol=1e-15)
    np.testing.assert_allclose(s1, (1 - B2) * (6.25e-5 * g) ** 2, rtol=1e-14)


def test_constant_gradient_closed_form():
    """A constant gradient c with LARC off: the moments are c(1 - beta1^k) and
    c^2(1 - beta2^k), so step k moves v by eta_t c sqrt(1-b2^k) / (|c| sqrt(1-b2^k) + eps_hat),
    with eta_t on the paper's decay."""
    n, td, eps_hat = 5, 20, 1e-4
    c = np.array([1.0, -2.0, 0.5, 3e-5, -1e-3])
    v = np.ones(n)  # nonzero: zero weights would take the fallback branch
    m = np.zeros(n)
    s = np.zeros(n)
    for t in range(25):
        v0 = v
        v, m, s, _ = oracle.adam_larc_step([0, n], t, td, v, c, m, s, eps_hat=eps_hat, **NO_LARC)
        k = t + 1
        eta = 2e-3 - 1.9e-3 * min(t, td) / td
        r = np.sqrt(1 - B2 ** k)
        np.testing.assert_allclose(v0 - v, eta * c * r / (np.abs(c) * r + eps_hat), rtol=1e-9)


def test_groups_are_independent():
    """Updating groups together equals updating each group alone."""
    sizes = [13, 0, 64, 1, 200]
    off = np.concatenate([[0], np.cumsum(sizes)])
    N = off[-1]
    v = _rand(N, 18, 0.1)
    g = _rand(N, 19)
    m0 = _rand(N, 20, 1e-2)
    s0 = np.abs(_rand(N, 21, 1e-4))
    joint = oracle.adam_larc_step(off, 7, 50, v, g, m0, s0)
    for l in range(len(sizes)):
        sl = slice(off[l], off[l + 1])
        n = sizes[l]
        alone = oracle.adam_larc_step([0, n], 7, 50, v[sl], g[sl], m0[sl], s0[sl])
        for x, y in zip(joint[:3], alone[:3]):
            np.testing.assert_array_equal(x[sl], y)
        assert joint[3][l] == alone[3][0]
