"""Pins of the Phase-2 oracle (oracle.grpo): the closed-form upstream gradient
s_j = dL_j/dv_j of the PPO-clipped GRPO step loss (Eq. grpo_loss, Eq. logprob,
rectified-flow Euler mean) against central finite differences of L_j, against
torch autograd of the loss written with library ops, the PPO-clip remark's
exact zero for clipped steps, the advantage clamp, and a hand-evaluated case."""
import numpy as np
import pytest
import torch

import synth
from oracle import grpo, jagg


def case(B=2, n=6, seed=0):
    g = synth.rng(seed)
    z = g.standard_normal((B, n))
    zn = g.standard_normal((B, n))
    v = g.standard_normal((B, n))
    return z, zn, v


def logp_old_for(z, zn, v, t, tn, sigma, rho_target):
    """Old log-probability that puts the ratio at rho_target (rho = exp(lp - lp_old))."""
    lp = grpo.log_prob(zn, grpo.rf_mean(z, v, t, tn), sigma)
    return lp - np.log(rho_target)


# (A per sample, target ratios): unclipped inside the range, and both clip sides
CASES = [
    (np.array([1.3, -0.7]), np.array([1.0, 1.0])),
    (np.array([1.3, -0.7]), np.array([1.05, 0.93])),
    (np.array([1.3, -0.7]), np.array([1.4, 1.4])),    # A>0 clipped (0), A<0 unclipped
    (np.array([1.3, -0.7]), np.array([0.6, 0.6])),    # A>0 unclipped, A<0 clipped (0)
    (np.array([7.0, -9.0]), np.array([1.02, 0.99])),  # advantages beyond the clamp
]


@pytest.mark.parametrize("A,rho", CASES)
def test_upstream_grad_matches_finite_differences(A, rho):
    z, zn, v = case()
    t, tn, sigma, eps, W, ac = 0.8, 0.7, 0.35, 0.1, 4, 5.0
    lpo = logp_old_for(z, zn, v, t, tn, sigma, rho)
    s = grpo.upstream_grad(z, zn, v, t, tn, sigma, lpo, A, eps, W, ac)
    h = 1e-6
    fd = np.zeros_like(v)
    for b in range(v.shape[0]):
        for e in range(v.shape[1]):
            vp, vm = v.copy(), v.copy()
            vp[b, e] += h
            vm[b, e] -= h
            lp_ = grpo.step_loss(z, zn, vp, t, tn, sigma, lpo, A, eps, W, ac)[b]
            lm_ = grpo.step_loss(z, zn, vm, t, tn, sigma, lpo, A, eps, W, ac)[b]
            fd[b, e] = (lp_ - lm_) / (2 * h)
    assert np.allclose(s, fd, rtol=1e-6, atol=1e-9)


def test_clipped_step_has_exactly_zero_gradient():
    """PPO-clip remark: outside the clip range on the clipped side, s_j = 0."""
    z, zn, v = case()
    A = np.array([2.0, -2.0])
    rho = np.array([1.5, 0.5])  # A>0 above 1+eps, A<0 below 1-eps
    lpo = logp_old_for(z, zn, v, 0.9, 0.8, 0.4, rho)
    s = grpo.upstream_grad(z, zn, v, 0.9, 0.8, 0.4, lpo, A, 0.1, 4, 5.0)
    assert np.all(s == 0.0)


def test_matches_torch_autograd_of_the_loss():
    z, zn, v = case(B=3, n=10, seed=3)
    A = np.array([0.9, -1.7, 6.0])
    t, tn, sigma, eps, W, ac = 0.6, 0.55, 0.2, 0.1, 5, 5.0
    lpo = logp_old_for(z, zn, v, t, tn, sigma, np.array([1.02, 1.3, 0.95]))
    vt = torch.tensor(v, dtype=torch.float64, requires_grad=True)
    mu = torch.tensor(z) + vt * (tn - t)
    d = torch.tensor(zn) - mu
    n = v.shape[1]
    lp = -(d * d).sum(1) / (2 * sigma ** 2) - n * np.log(np.sqrt(2 * np.pi) * sigma)
    rho = torch.exp(lp - torch.tensor(lpo))
    Ac = torch.clamp(torch.tensor(A), -ac, ac)
    L = torch.maximum(-Ac * rho, -Ac * torch.clamp(rho, 1 - eps, 1 + eps)) / W
    L.sum().backward()
    s = grpo.upstream_grad(z, zn, v, t, tn, sigma, lpo, A, eps, W, ac)
    assert np.allclose(s, vt.grad.numpy(), rtol=1e-10, atol=1e-13)


def test_hand_evaluated_unit_ratio():
    """rho = 1, A = 1: s_j = -(1/W) (z_{j+1} - z_j - v_j dt) dt / sigma^2."""
    z = np.array([[0.5, -1.0]])
    zn = np.array([[0.25, 0.0]])
    v = np.array([[1.0, 2.0]])
    t, tn, sigma, W = 1.0, 0.75, 0.5, 4
    lpo = grpo.log_prob(zn, grpo.rf_mean(z, v, t, tn), sigma)
    s = grpo.upstream_grad(z, zn, v, t, tn, sigma, lpo, np.array([1.0]), 0.1, W, 5.0)
    # mu = z + v * (-0.25) = [0.25, -1.5]; r = zn - mu = [0, 1.5]; dt / sigma^2 = -1
    assert np.allclose(s, [[0.0, 1.5 / 4.0]])


def test_window_composites_sum_to_the_step_sum():
    W, B, n = 4, 2, 8
    g = synth.rng(11)
    zs = [g.standard_normal((B, n)) for _ in range(W + 1)]
    vs = [g.standard_normal((B, n)) for _ in range(W)]
    ts = synth.uniform_grid(8)[:W + 1]
    sig = 0.3 + 0.1 * np.arange(W)
    lpo = [grpo.log_prob(zs[j + 1], grpo.rf_mean(zs[j], vs[j], ts[j], ts[j + 1]), sig[j]) - 0.05 * (j - 1)
           for j in range(W)]
    A = np.array([0.8, -1.1])
    sb, sc = grpo.window_composites(zs, vs, ts, sig, lpo, A, 0.1, 5.0)
    s = grpo.window_upstream(zs, vs, ts, sig, lpo, A, 0.1, 5.0)
    assert np.allclose(sb + sc, sum(s), atol=1e-14)
    assert np.allclose(sc, sum(a * x for a, x in zip(jagg.alpha(ts[:W]), s)), atol=1e-14)
