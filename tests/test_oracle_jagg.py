"""Pins for the JAGG steps of the oracle: Eq. alpha, Eq. s_base/s_corr,
Theorem 1 and its Corollary on a linear toy, the W = 2 degenerate case, the
PPO-clip remark, the joint/sequential identity, and the routing rule against
the gradient-quality table.  CPU only."""
import json
import os

import numpy as np
import pytest

import synth
from oracle import jagg, mmdit

from test_oracle_model import TINY, TINY_BLOCK, cot, inputs, theta

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "jagg_quality.json")


# ------------------------------------------------------------------ alpha
def test_alpha_endpoints_monotone_and_uniform_grid():
    t = synth.uniform_grid(8)[:4]  # 1, .875, .75, .625
    a = jagg.alpha(t)
    assert a[0] == 0.0 and a[-1] == 1.0
    np.testing.assert_allclose(a, [0, 1 / 3, 2 / 3, 1], rtol=0, atol=1e-15)
    # unshifted uniform spacing gives j/(W-1) (remark on timestep shift)
    for W in (2, 3, 4, 5, 8):
        tt = synth.uniform_grid(40)[7:7 + W]
        np.testing.assert_allclose(jagg.alpha(tt), np.arange(W) / (W - 1), rtol=0, atol=1e-14)
    # a shifted (non-uniform) decreasing schedule is still monotone in [0, 1]
    ts = 3 * t / (1 + 2 * t)
    a = jagg.alpha(ts)
    assert a[0] == 0.0 and a[-1] == 1.0 and np.all(np.diff(a) > 0)


def test_alpha_rejects_degenerate_windows():
    with pytest.raises(ValueError):
        jagg.alpha([0.5])
    with pytest.raises(ValueError):
        jagg.alpha([0.5, 0.3, 0.5])


# ------------------------------------------------------------ composites
def test_composites_sum_to_total_and_w2_is_identity():
    s = [synth.normal((5, 7), 100 + j) for j in range(4)]
    t = synth.uniform_grid(8)[4:]
    sb, sc = jagg.aggregate(s, t)
    np.testing.assert_allclose(sb + sc, sum(s), rtol=1e-14, atol=1e-14)
    # weights: s_base gets 1, 2/3, 1/3, 0 of each step
    np.testing.assert_allclose(sb, s[0] + (2 / 3) * s[1] + (1 / 3) * s[2], rtol=1e-14, atol=1e-14)
    # W = 2: (s_base, s_corr) = (s_0, s_1) exactly
    sb, sc = jagg.aggregate(s[:2], [0.9, 0.4])
    assert np.array_equal(sb, s[0]) and np.array_equal(sc, s[1])


# -------------------------------------------------------------- Theorem 1
def _toy(n=64, seed=5):
    rs = np.random.default_rng(seed)
    return jagg.LinearToy(0.02 * rs.standard_normal((n, n)), 0.02 * rs.standard_normal(n),
                          0.02 * rs.standard_normal(n))


def test_theorem1_linear_toy_on_path_is_exact():
    toy = _toy()
    t = synth.uniform_grid(8)[:4]
    a = jagg.alpha(t)
    z0, z1 = synth.normal(64, 1), synth.normal(64, 2)
    zs = [(1 - aj) * z0 + aj * z1 for aj in a]
    ss = [synth.normal(64, 10 + j) for j in range(4)]
    ge, gj = toy.g_exact(zs, t, ss), toy.g_jagg(zs, t, ss)
    for x, y in zip(ge, gj):
        np.testing.assert_allclose(y, x, rtol=1e-12, atol=1e-14)
    # shifted timesteps with z on the same affine path in alpha: still exact
    ts = 3 * t / (1 + 2 * t)
    a = jagg.alpha(ts)
    zs = [(1 - aj) * z0 + aj * z1 for aj in a]
    for x, y in zip(toy.g_exact(zs, ts, ss), toy.g_jagg(zs, ts, ss)):
        np.testing.assert_allclose(y, x, rtol=1e-12, atol=1e-14)


def test_theorem1_off_path_negative_control():
    """Off the affine path the A-gradient differs, but the b and c gradients
    stay exact (the weights sum to one and t is on its own affine grid)."""
    toy = _toy()
    t = synth.uniform_grid(8)[:4]
    zs = [synth.normal(64, 20 + j) for j in range(4)]
    ss = [synth.normal(64, 30 + j) for j in range(4)]
    (dA_e, db_e, dc_e), (dA_j, db_j, dc_j) = toy.g_exact(zs, t, ss), toy.g_jagg(zs, t, ss)
    np.testing.assert_allclose(db_j, db_e, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dc_j, dc_e, rtol=1e-12, atol=1e-14)
    assert np.linalg.norm(dA_j - dA_e) > 0.1 * np.linalg.norm(dA_e)


# ----------------------------------------------------------- MMDiT groups
def _window(cfg, W, seed, B=1):
    t = synth.uniform_grid(2 * W)[:W]
    inps = [jagg.step_inputs(inputs(cfg, B, seed + 7 * j), t[j]) for j in range(W)]
    ss = [cot(cfg, B, seed + 100 + 7 * j) for j in range(W)]
    return t, inps, ss


def _flat(cfg, G):
    return mmdit.flatten(cfg, G)


@pytest.mark.parametrize("cfg", [TINY, TINY_BLOCK], ids=["full", "block_only"])
def test_w2_jagg_equals_exact(cfg):
    P = mmdit.unflatten(cfg, theta(cfg))
    t, inps, ss = _window(cfg, 2, 300)
    np.testing.assert_allclose(_flat(cfg, jagg.g_jagg(cfg, P, inps, ss, t)),
                               _flat(cfg, jagg.g_exact(cfg, P, inps, ss)), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("cfg", [TINY, TINY_BLOCK], ids=["full", "block_only"])
def test_joint_equals_sequential_and_zero_step_is_dropped(cfg):
    """One backward over the endpoint pair equals two endpoint backwards
    (implementation-variants section); a clipped step (s_j = 0) contributes
    nothing (PPO-clip remark)."""
    P = mmdit.unflatten(cfg, theta(cfg))
    W = 4
    t, inps, ss = _window(cfg, W, 400)
    gj = _flat(cfg, jagg.g_jagg(cfg, P, inps, ss, t))
    sb, sc = jagg.aggregate_any(ss, t)
    seq = jagg.g_exact(cfg, P, [inps[0], inps[-1]], [sb, sc])
    np.testing.assert_allclose(gj, _flat(cfg, seq), rtol=1e-12, atol=1e-13)
    zero = tuple(np.zeros_like(a) for a in ss[1]) if isinstance(ss[1], tuple) else np.zeros_like(ss[1])
    ss0 = [ss[0], zero, ss[2], ss[3]]
    t3 = [t[0], t[2], t[3]]
    # with s_1 = 0 the composites equal those of the remaining steps at their alphas
    sb0, sc0 = jagg.aggregate_any(ss0, t)
    a = jagg.alpha(t)
    want_b = [(1 - a[j]) for j in (0, 2, 3)]
    if not isinstance(sb0, tuple):
        np.testing.assert_allclose(sb0, sum(w * ss[j] for w, j in zip(want_b, (0, 2, 3))), rtol=1e-14, atol=1e-14)
    ge0 = _flat(cfg, jagg.g_exact(cfg, P, inps, ss0))
    ge3 = _flat(cfg, jagg.g_exact(cfg, P, [inps[0], inps[2], inps[3]], [ss[0], ss[2], ss[3]]))
    np.testing.assert_allclose(ge0, ge3, rtol=1e-12, atol=1e-13)
    assert len(t3) == 3


def test_final_bias_is_exact_under_jagg():
    """d(final.b) does not depend on the input, so JAGG reproduces it exactly."""
    cfg = TINY
    P = mmdit.unflatten(cfg, theta(cfg))
    t, inps, ss = _window(cfg, 4, 500)
    gj, ge = jagg.g_jagg(cfg, P, inps, ss, t), jagg.g_exact(cfg, P, inps, ss)
    np.testing.assert_allclose(gj["final.b"], ge["final.b"], rtol=1e-12, atol=1e-13)
    assert np.linalg.norm(_flat(cfg, gj) - _flat(cfg, ge)) > 1e-6 * np.linalg.norm(_flat(cfg, ge))


# ---------------------------------------------------------------- routing
def test_routing_reproduces_gradient_quality_table():
    g = json.load(open(GOLDEN))
    tau = g["tau"]
    for name, m in g["models"].items():
        mask, frac = jagg.route(len(m["cos"]), scores=m["cos"], tau=tau)
        assert int(mask.sum()) == m["literal_rule_prefix"], name
        assert list(mask) == [1] * m["literal_rule_prefix"] + [0] * (5 - m["literal_rule_prefix"])
    # QwenImage: the rule yields exactly the paper's jagg_frac of 0.6
    _, frac = jagg.route(5, scores=g["models"]["QwenImage"]["cos"], tau=tau)
    assert frac == g["models"]["QwenImage"]["paper_chosen_frac"]
    for case in g["static_frac"]:
        mask, frac = jagg.route(case["n_groups"], frac=case["frac"])
        assert int(mask.sum()) == case["n_jagg"]


def test_routing_edges():
    assert list(jagg.route(4, scores=[0.9, 0.8, 0.7, 0.6])[0]) == [1, 1, 1, 1]
    assert list(jagg.route(4, scores=[0.4, 0.8, 0.7, 0.6])[0]) == [0, 0, 0, 0]
    # prefix only: a later qualifying group after a failing one is not routed
    assert list(jagg.route(4, scores=[0.9, 0.3, 0.9, 0.9])[0]) == [1, 0, 0, 0]
    assert list(jagg.route(3, scores=[0.5, 0.5, np.nextafter(0.5, 0)])[0]) == [1, 1, 0]
    assert list(jagg.route(4, frac=0.6)[0]) == [1, 1, 0, 0]
    assert list(jagg.route(2, frac=0.5)[0]) == [1, 0]
    assert jagg.route(3, frac=1.0)[1] == 1.0 and jagg.route(3, frac=0.0)[1] == 0.0
    with pytest.raises(ValueError):
        jagg.route(0, frac=0.5)


def test_group_score_closed_form():
    for rho in (0.5, 0.73, 0.99):
        h = synth.hidden_profile(4, 257, rho, seed=int(rho * 100))
        assert abs(jagg.group_score(list(h)) - rho) < 1e-13
        # invariance to positive rescaling of each step
        assert abs(jagg.group_score([h[0] * 3, h[1], h[2] * 0.1, h[3]]) - rho) < 1e-13


def test_windows_with_tail():
    full, tail = jagg.windows(20, 8)
    assert full == [list(range(8)), list(range(8, 16))] and tail == [16, 17, 18, 19]
    full, tail = jagg.windows(16, 4)
    assert len(full) == 4 and tail == []


def test_alpha_rejects_non_monotone_windows():
    with pytest.raises(ValueError):
        jagg.alpha([0.9, 0.95, 0.3])
    with pytest.raises(ValueError):
        jagg.alpha([0.3, 0.5])  # increasing


# ---------------------------------------------------------------- ablation
def test_ablate_is_the_endpoint_only_backward():
    """Endpoint-only ablation (Experiments): the gradient of
    <v(z_0, t_0), s_0> + <v(z_{W-1}, t_{W-1}), s_{W-1}> with weight one each,
    checked against central finite differences of that scalar in random
    parameter directions.  It equals JAGG when the middle signals vanish
    (then s_base = s_0 and s_corr = s_{W-1}) and differs otherwise."""
    from test_oracle_model import loss
    cfg = TINY
    th = theta(cfg)
    P = mmdit.unflatten(cfg, th)
    W = 4
    t, inps, ss = _window(cfg, W, 600)
    ga = _flat(cfg, jagg.g_ablate(cfg, P, inps, ss))
    rs = np.random.default_rng(7)
    h = 1e-5
    for _ in range(4):
        d = rs.standard_normal(ga.shape[0])
        f = lambda x: loss(cfg, x, inps[0], ss[0]) + loss(cfg, x, inps[W - 1], ss[W - 1])  # noqa: E731
        fd = (f(th + h * d) - f(th - h * d)) / (2 * h)
        assert abs(fd - float(np.dot(ga, d))) <= 1e-7 * max(1.0, abs(fd))
    zero = np.zeros_like(ss[1])
    ss0 = [ss[0], zero, zero, ss[3]]
    np.testing.assert_allclose(_flat(cfg, jagg.g_jagg(cfg, P, inps, ss0, t)), ga, rtol=1e-12, atol=1e-13)
    gj = _flat(cfg, jagg.g_jagg(cfg, P, inps, ss, t))
    assert np.linalg.norm(gj - ga) > 1e-2 * np.linalg.norm(ga)


# ------------------------------------------------------------- trajectory
def _traj(cfg, T, seed, B=1):
    t = synth.uniform_grid(T)
    inps = [jagg.step_inputs(inputs(cfg, B, seed + 7 * j), t[j]) for j in range(T)]
    ss = [cot(cfg, B, seed + 500 + 7 * j) for j in range(T)]
    return t, inps, ss


def _batched_vjp(cfg, th, inps, ss):
    """One VJP over all steps stacked as one batch (batch additivity)."""
    cat = lambda xs: None if xs[0] is None else np.concatenate(xs, axis=0)  # noqa: E731
    inp = mmdit.Inputs(t=np.concatenate([i.t for i in inps]), z=cat([i.z for i in inps]),
                       txt=cat([i.txt for i in inps]), x_txt=cat([i.x_txt for i in inps]),
                       x_img=cat([i.x_img for i in inps]))
    return mmdit.vjp_flat(cfg, th, inp, np.concatenate(ss, axis=0))


def test_trajectory_per_step_and_w2_equal_one_batched_vjp():
    """All windows per step (and W = 2, where JAGG is exact) give the plain
    gradient of the whole trajectory, here formed as a single VJP of all T
    steps stacked as one batch: every step, the tail included, counted once."""
    cfg = TINY
    th = theta(cfg)
    P = mmdit.unflatten(cfg, th)
    T = 7
    t, inps, ss = _traj(cfg, T, 700)
    want = _batched_vjp(cfg, th, inps, ss)
    m, g = jagg.trajectory(cfg, P, inps, ss, t, 3, frac=0.0)     # windows [0..2], [3..5], tail [6]
    assert list(m) == [0, 0]
    np.testing.assert_allclose(_flat(cfg, g), want, rtol=1e-11, atol=1e-12)
    m, g = jagg.trajectory(cfg, P, inps, ss, t, 2, frac=1.0)     # 3 JAGG windows of 2, tail [6]
    assert list(m) == [1, 1, 1]
    np.testing.assert_allclose(_flat(cfg, g), want, rtol=1e-11, atol=1e-12)


def test_trajectory_final_bias_exact_and_routing_matters():
    cfg = TINY
    th = theta(cfg)
    P = mmdit.unflatten(cfg, th)
    T, W = 10, 4                                               # windows [0..3], [4..7], tail [8, 9]
    t, inps, ss = _traj(cfg, T, 800)
    _, g_j = jagg.trajectory(cfg, P, inps, ss, t, W, mask=[1, 1])
    _, g_e = jagg.trajectory(cfg, P, inps, ss, t, W, mask=[0, 0])
    want_b = sum(mmdit.patchify(cfg, s).sum(axis=(0, 1)) for s in ss)
    np.testing.assert_allclose(g_j["final.b"], want_b, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(g_e["final.b"], want_b, rtol=1e-12, atol=1e-13)
    fj, fe = _flat(cfg, g_j), _flat(cfg, g_e)
    assert np.linalg.norm(fj - fe) > 1e-3 * np.linalg.norm(fe)
    # a mixed mask changes only its window: (JAGG, per step) - (per step, per step)
    # equals (JAGG, JAGG) - (per step, JAGG)
    _, g_10 = jagg.trajectory(cfg, P, inps, ss, t, W, mask=[1, 0])
    _, g_01 = jagg.trajectory(cfg, P, inps, ss, t, W, mask=[0, 1])
    np.testing.assert_allclose(_flat(cfg, g_10) - fe, fj - _flat(cfg, g_01), rtol=1e-9, atol=1e-12)


def test_trajectory_linear_toy_exact_on_each_windows_path():
    """Theorem 1 window by window: when every window's latents lie on its own
    affine path in alpha, the all-JAGG trajectory gradient (tail per step)
    equals the exact one; off the paths it does not."""
    toy = _toy()
    T, W = 10, 4
    t = synth.uniform_grid(T)
    zs = []
    for g in range(T // W):
        a = jagg.alpha(t[g * W:(g + 1) * W])
        za, zb = synth.normal(64, 40 + g), synth.normal(64, 50 + g)
        zs += [(1 - aj) * za + aj * zb for aj in a]
    zs += [synth.normal(64, 60 + k) for k in range(T % W)]
    ss = [synth.normal(64, 70 + k) for k in range(T)]
    ge = toy.g_exact(zs, t, ss)
    for x, y in zip(ge, toy.trajectory(zs, t, ss, W, [1, 1])):
        np.testing.assert_allclose(y, x, rtol=1e-12, atol=1e-14)
    zs_off = [synth.normal(64, 90 + k) for k in range(T)]
    dA = toy.trajectory(zs_off, t, ss, W, [1, 1])[0] - toy.g_exact(zs_off, t, ss)[0]
    assert np.linalg.norm(dA) > 0.1 * np.linalg.norm(toy.g_exact(zs_off, t, ss)[0])


def test_trajectory_plan_routing_and_tail():
    """T = 20, W = 8: two full windows and a 4-step per-step tail; with half
    the windows falling back, window 0 (highest noise) takes JAGG.  T = 20,
    W = 4 with the gradient-quality table's QwenImage cosines: 3 JAGG windows."""
    plan = jagg.trajectory_plan(20, 8, jagg.route(2, frac=0.5)[0])
    assert plan == [(list(range(8)), True), (list(range(8, 16)), False), ([16, 17, 18, 19], False)]
    g = json.load(open(GOLDEN))
    m, _ = jagg.route(5, scores=g["models"]["QwenImage"]["cos"], tau=g["tau"])
    plan = jagg.trajectory_plan(20, 4, m)
    assert [u for _, u in plan] == [True, True, True, False, False] and plan[-1][0] == [16, 17, 18, 19]
    with pytest.raises(ValueError):
        jagg.trajectory_plan(20, 8, [1, 0, 1])
    with pytest.raises(ValueError):
        jagg.trajectory(TINY, None, [None] * 3, [None] * 3, [0.5, 0.6, 0.1], 2)
