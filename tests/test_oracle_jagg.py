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
