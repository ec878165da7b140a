"""Oracle for the JAGG steps: interpolation weights, composites, group gradients,
routing and group scores, plus the linear-velocity toy of Theorem 1.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).  Each function follows the
paper's steps in its order and notation:

* alpha_j = (t_0 - t_j) / (t_0 - t_{W-1})                       (Eq. alpha)
* s_base = sum_j (1 - alpha_j) s_j,  s_corr = sum_j alpha_j s_j   (Eq. s_base/s_corr)
* g_jagg = J_0^T s_base + J_{W-1}^T s_corr, one backward over the
  endpoint pair                                   (Phase 4; Corollary of Thm 1)
* g_exact = sum_j J_j^T s_j with the same detach of z_j   (per-step baseline,
  Phase 2 remark and the gradient-quality appendix)
* routing: groups ordered from high to low noise; the first fraction use JAGG
  (high-noise vs low-noise scheduling); calibrated by cos >= 0.5
  (gradient-quality appendix);
* trajectory: the routed windows take g_jagg, the others and the T mod W tail
  take g_exact, summed over the trajectory (gradient accumulation over groups).
"""
from __future__ import annotations

import numpy as np

from . import mmdit


# ---------------------------------------------------------------- Eq. alpha
def alpha(t) -> np.ndarray:
    """Interpolation coefficients of one window, in fp64.

    A window is W consecutive denoising steps, which run from high noise to low
    noise, so its timesteps are strictly decreasing (reading of the problem
    statement: sampling integrates from t = 1 towards t = 0).  Raises
    ValueError when W < 2 or t is not strictly decreasing (which includes
    t_0 == t_{W-1}, where the weights are undefined)."""
    t = np.asarray(t, dtype=np.float64)
    W = t.shape[0]
    if W < 2:
        raise ValueError("a window needs at least two timesteps")
    if not np.all(t[1:] < t[:-1]):
        raise ValueError("the timesteps of a window must be strictly decreasing")
    den = t[0] - t[W - 1]
    return (t[0] - t) / den


# ------------------------------------------------------ Eq. s_base / s_corr
def aggregate(s_list, t, acc_dtype=np.float64):
    """Composite upstream gradients, accumulated in j order in ``acc_dtype``."""
    a = alpha(t).astype(acc_dtype)
    one = acc_dtype(1.0)
    s_base = np.zeros(np.shape(s_list[0]), dtype=acc_dtype)
    s_corr = np.zeros(np.shape(s_list[0]), dtype=acc_dtype)
    for j, s in enumerate(s_list):
        s = np.asarray(s, dtype=acc_dtype)
        s_base = s_base + (one - a[j]) * s
        s_corr = s_corr + a[j] * s
    return s_base, s_corr


# -------------------------------------------------- group gradients (MMDiT)
def pair_inputs(cfg, inp0: mmdit.Inputs, inp1: mmdit.Inputs) -> mmdit.Inputs:
    """The endpoint pair as one batch-2B input (endpoint 0 first)."""
    def cat(a, b):
        return None if a is None else np.concatenate([a, b], axis=0)
    return mmdit.Inputs(t=cat(inp0.t, inp1.t), z=cat(inp0.z, inp1.z), txt=cat(inp0.txt, inp1.txt),
                        x_txt=cat(inp0.x_txt, inp1.x_txt), x_img=cat(inp0.x_img, inp1.x_img))


def step_inputs(inp: mmdit.Inputs, t_scalar: float) -> mmdit.Inputs:
    B = (inp.z if inp.z is not None else inp.x_img).shape[0]
    return mmdit.Inputs(t=np.full(B, t_scalar), z=inp.z, txt=inp.txt, x_txt=inp.x_txt, x_img=inp.x_img)


def aggregate_any(s_list, t):
    """aggregate() for plain arrays or for (txt, img) tuples (block-only model)."""
    if isinstance(s_list[0], tuple):
        parts = [aggregate([s[c] for s in s_list], t) for c in range(len(s_list[0]))]
        return tuple(p[0] for p in parts), tuple(p[1] for p in parts)
    return aggregate(s_list, t)


def g_jagg(cfg, P, inputs, s_list, t):
    """JAGG group gradient: composites (Eq. s_base/s_corr) then one backward over
    the batched endpoint pair [v_0, v_{W-1}] with cotangents [s_base, s_corr]."""
    W = len(inputs)
    s_base, s_corr = aggregate_any(s_list, t)
    dt = P["t_in.w"].dtype
    if isinstance(s_base, tuple):
        cot = tuple(np.concatenate([b.astype(dt), c.astype(dt)], axis=0) for b, c in zip(s_base, s_corr))
    else:
        cot = np.concatenate([s_base.astype(dt), s_corr.astype(dt)], axis=0)
    pair = pair_inputs(cfg, inputs[0], inputs[W - 1])
    _, cache = mmdit.forward(cfg, P, pair)
    return mmdit.vjp(cfg, P, cache, cot)


def g_exact(cfg, P, inputs, s_list):
    """Per-step baseline: sum_j J_j^T s_j, one backward per step."""
    total = None
    for inp, s in zip(inputs, s_list):
        _, cache = mmdit.forward(cfg, P, inp)
        G = mmdit.vjp(cfg, P, cache, s)
        total = G if total is None else {k: total[k] + G[k] for k in total}
    return total


def g_ablate(cfg, P, inputs, s_list):
    """Ablate variant (Experiments): endpoint-only signals with equal weight,
    backward on [v_0, v_{W-1}] with [s_0, s_{W-1}]."""
    W = len(inputs)
    return g_exact(cfg, P, [inputs[0], inputs[W - 1]], [s_list[0], s_list[W - 1]])


# ---------------------------------------------------------------- routing
def route(n_groups: int, frac: float | None = None, scores=None, tau: float = 0.5):
    """Which groups take the JAGG backward.

    Static mode (frac given): the first floor(frac * n_groups + 1e-6) groups,
    high-noise first.  Score mode (scores given): the longest prefix whose
    scores are all >= tau.  Returns (uint8 mask, realised fraction)."""
    if n_groups <= 0:
        raise ValueError("n_groups must be positive")
    if frac is not None:
        if not (0.0 <= frac <= 1.0):
            raise ValueError("frac must lie in [0, 1]")
        n = int(np.floor(frac * n_groups + 1e-6))
    else:
        n = 0
        for s in scores:
            if not (float(s) >= tau):
                break
            n += 1
    mask = np.zeros(n_groups, dtype=np.uint8)
    mask[:n] = 1
    return mask, n / n_groups


def group_score(h_list) -> float:
    """Mean pairwise cosine similarity of the W per-step vectors (fp64, pair order
    (0,1), (0,2), ..., (W-2, W-1))."""
    hs = [np.asarray(h, dtype=np.float64).reshape(-1) for h in h_list]
    W = len(hs)
    tot = 0.0
    cnt = 0
    for i in range(W):
        for j in range(i + 1, W):
            tot += float(np.dot(hs[i], hs[j]) / (np.linalg.norm(hs[i]) * np.linalg.norm(hs[j])))
            cnt += 1
    return tot / cnt


def windows(T: int, W: int):
    """Split steps 0..T-1 into full windows of W plus a tail of T mod W steps."""
    full = [list(range(g * W, (g + 1) * W)) for g in range(T // W)]
    tail = list(range((T // W) * W, T))
    return full, tail


# ------------------------------------------------------------- trajectory
def trajectory_plan(T: int, W: int, mask):
    """The backward passes of a whole trajectory of T steps (high-noise vs
    low-noise scheduling): steps are taken in sampling order, i.e. from high to
    low noise; they form floor(T / W) full windows, window g takes the JAGG
    backward when mask[g] is 1 and the per-step backward otherwise, and the
    last T mod W steps (a tail the paper avoids by choosing T divisible by W)
    always take the per-step backward.  Returns [(step indices, use_jagg)]."""
    if W < 2 or T < 1:
        raise ValueError("need W >= 2 and T >= 1")
    full, tail = windows(T, W)
    mask = np.asarray(mask, dtype=np.uint8).reshape(-1)
    if mask.shape[0] != len(full) or np.any(mask > 1):
        raise ValueError("the mask needs one 0/1 entry per full window")
    plan = [(idx, bool(m)) for idx, m in zip(full, mask)]
    if tail:
        plan.append((tail, False))
    return plan


def trajectory(cfg, P, inputs, s_list, t, W, mask=None, frac=None, scores=None, tau: float = 0.5):
    """Gradient of a whole trajectory of T = len(inputs) steps: the sum over
    its windows of the JAGG group gradient (routed windows) or the per-step
    gradient (the rest and the tail), as gradient accumulation over groups
    does.  The mask comes from ``route`` (static frac or per-window scores)
    unless given.  t: the T timesteps, strictly decreasing.  Returns
    (mask, {name: grad})."""
    T = len(inputs)
    t = np.asarray(t, dtype=np.float64)
    if t.shape[0] != T or len(s_list) != T:
        raise ValueError("one timestep and one upstream gradient per step")
    if not np.all(t[1:] < t[:-1]):
        raise ValueError("a trajectory's timesteps must be strictly decreasing")
    n_full = T // W
    if mask is None:
        mask = route(n_full, frac=frac, scores=scores, tau=tau)[0] if n_full else np.zeros(0, np.uint8)
    total = None
    for idx, use_jagg in trajectory_plan(T, W, mask):
        ins = [inputs[k] for k in idx]
        ss = [s_list[k] for k in idx]
        G = g_jagg(cfg, P, ins, ss, t[idx]) if use_jagg else g_exact(cfg, P, ins, ss)
        total = G if total is None else {k: total[k] + G[k] for k in total}
    return np.asarray(mask, dtype=np.uint8), total


# ----------------------------------------------------- Theorem 1 linear toy
class LinearToy:
    """v_theta(z, t) = A z + b t + c, theta = (A, b, c): linear in (z, t)."""

    def __init__(self, A, b, c):
        self.A, self.b, self.c = (np.asarray(x, dtype=np.float64) for x in (A, b, c))

    def v(self, z, t):
        return self.A @ z + self.b * t + self.c

    @staticmethod
    def vjp(z, t, s):
        """J(z, t)^T s in closed form: dA = s z^T, db = s t, dc = s."""
        return np.outer(s, z), s * t, s.copy()

    def g_exact(self, zs, ts, ss):
        out = [np.zeros_like(self.A), np.zeros_like(self.b), np.zeros_like(self.c)]
        for z, t, s in zip(zs, ts, ss):
            for k, g in enumerate(self.vjp(z, t, s)):
                out[k] = out[k] + g
        return out

    def g_jagg(self, zs, ts, ss):
        W = len(zs)
        sb, sc = aggregate(ss, ts)
        g0 = self.vjp(zs[0], ts[0], sb)
        g1 = self.vjp(zs[W - 1], ts[W - 1], sc)
        return [x + y for x, y in zip(g0, g1)]

    def trajectory(self, zs, ts, ss, W, mask):
        """Whole-trajectory gradient under ``trajectory_plan`` (same windows,
        routing and tail as the MMDiT trajectory)."""
        out = [np.zeros_like(self.A), np.zeros_like(self.b), np.zeros_like(self.c)]
        for idx, use_jagg in trajectory_plan(len(zs), W, mask):
            args = ([zs[k] for k in idx], [ts[k] for k in idx], [ss[k] for k in idx])
            g = self.g_jagg(*args) if use_jagg else self.g_exact(*args)
            out = [a + b for a, b in zip(out, g)]
        return out
