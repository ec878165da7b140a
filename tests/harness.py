"""Shared helpers for the GPU parity tests: build one seeded case, feed the same
(dtype-rounded) values to the HIP path and to the oracle, and compare.

The oracle never sees a value produced by the HIP path: both sides start from
the seeded generators in ``synth``; for a bf16 run the inputs are rounded to
bf16 once and the oracle receives those rounded values in fp64 (or fp32)."""
from __future__ import annotations

import numpy as np
import torch

import paper_2607_17572_amd as pk
import synth
from oracle import jagg, mmdit


def oracle_cfg(c: pk.Config) -> mmdit.Config:
    return mmdit.Config(n_double=c.n_double, n_single=c.n_single, hidden=c.hidden, heads=c.heads,
                        head_dim=c.head_dim, mlp_hidden=c.mlp_hidden, in_ch=c.in_ch, patch=c.patch, lat_h=c.lat_h,
                        lat_w=c.lat_w, n_txt=c.n_txt, txt_dim=c.txt_dim, t_freq_dim=c.t_freq_dim,
                        block_only=bool(c.block_only))


def tdtype(c: pk.Config):
    return torch.bfloat16 if c.act_dtype == pk.BF16 else torch.float32


def to_dev(x: np.ndarray, dt) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(dt).cuda()


def rounded(x: np.ndarray, dt) -> np.ndarray:
    """x rounded to the device dtype, back in fp64 (what the oracle is fed)."""
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(dt).to(torch.float64).numpy()


def stream_major(x_txt: np.ndarray, x_img: np.ndarray) -> np.ndarray:
    """(B, nt, D), (B, ni, D) -> rows [B*nt text rows; B*ni image rows] x D."""
    return np.concatenate([x_txt.reshape(-1, x_txt.shape[-1]), x_img.reshape(-1, x_img.shape[-1])], axis=0)


def from_stream_major(rows: np.ndarray, B: int, nt: int, ni: int):
    D = rows.shape[-1]
    return rows[:B * nt].reshape(B, nt, D), rows[B * nt:].reshape(B, ni, D)


class Case:
    """A seeded model + window.  ``W`` steps with per-sample batch ``B``."""

    def __init__(self, c: pk.Config, B: int = 1, W: int = 4, seed: int = 0, theta_std: float = 0.02,
                 gain_std: float = 0.02, T: int | None = None, t=None):
        self.c, self.B, self.W = c, B, W
        self.oc = oracle_cfg(c)
        self.dt = tdtype(c)
        lay, total = mmdit.param_layout(self.oc)
        entries = [(n, off, int(np.prod(s))) for n, s, off in lay]
        th = synth.theta(entries, seed=synth.THETA_SEED + seed, std=theta_std, gain_std=gain_std, total=total)
        self.theta_dev = to_dev(th, self.dt)
        self.theta = self.theta_dev.to(torch.float64).cpu().numpy()
        if t is None:
            t = synth.uniform_grid(T or 2 * W)[:W]
        self.t = np.asarray(t, dtype=np.float32).astype(np.float64)
        dseed = synth.DATA_SEED + 1000 * seed
        self.inputs_dev, self.inputs = [], []
        for j in range(W):
            if c.block_only:
                xt = rounded(synth.normal((B, c.n_txt, c.hidden), dseed + 10 * j), self.dt)
                xi = rounded(synth.normal((B, c.n_img, c.hidden), dseed + 10 * j + 1), self.dt)
                self.inputs.append(mmdit.Inputs(t=np.full(B, self.t[j]), x_txt=xt, x_img=xi))
                self.inputs_dev.append((to_dev(stream_major(xt, xi), self.dt), None))
            else:
                z = rounded(synth.normal((B, c.in_ch, c.lat_h, c.lat_w), dseed + 10 * j), self.dt)
                tx = rounded(synth.normal((B, c.n_txt, c.txt_dim), dseed + 10 * j + 1), self.dt)
                self.inputs.append(mmdit.Inputs(t=np.full(B, self.t[j]), z=z, txt=tx))
                self.inputs_dev.append((to_dev(z, self.dt), to_dev(tx, self.dt)))
        self.s, self.s_dev = [], []
        g = synth.rng(dseed + 777)
        adv = g.standard_normal(B)
        for j in range(W):
            if c.block_only:
                st = rounded(g.standard_normal((B, c.n_txt, c.hidden)) * adv[:, None, None], self.dt)
                si = rounded(g.standard_normal((B, c.n_img, c.hidden)) * adv[:, None, None], self.dt)
                self.s.append((st, si))
                self.s_dev.append(to_dev(stream_major(st, si), self.dt))
            else:
                sj = rounded(g.standard_normal((B, c.in_ch, c.lat_h, c.lat_w)) * adv[:, None, None, None], self.dt)
                self.s.append(sj)
                self.s_dev.append(to_dev(sj, self.dt))
        self.ctx = pk.Context(c)

    # ---------------------------------------------------------------- GPU side
    def forward(self, j: int, saved=True):
        z, tx = self.inputs_dev[j]
        sv = self.ctx.new_saved(self.B) if saved else None
        v = self.ctx.forward_save(self.theta_dev, z, [self.t[j]] * self.B, tx, saved=sv, batch=self.B)
        return v, sv

    def pair_inputs_dev(self):
        """The endpoint pair as one batch-2B device input (endpoint 0 first)."""
        c, B = self.c, self.B
        (z0, t0), (z1, t1) = self.inputs_dev[0], self.inputs_dev[-1]
        if c.block_only:
            D = c.hidden
            nt = B * c.n_txt
            z = torch.cat([z0[:nt], z1[:nt], z0[nt:], z1[nt:]], dim=0)
            return z, None
        return torch.cat([z0, z1], 0), torch.cat([t0, t1], 0)

    def saved_pair(self):
        z, tx = self.pair_inputs_dev()
        sv = self.ctx.new_saved(2 * self.B)
        tt = [self.t[0]] * self.B + [self.t[-1]] * self.B
        self.ctx.forward_save(self.theta_dev, z, tt, tx, saved=sv, batch=2 * self.B)
        return sv

    def new_grad(self):
        return torch.zeros(self.ctx.n_params, dtype=self.ctx.grad_dtype, device="cuda")

    def gpu_jagg(self, dtheta=None, beta=0.0):
        sv = self.saved_pair()
        d = self.new_grad() if dtheta is None else dtheta
        self.ctx.group_backward(self.theta_dev, sv, self.B, self.s_dev, self.t, d, beta)
        return d

    def gpu_perstep(self, dtheta=None, beta=0.0):
        saved = [self.forward(j)[1] for j in range(self.W)]
        d = self.new_grad() if dtheta is None else dtheta
        self.ctx.perstep_group_backward(self.theta_dev, saved, self.B, self.s_dev, d, beta)
        return d

    # ------------------------------------------------------------- oracle side
    def P(self, dtype=np.float64):
        return mmdit.unflatten(self.oc, self.theta, dtype)

    def oracle_jagg(self, dtype=np.float64):
        P = self.P(dtype)
        inps = [self._cast(i, dtype) for i in self.inputs]
        return mmdit.flatten(self.oc, jagg.g_jagg(self.oc, P, inps, self.s, self.t))

    def oracle_exact(self, dtype=np.float64):
        P = self.P(dtype)
        inps = [self._cast(i, dtype) for i in self.inputs]
        ss = [tuple(x.astype(dtype) for x in s) if isinstance(s, tuple) else s.astype(dtype) for s in self.s]
        return mmdit.flatten(self.oc, jagg.g_exact(self.oc, P, inps, ss))

    @staticmethod
    def _cast(i, dtype):
        f = (lambda a: None if a is None else a.astype(dtype))
        return mmdit.Inputs(t=i.t, z=f(i.z), txt=f(i.txt), x_txt=f(i.x_txt), x_img=f(i.x_img))


def rel_l2(a: np.ndarray, b: np.ndarray) -> float:
    nb = float(np.linalg.norm(b))
    return float(np.linalg.norm(a - b)) / (nb if nb > 0 else 1.0)


def compare_grads(case: Case, got: torch.Tensor, want: np.ndarray, tol: float, per_tensor_tol: float | None = None,
                  report: bool = False):
    """Global and raw per-tensor relative L2 against the bar (``per_tensor_tol``
    defaults to ``tol``): each tensor is judged on its own norm,
    ||got - want|| / ||want||.  Tensors whose reference is exactly zero must be
    exactly zero.  Every tensor is checked before anything is asserted, so a
    failure lists all offenders.  Returns (global error, (worst per-tensor
    error, name))."""
    g = got.to(torch.float64).cpu().numpy()
    lay, _ = mmdit.param_layout(case.oc)
    mask = np.zeros_like(g, dtype=bool)
    worst = (0.0, "")
    bar = per_tensor_tol or tol
    bad, rows = [], []
    for name, shape, off in lay:
        n = int(np.prod(shape))
        mask[off:off + n] = True
        a, b = g[off:off + n], want[off:off + n]
        if not np.any(b):
            if np.any(a):
                bad.append(f"{name}: reference is exactly zero, GPU is not (max |g| {np.abs(a).max():.3e})")
            continue
        e = rel_l2(a, b)
        rows.append((e, name))
        if e > worst[0]:
            worst = (e, name)
        if not e <= bar:
            bad.append(f"{name}: rel L2 {e:.3e} > {bar}")
    eg = rel_l2(g[mask], want[mask])
    if report or bad:
        rows.sort(reverse=True)
        print("per-tensor rel L2 (worst 8): " + ", ".join(f"{n} {e:.2e}" for e, n in rows[:8]), flush=True)
    assert not bad, "; ".join(bad[:20])
    assert eg <= tol, f"global rel L2 {eg:.3e} > {tol}"
    return eg, worst
