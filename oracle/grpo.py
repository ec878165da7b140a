"""Oracle for Phase 2 of JAGG: the per-step upstream gradients s_j of the GRPO
objective and their composites.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).  Written from the paper's
GRPO section, in its order and notation, fp64 throughout:

* rectified-flow transition mean, one Euler step of the SDE:
      mu_j = z_j + v_j (t_{j+1} - t_j)                     (text of Eq. logprob)
* Gaussian log-probability of the observed next latent (summed over the n
  elements of one sample: the squared norm of Eq. logprob):
      log pi_j = -|z_{j+1} - mu_j|^2 / (2 sigma_j^2) - n log(sqrt(2 pi) sigma_j)
* probability ratio rho_j = exp(log pi_j - log pi_old_j)           (Eq. grpo_loss)
* per-step PPO-clipped term, the window average over j:
      L_j = (1/W) max(-A rho_j, -A clip(rho_j, 1 - eps, 1 + eps))   (Eq. grpo_loss)
  with the advantage clamped to [-adv_clip, adv_clip] (hyperparameter
  appendix: advantage clamp 5.0, clip range 0.1);
* s_j = dL_j / dv_j with z_j, z_{j+1} and pi_old fixed (Phase 2: detached
  proxy, z_j a fixed sample).

Closed form of the last step (chain rule through the three definitions):
      dL_j/drho_j = -A/W when the unclipped term is the maximum, 0 when the
                    clipped term is strictly larger (then rho_j lies outside
                    [1 - eps, 1 + eps] on the side the clip cuts: the PPO-clip
                    remark's zero upstream gradient);
      drho_j/dlog pi_j = rho_j;
      dlog pi_j/dv_j = (z_{j+1} - mu_j) (t_{j+1} - t_j) / sigma_j^2.
It is pinned against central finite differences of L_j (tests).
"""
from __future__ import annotations

import numpy as np

from . import jagg


def rf_mean(z, v, t, t_next):
    """Euler step of the rectified-flow SDE drift: the transition mean."""
    return z + v * (t_next - t)


def log_prob(z_next, mu, sigma):
    """Eq. logprob per sample (leading axis = batch), elements summed."""
    d = (np.asarray(z_next, np.float64) - np.asarray(mu, np.float64)).reshape(len(z_next), -1)
    n = d.shape[1]
    return -(d * d).sum(axis=1) / (2.0 * sigma * sigma) - n * np.log(np.sqrt(2.0 * np.pi) * sigma)


def clamp_adv(A, adv_clip):
    return np.clip(np.asarray(A, np.float64), -adv_clip, adv_clip)


def step_loss(z, z_next, v, t, t_next, sigma, logp_old, A, eps, W, adv_clip):
    """L_j of Eq. grpo_loss for every sample of the batch."""
    A = clamp_adv(A, adv_clip)
    lp = log_prob(z_next, rf_mean(z, v, t, t_next), sigma)
    rho = np.exp(lp - logp_old)
    return np.maximum(-A * rho, -A * np.clip(rho, 1.0 - eps, 1.0 + eps)) / W


def step_stats(z, z_next, v, t, t_next, sigma, logp_old, A, eps, W, adv_clip):
    """(log pi_j, rho_j, dL_j/drho_j) per sample."""
    A = clamp_adv(A, adv_clip)
    lp = log_prob(z_next, rf_mean(z, v, t, t_next), sigma)
    rho = np.exp(lp - logp_old)
    unclipped = -A * rho
    clipped = -A * np.clip(rho, 1.0 - eps, 1.0 + eps)
    dl_drho = np.where(clipped > unclipped, 0.0, -A / W)
    return lp, rho, dl_drho


def upstream_grad(z, z_next, v, t, t_next, sigma, logp_old, A, eps, W, adv_clip):
    """s_j = dL_j / dv_j (closed form, module docstring)."""
    _, rho, dl_drho = step_stats(z, z_next, v, t, t_next, sigma, logp_old, A, eps, W, adv_clip)
    r = np.asarray(z_next, np.float64) - rf_mean(np.asarray(z, np.float64), np.asarray(v, np.float64), t, t_next)
    coef = dl_drho * rho * (t_next - t) / (sigma * sigma)
    return coef.reshape((-1,) + (1,) * (r.ndim - 1)) * r


def window_upstream(zs, vs, ts, sigmas, logp_old, A, eps, adv_clip):
    """All W upstream gradients of a window: zs = z_0..z_W, vs = v_0..v_{W-1},
    ts = t_0..t_W, sigmas and logp_old[j][b] per step."""
    W = len(vs)
    return [upstream_grad(zs[j], zs[j + 1], vs[j], ts[j], ts[j + 1], sigmas[j], logp_old[j], A, eps, W, adv_clip)
            for j in range(W)]


def window_composites(zs, vs, ts, sigmas, logp_old, A, eps, adv_clip):
    """Phase 3 on the Phase-2 gradients: (s_base, s_corr) over t_0..t_{W-1}."""
    W = len(vs)
    s = window_upstream(zs, vs, ts, sigmas, logp_old, A, eps, adv_clip)
    return jagg.aggregate(s, np.asarray(ts[:W], np.float64))
