"""Gradient-quality tool (gradient-quality appendix and the endpoint-only
ablation of the experiments): for one window it forms

  g_jagg   -- JAGG: composites + one backward over the endpoint pair,
  g_exact  -- the per-step backward sum_j J_j^T s_j,
  g_ablate -- the endpoint-only ablation J_0^T s_0 + J_{W-1}^T s_{W-1}
              (the joint backward driven by the endpoint signals alone; it is
              the JAGG call with the window shrunk to its two endpoints),

and reports cos(g, g_exact) and the norm ratio rho = |g| / |g_exact| for the
two approximations.  The routing rule (jagg_route, score >= tau) consumes
these cosines per group.  Every step runs in libjagg.so; torch only allocates
the gradient buffers (zeroed, so the layout padding adds nothing to the sums).
"""
from __future__ import annotations

import math


def cos_rho(ctx, a, b):
    """cos(a, b) and |a| / |b| from the library's fp64 sums."""
    ab, aa, bb = ctx.grad_compare(a, b)
    return ab / math.sqrt(aa * bb), math.sqrt(aa / bb)


def gradient_quality(ctx, theta, saved_pair, saved_steps, batch: int, s_list, t) -> dict:
    """cos and rho of g_jagg and g_ablate against g_exact for one window.

    saved_pair: batch-2B forward of the endpoint pair; saved_steps: the W
    batch-B forwards of every step; s_list: the W upstream gradients; t: the
    W timesteps of the window."""
    import torch

    def zeros():
        return torch.zeros(ctx.n_params, dtype=ctx.grad_dtype, device="cuda")

    g_jagg, g_exact, g_abl = zeros(), zeros(), zeros()
    ctx.group_backward(theta, saved_pair, batch, s_list, t, g_jagg, beta=0.0)
    ctx.perstep_group_backward(theta, saved_steps, batch, s_list, g_exact, beta=0.0)
    ctx.group_backward(theta, saved_pair, batch, [s_list[0], s_list[-1]], [t[0], t[-1]], g_abl, beta=0.0)
    cj, rj = cos_rho(ctx, g_jagg, g_exact)
    ca, ra = cos_rho(ctx, g_abl, g_exact)
    return {"cos_jagg": cj, "rho_jagg": rj, "cos_ablate": ca, "rho_ablate": ra}
