"""Gradient-quality tool and routing calibration (gradient-quality appendix;
the endpoint-only ablation of the experiments).

For each window of a trajectory the library's ``jagg_window_quality`` forms
g_jagg (composites + one backward over the endpoint pair), g_exact (the
per-step backward) and g_ablate (the endpoint signals alone), and returns
cos(g, g_exact) and rho = |g| / |g_exact| for the two approximations (fp64
sums in the comparison kernel, the ratios formed in the library).  The table
of per-window cosines then calibrates the routing rule: ``jagg_route`` in
score mode routes the longest high-noise prefix of windows whose cosine is at
least tau.  Python only marshals the calls and collects the rows.
"""
from __future__ import annotations


def quality_table(ctx, theta, windows, batch: int) -> list:
    """One row per window, in the given (high-to-low noise) order.

    windows: [(saved_pair, saved_steps, s_list, t)] with saved_pair the
    batch-2B endpoint-pair forward, saved_steps the W batch-B step forwards,
    s_list the W upstream gradients, t the W timesteps."""
    import torch

    def zeros():
        return torch.zeros(ctx.n_params, dtype=ctx.grad_dtype, device="cuda")

    gj, ge, ga = zeros(), zeros(), zeros()
    rows = []
    for saved_pair, saved_steps, s_list, t in windows:
        cj, rj, ca, ra = ctx.window_quality(theta, saved_pair, saved_steps, batch, s_list, t, gj, ge, ga)
        rows.append({"cos_jagg": cj, "rho_jagg": rj, "cos_ablate": ca, "rho_ablate": ra})
    return rows


def calibrate(rows, tau: float = 0.5):
    """Routing mask and realised jagg_frac from the table's JAGG cosines
    (score mode of jagg_route: longest prefix with cos >= tau)."""
    from .api import route
    return route(len(rows), scores=[r["cos_jagg"] for r in rows], tau=tau)


def gradient_quality(ctx, theta, saved_pair, saved_steps, batch: int, s_list, t) -> dict:
    """cos and rho of g_jagg and g_ablate against g_exact for one window."""
    return quality_table(ctx, theta, [(saved_pair, saved_steps, s_list, t)], batch)[0]
