"""GPU parity of the sequential-graph variant (one endpoint backward at a
time) and of the gradient-quality tool (cos and norm ratio against the
per-step gradient, plus the endpoint-only ablation), against the oracle."""
import sys

import numpy as np
import pytest
import torch

import paper_2607_17572_amd as pk
import synth
from harness import Case, compare_grads, rel_l2
from oracle import jagg, mmdit
from paper_2607_17572_amd import quality

pytestmark = pytest.mark.gpu

TINY = pk.config("tiny")
BLOCK_SMALL = pk.Config(n_double=1, n_single=0, hidden=256, heads=2, head_dim=128, mlp_hidden=1024, in_ch=16, patch=2,
                        lat_h=16, lat_w=16, n_txt=40, txt_dim=256, t_freq_dim=256, block_only=1, act_dtype=pk.BF16,
                        grad_dtype=pk.F32)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def sequential(cs: Case):
    """Endpoint 0 then endpoint 1 with ONE saved buffer, re-filled in between."""
    d = cs.new_grad()
    sv = cs.ctx.new_saved(cs.B)
    for e, j in ((0, 0), (1, cs.W - 1)):
        z, tx = cs.inputs_dev[j]
        cs.ctx.forward_save(cs.theta_dev, z, [cs.t[j]] * cs.B, tx, saved=sv, batch=cs.B)
        cs.ctx.endpoint_backward(cs.theta_dev, sv, cs.B, cs.s_dev, cs.t, e, d, beta=0.0 if e == 0 else 1.0)
    return d


def test_sequential_variant_fp32_matches_joint_and_oracle():
    say("case: tiny fp32 sequential-graph JAGG W=4 B=2")
    cs = Case(TINY, B=2, W=4)
    seq = sequential(cs)
    joint = cs.gpu_jagg()
    torch.cuda.synchronize()
    e = rel_l2(seq.double().cpu().numpy(), joint.double().cpu().numpy())
    say(f"  sequential vs joint rel L2 {e:.2e}")
    assert e < 1e-6
    eg, _ = compare_grads(cs, seq, cs.oracle_jagg(), 1e-4)
    say(f"  sequential vs oracle rel L2 {eg:.2e}")


def test_sequential_variant_bf16_block():
    say("case: bf16 block sequential-graph JAGG W=4 B=1")
    cs = Case(BLOCK_SMALL, B=1, W=4)
    seq = sequential(cs)
    joint = cs.gpu_jagg()
    torch.cuda.synchronize()
    e = rel_l2(seq.double().cpu().numpy(), joint.double().cpu().numpy())
    say(f"  sequential vs joint rel L2 {e:.2e}")
    assert e < 1e-2
    eg, _ = compare_grads(cs, seq, cs.oracle_jagg(), 2e-2)
    say(f"  sequential vs oracle rel L2 {eg:.2e}")


@pytest.mark.parametrize("n", [1, 7, 4096, 1000003])
@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16])
def test_grad_compare_sums(n, dt):
    say(f"case: grad compare n={n} {dt}")
    ctx = pk.Context(TINY)
    a = synth.normal((n,), 300 + n)
    b = 0.5 * a + synth.normal((n,), 301 + n)
    ad = torch.from_numpy(a.astype(np.float32)).to(dt).cuda()
    bd = torch.from_numpy(b.astype(np.float32)).to(dt).cuda()
    got = ctx.grad_compare(ad, bd)
    x, y = ad.double().cpu().numpy(), bd.double().cpu().numpy()
    want = (float(x @ y), float(x @ x), float(y @ y))
    for g, w in zip(got, want):
        assert abs(g - w) <= 1e-12 * max(1.0, abs(want[1]) + abs(want[2])), (got, want)
    # the library's quality figures: cos = a.b / sqrt(a.a b.b), rho = sqrt(a.a / b.b)
    cos = float(x @ y) / (np.linalg.norm(x) * np.linalg.norm(y))
    rho = np.linalg.norm(x) / np.linalg.norm(y)
    assert abs(got[3] - cos) <= 1e-10 and abs(got[4] - rho) <= 1e-10 * rho


def test_gradient_quality_tool_matches_oracle():
    """cos and rho of JAGG and of the endpoint-only ablation against the exact
    per-step gradient, on the tiny fp32 model; the oracle computes the three
    gradients itself (g_jagg, g_exact, g_ablate) and the two ratios by their
    definition."""
    say("case: tiny fp32 gradient quality W=4")
    cs = Case(TINY, B=1, W=4)
    saved = [cs.forward(j)[1] for j in range(cs.W)]
    q = quality.gradient_quality(cs.ctx, cs.theta_dev, cs.saved_pair(), saved, cs.B, cs.s_dev, cs.t)
    P = cs.P()
    gj = cs.oracle_jagg()
    ge = cs.oracle_exact()
    ga = mmdit.flatten(cs.oc, jagg.g_ablate(cs.oc, P, cs.inputs, cs.s))

    def cr(a, b):
        return float(a @ b / (np.linalg.norm(a) * np.linalg.norm(b))), float(np.linalg.norm(a) / np.linalg.norm(b))

    want = dict(zip(("cos_jagg", "rho_jagg"), cr(gj, ge)))
    want.update(zip(("cos_ablate", "rho_ablate"), cr(ga, ge)))
    say(f"  gpu {q}\n  oracle {want}")
    for k in want:
        assert abs(q[k] - want[k]) <= 1e-5, k
    assert q["cos_jagg"] < 1.0 - 1e-6  # a random MMDiT is not linear in (z, t)


def test_gradient_quality_w2_is_exact():
    """W = 2: alpha = (0, 1) makes JAGG, the ablation and the exact gradient
    the same quantity: cos = rho = 1."""
    say("case: tiny fp32 gradient quality W=2")
    cs = Case(TINY, B=2, W=2)
    saved = [cs.forward(j)[1] for j in range(cs.W)]
    q = quality.gradient_quality(cs.ctx, cs.theta_dev, cs.saved_pair(), saved, cs.B, cs.s_dev, cs.t)
    say(f"  {q}")
    for k, v in q.items():
        assert abs(v - 1.0) <= 1e-6, (k, v)


@pytest.mark.parametrize("n", [1, 7, 4096, 1000003])
@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16])
def test_count_nonfinite_matches_numpy(n, dt):
    """NaN / +-Inf count of a device vector: exact against numpy's isfinite on
    the same values, with planted NaN, +-Inf, the largest finite magnitudes and
    subnormals, in the vector body and in its ragged tail."""
    say(f"case: count non-finite n={n} {dt}")
    ctx = pk.Context(TINY)
    x = synth.normal((n,), 900 + n).astype(np.float32)
    rng = np.random.default_rng(901 + n)
    big = np.float32(3.3895314e38) if dt == torch.bfloat16 else np.finfo(np.float32).max  # largest finite
    specials = [np.nan, np.inf, -np.inf, big, -big, np.float32(1e-40), -np.nan]
    k = min(n, 3 * len(specials))
    pos = rng.choice(n, size=k, replace=False)
    for i, p in enumerate(pos):
        x[p] = specials[i % len(specials)]
    if n % 8:
        x[-1] = np.inf  # the ragged tail is scanned too
    xd = torch.from_numpy(x).to(dt).cuda()
    got = ctx.count_nonfinite(xd)
    want = int(np.count_nonzero(~np.isfinite(xd.float().cpu().numpy())))
    say(f"  count {got} (numpy {want})")
    assert got == want
    assert ctx.count_nonfinite(torch.zeros(n, dtype=dt, device="cuda")) == 0
