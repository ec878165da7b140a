"""GPU parity of Phase 2 (GRPO upstream gradients through the rectified-flow
Euler step and the PPO-clipped loss) and of its fusion with the composites,
against oracle.grpo on the same bf16/fp32-rounded inputs.  Clip decisions
(which steps get a zero gradient) must match exactly: both sides take them in
fp64.  log pi_j: relative 1e-12, rho_j and loss: 1e-12 x |log pi_j| (at least
1e-9, see check_stats); s_j and the
composites: relative L2 1e-6 (fp32), 8e-3 (bf16, one rounding on store)."""
import sys

import numpy as np
import pytest
import torch

import paper_2607_17572_amd as pk
import synth
from harness import Case, compare_grads, rel_l2, rounded, stream_major, to_dev
from oracle import grpo, jagg, mmdit

pytestmark = pytest.mark.gpu

TINY = pk.config("tiny")
BLOCK_SMALL = pk.Config(n_double=1, n_single=0, hidden=256, heads=2, head_dim=128, mlp_hidden=1024, in_ch=16, patch=2,
                        lat_h=16, lat_w=16, n_txt=40, txt_dim=256, t_freq_dim=256, block_only=1, act_dtype=pk.BF16,
                        grad_dtype=pk.F32)
FULL_BF16 = pk.Config(n_double=1, n_single=1, hidden=256, heads=2, head_dim=128, mlp_hidden=512, in_ch=16, patch=2,
                      lat_h=16, lat_w=20, n_txt=24, txt_dim=128, t_freq_dim=256, act_dtype=pk.BF16, grad_dtype=pk.F32)
EPS, ADV_CLIP = 0.1, 5.0
# the clip range crosses the C ABI as an fp32 value; the oracle is given that value
EPS_ABI = float(np.float32(EPS))
# target ratios per (step, sample): inside the clip range, above and below it
RHO = np.array([[1.05, 0.93], [1.3, 1.3], [0.7, 0.7], [1.0, 1.16]])


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


class Window:
    """Seeded rollout data of one window in the model's batch-B output layout."""

    def __init__(self, c: pk.Config, B: int, W: int = 4, seed: int = 0):
        self.c, self.B, self.W = c, B, W
        self.dt = torch.bfloat16 if c.act_dtype == pk.BF16 else torch.float32
        if c.block_only:
            self.shape = (B * (c.n_txt + c.n_img), c.hidden)
        else:
            self.shape = (B, c.in_ch, c.lat_h, c.lat_w)
        sd = synth.DATA_SEED + 500 + seed
        self.z = [rounded(synth.normal(self.shape, sd + j), self.dt) for j in range(W + 1)]
        self.v = [rounded(synth.normal(self.shape, sd + 100 + j), self.dt) for j in range(W)]
        self.t = np.asarray(synth.uniform_grid(16)[3:3 + W + 1], np.float32)
        self.sigma = np.asarray(0.2 + 0.05 * np.arange(W), np.float32)
        self.adv = np.asarray([1.4, -0.8], np.float32)[:B]  # B <= 2 here
        # old log-probabilities that put the ratios at RHO (oracle arithmetic only)
        self.set_old_logp()

    def set_old_logp(self):
        self.lpo = np.stack([self.logp(j) - np.log(RHO[j % 4, :self.B]) for j in range(self.W)])

    def per_sample(self, x):
        """(B, n) view of a batch-B array in the output layout."""
        c, B = self.c, self.B
        if not c.block_only:
            return x.reshape(B, -1)
        nt = B * c.n_txt
        xt = x[:nt].reshape(B, -1)
        xi = x[nt:].reshape(B, -1)
        return np.concatenate([xt, xi], axis=1)

    def from_per_sample(self, y):
        c, B = self.c, self.B
        if not c.block_only:
            return y.reshape(self.shape)
        ntd = c.n_txt * c.hidden
        return np.concatenate([y[:, :ntd].reshape(-1, c.hidden), y[:, ntd:].reshape(-1, c.hidden)], axis=0)

    def logp(self, j):
        ps = self.per_sample
        t = self.t.astype(np.float64)
        return grpo.log_prob(ps(self.z[j + 1]), grpo.rf_mean(ps(self.z[j]), ps(self.v[j]), t[j], t[j + 1]),
                             float(self.sigma[j]))

    def oracle(self):
        ps = self.per_sample
        t = self.t.astype(np.float64)
        s = grpo.window_upstream([ps(x) for x in self.z], [ps(x) for x in self.v], t,
                                 self.sigma.astype(np.float64), self.lpo, self.adv.astype(np.float64), EPS_ABI, ADV_CLIP)
        stats = []
        for j in range(self.W):
            lp, rho, _ = grpo.step_stats(ps(self.z[j]), ps(self.z[j + 1]), ps(self.v[j]), t[j], t[j + 1],
                                         float(self.sigma[j]), self.lpo[j], self.adv.astype(np.float64), EPS_ABI,
                                         self.W, ADV_CLIP)
            L = grpo.step_loss(ps(self.z[j]), ps(self.z[j + 1]), ps(self.v[j]), t[j], t[j + 1], float(self.sigma[j]),
                               self.lpo[j], self.adv.astype(np.float64), EPS_ABI, self.W, ADV_CLIP)
            stats.append(np.stack([lp, rho, L], axis=1))
        return [self.from_per_sample(x) for x in s], np.stack(stats)

    def dev(self):
        return ([to_dev(x, self.dt) for x in self.v], [to_dev(x, self.dt) for x in self.z],
                torch.from_numpy(self.lpo).cuda(), torch.from_numpy(self.adv).cuda())


def check_stats(got, want):
    """log pi to 1e-12 relative (fp64 sums in a different order); rho = exp(log pi -
    log pi_old) then carries the ABSOLUTE error of log pi as its relative error:
    1e-12 x |log pi| (~1e-4 for a 14M-element sample, whose |log pi| ~ 1e8),
    at least 1e-9; the loss is -A rho / W or a constant."""
    got = got.cpu().numpy()
    assert np.allclose(got[..., 0], want[..., 0], rtol=1e-12, atol=0)
    rt = max(1e-9, 1e-12 * float(np.max(np.abs(want[..., 0]))))
    assert np.allclose(got[..., 1], want[..., 1], rtol=rt, atol=0)
    assert np.allclose(got[..., 2], want[..., 2], rtol=rt, atol=1e-15)


@pytest.mark.parametrize("name,B", [("tiny", 2), ("block", 2), ("full", 1)])
def test_grpo_upstream_and_composites_match_oracle(name, B):
    c = {"tiny": TINY, "block": BLOCK_SMALL, "full": FULL_BF16}[name]
    say(f"case: GRPO window {name} B={B} W=4")
    w = Window(c, B)
    s_want, st_want = w.oracle()
    # clip decisions of the chosen ratios: some (step, sample) gradients are
    # exactly zero, the others are not
    zero = np.array([[np.all(r == 0) for r in w.per_sample(x)] for x in s_want])
    assert zero.any() and not zero.all()
    ctx = pk.Context(c)
    v, z, lpo, adv = w.dev()
    s_out = [torch.empty(w.shape, dtype=w.dt, device="cuda") for _ in range(w.W)]
    stats = torch.zeros((w.W, B, 3), dtype=torch.float64, device="cuda")
    ctx.grpo_upstream(v, z, w.t, w.sigma, lpo, adv, s_out, EPS, ADV_CLIP, stats=stats)
    torch.cuda.synchronize()
    check_stats(stats, st_want)
    tol = 8e-3 if w.dt == torch.bfloat16 else 1e-6
    for j in range(w.W):
        got = s_out[j].double().cpu().numpy()
        gz = np.array([np.all(r == 0) for r in w.per_sample(got)])
        assert np.array_equal(gz, zero[j]), (j, gz, zero[j])
        e = rel_l2(got, s_want[j])
        say(f"  s_{j} rel L2 {e:.2e}")
        assert e <= tol
    # fused composites
    sb = torch.empty(w.shape, dtype=w.dt, device="cuda")
    sc = torch.empty_like(sb)
    ctx.grpo_composites(v, z, w.t, w.sigma, lpo, adv, sb, sc, EPS, ADV_CLIP)
    wb, wc = jagg.aggregate(s_want, w.t[:w.W].astype(np.float64))
    eb, ec = rel_l2(sb.double().cpu().numpy(), wb), rel_l2(sc.double().cpu().numpy(), wc)
    say(f"  composites rel L2 {eb:.2e} {ec:.2e}")
    assert eb <= tol and ec <= tol


def test_grpo_group_backward_matches_oracle():
    """Phases 2-4 on the tiny fp32 MMDiT: the rollout latents z_0, z_{W-1} are
    the network inputs of the window's endpoints; the oracle forms s_j from
    the same data and runs its own JAGG group gradient."""
    say("case: tiny fp32 GRPO group backward W=4 B=2")
    cs = Case(TINY, B=2, W=4)
    w = Window(TINY, 2)
    # the model's inputs at the endpoints are the rollout latents of the window
    w.z[0] = cs.inputs[0].z
    w.z[w.W - 1] = cs.inputs[-1].z
    w.t = np.concatenate([cs.t, [cs.t[-1] - (cs.t[0] - cs.t[1])]]).astype(np.float32)
    w.set_old_logp()
    s_want, _ = w.oracle()
    v, z, lpo, adv = w.dev()
    d = cs.new_grad()
    cs.ctx.grpo_group_backward(cs.theta_dev, cs.saved_pair(), 2, v, z, w.t, w.sigma, lpo, adv, d, 0.0, EPS, ADV_CLIP)
    P = cs.P()
    want = mmdit.flatten(cs.oc, jagg.g_jagg(cs.oc, P, cs.inputs, s_want, cs.t))
    eg, worst = compare_grads(cs, d, want, 1e-4)
    say(f"  GRPO JAGG group backward rel L2 {eg:.2e}")


def batch_of(c: pk.Config, B: int, arrays):
    """Several batch-B arrays in the output layout as one batch-(k B) array
    (stream-major rows for a block-only model: all text rows, then all image rows)."""
    if not c.block_only:
        return torch.cat(arrays, 0)
    nt = B * c.n_txt
    return torch.cat([x[:nt] for x in arrays] + [x[nt:] for x in arrays], 0)


@pytest.mark.parametrize("name", ["tiny", "block"])
def test_grpo_reads_v_from_sub_batches(name):
    """v_0 and v_{W-1} taken from one endpoint-pair output (batch 2B) and the
    middle steps from one batch-(W-2)B output give the same bits as separate
    batch-B arrays."""
    c = {"tiny": TINY, "block": BLOCK_SMALL}[name]
    say(f"case: GRPO sub-batch addressing {name}")
    B = 2
    w = Window(c, B)
    ctx = pk.Context(c)
    v, z, lpo, adv = w.dev()
    sb0 = torch.empty(w.shape, dtype=w.dt, device="cuda")
    sc0 = torch.empty_like(sb0)
    ctx.grpo_composites(v, z, w.t, w.sigma, lpo, adv, sb0, sc0, EPS, ADV_CLIP)
    pair = batch_of(c, B, [v[0], v[-1]])
    mid = batch_of(c, B, v[1:-1])
    vs = [(pair, 2 * B, 0)] + [(mid, (w.W - 2) * B, j * B) for j in range(w.W - 2)] + [(pair, 2 * B, B)]
    sb1, sc1 = torch.empty_like(sb0), torch.empty_like(sb0)
    ctx.grpo_composites(vs, z, w.t, w.sigma, lpo, adv, sb1, sc1, EPS, ADV_CLIP)
    torch.cuda.synchronize()
    assert torch.equal(sb0, sb1) and torch.equal(sc0, sc1)
