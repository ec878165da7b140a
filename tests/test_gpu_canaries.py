"""Out-of-bounds write guard (GPU): every caller-owned buffer the library
writes (the workspace, saved activations, forward outputs, dtheta, the
no-allocation score slot) sits inside a larger allocation whose margins hold a
fixed byte pattern.  After the forwards, the JAGG group backward, the per-step
baseline, a trajectory (one window through each path) and the scoring and
comparison calls, the margins must be unchanged byte for byte.  The bf16
configurations have ragged token counts (104 tokens), so the MFMA attention
path's padded tiles and the GEMMs' edge tiles are exercised."""
import ctypes

import pytest
import torch

import paper_2607_17572_amd as pk
from harness import Case

pytestmark = pytest.mark.gpu

MARGIN = 1 << 16  # bytes of pattern before and after each buffer
PAT = 0xA5

BLOCK_SMALL = pk.Config(n_double=1, n_single=0, hidden=256, heads=2, head_dim=128, mlp_hidden=1024, in_ch=16, patch=2,
                        lat_h=16, lat_w=16, n_txt=40, txt_dim=256, t_freq_dim=256, block_only=1, act_dtype=pk.BF16,
                        grad_dtype=pk.F32)
FULL_SMALL = pk.Config(n_double=1, n_single=1, hidden=256, heads=2, head_dim=128, mlp_hidden=512, in_ch=16, patch=2,
                       lat_h=16, lat_w=20, n_txt=24, txt_dim=128, t_freq_dim=256, act_dtype=pk.BF16, grad_dtype=pk.BF16)


def say(*a):
    print(*a, flush=True)


class Guarded:
    """nbytes of device memory with MARGIN bytes of pattern on each side."""

    def __init__(self, nbytes: int):
        self.n = int(nbytes)
        self.full = torch.full((self.n + 2 * MARGIN,), PAT, dtype=torch.uint8, device="cuda")

    def bytes(self):
        return self.full[MARGIN:MARGIN + self.n]

    def as_(self, dtype, shape=None):
        v = self.bytes().view(dtype)
        return v if shape is None else v.view(shape)

    def intact(self) -> bool:
        head, tail = self.full[:MARGIN], self.full[MARGIN + self.n:]
        return bool((head == PAT).all().item()) and bool((tail == PAT).all().item())


def _esize(dt):
    return torch.empty((), dtype=dt).element_size()


@pytest.mark.parametrize("cfg_name", ["BLOCK_SMALL", "FULL_SMALL"])
def test_calls_leave_buffer_margins_untouched(cfg_name):
    cfg = {"BLOCK_SMALL": BLOCK_SMALL, "FULL_SMALL": FULL_SMALL}[cfg_name]
    say(f"case: canaries {cfg_name}")
    cs = Case(cfg, B=1, W=4)
    ctx = cs.ctx
    L = pk.lib()
    guards = {}

    # workspace for the pair (the largest batch used below), bound by hand
    ws = Guarded(ctx.workspace_bytes(2))
    assert L.jagg_ctx_set_workspace(ctx._h, ctypes.c_void_p(ws.bytes().data_ptr()), ws.n) == 0
    ctx._ws, ctx._ws_batch = ws.full, 1 << 20  # keep the binding from replacing it
    guards["workspace"] = ws

    # forwards: the endpoint pair and the W steps, saved activations and outputs guarded
    z, tx = cs.pair_inputs_dev()
    sv_pair = Guarded(ctx.saved_bytes(2))
    v_pair = Guarded(z.numel() * z.element_size())
    tt = [cs.t[0], cs.t[-1]]
    ctx.forward_save(cs.theta_dev, z, tt, tx, saved=sv_pair.bytes(), batch=2, v_out=v_pair.as_(z.dtype, z.shape))
    guards["saved pair"], guards["pair output"] = sv_pair, v_pair
    saved_steps = []
    for j in range(cs.W):
        zj, txj = cs.inputs_dev[j]
        sv = Guarded(ctx.saved_bytes(1))
        vo = Guarded(zj.numel() * zj.element_size())
        ctx.forward_save(cs.theta_dev, zj, [cs.t[j]], txj, saved=sv.bytes(), batch=1, v_out=vo.as_(zj.dtype, zj.shape))
        saved_steps.append(sv.bytes())
        guards[f"saved step {j}"], guards[f"output step {j}"] = sv, vo

    gdt = ctx.grad_dtype
    nbytes = ctx.n_params * _esize(gdt)

    def grad():
        g = Guarded(nbytes)
        g.as_(gdt).zero_()
        return g

    d_jagg, d_step, d_traj, d_traj_ps = grad(), grad(), grad(), grad()
    ctx.group_backward(cs.theta_dev, sv_pair.bytes(), 1, cs.s_dev, cs.t, d_jagg.as_(gdt), 0.0)
    ctx.perstep_group_backward(cs.theta_dev, saved_steps, 1, cs.s_dev, d_step.as_(gdt), 0.0)
    ctx.trajectory_backward(cs.theta_dev, cs.W, 1, [sv_pair.bytes()], [None] * cs.W, cs.s_dev, cs.t, [1],
                            d_traj.as_(gdt), 0.0)
    ctx.trajectory_backward(cs.theta_dev, cs.W, 1, [None], saved_steps, cs.s_dev, cs.t, [0], d_traj_ps.as_(gdt), 0.0)
    guards.update({"dtheta jagg": d_jagg, "dtheta per step": d_step, "dtheta trajectory (JAGG)": d_traj,
                   "dtheta trajectory (per step)": d_traj_ps})

    # head-of-workspace calls and the allocation-free score slot
    ctx.grad_compare(d_jagg.as_(gdt), d_step.as_(gdt))
    assert ctx.count_nonfinite(d_jagg.as_(gdt)) == 0
    ctx.group_score(cs.s_dev)
    slot = Guarded(8)
    ctx.group_score_noalloc(cs.s_dev, slot.as_(torch.float64))
    guards["no-allocation score slot"] = slot
    torch.cuda.synchronize()

    bad = [name for name, g in guards.items() if not g.intact()]
    say(f"  {len(guards)} guarded buffers, margins touched: {bad}")
    assert not bad, bad
    # the guarded runs computed what the plain calls compute
    ref = cs.gpu_jagg()
    assert torch.equal(d_jagg.as_(gdt), ref)
