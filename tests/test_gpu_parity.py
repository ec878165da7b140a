"""GPU parity: the HIP path (through the C ABI) against the oracle on the same
seeded inputs.  fp32 path: relative L2 <= 1e-4; bf16 path: <= 2e-2 (the
oracle is fed the same bf16-rounded parameters, inputs and upstream
gradients); routing decisions bit-exact."""
import sys

import numpy as np
import pytest
import torch

import paper_2607_17572_amd as pk
import synth
from harness import Case, compare_grads, rel_l2, rounded, to_dev
from oracle import jagg, mmdit

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


TINY = pk.config("tiny")
# multi-tile bf16 shapes with ragged row counts: 2*(40 + 64) = 208 rows per stream pair
BLOCK_SMALL = pk.Config(n_double=1, n_single=0, hidden=256, heads=2, head_dim=128, mlp_hidden=1024, in_ch=16, patch=2,
                        lat_h=16, lat_w=16, n_txt=40, txt_dim=256, t_freq_dim=256, block_only=1, act_dtype=pk.BF16,
                        grad_dtype=pk.F32)
# hidden 512: the wave-per-row LayerNorm backward and 8-column vector kernels
BLOCK_MID = pk.Config(n_double=1, n_single=0, hidden=512, heads=4, head_dim=128, mlp_hidden=2048, in_ch=16, patch=2,
                      lat_h=16, lat_w=18, n_txt=37, txt_dim=512, t_freq_dim=256, block_only=1, act_dtype=pk.BF16,
                      grad_dtype=pk.F32)
# token rows in multiples of 32 (2 x 32 text, 2 x 64 image rows per sample pair): the two
# streams' products of each layer run as one grouped GEMM launch with different
# contraction lengths (weight gradients) and row counts (input gradients); widths
# 384 / 1152 / 1536 leave ragged tile edges
BLOCK_GRP = pk.Config(n_double=1, n_single=0, hidden=384, heads=3, head_dim=128, mlp_hidden=1536, in_ch=16, patch=2,
                      lat_h=16, lat_w=16, n_txt=32, txt_dim=384, t_freq_dim=256, block_only=1, act_dtype=pk.BF16,
                      grad_dtype=pk.F32)
# 144 image + 37 text tokens: two 128-key blocks of the attention backward,
# the second ragged, and a ragged last 64-query tile
BLOCK_2KB = pk.Config(n_double=1, n_single=0, hidden=256, heads=2, head_dim=128, mlp_hidden=1024, in_ch=16, patch=2,
                      lat_h=24, lat_w=24, n_txt=37, txt_dim=256, t_freq_dim=256, block_only=1, act_dtype=pk.BF16,
                      grad_dtype=pk.F32)
FULL_SMALL = pk.Config(n_double=1, n_single=1, hidden=256, heads=2, head_dim=128, mlp_hidden=512, in_ch=16, patch=2,
                       lat_h=16, lat_w=20, n_txt=24, txt_dim=128, t_freq_dim=256, act_dtype=pk.BF16, grad_dtype=pk.F32)


# ------------------------------------------------------------------ fp32
def test_tiny_fp32_forward_matches_oracle():
    say("case: tiny fp32 forward")
    cs = Case(TINY, B=1, W=4)
    v, _ = cs.forward(0, saved=False)
    want, _ = mmdit.forward(cs.oc, cs.P(), cs.inputs[0])
    assert rel_l2(v.double().cpu().numpy(), want) < 1e-5


def test_tiny_fp32_vjp_matches_oracle():
    say("case: tiny fp32 vjp")
    cs = Case(TINY, B=2, W=1, t=[0.7])
    v, sv = cs.forward(0)
    d = cs.new_grad()
    cs.ctx.vjp(cs.theta_dev, sv, 2, cs.s_dev[0], d)
    want = cs.oracle_exact()
    eg, worst = compare_grads(cs, d, want, 1e-4)
    say(f"tiny vjp rel L2 {eg:.2e}, worst tensor {worst}")


def test_tiny_fp32_jagg_and_perstep_match_oracle():
    say("case: tiny fp32 jagg/perstep W=4")
    cs = Case(TINY, B=1, W=4)
    compare_grads(cs, cs.gpu_jagg(), cs.oracle_jagg(), 1e-4)
    compare_grads(cs, cs.gpu_perstep(), cs.oracle_exact(), 1e-4)


def test_tiny_fp32_second_window_and_accumulate():
    """Gradient accumulation over windows: beta = 1 adds the second window."""
    say("case: tiny fp32 two windows, accumulate")
    w0 = Case(TINY, B=1, W=4, t=synth.uniform_grid(8)[:4])
    w1 = Case(TINY, B=1, W=4, t=synth.uniform_grid(8)[4:], seed=0)
    w1.theta_dev = w0.theta_dev
    d = w0.gpu_jagg()
    w1.gpu_perstep(dtheta=d, beta=1.0)
    want = w0.oracle_jagg() + w1.oracle_exact()
    compare_grads(w0, d, want, 1e-4)


def test_w2_jagg_equals_perstep_on_gpu():
    """W = 2: alpha = (0, 1), so the composites are s_0, s_1 and JAGG is exact."""
    say("case: tiny fp32 W=2")
    cs = Case(TINY, B=2, W=2)
    a = cs.gpu_jagg().double().cpu().numpy()
    b = cs.gpu_perstep().double().cpu().numpy()
    assert rel_l2(a, b) < 1e-6


# ------------------------------------------------------------------ bf16
def test_bf16_block_jagg_matches_oracle():
    say("case: bf16 block (D=256, ragged rows) jagg W=4 B=1")
    cs = Case(BLOCK_SMALL, B=1, W=4)
    eg, worst = compare_grads(cs, cs.gpu_jagg(), cs.oracle_jagg(), 2e-2)
    say(f"bf16 block jagg rel L2 {eg:.2e}, worst {worst}")


def test_bf16_block_hidden512_matches_oracle():
    say("case: bf16 block hidden 512 (vector row kernels) jagg W=4 B=2")
    cs = Case(BLOCK_MID, B=2, W=4)
    eg, worst = compare_grads(cs, cs.gpu_jagg(), cs.oracle_jagg(), 2e-2)
    say(f"bf16 block512 jagg rel L2 {eg:.2e}, worst {worst}")


def test_bf16_full_model_forward_matches_oracle():
    """The bf16 forward output (MFMA attention forward over two 128-query
    blocks and a ragged last 64-key tile, 168 tokens) against the oracle on
    the same bf16-rounded parameters and inputs."""
    import dataclasses
    say("case: bf16 full model forward, 144+24 tokens")
    cs = Case(dataclasses.replace(FULL_SMALL, lat_h=24, lat_w=24), B=2, W=1, t=[0.6])
    v, _ = cs.forward(0, saved=False)
    want, _ = mmdit.forward(cs.oc, cs.P(), cs.inputs[0])
    err = rel_l2(v.double().cpu().numpy(), want)
    say(f"  forward rel L2 {err:.2e}")
    assert err <= 2e-2


@pytest.mark.parametrize("lat,n_txt", [(8, 10), (16, 64)], ids=["26_tokens", "128_tokens"])
def test_bf16_block_tile_edges_match_oracle(lat, n_txt):
    """Sequence lengths at the attention kernels' tile edges: 26 tokens (less
    than one 64-key tile, only the masked tile) and 128 tokens (whole tiles,
    no masked tile), forward output and JAGG gradient."""
    import dataclasses
    cfg = dataclasses.replace(BLOCK_SMALL, lat_h=lat, lat_w=lat, n_txt=n_txt)
    say(f"case: bf16 block, {(lat // 2) ** 2}+{n_txt} tokens")
    cs = Case(cfg, B=2, W=4)
    v, _ = cs.forward(0, saved=False)
    (wt, wi), _ = mmdit.forward(cs.oc, cs.P(), cs.inputs[0])
    from harness import stream_major
    err = rel_l2(v.double().cpu().numpy(), stream_major(wt, wi))
    say(f"  forward rel L2 {err:.2e}")
    assert err <= 2e-2
    eg, worst = compare_grads(cs, cs.gpu_jagg(), cs.oracle_jagg(), 2e-2)
    say(f"  jagg rel L2 {eg:.2e}, worst {worst}")


def test_bf16_block_two_key_blocks_ragged_matches_oracle():
    """The stored dS^T chunks (128 keys x 64 queries) across two key blocks
    and four query tiles, with a ragged key block and query tile."""
    say("case: bf16 block 144+37 tokens (two key blocks, ragged) jagg W=4 B=2")
    cs = Case(BLOCK_2KB, B=2, W=4)
    eg, worst = compare_grads(cs, cs.gpu_jagg(), cs.oracle_jagg(), 2e-2)
    say(f"bf16 block 181 tokens jagg rel L2 {eg:.2e}, worst {worst}")
    eg, worst = compare_grads(cs, cs.gpu_perstep(), cs.oracle_exact(), 2e-2)
    say(f"  per-step rel L2 {eg:.2e}, worst {worst}")


@pytest.mark.parametrize("gdt", [pk.F32, pk.BF16], ids=["f32grad", "bf16grad"])
def test_bf16_block_grouped_streams_match_oracle(gdt):
    import dataclasses
    say(f"case: bf16 block, grouped text/image products, grad dtype {gdt}")
    cs = Case(dataclasses.replace(BLOCK_GRP, grad_dtype=gdt), B=2, W=4)
    eg, worst = compare_grads(cs, cs.gpu_jagg(), cs.oracle_jagg(), 2e-2)
    say(f"  jagg rel L2 {eg:.2e}, worst {worst}")
    eg, worst = compare_grads(cs, cs.gpu_perstep(), cs.oracle_exact(), 2e-2)
    say(f"  per-step rel L2 {eg:.2e}, worst {worst}")


def test_bf16_block_perstep_batch2_matches_oracle():
    say("case: bf16 block perstep W=3 B=2")
    cs = Case(BLOCK_SMALL, B=2, W=3)
    compare_grads(cs, cs.gpu_perstep(), cs.oracle_exact(), 2e-2)


def test_bf16_full_model_with_single_block_matches_oracle():
    say("case: bf16 full model 1 double + 1 single")
    cs = Case(FULL_SMALL, B=1, W=4)
    eg, worst = compare_grads(cs, cs.gpu_jagg(), cs.oracle_jagg(), 2e-2)
    say(f"bf16 full jagg rel L2 {eg:.2e}, worst {worst}")
    compare_grads(cs, cs.gpu_perstep(), cs.oracle_exact(), 2e-2)


def test_checkpoint_recompute_is_bitwise_identical():
    """Per-block activation checkpointing recomputes the block forward with the
    same kernels, so the gradient is bitwise the one from saved activations."""
    say("case: checkpoint vs saved")
    a = Case(FULL_SMALL, B=1, W=4).gpu_jagg()
    cfg = pk.Config(**{**FULL_SMALL.__dict__, "checkpoint": 1})
    b = Case(cfg, B=1, W=4).gpu_jagg()
    assert torch.equal(a, b)


def test_determinism_bitwise():
    say("case: determinism")
    cs = Case(BLOCK_SMALL, B=1, W=4)
    a = cs.gpu_jagg()
    b = cs.gpu_jagg()
    assert torch.equal(a, b)


def test_timing_hook_leaves_results_bitwise():
    """Arming the per-class timing hook binds events to the timed launches and
    changes nothing else: the gradient is bitwise the unhooked one."""
    say("case: timing hook on vs off, bf16 block hidden 512, B=2")
    cs = Case(BLOCK_MID, B=2, W=4)
    sv = cs.saved_pair()
    a = cs.new_grad()
    cs.ctx.group_backward(cs.theta_dev, sv, cs.B, cs.s_dev, cs.t, a)
    torch.cuda.synchronize()
    b = cs.new_grad()
    pk.prof_begin(pk.PROF_GEMM_WGRAD)
    try:
        cs.ctx.group_backward(cs.theta_dev, sv, cs.B, cs.s_dev, cs.t, b)
    finally:
        n, ms, work = pk.prof_end()
    torch.cuda.synchronize()
    assert n > 0 and ms > 0 and work > 0
    assert torch.equal(a, b)


# ------------------------------------------------------------ aggregation
@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("n,W", [(1, 4), (77, 4), (4096, 2), (100003, 5), (262144, 8)])
def test_aggregate_matches_oracle(dt, n, W):
    say(f"case: aggregate n={n} W={W} {dt}")
    ctx = pk.Context(TINY)
    t = np.asarray(synth.uniform_grid(2 * W)[:W], dtype=np.float32)
    s_np = [rounded(synth.normal(n, 50 + j), dt) for j in range(W)]
    s = [to_dev(x, dt) for x in s_np]
    sb, sc = torch.empty_like(s[0]), torch.empty_like(s[0])
    ctx.aggregate(s, t, sb, sc)
    wb, wc = jagg.aggregate(s_np, t.astype(np.float64))
    gb, gc = sb.double().cpu().numpy(), sc.double().cpu().numpy()
    a = jagg.alpha(t.astype(np.float64))
    # error bound of W fused multiply-adds in fp32 (weights rounded to fp32 too):
    # (W + 1) * 2^-24 * sum_j |w_j s_j|, plus one rounding of the result to the
    # storage dtype (half an ulp: 2^-24 fp32, 2^-8 bf16, relative)
    mag_b = sum(abs(1 - a[j]) * np.abs(s_np[j]) for j in range(W))
    mag_c = sum(abs(a[j]) * np.abs(s_np[j]) for j in range(W))
    rnd = 2.0 ** -24 if dt == torch.float32 else 2.0 ** -8
    assert np.all(np.abs(gb - wb) <= (W + 1) * 2.0 ** -24 * mag_b + rnd * np.abs(wb) + 1e-30)
    assert np.all(np.abs(gc - wc) <= (W + 1) * 2.0 ** -24 * mag_c + rnd * np.abs(wc) + 1e-30)
    if W == 2:
        assert torch.equal(sb, s[0]) and torch.equal(sc, s[1])


# ---------------------------------------------------------- routing scores
def test_group_scores_and_routing_bit_exact():
    say("case: group scores + routing")
    ctx = pk.Context(TINY)
    rhos = [0.97, 0.9, 0.81, 0.62, 0.4]
    W, n = 4, 262144
    scores, oscores = [], []
    for g, rho in enumerate(rhos):
        h = synth.hidden_profile(W, n, rho, seed=900 + g)
        hd = [to_dev(x, torch.float32) for x in h]
        hf = [x.double().cpu().numpy() for x in hd]
        scores.append(ctx.group_score(hd))
        oscores.append(jagg.group_score(hf))
    for s, o, r in zip(scores, oscores, rhos):
        assert abs(s - o) < 1e-9 and abs(s - r) < 1e-5
    for tau in (0.5, 0.7, 0.85):
        m, f = pk.route(len(rhos), scores=scores, tau=tau)
        om, of = jagg.route(len(rhos), scores=oscores, tau=tau)
        assert m == list(om) and f == of
