"""Full-size parity of the bench workload: one double-stream block, hidden
3072, 24 x 128 heads, MLP 12288, 4096 image + 512 text tokens, batch 1, W = 4,
bf16.  The JAGG group backward (composites + one VJP over the batched endpoint
pair, the launch configuration the bench times) is compared with the oracle
run in fp32 on the same bf16-rounded values: relative L2 <= 2e-2, globally and
per tensor.  The per-step path is checked through the W = 2 identity and its
agreement with the JAGG path's kernels at full size."""
import sys

import numpy as np
import pytest
import torch

import paper_2607_17572_amd as pk
from harness import Case, compare_grads, rel_l2

pytestmark = pytest.mark.gpu


def test_fullsize_block_jagg_matches_oracle():
    print("case: full-size block JAGG W=4 vs fp32 oracle", flush=True)
    cs = Case(pk.config("block"), B=1, W=4, T=16)
    got = cs.gpu_jagg()
    torch.cuda.synchronize()
    print("gpu done; running oracle (fp32)", flush=True)
    want = cs.oracle_jagg(dtype=np.float32)
    eg, worst = compare_grads(cs, got, want, 2e-2)
    print(f"full-size JAGG rel L2 {eg:.3e}, worst tensor {worst}", flush=True)


def test_fullsize_block_w2_identity_and_linearity():
    """W = 2 makes JAGG the exact per-step gradient; at full size the two paths
    (one batch-2 VJP vs two batch-1 VJPs) must agree to bf16 accumulation noise."""
    print("case: full-size block W=2 identity", flush=True)
    cs = Case(pk.config("block"), B=1, W=2, T=16)
    a = cs.gpu_jagg().double().cpu().numpy()
    b = cs.gpu_perstep().double().cpu().numpy()
    e = rel_l2(a, b)
    print(f"W=2 jagg vs perstep rel L2 {e:.3e}", flush=True)
    assert e < 1e-2


def test_fullsize_grpo_composites_match_oracle():
    """Phases 2+3 fused at the bench's size (block workload, 4608 x 3072 per
    sample, W = 4, batch 1), with v_0 / v_{W-1} read in place from an endpoint
    pair output and the middle steps from one batched output, as the bench's
    update stage does.  Stats (log pi, rho, loss) and clip decisions against
    the oracle in fp64; composites within the bf16 bar."""
    print("case: full-size GRPO composites, block workload W=4", flush=True)
    from test_gpu_grpo import EPS, ADV_CLIP, Window, batch_of, check_stats
    from oracle import jagg
    c = pk.config("block")
    w = Window(c, 1)
    s_want, st_want = w.oracle()
    ctx = pk.Context(c)
    v, z, lpo, adv = w.dev()
    pair = batch_of(c, 1, [v[0], v[-1]])
    mid = batch_of(c, 1, v[1:-1])
    vs = [(pair, 2, 0)] + [(mid, w.W - 2, j) for j in range(w.W - 2)] + [(pair, 2, 1)]
    del v
    sb = torch.empty(w.shape, dtype=w.dt, device="cuda")
    sc = torch.empty_like(sb)
    stats = torch.zeros((w.W, 1, 3), dtype=torch.float64, device="cuda")
    ctx.grpo_composites(vs, z, w.t, w.sigma, lpo, adv, sb, sc, EPS, ADV_CLIP, stats=stats)
    torch.cuda.synchronize()
    check_stats(stats, st_want)
    wb, wc = jagg.aggregate(s_want, w.t[:w.W].astype(np.float64))
    eb, ec = rel_l2(sb.double().cpu().numpy(), wb), rel_l2(sc.double().cpu().numpy(), wc)
    print(f"full-size GRPO composites rel L2 {eb:.2e} {ec:.2e}", flush=True)
    assert eb <= 8e-3 and ec <= 8e-3


# Full-width slice: one double-stream and one single-stream block at the
# model width of the Flux-like workloads (hidden 3072, 24 x 128 heads, MLP
# 12288, text width 4096, 16 latent channels, 2x2 patches), with the full
# embeddings and final layer, at token counts the oracle runs in seconds.
WIDE = dict(n_double=1, n_single=1, hidden=3072, heads=24, head_dim=128, mlp_hidden=12288, in_ch=16, patch=2,
            txt_dim=4096, t_freq_dim=256, act_dtype=pk.BF16)


@pytest.mark.parametrize("B,lat,n_txt", [(2, 32, 64), (8, 16, 32)], ids=["batch2_256+64", "batch8_64+32"])
def test_fullwidth_slice_matches_oracle(B, lat, n_txt):
    """JAGG group backward (W = 4, batch-2B endpoint pair) of the full-width
    slice against the fp32 oracle on the same bf16-rounded values, with fp32
    and with bf16 parameter gradients; raw per-tensor and global relative L2
    <= 2e-2.  The batch-8 case also runs the per-step baseline into a bf16
    gradient (four accumulating VJPs, the bf16 accumulate epilogue)."""
    import dataclasses
    print(f"case: full-width slice 1d+1s, batch {B}, {lat // 2}^2 image + {n_txt} text tokens", flush=True)
    cfg = pk.Config(**WIDE, lat_h=lat, lat_w=lat, n_txt=n_txt, grad_dtype=pk.F32)
    cs = Case(cfg, B=B, W=4, T=16)
    got32 = cs.gpu_jagg()
    ctx16 = pk.Context(dataclasses.replace(cfg, grad_dtype=pk.BF16))
    sv = cs.saved_pair()
    got16 = torch.zeros(ctx16.n_params, dtype=torch.bfloat16, device="cuda")
    ctx16.group_backward(cs.theta_dev, sv, B, cs.s_dev, cs.t, got16, 0.0)
    ps16 = None
    if B == 8:
        saved = [cs.forward(j)[1] for j in range(cs.W)]
        ps16 = torch.zeros_like(got16)
        ctx16.perstep_group_backward(cs.theta_dev, saved, B, cs.s_dev, ps16, 0.0)
    torch.cuda.synchronize()
    print("gpu done; running oracle (fp32)", flush=True)
    want = cs.oracle_jagg(dtype=np.float32)
    eg, worst = compare_grads(cs, got32, want, 2e-2, report=True)
    print(f"  fp32 dtheta: rel L2 {eg:.3e}, worst tensor {worst}", flush=True)
    eg, worst = compare_grads(cs, got16, want, 2e-2, report=True)
    print(f"  bf16 dtheta: rel L2 {eg:.3e}, worst tensor {worst}", flush=True)
    if ps16 is not None:
        want_e = cs.oracle_exact(dtype=np.float32)
        eg, worst = compare_grads(cs, ps16, want_e, 2e-2, report=True)
        print(f"  per-step, bf16 dtheta: rel L2 {eg:.3e}, worst tensor {worst}", flush=True)
