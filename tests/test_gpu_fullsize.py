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
