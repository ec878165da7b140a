"""Allocation-free group scores (jagg_group_scores_noalloc) against the
workspace-backed entry point (jagg_group_scores): same kernels, so the scores
must be bitwise equal.  Two calls in a row, the second with fewer elements and
a smaller W, both on a context that has no workspace bound when the
allocation-free call runs; bf16 and fp32 inputs."""
import sys

import numpy as np
import pytest
import torch

import paper_2607_17572_amd as pk
import synth
from harness import to_dev
from oracle import jagg

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16])
def test_noalloc_scores_equal_workspace_scores(dt):
    for (W, n, rho, seed) in ((8, 1000003, 0.83, 11), (3, 4097, 0.41, 12)):
        say(f"case: no-alloc group scores W={W} n={n} {dt}")
        ctx = pk.Context(pk.config("tiny"))
        h = [to_dev(x, dt) for x in synth.hidden_profile(W, n, rho, seed=seed)]
        out = torch.full((1,), float("nan"), dtype=torch.float64, device="cuda")
        ctx.group_score_noalloc(h, out)          # no workspace bound yet
        torch.cuda.synchronize()
        got = out.item()
        want = ctx.group_score(h)                # binds a workspace, uses its head
        o = jagg.group_score([x.double().cpu().numpy() for x in h])
        say(f"  no-alloc {got!r}  workspace {want!r}  oracle {o!r}")
        assert got == want
        assert abs(got - o) < 1e-9
