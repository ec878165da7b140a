"""GPU parity of the linear-layer backward products (jagg_linear_grad), the
kernels that carry most of the backward's FLOPs: input gradient dY W, input
gradient through the tanh-GELU derivative, and weight gradient dY^T X with
fp32 accumulation into the gradient (beta = 1).  The oracle gets the same
bf16-rounded operands in fp64 (mmdit.wgrad, mmdit.gelu_tanh_grad and a plain
matrix product).  Bars: fp32 results relative L2 <= 1e-5 (fp32 accumulation
of bf16 products over K <= 12288 terms); bf16 results <= 8e-3 (one rounding
to bf16, 2^-9 relative, on every element).  Shapes span several 256 x 256
tiles with ragged edges in every dimension; the full-size shapes of the block
workload are checked on sampled rows and columns."""
import sys

import numpy as np
import pytest
import torch

import paper_2607_17572_amd as pk
import synth
from harness import rel_l2, rounded, to_dev
from oracle import mmdit

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


_CTX = {}


def ctx():
    if "c" not in _CTX:
        _CTX["c"] = pk.Context(pk.config("tiny"))
    return _CTX["c"]


def operands(rows, n_out, n_in, seed):
    dY = rounded(synth.normal((rows, n_out), seed), torch.bfloat16)
    X = rounded(synth.normal((rows, n_in), seed + 1), torch.bfloat16)
    W = rounded(synth.normal((n_out, n_in), seed + 2, scale=0.02), torch.bfloat16)
    C0 = synth.normal((n_out, n_in), seed + 3)
    return dY, X, W, C0


# ragged in every dimension, several tiles, K not a multiple of the k tile;
# the last shape gives both products 16 x 16 tiles of 256 x 256 (one round of
# 256 CUs, against two rounds of the smaller tiles), so they run the 8-wave
# 256 x 256 direct-to-LDS kernel with a ragged N edge and a ragged k-tile count
SHAPES = [(37, 20, 12), (8, 8, 8), (200, 136, 72), (1000, 520, 776), (1032, 3072, 264), (520, 1048, 3080),
          (4000, 4064, 4040)]


@pytest.mark.parametrize("rows,n_out,n_in", SHAPES)
def test_linear_grad_matches_oracle(rows, n_out, n_in):
    say(f"case: linear grad rows={rows} n_out={n_out} n_in={n_in}")
    dY, X, W, C0 = operands(rows, n_out, n_in, 100 + rows)
    dYd, Xd, Wd = to_dev(dY, torch.bfloat16), to_dev(X, torch.bfloat16), to_dev(W, torch.bfloat16)
    c = ctx()
    # input gradient, fp32 and bf16 results
    want = dY @ W
    out = torch.empty(rows, n_in, dtype=torch.float32, device="cuda")
    c.linear_grad(pk.DGRAD, dYd, Wd, out)
    e = rel_l2(out.double().cpu().numpy(), want)
    say(f"  dgrad fp32 rel L2 {e:.2e}")
    assert e <= 1e-5
    outb = torch.empty(rows, n_in, dtype=torch.bfloat16, device="cuda")
    c.linear_grad(pk.DGRAD, dYd, Wd, outb)
    e = rel_l2(outb.double().cpu().numpy(), want)
    say(f"  dgrad bf16 rel L2 {e:.2e}")
    assert e <= 8e-3
    # input gradient through GELU'
    pre = rounded(synth.normal((rows, n_in), 7 + rows), torch.bfloat16)
    c.linear_grad(pk.DGRAD_GELU, dYd, Wd, outb, pre=to_dev(pre, torch.bfloat16))
    e = rel_l2(outb.double().cpu().numpy(), want * mmdit.gelu_tanh_grad(pre))
    say(f"  dgrad gelu rel L2 {e:.2e}")
    assert e <= 8e-3
    # weight gradient: overwrite, then accumulate onto an existing gradient
    gw = mmdit.wgrad(dY, X)
    dW = torch.empty(n_out, n_in, dtype=torch.float32, device="cuda")
    c.linear_grad(pk.WGRAD, dYd, Xd, dW, beta=0.0)
    e = rel_l2(dW.double().cpu().numpy(), gw)
    say(f"  wgrad beta=0 rel L2 {e:.2e}")
    assert e <= 1e-5
    dW.copy_(torch.from_numpy(C0.astype(np.float32)))
    c.linear_grad(pk.WGRAD, dYd, Xd, dW, beta=1.0)
    e = rel_l2(dW.double().cpu().numpy(), C0.astype(np.float32).astype(np.float64) + gw)
    say(f"  wgrad beta=1 rel L2 {e:.2e}")
    assert e <= 1e-5


# the block workload's weight-gradient and input-gradient products at full
# size (pair batch: 8192 image rows, 1024 text rows), sampled
FULL = [(8192, 12288, 3072), (8192, 3072, 12288), (8192, 9216, 3072), (1024, 3072, 3072), (1024, 12288, 3072)]


@pytest.mark.parametrize("rows,n_out,n_in", FULL)
def test_linear_grad_fullsize_sampled(rows, n_out, n_in):
    say(f"case: full-size linear grad rows={rows} n_out={n_out} n_in={n_in}")
    sd = rows + n_out + n_in
    dY = torch.from_numpy(synth.normal((rows, n_out), sd, dtype=np.float32)).to(torch.bfloat16)
    X = torch.from_numpy(synth.normal((rows, n_in), sd + 1, dtype=np.float32)).to(torch.bfloat16)
    W = torch.from_numpy(synth.normal((n_out, n_in), sd + 2, scale=0.02, dtype=np.float32)).to(torch.bfloat16)
    c = ctx()
    dW = torch.ones(n_out, n_in, dtype=torch.float32, device="cuda")
    c.linear_grad(pk.WGRAD, dY.cuda(), X.cuda(), dW, beta=1.0)
    dX = torch.empty(rows, n_in, dtype=torch.float32, device="cuda")
    c.linear_grad(pk.DGRAD, dY.cuda(), W.cuda(), dX)
    dW, dX = dW.cpu().double().numpy(), dX.cpu().double().numpy()
    rs = np.random.default_rng(5)
    oi = rs.choice(n_out, 48, replace=False)
    ii = rs.choice(n_in, 48, replace=False)
    ri = rs.choice(rows, 48, replace=False)
    dYn, Xn, Wn = dY.double().numpy(), X.double().numpy(), W.double().numpy()
    want_w = 1.0 + mmdit.wgrad(dYn[:, oi], Xn[:, ii])
    want_x = dYn[ri] @ Wn[:, ii]
    ew = rel_l2(dW[np.ix_(oi, ii)], want_w)
    ex = rel_l2(dX[np.ix_(ri, ii)], want_x)
    say(f"  sampled wgrad rel L2 {ew:.2e}, dgrad {ex:.2e}")
    assert ew <= 1e-5 and ex <= 1e-5
