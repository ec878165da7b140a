"""Pins for the oracle network and its VJP: central finite differences,
closed-form special cases, structural zeros and batch linearity.  CPU only."""
import numpy as np
import pytest

import synth
from oracle import mmdit

TINY = mmdit.Config(n_double=2, n_single=1, hidden=16, heads=2, head_dim=8, mlp_hidden=24,
                    in_ch=2, patch=2, lat_h=4, lat_w=6, n_txt=3, txt_dim=8, t_freq_dim=16)
TINY_DBL = mmdit.Config(n_double=2, n_single=0, hidden=16, heads=2, head_dim=8, mlp_hidden=24,
                        in_ch=2, patch=1, lat_h=2, lat_w=3, n_txt=3, txt_dim=8, t_freq_dim=16)
TINY_BLOCK = mmdit.Config(n_double=1, n_single=0, hidden=16, heads=2, head_dim=8, mlp_hidden=24,
                          lat_h=2, lat_w=2, n_txt=3, t_freq_dim=16, block_only=True)


def layout(cfg):
    lay, _ = mmdit.param_layout(cfg)
    return [(n, off, int(np.prod(s))) for n, s, off in lay]


def theta(cfg, std=0.3, seed=1):
    # a large std so that the network is far from linear and every term matters
    return synth.theta(layout(cfg), seed=seed, std=std, gain_std=0.3, total=mmdit.param_layout(cfg)[1])


def inputs(cfg, B, seed, t=None):
    t = np.linspace(0.9, 0.3, B) if t is None else np.asarray(t, dtype=np.float64)
    if cfg.block_only:
        return mmdit.Inputs(t=t, x_txt=synth.normal((B, cfg.n_txt, cfg.hidden), seed),
                            x_img=synth.normal((B, cfg.n_img, cfg.hidden), seed + 1))
    return mmdit.Inputs(t=t, z=synth.normal((B, cfg.in_ch, cfg.lat_h, cfg.lat_w), seed),
                        txt=synth.normal((B, cfg.n_txt, cfg.txt_dim), seed + 1))


def cot(cfg, B, seed):
    if cfg.block_only:
        return (synth.normal((B, cfg.n_txt, cfg.hidden), seed), synth.normal((B, cfg.n_img, cfg.hidden), seed + 1))
    return synth.normal((B, cfg.in_ch, cfg.lat_h, cfg.lat_w), seed)


def loss(cfg, th, inp, s):
    v, _ = mmdit.forward(cfg, mmdit.unflatten(cfg, th), inp)
    if isinstance(v, tuple):
        return sum(float(np.sum(a * b)) for a, b in zip(v, s))
    return float(np.sum(v * s))


@pytest.mark.parametrize("cfg", [TINY, TINY_DBL, TINY_BLOCK], ids=["full", "double_only", "block_only"])
def test_vjp_matches_central_finite_differences_per_tensor(cfg):
    """<J^T s, d> = d/dh <v(theta + h d), s> for a random direction d in each tensor."""
    B = 2
    th = theta(cfg)
    inp = inputs(cfg, B, 10)
    s = cot(cfg, B, 20)
    g = mmdit.vjp_flat(cfg, th, inp, s)
    lay, total = mmdit.param_layout(cfg)
    rs = np.random.default_rng(3)
    h = 1e-5
    for name, shape, off in lay:
        n = int(np.prod(shape))
        d = np.zeros(total)
        d[off:off + n] = rs.standard_normal(n)
        fd = (loss(cfg, th + h * d, inp, s) - loss(cfg, th - h * d, inp, s)) / (2 * h)
        an = float(np.dot(g, d))
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(fd)), (name, fd, an)


def test_double_block_closed_form_constant_value_path():
    """W_mod = 0, scale1 = scale2 = -1: the LayerNorm branches collapse to the
    shifts.  With the value rows of both streams' projections zero and one
    shared value bias b_v, every joint token carries v = b_v, attention returns
    it whatever q and k are, and each stream's output is
    x + g1*(W_o b_v + b_o) + g2*(W_2 gelu(W_1 sh2 + b_1) + b_2)."""
    cfg = TINY_BLOCK
    D, F = cfg.hidden, cfg.mlp_hidden
    th = theta(cfg, std=0.5, seed=7)
    P = mmdit.unflatten(cfg, th)
    rs = np.random.default_rng(8)
    bv_shared = rs.standard_normal(D)
    for s in ("txt", "img"):
        pre = f"double.0.{s}."
        P[pre + "qkv.w"][2 * D:3 * D] = 0.0
        P[pre + "qkv.b"][2 * D:3 * D] = bv_shared
        P[pre + "mod.w"][:] = 0.0
        b = rs.standard_normal(6 * D)
        b[D:2 * D] = -1.0      # scale1
        b[4 * D:5 * D] = -1.0  # scale2
        P[pre + "mod.b"][:] = b
    inp = inputs(cfg, 2, 30)
    (ot, oi), _ = mmdit.forward(cfg, P, inp)
    for s, x, o in (("txt", inp.x_txt, ot), ("img", inp.x_img, oi)):
        pre = f"double.0.{s}."
        b = P[pre + "mod.b"]
        sh2, g1, g2 = b[3 * D:4 * D], b[2 * D:3 * D], b[5 * D:6 * D]
        bv = bv_shared
        Wo, bo = P[pre + "o.w"], P[pre + "o.b"]
        W1, b1, W2, b2 = P[pre + "fc1.w"], P[pre + "fc1.b"], P[pre + "fc2.w"], P[pre + "fc2.b"]
        y1 = [sum(Wo[r, c] * bv[c] for c in range(D)) + bo[r] for r in range(D)]
        pre_act = [sum(W1[r, c] * sh2[c] for c in range(D)) + b1[r] for r in range(F)]
        hh = [0.5 * u * (1 + np.tanh(np.sqrt(2 / np.pi) * (u + 0.044715 * u ** 3))) for u in pre_act]
        y2 = [sum(W2[r, c] * hh[c] for c in range(F)) + b2[r] for r in range(D)]
        want = x + np.array([g1[r] * y1[r] + g2[r] * y2[r] for r in range(D)])[None, None, :]
        np.testing.assert_allclose(o, want, rtol=1e-12, atol=1e-12)


def test_single_block_and_time_mlp_closed_form():
    """Single block with W_mod = 0, scale = -1: the normalised input collapses to
    the shift, so v = W_v sh + b_v and the MLP input u = W_u sh + b_u are the same
    for every token; output = x + gate*(W_out [v, gelu(u)] + b_out).  The time MLP
    with W_t1 = 0 gives vec = W_t2 silu(b_t1) + b_t2."""
    cfg = mmdit.Config(n_double=0, n_single=1, hidden=16, heads=2, head_dim=8, mlp_hidden=24,
                       in_ch=2, patch=1, lat_h=2, lat_w=2, n_txt=2, txt_dim=8, t_freq_dim=16)
    D, F = cfg.hidden, cfg.mlp_hidden
    P = mmdit.unflatten(cfg, theta(cfg, std=0.5, seed=9))
    P["single.0.mod.w"][:] = 0.0
    P["single.0.mod.b"][D:2 * D] = -1.0
    P["t_in.w"][:] = 0.0
    inp = inputs(cfg, 1, 40)
    _, cache = mmdit.forward(cfg, P, inp)
    x_in = np.concatenate([mmdit.linear(inp.txt, P["txt_in.w"], P["txt_in.b"]),
                           mmdit.linear(mmdit.patchify(cfg, inp.z), P["img_in.w"], P["img_in.b"])], axis=1)
    b = P["single.0.mod.b"]
    gate = b[2 * D:3 * D]
    sh = b[:D]
    Win, bin_ = P["single.0.in.w"], P["single.0.in.b"]
    proj = [sum(Win[r, c] * sh[c] for c in range(D)) + bin_[r] for r in range(3 * D + F)]
    catv = proj[2 * D:3 * D] + [0.5 * u * (1 + np.tanh(np.sqrt(2 / np.pi) * (u + 0.044715 * u ** 3)))
                                for u in proj[3 * D:]]
    Wout, bout = P["single.0.out.w"], P["single.0.out.b"]
    y = np.array([sum(Wout[r, c] * catv[c] for c in range(D + F)) + bout[r] for r in range(D)])
    np.testing.assert_allclose(cache["x_last"], x_in + gate * y, rtol=1e-12, atol=1e-12)
    h1 = P["t_in.b"]
    sh = [u / (1 + np.exp(-u)) for u in h1]
    vec = [sum(P["t_out.w"][r, c] * sh[c] for c in range(D)) + P["t_out.b"][r] for r in range(D)]
    np.testing.assert_allclose(cache["vec"][0], vec, rtol=1e-12, atol=1e-12)


def test_no_block_model_closed_form():
    """No blocks, final modulation zero: v = unpatchify(LN(patches W_in^T + b_in) W_f^T + b_f),
    written with explicit pixel loops over the (c, py, px) feature convention."""
    cfg = mmdit.Config(n_double=0, n_single=0, hidden=8, heads=1, head_dim=8, mlp_hidden=8,
                       in_ch=2, patch=2, lat_h=4, lat_w=2, n_txt=1, txt_dim=4, t_freq_dim=8)
    P = mmdit.unflatten(cfg, theta(cfg, std=0.5, seed=11))
    P["final.mod.w"][:] = 0.0
    P["final.mod.b"][:] = 0.0
    inp = inputs(cfg, 1, 50)
    v, _ = mmdit.forward(cfg, P, inp)
    z = inp.z[0]
    D, p = cfg.hidden, 2
    for r in range(2):
        for c in range(1):
            feat = [z[ch, r * p + py, c * p + px] for ch in range(2) for py in range(p) for px in range(p)]
            x = [sum(P["img_in.w"][d, f] * feat[f] for f in range(8)) + P["img_in.b"][d] for d in range(D)]
            mu = sum(x) / D
            var = sum((a - mu) ** 2 for a in x) / D
            xh = [(a - mu) / np.sqrt(var + 1e-6) for a in x]
            out = [sum(P["final.w"][f, d] * xh[d] for d in range(D)) + P["final.b"][f] for f in range(8)]
            for ch in range(2):
                for py in range(p):
                    for px in range(p):
                        assert abs(v[0, ch, r * p + py, c * p + px] - out[ch * 4 + py * 2 + px]) < 1e-12


def test_structural_zero_gradients_of_last_text_stream():
    """With double blocks only, the final layer reads image tokens only, so in the
    last block every parameter that reaches nothing but the text output gets an
    exactly zero gradient: text out-projection, text MLP, text query path and
    the text modulation chunks gate1, shift2, scale2, gate2."""
    cfg = TINY_DBL
    B = 2
    th = theta(cfg)
    G = mmdit.vjp(cfg, mmdit.unflatten(cfg, th), mmdit.forward(cfg, mmdit.unflatten(cfg, th), inputs(cfg, B, 60))[1],
                  cot(cfg, B, 61))
    D = cfg.hidden
    last = f"double.{cfg.n_double - 1}.txt."
    for n in ("o.w", "o.b", "fc1.w", "fc1.b", "fc2.w", "fc2.b", "q_gain"):
        assert np.all(G[last + n] == 0.0), n
    assert np.all(G[last + "qkv.w"][:D] == 0.0) and np.all(G[last + "qkv.b"][:D] == 0.0)
    assert np.all(G[last + "mod.w"][2 * D:] == 0.0) and np.all(G[last + "mod.b"][2 * D:] == 0.0)
    # ... while the key/value path and the first block's text stream do get gradient
    assert np.abs(G[last + "qkv.w"][D:]).max() > 0
    assert np.abs(G[last + "k_gain"]).max() > 0
    assert np.abs(G["double.0.txt.o.w"]).max() > 0


def test_final_bias_gradient_is_input_independent():
    """d(final.b)[f] = sum over samples and tokens of s at feature f, exactly."""
    cfg = TINY
    th = theta(cfg)
    s = cot(cfg, 2, 70)
    G = mmdit.vjp(cfg, mmdit.unflatten(cfg, th), mmdit.forward(cfg, mmdit.unflatten(cfg, th), inputs(cfg, 2, 71))[1], s)
    want = mmdit.patchify(cfg, s).sum(axis=(0, 1))
    np.testing.assert_allclose(G["final.b"], want, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("cfg", [TINY, TINY_BLOCK], ids=["full", "block_only"])
def test_vjp_is_additive_over_the_batch(cfg):
    """The VJP of a batch is the sum of the per-sample VJPs (what makes the
    joint endpoint pass equal to two separate endpoint passes)."""
    th = theta(cfg)
    inp = inputs(cfg, 2, 80)
    s = cot(cfg, 2, 81)
    g = mmdit.vjp_flat(cfg, th, inp, s)

    def one(b):
        sl = slice(b, b + 1)
        i = mmdit.Inputs(t=inp.t[sl], z=None if inp.z is None else inp.z[sl],
                         txt=None if inp.txt is None else inp.txt[sl],
                         x_txt=None if inp.x_txt is None else inp.x_txt[sl],
                         x_img=None if inp.x_img is None else inp.x_img[sl])
        sb = tuple(a[sl] for a in s) if isinstance(s, tuple) else s[sl]
        return mmdit.vjp_flat(cfg, th, i, sb)

    np.testing.assert_allclose(g, one(0) + one(1), rtol=1e-12, atol=1e-13)


def test_param_counts_match_architecture_sizes():
    """Double block 36 D^2 + biases; single block 15 D^2 + biases (D=3072, MLP=4D)."""
    cfg = mmdit.Config(n_double=1, n_single=1, hidden=3072, heads=24, head_dim=128, mlp_hidden=12288,
                       in_ch=16, patch=2, lat_h=128, lat_w=128, n_txt=512, txt_dim=4096, t_freq_dim=256)
    shapes = dict(mmdit.param_shapes(cfg))
    dbl = sum(int(np.prod(v)) for k, v in shapes.items() if k.startswith("double.0."))
    sgl = sum(int(np.prod(v)) for k, v in shapes.items() if k.startswith("single.0."))
    D = 3072
    assert dbl == 36 * D * D + 2 * (6 * D + 3 * D + D + 4 * D + D + 2 * 128)
    assert sgl == 15 * D * D + 3 * D + 7 * D + D + 2 * 128


def test_attention_composition_worked_example():
    """One double block, one head of Dh = 4, one text token and a 2 x 2 image
    grid, written so that the block's output minus its input is the attention
    output itself: modulation weights zero with gate1 = 1 and every other
    chunk 0, query and key rows of the qkv projection zero with bias (1, 1, 1,
    1), value rows the identity, output projection the identity, MLP gate 0.
    Every token row has mean 0 and variance 1, so LayerNorm divides it by
    r = sqrt(1 + eps), and the RMS of the all-ones query/key bias is the same r.

    Worked by hand: the normalised query of a token is g_q / r (its stream's
    gain), the key g_k / r; RoPE turns pair (0,1) by the token's grid row and
    pair (2,3) by its grid column (frequency 1 for Dh = 4; text at (0, 0)).
    For rotations R(a), R(b): R(a)x . R(b)y = (x0 y0 + x1 y1) cos(b - a) +
    (x1 y0 - x0 y1) sin(b - a), so the logit of query i and key j is half the
    sum of that expression over the two pairs; the probabilities are the
    softmax of row i over the keys j, and the output of token i is
    sum_j p_ij x_j / r.  The gains differ within each pair, so RoPE applied
    before the RMSNorm gain, pairs taken as halves instead of interleaved,
    another logit scale, or a softmax over queries would all change it."""
    import math
    cfg = mmdit.Config(n_double=1, n_single=0, hidden=4, heads=1, head_dim=4, mlp_hidden=4, patch=1,
                       lat_h=2, lat_w=2, n_txt=1, t_freq_dim=4, block_only=True)
    P = mmdit.unflatten(cfg, np.zeros(mmdit.param_layout(cfg)[1]))
    gains = {"txt": ((1.5, 0.5, 1.0, 2.0), (1.0, 2.0, 0.5, 1.0)),
             "img": ((0.5, 2.5, 2.0, 1.0), (2.0, 0.5, 1.0, 1.5))}
    for s in ("txt", "img"):
        pre = f"double.0.{s}."
        P[pre + "mod.b"][8:12] = 1.0                       # gate1
        P[pre + "qkv.b"][0:8] = 1.0                        # query and key bias
        P[pre + "qkv.w"][8:12] = np.eye(4)                 # value = normalised input
        P[pre + "o.w"][:] = np.eye(4)
        P[pre + "q_gain"][:] = gains[s][0]
        P[pre + "k_gain"][:] = gains[s][1]
    rows = [(1, -1, 1, -1), (-1, 1, -1, 1), (1, 1, -1, -1), (-1, -1, 1, 1), (1, -1, -1, 1)]
    pos = [(0, 0), (0, 0), (0, 1), (1, 0), (1, 1)]        # text token, then the image grid row-major
    stream = ["txt", "img", "img", "img", "img"]
    x = np.array(rows, dtype=np.float64)
    inp = mmdit.Inputs(t=np.array([0.5]), x_txt=x[None, :1], x_img=x[None, 1:])
    (ot, oi), _ = mmdit.forward(cfg, P, inp)
    got = np.concatenate([ot[0], oi[0]], axis=0) - x
    r = math.sqrt(1.0 + 1e-6)

    def dot_rot(xv, a, yv, b):
        return (xv[0] * yv[0] + xv[1] * yv[1]) * math.cos(b - a) + (xv[1] * yv[0] - xv[0] * yv[1]) * math.sin(b - a)

    for i in range(5):
        q = [g / r for g in gains[stream[i]][0]]
        logits = []
        for j in range(5):
            k = [g / r for g in gains[stream[j]][1]]
            l0 = dot_rot(q[0:2], pos[i][0], k[0:2], pos[j][0])
            l1 = dot_rot(q[2:4], pos[i][1], k[2:4], pos[j][1])
            logits.append(0.5 * (l0 + l1))
        e = [math.exp(v) for v in logits]
        p = [v / sum(e) for v in e]
        want = [sum(p[j] * rows[j][d] / r for j in range(5)) for d in range(4)]
        np.testing.assert_allclose(got[i], want, rtol=1e-12, atol=1e-13)
