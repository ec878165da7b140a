"""Oracle MMDiT: plain numpy forward and hand-derived VJP to the parameters.

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously correct CPU
reference that the HIP path is checked against.  Only the tests, the smoke
entry and the bench's CPU-baseline leg may import it; the product path never
does.  It shares no code with the HIP library.

What it computes.  The paper gives no architecture for its DiT beyond the
attention equations of the backward-cost appendix (attention backward,
equations for dV, dP, dS, dQ, dK); it trains Flux- and QwenImage-class
MMDiTs (Experiments, setup).  The network below is the standard MMDiT written
out from that description; every choice the paper leaves open is a stated
reading:

* time embedding: temb(t)_k = cos(1000 t w_k), temb(t)_{F/2+k} = sin(1000 t w_k),
  w_k = 10000^(-k/(F/2)); vec = SiLU(temb W_t1^T + b_t1) W_t2^T + b_t2;
* image tokens: p x p patches, feature index (c, py, px), row-major token
  order, embedded by a linear layer; text tokens by a linear layer;
* double-stream block (separate weights per stream, joint attention over
  [text; image] tokens): adaLN modulation (shift1, scale1, gate1, shift2,
  scale2, gate2) = SiLU(vec) W_mod^T + b_mod; LayerNorm without affine
  (eps 1e-6); q, k RMS-normalised per head (eps 1e-6) with a learned gain;
  2-D rotary embedding; softmax attention with scale 1/sqrt(Dh); gated
  residuals; tanh-GELU MLP;
* single-stream block: (shift, scale, gate); one input projection to
  [q, k, v, mlp]; output projection of [attention, GELU(mlp)];
* final layer: (shift, scale) modulation of LayerNorm(image tokens), linear
  to patch features, unpatchify;
* rotary layout: head dim split in halves (row axis, column axis), rotating
  interleaved pairs (2i, 2i+1) with frequency theta^(-2i/(Dh/2)), theta=1e4;
  text tokens sit at position (0, 0); image token (r, c) at (r, c);
* every linear weight is stored [out][in] and applied as x W^T + b.

A "block only" model (kernel-level workload) keeps the time-embedding MLP and
the double-stream blocks but has no input embeddings and no final layer: its
input and output are the two token streams.

The VJP uses the textbook derivatives (LayerNorm, RMSNorm, rotation
transpose, softmax, tanh-GELU, SiLU).  It returns gradients for every
parameter; no input gradient is needed.  Pins: finite differences, library
routines for each operator, closed-form special cases, structural zeros
(see the oracle tests).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

LN_EPS = 1e-6
RMS_EPS = 1e-6
ROPE_THETA = 10000.0
GELU_C = np.sqrt(2.0 / np.pi)


@dataclass(frozen=True)
class Config:
    n_double: int
    n_single: int
    hidden: int
    heads: int
    head_dim: int
    mlp_hidden: int
    in_ch: int = 4
    patch: int = 1
    lat_h: int = 4
    lat_w: int = 4
    n_txt: int = 8
    txt_dim: int = 64
    t_freq_dim: int = 256
    block_only: bool = False

    @property
    def grid_h(self):
        return self.lat_h // self.patch

    @property
    def grid_w(self):
        return self.lat_w // self.patch

    @property
    def n_img(self):
        return self.grid_h * self.grid_w

    @property
    def n_tok(self):
        return self.n_txt + self.n_img

    @property
    def patch_dim(self):
        return self.in_ch * self.patch * self.patch


# ----------------------------------------------------------------------------
# parameter layout (names, shapes) and flat packing
# ----------------------------------------------------------------------------
ALIGN = 128  # every tensor starts at a multiple of 128 elements


def param_shapes(cfg: Config):
    D, Dh, F, M = cfg.hidden, cfg.head_dim, cfg.mlp_hidden, cfg.t_freq_dim
    out = [("t_in.w", (D, M)), ("t_in.b", (D,)), ("t_out.w", (D, D)), ("t_out.b", (D,))]
    if not cfg.block_only:
        out += [("img_in.w", (D, cfg.patch_dim)), ("img_in.b", (D,)),
                ("txt_in.w", (D, cfg.txt_dim)), ("txt_in.b", (D,))]
    for i in range(cfg.n_double):
        for s in ("txt", "img"):
            p = f"double.{i}.{s}."
            out += [(p + "mod.w", (6 * D, D)), (p + "mod.b", (6 * D,)),
                    (p + "qkv.w", (3 * D, D)), (p + "qkv.b", (3 * D,)),
                    (p + "q_gain", (Dh,)), (p + "k_gain", (Dh,)),
                    (p + "o.w", (D, D)), (p + "o.b", (D,)),
                    (p + "fc1.w", (F, D)), (p + "fc1.b", (F,)),
                    (p + "fc2.w", (D, F)), (p + "fc2.b", (D,))]
    for i in range(cfg.n_single):
        p = f"single.{i}."
        out += [(p + "mod.w", (3 * D, D)), (p + "mod.b", (3 * D,)),
                (p + "in.w", (3 * D + F, D)), (p + "in.b", (3 * D + F,)),
                (p + "q_gain", (Dh,)), (p + "k_gain", (Dh,)),
                (p + "out.w", (D, D + F)), (p + "out.b", (D,))]
    if not cfg.block_only:
        out += [("final.mod.w", (2 * D, D)), ("final.mod.b", (2 * D,)),
                ("final.w", (cfg.patch_dim, D)), ("final.b", (cfg.patch_dim,))]
    return out


def param_layout(cfg: Config):
    """[(name, shape, offset)] and the padded total length."""
    off = 0
    lay = []
    for name, shape in param_shapes(cfg):
        n = int(np.prod(shape))
        lay.append((name, shape, off))
        off += (n + ALIGN - 1) // ALIGN * ALIGN
    return lay, off


def unflatten(cfg: Config, theta: np.ndarray, dtype=np.float64):
    lay, _ = param_layout(cfg)
    return {name: theta[off:off + int(np.prod(shape))].astype(dtype).reshape(shape)
            for name, shape, off in lay}


def flatten(cfg: Config, grads: dict, dtype=np.float64):
    lay, total = param_layout(cfg)
    out = np.zeros(total, dtype=dtype)
    for name, shape, off in lay:
        g = grads.get(name)
        if g is not None:
            out[off:off + int(np.prod(shape))] = np.asarray(g).reshape(-1)
    return out


# ----------------------------------------------------------------------------
# elementary operators (forward); each one is pinned against a library routine
# ----------------------------------------------------------------------------
def silu(x):
    return x / (1.0 + np.exp(-x))


def silu_grad(x):
    s = 1.0 / (1.0 + np.exp(-x))
    return s * (1.0 + x * (1.0 - s))


def gelu_tanh(x):
    return 0.5 * x * (1.0 + np.tanh(GELU_C * (x + 0.044715 * x ** 3)))


def gelu_tanh_grad(x):
    th = np.tanh(GELU_C * (x + 0.044715 * x ** 3))
    return 0.5 * (1.0 + th) + 0.5 * x * (1.0 - th * th) * GELU_C * (1.0 + 3 * 0.044715 * x * x)


def layer_norm(x):
    """LayerNorm without affine over the last axis; returns (xhat, rstd)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + LN_EPS)
    return (x - mu) * rstd, rstd


def layer_norm_bwd(dxhat, xhat, rstd):
    m1 = dxhat.mean(axis=-1, keepdims=True)
    m2 = (dxhat * xhat).mean(axis=-1, keepdims=True)
    return rstd * (dxhat - m1 - xhat * m2)


def rms_norm(x, gain):
    """x * gain / sqrt(mean(x^2) + eps) over the last axis; returns (y, rinv)."""
    rinv = 1.0 / np.sqrt((x * x).mean(axis=-1, keepdims=True) + RMS_EPS)
    return x * rinv * gain, rinv


def rms_norm_bwd(dy, x, rinv, gain):
    n = x.shape[-1]
    gdy = dy * gain
    dx = gdy * rinv - x * rinv ** 3 * (gdy * x).sum(axis=-1, keepdims=True) / n
    dgain = (dy * x * rinv).reshape(-1, n).sum(axis=0)
    return dx, dgain


def timestep_embedding(t, dim):
    half = dim // 2
    k = np.arange(half, dtype=np.float64)
    w = ROPE_THETA ** (-k / half)
    arg = 1000.0 * np.asarray(t, dtype=np.float64)[:, None] * w[None, :]
    return np.concatenate([np.cos(arg), np.sin(arg)], axis=1)


def positions(cfg: Config):
    """(N, 2) positions of the joint sequence [text; image]."""
    pos = np.zeros((cfg.n_tok, 2), dtype=np.float64)
    r, c = np.meshgrid(np.arange(cfg.grid_h), np.arange(cfg.grid_w), indexing="ij")
    pos[cfg.n_txt:, 0] = r.reshape(-1)
    pos[cfg.n_txt:, 1] = c.reshape(-1)
    return pos


def rope_angles(cfg: Config):
    """(N, Dh/2) rotation angle of each interleaved pair."""
    dh = cfg.head_dim
    quarter = dh // 4
    i = np.arange(quarter, dtype=np.float64)
    freq = ROPE_THETA ** (-2.0 * i / (dh // 2))
    pos = positions(cfg)
    return np.concatenate([pos[:, :1] * freq[None, :], pos[:, 1:] * freq[None, :]], axis=1)


def rope(x, ang):
    """Rotate pairs (2i, 2i+1) of the last axis by ang[..., i] (ang broadcast over heads)."""
    c, s = np.cos(ang).astype(x.dtype), np.sin(ang).astype(x.dtype)
    x0, x1 = x[..., 0::2], x[..., 1::2]
    y = np.empty_like(x)
    y[..., 0::2] = x0 * c - x1 * s
    y[..., 1::2] = x0 * s + x1 * c
    return y


def rope_bwd(dy, ang):
    return rope(dy, -ang)


def softmax_probs(q, k):
    """P = softmax(q k^T / sqrt(Dh)) for one (batch, head): q (N, Dh), k (N, Dh)."""
    s = np.matmul(q, k.T) * (1.0 / np.sqrt(q.shape[-1]))
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    return p / p.sum(axis=-1, keepdims=True)


def attention(q, k, v):
    """Softmax attention; q, k, v: (B, H, N, Dh).  One (batch, head) at a time."""
    o = np.empty_like(v)
    for b in range(q.shape[0]):
        for h in range(q.shape[1]):
            o[b, h] = np.matmul(softmax_probs(q[b, h], k[b, h]), v[b, h])
    return o


def attention_bwd(do, q, k, v):
    """Backward-cost appendix: dV = P^T dO, dP = dO V^T, dS = softmax_bwd(P, dP),
    dQ = dS K / sqrt(Dh), dK = dS^T Q / sqrt(Dh).  P is recomputed per head."""
    scale = 1.0 / np.sqrt(q.shape[-1])
    dq, dk, dv = np.empty_like(q), np.empty_like(k), np.empty_like(v)
    for b in range(q.shape[0]):
        for h in range(q.shape[1]):
            p = softmax_probs(q[b, h], k[b, h])
            dv[b, h] = np.matmul(p.T, do[b, h])
            dp = np.matmul(do[b, h], v[b, h].T)
            ds = p * (dp - (dp * p).sum(axis=-1, keepdims=True))
            dq[b, h] = np.matmul(ds, k[b, h]) * scale
            dk[b, h] = np.matmul(ds.T, q[b, h]) * scale
    return dq, dk, dv


def linear(x, w, b):
    return np.matmul(x, w.T) + b


def wgrad(dy, x):
    """Weight gradient sum over batch and tokens of dy^T x: (..., out), (..., in) -> (out, in)."""
    return np.matmul(dy.reshape(-1, dy.shape[-1]).T, x.reshape(-1, x.shape[-1]))


def patchify(cfg: Config, z):
    """(B, C, H, W) -> (B, n_img, C*p*p) with feature index (c, py, px)."""
    B, C = z.shape[:2]
    p, gh, gw = cfg.patch, cfg.grid_h, cfg.grid_w
    x = z.reshape(B, C, gh, p, gw, p).transpose(0, 2, 4, 1, 3, 5)
    return x.reshape(B, gh * gw, C * p * p)


def unpatchify(cfg: Config, x):
    B = x.shape[0]
    p, gh, gw, C = cfg.patch, cfg.grid_h, cfg.grid_w, cfg.in_ch
    z = x.reshape(B, gh, gw, C, p, p).transpose(0, 3, 1, 4, 2, 5)
    return z.reshape(B, C, gh * p, gw * p)


# ----------------------------------------------------------------------------
# blocks
# ----------------------------------------------------------------------------
def _heads(x, H):
    B, N, D = x.shape
    return x.reshape(B, N, H, D // H).transpose(0, 2, 1, 3)


def _unheads(x):
    B, H, N, dh = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B, N, H * dh)


def _qk(cfg, P, pre, qkv, ang):
    """Per-stream q, k, v from a (B, n, 3D) projection: RMS-norm q, k; no rotation yet."""
    D, H = cfg.hidden, cfg.heads
    q, k, v = _heads(qkv[..., :D], H), _heads(qkv[..., D:2 * D], H), _heads(qkv[..., 2 * D:3 * D], H)
    qn, qr = rms_norm(q, P[pre + "q_gain"])
    kn, kr = rms_norm(k, P[pre + "k_gain"])
    return (q, qn, qr), (k, kn, kr), v


def double_block_fwd(cfg, P, i, x_txt, x_img, mvec, ang):
    D, H = cfg.hidden, cfg.heads
    nt = x_txt.shape[1]
    c = {"x_txt": x_txt, "x_img": x_img}
    streams = {"txt": x_txt, "img": x_img}
    qs, ks, vs = [], [], []
    for s in ("txt", "img"):
        pre = f"double.{i}.{s}."
        mod = linear(mvec, P[pre + "mod.w"], P[pre + "mod.b"])  # (B, 6D)
        ch = [mod[:, None, j * D:(j + 1) * D] for j in range(6)]
        xhat, rstd = layer_norm(streams[s])
        a = xhat * (1.0 + ch[1]) + ch[0]
        qkv = linear(a, P[pre + "qkv.w"], P[pre + "qkv.b"])
        (q, qn, qr), (k, kn, kr), v = _qk(cfg, P, pre, qkv, ang)
        c[s] = dict(mod=mod, ch=ch, xhat1=xhat, rstd1=rstd, a1=a, q=q, qn=qn, qr=qr, k=k, kn=kn, kr=kr)
        qs.append(qn), ks.append(kn), vs.append(v)
    qj = rope(np.concatenate(qs, axis=2), ang)
    kj = rope(np.concatenate(ks, axis=2), ang)
    vj = np.concatenate(vs, axis=2)
    o = attention(qj, kj, vj)
    c.update(qj=qj, kj=kj, vj=vj)
    o = _unheads(o)
    outs = {}
    for s, o_s in (("txt", o[:, :nt]), ("img", o[:, nt:])):
        pre = f"double.{i}.{s}."
        d = c[s]
        ch = d["ch"]
        y1 = linear(o_s, P[pre + "o.w"], P[pre + "o.b"])
        xm = streams[s] + ch[2] * y1
        xhat2, rstd2 = layer_norm(xm)
        a2 = xhat2 * (1.0 + ch[4]) + ch[3]
        pre_act = linear(a2, P[pre + "fc1.w"], P[pre + "fc1.b"])
        h = gelu_tanh(pre_act)
        y2 = linear(h, P[pre + "fc2.w"], P[pre + "fc2.b"])
        outs[s] = xm + ch[5] * y2
        d.update(o=o_s, y1=y1, xhat2=xhat2, rstd2=rstd2, a2=a2, pre_act=pre_act, h=h, y2=y2)
    return outs["txt"], outs["img"], c


def double_block_bwd(cfg, P, i, c, g_txt, g_img, mvec, ang, G):
    """Returns (dx_txt, dx_img, dmvec); parameter gradients accumulate into G."""
    D, H = cfg.hidden, cfg.heads
    gs = {"txt": g_txt, "img": g_img}
    dmods, dxm, do_parts = {}, {}, []
    for s in ("txt", "img"):
        pre = f"double.{i}.{s}."
        d = c[s]
        ch = d["ch"]
        g = gs[s]
        dmod = [None] * 6
        # MLP branch: x_out = xm + gate2 * y2
        dmod[5] = (g * d["y2"]).sum(axis=1)
        dy2 = g * ch[5]
        G[pre + "fc2.w"] += wgrad(dy2, d["h"])
        G[pre + "fc2.b"] += dy2.sum(axis=(0, 1))
        dh = np.matmul(dy2, P[pre + "fc2.w"])
        dpre = dh * gelu_tanh_grad(d["pre_act"])
        G[pre + "fc1.w"] += wgrad(dpre, d["a2"])
        G[pre + "fc1.b"] += dpre.sum(axis=(0, 1))
        da2 = np.matmul(dpre, P[pre + "fc1.w"])
        dmod[4] = (da2 * d["xhat2"]).sum(axis=1)
        dmod[3] = da2.sum(axis=1)
        dxm_s = g + layer_norm_bwd(da2 * (1.0 + ch[4]), d["xhat2"], d["rstd2"])
        # attention branch: xm = x + gate1 * y1
        dmod[2] = (dxm_s * d["y1"]).sum(axis=1)
        dy1 = dxm_s * ch[2]
        G[pre + "o.w"] += wgrad(dy1, d["o"])
        G[pre + "o.b"] += dy1.sum(axis=(0, 1))
        do_parts.append(np.matmul(dy1, P[pre + "o.w"]))
        dmods[s], dxm[s] = dmod, dxm_s
    do = _heads(np.concatenate(do_parts, axis=1), H)
    dqj, dkj, dvj = attention_bwd(do, c["qj"], c["kj"], c["vj"])
    dqn = rope_bwd(dqj, ang)
    dkn = rope_bwd(dkj, ang)
    nt = g_txt.shape[1]
    dmvec = 0.0
    dx = {}
    for s, sl in (("txt", slice(0, nt)), ("img", slice(nt, None))):
        pre = f"double.{i}.{s}."
        d = c[s]
        ch = d["ch"]
        dq, dgq = rms_norm_bwd(dqn[:, :, sl], d["q"], d["qr"], P[pre + "q_gain"])
        dk, dgk = rms_norm_bwd(dkn[:, :, sl], d["k"], d["kr"], P[pre + "k_gain"])
        G[pre + "q_gain"] += dgq
        G[pre + "k_gain"] += dgk
        dqkv = np.concatenate([_unheads(dq), _unheads(dk), _unheads(dvj[:, :, sl])], axis=-1)
        G[pre + "qkv.w"] += wgrad(dqkv, d["a1"])
        G[pre + "qkv.b"] += dqkv.sum(axis=(0, 1))
        da1 = np.matmul(dqkv, P[pre + "qkv.w"])
        dmod = dmods[s]
        dmod[1] = (da1 * d["xhat1"]).sum(axis=1)
        dmod[0] = da1.sum(axis=1)
        dx[s] = dxm[s] + layer_norm_bwd(da1 * (1.0 + ch[1]), d["xhat1"], d["rstd1"])
        dmod_full = np.concatenate(dmod, axis=-1)  # (B, 6D)
        G[pre + "mod.w"] += np.matmul(dmod_full.T, mvec)
        G[pre + "mod.b"] += dmod_full.sum(axis=0)
        dmvec = dmvec + np.matmul(dmod_full, P[pre + "mod.w"])
    return dx["txt"], dx["img"], dmvec


def single_block_fwd(cfg, P, i, x, mvec, ang):
    D, H, F = cfg.hidden, cfg.heads, cfg.mlp_hidden
    pre = f"single.{i}."
    mod = linear(mvec, P[pre + "mod.w"], P[pre + "mod.b"])
    ch = [mod[:, None, j * D:(j + 1) * D] for j in range(3)]
    xhat, rstd = layer_norm(x)
    a = xhat * (1.0 + ch[1]) + ch[0]
    proj = linear(a, P[pre + "in.w"], P[pre + "in.b"])
    (q, qn, qr), (k, kn, kr), v = _qk(cfg, P, pre, proj[..., :3 * D], ang)
    qj, kj = rope(qn, ang), rope(kn, ang)
    o = _unheads(attention(qj, kj, v))
    u = proj[..., 3 * D:]
    cat = np.concatenate([o, gelu_tanh(u)], axis=-1)
    y = linear(cat, P[pre + "out.w"], P[pre + "out.b"])
    c = dict(x=x, ch=ch, xhat=xhat, rstd=rstd, a=a, q=q, qr=qr, k=k, kr=kr, qj=qj, kj=kj, vj=v,
             u=u, cat=cat, y=y)
    return x + ch[2] * y, c


def single_block_bwd(cfg, P, i, c, g, mvec, ang, G):
    D, H = cfg.hidden, cfg.heads
    pre = f"single.{i}."
    ch = c["ch"]
    dmod = [None] * 3
    dmod[2] = (g * c["y"]).sum(axis=1)
    dy = g * ch[2]
    G[pre + "out.w"] += wgrad(dy, c["cat"])
    G[pre + "out.b"] += dy.sum(axis=(0, 1))
    dcat = np.matmul(dy, P[pre + "out.w"])
    do, dgu = dcat[..., :D], dcat[..., D:]
    du = dgu * gelu_tanh_grad(c["u"])
    dqj, dkj, dv = attention_bwd(_heads(do, H), c["qj"], c["kj"], c["vj"])
    dq, dgq = rms_norm_bwd(rope_bwd(dqj, ang), c["q"], c["qr"], P[pre + "q_gain"])
    dk, dgk = rms_norm_bwd(rope_bwd(dkj, ang), c["k"], c["kr"], P[pre + "k_gain"])
    G[pre + "q_gain"] += dgq
    G[pre + "k_gain"] += dgk
    dproj = np.concatenate([_unheads(dq), _unheads(dk), _unheads(dv), du], axis=-1)
    G[pre + "in.w"] += wgrad(dproj, c["a"])
    G[pre + "in.b"] += dproj.sum(axis=(0, 1))
    da = np.matmul(dproj, P[pre + "in.w"])
    dmod[1] = (da * c["xhat"]).sum(axis=1)
    dmod[0] = da.sum(axis=1)
    dx = g + layer_norm_bwd(da * (1.0 + ch[1]), c["xhat"], c["rstd"])
    dmod_full = np.concatenate(dmod, axis=-1)
    G[pre + "mod.w"] += np.matmul(dmod_full.T, mvec)
    G[pre + "mod.b"] += dmod_full.sum(axis=0)
    return dx, np.matmul(dmod_full, P[pre + "mod.w"])


# ----------------------------------------------------------------------------
# whole model
# ----------------------------------------------------------------------------
@dataclass
class Inputs:
    """Model inputs for one batch.

    Full model: z (B, C, H, W) latent and txt (B, n_txt, txt_dim).
    Block only: x_txt (B, n_txt, D) and x_img (B, n_img, D) token streams.
    t: (B,) network-input timesteps."""
    t: np.ndarray
    z: np.ndarray | None = None
    txt: np.ndarray | None = None
    x_txt: np.ndarray | None = None
    x_img: np.ndarray | None = None


def forward(cfg: Config, P: dict, inp: Inputs):
    """Returns (v_hat, cache).  Block only: v_hat = (x_txt_out, x_img_out)."""
    cache = {}
    dt = P["t_in.w"].dtype
    e = timestep_embedding(inp.t, cfg.t_freq_dim).astype(dt)
    h1 = linear(e, P["t_in.w"], P["t_in.b"])
    vec = linear(silu(h1), P["t_out.w"], P["t_out.b"])
    mvec = silu(vec)
    cache.update(e=e, h1=h1, vec=vec, mvec=mvec)
    ang = rope_angles(cfg)
    if cfg.block_only:
        x_txt, x_img = inp.x_txt, inp.x_img
    else:
        patches = patchify(cfg, inp.z)
        x_img = linear(patches, P["img_in.w"], P["img_in.b"])
        x_txt = linear(inp.txt, P["txt_in.w"], P["txt_in.b"])
        cache.update(patches=patches, txt=inp.txt)
    dbl = []
    for i in range(cfg.n_double):
        x_txt, x_img, c = double_block_fwd(cfg, P, i, x_txt, x_img, mvec, ang)
        dbl.append(c)
    cache["double"] = dbl
    if cfg.block_only:
        return (x_txt, x_img), cache
    x = np.concatenate([x_txt, x_img], axis=1)
    sgl = []
    for i in range(cfg.n_single):
        x, c = single_block_fwd(cfg, P, i, x, mvec, ang)
        sgl.append(c)
    cache["single"] = sgl
    D = cfg.hidden
    fmod = linear(mvec, P["final.mod.w"], P["final.mod.b"])
    shift, scale = fmod[:, None, :D], fmod[:, None, D:]
    xi = x[:, cfg.n_txt:]
    xhat, rstd = layer_norm(xi)
    a = xhat * (1.0 + scale) + shift
    out = linear(a, P["final.w"], P["final.b"])
    cache.update(fmod=fmod, fxhat=xhat, frstd=rstd, fa=a, x_last=x)
    return unpatchify(cfg, out), cache


def vjp(cfg: Config, P: dict, cache: dict, s):
    """Parameter gradient J(z, t)^T s for the cached forward.  Returns {name: grad}.

    s has the shape of v_hat (block only: a (s_txt, s_img) pair)."""
    G = {name: np.zeros(shape, dtype=P[name].dtype) for name, shape in param_shapes(cfg)}
    ang = rope_angles(cfg)
    mvec = cache["mvec"]
    D = cfg.hidden
    dmvec = np.zeros_like(mvec)
    if cfg.block_only:
        g_txt, g_img = s
    else:
        dout = patchify(cfg, s)
        G["final.w"] += wgrad(dout, cache["fa"])
        G["final.b"] += dout.sum(axis=(0, 1))
        da = np.matmul(dout, P["final.w"])
        dshift = da.sum(axis=1)
        dscale = (da * cache["fxhat"]).sum(axis=1)
        dfmod = np.concatenate([dshift, dscale], axis=-1)
        G["final.mod.w"] += np.matmul(dfmod.T, mvec)
        G["final.mod.b"] += dfmod.sum(axis=0)
        dmvec += np.matmul(dfmod, P["final.mod.w"])
        scale = cache["fmod"][:, None, D:]
        gx = np.zeros_like(cache["x_last"])
        gx[:, cfg.n_txt:] = layer_norm_bwd(da * (1.0 + scale), cache["fxhat"], cache["frstd"])
        for i in reversed(range(cfg.n_single)):
            gx, dm = single_block_bwd(cfg, P, i, cache["single"][i], gx, mvec, ang, G)
            dmvec += dm
        g_txt, g_img = gx[:, :cfg.n_txt], gx[:, cfg.n_txt:]
    for i in reversed(range(cfg.n_double)):
        g_txt, g_img, dm = double_block_bwd(cfg, P, i, cache["double"][i], g_txt, g_img, mvec, ang, G)
        dmvec += dm
    if not cfg.block_only:
        G["img_in.w"] += wgrad(g_img, cache["patches"])
        G["img_in.b"] += g_img.sum(axis=(0, 1))
        G["txt_in.w"] += wgrad(g_txt, cache["txt"])
        G["txt_in.b"] += g_txt.sum(axis=(0, 1))
    dvec = dmvec * silu_grad(cache["vec"])
    G["t_out.w"] += np.matmul(dvec.T, silu(cache["h1"]))
    G["t_out.b"] += dvec.sum(axis=0)
    dh1 = np.matmul(dvec, P["t_out.w"]) * silu_grad(cache["h1"])
    G["t_in.w"] += np.matmul(dh1.T, cache["e"])
    G["t_in.b"] += dh1.sum(axis=0)
    return G


def vjp_flat(cfg: Config, theta: np.ndarray, inp: Inputs, s, dtype=np.float64):
    """Convenience: forward + VJP from a flat parameter vector; returns flat dθ."""
    P = unflatten(cfg, theta, dtype)
    _, cache = forward(cfg, P, inp)
    return flatten(cfg, vjp(cfg, P, cache, s), dtype)
