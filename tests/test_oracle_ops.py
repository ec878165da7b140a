"""Pins for the oracle's elementary operators: each reduces to a library routine
(torch CPU, fp64) or a textbook identity.  CPU only."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import mmdit

torch.set_default_dtype(torch.float64)


def _rs(seed):
    return np.random.default_rng(seed)


def test_layer_norm_matches_torch_and_backward():
    x = _rs(0).standard_normal((3, 5, 24)) * 3 + 1
    xhat, rstd = mmdit.layer_norm(x)
    tx = torch.tensor(x, requires_grad=True)
    ty = F.layer_norm(tx, (24,), eps=mmdit.LN_EPS)
    np.testing.assert_allclose(xhat, ty.detach().numpy(), rtol=1e-12, atol=1e-12)
    g = _rs(1).standard_normal(x.shape)
    ty.backward(torch.tensor(g))
    np.testing.assert_allclose(mmdit.layer_norm_bwd(g, xhat, rstd), tx.grad.numpy(), rtol=1e-10, atol=1e-12)
    # invariants of the no-affine LayerNorm backward: sum dx = 0 exactly, and
    # <dx, xhat> = 0 up to the eps term (mean(xhat^2) = var / (var + eps))
    dx = mmdit.layer_norm_bwd(g, xhat, rstd)
    assert np.abs(dx.sum(-1)).max() < 1e-10
    assert np.abs((dx * xhat).sum(-1)).max() < 1e-5


def test_rms_norm_matches_torch_and_backward():
    x = _rs(2).standard_normal((2, 3, 7, 16))
    gain = 1 + 0.3 * _rs(3).standard_normal(16)
    y, rinv = mmdit.rms_norm(x, gain)
    tx = torch.tensor(x, requires_grad=True)
    tg = torch.tensor(gain, requires_grad=True)
    ty = F.rms_norm(tx, (16,), weight=tg, eps=mmdit.RMS_EPS)
    np.testing.assert_allclose(y, ty.detach().numpy(), rtol=1e-12, atol=1e-12)
    g = _rs(4).standard_normal(x.shape)
    ty.backward(torch.tensor(g))
    dx, dgain = mmdit.rms_norm_bwd(g, x, rinv, gain)
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dgain, tg.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_gelu_silu_match_torch_and_derivatives():
    x = np.linspace(-6, 6, 1001)
    tx = torch.tensor(x, requires_grad=True)
    y = F.gelu(tx, approximate="tanh")
    np.testing.assert_allclose(mmdit.gelu_tanh(x), y.detach().numpy(), rtol=1e-13, atol=1e-14)
    y.sum().backward()
    np.testing.assert_allclose(mmdit.gelu_tanh_grad(x), tx.grad.numpy(), rtol=1e-12, atol=1e-13)
    tx = torch.tensor(x, requires_grad=True)
    y = F.silu(tx)
    np.testing.assert_allclose(mmdit.silu(x), y.detach().numpy(), rtol=1e-13, atol=1e-14)
    y.sum().backward()
    np.testing.assert_allclose(mmdit.silu_grad(x), tx.grad.numpy(), rtol=1e-12, atol=1e-13)


def test_attention_matches_sdpa_and_backward():
    rs = _rs(5)
    q, k, v = (rs.standard_normal((2, 3, 11, 8)) for _ in range(3))
    o = mmdit.attention(q, k, v)
    tq, tk, tv = (torch.tensor(a, requires_grad=True) for a in (q, k, v))
    to = F.scaled_dot_product_attention(tq, tk, tv)
    np.testing.assert_allclose(o, to.detach().numpy(), rtol=1e-11, atol=1e-12)
    do = rs.standard_normal(o.shape)
    to.backward(torch.tensor(do))
    dq, dk, dv = mmdit.attention_bwd(do, q, k, v)
    for a, b in ((dq, tq), (dk, tk), (dv, tv)):
        np.testing.assert_allclose(a, b.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_rope_is_complex_rotation_and_relative():
    cfg = mmdit.Config(n_double=1, n_single=0, hidden=32, heads=2, head_dim=16, mlp_hidden=64,
                       in_ch=2, patch=1, lat_h=3, lat_w=5, n_txt=2, txt_dim=8)
    ang = mmdit.rope_angles(cfg)  # (N, 8)
    assert ang.shape == (cfg.n_tok, 8)
    # text tokens are at (0, 0): no rotation
    assert np.all(ang[:cfg.n_txt] == 0.0)
    # first quarter of pairs follow the row index, second quarter the column index
    tok = cfg.n_txt + 2 * cfg.grid_w + 3  # image token at row 2, col 3
    assert ang[tok, 0] == 2.0 and ang[tok, 4] == 3.0
    assert np.isclose(ang[tok, 1], 2.0 * 10000.0 ** (-2.0 / 8))
    x = _rs(6).standard_normal((cfg.n_tok, 16))
    y = mmdit.rope(x, ang)
    zc = (x[:, 0::2] + 1j * x[:, 1::2]) * np.exp(1j * ang)
    np.testing.assert_allclose(y[:, 0::2], zc.real, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(y[:, 1::2], zc.imag, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    np.testing.assert_allclose(mmdit.rope_bwd(y, ang), x, rtol=1e-12, atol=1e-13)
    # scores depend only on relative position: shifting both rows by one keeps <q,k>
    a = cfg.n_txt + 0 * cfg.grid_w + 1
    b = cfg.n_txt + 1 * cfg.grid_w + 4
    a2, b2 = a + cfg.grid_w, b + cfg.grid_w
    q, k = x[0], x[1]
    s1 = mmdit.rope(q, ang[a]) @ mmdit.rope(k, ang[b])
    s2 = mmdit.rope(q, ang[a2]) @ mmdit.rope(k, ang[b2])
    assert abs(s1 - s2) < 1e-12


def test_timestep_embedding_special_values():
    e = mmdit.timestep_embedding(np.array([0.0, 0.25]), 16)
    assert np.all(e[0, :8] == 1.0) and np.all(e[0, 8:] == 0.0)
    # frequency 0 is 1: first cosine is cos(1000 t); last frequency is 10000^(-7/8)
    assert np.isclose(e[1, 0], np.cos(250.0)) and np.isclose(e[1, 8], np.sin(250.0))
    assert np.isclose(e[1, 7], np.cos(250.0 * 10000.0 ** (-7 / 8)))


def test_patchify_index_convention():
    cfg = mmdit.Config(n_double=0, n_single=0, hidden=8, heads=1, head_dim=8, mlp_hidden=8,
                       in_ch=3, patch=2, lat_h=4, lat_w=6)
    z = _rs(7).standard_normal((2, 3, 4, 6))
    x = mmdit.patchify(cfg, z)
    assert x.shape == (2, 6, 12)
    for b in range(2):
        for r in range(2):
            for c in range(3):
                for ch in range(3):
                    for py in range(2):
                        for px in range(2):
                            assert x[b, r * 3 + c, ch * 4 + py * 2 + px] == z[b, ch, r * 2 + py, c * 2 + px]
    np.testing.assert_array_equal(mmdit.unpatchify(cfg, x), z)
