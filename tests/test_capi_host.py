"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function declared in include/jagg.h, its parameter layout equals the
oracle's, and the host-only routing and interpolation-weight calls agree with
the oracle bit for bit."""
import json
import os
import re

import numpy as np
import pytest

import paper_2607_17572_amd as pk
from oracle import jagg, mmdit

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib_or_skip():
    if not os.path.exists(pk.api.LIB_PATH):
        pytest.skip("libjagg.so not built")
    return pk.lib()


def test_library_exports_every_declared_function():
    L = _lib_or_skip()
    hdr = open(os.path.join(ROOT, "include", "jagg.h")).read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    names = set(re.findall(r"\b(\w+)\s*\([^;{]*\)\s*;", hdr))
    names -= {"if", "while", "for", "return"}
    assert {"dit_forward_save", "dit_vjp", "jagg_aggregate", "jagg_route", "jagg_group_backward"} <= names
    for n in sorted(names):
        assert hasattr(L, n), n


def _oracle_cfg(c: pk.Config) -> mmdit.Config:
    return mmdit.Config(n_double=c.n_double, n_single=c.n_single, hidden=c.hidden, heads=c.heads,
                        head_dim=c.head_dim, mlp_hidden=c.mlp_hidden, in_ch=c.in_ch, patch=c.patch, lat_h=c.lat_h,
                        lat_w=c.lat_w, n_txt=c.n_txt, txt_dim=c.txt_dim, t_freq_dim=c.t_freq_dim,
                        block_only=bool(c.block_only))


@pytest.mark.parametrize("name", ["tiny", "block", "slice", "flux", "qwen"])
def test_param_layout_matches_oracle(name):
    _lib_or_skip()
    c = pk.config(name)
    lay, total = pk.param_layout(c)
    olay, ototal = mmdit.param_layout(_oracle_cfg(c))
    assert total == ototal
    assert len(lay) == len(olay)
    for (n, off, numel, r, cc), (on, oshape, ooff) in zip(lay, olay):
        assert n == on and off == ooff and numel == int(np.prod(oshape))
        assert (r, cc) == (oshape if len(oshape) == 2 else (oshape[0], 1))


def test_flux_like_parameter_count():
    _lib_or_skip()
    lay, _ = pk.param_layout(pk.config("flux"))
    n = sum(x[2] for x in lay)
    assert 11.5e9 < n < 12.2e9  # "~12B" full-depth Flux-like MMDiT


def test_alpha_host_matches_oracle():
    _lib_or_skip()
    for t in ([1.0, 0.875, 0.75, 0.625], [0.5, 0.375, 0.25, 0.125], [0.9, 0.4],
              list(np.float32(3 * np.array([1, .9, .8, .7, .6]) / (1 + 2 * np.array([1, .9, .8, .7, .6]))))):
        a = pk.alpha(t)
        want = jagg.alpha(np.asarray(t, dtype=np.float32).astype(np.float64)).astype(np.float32)
        assert list(np.asarray(a, dtype=np.float32)) == list(want)
        assert a[0] == 0.0 and a[-1] == 1.0
    with pytest.raises(pk.JaggError):
        pk.alpha([0.5])
    with pytest.raises(pk.JaggError):
        pk.alpha([0.5, 0.2, 0.5])
    with pytest.raises(pk.JaggError):
        pk.alpha([0.3, 0.5])            # increasing: not a denoising window
    with pytest.raises(pk.JaggError):
        pk.alpha([0.9, 0.95, 0.3])      # not monotone


def test_route_host_bit_exact_against_oracle():
    _lib_or_skip()
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "jagg_quality.json")))
    for m in g["models"].values():
        mask, frac = pk.route(5, scores=m["cos"], tau=g["tau"])
        omask, ofrac = jagg.route(5, scores=m["cos"], tau=g["tau"])
        assert mask == list(omask) and frac == ofrac
    rs = np.random.default_rng(0)
    for _ in range(200):
        n = int(rs.integers(1, 12))
        sc = list(np.round(rs.uniform(0.3, 0.7, n), 3))
        tau = float(rs.choice([0.4, 0.5, 0.6]))
        mask, frac = pk.route(n, scores=sc, tau=tau)
        omask, ofrac = jagg.route(n, scores=sc, tau=tau)
        assert mask == list(omask) and frac == ofrac
        fr = float(rs.choice([0.0, 0.2, 0.4, 0.5, 0.6, 0.75, 1.0]))
        mask, frac = pk.route(n, frac=fr)
        omask, ofrac = jagg.route(n, frac=fr)
        assert mask == list(omask) and frac == ofrac


def test_invalid_arguments_are_rejected_before_any_launch():
    L = _lib_or_skip()
    bad = pk.Config(n_double=1, n_single=0, hidden=64, heads=3, head_dim=16, mlp_hidden=64)  # 3*16 != 64
    with pytest.raises(pk.JaggError) as e:
        pk.param_layout(bad)
    assert e.value.status == 1
    with pytest.raises(pk.JaggError):
        pk.route(0, frac=0.5)
    with pytest.raises(pk.JaggError):
        pk.route(3, frac=1.5)
    import ctypes
    assert L.dit_vjp(None, None, None, 1, None, None, 0.0) == 1
    assert L.jagg_group_backward(None, None, None, 1, None, None, 4, None, 0.0) == 1
    # linear-layer products: every argument error is caught on the host
    c = pk.config("tiny").c()
    h = ctypes.c_void_p()
    assert L.jagg_ctx_create(ctypes.byref(c), None, ctypes.byref(h)) == 0
    try:
        p16, p8 = 4096, 4104  # never dereferenced: every call below fails validation first
        assert L.jagg_linear_grad(h, 3, p16, p16, None, 8, 8, 8, p16, 0, 0.0) == 1       # unknown kind
        assert L.jagg_linear_grad(h, 0, p16, None, None, 8, 8, 8, p16, 0, 0.0) == 1      # null operand
        assert L.jagg_linear_grad(h, 0, p8, p16, None, 8, 8, 8, p16, 0, 0.0) == 1        # unaligned
        assert L.jagg_linear_grad(h, 0, p16, p16, None, 0, 8, 8, p16, 0, 0.0) == 1       # empty
        assert L.jagg_linear_grad(h, 0, p16, p16, None, 8, 8, 8, p16, 0, 1.0) == 1       # beta on dgrad
        assert L.jagg_linear_grad(h, 1, p16, p16, None, 8, 8, 8, p16, 1, 0.0) == 1       # GELU without pre
        assert L.jagg_linear_grad(h, 1, p16, p16, p16, 8, 8, 8, p16, 0, 0.0) == 1        # GELU to fp32
        assert L.jagg_linear_grad(h, 2, p16, p16, None, 8, 8, 8, p16, 0, 0.5) == 1       # beta not 0/1
        assert L.jagg_linear_grad(h, 2, p16, p16, None, 8, 8, 8, p16, 7, 0.0) == 1       # unknown dtype
    finally:
        L.jagg_ctx_destroy(h)


def test_variant_entry_points_reject_bad_arguments():
    """Sequential-graph endpoint backward and gradient comparison: argument
    errors are reported on the host before any launch."""
    L = _lib_or_skip()
    import ctypes
    c = pk.config("tiny").c()
    h = ctypes.c_void_p()
    assert L.jagg_ctx_create(ctypes.byref(c), None, ctypes.byref(h)) == 0
    try:
        p = 4096
        s2 = (ctypes.c_void_p * 2)(p, p)
        t2 = (ctypes.c_float * 2)(1.0, 0.5)
        # endpoint must be 0 or 1; beta 0 or 1; W >= 2 and t_0 != t_{W-1} (workspace checked after these)
        assert L.jagg_endpoint_backward(h, p, p, 1, s2, t2, 2, 2, p, 0.0) == 1
        assert L.jagg_endpoint_backward(h, p, p, 1, s2, t2, 2, 0, p, 0.5) == 1
        assert L.jagg_endpoint_backward(h, p, p, 0, s2, t2, 2, 0, p, 0.0) == 1
        assert L.jagg_endpoint_backward(h, p, None, 1, s2, t2, 2, 0, p, 0.0) == 1
        out = (ctypes.c_double * 5)()
        assert L.jagg_grad_compare(h, p, p, 0, 0, out) == 1          # empty
        assert L.jagg_grad_compare(h, p, p + 4, 8, 0, out) == 1      # unaligned
        assert L.jagg_grad_compare(h, p, p, 8, 5, out) == 1          # dtype
        assert L.jagg_grad_compare(h, p, p, 8, 0, out) == 1          # no workspace bound
        cnt = ctypes.c_ulonglong(7)
        assert L.jagg_count_nonfinite(h, None, 8, 0, ctypes.byref(cnt)) == 1   # null vector
        assert L.jagg_count_nonfinite(h, p, 8, 0, None) == 1                   # null count
        assert L.jagg_count_nonfinite(h, p, 0, 0, ctypes.byref(cnt)) == 1      # empty
        assert L.jagg_count_nonfinite(h, p + 4, 8, 0, ctypes.byref(cnt)) == 1  # unaligned
        assert L.jagg_count_nonfinite(h, p, 8, 5, ctypes.byref(cnt)) == 1      # dtype
        assert L.jagg_count_nonfinite(h, p, 8, 0, ctypes.byref(cnt)) == 1      # no workspace bound
        assert cnt.value == 7                                                 # untouched on error
    finally:
        L.jagg_ctx_destroy(h)


def test_grpo_entry_points_reject_bad_arguments():
    """GRPO Phase-2 calls: window and argument errors are caught on the host."""
    L = _lib_or_skip()
    import ctypes
    from paper_2607_17572_amd.api import _GrpoWindow
    c = pk.config("tiny").c()
    h = ctypes.c_void_p()
    assert L.jagg_ctx_create(ctypes.byref(c), None, ctypes.byref(h)) == 0
    try:
        p = 4096
        W = 4
        v = (ctypes.c_void_p * W)(*[p] * W)
        z = (ctypes.c_void_p * (W + 1))(*[p] * (W + 1))
        t = (ctypes.c_float * (W + 1))(1.0, 0.9, 0.8, 0.7, 0.6)
        sg = (ctypes.c_float * W)(0.3, 0.3, 0.3, 0.3)

        def win(**kw):
            d = dict(v_hat=v, z=z, t=t, sigma=sg, logp_old=p, adv=p, clip_eps=0.1, adv_clip=5.0, W=W,
                     v_batch=None, v_index=None)
            d.update(kw)
            return _GrpoWindow(**d)

        out = (ctypes.c_void_p * W)(*[p] * W)
        ok = win()
        assert L.jagg_grpo_composites(h, ctypes.byref(ok), 0, p, p, None) == 1          # batch 0
        assert L.jagg_grpo_composites(h, ctypes.byref(ok), 17, p, p, None) == 1         # batch > 16
        assert L.jagg_grpo_composites(h, ctypes.byref(win(W=1)), 1, p, p, None) == 1   # W < 2
        assert L.jagg_grpo_composites(h, ctypes.byref(win(W=17)), 1, p, p, None) == 1  # W > 16
        bad_sg = (ctypes.c_float * W)(0.3, 0.0, 0.3, 0.3)
        assert L.jagg_grpo_composites(h, ctypes.byref(win(sigma=bad_sg)), 1, p, p, None) == 1  # sigma <= 0
        flat = (ctypes.c_float * (W + 1))(0.5, 0.4, 0.3, 0.5, 0.2)
        assert L.jagg_grpo_composites(h, ctypes.byref(win(t=flat)), 1, p, p, None) == 1  # t_0 == t_{W-1}
        assert L.jagg_grpo_composites(h, ctypes.byref(win(logp_old=None)), 1, p, p, None) == 1
        assert L.jagg_grpo_composites(h, ctypes.byref(win(adv_clip=0.0)), 1, p, p, None) == 1
        vb = (ctypes.c_int * W)(2, 2, 2, 2)
        vk = (ctypes.c_int * W)(0, 1, 2, 0)  # index 2 of a batch-2 output: out of range
        assert L.jagg_grpo_composites(h, ctypes.byref(win(v_batch=vb, v_index=vk)), 1, p, p, None) == 1
        unal = (ctypes.c_void_p * W)(p, p + 4, p, p)
        assert L.jagg_grpo_upstream(h, ctypes.byref(ok), 1, unal, None) == 1           # unaligned s_j
        assert L.jagg_grpo_group_backward(h, p, p, 1, ctypes.byref(ok), p, 0.5, None) == 1  # beta
        assert L.jagg_grpo_composites(h, ctypes.byref(ok), 1, p, p, None) == 1          # no workspace
    finally:
        L.jagg_ctx_destroy(h)


def test_workspace_head_too_small_is_rejected_before_any_launch():
    """The scoring, comparison and GRPO calls use the batch-independent head of
    the workspace (partial sums, score slot, GRPO coefficients); a bound
    workspace shorter than that head is an argument error, whatever its size
    relative to the scoring partials alone."""
    L = _lib_or_skip()
    import ctypes
    c = pk.config("tiny").c()
    h = ctypes.c_void_p()
    assert L.jagg_ctx_create(ctypes.byref(c), None, ctypes.byref(h)) == 0
    try:
        p = 1 << 20  # a fake, aligned device address: never dereferenced
        score = ctypes.c_double()
        hs = (ctypes.c_void_p * 4)(*[p] * 4)
        out = (ctypes.c_double * 5)()
        for nbytes in (147712, 200000, 262144):
            assert L.jagg_ctx_set_workspace(h, ctypes.c_void_p(p), nbytes) == 0
            assert L.jagg_group_scores(h, hs, 1024, 4, 0, ctypes.byref(score)) == 1
            assert b"head" in L.jagg_last_error()
            assert L.jagg_grad_compare(h, p, p, 1024, 0, out) == 1
    finally:
        L.jagg_ctx_destroy(h)


def test_trajectory_and_quality_reject_bad_arguments():
    """Trajectory backward and window quality: every argument error is found
    on the host before the first launch (no workspace is bound, so a call that
    passed validation would fail on that instead)."""
    L = _lib_or_skip()
    import ctypes
    c = pk.config("tiny").c()
    h = ctypes.c_void_p()
    assert L.jagg_ctx_create(ctypes.byref(c), None, ctypes.byref(h)) == 0
    try:
        p = 1 << 20
        T, W = 10, 4
        vp = ctypes.c_void_p
        steps = (vp * T)(*[p] * T)
        pairs = (vp * 2)(p, p)
        s = (vp * T)(*[p] * T)
        t = (ctypes.c_float * T)(*[1.0 - k / T for k in range(T)])
        mask = (ctypes.c_ubyte * 2)(1, 0)

        def call(**kw):
            a = dict(T=T, W=W, batch=1, pairs=pairs, steps=steps, s=s, t=t, mask=mask, beta=0.0)
            a.update(kw)
            r = L.jagg_trajectory_backward(h, p, a["T"], a["W"], a["batch"], a["pairs"], a["steps"], a["s"], a["t"],
                                           a["mask"], p, a["beta"])
            return r, L.jagg_last_error()

        r, e = call()
        assert r == 1 and b"workspace" in e                      # valid arguments: stops at the workspace
        t_up = (ctypes.c_float * T)(*[0.1 + k / T for k in range(T)])
        assert call(t=t_up)[0] == 1                              # t increasing
        assert call(mask=(ctypes.c_ubyte * 2)(2, 0))[0] == 1     # mask byte not 0/1
        assert call(W=1)[0] == 1
        assert call(T=0)[0] == 1
        assert call(beta=0.5)[0] == 1
        assert call(pairs=(vp * 2)(None, p))[0] == 1             # JAGG window without its pair
        r, e = call(pairs=(vp * 2)(p, None))                     # per-step window needs no pair
        assert r == 1 and b"workspace" in e
        st = (vp * T)(*([p] * 4 + [None] + [p] * 5))
        assert call(steps=st)[0] == 1                            # per-step step 4 without its forward
        st = (vp * T)(*([None] + [p] * 9))
        r, e = call(steps=st)                                    # step 0 is in a JAGG window
        assert r == 1 and b"workspace" in e
        assert call(s=(vp * T)(*([p] * 9 + [p + 4])))[0] == 1   # unaligned s_k
        assert call(batch=17)[0] == 1                            # a JAGG window's pair would exceed 32
        r, e = call(mask=None, T=3)                              # no full window: no mask needed
        assert r == 1 and b"workspace" in e
        out = (ctypes.c_double * 4)()
        st4 = (vp * 4)(*[p] * 4)
        t4 = (ctypes.c_float * 4)(1.0, 0.9, 0.8, 0.7)
        assert L.jagg_window_quality(h, p, p, st4, 1, st4, t4, 1, p, p, p, out) == 1    # W < 2
        assert L.jagg_window_quality(h, p, p, st4, 1, st4, t4, 4, p, p + 8, p, out) == 1  # unaligned
        t4b = (ctypes.c_float * 4)(1.0, 0.9, 0.95, 0.7)
        assert L.jagg_window_quality(h, p, p, st4, 1, st4, t4b, 4, p, p, p, out) == 1  # t not decreasing
        assert L.jagg_window_quality(h, p, None, st4, 1, st4, t4, 4, p, p, p, out) == 1
    finally:
        L.jagg_ctx_destroy(h)
