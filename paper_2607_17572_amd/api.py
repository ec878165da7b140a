"""Thin Python binding over the JAGG C ABI (include/jagg.h).

Argument marshalling only: every step of the path runs in libjagg.so.  PyTorch
supplies device memory (tensors) and the HIP stream.  If the library is not
built, every entry point raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import asdict, dataclass

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libjagg.so")

F32, BF16 = 0, 1
DGRAD, DGRAD_GELU, WGRAD = 0, 1, 2


class _DitConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in (
        "n_double", "n_single", "hidden", "heads", "head_dim", "mlp_hidden", "in_ch", "patch", "lat_h",
        "lat_w", "n_txt", "txt_dim", "t_freq_dim", "block_only", "act_dtype", "grad_dtype", "checkpoint")]


class _GrpoWindow(ctypes.Structure):
    _fields_ = [("v_hat", ctypes.POINTER(ctypes.c_void_p)), ("z", ctypes.POINTER(ctypes.c_void_p)),
                ("t", ctypes.POINTER(ctypes.c_float)), ("sigma", ctypes.POINTER(ctypes.c_float)),
                ("logp_old", ctypes.c_void_p), ("adv", ctypes.c_void_p), ("clip_eps", ctypes.c_float),
                ("adv_clip", ctypes.c_float), ("W", ctypes.c_int), ("v_batch", ctypes.POINTER(ctypes.c_int)),
                ("v_index", ctypes.POINTER(ctypes.c_int))]


class _TensorDesc(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("offset", ctypes.c_size_t), ("numel", ctypes.c_size_t),
                ("rows", ctypes.c_int), ("cols", ctypes.c_int)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises RuntimeError if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2607_17572_amd.build.build() "
                               "(there is no fallback path)")
        L = ctypes.CDLL(LIB_PATH)
        vp, sz, i, f, d = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_float, ctypes.c_double
        pcfg = ctypes.POINTER(_DitConfig)
        L.jagg_last_error.restype = ctypes.c_char_p
        sig = {
            "dit_param_layout": [pcfg, ctypes.POINTER(sz), ctypes.POINTER(sz), ctypes.POINTER(_TensorDesc), sz],
            "jagg_ctx_create": [pcfg, vp, ctypes.POINTER(vp)],
            "dit_saved_bytes": [vp, i, ctypes.POINTER(sz)],
            "dit_workspace_bytes": [vp, i, ctypes.POINTER(sz)],
            "jagg_ctx_set_workspace": [vp, vp, sz],
            "dit_forward_save": [vp, vp, vp, ctypes.POINTER(f), vp, vp, vp, i],
            "dit_vjp": [vp, vp, vp, i, vp, vp, f],
            "jagg_alpha": [ctypes.POINTER(f), i, ctypes.POINTER(f)],
            "jagg_aggregate": [vp, ctypes.POINTER(vp), ctypes.POINTER(f), i, sz, i, vp, vp],
            "jagg_group_scores": [vp, ctypes.POINTER(vp), sz, i, i, ctypes.POINTER(d)],
            "jagg_group_scores_noalloc": [vp, ctypes.POINTER(vp), sz, i, i, vp],
            "jagg_route": [ctypes.POINTER(d), i, d, d, ctypes.POINTER(ctypes.c_ubyte), ctypes.POINTER(d)],
            "jagg_group_backward": [vp, vp, vp, i, ctypes.POINTER(vp), ctypes.POINTER(f), i, vp, f],
            "perstep_group_backward": [vp, vp, ctypes.POINTER(vp), i, ctypes.POINTER(vp), i, vp, f],
            "jagg_trajectory_backward": [vp, vp, i, i, i, ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp),
                                         ctypes.POINTER(f), ctypes.POINTER(ctypes.c_ubyte), vp, f],
            "jagg_linear_grad": [vp, i, vp, vp, vp, i, i, i, vp, i, f],
            "jagg_endpoint_backward": [vp, vp, vp, i, ctypes.POINTER(vp), ctypes.POINTER(f), i, i, vp, f],
            "jagg_grad_compare": [vp, vp, vp, sz, i, ctypes.POINTER(d)],
            "jagg_count_nonfinite": [vp, vp, sz, i, ctypes.POINTER(ctypes.c_ulonglong)],
            "jagg_window_quality": [vp, vp, vp, ctypes.POINTER(vp), i, ctypes.POINTER(vp), ctypes.POINTER(f), i, vp, vp,
                                    vp, ctypes.POINTER(d)],
            "jagg_grpo_composites": [vp, ctypes.POINTER(_GrpoWindow), i, vp, vp, vp],
            "jagg_grpo_upstream": [vp, ctypes.POINTER(_GrpoWindow), i, ctypes.POINTER(vp), vp],
            "jagg_grpo_group_backward": [vp, vp, vp, i, ctypes.POINTER(_GrpoWindow), vp, f, vp],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        L.jagg_ctx_destroy.argtypes = [vp]
        L.jagg_ctx_destroy.restype = None
        L.jagg_prof_begin.argtypes = [i]
        L.jagg_prof_begin.restype = ctypes.c_int
        L.jagg_prof_end.argtypes = [ctypes.POINTER(ctypes.c_long), ctypes.POINTER(d), ctypes.POINTER(d)]
        L.jagg_prof_end.restype = ctypes.c_int
        _lib = L
    return _lib


class JaggError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"JAGG status {status}: {msg}")
        self.status = status


def _check(rc: int):
    if rc != 0:
        raise JaggError(rc, lib().jagg_last_error().decode())


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
    block_only: int = 0
    act_dtype: int = F32
    grad_dtype: int = F32
    checkpoint: int = 0

    def c(self) -> _DitConfig:
        return _DitConfig(**{k: int(v) for k, v in asdict(self).items()})

    @property
    def n_img(self) -> int:
        return (self.lat_h // self.patch) * (self.lat_w // self.patch)

    @property
    def n_tok(self) -> int:
        return self.n_txt + self.n_img


def param_layout(cfg: Config):
    """[(name, offset, numel, rows, cols)], flat length."""
    c = cfg.c()
    nt, ne = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().dit_param_layout(ctypes.byref(c), ctypes.byref(nt), ctypes.byref(ne), None, 0))
    arr = (_TensorDesc * nt.value)()
    _check(lib().dit_param_layout(ctypes.byref(c), ctypes.byref(nt), ctypes.byref(ne), arr, nt.value))
    return [(d.name.decode(), d.offset, d.numel, d.rows, d.cols) for d in arr], ne.value


def alpha(t):
    W = len(t)
    tt = (ctypes.c_float * W)(*[float(x) for x in t])
    out = (ctypes.c_float * W)()
    _check(lib().jagg_alpha(tt, W, out))
    return list(out)


def route(n_groups: int, frac: float | None = None, scores=None, tau: float = 0.5):
    """(list of 0/1 per group, realised fraction)."""
    sc = None
    if scores is not None:
        sc = (ctypes.c_double * n_groups)(*[float(x) for x in scores])
    mask = (ctypes.c_ubyte * n_groups)()
    fr = ctypes.c_double()
    _check(lib().jagg_route(sc, n_groups, float(tau), -1.0 if frac is None else float(frac), mask, ctypes.byref(fr)))
    return list(mask), fr.value


PROF_GEMM_FWD, PROF_GEMM_DGRAD, PROF_GEMM_WGRAD = 1, 2, 3
PROF_ATTN_FWD, PROF_ATTN_BWD_KV, PROF_ATTN_BWD_Q, PROF_AGGREGATE = 4, 5, 6, 7
PROF_COMPARE, PROF_UPSTREAM = 8, 9


def prof_begin(cls: int):
    """Arm HIP-event timing of every launch of kernel class ``cls``."""
    _check(lib().jagg_prof_begin(cls))


def prof_end():
    """(launches, total kernel ms, total algorithmic work) of the armed class."""
    n, ms, work = ctypes.c_long(), ctypes.c_double(), ctypes.c_double()
    _check(lib().jagg_prof_end(ctypes.byref(n), ctypes.byref(ms), ctypes.byref(work)))
    return n.value, ms.value, work.value


def _ptrs(tensors):
    return (ctypes.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])


def _torch():
    import torch
    return torch


class Context:
    """One model configuration bound to a HIP stream, with a workspace tensor."""

    def __init__(self, cfg: Config, stream=None):
        torch = _torch()
        self.cfg = cfg
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        h = ctypes.c_void_p()
        c = cfg.c()
        _check(lib().jagg_ctx_create(ctypes.byref(c), ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(h)))
        self._h = h
        self._ws = None
        self._ws_batch = 0
        self.layout, self.n_params = param_layout(cfg)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.jagg_ctx_destroy(h)
            self._h = None

    @property
    def dtype(self):
        torch = _torch()
        return torch.bfloat16 if self.cfg.act_dtype == BF16 else torch.float32

    @property
    def grad_dtype(self):
        torch = _torch()
        return torch.bfloat16 if self.cfg.grad_dtype == BF16 else torch.float32

    def saved_bytes(self, batch: int) -> int:
        n = ctypes.c_size_t()
        _check(lib().dit_saved_bytes(self._h, batch, ctypes.byref(n)))
        return n.value

    def workspace_bytes(self, batch: int) -> int:
        n = ctypes.c_size_t()
        _check(lib().dit_workspace_bytes(self._h, batch, ctypes.byref(n)))
        return n.value

    def ensure_workspace(self, batch: int):
        if self._ws is not None and self._ws_batch >= batch:
            return
        torch = _torch()
        nb = self.workspace_bytes(batch)
        self._ws = torch.empty(nb + 256, dtype=torch.uint8, device="cuda")
        base = self._ws.data_ptr()
        off = (-base) % 256
        _check(lib().jagg_ctx_set_workspace(self._h, ctypes.c_void_p(base + off), nb))
        self._ws_batch = batch

    def new_saved(self, batch: int):
        torch = _torch()
        return torch.empty(self.saved_bytes(batch), dtype=torch.uint8, device="cuda")

    def forward_save(self, theta, z, t, txt=None, saved=None, batch=None, v_out=None):
        """v = v_theta(z, t); `saved` (uint8 tensor of saved_bytes(batch)) or None (no graph)."""
        torch = _torch()
        B = len(t) if batch is None else batch
        self.ensure_workspace(B)
        if v_out is None:
            v_out = torch.empty_like(z)
        tt = (ctypes.c_float * B)(*[float(x) for x in t])
        _check(lib().dit_forward_save(self._h, theta.data_ptr(), z.data_ptr(), tt,
                                      None if txt is None else txt.data_ptr(), v_out.data_ptr(),
                                      None if saved is None else saved.data_ptr(), B))
        return v_out

    def vjp(self, theta, saved, batch: int, s, dtheta, beta: float = 0.0):
        self.ensure_workspace(batch)
        _check(lib().dit_vjp(self._h, theta.data_ptr(), saved.data_ptr(), batch, s.data_ptr(), dtheta.data_ptr(),
                             float(beta)))
        return dtheta

    def aggregate(self, s_list, t, s_base, s_corr):
        W = len(s_list)
        tt = (ctypes.c_float * W)(*[float(x) for x in t])
        dt = BF16 if s_list[0].dtype == _torch().bfloat16 else F32
        _check(lib().jagg_aggregate(self._h, _ptrs(s_list), tt, W, s_list[0].numel(), dt, s_base.data_ptr(),
                                    s_corr.data_ptr()))
        return s_base, s_corr

    def group_score(self, h_list) -> float:
        self.ensure_workspace(1)
        out = ctypes.c_double()
        dt = BF16 if h_list[0].dtype == _torch().bfloat16 else F32
        _check(lib().jagg_group_scores(self._h, _ptrs(h_list), h_list[0].numel(), len(h_list), dt, ctypes.byref(out)))
        return out.value

    def group_score_noalloc(self, h_list, score_dev):
        """Allocation-free group score: written into score_dev (a device fp64
        tensor of one element) on the stream; needs no workspace."""
        dt = BF16 if h_list[0].dtype == _torch().bfloat16 else F32
        _check(lib().jagg_group_scores_noalloc(self._h, _ptrs(h_list), h_list[0].numel(), len(h_list), dt,
                                               score_dev.data_ptr()))
        return score_dev

    def group_backward(self, theta, saved_pair, batch: int, s_list, t, dtheta, beta: float = 0.0):
        """JAGG: composites + one VJP over the batch-2B endpoint pair."""
        W = len(s_list)
        self.ensure_workspace(2 * batch)
        tt = (ctypes.c_float * W)(*[float(x) for x in t])
        _check(lib().jagg_group_backward(self._h, theta.data_ptr(), saved_pair.data_ptr(), batch, _ptrs(s_list), tt,
                                         W, dtheta.data_ptr(), float(beta)))
        return dtheta

    def endpoint_backward(self, theta, saved, batch: int, s_list, t, endpoint: int, dtheta, beta: float = 0.0):
        """Sequential-graph JAGG: the backward of one endpoint (0: s_base, 1: s_corr)."""
        W = len(s_list)
        self.ensure_workspace(batch)
        tt = (ctypes.c_float * W)(*[float(x) for x in t])
        _check(lib().jagg_endpoint_backward(self._h, theta.data_ptr(), saved.data_ptr(), batch, _ptrs(s_list), tt, W,
                                            int(endpoint), dtheta.data_ptr(), float(beta)))
        return dtheta

    def grad_compare(self, a, b):
        """(a.b, a.a, b.b, cos, rho) over every element of two equal-size device
        tensors: the fp64 sums and the quality figures the library forms from them."""
        self.ensure_workspace(1)
        out = (ctypes.c_double * 5)()
        dt = BF16 if a.dtype == _torch().bfloat16 else F32
        assert a.numel() == b.numel() and a.dtype == b.dtype
        _check(lib().jagg_grad_compare(self._h, a.data_ptr(), b.data_ptr(), a.numel(), dt, out))
        return tuple(out)

    def count_nonfinite(self, x) -> int:
        """Number of NaN / +-Inf elements of a device tensor (fp32 or bf16)."""
        self.ensure_workspace(1)
        out = ctypes.c_ulonglong()
        dt = BF16 if x.dtype == _torch().bfloat16 else F32
        _check(lib().jagg_count_nonfinite(self._h, x.data_ptr(), x.numel(), dt, ctypes.byref(out)))
        return int(out.value)

    def window_quality(self, theta, saved_pair, saved_steps, batch: int, s_list, t, g_jagg, g_exact, g_ablate):
        """(cos_jagg, rho_jagg, cos_ablate, rho_ablate) of one window; the three
        group gradients are left in the given (zero-padded) buffers."""
        W = len(s_list)
        self.ensure_workspace(2 * batch)
        tt = (ctypes.c_float * W)(*[float(x) for x in t])
        out = (ctypes.c_double * 4)()
        _check(lib().jagg_window_quality(self._h, theta.data_ptr(), saved_pair.data_ptr(), _ptrs(saved_steps), batch,
                                         _ptrs(s_list), tt, W, g_jagg.data_ptr(), g_exact.data_ptr(),
                                         g_ablate.data_ptr(), out))
        return tuple(out)

    @staticmethod
    def _grpo_window(v_list, z_list, t, sigma, logp_old, adv, clip_eps, adv_clip):
        """The C struct of one GRPO window; returns (struct, keep-alive list).
        logp_old: device fp64 tensor [W][B]; adv: device fp32 tensor [B].
        An entry of v_list may be (tensor, batch, index): samples index ..
        index + B - 1 of a batch-``batch`` model output."""
        W = len(v_list)
        assert len(z_list) == W + 1 and len(t) == W + 1 and len(sigma) == W
        vt = [x[0] if isinstance(x, tuple) else x for x in v_list]
        B = adv.numel()
        vb = (ctypes.c_int * W)(*[x[1] if isinstance(x, tuple) else B for x in v_list])
        vk = (ctypes.c_int * W)(*[x[2] if isinstance(x, tuple) else 0 for x in v_list])
        vp, zp = _ptrs(vt), _ptrs(z_list)
        tt = (ctypes.c_float * (W + 1))(*[float(x) for x in t])
        sg = (ctypes.c_float * W)(*[float(x) for x in sigma])
        w = _GrpoWindow(vp, zp, tt, sg, logp_old.data_ptr(), adv.data_ptr(), float(clip_eps), float(adv_clip), W,
                        vb, vk)
        return w, [vp, zp, tt, sg, vb, vk]

    def grpo_composites(self, v_list, z_list, t, sigma, logp_old, adv, s_base, s_corr, clip_eps=0.1, adv_clip=5.0,
                        stats=None, batch=None):
        """Phases 2 + 3 fused: composites of the window's GRPO upstream gradients."""
        B = adv.numel() if batch is None else batch
        self.ensure_workspace(1)
        w, keep = self._grpo_window(v_list, z_list, t, sigma, logp_old, adv, clip_eps, adv_clip)
        _check(lib().jagg_grpo_composites(self._h, ctypes.byref(w), B, s_base.data_ptr(), s_corr.data_ptr(),
                                          None if stats is None else stats.data_ptr()))
        return s_base, s_corr

    def grpo_upstream(self, v_list, z_list, t, sigma, logp_old, adv, s_out, clip_eps=0.1, adv_clip=5.0, stats=None,
                      batch=None):
        """Phase 2: the W upstream gradients s_j (written into s_out)."""
        B = adv.numel() if batch is None else batch
        self.ensure_workspace(1)
        w, keep = self._grpo_window(v_list, z_list, t, sigma, logp_old, adv, clip_eps, adv_clip)
        _check(lib().jagg_grpo_upstream(self._h, ctypes.byref(w), B, _ptrs(s_out),
                                        None if stats is None else stats.data_ptr()))
        return s_out

    def grpo_group_backward(self, theta, saved_pair, batch: int, v_list, z_list, t, sigma, logp_old, adv, dtheta,
                            beta: float = 0.0, clip_eps=0.1, adv_clip=5.0, stats=None):
        """Phases 2-4: fused composites into the pair cotangent, one joint VJP."""
        self.ensure_workspace(2 * batch)
        w, keep = self._grpo_window(v_list, z_list, t, sigma, logp_old, adv, clip_eps, adv_clip)
        _check(lib().jagg_grpo_group_backward(self._h, theta.data_ptr(), saved_pair.data_ptr(), batch,
                                              ctypes.byref(w), dtheta.data_ptr(), float(beta),
                                              None if stats is None else stats.data_ptr()))
        return dtheta

    def linear_grad(self, kind: int, dY, other, result, beta: float = 0.0, pre=None):
        """One product of a linear layer's backward (DGRAD, DGRAD_GELU or WGRAD)."""
        torch = _torch()
        rows, n_out = dY.shape
        n_in = other.shape[1]
        rdt = BF16 if result.dtype == torch.bfloat16 else F32
        _check(lib().jagg_linear_grad(self._h, kind, dY.data_ptr(), other.data_ptr(),
                                      None if pre is None else pre.data_ptr(), rows, n_out, n_in, result.data_ptr(),
                                      rdt, float(beta)))
        return result

    def trajectory_backward(self, theta, W: int, batch: int, saved_pairs, saved_steps, s_list, t, use_jagg, dtheta,
                            beta: float = 0.0):
        """Whole trajectory: JAGG for the windows use_jagg marks, per step for
        the rest and the T mod W tail.  saved_pairs: one entry per full window
        (None where it takes the per-step backward); saved_steps: one per step
        (None for steps of JAGG windows)."""
        T = len(s_list)
        n = T // W
        any_jagg = any(int(u) for u in use_jagg)
        self.ensure_workspace(2 * batch if any_jagg else batch)
        vp = ctypes.c_void_p
        pairs = (vp * max(n, 1))(*[None if x is None else x.data_ptr() for x in saved_pairs])
        steps = (vp * T)(*[None if x is None else x.data_ptr() for x in saved_steps])
        tt = (ctypes.c_float * T)(*[float(x) for x in t])
        mk = (ctypes.c_ubyte * max(n, 1))(*[int(u) for u in use_jagg])
        _check(lib().jagg_trajectory_backward(self._h, theta.data_ptr(), T, W, batch, pairs, steps, _ptrs(s_list), tt,
                                              mk, dtheta.data_ptr(), float(beta)))
        return dtheta

    def perstep_group_backward(self, theta, saved_list, batch: int, s_list, dtheta, beta: float = 0.0):
        self.ensure_workspace(batch)
        _check(lib().perstep_group_backward(self._h, theta.data_ptr(), _ptrs(saved_list), batch, _ptrs(s_list),
                                            len(s_list), dtheta.data_ptr(), float(beta)))
        return dtheta


# ------------------------------------------------------------------ configs
def config(name: str, **over) -> Config:
    """The five workloads: tiny (C1), block (C2), slice (C3), flux (C4), qwen (C5)."""
    big = dict(hidden=3072, heads=24, head_dim=128, mlp_hidden=12288, in_ch=16, patch=2, t_freq_dim=256,
               act_dtype=BF16, grad_dtype=F32)
    table = {
        "tiny": dict(n_double=2, n_single=0, hidden=64, heads=4, head_dim=16, mlp_hidden=256, in_ch=4, patch=1,
                     lat_h=4, lat_w=4, n_txt=8, txt_dim=64, t_freq_dim=256, act_dtype=F32, grad_dtype=F32),
        "block": dict(big, n_double=1, n_single=0, lat_h=128, lat_w=128, n_txt=512, txt_dim=3072, block_only=1),
        "slice": dict(big, n_double=4, n_single=8, lat_h=64, lat_w=64, n_txt=512, txt_dim=4096),
        "flux": dict(big, n_double=19, n_single=38, lat_h=128, lat_w=128, n_txt=512, txt_dim=4096,
                     grad_dtype=BF16, checkpoint=1),
        "qwen": dict(big, n_double=60, n_single=0, lat_h=128, lat_w=128, n_txt=256, txt_dim=4096, checkpoint=1),
    }
    d = dict(table[name])
    d.update(over)
    return Config(**d)
