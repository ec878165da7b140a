"""Group-backward throughput of the JAGG hot path on one MI355X.

Headline workload (the one the metric is quoted on): one double-stream MMDiT
block (hidden 3072, 24 heads x 128, MLP 12288), 4096 image tokens (1024^2
image -> 128^2 latent, 16 channels, 2x2 patches) + 512 text tokens, batch 1,
bf16 storage with fp32 accumulation, window W = 4.  A bench "step" is the
backward of one window: JAGG = composites + one VJP over the batched endpoint
pair (W denoising steps); per step = W VJPs with the same kernels.  Saved
activations come from the forward, which runs before the timed region;
parameter gradients accumulate (beta = 1) across windows.  `value` is JAGG
denoising steps per second; `ms_per_step` is milliseconds per window.

Also measured on the headline workload (reported beside it, not as `value`):
  * the batched per-step control: the W steps as ONE batch-W VJP with the same
    kernels (separates JAGG's pass count from the better GEMM shapes of a
    larger batch);
  * the update stage of one window, Phases 1-4 (forwards + GRPO loss + VJPs);
  * per-kernel-class time from HIP events bound to each kernel's dispatch, and
    achieved HBM bandwidth of the aggregation, GRPO and comparison kernels.
Further workloads of the default run (each its own object; `--no-extra`
skips them):
  * flux: the full-depth Flux-like model (19 double + 38 single blocks, ~11.8B
    parameters, 4096 + 512 tokens, batch 1, activation checkpointing, bf16
    gradients), W = 8: JAGG window vs per-step window;
  * qwen_routed: the Qwen-Image-like model (60 double blocks, 4096 + 256
    tokens, checkpointing), a T = 20, W = 8 trajectory (two windows and a
    4-step tail) whose routing comes from group scores of synthetic per-step
    hidden states: half the windows fall back to the per-step backward;
  * slice_sweep: the Flux-like slice (4 double + 8 single blocks, 1024 + 512
    tokens, batch 8), a T = 16, W = 4 trajectory routed by scores of
    synthetic hidden states whose pairwise cosine is swept 0.5 - 0.99, at
    several thresholds tau.
--workload slice|flux|qwen runs the headline measurements on that workload
instead (used for kernel traces).

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK = 2.5e15     # dense bf16 MFMA, MI355X
HBM_PEAK = 8.0e12

# HBM traffic of the weight-gradient GEMM class per launch in the block
# workload (one launch = both streams' products of one layer), from two
# rocprofv3 --pmc passes (FETCH_SIZE, WRITE_SIZE) scaled by the same counters
# on a 1 GiB device copy (FETCH_SIZE reads 0.5x, WRITE_SIZE 1.0x the bytes);
# valid only for the GEMM source it was measured on (sha256 of gemm.hip,
# first 16 hex digits).
WGRAD_TRAFFIC = {"gemm_src": "93aef00644e157f4", "bytes_per_launch": 1440.0e6}

CLASSES = {"gemm_fwd": 1, "gemm_dgrad": 2, "gemm_wgrad": 3, "attn_fwd": 4, "attn_bwd_kv": 5, "attn_bwd_q": 6,
           "aggregate": 7}


def say(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def block_flops(D, F, N, B):
    """Algorithmic FLOPs of one transformer-block parameter VJP for a batch of B.

    GEMMs: per token 4 D^2 + 2 D F weights (double block per stream: qkv, out,
    fc1, fc2; single block: the fused input and output projections, the same
    count), 2 flops per multiply-add; the backward does the input-gradient and
    the weight-gradient products (2x forward).  Attention backward: four
    N x N x Dh products per head (dV, dP, dQ, dK), 8 N^2 Dh flops, twice the
    forward's (backward-cost appendix).  The per-sample modulation products
    and the embeddings are excluded."""
    tok = B * N
    gemm_fwd = 2.0 * tok * (3 * D * D + D * D + 2 * D * F)
    attn_bwd = 8.0 * B * N * N * D
    return 2.0 * gemm_fwd + attn_bwd


def block_recompute_flops(D, F, N, B):
    """FLOPs a block's backward executes beyond the algorithmic ones: with
    activation checkpointing the block forward (GEMMs + attention QK^T and PV),
    and in every backward the flash-style recompute of the scores S = QK^T."""
    tok = B * N
    return 2.0 * tok * (3 * D * D + D * D + 2 * D * F) + 4.0 * B * N * N * D, 2.0 * B * N * N * D


def gemm_src_hash():
    p = os.path.join(ROOT, "paper_2607_17572_amd", "csrc", "gemm.hip")
    return hashlib.sha256(open(p, "rb").read()).hexdigest()[:16]


class Workload:
    """Seeded synthetic inputs of W steps: parameters, the W + 1 rollout
    latents (block workload: token streams), text embeddings, upstream
    gradients (per-sample advantage times N(0, 1)), GRPO settings.  The
    timesteps are the first W + 1 points of the uniform grid t_k = 1 - k/T."""

    def __init__(self, pk, synth, torch, name, W, B, T=16):
        self.cfg = cfg = pk.config(name)
        self.W, self.B = W, B
        self.ctx = ctx = pk.Context(cfg)
        self.dt = dt = torch.bfloat16
        th = torch.zeros(ctx.n_params, dtype=dt, device="cuda")
        th.copy_(synth.device_normal((ctx.n_params,), synth.THETA_SEED, std=0.02, dtype=dt))
        for nm, off, numel, r, c in ctx.layout:
            if nm.endswith("_gain"):
                th[off:off + numel] = 1.0 + 0.02 * synth.device_normal((numel,), synth.THETA_SEED + off)
        self.theta = th
        self.t = [1.0 - k / T for k in range(W + 1)]
        if cfg.block_only:
            shape = (B * cfg.n_tok, cfg.hidden)
            self.txt = [None] * (W + 1)
        else:
            shape = (B, cfg.in_ch, cfg.lat_h, cfg.lat_w)
            self.txt = [synth.device_normal((B, cfg.n_txt, cfg.txt_dim), synth.DATA_SEED + 50 + j, dtype=dt)
                        for j in range(W + 1)]
        self.shape = shape
        self.z = [synth.device_normal(shape, synth.DATA_SEED + j, dtype=dt) for j in range(W + 1)]
        a = synth.device_normal((B,), synth.DATA_SEED + 99)
        self.adv = a.float().contiguous()
        # per-sample advantage scale of the upstream gradients (block: B = 1)
        scale = a[0] if cfg.block_only else a.view((-1,) + (1,) * (len(shape) - 1))
        self.s = [(synth.device_normal(shape, synth.DATA_SEED + 100 + j) * scale).to(dt) for j in range(W)]
        self.sigma = [0.3] * W

    def batch_of(self, torch, arrays):
        """Several batch-B inputs as one batch-(k B) input (stream-major rows for a block)."""
        if self.cfg.block_only:
            nt = self.B * self.cfg.n_txt
            return torch.cat([x[:nt] for x in arrays] + [x[nt:] for x in arrays], 0)
        return torch.cat(arrays, 0)

    def txt_of(self, torch, idx):
        return None if self.cfg.block_only else torch.cat([self.txt[j] for j in idx], 0)

    def saved_pair(self, torch, i, j):
        """Batch-2B saving forward of steps i and j (endpoint i first)."""
        B, ctx = self.B, self.ctx
        sv = ctx.new_saved(2 * B)
        ctx.forward_save(self.theta, self.batch_of(torch, [self.z[i], self.z[j]]), [self.t[i]] * B + [self.t[j]] * B,
                         self.txt_of(torch, [i, j]), saved=sv, batch=2 * B)
        return sv

    def saved_step(self, k):
        sv = self.ctx.new_saved(self.B)
        self.ctx.forward_save(self.theta, self.z[k], [self.t[k]] * self.B, self.txt[k], saved=sv, batch=self.B)
        return sv


def timed(torch, fn, k):
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(k):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / 1e3


def class_times(pk, fn, k, names):
    """Per-kernel-class time of k calls of fn from HIP events bound to each
    kernel's dispatch (the library runs on one stream while timing)."""
    out = {}
    for name in names:
        pk.prof_begin(CLASSES[name])
        for _ in range(k):
            fn()
        n, ms, work = pk.prof_end()
        out[name] = {"launches_per_window": n // k, "avg_us": 1e3 * ms / max(n, 1), "work_per_window": work / k,
                     "ms_per_window": ms / k}
        if ms > 0 and name != "aggregate":
            out[name]["tflops"] = work / (ms * 1e-3) / 1e12
    return out


def free(torch):
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


# ---------------------------------------------------------------- headline
def leg_headline(args, pk, synth, torch):
    W = args.W or (4 if args.workload in ("block", "slice") else 8)
    B = 8 if args.workload == "slice" else 1
    wl = Workload(pk, synth, torch, args.workload, W, B)
    cfg, ctx, theta, t = wl.cfg, wl.ctx, wl.theta, wl.t
    D, F, N = cfg.hidden, cfg.mlp_hidden, cfg.n_tok
    nblk = cfg.n_double + cfg.n_single

    # forward: endpoint pair (batch 2B) for JAGG; every step (batch B) for the
    # baseline; all W steps as one batch-W B input for the batched control
    saved_pair = wl.saved_pair(torch, 0, W - 1)
    saved = [wl.saved_step(j) for j in range(W)]
    saved_all = None
    if args.only == "all" and W * B <= 32:
        saved_all = ctx.new_saved(W * B)
        ctx.forward_save(theta, wl.batch_of(torch, wl.z[:W]), [t[j] for j in range(W) for _ in range(B)],
                         wl.txt_of(torch, range(W)), saved=saved_all, batch=W * B)
        s_all = wl.batch_of(torch, wl.s)
    dth = torch.zeros(ctx.n_params, dtype=ctx.grad_dtype, device="cuda")
    torch.cuda.synchronize()
    ss = wl.s

    def run_jagg():
        ctx.group_backward(theta, saved_pair, B, ss, t[:W], dth, beta=1.0)

    def run_perstep():
        ctx.perstep_group_backward(theta, saved, B, ss, dth, beta=1.0)

    def run_batched():
        ctx.vjp(theta, saved_all, W * B, s_all, dth, beta=1.0)

    for _ in range(args.warmup):
        run_jagg()
        if args.only == "all":
            run_perstep()
            if saved_all is not None:
                run_batched()
    t_jagg = timed(torch, run_jagg, args.steps)
    t_ps = timed(torch, run_perstep, args.steps) if args.only == "all" else float("nan")
    t_bt = timed(torch, run_batched, args.steps) if saved_all is not None else float("nan")
    say(f"{args.workload}: jagg {1e3 * t_jagg / args.steps:.3f} ms/window, per-step {1e3 * t_ps / args.steps:.3f}, "
        f"batched per-step {1e3 * t_bt / args.steps:.3f}")

    kernels = class_times(pk, run_jagg, args.steps,
                          ["gemm_wgrad", "gemm_dgrad", "attn_bwd_kv", "attn_bwd_q", "aggregate"] +
                          (["gemm_fwd", "attn_fwd"] if cfg.checkpoint else []))
    wg = kernels["gemm_wgrad"]
    achieved = wg["work_per_window"] / (wg["ms_per_window"] * 1e-3) / 1e12
    agg = kernels["aggregate"]
    say(f"kernels {json.dumps(kernels)}")

    update = None
    if args.only == "all":
        update = update_stage(torch, pk, synth, wl, saved_pair, saved, dth, args.steps, args.warmup)
        kernels.update(update.pop("kernels"))
    ms_jagg = 1e3 * t_jagg / args.steps
    ms_ps = 1e3 * t_ps / args.steps
    ms_bt = 1e3 * t_bt / args.steps
    fl_pair = nblk * block_flops(D, F, N, 2 * B)
    fl_one = nblk * block_flops(D, F, N, B)
    traffic = None
    if WGRAD_TRAFFIC["gemm_src"] == gemm_src_hash() and args.workload == "block":
        traffic = WGRAD_TRAFFIC["bytes_per_launch"]
    wl_desc = {
        "block": "one double-stream MMDiT block, hidden 3072, 24x128 heads, MLP 12288, 4096 image + 512 text "
                 "tokens, batch 1, W=4 (JAGG joint endpoint pair)",
        "slice": "Flux-like MMDiT slice, 4 double + 8 single blocks, hidden 3072, 1024 image + 512 text tokens, "
                 "batch 8, W=4",
        "flux": "full-depth Flux-like MMDiT, 19 double + 38 single blocks (~11.8B params), 4096 image + 512 text "
                "tokens, batch 1, activation checkpointing, bf16 gradients, W=8",
        "qwen": "Qwen-Image-like MMDiT, 60 double blocks, 4096 image + 256 text tokens, batch 1, activation "
                "checkpointing, W=8",
    }[args.workload]
    out = {
        "metric": "denoising-step backward throughput (steps/s) + MFMA util, JAGG vs per-step bwd",
        "value": W * args.steps / t_jagg,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_jagg,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl_desc, "W": W, "batch": B, "tokens": N, "hidden": D, "blocks": nblk,
                   "step": f"one bench step = the backward of one window of W={W} denoising steps; ms_per_step is "
                           f"ms per window, value counts denoising steps"},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK / 1e12, "unit": "TFLOP/s",
                     "frac": achieved * 1e12 / MFMA_BF16_PEAK, "traffic": traffic,
                     "kernel": "gemm_dtl_kernel (weight-gradient GEMMs, dW = dY^T X)",
                     "avg_launch_us": wg["avg_us"], "launches_per_window": wg["launches_per_window"],
                     "timing": "HIP events bound to each launch's dispatch (hipExtLaunchKernelGGL), library stream"},
        "ms_per_window": ms_jagg,
        "perstep": {"value": W * args.steps / t_ps, "ms_per_window": ms_ps},
        "speedup_vs_perstep": t_ps / t_jagg,
        "tflops_jagg": fl_pair / (ms_jagg * 1e-3) / 1e12,
        "tflops_perstep": W * fl_one / (ms_ps * 1e-3) / 1e12,
        "aggregate_gbps": agg["work_per_window"] / (agg["ms_per_window"] * 1e-3) / 1e9,
        "kernels": kernels,
    }
    if saved_all is not None:
        out["perstep_batched"] = {"value": W * args.steps / t_bt, "ms_per_window": ms_bt,
                                  "tflops": W * fl_one / (ms_bt * 1e-3) / 1e12,
                                  "what": f"the W={W} steps as one batch-{W * B} VJP, same kernels"}
        out["speedup_vs_perstep_batched"] = t_bt / t_jagg
    if update is not None:
        out["update_stage"] = update
    out["mfma_frac_whole_backward"] = out["tflops_jagg"] * 1e12 / MFMA_BF16_PEAK
    cpu_inputs = (cfg, theta, wl.z, ss, t[:W], W) if args.workload == "block" else None
    del saved_pair, saved, saved_all, dth, wl
    return out, cpu_inputs


def update_stage(torch, pk, synth, wl, saved_pair, saved, dth, steps, warmup):
    """Phases 1-4 of one window (the paper's update stage on stored rollouts)
    with the GRPO loss of the window: JAGG against per step."""
    ctx, theta, t, W, B = wl.ctx, wl.theta, wl.t, wl.W, wl.B
    pair_in = wl.batch_of(torch, [wl.z[0], wl.z[W - 1]])
    pair_txt = wl.txt_of(torch, [0, W - 1])
    mid_in = wl.batch_of(torch, wl.z[1:W - 1])
    mid_txt = wl.txt_of(torch, range(1, W - 1))
    t_pair = [t[0]] * B + [t[W - 1]] * B
    t_mid = [t[j] for j in range(1, W - 1) for _ in range(B)]
    v_pair = torch.empty((2 * wl.shape[0],) + wl.shape[1:], dtype=wl.dt, device="cuda")
    v_mid = torch.empty(((W - 2) * wl.shape[0],) + wl.shape[1:], dtype=wl.dt, device="cuda")
    v_step = [torch.empty(wl.shape, dtype=wl.dt, device="cuda") for _ in range(W)]
    s_out = [torch.empty(wl.shape, dtype=wl.dt, device="cuda") for _ in range(W)]
    # v_0 and v_{W-1} are read from the pair output, the middle steps from the
    # batched middle output, in place
    vs = [(v_pair, 2 * B, 0)] + [(v_mid, (W - 2) * B, (j - 1) * B) for j in range(1, W - 1)] + [(v_pair, 2 * B, B)]
    adv = wl.adv
    # old log-probabilities near the current ones (ratios ~ exp(N(0, 0.1))):
    # one untimed pass gives log pi_j, a seeded perturbation gives log pi_old
    for j in range(W):
        ctx.forward_save(theta, wl.z[j], [t[j]] * B, wl.txt[j], saved=None, batch=B, v_out=v_step[j])
    stats = torch.zeros((W, B, 3), dtype=torch.float64, device="cuda")
    zero = torch.zeros((W, B), dtype=torch.float64, device="cuda")
    ctx.grpo_upstream(v_step, wl.z, t, wl.sigma, zero, adv, s_out, stats=stats)
    logp_old = (stats[..., 0] - 0.1 * synth.device_normal((W, B), synth.DATA_SEED + 321).double()).contiguous()

    def jagg_update():
        ctx.forward_save(theta, pair_in, t_pair, pair_txt, saved=saved_pair, batch=2 * B, v_out=v_pair)
        ctx.forward_save(theta, mid_in, t_mid, mid_txt, saved=None, batch=(W - 2) * B, v_out=v_mid)
        ctx.grpo_group_backward(theta, saved_pair, B, vs, wl.z, t, wl.sigma, logp_old, adv, dth, beta=1.0)

    def perstep_update():
        for j in range(W):
            ctx.forward_save(theta, wl.z[j], [t[j]] * B, wl.txt[j], saved=saved[j], batch=B, v_out=v_step[j])
        ctx.grpo_upstream(v_step, wl.z, t, wl.sigma, logp_old, adv, s_out)
        ctx.perstep_group_backward(theta, saved, B, s_out, dth, beta=1.0)

    for _ in range(warmup):
        jagg_update()
        perstep_update()
    tj = timed(torch, jagg_update, steps)
    tp = timed(torch, perstep_update, steps)
    kernels = {}
    pk.prof_begin(pk.PROF_UPSTREAM)
    for _ in range(steps):
        jagg_update()
    n, ms, work = pk.prof_end()
    kernels["grpo_composites"] = {"launches_per_window": n // steps, "avg_us": 1e3 * ms / max(n, 1),
                                  "work_per_window": work / steps, "ms_per_window": ms / steps,
                                  "gbps": work / (ms * 1e-3) / 1e9 if ms else None}
    g2 = torch.zeros_like(dth)
    pk.prof_begin(pk.PROF_COMPARE)
    for _ in range(steps):
        ctx.grad_compare(dth, g2)
    n, ms, work = pk.prof_end()
    kernels["grad_compare"] = {"launches_per_call": n // steps, "avg_us": 1e3 * ms / max(n, 1),
                               "bytes_per_call": work / steps, "gbps": work / (ms * 1e-3) / 1e9 if ms else None}
    res = {"jagg_ms_per_window": 1e3 * tj / steps, "perstep_ms_per_window": 1e3 * tp / steps,
           "speedup": tp / tj, "jagg_steps_s": W * steps / tj, "perstep_steps_s": W * steps / tp,
           "kernels": kernels}
    say(f"update stage: jagg {res['jagg_ms_per_window']:.3f} ms, per-step {res['perstep_ms_per_window']:.3f} ms "
        f"per window")
    return res


# ------------------------------------------------------- further workloads
def leg_flux(pk, synth, torch, windows=2):
    """Full-depth Flux-like model, W = 8: JAGG window against per-step window,
    with per-class kernel time over one JAGG window."""
    W, B = 8, 1
    wl = Workload(pk, synth, torch, "flux", W, B)
    cfg, ctx, theta, t = wl.cfg, wl.ctx, wl.theta, wl.t
    saved_pair = wl.saved_pair(torch, 0, W - 1)
    saved = [wl.saved_step(j) for j in range(W)]
    dth = torch.zeros(ctx.n_params, dtype=ctx.grad_dtype, device="cuda")

    def run_jagg():
        ctx.group_backward(theta, saved_pair, B, wl.s, t[:W], dth, beta=1.0)

    def run_perstep():
        ctx.perstep_group_backward(theta, saved, B, wl.s, dth, beta=1.0)

    run_jagg()
    run_perstep()
    tj = timed(torch, run_jagg, windows)
    tp = timed(torch, run_perstep, windows)
    say(f"flux: jagg {1e3 * tj / windows:.1f} ms/window, per-step {1e3 * tp / windows:.1f} ms/window")
    kernels = class_times(pk, run_jagg, 1, ["gemm_fwd", "gemm_wgrad", "gemm_dgrad", "attn_fwd", "attn_bwd_kv",
                                            "attn_bwd_q", "aggregate"])
    D, F, N, nblk = cfg.hidden, cfg.mlp_hidden, cfg.n_tok, cfg.n_double + cfg.n_single
    alg_j = nblk * block_flops(D, F, N, 2 * B)
    rc_j, fl_j = block_recompute_flops(D, F, N, 2 * B)
    alg_p = W * nblk * block_flops(D, F, N, B)
    rc_p, fl_p = block_recompute_flops(D, F, N, B)
    exe_j = alg_j + nblk * (rc_j + fl_j)
    exe_p = alg_p + W * nblk * (rc_p + fl_p)
    ms_j, ms_p = 1e3 * tj / windows, 1e3 * tp / windows
    dom = max((k for k in kernels if k != "aggregate"), key=lambda k: kernels[k]["ms_per_window"])
    res = {"workload": "full-depth Flux-like MMDiT, 19 double + 38 single blocks (~11.8B params), 4096 image + 512 "
                       "text tokens, batch 1, activation checkpointing, bf16 parameters and gradients, W=8",
           "windows_timed": windows, "jagg_ms_per_window": ms_j, "perstep_ms_per_window": ms_p,
           "value": W / (ms_j * 1e-3), "perstep_value": W / (ms_p * 1e-3), "unit": "steps/s",
           "speedup_vs_perstep": ms_p / ms_j,
           "jagg_tflop_algorithmic": alg_j / 1e12, "jagg_tflop_executed": exe_j / 1e12,
           "perstep_tflop_algorithmic": alg_p / 1e12, "perstep_tflop_executed": exe_p / 1e12,
           "jagg_tflops_algorithmic": alg_j / (ms_j * 1e-3) / 1e12, "jagg_tflops_executed": exe_j / (ms_j * 1e-3) / 1e12,
           "dominant_kernel": dom, "dominant_frac_of_peak": kernels[dom].get("tflops", 0.0) * 1e12 / MFMA_BF16_PEAK,
           "kernels": kernels}
    del saved_pair, saved, dth, wl
    return res


def leg_qwen_routed(pk, synth, torch):
    """Qwen-Image-like model, T = 20, W = 8: windows [0..7], [8..15] and a
    4-step per-step tail.  Routing from K14 scores of synthetic per-step hidden
    states (pairwise cosine 0.9 for window 0, 0.35 for window 1; tau 0.5):
    window 0 takes JAGG, window 1 falls back.  Timed against the same
    trajectory with every window per step."""
    T, W, B = 20, 8, 1
    wl = Workload(pk, synth, torch, "qwen", T, B, T=T)
    ctx, theta, t = wl.ctx, wl.theta, wl.t[:T]
    rhos, tau = [0.9, 0.35], 0.5
    scores = []
    for g, rho in enumerate(rhos):
        h = synth.hidden_profile(W, 1 << 20, rho, seed=7000 + g)
        scores.append(ctx.group_score([torch.from_numpy(x.astype("float32")).cuda() for x in h]))
    mask, frac = pk.route(T // W, scores=scores, tau=tau)
    pairs = [wl.saved_pair(torch, g * W, g * W + W - 1) if mask[g] else None for g in range(T // W)]
    steps = [wl.saved_step(k) for k in range(T)]
    dth = torch.zeros(ctx.n_params, dtype=ctx.grad_dtype, device="cuda")

    def routed():
        ctx.trajectory_backward(theta, W, B, pairs, steps, wl.s, t, mask, dth, beta=1.0)

    def all_perstep():
        ctx.trajectory_backward(theta, W, B, [None] * (T // W), steps, wl.s, t, [0] * (T // W), dth, beta=1.0)

    tr = timed(torch, routed, 1)
    tp = timed(torch, all_perstep, 1)
    say(f"qwen routed trajectory: mask {mask}, {1e3 * tr:.1f} ms vs all per-step {1e3 * tp:.1f} ms")
    n_j = sum(mask)
    res = {"workload": "Qwen-Image-like MMDiT, 60 double blocks, 4096 image + 256 text tokens, batch 1, activation "
                       "checkpointing, T=20 steps, W=8: windows [0-7], [8-15] + a 4-step per-step tail",
           "routing": {"scores": scores, "tau": tau, "mask": mask, "jagg_frac": frac,
                       "hidden_state_cosines": rhos},
           "routed_ms": 1e3 * tr, "all_perstep_ms": 1e3 * tp, "value": T / tr, "all_perstep_value": T / tp,
           "unit": "steps/s", "speedup": tp / tr,
           "pass_count_speedup": T / (2 * n_j + W * (T // W - n_j) + T % W)}
    del pairs, steps, dth, wl
    return res


def leg_slice_sweep(pk, synth, torch):
    """Flux-like slice, batch 8, T = 16, W = 4 (four windows, no tail).  For
    each swept cosine rho_0 the windows' synthetic hidden states have pairwise
    cosine rho_0 - 0.1 g (window g, high noise first); K14 scores them,
    jagg_route decides at each tau, and the trajectory runs with that mask.
    Every window's backward reads the first window's saved activations (same
    shapes; the time does not depend on the values), the upstream gradients
    are per step; each distinct mask is timed once."""
    T, W, B = 16, 4, 8
    wl = Workload(pk, synth, torch, "slice", T, B, T=T)
    ctx, theta, t = wl.ctx, wl.theta, wl.t[:T]
    n_win = T // W
    pair = wl.saved_pair(torch, 0, W - 1)
    step = [wl.saved_step(k) for k in range(W)]
    steps = [step[k % W] for k in range(T)]
    dth = torch.zeros(ctx.n_params, dtype=ctx.grad_dtype, device="cuda")
    rho0s, taus = [0.5, 0.6, 0.7, 0.8, 0.9, 0.99], [0.5, 0.7, 0.9]
    score = {}
    for r0 in rho0s:
        sc = []
        for g in range(n_win):
            rho = max(r0 - 0.1 * g, 0.05)
            h = synth.hidden_profile(W, 1 << 18, rho, seed=int(7100 + 100 * r0 + g))
            sc.append(ctx.group_score([torch.from_numpy(x.astype("float32")).cuda() for x in h]))
        score[r0] = sc
    times = {}

    def run(mask):
        ctx.trajectory_backward(theta, W, B, [pair] * n_win, steps, wl.s, t, mask, dth, beta=1.0)

    run([1] * n_win)  # warm-up
    rows = []
    for r0 in rho0s:
        for tau in taus:
            mask, frac = pk.route(n_win, scores=score[r0], tau=tau)
            key = tuple(mask)
            if key not in times:
                times[key] = timed(torch, lambda: run(list(key)), 1)
            rows.append({"rho0": r0, "tau": tau, "scores": score[r0], "mask": mask, "jagg_frac": frac,
                         "ms": 1e3 * times[key], "steps_s": T / times[key]})
    base = (0,) * n_win
    if base not in times:
        times[base] = timed(torch, lambda: run(list(base)), 1)
    for r in rows:
        r["speedup_vs_all_perstep"] = times[base] / (r["ms"] * 1e-3)
    say("slice sweep: " + ", ".join(f"{k}: {1e3 * v:.1f} ms" for k, v in sorted(times.items())))
    res = {"workload": "Flux-like MMDiT slice, 4 double + 8 single blocks, hidden 3072, 1024 image + 512 text "
                       "tokens, batch 8, T=16, W=4 (4 windows)",
           "all_perstep_ms": 1e3 * times[base], "rows": rows,
           "note": "windows reuse the first window's saved activations; each distinct mask timed once"}
    del pair, step, steps, dth, wl
    return res


# ------------------------------------------------------------ CPU baseline
def cpu_baseline(cfg, theta, zs, ss, t, W):
    """The oracle, timed on this host's cores on bounded samples of the block
    workload, scaled to the metric's unit (denoising steps/s of the window
    backward):
      * all cores: the composites of one W = 4 window and ONE batch-1 endpoint
        VJP of the full-size block (fp32); JAGG window = composites + 2 VJPs,
        per-step window = W VJPs (extrapolated from the one measured VJP);
      * one thread: one batch-1 VJP of the same block with 256 image + 64 text
        tokens, scaled to the full size by the ratio of algorithmic FLOPs
        (extrapolated)."""
    import numpy as np
    import threadpoolctl
    from oracle import jagg as ojagg, mmdit

    def ocfg(lat, n_txt):
        return mmdit.Config(n_double=cfg.n_double, n_single=0, hidden=cfg.hidden, heads=cfg.heads,
                            head_dim=cfg.head_dim, mlp_hidden=cfg.mlp_hidden, in_ch=cfg.in_ch, patch=cfg.patch,
                            lat_h=lat, lat_w=lat, n_txt=n_txt, txt_dim=cfg.txt_dim, t_freq_dim=cfg.t_freq_dim,
                            block_only=True)

    oc = ocfg(cfg.lat_h, cfg.n_txt)
    nt = cfg.n_txt
    P = mmdit.unflatten(oc, theta.float().cpu().numpy(), np.float32)
    x0 = zs[0].float().cpu().numpy()
    s_np = [s.float().cpu().numpy() for s in ss]
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    nproc = os.cpu_count()
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = nproc
    threads = max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] + [1])
    say("oracle forward, full-size block (untimed)")
    inp = mmdit.Inputs(t=np.array([t[0]]), x_txt=x0[:nt][None], x_img=x0[nt:][None])
    _, cache = mmdit.forward(oc, P, inp)
    t0 = time.perf_counter()
    sb, sc = ojagg.aggregate(s_np, np.asarray(t, dtype=np.float64), acc_dtype=np.float32)
    t_agg = time.perf_counter() - t0
    t0 = time.perf_counter()
    mmdit.vjp(oc, P, cache, (sb[:nt][None], sb[nt:][None]))
    t_vjp = time.perf_counter() - t0
    del cache
    jagg_s = t_agg + 2.0 * t_vjp
    ps_s = W * t_vjp
    say(f"oracle, {threads} threads: aggregate {t_agg:.2f}s, one endpoint VJP {t_vjp:.2f}s")
    # one thread, token sample: 16 x 16 image grid (lat 32, patch 2) + 64 text tokens
    small = ocfg(32, 64)
    n_img_s = small.n_img
    D = cfg.hidden
    xs = np.concatenate([x0[:64], x0[nt:nt + n_img_s]], axis=0)
    inp_s = mmdit.Inputs(t=np.array([t[0]]), x_txt=xs[:64][None], x_img=xs[64:][None])
    sbs = np.concatenate([sb[:64], sb[nt:nt + n_img_s]], axis=0)
    with threadpoolctl.threadpool_limits(1):
        _, cache_s = mmdit.forward(small, P, inp_s)
        t0 = time.perf_counter()
        mmdit.vjp(small, P, cache_s, (sbs[:64][None], sbs[64:][None]))
        t_vjp1_s = time.perf_counter() - t0
    scale = block_flops(D, cfg.mlp_hidden, cfg.n_tok, 1) / block_flops(D, cfg.mlp_hidden, small.n_tok, 1)
    t_vjp1 = t_vjp1_s * scale
    say(f"oracle, 1 thread: VJP of a {small.n_tok}-token sample {t_vjp1_s:.2f}s -> full size {t_vjp1:.1f}s")
    return {"value": W / jagg_s, "unit": "steps/s", "cores": threads, "kind": "oracle",
            "extrapolated": True,
            "sample": "numpy fp32 oracle, block workload: composites of one W=4 window + one batch-1 endpoint VJP "
                      "of the full-size block timed on all threads; JAGG window = composites + 2 VJPs, per-step "
                      "window = 4 VJPs",
            "nproc": nproc, "cpus_available": avail, "cpu_model": model,
            "jagg_window_s": jagg_s, "perstep_window_s": ps_s, "perstep_value": W / ps_s,
            "measured_s": {"aggregate": t_agg, "endpoint_vjp": t_vjp},
            "single_thread": {"value": W / (t_agg + 2.0 * t_vjp1), "perstep_value": W / (W * t_vjp1),
                              "jagg_window_s": t_agg + 2.0 * t_vjp1, "perstep_window_s": W * t_vjp1,
                              "sample": f"one batch-1 VJP of the block with {small.n_tok} tokens on one thread "
                                        f"({t_vjp1_s:.2f} s), scaled by the algorithmic FLOP ratio {scale:.1f}; "
                                        "the composites' time is the one measured above (numpy's elementwise "
                                        "arithmetic runs on one thread)",
                              "extrapolated": True}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", choices=["block", "slice", "flux", "qwen"], default="block")
    ap.add_argument("--W", type=int, default=0, help="window size (default: 4 for block and slice, 8 for flux and qwen)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-extra", action="store_true", help="skip the flux, qwen and slice workloads")
    ap.add_argument("--calib-copy", action="store_true",
                    help="first run a plain 1 GiB device copy, larger than the 256 MB last-level cache "
                         "(calibrates rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    ap.add_argument("--only", choices=["all", "jagg"], default="all",
                    help="jagg: time the JAGG windows only (for a kernel trace of exactly those launches)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU (the path has no multi-GPU sharding); "
                                   "--gpus must be 1"}))
        sys.exit(2)

    import torch
    import paper_2607_17572_amd as pk
    import synth

    pk.lib()  # fails loudly if the HIP library is not built
    if args.calib_copy:
        # a copy kernel of known size: reads and writes exactly 1 GiB
        src = torch.ones(512 << 20, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    out, cpu_in = leg_headline(args, pk, synth, torch)
    free(torch)
    extra = args.workload == "block" and args.only == "all" and not args.no_extra
    if extra:
        for name, fn in (("flux", leg_flux), ("qwen_routed", leg_qwen_routed), ("slice_sweep", leg_slice_sweep)):
            t0 = time.perf_counter()
            try:
                out[name] = fn(pk, synth, torch)
            except Exception as e:  # a secondary workload must not lose the headline line
                out[name] = {"error": f"{type(e).__name__}: {e}"}
                say(f"{name} failed: {e}")
            free(torch)
            say(f"{name} leg: {time.perf_counter() - t0:.1f} s")
    if not args.no_cpu and cpu_in is not None:
        out["cpu_baseline"] = cpu_baseline(*cpu_in)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
