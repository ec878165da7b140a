"""Group-backward throughput of the JAGG hot path on one MI355X.

Default workload: one double-stream MMDiT block (hidden 3072, 24 heads x 128,
MLP 12288), 4096 image tokens (1024^2 image -> 128^2 latent, 16 channels,
2x2 patches) + 512 text tokens, batch 1, bf16 storage with fp32
accumulation, window W = 4.  A "step" is the backward of one window: JAGG =
composites + one VJP over the batched endpoint pair; per step = W VJPs with
the same kernels.  Saved activations come from the forward, which runs before
the timed region; parameter gradients accumulate (beta = 1) across windows.

Also measured (reported beside the headline, not as `value`):
  * the update stage of one window, Phases 1-4: JAGG = forward of the endpoint
    pair with saved activations + one batched no-grad forward of the W - 2
    middle steps + the fused GRPO upstream gradients and composites + the
    joint VJP; per step = W forwards with saved activations + the W GRPO
    upstream gradients + W VJPs;
  * achieved HBM bandwidth of the aggregation, of the fused GRPO upstream
    kernels and of the gradient-quality comparison.
--workload slice|flux|qwen runs the same measurements on the full-model
workloads (checkpointed for flux and qwen); the block workload is the one the
metric is quoted on.

Prints one JSON line (value = JAGG denoising-step backward throughput).
"""
from __future__ import annotations

import argparse
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
# workload, from two rocprofv3 --pmc passes (FETCH_SIZE, WRITE_SIZE) scaled by
# the same counters on a 1 GiB device copy; valid only for the GEMM source
# it was measured on (sha256 of gemm.hip, first 16 hex digits).
WGRAD_TRAFFIC = {"gemm_src": "ee046861998b99f4", "bytes_per_launch": 710.12e6}


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


def gemm_src_hash():
    p = os.path.join(ROOT, "paper_2607_17572_amd", "csrc", "gemm.hip")
    return hashlib.sha256(open(p, "rb").read()).hexdigest()[:16]


class Workload:
    """Seeded synthetic inputs of one window: parameters, the W + 1 rollout
    latents (block workload: token streams), text embeddings, upstream
    gradients (per-sample advantage times N(0, 1)), GRPO settings."""

    def __init__(self, pk, synth, torch, name, W, B):
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
        T = 16
        self.t = [1.0 - k / T for k in range(W + 1)]  # first window of a T = 16 uniform grid, plus t_W
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


def timed(torch, fn, k):
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(k):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / 1e3


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", choices=["block", "slice", "flux", "qwen"], default="block")
    ap.add_argument("--W", type=int, default=0, help="window size (default: 4 for block and slice, 8 for flux and qwen)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
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
    W = args.W or (4 if args.workload in ("block", "slice") else 8)
    B = 8 if args.workload == "slice" else 1
    wl = Workload(pk, synth, torch, args.workload, W, B)
    cfg, ctx, theta, t = wl.cfg, wl.ctx, wl.theta, wl.t
    D, F, N = cfg.hidden, cfg.mlp_hidden, cfg.n_tok
    nblk = cfg.n_double + cfg.n_single

    # forward: endpoint pair (batch 2B) for JAGG; every step (batch B) for the baseline
    pair_in = wl.batch_of(torch, [wl.z[0], wl.z[W - 1]])
    pair_txt = wl.txt_of(torch, [0, W - 1])
    t_pair = [t[0]] * B + [t[W - 1]] * B
    saved_pair = ctx.new_saved(2 * B)
    ctx.forward_save(theta, pair_in, t_pair, pair_txt, saved=saved_pair, batch=2 * B)
    saved = []
    for j in range(W):
        sv = ctx.new_saved(B)
        ctx.forward_save(theta, wl.z[j], [t[j]] * B, wl.txt[j], saved=sv, batch=B)
        saved.append(sv)
    dth = torch.zeros(ctx.n_params, dtype=ctx.grad_dtype, device="cuda")
    torch.cuda.synchronize()

    ss = wl.s

    def run_jagg():
        ctx.group_backward(theta, saved_pair, B, ss, t[:W], dth, beta=1.0)

    def run_perstep():
        ctx.perstep_group_backward(theta, saved, B, ss, dth, beta=1.0)

    for _ in range(args.warmup):
        run_jagg()
        if args.only == "all":
            run_perstep()
    t_jagg = timed(torch, run_jagg, args.steps)
    t_ps = timed(torch, run_perstep, args.steps) if args.only == "all" else float("nan")
    print(f"[bench] {args.workload}: jagg {1e3 * t_jagg / args.steps:.3f} ms/window, "
          f"per-step {1e3 * t_ps / args.steps:.3f} ms/window", file=sys.stderr, flush=True)

    # dominant kernel: the weight-gradient GEMMs (the products that contract
    # over the token rows of both endpoints).  Live HIP-event timing of every
    # launch of each class over K JAGG windows, on the library's stream.
    ksteps = args.steps
    kernels = {}
    for name, cls in (("gemm_wgrad", pk.PROF_GEMM_WGRAD), ("gemm_dgrad", pk.PROF_GEMM_DGRAD),
                      ("attn_bwd_kv", pk.PROF_ATTN_BWD_KV), ("attn_bwd_q", pk.PROF_ATTN_BWD_Q),
                      ("aggregate", pk.PROF_AGGREGATE)):
        pk.prof_begin(cls)
        for _ in range(ksteps):
            run_jagg()
        n, ms, work = pk.prof_end()
        kernels[name] = {"launches_per_window": n // ksteps, "avg_us": 1e3 * ms / max(n, 1),
                         "work_per_window": work / ksteps, "ms_per_window": ms / ksteps}
    wg = kernels["gemm_wgrad"]
    achieved = wg["work_per_window"] / (wg["ms_per_window"] * 1e-3) / 1e12
    agg = kernels["aggregate"]
    print(f"[bench] kernels {json.dumps(kernels)}", file=sys.stderr, flush=True)

    update = None
    if args.only == "all":
        update = update_stage(torch, pk, synth, wl, saved_pair, saved, dth, args.steps, args.warmup)
        kernels.update(update.pop("kernels"))
    ms_jagg = 1e3 * t_jagg / args.steps
    ms_ps = 1e3 * t_ps / args.steps
    steps_s = W * args.steps / t_jagg
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
        "value": steps_s,
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
        "config": {"workload": wl_desc, "W": W, "batch": B, "tokens": N, "hidden": D, "blocks": nblk},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK / 1e12, "unit": "TFLOP/s",
                     "frac": achieved * 1e12 / MFMA_BF16_PEAK, "traffic": traffic,
                     "kernel": "gemm_dtl_kernel (weight-gradient GEMMs, dW = dY^T X)",
                     "avg_launch_us": wg["avg_us"], "launches_per_window": wg["launches_per_window"]},
        "perstep": {"value": W * args.steps / t_ps, "ms_per_window": ms_ps},
        "speedup_vs_perstep": t_ps / t_jagg,
        "tflops_jagg": fl_pair / (ms_jagg * 1e-3) / 1e12,
        "tflops_perstep": W * fl_one / (ms_ps * 1e-3) / 1e12,
        "aggregate_gbps": agg["work_per_window"] / (agg["ms_per_window"] * 1e-3) / 1e9,
        "kernels": kernels,
    }
    if update is not None:
        out["update_stage"] = update
    out["mfma_frac_whole_backward"] = out["tflops_jagg"] * 1e12 / MFMA_BF16_PEAK
    if not args.no_cpu and args.workload == "block":
        out["cpu_baseline"] = cpu_baseline(cfg, theta, wl.z, ss, t[:W], W)
    print(json.dumps(out), flush=True)


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
    print(f"[bench] update stage: jagg {res['jagg_ms_per_window']:.3f} ms, per-step "
          f"{res['perstep_ms_per_window']:.3f} ms per window", file=sys.stderr, flush=True)
    return res


def cpu_baseline(cfg, theta, zs, ss, t, W):
    """The oracle, timed on this host on a bounded sample of the same workload:
    the composites of one window plus ONE endpoint VJP (batch 1, full size, fp32),
    scaled to the window (two endpoint VJPs) and reported in steps/s."""
    import numpy as np
    import threadpoolctl
    from oracle import jagg as ojagg, mmdit

    oc = mmdit.Config(n_double=cfg.n_double, n_single=0, hidden=cfg.hidden, heads=cfg.heads,
                      head_dim=cfg.head_dim, mlp_hidden=cfg.mlp_hidden, in_ch=cfg.in_ch, patch=cfg.patch,
                      lat_h=cfg.lat_h, lat_w=cfg.lat_w, n_txt=cfg.n_txt, txt_dim=cfg.txt_dim,
                      t_freq_dim=cfg.t_freq_dim, block_only=True)
    nt = cfg.n_txt
    P = mmdit.unflatten(oc, theta.float().cpu().numpy(), np.float32)
    x0 = zs[0].float().cpu().numpy()
    inp = mmdit.Inputs(t=np.array([t[0]]), x_txt=x0[:nt][None], x_img=x0[nt:][None])
    s_np = [s.float().cpu().numpy() for s in ss]
    print("[bench] oracle forward (untimed)", file=sys.stderr, flush=True)
    _, cache = mmdit.forward(oc, P, inp)
    info = threadpoolctl.threadpool_info()
    cores = max([i.get("num_threads", 1) for i in info] + [1])
    t0 = time.perf_counter()
    sb, sc = ojagg.aggregate(s_np, np.asarray(t, dtype=np.float64), acc_dtype=np.float32)
    t_agg = time.perf_counter() - t0
    t0 = time.perf_counter()
    mmdit.vjp(oc, P, cache, (sb[:nt][None], sb[nt:][None]))
    t_vjp = time.perf_counter() - t0
    t_window = t_agg + 2.0 * t_vjp
    print(f"[bench] oracle: aggregate {t_agg:.2f}s, one endpoint VJP {t_vjp:.2f}s", file=sys.stderr, flush=True)
    return {"value": W / t_window, "unit": "steps/s", "cores": cores, "kind": "oracle",
            "sample": "numpy fp32 oracle: composites of one W=4 window + one batch-1 endpoint VJP of the "
                      "full-size block, timed; window = composites + 2 endpoint VJPs",
            "seconds_measured": t_agg + t_vjp}


if __name__ == "__main__":
    main()
