"""Group-backward throughput of the JAGG hot path on one MI355X.

Workload: one double-stream MMDiT block (hidden 3072, 24 heads x 128, MLP
12288), 4096 image tokens (1024^2 image -> 128^2 latent, 16 channels, 2x2
patches) + 512 text tokens, batch 1, bf16 storage with fp32 accumulation,
window W = 4.  A "step" is the backward of one window: JAGG = composites +
one VJP over the batched endpoint pair; per step = W VJPs with the same
kernels.  Saved activations come from the forward, which runs before the
timed region; parameter gradients accumulate (beta = 1) across windows.

Prints one JSON line (value = JAGG denoising-step backward throughput).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK = 2.5e15     # dense bf16 MFMA, MI355X
HBM_PEAK = 8.0e12


def block_flops(D, F, N, nt, ni, B):
    """Algorithmic FLOPs of one double-block parameter VJP for a batch of B.

    GEMMs: per token 4 D^2 + 2 D F weights per stream (qkv, out, fc1, fc2; the
    per-sample modulation is excluded), 2 flops per multiply-add; the backward
    does the input-gradient and the weight-gradient products (2x forward).
    Attention backward: four N x N x Dh products per head (dV, dP, dQ, dK),
    8 N^2 Dh flops, twice the forward's (backward-cost appendix)."""
    tok = B * N
    gemm_fwd = 2.0 * tok * (3 * D * D + D * D + 2 * D * F)
    attn_bwd = 8.0 * B * N * N * D
    return 2.0 * gemm_fwd + attn_bwd


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--calib-copy", action="store_true",
                    help="first run a plain 256 MiB device copy (calibrates rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    ap.add_argument("--only", choices=["all", "jagg"], default="all",
                    help="jagg: time the JAGG windows only (for a kernel trace of exactly those launches)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1"}))
        sys.exit(2)

    import torch
    import paper_2607_17572_amd as pk
    import synth

    pk.lib()  # fails loudly if the HIP library is not built
    if args.calib_copy:
        # a copy kernel of known size: reads and writes exactly 256 MiB
        src = torch.ones(128 << 20, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    cfg = pk.config("block")
    D, F, nt, ni = cfg.hidden, cfg.mlp_hidden, cfg.n_txt, cfg.n_img
    N = nt + ni
    W, B = 4, 1
    ctx = pk.Context(cfg)
    dt = torch.bfloat16
    theta = torch.zeros(ctx.n_params, dtype=dt, device="cuda")
    theta.copy_(synth.device_normal((ctx.n_params,), synth.THETA_SEED, std=0.02, dtype=dt))
    for name, off, numel, r, c in ctx.layout:
        if name.endswith("_gain"):
            theta[off:off + numel] = 1.0 + 0.02 * synth.device_normal((numel,), synth.THETA_SEED + off)
    t = [1.0 - k / 16 for k in range(W)]  # first window of a T = 16 uniform grid
    xs = [synth.device_normal((B * N, D), synth.DATA_SEED + j, dtype=dt) for j in range(W)]
    adv = float(synth.device_normal((1,), synth.DATA_SEED + 99).item())
    ss = [(synth.device_normal((B * N, D), synth.DATA_SEED + 100 + j) * adv).to(dt) for j in range(W)]

    # forward: endpoint pair (batch 2B) for JAGG; every step (batch B) for the baseline
    pair = torch.cat([xs[0][:B * nt], xs[-1][:B * nt], xs[0][B * nt:], xs[-1][B * nt:]], 0)
    saved_pair = ctx.new_saved(2 * B)
    ctx.forward_save(theta, pair, [t[0]] * B + [t[-1]] * B, None, saved=saved_pair, batch=2 * B)
    saved = []
    for j in range(W):
        sv = ctx.new_saved(B)
        ctx.forward_save(theta, xs[j], [t[j]] * B, None, saved=sv, batch=B)
        saved.append(sv)
    dth = torch.zeros(ctx.n_params, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()

    # forward (no graph) time, for the update-stage context number
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    vtmp = torch.empty_like(xs[0])
    ev0.record()
    for j in range(W):
        ctx.forward_save(theta, xs[j], [t[j]] * B, None, saved=None, batch=B, v_out=vtmp)
    ev1.record()
    torch.cuda.synchronize()
    fwd_ms = ev0.elapsed_time(ev1) / W

    def run_jagg():
        ctx.group_backward(theta, saved_pair, B, ss, t, dth, beta=1.0)

    def run_perstep():
        ctx.perstep_group_backward(theta, saved, B, ss, dth, beta=1.0)

    def timed(fn, k):
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(k):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / 1e3

    for _ in range(args.warmup):
        run_jagg()
        if args.only == "all":
            run_perstep()
    t_jagg = timed(run_jagg, args.steps)
    t_ps = timed(run_perstep, args.steps) if args.only == "all" else float("nan")
    print(f"[bench] jagg {1e3 * t_jagg / args.steps:.3f} ms/window, per-step {1e3 * t_ps / args.steps:.3f} ms/window",
          file=sys.stderr, flush=True)

    # dominant kernel: the weight-gradient GEMMs (the products that contract
    # over the token rows of both endpoints).  Live HIP-event timing of every
    # launch of that class over K JAGG windows, on the library's stream.
    kernels = {}
    for name, cls in (("gemm_wgrad", pk.PROF_GEMM_WGRAD), ("gemm_dgrad", pk.PROF_GEMM_DGRAD),
                      ("attn_bwd_kv", pk.PROF_ATTN_BWD_KV), ("attn_bwd_q", pk.PROF_ATTN_BWD_Q),
                      ("aggregate", pk.PROF_AGGREGATE)):
        pk.prof_begin(cls)
        for _ in range(args.steps):
            run_jagg()
        n, ms, work = pk.prof_end()
        kernels[name] = {"launches_per_window": n // args.steps, "avg_us": 1e3 * ms / max(n, 1),
                         "work_per_window": work / args.steps, "ms_per_window": ms / args.steps}
    wg = kernels["gemm_wgrad"]
    achieved = wg["work_per_window"] / (wg["ms_per_window"] * 1e-3) / 1e12
    agg = kernels["aggregate"]
    print(f"[bench] kernels {json.dumps(kernels)}", file=sys.stderr, flush=True)

    ms_jagg = 1e3 * t_jagg / args.steps
    ms_ps = 1e3 * t_ps / args.steps
    steps_s = W * args.steps / t_jagg
    fl_pair = block_flops(D, F, N, nt, ni, 2 * B)
    fl_one = block_flops(D, F, N, nt, ni, B)
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
        "config": {"workload": "one double-stream MMDiT block, hidden 3072, 24x128 heads, MLP 12288, "
                               "4096 image + 512 text tokens, batch 1, W=4 (JAGG joint endpoint pair)",
                   "W": W, "batch": B, "tokens": N, "hidden": D},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK / 1e12, "unit": "TFLOP/s",
                     "frac": achieved * 1e12 / MFMA_BF16_PEAK, "traffic": None,
                     "kernel": "gemm_mfma_kernel (weight-gradient GEMMs, dW = dY^T X)",
                     "avg_launch_us": wg["avg_us"], "launches_per_window": wg["launches_per_window"]},
        "perstep": {"value": W * args.steps / t_ps, "ms_per_window": ms_ps},
        "speedup_vs_perstep": t_ps / t_jagg,
        "tflops_jagg": fl_pair / (ms_jagg * 1e-3) / 1e12,
        "tflops_perstep": W * fl_one / (ms_ps * 1e-3) / 1e12,
        "forward_ms_per_step": fwd_ms,
        "aggregate_gbps": agg["work_per_window"] / (agg["ms_per_window"] * 1e-3) / 1e9,
        "kernels": kernels,
    }
    out["mfma_frac_whole_backward"] = out["tflops_jagg"] * 1e12 / MFMA_BF16_PEAK
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(cfg, theta, xs, ss, t, W)
    print(json.dumps(out), flush=True)


def cpu_baseline(cfg, theta, xs, ss, t, W):
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
    nt, ni, D = cfg.n_txt, cfg.n_img, cfg.hidden
    P = mmdit.unflatten(oc, theta.float().cpu().numpy(), np.float32)
    x0 = xs[0].float().cpu().numpy()
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
