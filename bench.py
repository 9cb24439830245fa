"""Meta-gradients/sec of the MixFlow-MG path on one MI355X.

Workload: 8-layer ReLU MLP, width 4096, 1000 classes (121,566,184 parameters),
1024-row batches, SGD with per-parameter log learning rates (eta has the shape
of theta), bf16 GEMM operands with float32 accumulation; the meta-gradient
dV/deta through T inner steps (default T = 8).  Inputs are seeded synthetic
Gaussian batches with uniform labels, resident in HBM before timing starts.

One "step" is one mfmg_meta_grad call: T forward inner steps with
checkpoints, the validation pass, and T forward-over-reverse reverse steps.
The line also carries the peak device bytes at every T of the memory sweep,
the roofline of the dominant kernel (timed with HIP events on the stream it
runs on) and the float64 CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 matrix
PEAK_HBM_GBS = 8000.0

KERNEL_CLASSES = ["fwd_gemm", "bwd_data_gemm", "bwd_weight_gemm_update", "dual_fwd_gemm",
                  "dual_bwd_data_gemm", "dual_bwd_weight_gemm_reverse_first_layer", "loss_head",
                  "elementwise", "dual_bwd_weight_gemm_reverse"]


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_flops(cfg: W.Config, T: int):
    """Matrix-product flops the method must compute, per kernel class, per meta-gradient.
    One unit = 2 rows in out flops of one layer's product."""
    R, Rv = cfg.rows, cfg.val_rows
    f = [0.0] * len(KERNEL_CLASSES)
    adam = cfg.optimizer == W.OPT_ADAM
    for l in range(cfg.n_layers):
        u = 2.0 * cfg.widths[l] * cfg.widths[l + 1]
        f[0] += (T * R + Rv) * u                         # forward (unroll + validation)
        f[2] += (T * R + Rv) * u                         # backward-weight (update / seed)
        if l > 0:
            f[1] += (T * R + Rv) * u                     # backward-data
            f[4] += T * R * u * 3                        # dual backward-data
        f[3] += T * R * u * (3 if l > 0 else 2)          # dual forward
        if adam:                                         # tangent products only
            f[5] += T * R * u * (2 if l > 0 else 1)
        elif l > 0:                                      # G and G' = H v, three products
            f[8] += T * R * u * 3
        else:                                            # layer 0: A' = 0, two products
            f[5] += T * R * u * 2
    return f


def desc_of(cfg: W.Config):
    from paper_2505_00793_amd import _lib as M
    return M.make_desc(widths=cfg.widths, act=cfg.act, loss=cfg.loss, optimizer=cfg.optimizer,
                       meta=cfg.meta, precision=cfg.precision, has_bias=cfg.has_bias,
                       rows=cfg.rows, val_rows=cfg.val_rows, sgd_lr=cfg.sgd_lr,
                       adam_b1=cfg.adam_b1, adam_b2=cfg.adam_b2, adam_eps=cfg.adam_eps)


def cpu_baseline(cfg: W.Config, inp: dict, T: int):
    """The float64 oracle on the host cores, on a bounded sample of the workload:
    one forward inner step, the validation seed and one reverse step of the
    step-checkpointed oracle at full size, extrapolated to T steps."""
    import torch
    import oracle
    from oracle.metagrad import _Inputs, reverse_step, seed
    one = dict(inp)
    one["train_x"], one["train_y"] = inp["train_x"][:1], inp["train_y"][:1]
    I = _Inputs(cfg, one)
    t0 = time.perf_counter()
    th1, _, _, _ = oracle.inner_step(cfg, inp["theta0"], None, inp["eta"], inp["train_x"][0],
                                     inp["train_y"][0], 0)
    t1 = time.perf_counter()
    th1 = torch.from_numpy(th1)
    V, thbar = seed(cfg, I, th1, False)
    t2 = time.perf_counter()
    reverse_step(cfg, I, 0, I.theta0, None, thbar, None, False)
    t3 = time.perf_counter()
    per = T * ((t1 - t0) + (t3 - t2)) + (t2 - t1)
    return {"value": 1.0 / per, "unit": "meta-gradients/s", "cores": torch.get_num_threads(),
            "kind": "oracle",
            "sample": (f"float64 reverse-over-reverse oracle at full size: one inner step "
                       f"({t1 - t0:.2f} s), the validation seed ({t2 - t1:.2f} s) and one "
                       f"reverse step ({t3 - t2:.2f} s), extrapolated to T={T}: "
                       f"{per:.1f} s per meta-gradient")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--T", type=int, default=8)
    ap.add_argument("--sweep-steps", type=int, default=3,
                    help="timed calls per T of the memory sweep (0 = sizes only)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="first run a plain device copy of this many bytes (a known-size "
                         "reference for hardware traffic counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the meta-gradient path is single-device "
              f"(--gpus {args.gpus} is not supported)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2505_00793_amd import _lib as M

    if args.copy_bytes > 0:
        src = torch.ones(args.copy_bytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        torch.cuda.empty_cache()

    cfg = W.C5.with_(T=args.T)
    T = args.T
    Tmax = max([T] + list(W.C5_TS))
    log(f"[bench] generating inputs (T up to {Tmax})")
    inp = W.make_inputs(cfg, T=Tmax)
    dev = torch.device("cuda")

    def up(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    theta0, eta = up(inp["theta0"]), up(inp["eta"])
    xs = [up(x) for x in inp["train_x"]]
    ys = [up(y) for y in inp["train_y"]]
    vx, vy = up(inp["val_x"]), up(inp["val_y"])
    P = M.Problem(desc_of(cfg))
    n_eta = W.n_eta(cfg)
    d_eta = torch.empty(n_eta, device=dev)
    vloss = torch.empty(1, device=dev)
    sizes = P.mfmg_query_sizes(T)
    ws = P.workspace(sizes.workspace_bytes)
    stream = torch.cuda.current_stream()

    def call(Tc, wsc):
        return P.mfmg_meta_grad(theta0, None, eta, xs[:Tc], ys[:Tc], vx, vy, d_eta, vloss, ws=wsc)

    log(f"[bench] warmup {args.warmup}")
    for _ in range(args.warmup):
        peak = call(T, ws)
    torch.cuda.synchronize()
    M.mfmg_timing_enable(True)
    for c in range(len(KERNEL_CLASSES)):
        M.mfmg_timing_read(c)
    log(f"[bench] timing {args.steps} meta-gradients at T={T}")
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        peak = call(T, ws)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    M.mfmg_timing_enable(False)
    ms = start.elapsed_time(stop) / args.steps
    kern = {}
    flops = algorithmic_flops(cfg, T)
    for c, name in enumerate(KERNEL_CLASSES):
        n, tot = M.mfmg_timing_read(c)
        if n:
            kern[name] = {"launches_per_step": n / args.steps, "ms_per_step": tot / args.steps,
                          "tflops": (flops[c] * args.steps / (tot * 1e-3) / 1e12) if flops[c] else None}
    log(f"[bench] {ms:.2f} ms per meta-gradient (wall {wall / args.steps * 1e3:.2f} ms)")
    dom = max((k for k in kern if kern[k]["tflops"]), key=lambda k: kern[k]["ms_per_step"])
    achieved = kern[dom]["tflops"]
    c = KERNEL_CLASSES.index(dom)
    per_launch = flops[c] / kern[dom]["launches_per_step"]
    roof = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2),
            "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": None, "gflop_per_launch": round(per_launch / 1e9, 3),
            "us_per_launch": round(kern[dom]["ms_per_step"] / kern[dom]["launches_per_step"] * 1e3, 2)}
    finite = bool(torch.isfinite(d_eta).all().item())

    sweep = {}
    for Ts in W.C5_TS:
        s = P.mfmg_query_sizes(Ts)
        entry = {"peak_bytes": None, "static_bytes": s.static_bytes, "dynamic_bytes": s.dynamic_bytes,
                 "workspace_bytes": s.workspace_bytes}
        if args.sweep_steps > 0:
            log(f"[bench] sweep T={Ts}")
            wss = ws if s.workspace_bytes <= ws.numel() else P.workspace(s.workspace_bytes)
            entry["peak_bytes"] = call(Ts, wss)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(args.sweep_steps):
                call(Ts, wss)
            e1.record(stream)
            torch.cuda.synchronize()
            entry["ms_per_meta_grad"] = round(e0.elapsed_time(e1) / args.sweep_steps, 3)
            entry["meta_grads_per_s"] = round(1e3 / entry["ms_per_meta_grad"], 3)
            if wss is not ws:
                del wss
                torch.cuda.empty_cache()
        sweep[str(Ts)] = entry

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (float64 oracle sample)")
        cpu = cpu_baseline(cfg, inp, T)

    out = {
        "metric": "meta-gradients/sec + peak HBM bytes vs T on 1 MI355X; MFMA util of HVP GEMMs",
        "value": round(1e3 / ms, 4), "unit": "meta-gradients/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded Gaussian inputs, uniform labels)",
        "config": {"workload": ("MLP 4096-(4096x7)-1000 ReLU, CE, batch 1024, SGD with "
                                "per-parameter log learning rates, bf16 GEMM operands"),
                   "T": T, "rows": cfg.rows, "n_theta": W.n_theta(cfg), "n_eta": n_eta,
                   "parallelism": "single GPU"},
        "peak_bytes": peak, "static_bytes": sizes.static_bytes,
        "dynamic_bytes": sizes.dynamic_bytes, "memory_vs_T": sweep,
        "roofline": roof, "kernels": kern, "cpu_baseline": cpu, "d_eta_finite": finite,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
