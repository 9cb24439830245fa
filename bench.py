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
runs on) and one whole float64 CPU oracle meta-gradient, timed on the host.
"""
from __future__ import annotations

import argparse
import math
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


def algorithmic_bytes(cfg: W.Config, T: int):
    """HBM bytes per kernel class per meta-gradient that the method must move
    with this design (SGD with per-parameter log learning rates; bf16 operands
    in both layouts, float32 parameter streams): every operand tile read once,
    every output written once, no re-reads.  None for classes not modelled."""
    if cfg.optimizer != W.OPT_SGD or cfg.meta != W.META_LOGLR_PER_PARAM:
        return [None] * len(KERNEL_CLASSES)
    R, Rv, L = cfg.rows, cfg.val_rows, cfg.n_layers
    b = [0.0] * len(KERNEL_CLASSES)
    for l in range(L):
        i, o = cfg.widths[l], cfg.widths[l + 1]
        P = i * o
        last = l == L - 1
        for rows in [R] * T + [Rv]:
            # forward: A and W^T read; z (float32) written, and for hidden layers
            # the next operand in both bf16 layouts
            b[0] += 2 * rows * i + 2 * P + 4 * rows * o + (0 if last else 4 * rows * o)
            if l > 0:   # backward-data: dZ, W, z_{l-1} read; dZ_{l-1} written in both layouts
                b[1] += 2 * rows * o + 2 * P + 4 * rows * i + 4 * rows * i
        # backward-weight with the update (T steps): A^T, dZ^T read; theta, eta
        # read, theta' written, new operands W, W^T written
        b[2] += T * (2 * R * i + 2 * R * o + 16 * P)
        # validation seed: theta-bar written, eta read, tangent W, W^T written
        b[2] += 2 * Rv * i + 2 * Rv * o + 12 * P
        for t in range(T):
            first, last_rev = t == 0, t == T - 1      # reverse order: first = step T-1
            # dual forward: A, A' (not layer 0), W^T, W'^T read; z, z' written,
            # hidden layers write both operands in both layouts
            b[3] += (2 if l == 0 else 4) * R * i + 4 * P + 8 * R * o + (0 if last else 8 * R * o)
            if l > 0:   # dual backward-data: dZ, dZ', W, W', z, z' read; outputs in both layouts
                b[4] += 4 * R * o + 4 * P + 8 * R * i + 8 * R * i
            # dual backward-weight with the reverse epilogue: operands read once;
            # theta-bar read and written, eta read, eta-bar read (not on the first
            # reverse step) and written, next tangent W, W^T (not after the last)
            par = (8 + 4 + (0 if first else 4) + 4 + (0 if last_rev else 4)) * P
            ops = 2 * R * o * 2 + (2 if l == 0 else 4) * R * i
            b[5 if l == 0 else 8] += par + ops
    # loss head, per pass of `rows` rows over C classes: logits read (float32),
    # labels read, the output gradient written as bf16 operands in both layouts,
    # per-row losses written; dual passes also read the logit tangents and write
    # the gradient's tangent in both layouts
    C = cfg.widths[-1]
    for rows, dual in [(R, False)] * T + [(Rv, False)] + [(R, True)] * T:
        b[6] += rows * C * (16 if dual else 8) + rows * 8
    # other elementwise kernels: theta_0 to its operand copies once (float32 read,
    # bf16 W and W^T written); every pass converts its input rows (float32 read,
    # bf16 rows in both layouts); every pass's bias reductions read dZ^T (and its
    # tangent) in bf16 and touch the bias streams (~24 bytes per bias)
    n_w = sum(cfg.widths[l] * cfg.widths[l + 1] for l in range(L))
    n_b = sum(cfg.widths[1:]) if cfg.has_bias else 0
    b[7] += 8 * (n_w + n_b)
    for rows, dual in [(R, False)] * T + [(Rv, False)] + [(R, True)] * T:
        b[7] += rows * cfg.widths[0] * 8
        if cfg.has_bias:
            b[7] += sum(rows * o * (4 if dual else 2) for o in cfg.widths[1:]) + 24 * n_b
    return b


# Kernel instantiation that makes up each kernel class in the c5 run (bf16,
# 128 x 128 tiles on the direct-to-LDS path), for matching counter records.
# (Regular expressions over the kernel name: flags, tile and epilogue; any k depth and stages.)
CLASS_KERNEL = {
    "dual_bwd_weight_gemm_reverse": r"gemm_nt_ws<7, 128, 128, \d+, \d+, mfmg::\(anonymous namespace\)::ParamOp",
    "bwd_weight_gemm_update": r"gemm_nt_ws<1, 128, 128, \d+, \d+, mfmg::\(anonymous namespace\)::ParamOp",
    "dual_fwd_gemm": r"gemm_nt_ws<7, 128, 128, \d+, \d+, mfmg::\(anonymous namespace\)::ActFwdOp",
    "dual_bwd_data_gemm": r"gemm_nt_ws<7, 128, 128, \d+, \d+, mfmg::\(anonymous namespace\)::ActBwdOp",
}
KERNEL_SOURCES = ["paper_2505_00793_amd/csrc/gemm.hip", "paper_2505_00793_amd/csrc/param_epi.h",
                  "paper_2505_00793_amd/csrc/kernels.h", "paper_2505_00793_amd/csrc/common.h"]


def counters_file(cls: str) -> str:
    return os.path.join(ROOT, "profiles", f"{cls}_c5_mlp8x4096_T8_hbm_counters.md")


def kernel_sources_sha() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(cls: str):
    """HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE summary of
    this kernel class, or None if there is none or the kernel sources changed
    since the counters were taken."""
    path = counters_file(cls)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    i = text.find("```json")
    if i < 0:
        return None
    rec = json.loads(text[i + 7:text.index("```", i + 7)])
    if rec.get("kernel_sources_sha256") != kernel_sources_sha():
        return None
    return rec["hbm_bytes_per_launch"]


def pmc_summary(fetch_csv: str, write_csv: str, copy_bytes: int, cls: str, command: str):
    """Turns two rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE, KiB per
    dispatch) of `bench.py --copy-bytes N` into per-launch HBM bytes of one
    kernel class, each counter scaled by what it reads for the plain N-byte copy."""
    import csv
    import re

    def load(path, counter):
        per = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            per.setdefault(r["Dispatch_Id"], [r["Kernel_Name"], 0.0])[1] += float(r["Counter_Value"])
        return list(per.values())

    out = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = load(path, counter)
        copies = sorted((v for n, v in rows if "copyBuffer" in n), reverse=True)[:3]
        factor = (copy_bytes / 1024.0) / (sum(copies) / len(copies))
        ks = [v for n, v in rows if re.search(CLASS_KERNEL[cls], n)]
        names = sorted({n for n, _ in rows if re.search(CLASS_KERNEL[cls], n)})
        if not ks:
            raise SystemExit(f"no dispatch of {cls} ({CLASS_KERNEL[cls]}) in {path}")
        out[counter] = {"copy_kib_per_dispatch": round(sum(copies) / len(copies), 1),
                        "scale": round(factor, 4), "dispatches": len(ks),
                        "kib_per_dispatch": round(sum(ks) / len(ks), 1),
                        "bytes_per_launch": sum(ks) / len(ks) * 1024.0 * factor}
    kname = re.sub(r"^void |\(mfmg::GemmOperands.*$", "", names[0])
    rec = {"kernel_class": cls, "kernel": kname, "copy_bytes": copy_bytes,
           "fetch": out["FETCH_SIZE"], "write": out["WRITE_SIZE"],
           "hbm_bytes_per_launch": round(out["FETCH_SIZE"]["bytes_per_launch"]
                                         + out["WRITE_SIZE"]["bytes_per_launch"]),
           "kernel_sources_sha256": kernel_sources_sha()}
    cfg = W.C5
    T = 8
    alg = algorithmic_bytes(cfg, T)[KERNEL_CLASSES.index(cls)]
    launches = {"dual_bwd_weight_gemm_reverse": T * (cfg.n_layers - 1)}.get(cls)
    body = [f"# HBM traffic counters: `{cls}` (MLP 4096-(4096x7)-1000, batch 1024, T=8, bf16)",
            "", "Commands (repository root, one MI355X), one counter per pass:", "", "```",
            command, "```", "",
            f"Each counter is scaled by its reading for a plain device copy of {copy_bytes} bytes "
            f"(`__amd_rocclr_copyBuffer`, which reads and writes exactly that many bytes), then "
            f"averaged over the {out['FETCH_SIZE']['dispatches']} dispatches of "
            f"`{kname}`.", "",
            "| counter | copy reads (KiB) | scale | kernel (KiB/dispatch) | bytes per launch |",
            "|---|---:|---:|---:|---:|"]
    for counter in ("FETCH_SIZE", "WRITE_SIZE"):
        o = out[counter]
        body.append(f"| {counter} | {o['copy_kib_per_dispatch']} | {o['scale']} | "
                    f"{o['kib_per_dispatch']} | {o['bytes_per_launch'] / 1e6:.1f} MB |")
    if alg and launches:
        body += ["", f"Algorithmic bytes per launch (bench.py `algorithmic_bytes`): "
                 f"{alg / launches / 1e6:.1f} MB; measured / algorithmic = "
                 f"{rec['hbm_bytes_per_launch'] / (alg / launches):.3f}."]
    body += ["", "bench.py reads the record below for `roofline.traffic` while the kernel "
             "sources hash to the same value.", "", "```json", json.dumps(rec, indent=1), "```", ""]
    path = counters_file(cls)
    with open(path, "w") as f:
        f.write("\n".join(body))
    print(path)


def pmc_mfma_summary(csv_path: str, out_name: str, command: str):
    """Per-kernel MFMA counters from one rocprofv3 --pmc run of MfmaUtil (matrix-core
    busy cycles over the dispatch's active cycles, all SIMDs) and MfmaFlopsBF16 /
    MfmaFlopsF32 (512 x the MFMA ops the hardware counted): a markdown table per
    kernel instantiation, written under profiles/."""
    import csv
    import re
    per = {}
    for r in csv.DictReader(open(csv_path)):
        key = (r["Dispatch_Id"], r["Kernel_Name"])
        d = per.setdefault(key, {})
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        if r.get("Start_Timestamp") and r.get("End_Timestamp"):
            d["_ns"] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    kern = {}
    for (_, name), d in per.items():
        k = kern.setdefault(name, {"n": 0, "util": 0.0, "flops": 0.0, "ns": 0.0})
        k["n"] += 1
        k["util"] += d.get("MfmaUtil", 0.0)
        k["flops"] += d.get("MfmaFlopsBF16", 0.0) + d.get("MfmaFlopsF32", 0.0)
        k["ns"] += d.get("_ns", 0.0)
    rows = sorted(((n, k) for n, k in kern.items() if k["flops"] > 0),
                  key=lambda nk: -nk[1]["ns"])
    body = [f"# MFMA counters per GEMM kernel: {out_name}", "",
            "Command (repository root, one MI355X):", "", "```", command, "```", "",
            "`MfmaUtil` = matrix-core busy cycles summed over all SIMDs / (active cycles of the "
            "dispatch x SIMDs), in %; `MFMA GFLOP` = 512 x the MFMA ops counted "
            "(`SQ_INSTS_VALU_MFMA_MOPS_*`), per dispatch; the duration is the dispatch's own "
            "timestamps under counter collection (kernels serialised).", "",
            "| kernel | dispatches | MfmaUtil % | MFMA GFLOP / dispatch | us / dispatch | TFLOP/s |",
            "|---|---:|---:|---:|---:|---:|"]
    for name, k in rows:
        short = re.sub(r"^void |\(mfmg::GemmOperands.*$|mfmg::\(anonymous namespace\)::", "", name)
        short = short.replace("unsigned short", "bf16")[:110]
        us = k["ns"] / k["n"] / 1e3 if k["ns"] else float("nan")
        gf = k["flops"] / k["n"] / 1e9
        tf = gf / us * 1e3 if k["ns"] else float("nan")   # GFLOP per us = PFLOP/s
        body.append(f"| `{short}` | {k['n']} | {k['util'] / k['n']:.1f} | {gf:.2f} | {us:.1f} | "
                    f"{tf:.0f} |")
    path = os.path.join(ROOT, "profiles", f"gemm_mfma_counters_{out_name}.md")
    with open(path, "w") as f:
        f.write("\n".join(body) + "\n")
    print(path)


def pmc_traffic_summary(fetch_csv: str, write_csv: str, copy_bytes: int, regex: str, label: str,
                        command: str):
    """HBM bytes per dispatch of every kernel whose name matches `regex`, from two
    rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE) made with --copy-bytes, each
    counter scaled by its reading for the plain copy; written to
    profiles/LABEL_hbm_counters.md."""
    import csv
    import re

    def load(path, counter):
        per = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            per.setdefault(r["Dispatch_Id"], [r["Kernel_Name"], 0.0])[1] += float(r["Counter_Value"])
        return list(per.values())

    stats = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = load(path, counter)
        copies = sorted((v for n, v in rows if "copyBuffer" in n), reverse=True)[:3]
        factor = (copy_bytes / 1024.0) / (sum(copies) / len(copies))
        for n, v in rows:
            if re.search(regex, n):
                k = stats.setdefault(n, {}).setdefault(counter, [0, 0.0, factor])
                k[0] += 1
                k[1] += v
    body = [f"# HBM traffic counters: {label}", "", "Commands (repository root, one MI355X), "
            "one counter per pass:", "", "```", command, "```", "",
            f"Each counter is scaled by its reading for a plain device copy of {copy_bytes} "
            "bytes (`__amd_rocclr_copyBuffer`, which reads and writes exactly that many bytes) "
            "and averaged over the kernel's dispatches.", "",
            "| kernel | dispatches | FETCH (KB / dispatch) | WRITE (KB / dispatch) |",
            "|---|---:|---:|---:|"]
    for name, c in sorted(stats.items()):
        short = re.sub(r"^void |mfmg::\(anonymous namespace\)::|\(mfmg::.*$|\(.*$", "", name)
        f = c.get("FETCH_SIZE", [1, 0.0, 1.0])
        w = c.get("WRITE_SIZE", [1, 0.0, 1.0])
        body.append(f"| `{short[:100]}` | {f[0]} | {f[1] / f[0] * 1.024 * f[2]:.1f} | "
                    f"{w[1] / w[0] * 1.024 * w[2]:.1f} |")
    path = os.path.join(ROOT, "profiles", f"{label}_hbm_counters.md")
    with open(path, "w") as fh:
        fh.write("\n".join(body) + "\n")
    print(path)


def trace_summary(stats_csv: str, label: str, title: str, command: str, top: int = 25):
    """profiles/LABEL_kernel_trace.md from rocprofv3's run_kernel_stats.csv: the
    kernels by total time, with calls and average duration."""
    import csv
    import re
    rows = list(csv.DictReader(open(stats_csv)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    body = [f"# Kernel trace: {title}", "", "Command (repository root, one MI355X):", "", "```",
            command, "```", "", "The table is `run_kernel_stats.csv` of that run.", "",
            "| kernel | calls | avg (us) | total (ms) | % |", "|---|---:|---:|---:|---:|"]
    for r in rows[:top]:
        name = re.sub(r"^void |mfmg::\(anonymous namespace\)::|\(mfmg::.*$|\(.*$", "",
                      r["Name"])
        name = name.replace("unsigned short", "bf16")
        body.append(f"| `{name[:110]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                    f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.1f} |")
    path = os.path.join(ROOT, "profiles", f"{label}_kernel_trace.md")
    with open(path, "w") as fh:
        fh.write("\n".join(body) + "\n")
    print(path)


def desc_of(cfg: W.Config):
    from paper_2505_00793_amd import _lib as M
    if cfg.kind == W.KIND_TRANSFORMER:
        return M.make_desc(kind=1, widths=(1, 1), loss=cfg.loss, optimizer=cfg.optimizer,
                           meta=cfg.meta, precision=cfg.precision, has_bias=False,
                           rows=cfg.rows, val_rows=cfg.val_rows, sgd_lr=cfg.sgd_lr,
                           d_model=cfg.d_model, n_heads=cfg.n_heads, d_ff=cfg.d_ff,
                           vocab=cfg.vocab, seq=cfg.seq, n_blocks=cfg.n_blocks,
                           meta_hidden=cfg.meta_hidden, ln_eps=cfg.ln_eps, rope_base=cfg.rope_base,
                           fused_attention=cfg.fused_attention, block_remat=cfg.block_remat)
    return M.make_desc(widths=cfg.widths, act=cfg.act, loss=cfg.loss, optimizer=cfg.optimizer,
                       meta=cfg.meta, precision=cfg.precision, has_bias=cfg.has_bias,
                       rows=cfg.rows, val_rows=cfg.val_rows, sgd_lr=cfg.sgd_lr,
                       adam_b1=cfg.adam_b1, adam_b2=cfg.adam_b2, adam_eps=cfg.adam_eps,
                       map_steps=cfg.map_steps, ckpt_segment=cfg.ckpt_segment)


def cpu_model() -> str:
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_meta_grad_logged(cfg: W.Config, inp: dict):
    """oracle.meta_grad_checkpointed, step by step through the oracle's own
    functions, logging each step (a whole float64 meta-gradient of the large
    workloads takes minutes on the host)."""
    import torch
    from oracle.metagrad import _Inputs, reverse_step, seed, unroll
    I = _Inputs(cfg, inp)
    thetas, opts, _, _ = unroll(cfg, inp)
    log(f"[bench]   oracle: forward unroll of {I.T} steps done")
    V, thbar = seed(cfg, I, thetas[-1], False)
    obar = None if opts[-1] is None else torch.zeros_like(opts[-1])
    etabar = torch.zeros_like(I.eta)
    for i in reversed(range(I.T)):
        thbar, obar, d = reverse_step(cfg, I, i, thetas[i], opts[i], thbar, obar, False)
        etabar = etabar + d
        log(f"[bench]   oracle: reverse step {i} done")
    if cfg.meta == W.META_MAML:
        etabar = etabar + thbar
    return etabar.numpy(), float(V.detach())


def cpu_baseline(cfg: W.Config, inp: dict, runs: int = 1):
    """The float64 reverse-over-reverse oracle (step-checkpointed) on the host
    cores: `runs` whole meta-gradients of the workload, timed; 1 / median."""
    import torch
    times = []
    for _ in range(runs):
        t0 = time.perf_counter()
        oracle_meta_grad_logged(cfg, inp)
        times.append(time.perf_counter() - t0)
    med = sorted(times)[len(times) // 2]
    return {"value": 1.0 / med, "unit": "meta-gradients/s", "cores": torch.get_num_threads(),
            "kind": "oracle", "measured": True, "cpu": cpu_model(),
            "sample": (f"{runs} whole float64 oracle meta-gradient(s) at T={len(inp['train_x'])} "
                       f"(reverse-over-reverse, one inner step's graph at a time): "
                       f"{', '.join(f'{t:.2f}' for t in times)} s")}


WORKLOADS = {
    "c1_linreg": "linear regression 64 features, 256 rows, per-parameter log learning rates, fp32",
    "c2_mlp_tanh_lossweights": ("MLP 784-256-10 tanh, CE, 128 rows, SGD lr 0.1, per-example loss "
                                "weights, fp32"),
    "c3_mlp_gelu_adam": ("MLP 1024-(1024x3)-100 GELU, CE, 512 rows, Adam with per-layer log "
                         "learning rates and weight decay, bf16 GEMM operands"),
    "c4_transformer_tokenweights": ("decoder 4 blocks d 512, 8 heads, FF 2048, vocab 8192, RoPE, "
                                    "16x256 tokens, SGD lr 0.1, per-token loss weights from a "
                                    "512-128-1 meta-model, bf16 GEMM operands"),
    "maml_mlp_relu_8x4096": ("MLP 4096-(4096x7)-1000 ReLU, CE, batch 1024, T=8, MAML (eta = "
                             "theta_0), SGD lr 0.05, bf16 GEMM operands"),
    "c4_long_context": ("decoder 4 blocks d 512, 8 heads, FF 2048, vocab 8192, 8192 tokens per "
                        "batch as S x 8192/S sequences for S = 2048, 4096, 8192, T=2, per-token "
                        "loss weights, bf16 GEMM operands"),
    "toy_mstep_map": ("motivating example: y_0 = x w (1024 x 4096, w 4096 x 4096), M map steps "
                      "y_i = i (2 + sin y)^cos y, mean squared error, MAML, T=2, SGD lr 1e-3, "
                      "fp32"),
}
BENCH_CONFIGS = {**W.CONFIGS, W.MAML5.name: W.MAML5, W.TOY.name: W.TOY,
                 "c4_long_context": W.C4}


def c4_long(S: int) -> W.Config:
    return W.C4.with_(name=f"c4_S{S}", seq=S, rows=8192 // S, val_rows=8192 // S, T=2)


def with_attention(cfg: W.Config, form: str) -> W.Config:
    """A transformer workload with fused or materialised attention."""
    if cfg.kind != W.KIND_TRANSFORMER:
        return cfg
    return cfg.with_(fused_attention=int(form == "fused"))


def bench_config(name: str, args):
    """meta-gradients/s of one of the other workloads at its own T, same timing
    protocol as the main line (inputs resident, warm-up calls, HIP-event timing
    on the stream); no roofline, sweep or CPU baseline."""
    import torch
    from paper_2505_00793_amd import _lib as M
    cfg = with_attention(BENCH_CONFIGS[name], args.attention)
    if cfg.kind == W.KIND_TRANSFORMER:
        cfg = cfg.with_(block_remat=args.block_remat)
    ms, peak, finite = time_config(cfg, args)
    sizes = M.Problem(desc_of(cfg)).mfmg_query_sizes(cfg.T)
    extra = {"static_bytes": sizes.static_bytes, "dynamic_bytes": sizes.dynamic_bytes}
    if cfg.kind == W.KIND_TRANSFORMER:
        # the other block-rematerialisation setting, for its time and memory
        other = cfg.with_(block_remat=1 - cfg.block_remat)
        ms2, peak2, _ = time_config(other, args)
        s2 = M.Problem(desc_of(other)).mfmg_query_sizes(cfg.T)
        extra["block_remat"] = cfg.block_remat
        extra["vs_block_remat"] = {
            str(c.block_remat): {"ms_per_meta_grad": round(m, 4), "peak_bytes": pk,
                                 "static_bytes": z.static_bytes, "dynamic_bytes": z.dynamic_bytes}
            for c, m, pk, z in ((cfg, ms, peak, sizes), (other, ms2, peak2, s2))}
    cpu = None
    if not args.no_cpu_baseline and torch.cuda.is_available():
        inp = W.make_inputs(cfg)
        # three whole float64 oracle meta-gradients of the small workloads, one of
        # the large ones (about a minute on 16 host cores)
        runs = 3 if name in ("c1_linreg", "c2_mlp_tanh_lossweights", "c3_mlp_gelu_adam") else 1
        log(f"[bench] {name}: cpu baseline, {runs} whole float64 oracle meta-gradient(s)")
        cpu = cpu_baseline(cfg, inp, runs=runs)
    print(json.dumps({
        "metric": "meta-gradients/sec on 1 MI355X", "value": round(1e3 / ms, 4),
        "unit": "meta-gradients/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if cfg.precision == W.PREC_BF16 else "f32",
        "data": "synthetic (seeded, see workloads/)",
        "config": {"workload": WORKLOADS[name], "name": name, "T": cfg.T,
                   **({"attention": args.attention} if cfg.kind == W.KIND_TRANSFORMER else {})},
        "peak_bytes": peak, **extra, "roofline": None, "cpu_baseline": cpu,
        "d_eta_finite": finite,
        **({"graph_replay": {"ms_per_step": round(args.graph_ms, 4),
                             "meta_grads_per_s": round(1e3 / args.graph_ms, 4)}}
           if args.graph_ms else {})}))


def bench_toy(args):
    """The motivating example of Section 3.2 (B = 1024, D = 4096, T = 2, MAML) over
    the number of map steps M: time and peak device bytes per meta-gradient.
    The map's derivatives are carried in registers, so memory does not grow with
    M.  The map's derivative grows roughly like M!, so in float32 the meta-gradient
    itself overflows for the larger M (from M = 16 at this size); d_eta_finite
    records it per M."""
    rows = {}
    for m in W.TOY_MS:
        ms, peak, finite = time_config(W.TOY.with_(map_steps=m), args)
        rows[str(m)] = {"ms_per_meta_grad": round(ms, 4), "peak_bytes": peak,
                        "d_eta_finite": finite}
    ref = rows[str(W.TOY.map_steps)]
    print(json.dumps({
        "metric": "meta-gradients/sec on 1 MI355X",
        "value": round(1e3 / ref["ms_per_meta_grad"], 4),
        "unit": "meta-gradients/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ref["ms_per_meta_grad"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic (seeded, see workloads/)",
        "config": {"workload": WORKLOADS[W.TOY.name], "name": W.TOY.name, "T": W.TOY.T,
                   "M": W.TOY.map_steps},
        "vs_M": rows, "roofline": None, "cpu_baseline": None}))


def bench_long_context(args):
    """The config-4 decoder at long contexts: time and peak device bytes per
    meta-gradient for each S in C4_LONG_S (8192 tokens per batch, T = 2), with
    fused and with materialised attention; `value` is the --attention form at the
    longest S."""
    rows = {}
    seqs = (args.seq,) if args.seq else W.C4_LONG_S
    forms = (args.attention,) if args.seq else ("fused", "materialised")
    for S in seqs:
        rows[str(S)] = {}
        for form in forms:
            ms, peak, finite = time_config(with_attention(c4_long(S), form), args)
            rows[str(S)][form] = {"ms_per_meta_grad": round(ms, 4), "peak_bytes": peak,
                                  "d_eta_finite": finite}
    ref = rows[str(seqs[-1])][args.attention]
    print(json.dumps({
        "metric": "meta-gradients/sec on 1 MI355X",
        "value": round(1e3 / ref["ms_per_meta_grad"], 4),
        "unit": "meta-gradients/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ref["ms_per_meta_grad"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded, see workloads/)",
        "config": {"workload": WORKLOADS["c4_long_context"], "name": "c4_long_context", "T": 2,
                   "S": seqs[-1], "attention": args.attention},
        "vs_S": rows, "roofline": None, "cpu_baseline": None}))


def time_config(cfg: W.Config, args):
    """(ms per meta-gradient, peak device bytes, dV/deta finite) for one workload."""
    import torch
    from paper_2505_00793_amd import _lib as M
    name = cfg.name
    T = cfg.T
    log(f"[bench] {name}: generating inputs (T={T})")
    inp = W.make_inputs(cfg)
    dev = torch.device("cuda")

    def up(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    theta0, eta = up(inp["theta0"]), up(inp["eta"])
    xs = [up(x) for x in inp["train_x"]]
    vx = up(inp["val_x"])
    if cfg.kind == W.KIND_TRANSFORMER:   # next-token targets come from the token rows
        dummy = torch.zeros(1, dtype=torch.int32, device=dev)
        ys, vy = [dummy] * T, dummy
    else:
        ys, vy = [up(y) for y in inp["train_y"]], up(inp["val_y"])
    P = M.Problem(desc_of(cfg))
    d_eta = torch.empty(W.n_eta(cfg), device=dev)
    vloss = torch.empty(1, device=dev)
    ws = P.workspace(P.mfmg_query_sizes(T).workspace_bytes)
    stream = torch.cuda.current_stream()

    def call():
        return P.mfmg_meta_grad(theta0, None, eta, xs, ys, vx, vy, d_eta, vloss, ws=ws)

    for _ in range(args.warmup):
        peak = call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        peak = call()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    tag = f" (M={cfg.map_steps})" if cfg.loss == W.LOSS_MAPMSE else ""
    log(f"[bench] {name}{tag}: {ms:.3f} ms per meta-gradient")
    args.graph_ms = None
    if getattr(args, "graph", False):
        # the same call recorded once in a HIP graph and replayed (no host launch
        # cost per kernel); replays are bit-identical to eager calls
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            call()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            call()
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        args.graph_ms = e0.elapsed_time(e1) / args.steps
        log(f"[bench] {name}{tag}: {args.graph_ms:.3f} ms per meta-gradient as a graph replay")
    return ms, peak, bool(torch.isfinite(d_eta).all().item())


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
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the HBM counter summary of --pmc-class from two rocprofv3 "
                         "--pmc runs (made with --copy-bytes) and exit; no GPU needed")
    ap.add_argument("--pmc-class", default="dual_bwd_weight_gemm_reverse")
    ap.add_argument("--trace-summary", nargs=3, metavar=("STATS_CSV", "LABEL", "TITLE"),
                    help="write profiles/LABEL_kernel_trace.md from rocprofv3's kernel stats "
                         "and exit; no GPU needed")
    ap.add_argument("--pmc-traffic-summary", nargs=4,
                    metavar=("FETCH_CSV", "WRITE_CSV", "REGEX", "LABEL"),
                    help="write profiles/LABEL_hbm_counters.md for the kernels matching REGEX "
                         "and exit; no GPU needed")
    ap.add_argument("--pmc-mfma-summary", nargs=2, metavar=("CSV", "NAME"),
                    help="write profiles/gemm_mfma_counters_NAME.md from a rocprofv3 --pmc run "
                         "of MfmaUtil and MfmaFlopsBF16 and exit; no GPU needed")
    ap.add_argument("--config", default="c5_mlp_relu_8x4096", choices=list(BENCH_CONFIGS),
                    help="workload; the default (c5) line carries the roofline, the memory "
                         "sweep and the CPU baseline, the others throughput only")
    ap.add_argument("--pmc-command", default="", help="the commands that made the CSVs")
    ap.add_argument("--attention", default="fused", choices=["fused", "materialised"],
                    help="attention form of the transformer workloads")
    ap.add_argument("--block-remat", type=int, default=1, choices=[0, 1],
                    help="transformer workloads: block rematerialisation (the line also "
                         "times the other setting)")
    ap.add_argument("--graph", action="store_true",
                    help="other workloads: also time graph replays of the same call")
    ap.add_argument("--seq", type=int, default=0, choices=[0, *W.C4_LONG_S],
                    help="c4_long_context: time this sequence length and --attention form only")
    args = ap.parse_args()
    if args.trace_summary:
        trace_summary(*args.trace_summary, command=args.pmc_command)
        return
    if args.pmc_traffic_summary:
        f_csv, w_csv, rx, label = args.pmc_traffic_summary
        pmc_traffic_summary(f_csv, w_csv, args.copy_bytes or (1 << 30), rx, label, args.pmc_command)
        return
    if args.pmc_mfma_summary:
        pmc_mfma_summary(args.pmc_mfma_summary[0], args.pmc_mfma_summary[1], args.pmc_command)
        return
    if args.pmc_summary:
        pmc_summary(args.pmc_summary[0], args.pmc_summary[1], args.copy_bytes or (1 << 30),
                    args.pmc_class, args.pmc_command)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the meta-gradient path is single-device "
              f"(--gpus {args.gpus} is not supported)", file=sys.stderr)
        sys.exit(2)
    if args.config == W.TOY.name:
        bench_toy(args)
        return
    if args.config == "c4_long_context":
        bench_long_context(args)
        return
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

    if args.config != W.C5.name:
        bench_config(args.config, args)
        return

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
    log(f"[bench] timing {args.steps} meta-gradients at T={T}")
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        peak = call(T, ws)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(stop) / args.steps
    # Per-kernel durations: a second pass of the same calls with HIP events
    # recorded around every launch on the library's stream (the events cost a
    # few percent of a step, so the throughput above is timed without them).
    log(f"[bench] per-kernel HIP-event pass, {args.steps} meta-gradients")
    for c in range(len(KERNEL_CLASSES)):
        M.mfmg_timing_read(c)
    M.mfmg_timing_enable(True)
    for _ in range(args.steps):
        call(T, ws)
    torch.cuda.synchronize()
    M.mfmg_timing_enable(False)
    kern = {}
    flops = algorithmic_flops(cfg, T)
    for c, name in enumerate(KERNEL_CLASSES):
        n, tot = M.mfmg_timing_read(c)
        if n:
            kern[name] = {"launches_per_step": n / args.steps, "ms_per_step": tot / args.steps,
                          "tflops": (flops[c] * args.steps / (tot * 1e-3) / 1e12) if flops[c] else None}
    log(f"[bench] {ms:.2f} ms per meta-gradient (wall {wall / args.steps * 1e3:.2f} ms)")
    nbytes = algorithmic_bytes(cfg, T)
    for c, name in enumerate(KERNEL_CLASSES):
        if name in kern:
            k = kern[name]
            k["mfma_util"] = round(k["tflops"] / PEAK_BF16_TFLOPS, 4) if k["tflops"] else None
            k["gb_per_s"] = round(nbytes[c] / (k["ms_per_step"] * 1e-3) / 1e9, 1) if nbytes[c] else None
    dom = max((k for k in kern if kern[k]["tflops"]), key=lambda k: kern[k]["ms_per_step"])
    c = KERNEL_CLASSES.index(dom)
    launches = kern[dom]["launches_per_step"]
    us = kern[dom]["ms_per_step"] / launches * 1e3
    flop_launch = flops[c] / launches
    byte_launch = nbytes[c] / launches if nbytes[c] else None
    # the bound is whichever floor is higher: flops at the MFMA peak or bytes at the HBM peak
    t_mfma = flop_launch / (PEAK_BF16_TFLOPS * 1e12)
    t_hbm = byte_launch / (PEAK_HBM_GBS * 1e9) if byte_launch else 0.0
    if t_hbm > t_mfma:
        achieved = byte_launch / (us * 1e-6) / 1e9
        roof = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    else:
        achieved = flop_launch / (us * 1e-6) / 1e12
        roof = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4)}
    roof.update({"traffic": measured_traffic(dom), "algorithmic_bytes_per_launch": byte_launch,
                 "gflop_per_launch": round(flop_launch / 1e9, 3), "us_per_launch": round(us, 2),
                 "mfma_frac": round(flop_launch / (us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4),
                 "floor_us": {"mfma": round(t_mfma * 1e6, 2), "hbm": round(t_hbm * 1e6, 2)}})
    finite = bool(torch.isfinite(d_eta).all().item())

    def sweep_entry(Pq, Ts, label):
        s = Pq.mfmg_query_sizes(Ts)
        entry = {"peak_bytes": None, "static_bytes": s.static_bytes, "dynamic_bytes": s.dynamic_bytes,
                 "workspace_bytes": s.workspace_bytes}
        if args.sweep_steps > 0:
            log(f"[bench] sweep T={Ts}{label}")
            wss = ws if s.workspace_bytes <= ws.numel() else Pq.workspace(s.workspace_bytes)

            def callq():
                return Pq.mfmg_meta_grad(theta0, None, eta, xs[:Ts], ys[:Ts], vx, vy, d_eta, vloss,
                                         ws=wss)
            entry["peak_bytes"] = callq()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(args.sweep_steps):
                callq()
            e1.record(stream)
            torch.cuda.synchronize()
            entry["ms_per_meta_grad"] = round(e0.elapsed_time(e1) / args.sweep_steps, 3)
            entry["meta_grads_per_s"] = round(1e3 / entry["ms_per_meta_grad"], 3)
            if wss is not ws:
                del wss
                torch.cuda.empty_cache()
        return entry

    sweep = {str(Ts): sweep_entry(P, Ts, "") for Ts in W.C5_TS}
    # the same with segment checkpoints of length round(sqrt(T)) (static memory
    # ~ 2 sqrt(T) parameter copies instead of T + 1, bit-identical results)
    sweep_seg = {}
    for Ts in W.C5_TS:
        k = max(1, int(round(math.sqrt(Ts))))
        Pk = M.Problem(desc_of(cfg.with_(ckpt_segment=k)))
        sweep_seg[str(Ts)] = {"segment": k, **sweep_entry(Pk, Ts, f" segments of {k}")}
        del Pk

    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] cpu baseline: one whole float64 oracle meta-gradient at T={T}")
        one = dict(inp)
        one["train_x"], one["train_y"] = inp["train_x"][:T], inp["train_y"][:T]
        cpu = cpu_baseline(cfg, one, runs=1)
        log(f"[bench] cpu baseline: {1.0 / cpu['value']:.1f} s per meta-gradient")

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
        "memory_vs_T_segment_checkpoints": sweep_seg,
        "roofline": roof, "kernels": kern,
        "kernel_timing": "HIP events around each launch on the library stream, separate pass of the same calls",
        "cpu_baseline": cpu, "d_eta_finite": finite,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
