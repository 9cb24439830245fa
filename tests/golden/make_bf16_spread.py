"""Writes tests/golden/bf16_spread.json: how far bf16 operand rounding alone moves
the meta-gradient on the full-size bf16 workloads, and how far float32 GEMM
accumulation alone moves it on the full-size workloads gated in float32.

For each case the oracle computes dV/deta twice with bf16-rounded GEMM
operands, once accumulating the rounded products in float64 and once in
float32: two equally valid bf16 implementations.  Their normwise relative
distance (per eta group) is the noise floor a bf16 GPU result is compared
against; the distance of each to the unrounded float64 result is recorded
alongside.  Calls only oracle/ and workloads/.

    python tests/golden/make_bf16_spread.py [--only=NAME ...] [--T=T ...] [--fp32-only]
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import torch  # noqa: E402

import oracle  # noqa: E402
import workloads as W  # noqa: E402
from oracle.metagrad import working_precision  # noqa: E402

CASES = [("c5_mlp_relu_8x4096", 2), ("c5_mlp_relu_8x4096", 4), ("c5_mlp_relu_8x4096", 8),
         ("c3_mlp_gelu_adam", 16), ("c4_transformer_tokenweights", 2),
         ("c4_transformer_tokenweights", 8), ("c5_slice2", 2), ("c5_slice2", 8),
         ("c5_slice3", 2), ("c5_slice3", 8)]
FP32_CASES = [("c3_mlp_gelu_adam", 16)]


def groups(cfg):
    """The eta groups of the parity gates: each per-layer lr and the decay of
    Adam separately, each meta-model tensor separately, else all of eta."""
    n = W.n_eta(cfg)
    if cfg.meta == W.META_LOGLR_PER_LAYER_WD:
        return [[i] for i in range(n)]
    if cfg.meta == W.META_TOKEN_WEIGHT_MLP:
        return [list(range(off, off + int(np.prod(shape)))) for _, off, shape in W.meta_layout(cfg)]
    return [list(range(n))]


def rel(a, b, g):
    a, b = a[g], b[g]
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def main():
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "bf16_spread.json")
    only_fp32 = "--fp32-only" in sys.argv
    only = [a.split("=", 1)[1] for a in sys.argv if a.startswith("--only=")]
    only_T = [int(a.split("=", 1)[1]) for a in sys.argv if a.startswith("--T=")]
    out = json.load(open(path)) if (only_fp32 or only or only_T) and os.path.exists(path) else {"note": ("normwise relative distances per eta group between the oracle's bf16-operand "
                    "emulations accumulated in float64 ('emu64') and in float32 ('emu32'), and "
                    "each to the unrounded float64 oracle ('fp64'); '/fp32' entries: float32 "
                    "GEMMs ('fp32') and the whole oracle in float32 ('fp32all') against float64")}
    todo = [c for c in CASES if (not only or c[0] in only) and (not only_T or c[1] in only_T)]
    for name, T in ([] if only_fp32 else todo):
        cfg = W.get(name).with_(T=T)
        inp = W.make_inputs(cfg, T=T)
        d64, _ = oracle.meta_grad_checkpointed(cfg, inp)
        e64, _ = oracle.meta_grad_checkpointed(cfg, inp, bf16=True)
        e32, _ = oracle.meta_grad_checkpointed(cfg, inp, bf16="acc32")
        gs = groups(cfg)
        out[f"{name}/T{T}"] = {
            "emu32_vs_emu64": [rel(e32, e64, g) for g in gs],
            "emu64_vs_fp64": [rel(e64, d64, g) for g in gs],
            "emu32_vs_fp64": [rel(e32, d64, g) for g in gs],
        }
        print(name, T, out[f"{name}/T{T}"], flush=True)
        with open(path, "w") as f:   # keep what is done if a later case is interrupted
            json.dump(out, f, indent=1)
    for name, T in ([] if only else FP32_CASES):
        cfg = W.get(name).with_(T=T, precision=W.PREC_FP32)
        inp = W.make_inputs(cfg, T=T)
        d64, _ = oracle.meta_grad_checkpointed(cfg, inp)
        f32, _ = oracle.meta_grad_checkpointed(cfg, inp, bf16="fp32")
        with working_precision(torch.float32):
            a32, _ = oracle.meta_grad_checkpointed(cfg, inp)
        out[f"{name}/T{T}/fp32"] = {"fp32_vs_fp64": [rel(f32, d64, g) for g in groups(cfg)],
                                    "fp32all_vs_fp64": [rel(a32, d64, g) for g in groups(cfg)]}
        print(name, T, "fp32", out[f"{name}/T{T}/fp32"], flush=True)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
