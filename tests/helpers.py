"""Shared test helpers: workload config -> ABI description, device upload, error metrics."""
from __future__ import annotations

import json
import os

import numpy as np

import workloads as W

FP32_TOL = 1e-4   # float32 GEMM operands
BF16_TOL = 2e-2   # bfloat16 GEMM operands, against the oracle's bf16-emulation mode


def desc_of(cfg: W.Config):
    from paper_2505_00793_amd import _lib as M
    if cfg.kind == W.KIND_TRANSFORMER:
        return M.make_desc(kind=1, widths=(1, 1), loss=cfg.loss, optimizer=cfg.optimizer,
                           meta=cfg.meta, precision=cfg.precision, has_bias=False,
                           rows=cfg.rows, val_rows=cfg.val_rows, sgd_lr=cfg.sgd_lr,
                           d_model=cfg.d_model, n_heads=cfg.n_heads, d_ff=cfg.d_ff,
                           vocab=cfg.vocab, seq=cfg.seq, n_blocks=cfg.n_blocks,
                           meta_hidden=cfg.meta_hidden, ln_eps=cfg.ln_eps,
                           rope_base=cfg.rope_base, fused_attention=cfg.fused_attention,
                           block_remat=cfg.block_remat)
    return M.make_desc(widths=cfg.widths, act=cfg.act, loss=cfg.loss, optimizer=cfg.optimizer,
                       meta=cfg.meta, precision=cfg.precision, has_bias=cfg.has_bias,
                       rows=cfg.rows, val_rows=cfg.val_rows, sgd_lr=cfg.sgd_lr,
                       adam_b1=cfg.adam_b1, adam_b2=cfg.adam_b2, adam_eps=cfg.adam_eps,
                       map_steps=cfg.map_steps, ckpt_segment=cfg.ckpt_segment)


def tol_of(cfg: W.Config) -> float:
    return BF16_TOL if cfg.precision == W.PREC_BF16 else FP32_TOL


def relerr(a, b) -> float:
    a = np.asarray(a, dtype=np.float64).ravel()
    b = np.asarray(b, dtype=np.float64).ravel()
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def eta_groups(cfg: W.Config):
    """Index groups over which the normwise error of d eta is taken: each
    per-layer log-lr and the weight decay separately; each meta-model tensor;
    otherwise all of eta."""
    n = W.n_eta(cfg)
    if cfg.meta == W.META_LOGLR_PER_LAYER_WD:
        return [np.array([i]) for i in range(n)]
    if cfg.meta == W.META_TOKEN_WEIGHT_MLP:
        return [np.arange(off, off + int(np.prod(shape))) for _, off, shape in W.meta_layout(cfg)]
    return [np.arange(n)]


def group_errors(cfg, got, ref):
    return [relerr(np.asarray(got)[g], np.asarray(ref)[g]) for g in eta_groups(cfg)]


def to_device(inp: dict, device="cuda"):
    import torch

    def t(a):
        return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(device)

    return {
        "theta0": t(inp["theta0"]), "eta": t(inp["eta"]), "opt_state0": t(inp["opt_state0"]),
        "xs": [t(x) for x in inp["train_x"]], "ys": [t(y) for y in inp["train_y"]],
        "vx": t(inp["val_x"]), "vy": t(inp["val_y"]),
    }


def spread_of(key):
    """Per-eta-group distance between the oracle's float32- and
    float64-accumulated bf16 emulations, stored by tests/golden/make_bf16_spread.py."""
    with open(os.path.join(os.path.dirname(__file__), "golden", "bf16_spread.json")) as f:
        return json.load(f)[key]["emu32_vs_emu64"]
