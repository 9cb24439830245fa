"""Oracle inner/outer losses and meta-parameter maps (float64, CPU).

Test infrastructure only (see oracle/__init__.py).

Inner loss L(theta, eta, x) and outer loss V(theta, y) of the bilevel problem
(Section 2.1, eq. bilevel_opt_problem).  How eta enters follows the three
tasks of Section 5.2: learned (per-parameter or per-layer) learning rates
enter only the update; adaptive loss weighting multiplies each example's (or
token's) loss by alpha(eta, x): L = (1/N) sum_n alpha_n l_n.
"""
from __future__ import annotations

import math
from typing import Dict, Optional

import torch

from workloads import (Config, KIND_MLP, KIND_TRANSFORMER, LOSS_CE, LOSS_MAPMSE, LOSS_MSE,
                       META_EXAMPLE_WEIGHT_LOGITS, META_TOKEN_WEIGHT_MLP, ACT_NONE,
                       theta_layout, meta_layout)

from .ops import (activation, bias_add, bmm, cross_entropy_rows, gelu, layer_norm, mm)


def unpack(flat: torch.Tensor, layout) -> Dict[str, torch.Tensor]:
    """Views of the named tensors inside a flat parameter vector."""
    out = {}
    for name, off, shape in layout:
        size = 1
        for s in shape:
            size *= s
        out[name] = flat[off:off + size].view(*shape) if shape else flat[off]
    return out


# ---------------------------------------------------------------------------------------
# MLP (linear regression is the one-layer, no-bias, identity-activation case)
# ---------------------------------------------------------------------------------------
def mlp_outputs(cfg: Config, theta: torch.Tensor, x: torch.Tensor, bf16: bool) -> torch.Tensor:
    P = unpack(theta, theta_layout(cfg))
    a = x
    L = cfg.n_layers
    for l in range(L):
        z = mm(a, P[f"W{l}"], bf16)
        if cfg.has_bias:
            z = bias_add(z, P[f"b{l}"], bf16)
        a = activation(z, cfg.act) if l < L - 1 else z
    return a


def per_example_loss(cfg: Config, out: torch.Tensor, y: torch.Tensor) -> torch.Tensor:
    if cfg.loss == LOSS_CE:
        return cross_entropy_rows(out, y)
    if cfg.loss == LOSS_MSE:
        return ((out - y.reshape(out.shape)) ** 2).sum(-1)
    if cfg.loss == LOSS_MAPMSE:
        return ((toy_map(out, cfg.map_steps) - y.reshape(out.shape)) ** 2).mean(-1)
    raise ValueError(cfg.loss)


def toy_map(y: torch.Tensor, M: int) -> torch.Tensor:
    """The M-step recursive map of Section 3.2 (eq. motivational_example),
    elementwise: y_i = i * (2 + sin y_{i-1}) ** cos y_{i-1}, i = 1..M."""
    for i in range(1, M + 1):
        y = i * (2.0 + torch.sin(y)) ** torch.cos(y)
    return y


# ---------------------------------------------------------------------------------------
# Decoder-only pre-LN transformer with RoPE (Section 5: Chinchilla-style models)
# ---------------------------------------------------------------------------------------
def rope_tables(S: int, dh: int, base: float):
    j = torch.arange(dh // 2, dtype=torch.float64)
    freq = base ** (-2.0 * j / dh)
    ang = torch.arange(S, dtype=torch.float64)[:, None] * freq[None, :]
    cos = torch.cat([torch.cos(ang), torch.cos(ang)], -1)
    sin = torch.cat([torch.sin(ang), torch.sin(ang)], -1)
    return cos, sin


def apply_rope(q: torch.Tensor, cos: torch.Tensor, sin: torch.Tensor) -> torch.Tensor:
    h = q.shape[-1] // 2
    rot = torch.cat([-q[..., h:], q[..., :h]], -1)
    return q * cos + rot * sin


def transformer_logits(cfg: Config, theta: torch.Tensor, tokens: torch.Tensor,
                       bf16: bool) -> torch.Tensor:
    """Logits (B*S, V) for input tokens (B, S)."""
    P = unpack(theta, theta_layout(cfg))
    B, S = tokens.shape
    d, H = cfg.d_model, cfg.n_heads
    dh = d // H
    cos, sin = rope_tables(S, dh, cfg.rope_base)
    causal = torch.tril(torch.ones(S, S, dtype=torch.bool))
    h = P["emb"][tokens.long()]                                   # (B, S, d)
    for b in range(cfg.n_blocks):
        a = layer_norm(h, P[f"ln1_g{b}"], P[f"ln1_b{b}"], cfg.ln_eps)
        qkv = mm(a.reshape(B * S, d), P[f"wqkv{b}"], bf16).reshape(B, S, 3, H, dh)
        q = apply_rope(qkv[:, :, 0].transpose(1, 2), cos, sin)    # (B, H, S, dh)
        k = apply_rope(qkv[:, :, 1].transpose(1, 2), cos, sin)
        v = qkv[:, :, 2].transpose(1, 2)
        s = bmm(q, k.transpose(-2, -1), bf16) / math.sqrt(dh)
        s = s.masked_fill(~causal, float("-inf"))
        p = torch.softmax(s, dim=-1)
        o = bmm(p, v, bf16).transpose(1, 2).reshape(B * S, d)
        h = h + mm(o, P[f"wo{b}"], bf16).reshape(B, S, d)
        a2 = layer_norm(h, P[f"ln2_g{b}"], P[f"ln2_b{b}"], cfg.ln_eps)
        f = gelu(mm(a2.reshape(B * S, d), P[f"w1{b}"], bf16))
        h = h + mm(f, P[f"w2{b}"], bf16).reshape(B, S, d)
    hf = layer_norm(h, P["lnf_g"], P["lnf_b"], cfg.ln_eps)
    return mm(hf.reshape(B * S, d), P["unemb"], bf16)


def split_tokens(tokens: torch.Tensor):
    """Next-token prediction: inputs are positions 0..S-1, targets 1..S."""
    return tokens[:, :-1], tokens[:, 1:].reshape(-1)


# ---------------------------------------------------------------------------------------
# Losses
# ---------------------------------------------------------------------------------------
def per_row_losses(cfg: Config, theta: torch.Tensor, x: torch.Tensor, y, bf16: bool):
    if cfg.kind == KIND_MLP:
        return per_example_loss(cfg, mlp_outputs(cfg, theta, x, bf16), y)
    xin, tgt = split_tokens(x)
    return cross_entropy_rows(transformer_logits(cfg, theta, xin, bf16), tgt)


def inner_loss(cfg: Config, theta: torch.Tensor, alpha: Optional[torch.Tensor], x, y,
               bf16: bool) -> torch.Tensor:
    """L = (1/N) sum_n alpha_n l_n (alpha = 1 when eta does not weight the loss)."""
    l = per_row_losses(cfg, theta, x, y, bf16)
    if alpha is not None:
        l = alpha.reshape(l.shape) * l
    return l.sum() / l.numel()


def outer_loss(cfg: Config, theta: torch.Tensor, x, y, bf16: bool) -> torch.Tensor:
    """V: unweighted mean loss on the validation batch."""
    return inner_loss(cfg, theta, None, x, y, bf16)


def meta_mlp_alpha(cfg: Config, eta: torch.Tensor, e: torch.Tensor) -> torch.Tensor:
    """alpha = sigmoid(tanh(e W1 + b1) w2 + b2) per token; e is constant data."""
    M = unpack(eta, meta_layout(cfg))
    hdn = torch.tanh(e @ M["mW1"] + M["mb1"])
    return torch.sigmoid(hdn @ M["mw2"] + M["mb2"]).squeeze(-1)


def alpha_of(cfg: Config, eta: torch.Tensor, step: int, x, emb0: Optional[torch.Tensor]):
    """Loss weights of inner step ``step`` (None = all ones)."""
    if cfg.meta == META_EXAMPLE_WEIGHT_LOGITS:
        return torch.sigmoid(eta.view(cfg.T, cfg.rows)[step])
    if cfg.meta == META_TOKEN_WEIGHT_MLP:
        xin, _ = split_tokens(x)
        return meta_mlp_alpha(cfg, eta, emb0[xin.long()]).reshape(-1)
    return None
