"""Oracle building blocks: float64 tensor ops with optional bf16 operand rounding.

Test infrastructure only (see oracle/__init__.py).

The rounding emulation models a GPU that feeds bfloat16 operands to its
matrix units and accumulates in float32 or wider: each operand of a matrix
product is rounded f64 -> f32 -> bf16 (round-to-nearest-even), the product
is taken in float64.  Rounding is the identity for differentiation.  The
backward of a rounded product is again a rounded product, so gradients (and
gradients of gradients) round their GEMM operands at the same places.
"""
from __future__ import annotations

import math

import torch

F64 = torch.float64


def bf16_round(x: torch.Tensor) -> torch.Tensor:
    """Value of x rounded to bfloat16 (RNE), returned as float64, no gradient."""
    return x.detach().to(torch.float32).to(torch.bfloat16).to(F64)


class _RoundST(torch.autograd.Function):
    """Straight-through rounding: forward rounds to bf16, backward is identity."""

    @staticmethod
    def forward(ctx, x):
        return bf16_round(x)

    @staticmethod
    def backward(ctx, g):
        return g


def round_st(x: torch.Tensor, bf16: bool) -> torch.Tensor:
    return _RoundST.apply(x) if bf16 else x


class _RoundedMM(torch.autograd.Function):
    """C = round(A) @ round(B) for matrices; its VJP is built from the same op."""

    @staticmethod
    def forward(ctx, a, b):
        ctx.save_for_backward(a, b)
        return bf16_round(a) @ bf16_round(b)

    @staticmethod
    def backward(ctx, g):
        a, b = ctx.saved_tensors
        ga = _RoundedMM.apply(g, b.transpose(-2, -1)) if ctx.needs_input_grad[0] else None
        gb = _RoundedMM.apply(a.transpose(-2, -1), g) if ctx.needs_input_grad[1] else None
        return ga, gb


class _RoundedMM32(torch.autograd.Function):
    """As _RoundedMM, but the product of the rounded operands is accumulated in
    float32 (a second, equally valid bf16-operand implementation; the spread
    between the two measures how far rounding alone moves a result)."""

    @staticmethod
    def forward(ctx, a, b):
        ctx.save_for_backward(a, b)
        return (bf16_round(a).float() @ bf16_round(b).float()).to(F64)

    @staticmethod
    def backward(ctx, g):
        a, b = ctx.saved_tensors
        ga = _RoundedMM32.apply(g, b.transpose(-2, -1)) if ctx.needs_input_grad[0] else None
        gb = _RoundedMM32.apply(a.transpose(-2, -1), g) if ctx.needs_input_grad[1] else None
        return ga, gb


class _RoundedBMM(torch.autograd.Function):
    """Batched version: leading dims equal on both sides."""

    @staticmethod
    def forward(ctx, a, b):
        ctx.save_for_backward(a, b)
        return torch.matmul(bf16_round(a), bf16_round(b))

    @staticmethod
    def backward(ctx, g):
        a, b = ctx.saved_tensors
        ga = _RoundedBMM.apply(g, b.transpose(-2, -1)) if ctx.needs_input_grad[0] else None
        gb = _RoundedBMM.apply(a.transpose(-2, -1), g) if ctx.needs_input_grad[1] else None
        return ga, gb


class _MM32(torch.autograd.Function):
    """Float32 product of the (unrounded) operands; its VJP uses the same op.  A
    float32-GEMM implementation of the same method, for measuring how far
    float32 accumulation alone moves a result."""

    @staticmethod
    def forward(ctx, a, b):
        ctx.save_for_backward(a, b)
        return (a.float() @ b.float()).to(F64)

    @staticmethod
    def backward(ctx, g):
        a, b = ctx.saved_tensors
        ga = _MM32.apply(g, b.transpose(-2, -1)) if ctx.needs_input_grad[0] else None
        gb = _MM32.apply(a.transpose(-2, -1), g) if ctx.needs_input_grad[1] else None
        return ga, gb


def mm(a: torch.Tensor, b: torch.Tensor, bf16) -> torch.Tensor:
    """2-D matrix product.  ``bf16``: False = float64; True = bf16 operands;
    "acc32" = bf16 operands with float32 accumulation; "fp32" = float32
    operands and accumulation."""
    if bf16 == "acc32":
        return _RoundedMM32.apply(a, b)
    if bf16 == "fp32":
        return _MM32.apply(a, b)
    return _RoundedMM.apply(a, b) if bf16 else a @ b


def bmm(a: torch.Tensor, b: torch.Tensor, bf16: bool) -> torch.Tensor:
    """Batched matrix product over equal leading dimensions."""
    return _RoundedBMM.apply(a, b) if bf16 else torch.matmul(a, b)


class _BiasAdd(torch.autograd.Function):
    """z + b (b broadcast over rows); the bias gradient sums the *rounded*
    row gradients, as a GPU does when it reduces its bf16 copy of dZ."""

    @staticmethod
    def forward(ctx, z, b):
        return z + b

    @staticmethod
    def backward(ctx, g):
        return g, _RoundST.apply(g).sum(0)


def bias_add(z: torch.Tensor, b: torch.Tensor, bf16) -> torch.Tensor:
    return _BiasAdd.apply(z, b) if (bf16 and bf16 != "fp32") else z + b


def gelu(z: torch.Tensor) -> torch.Tensor:
    """Exact (erf) GELU: z * Phi(z)."""
    return 0.5 * z * (1.0 + torch.erf(z / math.sqrt(2.0)))


def activation(z: torch.Tensor, act: int) -> torch.Tensor:
    from workloads import ACT_GELU, ACT_NONE, ACT_RELU, ACT_TANH
    if act == ACT_TANH:
        return torch.tanh(z)
    if act == ACT_GELU:
        return gelu(z)
    if act == ACT_RELU:
        return torch.relu(z)
    if act == ACT_NONE:
        return z
    raise ValueError(act)


def cross_entropy_rows(z: torch.Tensor, y: torch.Tensor) -> torch.Tensor:
    """Per-row softmax cross-entropy l_n = logsumexp(z_n) - z_{n, y_n}."""
    return torch.logsumexp(z, dim=-1) - z.gather(-1, y.long().unsqueeze(-1)).squeeze(-1)


def layer_norm(x: torch.Tensor, g: torch.Tensor, b: torch.Tensor, eps: float) -> torch.Tensor:
    mu = x.mean(-1, keepdim=True)
    var = ((x - mu) ** 2).mean(-1, keepdim=True)
    return (x - mu) / torch.sqrt(var + eps) * g + b
