"""Oracle meta-gradient: Truncated-BPTT by reverse-over-reverse (Algorithm 1).

Test infrastructure only (see oracle/__init__.py).

``meta_grad`` is Algorithm 1 taken literally: ValLoss(eta, theta0, upsilon0,
{x_i}, val_x) runs T inner updates whose gradients are built with reverse
mode and kept in the graph (create_graph), then reverse mode over the whole
program gives dV/deta.  ``meta_grad_checkpointed`` computes the same quantity
one inner step at a time (per-inner-step gradient checkpointing, Section 4):
it stores (theta_i, upsilon_i), then for i = T-1..0 rebuilds step i's graph
and back-propagates <bar theta_{i+1}, theta_{i+1}> + <bar upsilon_{i+1},
upsilon_{i+1}> into (theta_i, upsilon_i, eta); this is the chain rule of
Section 3 (eq. dVdmeta seeds bar theta_T = dV/dtheta_T, bar upsilon_T = 0;
eq. bptt_recur is the one-step recurrence).
"""
from __future__ import annotations

from typing import List, Optional, Tuple

import numpy as np
import torch

from workloads import Config, KIND_TRANSFORMER, META_MAML, META_TOKEN_WEIGHT_MLP, theta_layout

from .models import alpha_of, inner_loss, outer_loss, unpack
from .optim import upsilon

F64 = torch.float64
_FLOAT = [F64]  # working precision of the oracle: float64 (float32 only to measure spreads)


class working_precision:
    """Context manager that runs the same oracle code in another float dtype.
    The oracle is float64; float32 runs measure how far float32 arithmetic
    alone moves a result (the noise floor a float32 GPU result is held to)."""

    def __init__(self, dtype):
        self.dtype = dtype

    def __enter__(self):
        _FLOAT.append(self.dtype)

    def __exit__(self, *exc):
        _FLOAT.pop()


def _t(a, dtype=None):
    if a is None:
        return None
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(dtype or _FLOAT[-1]) if t.dtype.is_floating_point else t.long()


class _Inputs:
    """inputs (numpy, as produced by workloads.make_inputs) as float64 tensors."""

    def __init__(self, cfg: Config, inputs: dict):
        self.cfg = cfg
        self.eta = _t(inputs["eta"])
        # MAML (the task list of Section 5.2, 'Sweeping over Bilevel Optimisation
        # Tasks'): the meta-parameters are the initial point theta_0
        self.theta0 = self.eta.clone() if cfg.meta == META_MAML else _t(inputs["theta0"])
        self.opt0 = _t(inputs.get("opt_state0"))
        self.xs = [_t(x) for x in inputs["train_x"]]
        self.ys = [_t(y) for y in inputs["train_y"]]
        self.vx = _t(inputs["val_x"])
        self.vy = _t(inputs["val_y"])
        self.T = len(self.xs)
        self.emb0 = None
        if cfg.meta == META_TOKEN_WEIGHT_MLP:
            self.emb0 = unpack(self.theta0, theta_layout(cfg))["emb"].detach().clone()


def val_loss_of_eta(cfg: Config, inputs: dict, eta: torch.Tensor, bf16: bool = False,
                    create_graph: bool = True) -> torch.Tensor:
    """ValLoss of Algorithm 1 as a differentiable function of eta."""
    I = _Inputs(cfg, inputs)
    theta = eta if cfg.meta == META_MAML else I.theta0.clone().requires_grad_(True)
    opt = I.opt0
    for i in range(I.T):
        alpha = alpha_of(cfg, eta, i, I.xs[i], I.emb0)
        L = inner_loss(cfg, theta, alpha, I.xs[i], I.ys[i], bf16)
        (g,) = torch.autograd.grad(L, theta, create_graph=create_graph)
        theta, opt = upsilon(cfg, g, theta, opt, eta, i)
    return outer_loss(cfg, theta, I.vx, I.vy, bf16)


def meta_grad(cfg: Config, inputs: dict, bf16: bool = False) -> Tuple[np.ndarray, float]:
    """(dV/deta, V) by reverse-over-reverse through the unrolled inner loop."""
    eta = _t(inputs["eta"]).requires_grad_(True)
    V = val_loss_of_eta(cfg, inputs, eta, bf16)
    (d_eta,) = torch.autograd.grad(V, eta)
    return d_eta.numpy(), float(V.detach())


def unroll(cfg: Config, inputs: dict, bf16: bool = False):
    """Forward unroll only: ([theta_0..theta_T], [opt_0..opt_T], [L_0..L_{T-1}], V)."""
    I = _Inputs(cfg, inputs)
    thetas, opts, losses = [I.theta0], [I.opt0], []
    for i in range(I.T):
        th = thetas[-1].detach().clone().requires_grad_(True)
        alpha = alpha_of(cfg, I.eta, i, I.xs[i], I.emb0)
        L = inner_loss(cfg, th, alpha, I.xs[i], I.ys[i], bf16)
        (g,) = torch.autograd.grad(L, th)
        with torch.no_grad():
            th1, op1 = upsilon(cfg, g, th.detach(), opts[-1], I.eta, i)
        thetas.append(th1)
        opts.append(op1)
        losses.append(float(L.detach()))
    with torch.no_grad():
        V = float(outer_loss(cfg, thetas[-1], I.vx, I.vy, bf16))
    return thetas, opts, losses, V


def reverse_step(cfg: Config, I: "_Inputs", i: int, theta_i, opt_i, thbar, obar, bf16: bool):
    """One step of the reverse sweep: rebuild inner step i from (theta_i, opt_i)
    and back-propagate <thbar, theta_{i+1}> + <obar, opt_{i+1}> into
    (theta_i, opt_i, eta).  Returns (bar theta_i, bar opt_i, d eta contribution)."""
    th = theta_i.clone().requires_grad_(True)
    op = None if opt_i is None else opt_i.clone().requires_grad_(True)
    et = I.eta.clone().requires_grad_(True)
    alpha = alpha_of(cfg, et, i, I.xs[i], I.emb0)
    L = inner_loss(cfg, th, alpha, I.xs[i], I.ys[i], bf16)
    (g,) = torch.autograd.grad(L, th, create_graph=True)
    th1, op1 = upsilon(cfg, g, th, op, et, i)
    s = (thbar * th1).sum()
    wrt = [th, et]
    if op is not None:
        s = s + (obar * op1).sum()
        wrt.append(op)
    grads = torch.autograd.grad(s, wrt, allow_unused=True)
    new_thbar = grads[0] if grads[0] is not None else torch.zeros_like(th)
    d_eta = grads[1] if grads[1] is not None else torch.zeros_like(et)
    new_obar = None
    if op is not None:
        new_obar = grads[2] if grads[2] is not None else torch.zeros_like(op)
    return new_thbar, new_obar, d_eta


def seed(cfg: Config, I: "_Inputs", theta_T, bf16: bool):
    """(V, dV/dtheta_T) at the end of the unroll."""
    thT = theta_T.clone().requires_grad_(True)
    V = outer_loss(cfg, thT, I.vx, I.vy, bf16)
    (thbar,) = torch.autograd.grad(V, thT)
    return V, thbar


def meta_grad_checkpointed(cfg: Config, inputs: dict, bf16: bool = False
                           ) -> Tuple[np.ndarray, float]:
    """Same quantity as ``meta_grad``, one inner step's graph at a time."""
    I = _Inputs(cfg, inputs)
    thetas, opts, _, _ = unroll(cfg, inputs, bf16)
    V, thbar = seed(cfg, I, thetas[-1], bf16)
    obar = None if opts[-1] is None else torch.zeros_like(opts[-1])
    etabar = torch.zeros_like(I.eta)
    for i in reversed(range(I.T)):
        thbar, obar, d = reverse_step(cfg, I, i, thetas[i], opts[i], thbar, obar, bf16)
        etabar = etabar + d
    if cfg.meta == META_MAML:   # theta_0 = eta: its adjoint is the rest of dV/deta
        etabar = etabar + thbar
    return etabar.double().numpy(), float(V.detach())


# ---------------------------------------------------------------------------------------
# Single-step quantities (the units the GPU entry points compute)
# ---------------------------------------------------------------------------------------
def _alpha_leaf(cfg: Config, alpha) -> Optional[torch.Tensor]:
    return None if alpha is None else _t(alpha).clone()


def grad_and_loss(cfg: Config, theta, x, y, alpha=None, bf16: bool = False):
    """(dL/dtheta, L) at theta on one batch (first order)."""
    th = _t(theta).clone().requires_grad_(True)
    L = inner_loss(cfg, th, _alpha_leaf(cfg, alpha), _t(x), _t(y), bf16)
    (g,) = torch.autograd.grad(L, th)
    return g.numpy(), float(L)


def inner_step(cfg: Config, theta, opt, eta, x, y, step: int, alpha=None, bf16: bool = False):
    """One inner update: (theta', opt', g, L)."""
    th = _t(theta).clone().requires_grad_(True)
    L = inner_loss(cfg, th, _alpha_leaf(cfg, alpha), _t(x), _t(y), bf16)
    (g,) = torch.autograd.grad(L, th)
    with torch.no_grad():
        th1, op1 = upsilon(cfg, g, th.detach(), _t(opt), _t(eta), step)
    return (th1.numpy(), None if op1 is None else op1.numpy(), g.numpy(), float(L))


def hvp_rev_rev(cfg: Config, theta, x, y, v, alpha=None, bf16: bool = False) -> np.ndarray:
    """H v = d/dtheta <dL/dtheta, v> (reverse-over-reverse, Section 2.2)."""
    th = _t(theta).clone().requires_grad_(True)
    L = inner_loss(cfg, th, _alpha_leaf(cfg, alpha), _t(x), _t(y), bf16)
    (g,) = torch.autograd.grad(L, th, create_graph=True)
    (hv,) = torch.autograd.grad((g * _t(v)).sum(), th)
    return hv.numpy()


def hvp_rev_fwd(cfg: Config, theta, x, y, v, alpha=None) -> Tuple[np.ndarray, np.ndarray]:
    """(H v, mixed product) by reverse-over-forward, the third mode of Section 2.2:
    the directional derivative <dL/dtheta, v> is formed in forward mode
    (torch.func.jvp of L along v) and then differentiated in reverse mode with
    respect to theta (giving H v) and to the per-row loss weights alpha (giving
    (d^2 L / d alpha d theta) v, one entry per loss row).  Unrounded operands
    only (float64)."""
    th = _t(theta).clone()
    xt, yt, vt = _t(x), _t(y), _t(v)
    n_rows = xt.shape[0] if cfg.kind != KIND_TRANSFORMER else xt.shape[0] * (xt.shape[1] - 1)
    a = torch.ones(n_rows, dtype=F64) if alpha is None else _t(alpha).clone()

    def directional(p, w):
        return torch.func.jvp(lambda q: inner_loss(cfg, q, w, xt, yt, False), (p,), (vt,))[1]

    hv, mv = torch.func.grad(directional, argnums=(0, 1))(th, a)
    return hv.numpy(), mv.numpy()


def mvp_rev_rev(cfg: Config, theta, x, y, v, alpha=None, bf16: bool = False) -> np.ndarray:
    """Mixed product (d^2 L / d alpha d theta) v, one entry per loss row.

    With L = (1/N) sum_n alpha_n l_n this is (1/N) <grad l_n, v> per row.
    """
    th = _t(theta).clone().requires_grad_(True)
    xt = _t(x)
    n_rows = xt.shape[0] if cfg.kind != KIND_TRANSFORMER else xt.shape[0] * (xt.shape[1] - 1)
    a = (torch.ones(n_rows, dtype=F64) if alpha is None else _t(alpha).clone()).requires_grad_(True)
    L = inner_loss(cfg, th, a, xt, _t(y), bf16)
    (g,) = torch.autograd.grad(L, th, create_graph=True)
    (m,) = torch.autograd.grad((g * _t(v)).sum(), a)
    return m.numpy()
