"""Independent numpy implementation of the MLP inner loop, for pinning the oracle.

Hand-written forward and backward passes (no autodiff library), written so
that every operation is complex-analytic: transposes are plain transposes,
never conjugates, so that complex-step differentiation dV/deta_k =
Im V(eta + i h e_k) / h is exact to rounding.  ReLU masks use the real part.

It implements: MLP (tanh, erf-GELU, ReLU, identity), softmax cross-entropy
and squared error heads with per-row loss weights, SGD with per-parameter
log learning rates, SGD with a fixed rate and per-example weight logits, Adam
with per-layer log learning rates and decoupled weight decay.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

import workloads as W


def _unpack(cfg, flat):
    P = {}
    for name, off, shape in W.theta_layout(cfg):
        size = int(np.prod(shape))
        P[name] = flat[off:off + size].reshape(shape)
    return P


def _act(z, act):
    if act == W.ACT_TANH:
        return np.tanh(z)
    if act == W.ACT_GELU:
        return 0.5 * z * (1.0 + erf(z / math.sqrt(2.0)))
    if act == W.ACT_RELU:
        return np.where(z.real > 0, z, 0.0)
    return z


def _dact(z, act):
    if act == W.ACT_TANH:
        t = np.tanh(z)
        return 1.0 - t * t
    if act == W.ACT_GELU:
        return 0.5 * (1.0 + erf(z / math.sqrt(2.0))) + z * np.exp(-0.5 * z * z) / math.sqrt(2 * math.pi)
    if act == W.ACT_RELU:
        return (z.real > 0).astype(np.float64)
    return np.ones_like(z)


def loss_and_grad(cfg, theta, x, y, alpha=None):
    """(L, dL/dtheta) with L = (1/N) sum_n alpha_n l_n."""
    P = _unpack(cfg, theta)
    L = cfg.n_layers
    N = x.shape[0]
    a = x
    acts, zs = [x], []
    for l in range(L):
        z = a @ P[f"W{l}"]
        if cfg.has_bias:
            z = z + P[f"b{l}"]
        zs.append(z)
        a = _act(z, cfg.act) if l < L - 1 else z
        acts.append(a)
    out = a
    al = np.ones(N) if alpha is None else alpha
    if cfg.loss == W.LOSS_CE:
        m = out.real.max(axis=1, keepdims=True)
        e = np.exp(out - m)
        s = e.sum(axis=1, keepdims=True)
        lse = (m + np.log(s))[:, 0]
        ln = lse - out[np.arange(N), y]
        dout = e / s
        dout[np.arange(N), y] -= 1.0
    elif cfg.loss == W.LOSS_MAPMSE:
        # forward through the map keeping each step's input, then the chain rule
        # back through d/dy [i (2 + sin y)^cos y] = y_i (cos^2 y / (2 + sin y) - sin y ln(2 + sin y))
        ys = [out]
        for i in range(1, cfg.map_steps + 1):
            ys.append(i * (2.0 + np.sin(ys[-1])) ** np.cos(ys[-1]))
        r = ys[-1] - y.reshape(out.shape)
        D = out.shape[1]
        ln = (r * r).sum(axis=1) / D
        dout = 2.0 * r / D
        for i in range(cfg.map_steps, 0, -1):
            yp = ys[i - 1]
            s, c = np.sin(yp), np.cos(yp)
            dout = dout * ys[i] * (c * c / (2.0 + s) - s * np.log(2.0 + s))
    else:
        r = out - y.reshape(out.shape)
        ln = (r * r).sum(axis=1)
        dout = 2.0 * r
    loss = (al * ln).sum() / N
    dz = dout * (al / N)[:, None]
    grads = {}
    for l in reversed(range(L)):
        grads[f"W{l}"] = acts[l].T @ dz
        if cfg.has_bias:
            grads[f"b{l}"] = dz.sum(axis=0)
        if l > 0:
            dz = (dz @ P[f"W{l}"].T) * _dact(zs[l - 1], cfg.act)
    g = np.concatenate([grads[name].reshape(-1) for name, _, _ in W.theta_layout(cfg)])
    return loss, g


def per_example_grads(cfg, theta, x, y):
    """Rows of grad l_n(theta), n = 0..N-1 (one backward per example)."""
    N = x.shape[0]
    rows = []
    for n in range(N):
        _, g = loss_and_grad(cfg, theta, x[n:n + 1], y[n:n + 1])
        rows.append(g)
    return np.stack(rows)


def _layer_index(cfg):
    return np.concatenate([np.full(int(np.prod(shape)), int(name[1:]))
                           for name, _, shape in W.theta_layout(cfg)])


def val_loss(cfg, inp, eta):
    """V(eta): T inner updates then the unweighted validation loss (any dtype)."""
    if cfg.meta == W.META_MAML:   # eta is the starting point theta_0
        theta = eta.reshape(-1).astype(np.result_type(eta.dtype, np.float64)).copy()
    else:
        theta = inp["theta0"].astype(np.float64) + 0 * eta.reshape(-1)[0]
    n = theta.size
    m = np.zeros(n, dtype=theta.dtype)
    v = np.zeros(n, dtype=theta.dtype)
    T = len(inp["train_x"])
    for i in range(T):
        x = inp["train_x"][i].astype(np.float64)
        y = inp["train_y"][i]
        if y.dtype.kind == "f":
            y = y.astype(np.float64)
        alpha = None
        if cfg.meta == W.META_EXAMPLE_WEIGHT_LOGITS:
            alpha = 1.0 / (1.0 + np.exp(-eta.reshape(cfg.T, cfg.rows)[i]))
        _, g = loss_and_grad(cfg, theta, x, y, alpha)
        if cfg.optimizer == W.OPT_SGD:
            if cfg.meta == W.META_LOGLR_PER_PARAM:
                theta = theta - np.exp(eta) * g
            else:
                theta = theta - cfg.sgd_lr * g
        else:
            t = i + 1
            b1, b2 = cfg.adam_b1, cfg.adam_b2
            m = b1 * m + (1 - b1) * g
            v = b2 * v + (1 - b2) * g * g
            u = (m / (1 - b1 ** t)) / (np.sqrt(v / (1 - b2 ** t)) + cfg.adam_eps)
            lr = np.exp(eta[:cfg.n_layers])[_layer_index(cfg)]
            theta = theta - lr * (u + eta[cfg.n_layers] * theta)
    vy = inp["val_y"]
    if vy.dtype.kind == "f":
        vy = vy.astype(np.float64)
    V, _ = loss_and_grad(cfg, theta, inp["val_x"].astype(np.float64), vy)
    return V


def complex_step_meta_grad(cfg, inp, h=1e-30):
    """dV/deta_k = Im V(eta + i h e_k) / h for every k."""
    eta = inp["eta"].astype(np.float64)
    out = np.zeros(eta.size)
    for k in range(eta.size):
        e = eta.astype(np.complex128)
        e[k] += 1j * h
        out[k] = val_loss(cfg, inp, e).imag / h
    return out
