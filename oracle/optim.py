"""Oracle inner update Upsilon (float64, CPU).

Test infrastructure only (see oracle/__init__.py).

Upsilon(g, theta, upsilon, eta) takes the inner gradient as an explicit
argument (Section 3, eq. reparam).  Three update rules:

* SGD with per-parameter learning rates exp(eta) (hyperparameter learning,
  Section 5.2): theta' = theta - exp(eta) * g.
* SGD with a fixed learning rate (loss-weighting task, Section 5.2):
  theta' = theta - lr * g.
* Adam (Section 5 uses Adam as the inner optimiser) with bias correction and
  decoupled weight decay, per-layer learning rates exp(eta_l) and a raw decay
  coefficient omega = eta[-1]:
  m' = b1 m + (1-b1) g;  v' = b2 v + (1-b2) g^2;
  u = (m'/(1-b1^t)) / (sqrt(v'/(1-b2^t)) + eps), t = step + 1;
  theta' = theta - lr_l (u + omega theta).
"""
from __future__ import annotations

import torch

from workloads import (Config, META_LOGLR_PER_LAYER_WD, META_LOGLR_PER_PARAM, OPT_ADAM,
                       OPT_SGD, theta_layout)


def layer_index(cfg: Config) -> torch.Tensor:
    """For each theta entry, the index of the MLP layer it belongs to."""
    idx = []
    for name, off, shape in theta_layout(cfg):
        size = 1
        for s in shape:
            size *= s
        idx.append(torch.full((size,), int(name[1:]), dtype=torch.long))
    return torch.cat(idx)


def upsilon(cfg: Config, g: torch.Tensor, theta: torch.Tensor, opt, eta: torch.Tensor,
            step: int):
    """One inner update; returns (theta', opt') with opt None for stateless SGD."""
    if cfg.optimizer == OPT_SGD:
        if cfg.meta == META_LOGLR_PER_PARAM:
            return theta - torch.exp(eta) * g, None
        return theta - cfg.sgd_lr * g, None
    if cfg.optimizer == OPT_ADAM:
        if cfg.meta != META_LOGLR_PER_LAYER_WD:
            raise ValueError("Adam workloads learn per-layer log-lr + weight decay")
        n = theta.numel()
        m, v = opt[:n], opt[n:]
        t = step + 1
        b1, b2 = cfg.adam_b1, cfg.adam_b2
        m1 = b1 * m + (1.0 - b1) * g
        v1 = b2 * v + (1.0 - b2) * g * g
        mhat = m1 / (1.0 - b1 ** t)
        vhat = v1 / (1.0 - b2 ** t)
        u = mhat / (torch.sqrt(vhat) + cfg.adam_eps)
        L = cfg.n_layers
        lr = torch.exp(eta[:L])[layer_index(cfg)]
        omega = eta[L]
        return theta - lr * (u + omega * theta), torch.cat([m1, v1])
    raise ValueError(cfg.optimizer)
