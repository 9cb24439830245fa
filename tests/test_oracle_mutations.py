"""Plant plausible mistakes in the oracle (CPU only) and check that a pin catches each.

Each case monkeypatches one oracle building block with a wrong variant (a
dropped term, a wrong sign, a wrong constant) and re-runs the pin that
should fail.  The pins themselves live in test_oracle_pins.py.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from oracle import models as OM
from oracle import ops as OPS
from oracle import optim as OO

import numpy_ref as R
from test_oracle_pins import TINY, linreg_closed_form, relerr, _transformer_logits_independent


def _complex_step_err(key):
    cfg = TINY[key]
    inp = W.make_inputs(cfg)
    return relerr(oracle.meta_grad(cfg, inp)[0], R.complex_step_meta_grad(cfg, inp))


def test_mutation_sgd_lr_without_exp(monkeypatch):
    orig = OO.upsilon

    def bad(cfg, g, theta, opt, eta, step):
        if cfg.optimizer == W.OPT_SGD and cfg.meta == W.META_LOGLR_PER_PARAM:
            return theta - eta * g, None
        return orig(cfg, g, theta, opt, eta, step)

    monkeypatch.setattr("oracle.metagrad.upsilon", bad)
    inp = W.make_inputs(W.C1)
    assert relerr(oracle.meta_grad(W.C1, inp)[0], linreg_closed_form(inp)) > 1e-3


def test_mutation_mse_half(monkeypatch):
    orig = OM.per_example_loss

    def bad(cfg, out, y):
        l = orig(cfg, out, y)
        return 0.5 * l if cfg.loss == W.LOSS_MSE else l

    monkeypatch.setattr(OM, "per_example_loss", bad)
    assert _complex_step_err("tanh_mse_pp") > 1e-3


def test_mutation_gelu_tanh_approximation(monkeypatch):
    def bad(z):
        return 0.5 * z * (1 + torch.tanh(math.sqrt(2 / math.pi) * (z + 0.044715 * z ** 3)))

    monkeypatch.setattr(OPS, "gelu", bad)
    assert _complex_step_err("gelu_ce_pp") > 1e-6


def test_mutation_loss_weights_normalised_by_sum(monkeypatch):
    def bad(cfg, theta, alpha, x, y, bf16):
        l = OM.per_row_losses(cfg, theta, x, y, bf16)
        if alpha is None:
            return l.mean()
        return (alpha * l).sum() / alpha.sum()

    monkeypatch.setattr("oracle.metagrad.inner_loss", bad)
    assert _complex_step_err("weights") > 1e-3


def test_mutation_adam_bias_correction_off_by_one():
    cfg = TINY["adam"]
    n = W.n_theta(cfg)
    g = torch.from_numpy(np.random.default_rng(0).standard_normal(n))
    th = torch.zeros(n, dtype=torch.float64)
    eta = torch.tensor([math.log(0.05)] * cfg.n_layers + [0.1], dtype=torch.float64)
    good, _ = OO.upsilon(cfg, g, th, torch.zeros(2 * n, dtype=torch.float64), eta, 0)
    bad, _ = OO.upsilon(cfg, g, th, torch.zeros(2 * n, dtype=torch.float64), eta, 1)
    # step 0 must equal AdamW's first step: theta - lr * g / (|g| + eps) (bias corrected)
    lr = math.exp(eta[0].item())
    first = -lr * g[:20] / (g[:20].abs() + cfg.adam_eps)
    assert torch.allclose(good[:20], first, rtol=1e-12)
    assert not torch.allclose(bad[:20], first, rtol=1e-3)


def test_mutation_rope_sign(monkeypatch):
    def bad(q, cos, sin):
        h = q.shape[-1] // 2
        rot = torch.cat([q[..., h:], -q[..., :h]], -1)
        return q * cos + rot * sin

    monkeypatch.setattr(OM, "apply_rope", bad)
    cfg = W.SMALL["c4_small"]
    inp = W.make_inputs(cfg)
    th = inp["theta0"]
    tok = inp["train_x"][0][:, :-1]
    ours = OM.transformer_logits(cfg, torch.from_numpy(th).double(), torch.from_numpy(tok), False)
    assert not torch.allclose(ours, _transformer_logits_independent(cfg, th, tok), rtol=1e-6)


def test_mutation_dropped_second_order_term(monkeypatch):
    """Detaching the inner gradient (first-order meta-gradient) drops the HVP term."""
    orig_grad = torch.autograd.grad

    def first_order(outputs, inputs, create_graph=False, **kw):
        return orig_grad(outputs, inputs, create_graph=False, **kw)

    cfg = TINY["tanh_ce_pp"]
    inp = W.make_inputs(cfg)
    eta = torch.from_numpy(inp["eta"].astype(np.float64)).requires_grad_(True)
    monkeypatch.setattr(torch.autograd, "grad", first_order)
    V = oracle.val_loss_of_eta(cfg, inp, eta)
    monkeypatch.setattr(torch.autograd, "grad", orig_grad)
    (d_bad,) = torch.autograd.grad(V, eta)
    assert relerr(d_bad.numpy(), R.complex_step_meta_grad(cfg, inp)) > 1e-4
