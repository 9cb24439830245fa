"""Pins for the float64 oracle: each check ties it to something other than itself.

* closed-form meta-gradient of SGD on a quadratic loss (linear regression);
* complex-step derivatives of V(eta) through an independent numpy inner loop
  with hand-written gradients (MLPs, all three update rules, both heads);
* central finite differences with Richardson extrapolation (transformer);
* T=1 closed forms for learned learning rates and for loss weights;
* Hessian symmetry u.Hv = v.Hu, a brute-force Hessian against finite
  differences of the gradient, forward-over-reverse == reverse-over-reverse;
* whole-graph == step-checkpointed;
* library cross-checks: AdamW, cross-entropy, GELU, layer norm, attention.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from oracle import models as OM
from oracle import optim as OO
from oracle.ops import bf16_round

import numpy_ref as R

# Tiny problems for exhaustive checks (<= a few hundred meta-parameters).
TINY = {
    "linreg": W.C1.with_(name="t_linreg", cfg_id=201, widths=(5, 1), rows=7, val_rows=6, T=3,
                         loglr_init=math.log(0.05)),
    "tanh_ce_pp": W.C5.with_(name="t_tanh", cfg_id=202, widths=(4, 5, 3), act=W.ACT_TANH,
                             precision=W.PREC_FP32, rows=6, val_rows=5, T=3,
                             loglr_init=math.log(0.3)),
    "gelu_ce_pp": W.C5.with_(name="t_gelu", cfg_id=203, widths=(3, 4, 4, 2), act=W.ACT_GELU,
                             precision=W.PREC_FP32, rows=6, val_rows=5, T=3,
                             loglr_init=math.log(0.3)),
    "relu_ce_pp": W.C5.with_(name="t_relu", cfg_id=204, widths=(4, 6, 3), act=W.ACT_RELU,
                             precision=W.PREC_FP32, rows=6, val_rows=5, T=2,
                             loglr_init=math.log(0.3)),
    "tanh_mse_pp": W.C5.with_(name="t_mse", cfg_id=205, widths=(3, 4, 1), act=W.ACT_TANH,
                              loss=W.LOSS_MSE, precision=W.PREC_FP32, rows=6, val_rows=5, T=3,
                              loglr_init=math.log(0.1)),
    "weights": W.C2.with_(name="t_weights", cfg_id=206, widths=(4, 5, 3), rows=6, val_rows=5,
                          T=3, sgd_lr=0.5),
    "adam": W.C3.with_(name="t_adam", cfg_id=207, widths=(4, 5, 3), precision=W.PREC_FP32,
                       rows=6, val_rows=5, T=3, loglr_init=math.log(0.05), wd_init=0.1),
    "adam_tanh": W.C3.with_(name="t_adam_tanh", cfg_id=208, widths=(3, 4, 2), act=W.ACT_TANH,
                            precision=W.PREC_FP32, rows=5, val_rows=4, T=4,
                            loglr_init=math.log(0.02), wd_init=0.05),
    "maml_tanh_ce": W.C5.with_(name="t_maml_ce", cfg_id=209, widths=(4, 5, 3), act=W.ACT_TANH,
                               precision=W.PREC_FP32, meta=W.META_MAML, sgd_lr=0.4, rows=6,
                               val_rows=5, T=3),
    "toy_map": W.TOY.with_(name="t_toy", cfg_id=212, widths=(6, 5), rows=7, val_rows=4,
                           map_steps=3, sgd_lr=0.05),
    "toy_map_m1": W.TOY.with_(name="t_toy1", cfg_id=213, widths=(4, 3), rows=5, val_rows=3,
                              map_steps=1, sgd_lr=0.2, T=3),
    "maml_gelu_mse": W.C5.with_(name="t_maml_mse", cfg_id=210, widths=(3, 4, 1),
                                act=W.ACT_GELU, loss=W.LOSS_MSE, has_bias=True,
                                precision=W.PREC_FP32, meta=W.META_MAML, sgd_lr=0.2, rows=6,
                                val_rows=5, T=2),
}


def relerr(a, b):
    return np.linalg.norm(np.asarray(a) - np.asarray(b)) / max(np.linalg.norm(b), 1e-300)


# ---------------------------------------------------------------------------------------
# Closed form: SGD with per-parameter learning rates on the squared loss
# ---------------------------------------------------------------------------------------
def linreg_closed_form(inp):
    """theta_{i+1} = (I - D A_i) theta_i + D b_i with A_i = (2/N) X^T X, b_i = (2/N) X^T y,
    D = diag(exp(eta)); adjoint a_T = grad V(theta_T), a_i = (I - A_i D) a_{i+1};
    dV/deta = - sum_i exp(eta) * g_i * a_{i+1}, g_i = A_i theta_i - b_i."""
    eta = inp["eta"].astype(np.float64)
    D = np.exp(eta)
    th = inp["theta0"].astype(np.float64)
    As, gs = [], []
    for X, y in zip(inp["train_x"], inp["train_y"]):
        X = X.astype(np.float64)
        y = y.astype(np.float64).reshape(-1)
        N = X.shape[0]
        A = 2.0 / N * X.T @ X
        b = 2.0 / N * X.T @ y
        g = A @ th - b
        As.append(A)
        gs.append(g)
        th = th - D * g
    Xv = inp["val_x"].astype(np.float64)
    yv = inp["val_y"].astype(np.float64).reshape(-1)
    a = 2.0 / Xv.shape[0] * Xv.T @ (Xv @ th - yv)
    d = np.zeros_like(eta)
    for i in reversed(range(len(As))):
        d += -D * gs[i] * a
        a = a - As[i] @ (D * a)
    return d


def maml_linreg_closed_form(inp, lr):
    """MAML on the squared loss: theta_{i+1} = (I - lr A_i) theta_i + lr b_i, so with
    a_T = grad V(theta_T) and a_i = (I - lr A_i) a_{i+1} (A_i symmetric), dV/dtheta_0 = a_0."""
    th = inp["eta"].astype(np.float64)
    As = []
    for X, y in zip(inp["train_x"], inp["train_y"]):
        X = X.astype(np.float64)
        y = y.astype(np.float64).reshape(-1)
        N = X.shape[0]
        A = 2.0 / N * X.T @ X
        th = th - lr * (A @ th - 2.0 / N * X.T @ y)
        As.append(A)
    Xv = inp["val_x"].astype(np.float64)
    yv = inp["val_y"].astype(np.float64).reshape(-1)
    a = 2.0 / Xv.shape[0] * Xv.T @ (Xv @ th - yv)
    for A in reversed(As):
        a = a - lr * (A @ a)
    return a


@pytest.mark.parametrize("T", [1, 3])
def test_maml_linreg_closed_form(T):
    cfg = W.C1.with_(name="t_maml_lin", cfg_id=211, meta=W.META_MAML, sgd_lr=0.05, T=T,
                     widths=(6, 1), rows=9, val_rows=7)
    inp = W.make_inputs(cfg)
    assert not np.any(inp["theta0"])   # the starting point comes from eta alone
    d_cf = maml_linreg_closed_form(inp, cfg.sgd_lr)
    assert relerr(oracle.meta_grad(cfg, inp)[0], d_cf) < 1e-12
    assert relerr(oracle.meta_grad_checkpointed(cfg, inp)[0], d_cf) < 1e-12


def test_maml_zero_lr_is_the_validation_gradient():
    """With a zero inner learning rate theta_T = theta_0 = eta, so dV/deta = grad V(eta)."""
    cfg = TINY["maml_tanh_ce"].with_(sgd_lr=0.0)
    inp = W.make_inputs(cfg)
    _, g = R.loss_and_grad(cfg, inp["eta"].astype(np.float64), inp["val_x"].astype(np.float64),
                           inp["val_y"])
    assert relerr(oracle.meta_grad_checkpointed(cfg, inp)[0], g) < 1e-12


@pytest.mark.parametrize("cfg", [W.C1, W.SMALL["c1_small"], TINY["linreg"]], ids=lambda c: c.name)
def test_linreg_closed_form(cfg):
    inp = W.make_inputs(cfg)
    d_or, _ = oracle.meta_grad(cfg, inp)
    d_cf = linreg_closed_form(inp)
    assert relerr(d_or, d_cf) < 1e-12


@pytest.mark.parametrize("T", [1, 2, 7])
def test_linreg_closed_form_various_T(T):
    cfg = W.C1.with_(T=T)
    inp = W.make_inputs(cfg)
    assert relerr(oracle.meta_grad(cfg, inp)[0], linreg_closed_form(inp)) < 1e-12


# ---------------------------------------------------------------------------------------
# Complex step through an independent numpy inner loop
# ---------------------------------------------------------------------------------------
@pytest.mark.parametrize("key", sorted(TINY))
def test_complex_step(key):
    cfg = TINY[key]
    inp = W.make_inputs(cfg)
    d_or, V_or = oracle.meta_grad(cfg, inp)
    assert abs(R.val_loss(cfg, inp, inp["eta"].astype(np.float64)) - V_or) < 1e-12 * max(1, abs(V_or))
    d_cs = R.complex_step_meta_grad(cfg, inp)
    assert np.linalg.norm(d_cs) > 0
    assert relerr(d_or, d_cs) < 1e-10, (d_or[:5], d_cs[:5])


def test_numpy_reference_gradient_by_fd():
    """The hand-written numpy gradient itself, against central differences."""
    for key in ("tanh_ce_pp", "gelu_ce_pp", "tanh_mse_pp"):
        cfg = TINY[key]
        inp = W.make_inputs(cfg)
        th = inp["theta0"].astype(np.float64)
        x, y = inp["train_x"][0].astype(np.float64), inp["train_y"][0]
        if y.dtype.kind == "f":
            y = y.astype(np.float64)
        _, g = R.loss_and_grad(cfg, th, x, y)
        h = 1e-6
        fd = np.array([(R.loss_and_grad(cfg, th + h * e, x, y)[0] - R.loss_and_grad(cfg, th - h * e, x, y)[0]) / (2 * h)
                       for e in np.eye(th.size)])
        assert relerr(g, fd) < 1e-8


# ---------------------------------------------------------------------------------------
# Finite differences (transformer and full-size small workloads)
# ---------------------------------------------------------------------------------------
def fd_directional(cfg, inp, u, h):
    eta0 = torch.from_numpy(inp["eta"].astype(np.float64))
    ut = torch.from_numpy(u)

    def V(e):
        with torch.no_grad():
            pass
        return float(oracle.val_loss_of_eta(cfg, inp, e, create_graph=False).detach())

    def D(hh):
        return (V(eta0 + hh * ut) - V(eta0 - hh * ut)) / (2 * hh)

    return (4 * D(h / 2) - D(h)) / 3


@pytest.mark.parametrize("name,h", [("c4_small", 1e-3), ("c2_small", 1e-2), ("c3_fp32", 1e-3)])
def test_fd_directional(name, h):
    cfg = W.SMALL[name]
    inp = W.make_inputs(cfg)
    d_or, _ = oracle.meta_grad(cfg, inp)
    rng = np.random.default_rng(7)
    for _ in range(2):
        u = rng.standard_normal(d_or.size)
        lhs = float(d_or @ u)
        rhs = fd_directional(cfg, inp, u, h)
        assert abs(lhs - rhs) <= 1e-7 * max(abs(lhs), np.linalg.norm(d_or) * np.linalg.norm(u) * 1e-3), (lhs, rhs)


# ---------------------------------------------------------------------------------------
# T = 1 closed forms
# ---------------------------------------------------------------------------------------
def test_T1_learned_lr_closed_form():
    """T=1, theta_1 = theta_0 - exp(eta) g_0:  dV/deta = -exp(eta) * g_0 * grad V(theta_1)."""
    cfg = TINY["gelu_ce_pp"].with_(T=1)
    inp = W.make_inputs(cfg)
    th0 = inp["theta0"].astype(np.float64)
    eta = inp["eta"].astype(np.float64)
    _, g0 = R.loss_and_grad(cfg, th0, inp["train_x"][0].astype(np.float64), inp["train_y"][0])
    th1 = th0 - np.exp(eta) * g0
    _, gV = R.loss_and_grad(cfg, th1, inp["val_x"].astype(np.float64), inp["val_y"])
    expect = -np.exp(eta) * g0 * gV
    assert relerr(oracle.meta_grad(cfg, inp)[0], expect) < 1e-12


def test_T1_loss_weight_closed_form():
    """T=1, L = (1/N) sum sigma(eta_n) l_n, theta_1 = theta_0 - lr g_0:
    dV/deta_n = sigma'(eta_n) * (-(lr/N) grad V(theta_1) . grad l_n(theta_0))."""
    cfg = TINY["weights"].with_(T=1)
    inp = W.make_inputs(cfg)
    inp["eta"] = np.random.default_rng(3).standard_normal(cfg.rows).astype(np.float32)
    th0 = inp["theta0"].astype(np.float64)
    eta = inp["eta"].astype(np.float64)
    x, y = inp["train_x"][0].astype(np.float64), inp["train_y"][0]
    s = 1 / (1 + np.exp(-eta))
    _, g0 = R.loss_and_grad(cfg, th0, x, y, s)
    th1 = th0 - cfg.sgd_lr * g0
    _, gV = R.loss_and_grad(cfg, th1, inp["val_x"].astype(np.float64), inp["val_y"])
    G = R.per_example_grads(cfg, th0, x, y)
    expect = s * (1 - s) * (-(cfg.sgd_lr / cfg.rows) * (G @ gV))
    assert relerr(oracle.meta_grad(cfg, inp)[0], expect) < 1e-12


# ---------------------------------------------------------------------------------------
# Hessian-vector products
# ---------------------------------------------------------------------------------------
HVP_CASES = ["tanh_ce_pp", "gelu_ce_pp", "relu_ce_pp", "tanh_mse_pp"]


def _one_batch(cfg):
    inp = W.make_inputs(cfg)
    return inp["theta0"], inp["train_x"][0], inp["train_y"][0]


@pytest.mark.parametrize("key", HVP_CASES)
def test_hessian_symmetry(key):
    cfg = TINY[key]
    th, x, y = _one_batch(cfg)
    n = th.size
    u = W.random_direction(n, 1).astype(np.float64)
    v = W.random_direction(n, 2).astype(np.float64)
    uHv = u @ oracle.hvp_rev_rev(cfg, th, x, y, v)
    vHu = v @ oracle.hvp_rev_rev(cfg, th, x, y, u)
    assert abs(uHv - vHu) < 1e-12 * max(1.0, abs(uHv))


@pytest.mark.parametrize("key", HVP_CASES)
def test_bruteforce_hessian_vs_fd_of_gradient(key):
    """Full Hessian from HVPs on basis vectors: symmetric, equal to the central
    difference of the independent numpy gradient."""
    cfg = TINY[key]
    th, x, y = _one_batch(cfg)
    x64 = x.astype(np.float64)
    y_ = y.astype(np.float64) if y.dtype.kind == "f" else y
    n = th.size
    assert n <= 60
    H = np.stack([oracle.hvp_rev_rev(cfg, th, x, y, e) for e in np.eye(n)])
    assert np.abs(H - H.T).max() < 1e-12 * max(1.0, np.abs(H).max())
    h = 1e-5
    th64 = th.astype(np.float64)
    Hfd = np.stack([(R.loss_and_grad(cfg, th64 + h * e, x64, y_)[1]
                     - R.loss_and_grad(cfg, th64 - h * e, x64, y_)[1]) / (2 * h) for e in np.eye(n)])
    assert np.abs(H - Hfd).max() < 1e-7 * max(1.0, np.abs(H).max())


@pytest.mark.parametrize("name", ["c2_small", "c5_small", "c3_small", "c4_small", "c4_fused"])
def test_three_hvp_modes_agree(name):
    """The three HVP modes of Section 2.2 on one batch: the JVP of the gradient map
    (forward-over-reverse), the gradient of the directional derivative <grad L, v>
    taken in forward mode (reverse-over-forward), both by torch.func, and the
    oracle's reverse-over-reverse HVP agree to rounding; the per-row loss tangents
    equal the mixed product, also when taken as the alpha-gradient of the
    forward-mode directional derivative."""
    cfg = W.SMALL[name]
    th, x, y = _one_batch(cfg)
    v = W.random_direction(th.size, 3).astype(np.float64)
    hv_rr = oracle.hvp_rev_rev(cfg, th, x, y, v)
    mv_rr = oracle.mvp_rev_rev(cfg, th, x, y, v)
    xt = torch.from_numpy(x) if x.dtype.kind != "f" else torch.from_numpy(x).double()
    yt = None if y is None else (torch.from_numpy(y).long() if y.dtype.kind != "f"
                                 else torch.from_numpy(y).double())

    def loss(p):
        return OM.inner_loss(cfg, p, None, xt, yt, False)

    def rows(p):
        return OM.per_row_losses(cfg, p, xt, yt, False)

    tht = torch.from_numpy(th).double()
    vt = torch.from_numpy(v)
    _, hv_fr = torch.func.jvp(torch.func.grad(loss), (tht,), (vt,))
    _, ldot = torch.func.jvp(rows, (tht,), (vt,))
    assert relerr(hv_fr.numpy(), hv_rr) < 1e-12
    assert relerr(ldot.numpy() / ldot.numel(), mv_rr) < 1e-12

    hv_rf, mv_rf = oracle.hvp_rev_fwd(cfg, th, x, y, v)
    assert relerr(hv_rf, hv_rr) < 1e-12
    assert relerr(mv_rf, mv_rr) < 1e-12


# ---------------------------------------------------------------------------------------
# Checkpointed == whole graph
# ---------------------------------------------------------------------------------------
@pytest.mark.parametrize("name", sorted(W.SMALL))
def test_checkpointed_equals_whole_graph(name):
    cfg = W.SMALL[name]
    inp = W.make_inputs(cfg)
    a, Va = oracle.meta_grad(cfg, inp)
    b, Vb = oracle.meta_grad_checkpointed(cfg, inp)
    assert relerr(b, a) <= 1e-12 and abs(Va - Vb) <= 1e-12 * abs(Va)


# ---------------------------------------------------------------------------------------
# Library cross-checks of the building blocks
# ---------------------------------------------------------------------------------------
def test_adam_update_matches_torch_adamw():
    cfg = TINY["adam"]
    inp = W.make_inputs(cfg)
    n = W.n_theta(cfg)
    eta = torch.tensor([math.log(0.05), math.log(0.02), 0.1], dtype=torch.float64)
    th = torch.from_numpy(inp["theta0"]).double()
    opt = torch.zeros(2 * n, dtype=torch.float64)
    lay = W.theta_layout(cfg)
    params = [torch.nn.Parameter(th[off:off + int(np.prod(s))].clone()) for _, off, s in lay]
    groups = [{"params": [p], "lr": math.exp(float(eta[int(name[1:])]))}
              for p, (name, _, _) in zip(params, lay)]
    ref = torch.optim.AdamW(groups, betas=(cfg.adam_b1, cfg.adam_b2), eps=cfg.adam_eps,
                            weight_decay=float(eta[-1]))
    rng = np.random.default_rng(0)
    for step in range(3):
        g = torch.from_numpy(rng.standard_normal(n))
        th, opt = OO.upsilon(cfg, g, th, opt, eta, step)
        for p, (_, off, s) in zip(params, lay):
            p.grad = g[off:off + int(np.prod(s))].clone()
        ref.step()
        flat = torch.cat([p.detach().reshape(-1) for p in params])
        assert torch.allclose(th, flat, rtol=1e-13, atol=1e-15)


def test_building_blocks_match_torch_functional():
    F = torch.nn.functional
    rng = np.random.default_rng(1)
    z = torch.from_numpy(rng.standard_normal((9, 7)))
    y = torch.from_numpy(rng.integers(0, 7, 9))
    from oracle.ops import cross_entropy_rows, gelu, layer_norm
    assert torch.allclose(cross_entropy_rows(z, y), F.cross_entropy(z, y, reduction="none"), atol=1e-14)
    assert torch.allclose(gelu(z), F.gelu(z), atol=1e-14)
    g = torch.from_numpy(rng.standard_normal(7))
    b = torch.from_numpy(rng.standard_normal(7))
    assert torch.allclose(layer_norm(z, g, b, 1e-5), F.layer_norm(z, (7,), g, b, 1e-5), atol=1e-12)


def _transformer_logits_independent(cfg, theta, tokens):
    """The same decoder written with torch.nn.functional and complex-number RoPE."""
    F = torch.nn.functional
    P = OM.unpack(torch.from_numpy(theta).double(), W.theta_layout(cfg))
    B, S = tokens.shape
    d, H = cfg.d_model, cfg.n_heads
    dh = d // H
    half = dh // 2
    pos = torch.arange(S, dtype=torch.float64)
    freqs = cfg.rope_base ** (-torch.arange(half, dtype=torch.float64) * 2 / dh)
    rot = torch.polar(torch.ones(S, half, dtype=torch.float64), pos[:, None] * freqs[None])

    def rope(t):  # pairs (j, j + dh/2) as complex numbers j + i (j + half)
        c = torch.complex(t[..., :half], t[..., half:]) * rot
        return torch.cat([c.real, c.imag], -1)

    h = F.embedding(torch.from_numpy(tokens).long(), P["emb"])
    for b in range(cfg.n_blocks):
        a = F.layer_norm(h, (d,), P[f"ln1_g{b}"], P[f"ln1_b{b}"], cfg.ln_eps)
        q, k, v = (a @ P[f"wqkv{b}"]).split(d, dim=-1)
        q, k, v = (t.reshape(B, S, H, dh).permute(0, 2, 1, 3) for t in (q, k, v))
        o = F.scaled_dot_product_attention(rope(q), rope(k), v, is_causal=True)
        h = h + o.permute(0, 2, 1, 3).reshape(B, S, d) @ P[f"wo{b}"]
        a2 = F.layer_norm(h, (d,), P[f"ln2_g{b}"], P[f"ln2_b{b}"], cfg.ln_eps)
        h = h + F.gelu(a2 @ P[f"w1{b}"]) @ P[f"w2{b}"]
    hf = F.layer_norm(h, (d,), P["lnf_g"], P["lnf_b"], cfg.ln_eps)
    return (hf @ P["unemb"]).reshape(B * S, -1)


def test_transformer_forward_matches_independent_version():
    cfg = W.SMALL["c4_small"]
    inp = W.make_inputs(cfg)
    th = inp["theta0"] + 0.05 * W.random_direction(W.n_theta(cfg), 5)  # non-trivial LN params
    tok = inp["train_x"][0][:, :-1]
    ours = OM.transformer_logits(cfg, torch.from_numpy(th).double(), torch.from_numpy(tok), False)
    ref = _transformer_logits_independent(cfg, th, tok)
    assert torch.allclose(ours, ref, rtol=1e-10, atol=1e-12)


def test_transformer_is_causal():
    cfg = W.SMALL["c4_small"]
    inp = W.make_inputs(cfg)
    th = torch.from_numpy(inp["theta0"]).double()
    tok = inp["train_x"][0][:, :-1].copy()
    a = OM.transformer_logits(cfg, th, torch.from_numpy(tok), False).reshape(cfg.rows, cfg.seq, -1)
    tok[:, 10] = (tok[:, 10] + 1) % cfg.vocab
    b = OM.transformer_logits(cfg, th, torch.from_numpy(tok), False).reshape(cfg.rows, cfg.seq, -1)
    assert torch.equal(a[:, :10], b[:, :10])
    assert not torch.allclose(a[:, 10:], b[:, 10:])


def test_bf16_rounding_is_rne():
    x = torch.tensor([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -(1.0 + 2 ** -8) - 2 ** -20],
                     dtype=torch.float64)
    r = bf16_round(x)
    assert r.tolist() == [1.0, 1.0 + 2 ** -6, 1.0, -(1.0 + 2 ** -7)]


@pytest.mark.parametrize("name", ["c3_small", "c5_small", "c4_small"])
def test_bf16_emulation_is_a_small_perturbation(name):
    cfg = W.SMALL[name]
    inp = W.make_inputs(cfg)
    a, _ = oracle.meta_grad(cfg, inp)
    b, _ = oracle.meta_grad(cfg, inp, bf16=True)
    assert 0 < relerr(b, a) < 2e-2


# ---------------------------------------------------------------------------------------
# Where the bf16 emulation rounds: a hand-written numpy forward/backward with every
# GEMM operand rounded (round-to-nearest-even written from the float32 bit layout,
# not through torch's conversion)
# ---------------------------------------------------------------------------------------
def rne_bf16(x):
    """float64 -> float32 -> bfloat16 (round to nearest, ties to even) as float64:
    add 0x7FFF plus the lowest kept bit to the float32 pattern, clear the low 16 bits."""
    u = np.ascontiguousarray(np.asarray(x, dtype=np.float32)).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def test_rne_bf16_matches_the_emulation_rounding():
    x = np.random.default_rng(5).standard_normal(10000) * np.exp(
        np.random.default_rng(6).uniform(-20, 20, 10000))
    assert np.array_equal(rne_bf16(x), bf16_round(torch.from_numpy(x)).numpy())
    # exact ties go to the even mantissa
    assert rne_bf16(np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8])).tolist() == [1.0, 1 + 2 ** -6]


def _softmax_rows(z):
    e = np.exp(z - z.max(1, keepdims=True))
    return e / e.sum(1, keepdims=True)


@pytest.mark.parametrize("act", [W.ACT_TANH, W.ACT_RELU])
def test_bf16_emulation_rounding_placement_two_layers(act):
    """Gradient of a two-layer CE network under the bf16 emulation equals the
    plain backward with these operands rounded: X, W1 | r(A1), W2 in the forward;
    dZ2 and W2 in the data product; r(A1), dZ2 and X, dZ1 in the weight products;
    bias gradients summing the rounded dZ (the reduction reads the same bf16
    operand copy the weight product does)."""
    r = rne_bf16
    cfg = W.C5.with_(name="t_emu2", cfg_id=230, widths=(9, 11, 5), act=act, rows=13,
                     val_rows=4, T=1, precision=W.PREC_BF16)
    inp = W.make_inputs(cfg)
    theta = inp["theta0"].astype(np.float64) + 0.1 * W.random_direction(W.n_theta(cfg), 60)
    theta = theta.astype(np.float32).astype(np.float64)
    x, y = inp["train_x"][0].astype(np.float64), inp["train_y"][0]
    lay = {n: (o, s) for n, o, s in W.theta_layout(cfg)}
    P = {n: theta[o:o + int(np.prod(s))].reshape(s) for n, (o, s) in lay.items()}
    N = x.shape[0]
    z1 = r(x) @ r(P["W0"]) + P["b0"]
    a1 = np.tanh(z1) if act == W.ACT_TANH else np.maximum(z1, 0)
    dphi = 1 - a1 ** 2 if act == W.ACT_TANH else (z1 > 0).astype(np.float64)
    z2 = r(a1) @ r(P["W1"]) + P["b1"]
    p = _softmax_rows(z2)
    dz2 = p.copy()
    dz2[np.arange(N), y] -= 1.0
    dz2 /= N
    g = {"W1": r(a1).T @ r(dz2), "b1": r(dz2).sum(0)}
    dz1 = (r(dz2) @ r(P["W1"]).T) * dphi
    g["W0"] = r(x).T @ r(dz1)
    g["b0"] = r(dz1).sum(0)
    want = np.concatenate([g[n].ravel() for n, _, _ in W.theta_layout(cfg)])
    got, _ = oracle.grad_and_loss(cfg, theta, x, y, bf16=True)
    assert relerr(got, want) <= 1e-12
    # and the rounding is visible: the unrounded gradient is measurably elsewhere
    plain, _ = oracle.grad_and_loss(cfg, theta, x, y)
    assert relerr(plain, want) > 1e-4


def test_bf16_emulation_hvp_one_layer():
    """H v of a one-layer CE model (z = x W + b) under the bf16 emulation: the
    tangent logits are r(x) r(V) + v_b, the tangent of the output gradient is
    p (zdot - <p, zdot>) / N, and H v = r(x)^T r(that), its bias part the sum of
    the rounded rows."""
    r = rne_bf16
    cfg = W.C5.with_(name="t_emu1", cfg_id=231, widths=(10, 6), rows=12, val_rows=4, T=1,
                     precision=W.PREC_BF16)
    inp = W.make_inputs(cfg)
    n = W.n_theta(cfg)
    theta = (0.5 * W.random_direction(n, 61)).astype(np.float64)
    v = W.random_direction(n, 62).astype(np.float64)
    x, y = inp["train_x"][0].astype(np.float64), inp["train_y"][0]
    lay = {nm: (o, s) for nm, o, s in W.theta_layout(cfg)}
    Wt = theta[lay["W0"][0]:lay["W0"][0] + 60].reshape(10, 6)
    bt = theta[lay["b0"][0]:lay["b0"][0] + 6]
    Vw = v[lay["W0"][0]:lay["W0"][0] + 60].reshape(10, 6)
    Vb = v[lay["b0"][0]:lay["b0"][0] + 6]
    N = x.shape[0]
    p = _softmax_rows(r(x) @ r(Wt) + bt)
    zd = r(x) @ r(Vw) + Vb
    dd = p * (zd - (p * zd).sum(1, keepdims=True)) / N
    want = np.concatenate([(r(x).T @ r(dd)).ravel(), r(dd).sum(0)])
    got = oracle.hvp_rev_rev(cfg, theta, x, y, v, bf16=True)
    assert relerr(got, want) <= 1e-12
