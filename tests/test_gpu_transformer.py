"""GPU parity for the transformer workload (decoder blocks with RoPE, causal
attention, LayerNorm, GELU MLP; per-token loss weights from a meta-model),
through the C ABI, against the float64 oracle."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from helpers import desc_of, group_errors, relerr, spread_of, to_device, tol_of
from oracle import models as OM

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_00793_amd import _lib
    _lib.lib()


def M():
    from paper_2505_00793_amd import _lib
    return _lib


def c(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


SMALL = W.SMALL["c4_small"]
CASES = {"fp32": SMALL.with_(precision=W.PREC_FP32), "bf16": SMALL}
# the full transformer workload: d 512, 8 heads, 4 blocks, vocab 8192, 16 x 256 tokens
FULL = {"fp32": W.C4.with_(precision=W.PREC_FP32), "bf16": W.C4,
        "bf16_fused": W.C4.with_(fused_attention=1)}
FUSED = W.SMALL["c4_fused"]


def token_alpha(cfg, theta, eta, tokens):
    """The loss weights the GPU uses in single-step calls: the meta-model on the
    embedding rows of the theta passed in."""
    th = torch.from_numpy(theta).double()
    emb = OM.unpack(th, W.theta_layout(cfg))["emb"]
    xin, _ = OM.split_tokens(torch.from_numpy(tokens).long())
    return OM.meta_mlp_alpha(cfg, torch.from_numpy(eta).double(), emb[xin]).reshape(-1).numpy()


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_tf_inner_step(prec):
    check_inner_step(CASES[prec], prec)


@pytest.mark.parametrize("prec", ["fp32", "bf16", "bf16_fused"])
def test_tf_inner_step_full_size(prec):
    check_inner_step(FULL[prec], prec)


@pytest.mark.parametrize("name", ["c4_d256", "c4_d256_n12"])
def test_tf_d256_paths(name):
    """d = 256, bf16: LayerNorm and RoPE outputs written as bf16 operand rows with bf16
    transposes (32 tokens), or through float32 and conversions (36 tokens); inner step,
    H v and the meta-gradient against the oracle's bf16 emulation, and the float32
    meta-gradient of the same shapes against the float64 oracle."""
    cfg = W.SMALL[name]
    c32 = cfg.with_(precision=W.PREC_FP32)
    inp32 = W.make_inputs(c32)
    got32, _, _ = run_meta_tf(c32, inp32)
    ref32, _ = oracle.meta_grad_checkpointed(c32, inp32)
    e32 = group_errors(c32, got32, ref32)
    print(f"\n[tf d256] {name} fp32 meta group errors {['%.2e' % e for e in e32]}", flush=True)
    assert max(e32) <= tol_of(c32)
    check_inner_step(cfg, "bf16")
    check_hvp(cfg, "bf16")
    inp = W.make_inputs(cfg)
    got, V, peak = run_meta_tf(cfg, inp)
    ref, Vref = oracle.meta_grad_checkpointed(cfg, inp, bf16=True)
    errs = group_errors(cfg, got, ref)
    print(f"  meta group errors {['%.2e' % e for e in errs]} V {V:.6f} ref {Vref:.6f}", flush=True)
    assert np.all(np.isfinite(got))
    assert max(errs) <= tol_of(cfg)


def test_tf_inner_step_fused():
    """Fused attention, primal forward and backward (three 64-query blocks)."""
    check_inner_step(FUSED, "bf16_fused")


def check_inner_step(cfg, prec):
    inp = W.make_inputs(cfg, T=1)
    n = W.n_theta(cfg)
    theta = inp["theta0"] + 0.02 * W.random_direction(n, 51)
    tok = inp["train_x"][0]
    alpha = token_alpha(cfg, theta, inp["eta"], tok)
    print(f"\n[tf inner_step] {cfg.name} {prec}", flush=True)
    th1_ref, _, g_ref, L_ref = oracle.inner_step(cfg, theta, None, inp["eta"], tok, None, 0,
                                                 alpha=alpha, bf16=prec.startswith("bf16"))
    P = M().Problem(desc_of(cfg))
    th1 = torch.empty(n, device="cuda")
    g = torch.empty(n, device="cuda")
    loss = torch.empty(1, device="cuda")
    dummy_y = torch.zeros(1, dtype=torch.int32, device="cuda")
    P.mfmg_inner_step(c(theta), None, c(inp["eta"]), c(tok), dummy_y, 0, th1, None, g, loss)
    torch.cuda.synchronize()
    e_g = relerr(g.cpu().numpy(), g_ref)
    e_up = relerr(th1.cpu().numpy() - theta, th1_ref - theta)
    print(f"  grad {e_g:.2e} update {e_up:.2e} loss {loss.item():.6f} ref {L_ref:.6f}", flush=True)
    lay = W.theta_layout(cfg)
    gg = g.cpu().numpy()
    for name, off, shape in lay:
        k = int(np.prod(shape))
        e = relerr(gg[off:off + k], g_ref[off:off + k])
        if e > tol_of(cfg):
            print(f"    {name}: {e:.2e}", flush=True)
    assert e_g <= tol_of(cfg) and e_up <= tol_of(cfg)
    assert abs(loss.item() - L_ref) <= tol_of(cfg) * abs(L_ref)


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_tf_hvp(prec):
    check_hvp(CASES[prec], prec)


def test_tf_hvp_full_size_fp32():
    check_hvp(FULL["fp32"], "fp32")


def test_tf_hvp_matches_reverse_over_forward():
    """Transformer H v and per-token mixed product (float32 operands) against the
    oracle's reverse-over-forward mode (Section 2.2)."""
    cfg = CASES["fp32"]
    inp = W.make_inputs(cfg, T=1)
    n = W.n_theta(cfg)
    theta = inp["theta0"] + 0.02 * W.random_direction(n, 54)
    v = 0.1 * W.random_direction(n, 55)
    tok = inp["train_x"][0]
    alpha = token_alpha(cfg, theta, inp["eta"], tok)
    print("\n[tf hvp vs rev-over-fwd] c4_small fp32", flush=True)
    hv_ref, mv_ref = oracle.hvp_rev_fwd(cfg, theta, tok, None, v, alpha=alpha)
    P = M().Problem(desc_of(cfg))
    hv = torch.empty(n, device="cuda")
    mv = torch.empty(cfg.rows * cfg.seq, device="cuda")
    dummy_y = torch.zeros(1, dtype=torch.int32, device="cuda")
    P.mfmg_hvp_fwd_over_rev(c(theta), c(inp["eta"]), c(tok), dummy_y, 0, c(v), None, hv, mv)
    torch.cuda.synchronize()
    e = (relerr(hv.cpu().numpy(), hv_ref), relerr(mv.cpu().numpy(), mv_ref))
    print(f"  hvp {e[0]:.2e} mvp {e[1]:.2e}", flush=True)
    assert max(e) <= tol_of(cfg)


@pytest.mark.parametrize("name", ["c4_fused", "c4_fused128", "c4_fused64"])
def test_tf_hvp_fused(name):
    """Fused attention, dual forward and backward: H v and the mixed product
    (S = 192: 64-row blocks throughout; S = 128: the 128-row dual forward; S = 64: one
    diagonal tile per head)."""
    check_hvp(W.SMALL[name], "bf16_fused")


def check_hvp(cfg, prec):
    inp = W.make_inputs(cfg, T=1)
    n = W.n_theta(cfg)
    theta = inp["theta0"] + 0.02 * W.random_direction(n, 52)
    v = 0.1 * W.random_direction(n, 53)
    tok = inp["train_x"][0]
    alpha = token_alpha(cfg, theta, inp["eta"], tok)
    bf16 = prec.startswith("bf16")
    print(f"\n[tf hvp] {cfg.name} {prec}", flush=True)
    hv_ref = oracle.hvp_rev_rev(cfg, theta, tok, None, v, alpha=alpha, bf16=bf16)
    mv_ref = oracle.mvp_rev_rev(cfg, theta, tok, None, v, alpha=alpha, bf16=bf16)
    g_ref, _ = oracle.grad_and_loss(cfg, theta, tok, None, alpha=alpha, bf16=bf16)
    P = M().Problem(desc_of(cfg))
    g = torch.empty(n, device="cuda")
    hv = torch.empty(n, device="cuda")
    mv = torch.empty(cfg.rows * cfg.seq, device="cuda")
    dummy_y = torch.zeros(1, dtype=torch.int32, device="cuda")
    P.mfmg_hvp_fwd_over_rev(c(theta), c(inp["eta"]), c(tok), dummy_y, 0, c(v), g, hv, mv)
    torch.cuda.synchronize()
    e = (relerr(g.cpu().numpy(), g_ref), relerr(hv.cpu().numpy(), hv_ref),
         relerr(mv.cpu().numpy(), mv_ref))
    print(f"  grad {e[0]:.2e} hvp {e[1]:.2e} mvp {e[2]:.2e}", flush=True)
    hh = hv.cpu().numpy()
    for name, off, shape in W.theta_layout(cfg):
        k = int(np.prod(shape))
        ee = relerr(hh[off:off + k], hv_ref[off:off + k])
        if ee > tol_of(cfg):
            print(f"    {name}: hvp {ee:.2e}", flush=True)
    assert max(e) <= tol_of(cfg)


def run_meta_tf(cfg, inp):
    P = M().Problem(desc_of(cfg))
    dev = to_device(inp)
    d = torch.full((W.n_eta(cfg),), float("nan"), device="cuda")
    vl = torch.full((1,), float("nan"), device="cuda")
    dummy = torch.zeros(1, dtype=torch.int32, device="cuda")
    peak = P.mfmg_meta_grad(dev["theta0"], None, dev["eta"], dev["xs"], [dummy] * len(dev["xs"]),
                            dev["vx"], dummy, d, vl)
    torch.cuda.synchronize()
    return d.cpu().numpy().astype(np.float64), float(vl.item()), peak


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_tf_meta_grad(prec):
    cfg = CASES[prec]
    inp = W.make_inputs(cfg)
    print(f"\n[tf meta_grad] {prec} T={cfg.T}", flush=True)
    got, V, peak = run_meta_tf(cfg, inp)
    ref, Vref = oracle.meta_grad_checkpointed(cfg, inp, bf16=prec == "bf16")
    errs = group_errors(cfg, got, ref)
    print(f"  group errors {['%.2e' % e for e in errs]} V {V:.6f} ref {Vref:.6f}", flush=True)
    assert np.all(np.isfinite(got))
    assert max(errs) <= tol_of(cfg)
    assert abs(V - Vref) <= tol_of(cfg) * abs(Vref)


def test_tf_meta_grad_mid_bf16():
    """8 x 160 tokens: the weight-gradient products over the token dimension take
    the split-K path (5 slices), the unembedding with an odd vocabulary (301)
    its scalar edge; bf16 operands against the oracle's bf16 emulation."""
    cfg = W.SMALL["c4_mid"]
    inp = W.make_inputs(cfg)
    print(f"\n[tf meta_grad] c4_mid bf16 T={cfg.T}", flush=True)
    got, V, peak = run_meta_tf(cfg, inp)
    ref, Vref = oracle.meta_grad_checkpointed(cfg, inp, bf16=True)
    errs = group_errors(cfg, got, ref)
    print(f"  group errors {['%.2e' % e for e in errs]} V {V:.6f} ref {Vref:.6f}", flush=True)
    assert np.all(np.isfinite(got))
    assert max(errs) <= tol_of(cfg)
    assert abs(V - Vref) <= tol_of(cfg) * abs(Vref)


@pytest.mark.parametrize("name", ["c4_fused", "c4_fused128", "c4_fused64", "c4_long_fused"])
def test_tf_meta_grad_fused(name):
    """Fused attention through the whole meta-gradient (192- and 1024-token
    sequences, head dim 64) against the oracle's bf16 emulation."""
    cfg = W.SMALL[name]
    inp = W.make_inputs(cfg)
    print(f"\n[tf meta_grad] {name} S={cfg.seq}", flush=True)
    got, V, peak = run_meta_tf(cfg, inp)
    ref, Vref = oracle.meta_grad_checkpointed(cfg, inp, bf16=True)
    errs = group_errors(cfg, got, ref)
    print(f"  group errors {['%.2e' % e for e in errs]} V {V:.6f} ref {Vref:.6f}", flush=True)
    assert np.all(np.isfinite(got))
    assert max(errs) <= tol_of(cfg)
    assert abs(V - Vref) <= tol_of(cfg) * abs(Vref)


def test_tf_fused_matches_materialised_full_size():
    """The full transformer workload at T=2 with both attention forms: the two
    differ only in where bf16 rounding happens (unnormalised probabilities in
    the fused form), and use less dynamic memory when fused."""
    base = W.C4.with_(T=2)
    inp = W.make_inputs(base, T=2)
    print("\n[tf fused vs materialised] full size T=2", flush=True)
    ref, Vr, peak_r = run_meta_tf(base, inp)
    got, V, peak = run_meta_tf(base.with_(fused_attention=1), inp)
    errs = group_errors(base, got, ref)
    print(f"  group errors {['%.2e' % e for e in errs]} V {V:.6f} / {Vr:.6f} "
          f"peak {peak / 1e9:.2f} / {peak_r / 1e9:.2f} GB", flush=True)
    assert np.all(np.isfinite(got))
    assert max(errs) <= tol_of(base)
    assert abs(V - Vr) <= 1e-3 * abs(Vr)
    assert peak < peak_r


def test_tf_fused_matches_materialised_S4096():
    """The long-context workload's model at S = 4096 (2 sequences per batch, T = 2):
    fused attention against materialised attention, both bf16 (the fused kernels at
    the lengths the long-context measurement runs; 64 query blocks per head)."""
    base = W.C4.with_(name="c4_S4096", seq=4096, rows=2, val_rows=2, T=2)
    inp = W.make_inputs(base, T=2)
    print("\n[tf fused vs materialised] S=4096 T=2", flush=True)
    ref, Vr, peak_r = run_meta_tf(base, inp)
    got, V, peak = run_meta_tf(base.with_(fused_attention=1), inp)
    errs = group_errors(base, got, ref)
    print(f"  group errors {['%.2e' % e for e in errs]} V {V:.6f} / {Vr:.6f} "
          f"peak {peak / 1e9:.2f} / {peak_r / 1e9:.2f} GB", flush=True)
    assert np.all(np.isfinite(got))
    assert max(errs) <= tol_of(base)
    assert abs(V - Vr) <= 1e-3 * abs(Vr)
    assert peak < peak_r


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_tf_meta_grad_long_context(prec):
    """1024-token sequences: causal attention of 1024 x 1024 per head, materialised."""
    cfg = W.SMALL["c4_long"]
    if prec == "fp32":
        cfg = cfg.with_(precision=W.PREC_FP32)
    inp = W.make_inputs(cfg)
    print(f"\n[tf meta_grad] c4_long {prec} S={cfg.seq}", flush=True)
    got, V, peak = run_meta_tf(cfg, inp)
    ref, Vref = oracle.meta_grad_checkpointed(cfg, inp, bf16=prec == "bf16")
    errs = group_errors(cfg, got, ref)
    print(f"  group errors {['%.2e' % e for e in errs]} V {V:.6f} ref {Vref:.6f}", flush=True)
    assert np.all(np.isfinite(got))
    assert max(errs) <= tol_of(cfg)
    assert abs(V - Vref) <= tol_of(cfg) * abs(Vref)


def test_tf_meta_grad_full_size_bf16():
    """The full transformer workload at T=2 with bf16 operands against the
    oracle's float64-accumulated bf16 emulation, each meta-model tensor gated at
    max(2e-2, 1.5 x the stored spread between two valid emulations)."""
    cfg = W.C4.with_(T=2)
    inp = W.make_inputs(cfg, T=2)
    print("\n[tf meta_grad full bf16] T=2", flush=True)
    got, V, peak = run_meta_tf(cfg, inp)
    ref, Vref = oracle.meta_grad_checkpointed(cfg, inp, bf16=True)
    spread = spread_of(f"{cfg.name}/T2")
    errs = group_errors(cfg, got, ref)
    print(f"  errors {['%.2e' % e for e in errs]} spread {['%.2e' % e for e in spread]} "
          f"V {V:.6f} ref {Vref:.6f}", flush=True)
    assert np.all(np.isfinite(got))
    for e, sp in zip(errs, spread):
        assert e <= max(tol_of(cfg), 1.5 * sp)
    assert abs(V - Vref) <= tol_of(cfg) * abs(Vref)


def test_tf_meta_grad_full_size_bf16_T8():
    """The transformer workload as specified (T = 8 inner steps, 16 x 256 tokens,
    d 512, 4 blocks, vocab 8192, bf16 operands, fused attention as bench.py runs
    it) against the oracle's float64-accumulated bf16 emulation at the plain 2e-2
    per meta-model tensor (two valid emulations differ by ~1e-3 here)."""
    cfg = W.C4.with_(fused_attention=1)
    inp = W.make_inputs(cfg)
    print(f"\n[tf meta_grad full bf16] T={cfg.T} fused attention", flush=True)
    got, V, peak = run_meta_tf(cfg, inp)
    ref, Vref = oracle.meta_grad_checkpointed(cfg, inp, bf16=True)
    errs = group_errors(cfg, got, ref)
    print(f"  errors {['%.2e' % e for e in errs]} spread "
          f"{['%.2e' % e for e in spread_of(f'{W.C4.name}/T8')]} V {V:.6f} ref {Vref:.6f}",
          flush=True)
    assert np.all(np.isfinite(got))
    assert max(errs) <= tol_of(cfg)
    assert abs(V - Vref) <= tol_of(cfg) * abs(Vref)


# ---------------------------------------------------------------------------------------
# Block rematerialisation (Section 4): each block's forward is recomputed from its
# input at the start of its backward, in the unroll, the seed and the dual reverse sweep
# ---------------------------------------------------------------------------------------
REMAT_CASES = {"c4_small_fp32": W.SMALL["c4_small"].with_(precision=W.PREC_FP32),
               "c4_small": W.SMALL["c4_small"], "c4_mid": W.SMALL["c4_mid"],
               "c4_fused": W.SMALL["c4_fused"], "c4_fused64": W.SMALL["c4_fused64"]}


@pytest.mark.parametrize("name", list(REMAT_CASES))
def test_tf_block_remat_meta_grad(name):
    """The meta-gradient with block rematerialisation: bit-identical to keeping
    every block's activations (the same kernels recompute the same values), and
    against the oracle (float64, or its bf16 emulation) at the stated tolerance."""
    base = REMAT_CASES[name]
    inp = W.make_inputs(base)
    print(f"\n[tf block remat] {name} blocks={base.n_blocks} T={base.T}", flush=True)
    d0, V0, _ = run_meta_tf(base, inp)
    d1, V1, _ = run_meta_tf(base.with_(block_remat=1), inp)
    ref, Vref = oracle.meta_grad_checkpointed(base, inp, bf16=base.precision == W.PREC_BF16)
    errs = group_errors(base, d1, ref)
    print(f"  bit-identical {np.array_equal(d0, d1)}; vs oracle {['%.2e' % e for e in errs]}",
          flush=True)
    assert np.array_equal(d0, d1) and V0 == V1
    assert max(errs) <= tol_of(base)
    assert abs(V1 - Vref) <= tol_of(base) * abs(Vref)


@pytest.mark.parametrize("name", ["c4_small", "c4_fused"])
def test_tf_block_remat_single_step(name):
    """The inner step and the forward-over-reverse pass with block rematerialisation."""
    cfg = W.SMALL[name].with_(block_remat=1)
    prec = "bf16_fused" if cfg.fused_attention else "bf16"
    check_inner_step(cfg, prec)
    check_hvp(cfg, prec)


def test_tf_block_remat_full_size():
    """The full transformer workload at T=2 (fused attention): rematerialised
    blocks give the same bits as kept ones, match the bf16 emulation at 2e-2,
    and use less dynamic memory."""
    base = W.C4.with_(T=2, fused_attention=1)
    inp = W.make_inputs(base, T=2)
    print("\n[tf block remat] full size T=2 fused attention", flush=True)
    d0, V0, peak0 = run_meta_tf(base, inp)
    d1, V1, peak1 = run_meta_tf(base.with_(block_remat=1), inp)
    ref, Vref = oracle.meta_grad_checkpointed(base, inp, bf16=True)
    errs = group_errors(base, d1, ref)
    print(f"  bit-identical {np.array_equal(d0, d1)}; vs oracle {['%.2e' % e for e in errs]}; "
          f"peak {peak0 / 1e9:.3f} -> {peak1 / 1e9:.3f} GB", flush=True)
    assert np.array_equal(d0, d1) and V0 == V1
    assert max(errs) <= tol_of(base)
    assert peak1 < peak0
