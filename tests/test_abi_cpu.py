"""C ABI checks that need no GPU: the library loads, exports every symbol the
header declares, validates descriptions and arguments on the host, and
reports sizes.  No call here reaches a kernel launch."""
import ctypes
import os
import re

import pytest

import workloads as W
from helpers import desc_of

M = pytest.importorskip("paper_2505_00793_amd._lib")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(M.LIB_PATH):
        pytest.skip("libmfmg.so not built")
    return M.lib()


def header_functions():
    src = open(os.path.join(ROOT, "include", "mfmg.h")).read()
    return sorted(set(re.findall(r"^(?:mfmg_status|void|const char\*)\s+(mfmg_\w+)\(", src, re.M)))


def test_exports_every_declared_symbol(L):
    declared = header_functions()
    assert len(declared) >= 9
    for name in declared:
        assert hasattr(L, name), name
    assert sorted(M.EXPORTED) == declared


def test_status_strings(L):
    for s in range(6):
        assert L.mfmg_status_string(s).decode().startswith("MFMG_")
    assert L.mfmg_status_string(M.ERR_NUMERIC) == b"MFMG_ERR_NUMERIC"


@pytest.mark.parametrize("cfg", [W.C1, W.C2, W.C3, W.C5], ids=lambda c: c.name)
def test_sizes_match_layout(L, cfg):
    p = M.Problem(desc_of(cfg))
    s = p.mfmg_query_sizes(cfg.T)
    assert s.n_theta == W.n_theta(cfg)
    assert s.n_eta == W.n_eta(cfg)
    assert s.n_opt_state == W.n_opt_state(cfg)
    assert s.workspace_bytes == s.static_bytes + s.dynamic_bytes or s.dynamic_bytes == 0


def test_static_memory_grows_only_with_checkpoints(L):
    """Workspace per extra inner step = one checkpoint of theta's GEMM operands
    (bf16, two layouts: 4 bytes per weight + 4 per bias, up to 256-byte
    alignment); the dynamic part does not depend on T."""
    cfg = W.C5
    p = M.Problem(desc_of(cfg))
    sizes = {T: p.mfmg_query_sizes(T) for T in W.C5_TS}
    n_w = sum(cfg.widths[l] * cfg.widths[l + 1] for l in range(cfg.n_layers))
    n_b = sum(cfg.widths[1:])
    per_step = 4 * n_w + 4 * n_b
    dyn = {s.dynamic_bytes for s in sizes.values()}
    assert len(dyn) == 1
    for a, b in zip(W.C5_TS, W.C5_TS[1:]):
        slope = (sizes[b].static_bytes - sizes[a].static_bytes) / (b - a)
        assert abs(slope - per_step) <= 3 * 256 * cfg.n_layers


@pytest.mark.parametrize("field,value,status", [
    ("n_layers", 0, M.ERR_INVALID_ARGUMENT if M else 1),
    ("act", 9, 1), ("loss", 5, 1), ("precision", 3, 1), ("rows", 0, 1),
    ("kind", 1, 2), ("meta", 3, 2), ("optimizer", 1, 2),
])
def test_create_rejects_bad_descriptions(L, field, value, status):
    d = desc_of(W.C2)
    setattr(d, field, value)
    h = ctypes.c_void_p()
    st = L.mfmg_problem_create(ctypes.byref(d), ctypes.byref(h))
    assert st == status
    assert not h.value
    assert len(L.mfmg_last_error_message()) > 0


@pytest.mark.parametrize("cfg,fields,status", [
    (W.SMALL["toy_small"], {"map_steps": 0}, 1),        # the map needs M >= 1
    (W.SMALL["toy_small"], {"map_steps": 1025}, 1),
    (W.C5, {"ckpt_segment": -1}, 1),
    (W.C5, {"meta": W.META_MAML, "optimizer": W.OPT_ADAM}, 2),   # MAML is SGD only
    (W.C4, {"meta": W.META_MAML}, 2),                  # and MLP only
    (W.C5, {"fused_attention": 1}, 1),                  # attention options are transformer only
    (W.C5, {"block_remat": 1}, 1),
    (W.C4, {"block_remat": 2}, 2),
    (W.C4, {"fused_attention": 2}, 2),
    (W.C4.with_(precision=W.PREC_FP32), {"fused_attention": 1}, 2),   # bf16 operands only
    (W.C4.with_(n_heads=4), {"fused_attention": 1}, 2),               # head dim 128
    (W.C4.with_(seq=160, rows=8, val_rows=8), {"fused_attention": 1}, 2),  # seq % 64 != 0
])
def test_create_rejects_bad_options(L, cfg, fields, status):
    d = desc_of(cfg)
    for k, v in fields.items():
        setattr(d, k, v)
    h = ctypes.c_void_p()
    assert L.mfmg_problem_create(ctypes.byref(d), ctypes.byref(h)) == status
    assert not h.value


def test_segment_checkpoints_shrink_static_memory():
    """Static bytes with segment checkpoints: (T/k - 1) float32 copies of theta and
    k + 1 operand checkpoints instead of T + 1 (size query only, no GPU)."""
    T = 32
    full = M.Problem(desc_of(W.C5)).mfmg_query_sizes(T)
    seg = M.Problem(desc_of(W.C5.with_(ckpt_segment=6))).mfmg_query_sizes(T)
    n = W.n_theta(W.C5)
    assert full.dynamic_bytes == seg.dynamic_bytes
    # 32 + 1 operand checkpoints (4 B per weight) against 6 + 1 and 5 float32 thetas
    saved = full.static_bytes - seg.static_bytes
    assert abs(saved - (26 * 4 * n - 5 * 4 * n)) < 0.01 * saved
    # Adam (c3) at T = 16, bytes per parameter: every step kept = 17 operand
    # checkpoints (4) + theta_1..16 (4) + m, v for 17 states (8) + 16 gradients (4)
    # = 332; segments of 4 = a ring of 5 operand checkpoints, theta, m, v (16 each)
    # + 4 gradients (4) + theta, m, v at 3 segment starts (12) = 132
    full = M.Problem(desc_of(W.C3)).mfmg_query_sizes(16)
    seg = M.Problem(desc_of(W.C3.with_(ckpt_segment=4))).mfmg_query_sizes(16)
    n = W.n_theta(W.C3)
    assert full.dynamic_bytes == seg.dynamic_bytes
    saved = full.static_bytes - seg.static_bytes
    assert abs(saved - (332 - 132) * n) < 0.01 * saved


def test_fused_attention_drops_quadratic_buffers():
    """Dynamic bytes of the full transformer workload with fused attention: the
    per-block probabilities (2 fp32 + 4 bf16 copies of B*H*S^2) and the shared
    score buffers (4 fp32 + 4 bf16) are gone; per-row statistics (2 floats per
    row and block, 2 shared) are added (size query only, no GPU)."""
    T = 8
    cfg = W.C4
    mat = M.Problem(desc_of(cfg)).mfmg_query_sizes(T)
    fus = M.Problem(desc_of(cfg.with_(fused_attention=1))).mfmg_query_sizes(T)
    assert mat.static_bytes == fus.static_bytes
    BH, S, L = cfg.val_rows * cfg.n_heads, cfg.seq, cfg.n_blocks
    quad = BH * S * S * (L * (2 * 4 + 4 * 2) + 4 * 4 + 4 * 2)
    rows = BH * S * 4 * (2 * L + 2)
    saved = mat.dynamic_bytes - fus.dynamic_bytes
    assert abs(saved - (quad - rows)) < 4096 * (L * 10 + 12)


FAKE = 0x7f0000000000  # never dereferenced: every call below fails validation first


def _meta_call(L, p, T, rows=None, ws_bytes=None, ws=FAKE, x=FAKE, d_eta=FAKE):
    cfg_rows = p.desc.rows
    b = (M.mfmg_batch * max(T, 1))(*[M.mfmg_batch(x, FAKE, rows or cfg_rows) for _ in range(max(T, 1))])
    vb = M.mfmg_batch(FAKE, FAKE, p.desc.val_rows)
    need = p.mfmg_query_sizes(max(T, 1)).workspace_bytes
    peak = ctypes.c_size_t(0)
    return L.mfmg_meta_grad(p.handle, ctypes.c_void_p(FAKE), None, ctypes.c_void_p(FAKE), b, T,
                            ctypes.byref(vb), ctypes.c_void_p(d_eta) if d_eta else None, None,
                            ctypes.byref(peak), ctypes.c_void_p(ws) if ws else None,
                            need if ws_bytes is None else ws_bytes, None)


def test_meta_grad_argument_errors(L):
    p = M.Problem(desc_of(W.C2))
    assert _meta_call(L, p, 0) == M.ERR_INVALID_ARGUMENT
    assert _meta_call(L, p, 2, rows=W.C2.rows + 1) == M.ERR_INVALID_ARGUMENT
    assert _meta_call(L, p, 2, ws_bytes=100) == M.ERR_WORKSPACE
    assert b"workspace" in L.mfmg_last_error_message()
    assert _meta_call(L, p, 2, ws=FAKE + 8) == M.ERR_INVALID_ARGUMENT
    assert _meta_call(L, p, 2, ws=0) == M.ERR_INVALID_ARGUMENT
    assert _meta_call(L, p, 2, d_eta=0) == M.ERR_INVALID_ARGUMENT
    assert _meta_call(L, p, 2, x=0) == M.ERR_INVALID_ARGUMENT


def test_step_argument_errors(L):
    p = M.Problem(desc_of(W.C3))
    b = M.mfmg_batch(FAKE, FAKE, W.C3.rows)
    need = p.mfmg_query_sizes(1).step_workspace_bytes
    # Adam without opt_state_next
    st = L.mfmg_inner_step(p.handle, FAKE, None, FAKE, ctypes.byref(b), 0, FAKE, None, None, None,
                           FAKE, need, None)
    assert st == M.ERR_INVALID_ARGUMENT
    st = L.mfmg_hvp_fwd_over_rev(p.handle, FAKE, FAKE, ctypes.byref(b), 0, FAKE, None, FAKE, None,
                                 FAKE, need - 1, None)
    assert st == M.ERR_WORKSPACE
    st = L.mfmg_hvp_fwd_over_rev(p.handle, FAKE, FAKE, ctypes.byref(b), -1, FAKE, None, FAKE, None,
                                 FAKE, need, None)
    assert st == M.ERR_INVALID_ARGUMENT


def test_timing_read_validates(L):
    n, ms = ctypes.c_int(), ctypes.c_double()
    assert L.mfmg_timing_read(99, ctypes.byref(n), ctypes.byref(ms)) == M.ERR_INVALID_ARGUMENT


def test_check_finite_validates(L):
    n = ctypes.c_size_t(7)
    assert L.mfmg_check_finite(None, 10, ctypes.byref(n), FAKE, 256, None) == M.ERR_INVALID_ARGUMENT
    assert L.mfmg_check_finite(FAKE, 10, ctypes.byref(n), FAKE, 255, None) == M.ERR_WORKSPACE
    assert L.mfmg_check_finite(FAKE, 10, ctypes.byref(n), FAKE + 8, 256, None) == \
        M.ERR_INVALID_ARGUMENT
    assert L.mfmg_check_finite(FAKE + 2, 10, ctypes.byref(n), FAKE, 256, None) == \
        M.ERR_INVALID_ARGUMENT
    assert n.value == 7   # untouched on a validation error


def test_noalloc_rejects_oversized_problems_before_any_device_work(L):
    """mfmg_meta_grad_noalloc checks the problem's workspace against its static
    scratch on the host: a problem that needs more is refused with
    MFMG_ERR_WORKSPACE (fake device pointers, never dereferenced)."""
    p = M.Problem(desc_of(W.C5))
    assert p.mfmg_query_sizes(2).workspace_bytes > M.NOALLOC_SCRATCH_BYTES
    b = (M.mfmg_batch * 2)(*[M.mfmg_batch(FAKE, FAKE, W.C5.rows) for _ in range(2)])
    vb = M.mfmg_batch(FAKE, FAKE, W.C5.val_rows)
    peak = ctypes.c_size_t(0)
    st = L.mfmg_meta_grad_noalloc(p.handle, ctypes.c_void_p(FAKE), None, ctypes.c_void_p(FAKE), b,
                                  2, ctypes.byref(vb), ctypes.c_void_p(FAKE), None,
                                  ctypes.byref(peak), None)
    assert st == M.ERR_WORKSPACE
    assert b"static scratch" in L.mfmg_last_error_message()
    assert L.mfmg_meta_grad_noalloc(p.handle, ctypes.c_void_p(FAKE), None, ctypes.c_void_p(FAKE),
                                    b, 0, ctypes.byref(vb), ctypes.c_void_p(FAKE), None,
                                    ctypes.byref(peak), None) == M.ERR_INVALID_ARGUMENT


def test_block_remat_dynamic_memory_flat_in_depth():
    """With block rematerialisation the transformer's dynamic bytes grow with the
    number of blocks only by the kept block inputs (the residual stream and its
    tangent, float32: 8 bytes per token and model dimension per block); without
    it every block's activations are kept (size query only, no GPU)."""
    T = 8
    size = lambda L, r: M.Problem(desc_of(W.C4.with_(n_blocks=L, block_remat=r,
                                                     fused_attention=1))).mfmg_query_sizes(T)
    N, d = W.C4.val_rows * W.C4.seq, W.C4.d_model
    for L in (4, 8):
        grow = size(L + 4, 1).dynamic_bytes - size(L, 1).dynamic_bytes
        assert abs(grow - 4 * 8 * N * d) <= 4 * 8 * 256
        assert size(L, 1).static_bytes == size(L, 0).static_bytes
    assert size(8, 1).dynamic_bytes < 1.06 * size(4, 1).dynamic_bytes
    assert size(8, 0).dynamic_bytes > 1.5 * size(4, 0).dynamic_bytes
    assert size(4, 1).dynamic_bytes < 0.65 * size(4, 0).dynamic_bytes
