"""ctypes binding of libmfmg.so (include/mfmg.h).  Argument marshalling only.

Every function here has the name of the C entry point it wraps.  Torch is
used for device memory, the current stream and pointers; all arithmetic of
the meta-gradient runs in the library's HIP kernels.  Loading fails loudly
when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int, c_int64, c_size_t, c_void_p

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmfmg.so")

MAX_LAYERS = 16
OK, ERR_INVALID_ARGUMENT, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP, ERR_NUMERIC = 0, 1, 2, 3, 4, 5

EXPORTED = [
    "mfmg_problem_create", "mfmg_problem_destroy", "mfmg_query_sizes", "mfmg_inner_step",
    "mfmg_hvp_fwd_over_rev", "mfmg_meta_grad", "mfmg_status_string", "mfmg_last_error_message",
    "mfmg_timing_enable", "mfmg_timing_read", "mfmg_check_finite", "mfmg_meta_grad_noalloc",
]
NOALLOC_SCRATCH_BYTES = 64 * 1024 * 1024   # MFMG_NOALLOC_SCRATCH_BYTES


class mfmg_problem_desc(ctypes.Structure):
    _fields_ = [
        ("kind", c_int), ("n_layers", c_int), ("widths", c_int * (MAX_LAYERS + 1)),
        ("act", c_int), ("loss", c_int), ("optimizer", c_int), ("meta", c_int),
        ("precision", c_int), ("has_bias", c_int), ("rows", c_int), ("val_rows", c_int),
        ("sgd_lr", c_float), ("adam_b1", c_float), ("adam_b2", c_float), ("adam_eps", c_float),
        ("d_model", c_int), ("n_heads", c_int), ("d_ff", c_int), ("vocab", c_int), ("seq", c_int),
        ("n_blocks", c_int), ("meta_hidden", c_int), ("ln_eps", c_float), ("rope_base", c_float),
        ("map_steps", c_int), ("ckpt_segment", c_int), ("fused_attention", c_int),
        ("block_remat", c_int),
    ]


class mfmg_sizes(ctypes.Structure):
    _fields_ = [("n_theta", c_size_t), ("n_opt_state", c_size_t), ("n_eta", c_size_t),
                ("workspace_bytes", c_size_t), ("static_bytes", c_size_t),
                ("dynamic_bytes", c_size_t), ("step_workspace_bytes", c_size_t)]


class mfmg_batch(ctypes.Structure):
    _fields_ = [("x", c_void_p), ("y", c_void_p), ("rows", c_int64)]


class MfmgError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2505_00793_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P = POINTER
    L.mfmg_problem_create.argtypes = [P(mfmg_problem_desc), P(c_void_p)]
    L.mfmg_problem_destroy.argtypes = [c_void_p]
    L.mfmg_problem_destroy.restype = None
    L.mfmg_query_sizes.argtypes = [c_void_p, c_int, P(mfmg_sizes)]
    L.mfmg_inner_step.argtypes = [c_void_p, c_void_p, c_void_p, c_void_p, P(mfmg_batch), c_int,
                                  c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                  c_void_p]
    L.mfmg_hvp_fwd_over_rev.argtypes = [c_void_p, c_void_p, c_void_p, P(mfmg_batch), c_int,
                                        c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                        c_size_t, c_void_p]
    L.mfmg_meta_grad.argtypes = [c_void_p, c_void_p, c_void_p, c_void_p, P(mfmg_batch), c_int,
                                 P(mfmg_batch), c_void_p, c_void_p, P(c_size_t), c_void_p,
                                 c_size_t, c_void_p]
    L.mfmg_meta_grad_noalloc.argtypes = [c_void_p, c_void_p, c_void_p, c_void_p, P(mfmg_batch),
                                         c_int, P(mfmg_batch), c_void_p, c_void_p, P(c_size_t),
                                         c_void_p]
    L.mfmg_check_finite.argtypes = [c_void_p, c_size_t, P(c_size_t), c_void_p, c_size_t,
                                    c_void_p]
    L.mfmg_status_string.argtypes = [c_int]
    L.mfmg_status_string.restype = c_char_p
    L.mfmg_last_error_message.argtypes = []
    L.mfmg_last_error_message.restype = c_char_p
    L.mfmg_timing_enable.argtypes = [c_int]
    L.mfmg_timing_read.argtypes = [c_int, P(c_int), P(c_double)]
    for name in ("mfmg_problem_create", "mfmg_query_sizes", "mfmg_inner_step",
                 "mfmg_hvp_fwd_over_rev", "mfmg_meta_grad", "mfmg_timing_enable",
                 "mfmg_timing_read", "mfmg_check_finite", "mfmg_meta_grad_noalloc"):
        getattr(L, name).restype = c_int
    _lib = L
    return L


def check(status: int) -> None:
    if status != OK:
        msg = lib().mfmg_last_error_message().decode()
        raise MfmgError(status, f"{lib().mfmg_status_string(status).decode()}: {msg}")


def _ptr(t):
    return None if t is None else c_void_p(t.data_ptr())


def _batch(x, y):
    """mfmg_batch of a CUDA tensor x (rows = its first dimension) and y (None: NULL)."""
    return mfmg_batch(x.data_ptr(), None if y is None else y.data_ptr(), x.shape[0])


def _stream():
    import torch
    return c_void_p(torch.cuda.current_stream().cuda_stream)


def make_desc(*, widths, act=0, loss=1, optimizer=0, meta=0, precision=0, has_bias=True, rows=1,
              val_rows=1, sgd_lr=0.1, adam_b1=0.9, adam_b2=0.999, adam_eps=1e-8,
              kind=0, **transformer) -> mfmg_problem_desc:
    d = mfmg_problem_desc()
    d.kind = kind
    d.n_layers = len(widths) - 1
    for i, w in enumerate(widths):
        d.widths[i] = int(w)
    d.act, d.loss, d.optimizer, d.meta, d.precision = act, loss, optimizer, meta, precision
    d.has_bias = int(bool(has_bias))
    d.rows, d.val_rows = rows, val_rows
    d.sgd_lr, d.adam_b1, d.adam_b2, d.adam_eps = sgd_lr, adam_b1, adam_b2, adam_eps
    for k, v in transformer.items():
        setattr(d, k, v)
    return d


class Problem:
    """Owns an mfmg_problem_t handle."""

    def __init__(self, desc: mfmg_problem_desc):
        self._h = c_void_p()
        check(lib().mfmg_problem_create(ctypes.byref(desc), ctypes.byref(self._h)))
        self.desc = desc

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.mfmg_problem_destroy(h)
            self._h = c_void_p()

    @property
    def handle(self):
        return self._h

    def mfmg_query_sizes(self, T: int) -> mfmg_sizes:
        s = mfmg_sizes()
        check(lib().mfmg_query_sizes(self._h, T, ctypes.byref(s)))
        return s

    def workspace(self, nbytes: int, device="cuda"):
        """A 256-byte-aligned uint8 CUDA tensor of at least nbytes (torch allocation)."""
        import torch
        return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)

    def mfmg_inner_step(self, theta, opt_state, eta, x, y, step_index, theta_next,
                        opt_state_next=None, grad_out=None, loss_out=None, ws=None):
        b = _batch(x, y)
        if ws is None:
            ws = self.workspace(self.mfmg_query_sizes(1).step_workspace_bytes, theta.device)
        check(lib().mfmg_inner_step(self._h, _ptr(theta), _ptr(opt_state), _ptr(eta),
                                    ctypes.byref(b), step_index, _ptr(theta_next),
                                    _ptr(opt_state_next), _ptr(grad_out), _ptr(loss_out),
                                    _ptr(ws), ws.numel(), _stream()))

    def mfmg_hvp_fwd_over_rev(self, theta, eta, x, y, step_index, v, grad_out, hvp_out,
                              mvp_out=None, ws=None):
        b = _batch(x, y)
        if ws is None:
            ws = self.workspace(self.mfmg_query_sizes(1).step_workspace_bytes, theta.device)
        check(lib().mfmg_hvp_fwd_over_rev(self._h, _ptr(theta), _ptr(eta), ctypes.byref(b),
                                          step_index, _ptr(v), _ptr(grad_out), _ptr(hvp_out),
                                          _ptr(mvp_out), _ptr(ws), ws.numel(), _stream()))

    def mfmg_meta_grad(self, theta0, opt_state0, eta, xs, ys, vx, vy, d_eta_out,
                       val_loss_out=None, ws=None) -> int:
        """Returns peak bytes."""
        T = len(xs)
        arr = (mfmg_batch * T)(*[_batch(x, y) for x, y in zip(xs, ys)])
        vb = _batch(vx, vy)
        if ws is None:
            ws = self.workspace(self.mfmg_query_sizes(T).workspace_bytes, theta0.device)
        peak = c_size_t(0)
        check(lib().mfmg_meta_grad(self._h, _ptr(theta0), _ptr(opt_state0), _ptr(eta), arr, T,
                                   ctypes.byref(vb), _ptr(d_eta_out), _ptr(val_loss_out),
                                   ctypes.byref(peak), _ptr(ws), ws.numel(), _stream()))
        return peak.value

    def mfmg_meta_grad_noalloc(self, theta0, opt_state0, eta, xs, ys, vx, vy, d_eta_out,
                               val_loss_out=None) -> int:
        """mfmg_meta_grad on the library's static scratch (no workspace); returns peak bytes."""
        T = len(xs)
        arr = (mfmg_batch * T)(*[_batch(x, y) for x, y in zip(xs, ys)])
        vb = _batch(vx, vy)
        peak = c_size_t(0)
        check(lib().mfmg_meta_grad_noalloc(self._h, _ptr(theta0), _ptr(opt_state0), _ptr(eta),
                                           arr, T, ctypes.byref(vb), _ptr(d_eta_out),
                                           _ptr(val_loss_out), ctypes.byref(peak), _stream()))
        return peak.value


def mfmg_check_finite(x, ws=None) -> int:
    """Number of NaN / infinite entries of the float32 CUDA tensor x (synchronises the
    current stream); raises MfmgError (status ERR_NUMERIC) when it is not zero."""
    import torch
    if ws is None:
        ws = torch.empty(256, dtype=torch.uint8, device=x.device)
    n = c_size_t(0)
    check(lib().mfmg_check_finite(_ptr(x), x.numel(), ctypes.byref(n), _ptr(ws), ws.numel(),
                                  _stream()))
    return n.value


def mfmg_timing_enable(enable: bool) -> None:
    check(lib().mfmg_timing_enable(int(enable)))


def mfmg_timing_read(kernel_class: int):
    n = c_int(0)
    ms = c_double(0.0)
    check(lib().mfmg_timing_read(kernel_class, ctypes.byref(n), ctypes.byref(ms)))
    return n.value, ms.value
