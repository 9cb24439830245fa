"""Float64 CPU oracle for the MixFlow-MG meta-gradient.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it.  It shares no code with the
HIP path; the only common module is ``workloads`` (seeded inputs, no method
arithmetic).

What it computes is the plain quantity dV/deta of the truncated bilevel
problem (Section 2.1, eq. bptt_bilevel): T inner updates
(theta_{i+1}, upsilon_{i+1}) = Upsilon(dL/dtheta_i, theta_i, upsilon_i, eta)
(Section 3, eq. reparam), then V(theta_T, val).  The route is the paper's
standard Truncated-BPTT (Algorithm 1): reverse-mode differentiation through
the unrolled inner loop, whose inner gradients are themselves built with
reverse mode and kept differentiable (reverse-over-reverse).  Every tensor is
torch.float64 on the CPU.

Pins (see tests/test_oracle_*.py): the closed-form meta-gradient of SGD on a
quadratic loss; complex-step and central finite differences in eta against an
independent numpy implementation with hand-written gradients; Hessian
symmetry u.Hv = v.Hu; forward-over-reverse == reverse-over-reverse HVPs;
brute-force Hessians; the T=1 closed forms; the step-checkpointed mode
against the whole-graph mode; library cross-checks (AdamW, log-softmax,
layer norm, attention).

The optional bf16-emulation mode (``bf16=True``) rounds every GEMM operand to
bfloat16 (round-to-nearest-even) with straight-through derivatives.  Its
parity against the fp64 mode is by construction only ("parity unpinned" for
the rounding pattern itself; the unrounded mode is pinned).
"""
from .metagrad import (meta_grad, meta_grad_checkpointed, unroll, inner_step, grad_and_loss,
                       hvp_rev_rev, hvp_rev_fwd, mvp_rev_rev, val_loss_of_eta)

__all__ = ["meta_grad", "meta_grad_checkpointed", "unroll", "inner_step", "grad_and_loss",
           "hvp_rev_rev", "hvp_rev_fwd", "mvp_rev_rev", "val_loss_of_eta"]
