// Per-parameter epilogue shared by the backward-weight GEMMs and the bias
// reductions: given g = dL/dtheta and hv = (H v) for one parameter, apply the
// inner update (forward unroll), seed the reverse sweep (validation pass), or
// accumulate one reverse step of the recurrence for dV/deta.
#pragma once

#include "kernels.h"

namespace mfmg {

// Returns the value the caller stores into the operand copies (new theta for
// the update modes, the next tangent v for the SGD seed/reverse modes).
//
// Reverse step of SGD with per-parameter log learning rates (Section 3,
// eq. bptt_recur with Upsilon = theta - exp(eta) g): the incoming adjoint
// tb = bar theta_{i+1} gives the tangent v = tb dUpsilon/dg = -exp(eta) tb
// (the "normal VJP" of eq. vhp_to_hvp), then
//   bar eta   += tb dUpsilon/deta = -exp(eta) g tb
//   bar theta  = tb dUpsilon/dtheta + H v = tb + hv
// and the next step's tangent is -exp(eta) bar theta.
template <typename T>
__device__ __forceinline__ float param_elem(const ParamArgs<T>& P, long idx, float g, float hv) {
  switch (P.mode) {
    case P_UPD_SGD_PP: {
      float t1 = P.theta[idx] - expf(P.eta[idx]) * g;
      P.theta_next[idx] = t1;
      if (P.grad_out) P.grad_out[idx] = g;
      return t1;
    }
    case P_UPD_SGD_FIXED: {
      float t1 = P.theta[idx] - P.lr * g;
      P.theta_next[idx] = t1;
      if (P.grad_out) P.grad_out[idx] = g;
      return t1;
    }
    case P_UPD_ADAM: {
      float m = P.m_in ? P.m_in[idx] : 0.0f;
      float v = P.v_in ? P.v_in[idx] : 0.0f;
      float m1 = P.b1 * m + (1.0f - P.b1) * g;
      float v1 = P.b2 * v + (1.0f - P.b2) * g * g;
      float u = (m1 / P.k1) / (sqrtf(v1 / P.k2) + P.eps);
      float lam = expf(P.eta[P.layer]);
      float om = P.eta[P.n_layers];
      float th = P.theta[idx];
      float t1 = th - lam * (u + om * th);
      P.theta_next[idx] = t1;
      P.m_out[idx] = m1;
      P.v_out[idx] = v1;
      if (P.g_save) P.g_save[idx] = g;
      if (P.grad_out) P.grad_out[idx] = g;
      return t1;
    }
    case P_SEED_SGD_PP:
      P.thetabar[idx] = g;
      return -expf(P.eta[idx]) * g;
    case P_SEED_SGD_FIXED:
      P.thetabar[idx] = g;
      return -P.lr * g;
    case P_SEED_ADAM:
      P.thetabar[idx] = g;
      return 0.0f;
    case P_REV_SGD_PP: {
      float lam = expf(P.eta[idx]);
      float tb = P.thetabar[idx];
      float eb = -lam * g * tb;
      P.etabar[idx] = P.first ? eb : P.etabar[idx] + eb;
      float tb2 = tb + hv;
      P.thetabar[idx] = tb2;
      return -lam * tb2;
    }
    case P_REV_SGD_FIXED: {
      float tb2 = P.thetabar[idx] + hv;
      P.thetabar[idx] = tb2;
      return -P.lr * tb2;
    }
    case P_REV_ADAM:
      P.thetabar[idx] += hv;
      return 0.0f;
    case P_HVP:
      if (P.grad_out) P.grad_out[idx] = g;
      P.hvp_out[idx] = hv;
      return 0.0f;
  }
  return 0.0f;
}

}  // namespace mfmg
