// Per-parameter epilogue shared by the backward-weight GEMMs and the bias
// reductions: given g = dL/dtheta and hv = (H v) for a parameter, apply the
// inner update (forward unroll), seed the reverse sweep (validation pass), or
// accumulate one reverse step of the recurrence for dV/deta.
//
// Reverse step of SGD with per-parameter log learning rates (Section 3,
// eq. bptt_recur with Upsilon = theta - exp(eta) g): the incoming adjoint
// tb = bar theta_{i+1} gives the tangent v = tb dUpsilon/dg = -exp(eta) tb
// (the "normal VJP" of eq. vhp_to_hvp), then
//   bar eta   += tb dUpsilon/deta = -exp(eta) g tb
//   bar theta  = tb dUpsilon/dtheta + H v = tb + hv
// and the next step's tangent is -exp(eta) bar theta.
#pragma once

#include "kernels.h"

namespace mfmg {

// Up to four consecutive parameters: loaded inputs, outputs to store.
struct P4 {
  float th[4], et[4], tb[4], eb[4], m[4], v[4];
};

__device__ __forceinline__ void ld4(const float* __restrict__ p, long idx, int cnt, bool vec,
                                    float* out) {
  if (vec) {
    const float4 v = *reinterpret_cast<const float4*>(p + idx);
    out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) out[k] = k < cnt ? p[idx + k] : 0.0f;
  }
}

__device__ __forceinline__ void st4(float* __restrict__ p, long idx, int cnt, bool vec,
                                    const float* v) {
  if (vec) {
    *reinterpret_cast<float4*>(p + idx) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (k < cnt) p[idx + k] = v[k];
  }
}

// cnt (1..4) consecutive parameters starting at flat index idx.  All loads are
// issued before any store.  cv receives the values for the operand copies
// (new theta for the update modes, the next tangent for the SGD seed/reverse
// modes, 0 otherwise).
template <typename T>
__device__ __forceinline__ void param_apply(const ParamArgs<T>& P, long idx, int cnt,
                                            const float* g, const float* hv, float* cv) {
  const bool vec = cnt == 4 && (idx & 3) == 0;
  float a[4], b[4], c[4];
  switch (P.mode) {
    case P_UPD_SGD_PP:
    case P_UPD_SGD_FIXED: {
      ld4(P.theta, idx, cnt, vec, a);
      if (P.mode == P_UPD_SGD_PP) ld4(P.eta, idx, cnt, vec, b);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float lam = P.mode == P_UPD_SGD_PP ? expf(b[k]) : P.lr;
        cv[k] = a[k] - lam * g[k];
      }
      st4(P.theta_next, idx, cnt, vec, cv);
      if (P.grad_out) st4(P.grad_out, idx, cnt, vec, g);
      return;
    }
    case P_UPD_ADAM: {
      ld4(P.theta, idx, cnt, vec, a);
      float m[4] = {0.f, 0.f, 0.f, 0.f}, v[4] = {0.f, 0.f, 0.f, 0.f};
      if (P.m_in) ld4(P.m_in, idx, cnt, vec, m);
      if (P.v_in) ld4(P.v_in, idx, cnt, vec, v);
      const float lam = expf(P.eta[P.layer]);
      const float om = P.eta[P.n_layers];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        m[k] = P.b1 * m[k] + (1.0f - P.b1) * g[k];
        v[k] = P.b2 * v[k] + (1.0f - P.b2) * g[k] * g[k];
        const float u = (m[k] / P.k1) / (sqrtf(v[k] / P.k2) + P.eps);
        cv[k] = a[k] - lam * (u + om * a[k]);
      }
      st4(P.theta_next, idx, cnt, vec, cv);
      st4(P.m_out, idx, cnt, vec, m);
      st4(P.v_out, idx, cnt, vec, v);
      if (P.g_save) st4(P.g_save, idx, cnt, vec, g);
      if (P.grad_out) st4(P.grad_out, idx, cnt, vec, g);
      return;
    }
    case P_SEED_SGD_PP:
    case P_SEED_SGD_FIXED:
    case P_SEED_ADAM: {
      if (P.mode == P_SEED_SGD_PP) ld4(P.eta, idx, cnt, vec, b);
#pragma unroll
      for (int k = 0; k < 4; ++k)
        cv[k] = P.mode == P_SEED_SGD_PP ? -expf(b[k]) * g[k]
                : P.mode == P_SEED_SGD_FIXED ? -P.lr * g[k] : 0.0f;
      st4(P.thetabar, idx, cnt, vec, g);
      return;
    }
    case P_REV_SGD_PP: {
      ld4(P.thetabar, idx, cnt, vec, a);
      ld4(P.eta, idx, cnt, vec, b);
      if (!P.first) ld4(P.etabar, idx, cnt, vec, c);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float lam = expf(b[k]);
        const float eb = -lam * g[k] * a[k];
        c[k] = P.first ? eb : c[k] + eb;
        a[k] = a[k] + hv[k];
        cv[k] = -lam * a[k];
      }
      st4(P.etabar, idx, cnt, vec, c);
      st4(P.thetabar, idx, cnt, vec, a);
      return;
    }
    case P_REV_SGD_FIXED:
    case P_REV_ADAM: {
      ld4(P.thetabar, idx, cnt, vec, a);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        a[k] = a[k] + hv[k];
        cv[k] = P.mode == P_REV_SGD_FIXED ? -P.lr * a[k] : 0.0f;
      }
      st4(P.thetabar, idx, cnt, vec, a);
      return;
    }
    case P_HVP: {
      if (P.grad_out) st4(P.grad_out, idx, cnt, vec, g);
      st4(P.hvp_out, idx, cnt, vec, hv);
#pragma unroll
      for (int k = 0; k < 4; ++k) cv[k] = 0.0f;
      return;
    }
    case P_STORE_G: {
      st4(P.grad_out, idx, cnt, vec, g);
#pragma unroll
      for (int k = 0; k < 4; ++k) cv[k] = 0.0f;
      return;
    }
  }
}

// One parameter (the bias reductions).
template <typename T>
__device__ __forceinline__ float param_elem(const ParamArgs<T>& P, long idx, float g, float hv) {
  float g4[4] = {g, 0.f, 0.f, 0.f}, h4[4] = {hv, 0.f, 0.f, 0.f}, cv[4];
  param_apply(P, idx, 1, g4, h4, cv);
  return cv[0];
}

}  // namespace mfmg
