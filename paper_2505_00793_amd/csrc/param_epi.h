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

// 16-byte load of 4 consecutive floats at a 16-byte aligned index.
__device__ __forceinline__ void ld4v(const float* __restrict__ p, long idx, float* out) {
  const float4 v = *reinterpret_cast<const float4*>(p + idx);
  out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
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

// Inputs of the per-parameter arithmetic for up to 4 consecutive parameters,
// loaded ahead of it so that a thread can keep many groups in flight.  Which
// slots hold what depends on the mode (see param_load).
struct ParamIn {
  float x[3][4];
};

// The arrays whose values the arithmetic of this mode needs, by input slot
// (null: slot unused).
template <typename T>
__device__ __forceinline__ void param_sources(const ParamArgs<T>& P, const float* (&src)[3]) {
  src[0] = src[1] = src[2] = nullptr;
  switch (P.mode) {
    case P_UPD_SGD_PP: src[0] = P.theta; src[1] = P.eta; return;
    case P_UPD_SGD_FIXED: src[0] = P.theta; return;
    case P_UPD_ADAM: src[0] = P.theta; src[1] = P.m_in; src[2] = P.v_in; return;
    case P_SEED_SGD_PP: src[1] = P.eta; return;
    case P_REV_SGD_PP: src[0] = P.thetabar; src[1] = P.eta; src[2] = P.first ? nullptr : P.etabar; return;
    case P_REV_SGD_FIXED:
    case P_REV_ADAM: src[0] = P.thetabar; return;
    default: return;
  }
}

// Loads the inputs of cnt (1..4) consecutive parameters starting at flat index idx.
template <typename T>
__device__ __forceinline__ void param_load(const ParamArgs<T>& P, long idx, int cnt, ParamIn& in) {
  const bool vec = cnt == 4 && (idx & 3) == 0;
  const float* src[3];
  param_sources(P, src);
#pragma unroll
  for (int s = 0; s < 3; ++s)
    if (src[s]) ld4(src[s], idx, cnt, vec, in.x[s]);
}

// The arithmetic and stores for cnt (1..4) consecutive parameters at flat index
// idx, given their inputs.  cv receives the values for the operand copies (new
// theta for the update modes, the next tangent for the SGD seed/reverse modes,
// 0 otherwise).
template <typename T>
__device__ __forceinline__ void param_finish(const ParamArgs<T>& P, long idx, int cnt,
                                             const ParamIn& in, const float* g, const float* hv,
                                             float* cv) {
  const bool vec = cnt == 4 && (idx & 3) == 0;
  switch (P.mode) {
    case P_UPD_SGD_PP:
    case P_UPD_SGD_FIXED: {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float lam = P.mode == P_UPD_SGD_PP ? expf(in.x[1][k]) : P.lr;
        cv[k] = in.x[0][k] - lam * g[k];
      }
      st4(P.theta_next, idx, cnt, vec, cv);
      if (P.grad_out) st4(P.grad_out, idx, cnt, vec, g);
      return;
    }
    case P_UPD_ADAM: {
      float m[4], v[4];
      const float lam = expf(P.eta[P.layer]);
      const float om = P.eta[P.n_layers];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float m0 = P.m_in ? in.x[1][k] : 0.0f, v0 = P.v_in ? in.x[2][k] : 0.0f;
        m[k] = P.b1 * m0 + (1.0f - P.b1) * g[k];
        v[k] = P.b2 * v0 + (1.0f - P.b2) * g[k] * g[k];
        const float u = (m[k] / P.k1) / (sqrtf(v[k] / P.k2) + P.eps);
        cv[k] = in.x[0][k] - lam * (u + om * in.x[0][k]);
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
#pragma unroll
      for (int k = 0; k < 4; ++k)
        cv[k] = P.mode == P_SEED_SGD_PP ? -expf(in.x[1][k]) * g[k]
                : P.mode == P_SEED_SGD_FIXED ? -P.lr * g[k] : 0.0f;
      st4(P.thetabar, idx, cnt, vec, g);
      return;
    }
    case P_REV_SGD_PP: {
      float tb[4], eb[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float lam = expf(in.x[1][k]);
        const float e = -lam * g[k] * in.x[0][k];
        eb[k] = P.first ? e : in.x[2][k] + e;
        tb[k] = in.x[0][k] + hv[k];
        cv[k] = -lam * tb[k];
      }
      st4(P.etabar, idx, cnt, vec, eb);
      st4(P.thetabar, idx, cnt, vec, tb);
      return;
    }
    case P_REV_SGD_FIXED:
    case P_REV_ADAM: {
      float tb[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        tb[k] = in.x[0][k] + hv[k];
        cv[k] = P.mode == P_REV_SGD_FIXED ? -P.lr * tb[k] : 0.0f;
      }
      st4(P.thetabar, idx, cnt, vec, tb);
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

// Loads, arithmetic and stores of cnt (1..4) consecutive parameters.
template <typename T>
__device__ __forceinline__ void param_apply(const ParamArgs<T>& P, long idx, int cnt,
                                            const float* g, const float* hv, float* cv) {
  ParamIn in;
  param_load(P, idx, cnt, in);
  param_finish(P, idx, cnt, in, g, hv, cv);
}

// One parameter (the bias reductions).
template <typename T>
__device__ __forceinline__ float param_elem(const ParamArgs<T>& P, long idx, float g, float hv) {
  float g4[4] = {g, 0.f, 0.f, 0.f}, h4[4] = {hv, 0.f, 0.f, 0.f}, cv[4];
  param_apply(P, idx, 1, g4, h4, cv);
  return cv[0];
}

}  // namespace mfmg
