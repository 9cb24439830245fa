// Elementwise and reduction kernels of the meta-gradient path (gfx950).
//
// All are HBM- or latency-bound: 64-lane wavefront reductions, coalesced
// row-major traffic, LDS-staged transposes where a second layout is written.
#include <algorithm>

#include "kernels.h"
#include "param_epi.h"

namespace mfmg {

namespace {

inline int cdiv(long a, long b) { return (int)((a + b - 1) / b); }

// ------------------------------------------------------------------------------------
// float32 [rows][cols] -> operand copies in both layouts, through a 64x64 LDS tile.
// ------------------------------------------------------------------------------------
// Several matrices of one shape per launch: z = job * batch + batch index.
template <typename T>
struct ConvPtrs {
  const float* src;
  T* dst;
  T* dstT;
};
template <typename T>
__device__ __forceinline__ ConvPtrs<T> conv_ptrs(const ConvJobs<T>& J, int batch, long s_src,
                                                 long s_dst, long s_dstT) {
  const int job = blockIdx.z / batch, bz = blockIdx.z - job * batch;
  ConvPtrs<T> p;
  p.src = J.src[job] + bz * s_src;
  p.dst = J.dst[job] ? J.dst[job] + bz * s_dst : nullptr;
  p.dstT = J.dstT[job] ? J.dstT[job] + bz * s_dstT : nullptr;
  return p;
}

template <typename T>
__global__ void __launch_bounds__(256) convert_kernel(ConvJobs<T> J, int batch, int rows,
                                                      int cols, int lds, int ldd, int lddT,
                                                      long s_src, long s_dst, long s_dstT) {
  __shared__ float tile[64][65];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const ConvPtrs<T> P = conv_ptrs(J, batch, s_src, s_dst, s_dstT);
  const float* src = P.src;
  T* dst = P.dst;
  T* dstT = P.dstT;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tx;
    float v = 0.0f;
    if (r < rows && c < cols) {
      v = src[(long)r * lds + c];
      if (dst) dst[(long)r * ldd + c] = Elem<T>::from_float(v);
    }
    tile[i][tx] = v;
  }
  if (!dstT) return;
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) dstT[(long)c * lddT + r] = Elem<T>::from_float(tile[tx][i]);
  }
}

// The same with 16-byte accesses: each thread converts 4 consecutive columns of a
// row (float4 in, 4 elements out) and writes the transposed copy 4 consecutive
// rows at a time.  Requires lds, ldd, lddT and the batch strides to be
// multiples of 4 and the arrays aligned to their 4-element width.
template <typename T>
__global__ void __launch_bounds__(256) convert_vec_kernel(ConvJobs<T> J, int batch, int rows,
                                                          int cols, int lds, int ldd, int lddT,
                                                          long s_src, long s_dst, long s_dstT) {
  __shared__ __attribute__((aligned(16))) float tile[64][68];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const ConvPtrs<T> P = conv_ptrs(J, batch, s_src, s_dst, s_dstT);
  const float* src = P.src;
  T* dst = P.dst;
  T* dstT = P.dstT;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int c = c0 + tx * 4;
  if ((cols & 3) == 0) {
    // every 16-byte chunk lies wholly inside or outside the matrix: the thread's
    // four rows are requested at once, from indices clamped into it, and the
    // chunks outside are zeroed on their way to LDS
    const int cl = min(c, cols - 4);
    float4 x[4];
#pragma unroll
    for (int it = 0; it < 4; ++it)
      x[it] = *reinterpret_cast<const float4*>(src + (long)min(r0 + ty + 16 * it, rows - 1) * lds +
                                               cl);
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int i = ty + 16 * it, r = r0 + i;
      const bool in = r < rows && c < cols;
      const float4 v = in ? x[it] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      if (in && dst) store4(dst + (long)r * ldd + c, v.x, v.y, v.z, v.w);
      *reinterpret_cast<float4*>(&tile[i][tx * 4]) = v;
    }
  } else {
    for (int i = ty; i < 64; i += 16) {
      const int r = r0 + i;
      float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      if (r < rows) {
        if (c + 4 <= cols) {
          const float4 x = *reinterpret_cast<const float4*>(src + (long)r * lds + c);
          v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
          if (dst) store4(dst + (long)r * ldd + c, v[0], v[1], v[2], v[3]);
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k)
            if (c + k < cols) {
              v[k] = src[(long)r * lds + c + k];
              if (dst) dst[(long)r * ldd + c + k] = Elem<T>::from_float(v[k]);
            }
        }
      }
      *reinterpret_cast<float4*>(&tile[i][tx * 4]) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
  if (!dstT) return;
  __syncthreads();
  const int r = r0 + tx * 4;
  for (int j = ty; j < 64; j += 16) {
    const int cc = c0 + j;
    if (cc >= cols || r >= rows) continue;
    const float w0 = tile[tx * 4][j], w1 = tile[tx * 4 + 1][j], w2 = tile[tx * 4 + 2][j],
                w3 = tile[tx * 4 + 3][j];
    if (r + 4 <= rows) {
      store4(dstT + (long)cc * lddT + r, w0, w1, w2, w3);
    } else {
      const float w[4] = {w0, w1, w2, w3};
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (r + k < rows) dstT[(long)cc * lddT + r + k] = Elem<T>::from_float(w[k]);
    }
  }
}

// bf16 / float [rows][ld] -> its transpose [cols][ldT], through a 64x64 LDS tile;
// the transposed copies of the loss head's outputs.  Two matrices per launch
// (z = 0, 1; the second may be null).
template <typename T>
__global__ void __launch_bounds__(256) transpose_kernel(const T* __restrict__ a0,
                                                        const T* __restrict__ a1, int rows,
                                                        int cols, int ld, T* t0, T* t1, int ldT) {
  __shared__ float tile[64][65];
  const T* src = blockIdx.z ? a1 : a0;
  T* dst = blockIdx.z ? t1 : t0;
  if (!src || !dst) return;
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tx;
    tile[i][tx] = (r < rows && c < cols) ? Elem<T>::to_float(src[(long)r * ld + c]) : 0.0f;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) dst[(long)c * ldT + r] = Elem<T>::from_float(tile[tx][i]);
  }
}

// bf16 version: a 64 x 64 tile goes in with one 16-byte load per 8 elements
// and out with one 16-byte store per 8 transposed elements.  Requires rows, ld,
// ldT and the batch strides to be multiples of 8 and ld >= roundup8(cols): cols
// itself may be ragged, in which case the loads read the rows' padding up to
// the next multiple of 8 (those lanes land in LDS but are never stored) and the
// output rows past cols are skipped.
// blockIdx.z = job * batch + matrix; matrix m of job j is src[j] + m s_src.
__global__ void __launch_bounds__(256) transpose_bf16_kernel(TrJobs J, int batch, int rows,
                                                             int cols, int ld, int ldT,
                                                             long s_src, long s_dst) {
  __shared__ bf16_t tile[64][64 + 2];
  const int job = blockIdx.z / batch, m = blockIdx.z - job * batch;
  const bf16_t* src = J.src[job] + m * s_src;
  bf16_t* dst = J.dst[job] + m * s_dst;
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = threadIdx.x + 256 * k, r = i >> 3, ch = (i & 7) * 8;
    union {
      uint4 v;
      bf16_t e[8];
    } u;
    u.v = make_uint4(0, 0, 0, 0);
    if (r0 + r < rows && c0 + ch < cols)
      u.v = *reinterpret_cast<const uint4*>(src + (long)(r0 + r) * ld + c0 + ch);
#pragma unroll
    for (int e = 0; e < 8; ++e) tile[r][ch + e] = u.e[e];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = threadIdx.x + 256 * k, c = i >> 3, rr = (i & 7) * 8;
    if (c0 + c >= cols || r0 + rr >= rows) continue;
    union {
      uint4 v;
      bf16_t e[8];
    } u;
#pragma unroll
    for (int e = 0; e < 8; ++e) u.e[e] = tile[rr + e][c];
    *reinterpret_cast<uint4*>(dst + (long)(c0 + c) * ldT + r0 + rr) = u.v;
  }
}

// ------------------------------------------------------------------------------------
// Bias entries: column sums of dZ (and its tangent) over the batch rows, read
// from the transposed copies (one wavefront per column, contiguous reads),
// then the per-parameter epilogue.  VEC: rows start 16-byte aligned, so each
// lane reads 16 bytes at a time; the rows % (elements per 16 bytes) tail is
// read element by element.
// ------------------------------------------------------------------------------------
__device__ __forceinline__ float chunk_sum(uint4 u, const bf16_t*) {
  const unsigned w[4] = {u.x, u.y, u.z, u.w};
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < 4; ++k) s += __uint_as_float(w[k] << 16) + __uint_as_float(w[k] & 0xffff0000u);
  return s;
}
__device__ __forceinline__ float chunk_sum(uint4 u, const float*) {
  return (__uint_as_float(u.x) + __uint_as_float(u.y)) + (__uint_as_float(u.z) + __uint_as_float(u.w));
}

template <typename T, bool VEC>
__global__ void __launch_bounds__(256) bias_kernel(const T* __restrict__ dZT,
                                                   const T* __restrict__ dZdT, int ld, int rows,
                                                   ParamArgs<T> P) {
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (n >= P.nout) return;
  float g = 0.0f, hv = 0.0f;
  int r0 = 0;
  if constexpr (VEC) {
    constexpr int VE = Elem<T>::VE;
    const int full = rows / VE * VE;
    const T* a = dZT + (long)n * ld;
    const T* b = dZdT ? dZdT + (long)n * ld : nullptr;
    for (int r = lane * VE; r < full; r += 64 * VE) {
      g += chunk_sum(*reinterpret_cast<const uint4*>(a + r), a);
      if (b) hv += chunk_sum(*reinterpret_cast<const uint4*>(b + r), b);
    }
    r0 = full;
  }
  for (int r = r0 + lane; r < rows; r += 64) {
    g += Elem<T>::to_float(dZT[(long)n * ld + r]);
    if (dZdT) hv += Elem<T>::to_float(dZdT[(long)n * ld + r]);
  }
  g = wave_sum(g);
  hv = wave_sum(hv);
  if (lane == 0) {
    const float cv = param_elem(P, P.b_off + n, g, hv);
    if (P.outb) P.outb[n] = cv;
  }
}

// ------------------------------------------------------------------------------------
// Loss head, one wavefront per row.  Softmax cross-entropy:
//   p = softmax(z), l = logsumexp(z) - z_y, dL/dz = (alpha/N)(p - e_y);
// with the tangent zd of z (forward mode):
//   ldot = <p - e_y, zd>,  d(dL/dz) = (alpha/N) p (zd - <p, zd>).
// Squared error: l = |z - t|^2, dL/dz = (2 alpha/N)(z - t), ldot = 2<z - t, zd>,
// d(dL/dz) = (2 alpha/N) zd.  ldot/N is the mixed product
// (d^2 L / d alpha_n d theta) v of Section 3 (eq. vmp_to_mvp) for loss weights.
// ------------------------------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) loss_kernel(LossArgs<T> a) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.rows) return;
  const int C = a.C;
  // the row's padding columns C .. pad_to - 1 of dL/dz (and its tangent) are
  // zero, so that a product may contract over them
  if (C + lane < a.pad_to) {
    a.d[(long)row * a.ld + C + lane] = Elem<T>::from_float(0.0f);
    if (a.dual) a.dd[(long)row * a.ld + C + lane] = Elem<T>::from_float(0.0f);
  }
  const float* z = a.Z + (long)row * C;
  const float* zd = a.dual ? a.Zd + (long)row * C : nullptr;
  // dL/dz (and its tangent) of class c in both layouts
  auto put = [&](int c, float v, float vd) {
    a.d[(long)row * a.ld + c] = Elem<T>::from_float(v);
    if (a.direct_t) a.dT[(long)c * a.ldT + row] = Elem<T>::from_float(v);
    if (a.dual) {
      a.dd[(long)row * a.ld + c] = Elem<T>::from_float(vd);
      if (a.direct_t) a.ddT[(long)c * a.ldT + row] = Elem<T>::from_float(vd);
    }
  };
  float w = 1.0f;
  if (a.alpha_logits) w = 1.0f / (1.0f + expf(-a.alpha_logits[row]));
  const float scale = w * a.inv_n;
  float loss = 0.0f, ldot = 0.0f;
  const bool vec = (C & 3) == 0 && (a.ld & 3) == 0 &&
                   (reinterpret_cast<uintptr_t>(a.Z) & 15) == 0 &&
                   (!a.dual || ((reinterpret_cast<uintptr_t>(a.Zd) & 15) == 0));
  if (a.loss == 1 && vec) {
    // One pass for the log-sum-exp and the tangent dot: per lane a running max
    // m with se = sum exp(z - m) and sd = sum exp(z - m) zd, rescaled when m
    // grows; lanes are then combined at the wave's max.
    float m = -INFINITY, se = 0.0f, sd = 0.0f;
    for (int c = lane * 4; c < C; c += 256) {
      const float4 x = *reinterpret_cast<const float4*>(z + c);
      const float mn = fmaxf(m, fmaxf(fmaxf(x.x, x.y), fmaxf(x.z, x.w)));
      if (mn == -INFINITY) continue;
      const float r = m == mn ? 1.0f : expf(m - mn);
      const float e0 = expf(x.x - mn), e1 = expf(x.y - mn), e2 = expf(x.z - mn),
                  e3 = expf(x.w - mn);
      se = se * r + ((e0 + e1) + (e2 + e3));
      if (a.dual) {
        const float4 xd = *reinterpret_cast<const float4*>(zd + c);
        sd = sd * r + ((e0 * xd.x + e1 * xd.y) + (e2 * xd.z + e3 * xd.w));
      }
      m = mn;
    }
    const float M = wave_max(m);
    const float f = m == -INFINITY ? 0.0f : expf(m - M);
    const float SE = wave_sum(se * f);
    const float lse = M + logf(SE);
    int y = a.labels[row];
    if (y < 0 || y >= C) {  // invalid label: NaN loss, no target term
      y = -1;
      loss = NAN;
    } else {
      loss = lse - z[y];
    }
    float sdot = 0.0f;
    if (a.dual) {
      sdot = wave_sum(sd * f) / SE;   // sum_c p_c zd_c
      ldot = y >= 0 ? sdot - zd[y] : NAN;
    }
    for (int c = lane * 4; c < C; c += 256) {
      const float4 x = *reinterpret_cast<const float4*>(z + c);
      const float xs[4] = {x.x, x.y, x.z, x.w};
      float dv[4], ddv[4];
      float xds[4] = {0.f, 0.f, 0.f, 0.f};
      if (a.dual) {
        const float4 xd = *reinterpret_cast<const float4*>(zd + c);
        xds[0] = xd.x; xds[1] = xd.y; xds[2] = xd.z; xds[3] = xd.w;
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float p = expf(xs[k] - lse);
        dv[k] = scale * (p - (c + k == y ? 1.0f : 0.0f));
        ddv[k] = scale * p * (xds[k] - sdot);
      }
      store4(a.d + (long)row * a.ld + c, dv[0], dv[1], dv[2], dv[3]);
      if (a.dual) store4(a.dd + (long)row * a.ld + c, ddv[0], ddv[1], ddv[2], ddv[3]);
      if (a.direct_t) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          a.dT[(long)(c + k) * a.ldT + row] = Elem<T>::from_float(dv[k]);
          if (a.dual) a.ddT[(long)(c + k) * a.ldT + row] = Elem<T>::from_float(ddv[k]);
        }
      }
    }
  } else if (a.loss == 2) {
    // Squared error after the M-step map y_i = i (2 + sin y_{i-1})^cos y_{i-1},
    // mean over the C outputs.  Per element the map's value y_M and its first
    // and second derivatives in z are carried through the M steps in registers
    // (with h = d/dy ln f_i = cos^2 y / (2 + sin y) - sin y ln(2 + sin y):
    // f_i' = f_i h, f_i'' = f_i (h^2 + h')), so no step is stored.
    const float* t = a.targets + (long)row * C;
    const float invC = 1.0f / (float)C;
    for (int c = lane; c < C; c += 64) {
      float g = z[c], g1 = 1.0f, g2 = 0.0f;
      for (int i = 1; i <= a.map_M; ++i) {
        float sn, cs;
        sincosf(g, &sn, &cs);
        const float u = 2.0f + sn, lu = logf(u), iu = 1.0f / u;
        const float f = (float)i * expf(cs * lu);
        const float h = cs * cs * iu - sn * lu;
        const float hp = -cs * lu - 3.0f * sn * cs * iu - cs * cs * cs * iu * iu;
        const float f1 = f * h, f2 = f * (h * h + hp);
        g2 = f2 * g1 * g1 + f1 * g2;
        g1 = f1 * g1;
        g = f;
      }
      const float r = g - t[c];
      loss += r * r * invC;
      float vd = 0.0f;
      if (a.dual) {
        const float zdc = zd[c];
        ldot += 2.0f * invC * r * g1 * zdc;
        vd = 2.0f * scale * invC * zdc * (g1 * g1 + r * g2);
      }
      put(c, 2.0f * scale * invC * r * g1, vd);
    }
    loss = wave_sum(loss);
    ldot = wave_sum(ldot);
  } else if (a.loss == 1) {
    float mx = -INFINITY;
    for (int c = lane; c < C; c += 64) mx = fmaxf(mx, z[c]);
    mx = wave_max(mx);
    float se = 0.0f;
    for (int c = lane; c < C; c += 64) se += expf(z[c] - mx);
    se = wave_sum(se);
    const float lse = mx + logf(se);
    int y = a.labels[row];
    if (y < 0 || y >= C) {  // invalid label: NaN loss, no target term
      y = -1;
      loss = NAN;
    } else {
      loss = lse - z[y];
    }
    float s = 0.0f;
    if (a.dual) {
      for (int c = lane; c < C; c += 64) s += expf(z[c] - lse) * zd[c];
      s = wave_sum(s);
      ldot = y >= 0 ? s - zd[y] : NAN;
    }
    for (int c = lane; c < C; c += 64) {
      const float p = expf(z[c] - lse);
      put(c, scale * (p - (c == y ? 1.0f : 0.0f)), a.dual ? scale * p * (zd[c] - s) : 0.0f);
    }
  } else {
    const float* t = a.targets + (long)row * C;
    for (int c = lane; c < C; c += 64) {
      const float r = z[c] - t[c];
      loss += r * r;
      if (a.dual) ldot += 2.0f * r * zd[c];
      put(c, 2.0f * scale * r, a.dual ? 2.0f * scale * zd[c] : 0.0f);
    }
    loss = wave_sum(loss);
    ldot = wave_sum(ldot);
  }
  if (lane == 0) {
    if (a.loss_rows) a.loss_rows[row] = loss;
    if (a.mvp_rows) a.mvp_rows[row] = ldot * a.inv_n;
    if (a.deta_rows) a.deta_rows[row] = w * (1.0f - w) * ldot * a.inv_n;
  }
}

// Deterministic single-workgroup weighted sum.
__global__ void __launch_bounds__(256) loss_reduce_kernel(const float* __restrict__ l,
                                                          const float* __restrict__ alpha_logits,
                                                          int rows, float inv_n, float* out) {
  __shared__ float red[256];
  float s = 0.0f;
  for (int r = threadIdx.x; r < rows; r += 256) {
    float w = alpha_logits ? 1.0f / (1.0f + expf(-alpha_logits[r])) : 1.0f;
    s += w * l[r];
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = red[0] * inv_n;
}

// ------------------------------------------------------------------------------------
// Adam, reverse step i before the dual pass.  With the step's recomputed
// (m', v') from (m_i, v_i, g_i), t = i + 1, k1 = 1 - b1^t, k2 = 1 - b2^t,
// D = sqrt(v'/k2) + eps, u = (m'/k1)/D, and incoming adjoints (tb, mb', vb'):
//   ub        = -lr tb                                (adjoint of u)
//   mb_tot    = mb' + ub / (k1 D)
//   vb_tot    = vb' - ub (m'/k1) / (D^2 2 sqrt(v'/k2) k2)   (0 where v' = 0)
//   v_g       = (1-b1) mb_tot + 2 (1-b2) g vb_tot     (tangent for the dual pass,
//                                                      the normal VJP of eq. vhp_to_hvp)
//   mb_i      = b1 mb_tot,  vb_i = b2 vb_tot
//   tb_i      = tb (1 - lr omega) + H v_g             (H v_g added by the dual pass)
//   d eta_l  += sum_layer -lr tb (u + omega theta)    (d lr / d eta_l = lr)
//   d omega  += sum_all   -lr tb theta
// ------------------------------------------------------------------------------------
// Blocks 0 .. tiles-1 take 16 x 64 tiles of W (coalesced reads of every stream,
// coalesced row-major tangent, the transposed tangent through an LDS tile in
// 32-byte runs); the remaining blocks take 256 bias entries each.  Each block
// writes the sums of its entries' eta and omega terms (fixed order) to
// partial[2 block ..].
template <typename T>
__device__ __forceinline__ void adam_vjp_elem(const AdamVjpArgs<T>& a, long idx, float& vg,
                                              float& pe, float& po) {
  const float g = a.g[idx], m = a.m[idx], v = a.v[idx], th = a.theta[idx];
  const float m1 = a.b1 * m + (1.0f - a.b1) * g;
  const float v1 = a.b2 * v + (1.0f - a.b2) * g * g;
  const float s = sqrtf(v1 / a.k2);
  const float D = s + a.eps;
  const float mh = m1 / a.k1;
  const float u = mh / D;
  const float lam = expf(a.eta[a.layer]);
  const float om = a.eta[a.n_layers];
  const float tb = a.thetabar[idx];
  const float ub = -lam * tb;
  const float mb = (a.first ? 0.0f : a.mbar[idx]) + ub / (a.k1 * D);
  const float vbt = (a.first ? 0.0f : a.vbar[idx]) +
                    (v1 > 0.0f ? -ub * mh / (D * D) / (2.0f * s * a.k2) : 0.0f);
  vg = (1.0f - a.b1) * mb + 2.0f * (1.0f - a.b2) * g * vbt;
  a.mbar[idx] = a.b1 * mb;
  a.vbar[idx] = a.b2 * vbt;
  a.thetabar[idx] = tb * (1.0f - lam * om);
  pe += -lam * tb * (u + om * th);
  po += -lam * tb * th;
}

template <typename T>
__device__ void adam_vjp_block(const AdamVjpArgs<T>& a, int blk, float* partial) {
  __shared__ float tile[16][65];
  __shared__ float red0[256], red1[256];
  const int tiles_n = (a.nout + 63) / 64;
  const int tiles = ((a.nin + 15) / 16) * tiles_n;
  const int tid = threadIdx.x;
  float pe = 0.0f, po = 0.0f;
  if (blk < tiles) {
    const int r0 = (blk / tiles_n) * 16, c0 = (blk % tiles_n) * 64;
    const int tx = tid & 63, ty = tid >> 6;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = ty + 4 * i, mm = r0 + r, nn = c0 + tx;
      float vg = 0.0f;
      if (mm < a.nin && nn < a.nout) {
        adam_vjp_elem(a, a.w_off + (long)mm * a.nout + nn, vg, pe, po);
        a.vW[(long)mm * a.ldW + nn] = Elem<T>::from_float(vg);
      }
      tile[r][tx] = vg;
    }
    __syncthreads();
    const int rr = tid & 15;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = (tid >> 4) + 16 * j, nn = c0 + c, mm = r0 + rr;
      if (nn < a.nout && mm < a.nin) a.vWT[(long)nn * a.ldWT + mm] = Elem<T>::from_float(tile[rr][c]);
    }
  } else {
    const long e = (long)(blk - tiles) * 256 + tid;
    if (a.b_off >= 0 && e < a.nout) {
      float vg = 0.0f;
      adam_vjp_elem(a, a.b_off + e, vg, pe, po);
      a.vb[e] = vg;
    }
  }
  red0[tid] = pe;
  red1[tid] = po;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (tid < o) {
      red0[tid] += red0[tid + o];
      red1[tid] += red1[tid + o];
    }
    __syncthreads();
  }
  if (tid == 0) {
    partial[0] = red0[0];
    partial[1] = red1[0];
  }
}

// The Adam reverse of every layer of one step in one launch: workgroups
// off[l] .. off[l + 1] - 1 take layer l, each writing its partial pair at its
// own index.
template <typename T>
struct AdamVjpLayers {
  AdamVjpArgs<T> a[MFMG_MAX_LAYERS];
  int off[MFMG_MAX_LAYERS + 1];
  int L;
};

template <typename T>
__global__ void __launch_bounds__(256) adam_vjp_kernel(AdamVjpLayers<T> A, float* partial) {
  int l = 0;
  while (l + 1 < A.L && (int)blockIdx.x >= A.off[l + 1]) ++l;
  adam_vjp_block(A.a[l], (int)blockIdx.x - A.off[l], partial + 2 * (long)blockIdx.x);
}

struct Offsets {
  int off[MFMG_MAX_LAYERS + 1];
};

// Per-layer sums of the adam_vjp_kernel partials, in a fixed order: thread t sums
// partials t, t + 1024, ... of each layer, waves combine by butterfly, and the 16
// wave sums of a layer are added in wave order; the weight-decay sums of the
// layers are then added in layer order.
__global__ void __launch_bounds__(1024) adam_reduce_kernel(const float* __restrict__ partial,
                                                           Offsets o, int n_layers, int first,
                                                           float* d_eta) {
  __shared__ float red[2][MFMG_MAX_LAYERS][16];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int l = 0; l < n_layers; ++l) {
    float s = 0.0f, so = 0.0f;
    for (int b = o.off[l] + threadIdx.x; b < o.off[l + 1]; b += 1024) {
      s += partial[2 * b];
      so += partial[2 * b + 1];
    }
    s = wave_sum(s);
    so = wave_sum(so);
    if (lane == 0) {
      red[0][l][w] = s;
      red[1][l][w] = so;
    }
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  float tot_om = 0.0f;
  for (int l = 0; l < n_layers; ++l) {
    float s = red[0][l][0], so = red[1][l][0];
    for (int k = 1; k < 16; ++k) {
      s += red[0][l][k];
      so += red[1][l][k];
    }
    d_eta[l] = (first ? 0.0f : d_eta[l]) + s;
    tot_om += so;
  }
  d_eta[n_layers] = (first ? 0.0f : d_eta[n_layers]) + tot_om;
}

// ------------------------------------------------------------------------------------
// Linear regression meta-gradient in one workgroup: squared loss
// L = (1/N)|X theta - y|^2, SGD theta' = theta - exp(eta) g, V on the
// validation batch.  Forward unroll with theta_t checkpoints, then the
// reverse sweep with the dual pass (r, rdot) = (X theta - y, X v):
// g = (2/N) X^T r, H v = (2/N) X^T rdot.
// 512 threads.  The batches are used in the order of the sweep: the T
// training batches, the validation batch, then the training batches again in
// reverse.  Each is staged in LDS (when it fits in 80 KB) with rows padded to a
// pitch of 16 (mod 32) floats, so that the four rows a quarter-wave reads with
// 16-byte accesses fall on distinct banks; the next batch's values are loaded
// into registers while the current one is used, so the sweep waits on global
// memory only for the first.  The checkpoints theta_t stay in LDS when
// (T + 1) d <= 4096.  Residuals take four threads per row (every fourth 16-byte
// group of the row, then a sum over the four lanes), X^T r takes 64 features x
// 8 row groups per pass with an ordered sum of the 8 partials.
// ------------------------------------------------------------------------------------
constexpr int LR_MAXD = 256;
constexpr int LR_MAXR = 1024;
constexpr int LR_MAXT = 64;
constexpr int LR_THREADS = 512;
constexpr int LR_RG = LR_THREADS / 64;   // row groups of the column pass
constexpr int LR_YPT = LR_MAXR / LR_THREADS;  // targets per thread
constexpr int LR_STAGE = 20480;  // floats of one batch staged in LDS, rows padded (80 KB)
constexpr int LR_PF = LR_STAGE / LR_THREADS;  // prefetched floats per thread (n <= LR_STAGE)
constexpr int LR_PF4 = LR_PF / 4;             // prefetched 16-byte groups per thread
constexpr int LR_CKPT = 4096;    // floats of checkpoints kept in LDS

struct LinregArgs {
  const float* theta0;
  const float* eta;
  const float* xs[LR_MAXT];  // device pointers of the T training batches
  const float* ys[LR_MAXT];
  int T, rows, d, vrows;
  int vec;                   // every batch 16-byte aligned and d % 4 == 0
  const float* vx;
  const float* vy;
  float* d_eta;
  float* val_loss;
  float* ckpt;  // (T + 1) x d
};

// Padded row pitch of a staged batch: d rounded up to 4, then to 16 (mod 32).
__host__ __device__ __forceinline__ int lr_spitch(int d) {
  const int p = (d + 3) & ~3;
  return p + ((16 - (p & 31)) & 31);
}
__host__ __device__ __forceinline__ bool lr_staged(int rows, int d) {
  return rows * lr_spitch(d) <= LR_STAGE;
}

// Batch k of the sweep (k = 0 .. 2T).
struct LrBatch {
  const float* X;
  const float* y;
  int rows;
};
__device__ __forceinline__ LrBatch lr_batch(const LinregArgs& a, int k) {
  if (k < a.T) return {a.xs[k], a.ys[k], a.rows};
  if (k == a.T) return {a.vx, a.vy, a.vrows};
  return {a.xs[2 * a.T - k], a.ys[2 * a.T - k], a.rows};
}

// Registers holding one batch on its way to LDS: 16-byte group tid + u *
// LR_THREADS of X (vec), or element tid + u * LR_THREADS, and y[tid].  The
// loads are unconditional (an index past the end reads the last element) so
// that a register is never both cleared and loaded: the compiler would then
// wait for every load in flight.
struct LrRegs {
  float x[LR_PF];   // vec: group u in x[4u .. 4u + 3]
  float y[LR_YPT];
};
template <bool VEC>
__device__ __forceinline__ void lr_load(const LrBatch& b, int d, LrRegs& g) {
  const int tid = threadIdx.x;
  if (lr_staged(b.rows, d)) {
    const int n = b.rows * d;
    if constexpr (VEC) {
      const float4* X4 = reinterpret_cast<const float4*>(b.X);
#pragma unroll
      for (int u = 0; u < LR_PF4; ++u) {
        const float4 v = X4[min(tid + u * LR_THREADS, n / 4 - 1)];
        g.x[4 * u] = v.x; g.x[4 * u + 1] = v.y; g.x[4 * u + 2] = v.z; g.x[4 * u + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int u = 0; u < LR_PF; ++u) g.x[u] = b.X[min(tid + u * LR_THREADS, n - 1)];
    }
  }
#pragma unroll
  for (int v = 0; v < LR_YPT; ++v) g.y[v] = b.y[min(tid + v * LR_THREADS, b.rows - 1)];
}
// Registers -> LDS (padded rows; the padding columns stay zero).  Callers
// synchronise before (the previous batch's readers are done) and after.
template <bool VEC>
__device__ __forceinline__ void lr_commit(const LrBatch& b, int d, const LrRegs& g, float* stage,
                                          float* ys) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int v = 0; v < LR_YPT; ++v)
    if (tid + v * LR_THREADS < b.rows) ys[tid + v * LR_THREADS] = g.y[v];
  if (!lr_staged(b.rows, d)) return;
  const int n = b.rows * d, P = lr_spitch(d);
  // element i = row * d + col goes to row * P + col; row and col advance by the
  // elements of one step without a division
  if constexpr (VEC) {
    const int st = 4 * LR_THREADS;
    const int qd = st / d, rd = st - qd * d;
    int row = 4 * tid / d, col = 4 * tid - row * d;
#pragma unroll
    for (int u = 0; u < LR_PF4; ++u) {
      if (4 * (tid + u * LR_THREADS) < n)
        *reinterpret_cast<float4*>(stage + row * P + col) =
            make_float4(g.x[4 * u], g.x[4 * u + 1], g.x[4 * u + 2], g.x[4 * u + 3]);
      row += qd;
      col += rd;
      while (col >= d) {
        col -= d;
        ++row;
      }
    }
  } else {
    const int qd = LR_THREADS / d, rd = LR_THREADS - qd * d;
    int row = tid / d, col = tid - row * d;
#pragma unroll
    for (int u = 0; u < LR_PF; ++u) {
      if (tid + u * LR_THREADS < n) stage[row * P + col] = g.x[u];
      row += qd;
      col += rd;
      if (col >= d) {
        col -= d;
        ++row;
      }
    }
  }
}

// Sum over the four lanes of a quad (DPP quad permutations, no LDS traffic).
__device__ __forceinline__ float quad_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, true));  // [1,0,3,2]
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, true));  // [2,3,0,1]
  return v;
}

// r[n] = X[n] . w - y[n] (and rd[n] = X[n] . u when DU).  Staged batches: four
// threads per row, thread q taking 16-byte groups q, q + 4, ... of the row (w
// and u zero past d, like the row's padding), and two rows (n and n + 128) per
// thread at once, sharing the reads of w and u; batches in global memory: one
// thread per row.  Returns this thread's share of sum_n r[n]^2.
template <bool DU>
__device__ float lr_rows_staged(const float* X, int P, const float* y, const float* w,
                                const float* u, int rows, int d, float* r, float* rd) {
  constexpr int RPP = LR_THREADS / 4;   // rows per pass and half
  const int q = threadIdx.x & 3;
  const int g4 = (d + 3) >> 2;
  const float4* w4 = reinterpret_cast<const float4*>(w);
  const float4* u4 = reinterpret_cast<const float4*>(u);
  float sq = 0.0f;
  for (int nb = 0; nb < rows; nb += 2 * RPP) {
    const int n0 = nb + (threadIdx.x >> 2), n1 = n0 + RPP;
    // rows past the end read the last row; their sums are not used
    const float4* x0 = reinterpret_cast<const float4*>(X + min(n0, rows - 1) * P);
    const float4* x1 = reinterpret_cast<const float4*>(X + min(n1, rows - 1) * P);
    float s0 = 0.0f, s1 = 0.0f, sd0 = 0.0f, sd1 = 0.0f;
#pragma unroll 2
    for (int j = q; j < g4; j += 4) {
      const float4 ww = w4[j], a = x0[j], b = x1[j];
      s0 += a.x * ww.x + a.y * ww.y + a.z * ww.z + a.w * ww.w;
      s1 += b.x * ww.x + b.y * ww.y + b.z * ww.z + b.w * ww.w;
      if (DU) {
        const float4 uu = u4[j];
        sd0 += a.x * uu.x + a.y * uu.y + a.z * uu.z + a.w * uu.w;
        sd1 += b.x * uu.x + b.y * uu.y + b.z * uu.z + b.w * uu.w;
      }
    }
    s0 = quad_sum(s0);
    s1 = quad_sum(s1);
    if (DU) {
      sd0 = quad_sum(sd0);
      sd1 = quad_sum(sd1);
    }
    if (q == 0) {
      if (n0 < rows) {
        const float res = s0 - y[n0];
        r[n0] = res;
        if (DU) rd[n0] = sd0;
        sq += res * res;
      }
      if (n1 < rows) {
        const float res = s1 - y[n1];
        r[n1] = res;
        if (DU) rd[n1] = sd1;
        sq += res * res;
      }
    }
  }
  __syncthreads();
  return sq;
}
template <bool DU>
__device__ float lr_rows_global(const float* X, const float* y, const float* w, const float* u,
                                int rows, int d, float* r, float* rd) {
  float sq = 0.0f;
  for (int n = threadIdx.x; n < rows; n += LR_THREADS) {
    const float* xr = X + (long)n * d;
    float s = 0.0f, sd = 0.0f;
    for (int j = 0; j < d; ++j) {
      const float x = xr[j];
      s += x * w[j];
      if (DU) sd += x * u[j];
    }
    const float res = s - y[n];
    r[n] = res;
    if (DU) rd[n] = sd;
    sq += res * res;
  }
  __syncthreads();
  return sq;
}

// out[j] = sum_n X[n][j] v[n] (and out2 with v2 when DU), j < d; X has row
// pitch P (LDS or global memory: separate instantiations, so that every access
// has a known address space; a flat access would wait for the next batch's
// loads).
template <bool DU>
__device__ void lr_cols(const float* X, int P, const float* v, const float* v2, int rows, int d,
                        float* part, float* part2, float* out, float* out2) {
  const int c = threadIdx.x & 63, q = threadIdx.x >> 6;
  for (int j0 = 0; j0 < d; j0 += 64) {
    const int j = j0 + c;
    float s = 0.0f, s2 = 0.0f;
    if (j < d) {
#pragma unroll 4
      for (int n = q; n < rows; n += LR_RG) {
        const float x = X[(long)n * P + j];
        s += x * v[n];
        if (DU) s2 += x * v2[n];
      }
    }
    part[q * 64 + c] = s;
    if (DU) part2[q * 64 + c] = s2;
    __syncthreads();
    if (threadIdx.x < 64 && j < d) {
      float a = 0.0f, b = 0.0f;
#pragma unroll
      for (int k = 0; k < LR_RG; ++k) {
        a += part[k * 64 + c];
        if (DU) b += part2[k * 64 + c];
      }
      out[j] = a;
      if (DU) out2[j] = b;
    }
    __syncthreads();
  }
}

// The column pass of a staged batch (row pitch P, a multiple of 4, zero past
// d): each thread takes a 16-byte group of 4 columns and every 32nd row, 16
// groups (64 columns) per round; the 32 partials of a column are then summed in
// order, 8 at a time by the 4 lanes of a quad, then across the quad.
constexpr int LR_CG = 16;                     // column groups per round
constexpr int LR_CRG = LR_THREADS / LR_CG;    // row groups
template <bool DU>
__device__ void lr_cols_staged(const float* X, int P, const float* v, const float* v2, int rows,
                               int d, float* part, float* part2, float* out, float* out2) {
  const int cg = threadIdx.x % LR_CG, q = threadIdx.x / LR_CG;
  for (int j0 = 0; j0 < d; j0 += 4 * LR_CG) {
    const int j = j0 + 4 * cg;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f), s2 = s;
    if (j < d) {
#pragma unroll 4
      for (int n = q; n < rows; n += LR_CRG) {
        const float4 x = *reinterpret_cast<const float4*>(X + n * P + j);
        const float vn = v[n];
        s.x += x.x * vn; s.y += x.y * vn; s.z += x.z * vn; s.w += x.w * vn;
        if (DU) {
          const float un = v2[n];
          s2.x += x.x * un; s2.y += x.y * un; s2.z += x.z * un; s2.w += x.w * un;
        }
      }
    }
    reinterpret_cast<float4*>(part)[q * LR_CG + cg] = s;
    if (DU) reinterpret_cast<float4*>(part2)[q * LR_CG + cg] = s2;
    __syncthreads();
    if (threadIdx.x < 4 * 4 * LR_CG) {
      // column c = threadIdx.x / 4 of the round, partials h * 8 .. h * 8 + 7
      const int c = threadIdx.x >> 2, h = threadIdx.x & 3;
      float a = 0.0f, b = 0.0f;
#pragma unroll
      for (int k = 0; k < LR_CRG / 4; ++k) {
        a += part[(h * (LR_CRG / 4) + k) * 4 * LR_CG + c];
        if (DU) b += part2[(h * (LR_CRG / 4) + k) * 4 * LR_CG + c];
      }
      a = quad_sum(a);
      if (DU) b = quad_sum(b);
      if (h == 0 && j0 + c < d) {
        out[j0 + c] = a;
        if (DU) out2[j0 + c] = b;
      }
    }
    __syncthreads();
  }
}

// One pass over batch b: residuals, then X^T r (and the tangents when DU).
template <bool DU>
__device__ float lr_pass(const LrBatch& b, int d, const float* stage, const float* ys,
                         const float* w, const float* u, float* r, float* rd, float* part,
                         float* part2, float* g, float* h) {
  float sq;
  if (lr_staged(b.rows, d)) {
    const int P = lr_spitch(d);
    sq = lr_rows_staged<DU>(stage, P, ys, w, u, b.rows, d, r, rd);
    lr_cols_staged<DU>(stage, P, r, rd, b.rows, d, part, part2, g, h);
  } else {
    sq = lr_rows_global<DU>(b.X, ys, w, u, b.rows, d, r, rd);
    lr_cols<DU>(b.X, d, r, rd, b.rows, d, part, part2, g, h);
  }
  return sq;
}

// VEC: every batch 16-byte aligned and d % 4 == 0 (16-byte prefetch loads).  The
// two forms are separate kernels so that the prefetch has one load site, whose
// registers the compiler then carries across the phase without copying them
// (a copy would wait for the loads it was meant to overlap).
template <bool VEC>
__global__ void __launch_bounds__(LR_THREADS) linreg_kernel(LinregArgs a) {
  __shared__ __attribute__((aligned(16))) float stage[LR_STAGE];
  __shared__ float ck[LR_CKPT];
  __shared__ __attribute__((aligned(16))) float th[LR_MAXD], vv[LR_MAXD];
  __shared__ float tb[LR_MAXD], lam[LR_MAXD], eb[LR_MAXD];
  __shared__ float gs[LR_MAXD], hs[LR_MAXD];
  __shared__ float r[LR_MAXR], rd[LR_MAXR], ys[LR_MAXR];
  constexpr int NPART = LR_CRG * 4 * LR_CG > LR_RG * 64 ? LR_CRG * 4 * LR_CG : LR_RG * 64;
  __shared__ __attribute__((aligned(16))) float part[NPART], part2[NPART];
  __shared__ float red[LR_THREADS / 64];
  const int tid = threadIdx.x, d = a.d, T = a.T;
  const bool ck_lds = (long)(T + 1) * d <= LR_CKPT;
  LrRegs g;
  lr_load<VEC>(lr_batch(a, 0), d, g);
  {
    // the columns d .. (d rounded up to 4) - 1 of every row that can be staged
    // stay zero (the 16-byte groups of the residual pass read them)
    const int P = lr_spitch(d), pad = ((d + 3) & ~3) - d;
    for (int i = tid; i < (LR_STAGE / P) * pad; i += LR_THREADS)
      stage[(i / pad) * P + d + i % pad] = 0.0f;
  }
  for (int j = tid; j < LR_MAXD; j += LR_THREADS) {
    th[j] = j < d ? a.theta0[j] : 0.0f;
    vv[j] = 0.0f;
    if (j < d) {
      lam[j] = expf(a.eta[j]);
      eb[j] = 0.0f;
      if (ck_lds) ck[j] = th[j];
      else a.ckpt[j] = th[j];
    }
  }
  for (int k = 0; k <= 2 * T; ++k) {
    const LrBatch b = lr_batch(a, k);
    const int i = k < T ? k : 2 * T - k;   // training step of a forward or reverse phase
    if (k > T) {
      for (int j = tid; j < d; j += LR_THREADS) {
        th[j] = ck_lds ? ck[i * d + j] : a.ckpt[(long)i * d + j];
        vv[j] = -lam[j] * tb[j];
      }
    }
    __syncthreads();   // the previous batch's readers are done; th, vv published
    lr_commit<VEC>(b, d, g, stage, ys);
    if (k < 2 * T) lr_load<VEC>(lr_batch(a, k + 1), d, g);   // in flight during this phase
    __syncthreads();
    const float inv = 2.0f / b.rows;
    if (k < T) {
      // forward unroll step
      lr_pass<false>(b, d, stage, ys, th, nullptr, r, nullptr, part, nullptr, gs, nullptr);
      for (int j = tid; j < d; j += LR_THREADS) {
        th[j] -= lam[j] * inv * gs[j];
        if (ck_lds) ck[(k + 1) * d + j] = th[j];
        else a.ckpt[(long)(k + 1) * d + j] = th[j];
      }
    } else if (k == T) {
      // validation loss and its gradient (the seed of the reverse sweep)
      float sq = lr_pass<false>(b, d, stage, ys, th, nullptr, r, nullptr, part, nullptr, gs,
                                nullptr);
      sq = wave_sum(sq);
      if ((tid & 63) == 0) red[tid >> 6] = sq;
      __syncthreads();
      if (tid == 0 && a.val_loss) {
        float ls = 0.0f;
        for (int w = 0; w < LR_THREADS / 64; ++w) ls += red[w];
        *a.val_loss = ls / b.rows;
      }
      for (int j = tid; j < d; j += LR_THREADS) tb[j] = inv * gs[j];
    } else {
      // reverse step i: v = -exp(eta) bar theta_{i+1}; bar theta_i = bar theta_{i+1} + H v;
      // bar eta += -exp(eta) g_i bar theta_{i+1}
      lr_pass<true>(b, d, stage, ys, th, vv, r, rd, part, part2, gs, hs);
      for (int j = tid; j < d; j += LR_THREADS) {
        eb[j] += -lam[j] * inv * gs[j] * tb[j];
        tb[j] += inv * hs[j];
      }
    }
  }
  __syncthreads();
  for (int j = tid; j < d; j += LR_THREADS) a.d_eta[j] = eb[j];
}

// The same meta-gradient with each batch held in registers, for d <= 64 with
// d % 4 == 0, at most 256 rows in every batch and 16-byte aligned batches.
// Thread (q, c) = (tid / 16, tid % 16) holds the 16-byte group c of rows q,
// q + 32, .., q + 224 (32 registers); the 16 groups of a row lie in one DPP row
// of 16 lanes, which sums the row's dot products with rotations, so a residual
// needs neither LDS nor a barrier and every lane of the row receives it.  X^T r
// is summed over the thread's eight rows in registers, then over the 32 row
// slots in LDS, in a fixed order.  The next batch is loaded into a second set
// of registers one group per residual, between the residuals of the current
// batch: a compute unit takes in only ~20 bytes per clock, and a whole batch
// requested at once stalls every wave at the load instructions until most of
// it has arrived, whereas spread out the loads run under the arithmetic.
constexpr int LRR_RPT = 8;                          // rows per thread
constexpr int LRR_SLOTS = LR_THREADS / 16;          // row slots (32)
constexpr int LRR_MAXROWS = LRR_SLOTS * LRR_RPT;    // 256
constexpr int LRR_MAXD = 64;

struct LrrRegs {
  float4 x[LRR_RPT];  // group c of rows q + 32 u
  float y;            // y of row q + 32 (c % 8)
};
struct LrrSrc {
  const float4* x;
  const float* y;
  int n4, rows;
};
template <bool B>
struct LrrLoad {
  static constexpr bool value = B;
};

__device__ __forceinline__ LrrSrc lrr_src(const LrBatch& b, int g4) {
  return {reinterpret_cast<const float4*>(b.X), b.y, b.rows * g4, b.rows};
}
// Loads past the end read the last element (never cleared registers, see LrRegs).
__device__ __forceinline__ float4 lrr_group(const LrrSrc& s, int g4, int q, int c, int u) {
  return s.x[min((q + LRR_SLOTS * u) * g4 + c, s.n4 - 1)];
}
__device__ __forceinline__ float lrr_target(const LrrSrc& s, int q, int c) {
  return s.y[min(q + LRR_SLOTS * (c & 7), s.rows - 1)];
}
__device__ __forceinline__ float dot4(const float4& a, const float4& b) {
  return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w;
}
// Sum over the 16 lanes of a DPP row.  Every lane gets the same bits: each step
// adds two values that the partner lane adds in the other order.
__device__ __forceinline__ float row16_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x128, 0xF, 0xF, true));  // row_ror:8
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x124, 0xF, 0xF, true));  // row_ror:4
  return quad_sum(v);
}

// CKL: the checkpoints fit in LDS ((T + 1) d <= 4096).  A compile-time choice,
// since a runtime one merges the two checkpoint reads into one flat load, which
// waits for every global load in flight, the next batch's included.
template <bool CKL>
__global__ void __launch_bounds__(LR_THREADS) linreg_reg_kernel(LinregArgs a) {
  __shared__ float ck[CKL ? LR_CKPT : 1];
  __shared__ __attribute__((aligned(16))) float th[LRR_MAXD], vv[LRR_MAXD];
  __shared__ __attribute__((aligned(16))) float part[LRR_SLOTS * LRR_MAXD];
  __shared__ __attribute__((aligned(16))) float part2[LRR_SLOTS * LRR_MAXD];
  __shared__ float red[LR_THREADS / 64];
  const int tid = threadIdx.x, d = a.d, T = a.T, g4 = d >> 2;
  const int c = tid & 15, q = tid >> 4;
  // Column j < d is owned by thread 4 j (the first of the four that sum its
  // partials), which keeps exp(eta_j), theta_j, bar theta_j and bar eta_j in
  // registers through the sweep.
  const int jc = min(tid >> 2, d - 1);
  // theta_0 and eta, then the first batch; the set-up waits for the former only
  const float th0 = a.theta0[min(tid, d - 1)], etc = a.eta[jc], thc0 = a.theta0[jc];
  LrrRegs A, B;
  {
    const LrrSrc s0 = lrr_src(lr_batch(a, 0), g4);
    A.y = lrr_target(s0, q, c);
#pragma unroll
    for (int u = 0; u < LRR_RPT; ++u) A.x[u] = lrr_group(s0, g4, q, c, u);
  }
  __builtin_amdgcn_sched_barrier(0);
  const float lamr = expf(etc);
  float thr = thc0, tbr = 0.0f, ebr = 0.0f;
  if (tid < LRR_MAXD) {
    const bool in = tid < d;
    th[tid] = in ? th0 : 0.0f;   // zero past d, like vv: the groups past d add nothing
    vv[tid] = 0.0f;
    if (in) {
      if constexpr (CKL) ck[tid] = th0;
      else a.ckpt[tid] = th0;
    }
  }
  __syncthreads();

  // Phase k of the sweep on the batch in cur; with LOAD, batch k + 1 into nxt.
  auto phase = [&](int k, const LrrRegs& cur, LrrRegs& nxt, auto load) {
    constexpr bool LOAD = decltype(load)::value;
    const LrBatch b = lr_batch(a, k);
    const bool du = k > T;
    const float4 w4 = reinterpret_cast<const float4*>(th)[c];
    const float4 u4 = reinterpret_cast<const float4*>(vv)[c];
    LrrSrc ns{};
    if constexpr (LOAD) {
      ns = lrr_src(lr_batch(a, k + 1), g4);
      nxt.y = lrr_target(ns, q, c);
    }
    // residuals r = X th - y (and rd = X vv); lane u of the row holds y of row u
    float r[LRR_RPT], rd[LRR_RPT], sq = 0.0f;
    const bool in = c < g4;
#pragma unroll
    for (int u = 0; u < LRR_RPT; ++u) {
      if constexpr (LOAD) nxt.x[u] = lrr_group(ns, g4, q, c, u);
      const float4 x = cur.x[u];
      const bool valid = q + LRR_SLOTS * u < b.rows;
      float s = in ? dot4(x, w4) : 0.0f;
      s -= c == u ? cur.y : 0.0f;
      s = row16_sum(s);
      r[u] = valid ? s : 0.0f;
      sq += r[u] * r[u];
      if (du) {
        const float sd = row16_sum(in ? dot4(x, u4) : 0.0f);
        rd[u] = valid ? sd : 0.0f;
      }
      // two rows per scheduling group: their dependent sums interleave, and
      // the loads still go out spread over the residuals
      if (u & 1) __builtin_amdgcn_sched_barrier(0);
    }
    // X^T r (and X^T rd) over this thread's rows, then over the row slots
    float4 ga = make_float4(0.f, 0.f, 0.f, 0.f), ha = ga;
#pragma unroll
    for (int u = 0; u < LRR_RPT; ++u) {
      const float4 x = cur.x[u];
      ga.x += x.x * r[u]; ga.y += x.y * r[u]; ga.z += x.z * r[u]; ga.w += x.w * r[u];
      if (du) {
        ha.x += x.x * rd[u]; ha.y += x.y * rd[u]; ha.z += x.z * rd[u]; ha.w += x.w * rd[u];
      }
    }
    // the column owner's theta for the next reverse step, read ahead
    float thn = 0.0f;
    {
      const int i = 2 * T - k;
      if (k >= T && i >= 1 && (tid & 3) == 0 && tid < 4 * d) {
        if constexpr (CKL) thn = ck[(i - 1) * d + (tid >> 2)];
        else thn = a.ckpt[(long)(i - 1) * d + (tid >> 2)];
      }
    }
    reinterpret_cast<float4*>(part)[q * 16 + c] = ga;
    if (du) reinterpret_cast<float4*>(part2)[q * 16 + c] = ha;
    if (k == T) {
      const float v = wave_sum(c == 0 ? sq : 0.0f);
      if ((tid & 63) == 0) red[tid >> 6] = v;
    }
    __syncthreads();
    if (tid < 4 * LRR_MAXD) {
      // column j, row slots 8h .. 8h + 7 in order, then across the quad
      const int j = tid >> 2, h = tid & 3;
      float g = 0.0f, hv = 0.0f;
#pragma unroll
      for (int i = 0; i < LRR_SLOTS / 4; ++i) {
        g += part[(h * (LRR_SLOTS / 4) + i) * LRR_MAXD + j];
        if (du) hv += part2[(h * (LRR_SLOTS / 4) + i) * LRR_MAXD + j];
      }
      g = quad_sum(g);
      if (du) hv = quad_sum(hv);
      const float inv = 2.0f / b.rows;
      if (h == 0 && j < d) {
        if (k < T) {
          // forward step k: theta_{k+1}
          const float t = thr - lamr * inv * g;
          thr = t;
          th[j] = t;
          if constexpr (CKL) ck[(k + 1) * d + j] = t;
          else a.ckpt[(long)(k + 1) * d + j] = t;
        } else {
          // validation: bar theta_T = dV/dtheta_T; reverse step i = 2T - k:
          // bar eta += -exp(eta) g_i bar theta_{i+1}; bar theta_i = bar theta_{i+1} + H v
          float t;
          if (k == T) {
            t = inv * g;
          } else {
            t = tbr;
            ebr += -lamr * inv * g * t;
            t += inv * hv;
          }
          tbr = t;
          if (2 * T - k >= 1) {   // the next reverse step's theta_{i-1}, v = -exp(eta) bar theta_i
            th[j] = thn;
            vv[j] = -lamr * t;
          }
        }
      }
      if (k == T && tid == 0 && a.val_loss) {
        float ls = 0.0f;
        for (int w = 0; w < LR_THREADS / 64; ++w) ls += red[w];
        *a.val_loss = ls / b.rows;
      }
    }
    __syncthreads();
  };

  for (int k = 0; k < 2 * T; k += 2) {
    phase(k, A, B, LrrLoad<true>{});
    phase(k + 1, B, A, LrrLoad<true>{});
  }
  phase(2 * T, A, B, LrrLoad<false>{});
  if ((tid & 3) == 0 && tid < 4 * d) a.d_eta[tid >> 2] = ebr;
}

// Columns c0 .. c1 - 1 of rows 0 .. rows - 1 of each job's bf16 matrix set to
// zero; one workgroup per job and 256 rows.
__global__ void zero_cols_kernel(ZeroColJobs J) {
  const int j = blockIdx.y;
  if (j >= J.n) return;
  const int w = J.c1[j] - J.c0[j];
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < (long)J.rows[j] * w;
       i += (long)gridDim.x * 256)
    J.p[j][(i / w) * J.ld[j] + J.c0[j] + i % w] = 0;
}

__global__ void fill_kernel(float* p, long n, float v) {
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long)gridDim.x * 256) p[i] = v;
}

__global__ void copy_kernel(const float* __restrict__ src, float* __restrict__ dst, long n) {
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long)gridDim.x * 256)
    dst[i] = src[i];
}

// Number of NaN / infinite entries of x, added to *count by one atomic per wave.
__global__ void count_nonfinite_kernel(const float* __restrict__ x, long n,
                                       unsigned long long* count) {
  unsigned c = 0;
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long)gridDim.x * 256)
    c += (__float_as_uint(x[i]) & 0x7f800000u) == 0x7f800000u;
  for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
  if ((threadIdx.x & 63) == 0 && c) atomicAdd(count, (unsigned long long)c);
}

__global__ void zero_count_kernel(unsigned long long* count) {
  if (threadIdx.x == 0) count[threadIdx.x] = 0ull;
}

}  // namespace

hipError_t count_nonfinite(const float* x, long n, unsigned long long* count, hipStream_t s) {
  hipLaunchKernelGGL(zero_count_kernel, dim3(1), dim3(64), 0, s, count);
  if (n > 0)
    hipLaunchKernelGGL(count_nonfinite_kernel, dim3(min(cdiv(n, 256), 4096)), dim3(256), 0, s, x,
                       n, count);
  return hipGetLastError();
}

hipError_t zero_cols(const ZeroColJobs& J, hipStream_t s) {
  if (J.n < 0 || J.n > ZC_MAX_JOBS) return hipErrorInvalidValue;
  if (J.n == 0) return hipSuccess;
  long most = 0;
  for (int j = 0; j < J.n; ++j) {
    if (!J.p[j] || J.rows[j] < 0 || J.c0[j] < 0 || J.c1[j] < J.c0[j] || J.c1[j] > J.ld[j])
      return hipErrorInvalidValue;
    most = std::max(most, (long)J.rows[j] * (J.c1[j] - J.c0[j]));
  }
  if (most == 0) return hipSuccess;
  hipLaunchKernelGGL(zero_cols_kernel, dim3(min(cdiv(most, 256), 1024), J.n), dim3(256), 0, s, J);
  return hipGetLastError();
}

hipError_t fill(float* p, long n, float v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_kernel, dim3(min(cdiv(n, 256), 4096)), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t copy(const float* src, float* dst, long n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy_kernel, dim3(min(cdiv(n, 256), 4096)), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

template <typename T>
hipError_t convert_matrices(const ConvJobs<T>& J, int rows, int cols, int lds, int ldd, int lddT,
                            hipStream_t s, int batch, long s_src, long s_dst, long s_dstT) {
  if (J.n < 0 || J.n > CONV_MAX_JOBS) return hipErrorInvalidValue;
  if (rows <= 0 || cols <= 0 || batch <= 0 || J.n == 0) return hipSuccess;
  for (int k = 0; k < J.n; ++k)
    if (!J.src[k]) return hipErrorInvalidValue;
  dim3 grid(cdiv(cols, 64), cdiv(rows, 64), batch * J.n);
  const auto al = [](const void* q, uintptr_t a) { return (reinterpret_cast<uintptr_t>(q) % a) == 0; };
  const uintptr_t aw = 4 * sizeof(T);  // alignment of 4 elements
  bool vec = (lds % 4) == 0 && (s_src % 4) == 0;
  for (int k = 0; k < J.n; ++k)
    vec = vec && al(J.src[k], 16) &&
          (!J.dst[k] || ((ldd % 4) == 0 && (s_dst % 4) == 0 && al(J.dst[k], aw))) &&
          (!J.dstT[k] || ((lddT % 4) == 0 && (s_dstT % 4) == 0 && al(J.dstT[k], aw)));
  if (vec)
    hipLaunchKernelGGL(convert_vec_kernel<T>, grid, dim3(256), 0, s, J, batch, rows, cols, lds, ldd,
                       lddT, s_src, s_dst, s_dstT);
  else
    hipLaunchKernelGGL(convert_kernel<T>, grid, dim3(256), 0, s, J, batch, rows, cols, lds, ldd,
                       lddT, s_src, s_dst, s_dstT);
  return hipGetLastError();
}

hipError_t transpose_bf16_jobs(const TrJobs& J, int batch, int rows, int cols, int ld, int ldT,
                               long s_src, long s_dst, hipStream_t s) {
  // Source rows are read in 16-byte chunks up to the next multiple of 8 columns
  // (padding, present when ld >= that); transposed rows past cols are not written.
  if (rows % 8 || ld % 8 || ldT % 8 || s_src % 8 || s_dst % 8 || ld < (cols + 7) / 8 * 8 ||
      batch < 1 || J.n < 0 || J.n > TR_MAX_JOBS)
    return hipErrorInvalidValue;
  for (int j = 0; j < J.n; ++j)
    if (!J.src[j] || !J.dst[j]) return hipErrorInvalidValue;
  if (rows <= 0 || cols <= 0 || J.n == 0) return hipSuccess;
  hipLaunchKernelGGL(transpose_bf16_kernel, dim3(cdiv(cols, 64), cdiv(rows, 64), J.n * batch),
                     dim3(256), 0, s, J, batch, rows, cols, ld, ldT, s_src, s_dst);
  return hipGetLastError();
}

hipError_t transpose_bf16(const bf16_t* a0, const bf16_t* a1, int rows, int cols, int ld,
                          bf16_t* t0, bf16_t* t1, int ldT, hipStream_t s) {
  TrJobs J;
  J.n = a1 ? 2 : 1;
  J.src[0] = a0; J.dst[0] = t0;
  J.src[1] = a1; J.dst[1] = t1;
  return transpose_bf16_jobs(J, 1, rows, cols, ld, ldT, 0, 0, s);
}

template <typename T>
hipError_t convert_matrix(const float* src, int rows, int cols, int lds, T* dst, int ldd,
                          T* dstT, int lddT, hipStream_t s, int batch, long s_src, long s_dst,
                          long s_dstT) {
  ConvJobs<T> J;
  J.n = 1;
  J.src[0] = src;
  J.dst[0] = dst;
  J.dstT[0] = dstT;
  return convert_matrices<T>(J, rows, cols, lds, ldd, lddT, s, batch, s_src, s_dst, s_dstT);
}

template <typename T>
hipError_t bias_reduce(const T* dZT, const T* dZdT, int ld, int rows, const ParamArgs<T>& P,
                       hipStream_t s) {
  if (P.nout <= 0) return hipSuccess;
  const bool vec = (ld % Elem<T>::VE) == 0 && (reinterpret_cast<uintptr_t>(dZT) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(dZdT) & 15) == 0;
  if (vec)
    hipLaunchKernelGGL((bias_kernel<T, true>), dim3(cdiv(P.nout, 4)), dim3(256), 0, s, dZT, dZdT, ld,
                       rows, P);
  else
    hipLaunchKernelGGL((bias_kernel<T, false>), dim3(cdiv(P.nout, 4)), dim3(256), 0, s, dZT, dZdT,
                       ld, rows, P);
  return hipGetLastError();
}

template <typename T>
hipError_t loss_head(const LossArgs<T>& args, hipStream_t s) {
  // Up to 128 classes the loss kernel writes the transposed copies itself (a
  // wave's C strided stores per row cost less than a transpose launch); wider
  // heads are transposed through LDS tiles afterwards.
  LossArgs<T> a = args;
  a.direct_t = a.C <= 128 ? 1 : 0;
  hipLaunchKernelGGL(loss_kernel<T>, dim3(cdiv(a.rows, 4)), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.direct_t) return e;
  // transposed copies of dL/dz (and its tangent), coalesced through LDS
  const dim3 tg(cdiv(a.C, 64), cdiv(a.rows, 64), 2);
  if constexpr (sizeof(T) == 2) {
    if (a.rows % 8 == 0 && a.ld % 8 == 0 && a.ld >= (a.C + 7) / 8 * 8 && a.ldT % 8 == 0) {
      return transpose_bf16(a.d, a.dual ? a.dd : nullptr, a.rows, a.C, a.ld, a.dT,
                            a.dual ? a.ddT : nullptr, a.ldT, s);
    }
  }
  hipLaunchKernelGGL(transpose_kernel<T>, tg, dim3(256), 0, s, a.d, a.dual ? a.dd : nullptr,
                     a.rows, a.C, a.ld, a.dT, a.ddT, a.ldT);
  return hipGetLastError();
}

hipError_t loss_reduce(const float* loss_rows, const float* alpha_logits, int rows, float inv_n,
                       float* loss_out, hipStream_t s) {
  hipLaunchKernelGGL(loss_reduce_kernel, dim3(1), dim3(256), 0, s, loss_rows, alpha_logits, rows,
                     inv_n, loss_out);
  return hipGetLastError();
}

template <typename T>
hipError_t adam_vjp(const AdamVjpArgs<T>* a, int L, const int* part_off, float* partial,
                    hipStream_t s) {
  if (L < 1 || L > MFMG_MAX_LAYERS) return hipErrorInvalidValue;
  AdamVjpLayers<T> A;
  A.L = L;
  A.off[0] = 0;
  for (int l = 0; l < L; ++l) {
    // 16 x 64 tiles of W, then 256 bias entries per workgroup
    const long nb = (long)cdiv(a[l].nin, 16) * cdiv(a[l].nout, 64) +
                    (a[l].b_off >= 0 ? cdiv(a[l].nout, 256) : 0);
    if (nb != part_off[l + 1] - part_off[l] || part_off[l] != A.off[l])
      return hipErrorInvalidValue;
    A.a[l] = a[l];
    A.off[l + 1] = A.off[l] + (int)nb;
  }
  hipLaunchKernelGGL(adam_vjp_kernel<T>, dim3(A.off[L]), dim3(256), 0, s, A, partial);
  return hipGetLastError();
}

hipError_t adam_reduce(const float* partial, const int* block_offsets, int n_layers, int first,
                       float* d_eta, hipStream_t s) {
  Offsets o;
  for (int l = 0; l <= n_layers; ++l) o.off[l] = block_offsets[l];
  if (n_layers < 1 || n_layers > MFMG_MAX_LAYERS) return hipErrorInvalidValue;
  hipLaunchKernelGGL(adam_reduce_kernel, dim3(1), dim3(1024), 0, s, partial, o, n_layers, first,
                     d_eta);
  return hipGetLastError();
}

bool linreg_fits(int T, int rows, int vrows, int d) {
  return T >= 1 && T <= LR_MAXT && d >= 1 && d <= LR_MAXD && rows >= 1 && rows <= LR_MAXR &&
         vrows >= 1 && vrows <= LR_MAXR;
}

hipError_t linreg_meta_grad(const float* theta0, const float* eta, const float* const* xs,
                            const float* const* ys, int T, int rows, int d, const float* vx,
                            const float* vy, int vrows, float* d_eta, float* val_loss,
                            float* scratch, hipStream_t s) {
  LinregArgs a;
  a.theta0 = theta0;
  a.eta = eta;
  for (int t = 0; t < LR_MAXT; ++t) {
    a.xs[t] = t < T ? xs[t] : nullptr;
    a.ys[t] = t < T ? ys[t] : nullptr;
  }
  a.T = T;
  a.rows = rows;
  a.d = d;
  a.vrows = vrows;
  bool vec = (d % 4) == 0 && (reinterpret_cast<uintptr_t>(vx) & 15) == 0;
  for (int t = 0; t < T; ++t) vec = vec && (reinterpret_cast<uintptr_t>(xs[t]) & 15) == 0;
  a.vec = vec ? 1 : 0;
  a.vx = vx;
  a.vy = vy;
  a.d_eta = d_eta;
  a.val_loss = val_loss;
  a.ckpt = scratch;
  // batches that fit one register set per thread: the register-resident kernel;
  // else batches staged in LDS (16-byte or 4-byte loads) or read from global memory
  if (a.vec && d <= LRR_MAXD && rows <= LRR_MAXROWS && vrows <= LRR_MAXROWS) {
    if ((T + 1) * d <= LR_CKPT)
      hipLaunchKernelGGL(linreg_reg_kernel<true>, dim3(1), dim3(LR_THREADS), 0, s, a);
    else
      hipLaunchKernelGGL(linreg_reg_kernel<false>, dim3(1), dim3(LR_THREADS), 0, s, a);
  } else if (a.vec)
    hipLaunchKernelGGL(linreg_kernel<true>, dim3(1), dim3(LR_THREADS), 0, s, a);
  else
    hipLaunchKernelGGL(linreg_kernel<false>, dim3(1), dim3(LR_THREADS), 0, s, a);
  return hipGetLastError();
}

template hipError_t convert_matrices<bf16_t>(const ConvJobs<bf16_t>&, int, int, int, int, int, hipStream_t, int, long, long, long);
template hipError_t convert_matrices<float>(const ConvJobs<float>&, int, int, int, int, int, hipStream_t, int, long, long, long);
template hipError_t convert_matrix<bf16_t>(const float*, int, int, int, bf16_t*, int, bf16_t*, int, hipStream_t, int, long, long, long);
template hipError_t convert_matrix<float>(const float*, int, int, int, float*, int, float*, int, hipStream_t, int, long, long, long);
template hipError_t bias_reduce<bf16_t>(const bf16_t*, const bf16_t*, int, int, const ParamArgs<bf16_t>&, hipStream_t);
template hipError_t bias_reduce<float>(const float*, const float*, int, int, const ParamArgs<float>&, hipStream_t);
template hipError_t loss_head<bf16_t>(const LossArgs<bf16_t>&, hipStream_t);
template hipError_t loss_head<float>(const LossArgs<float>&, hipStream_t);
template hipError_t adam_vjp<bf16_t>(const AdamVjpArgs<bf16_t>*, int, const int*, float*, hipStream_t);
template hipError_t adam_vjp<float>(const AdamVjpArgs<float>*, int, const int*, float*, hipStream_t);

}  // namespace mfmg
