// Decoder-block dual kernels (gfx950): token gather, LayerNorm, RoPE head
// split/merge, causal softmax, embedding scatter and the loss-weighting
// meta-model, each with the tangent carried alongside (forward-over-reverse,
// Section 2.2; the transformer workloads of Section 5).  Matrix products go
// through gemm_nt; these kernels are the elementwise/row-wise pieces.
//
// Layouts: token rows n = b * seq + s; residual stream and LayerNorm values
// float32 [tokens][d]; per-head tensors float32 [batch * heads][seq][dh];
// attention scores/probabilities float32 [batch * heads][seq][seq].
#include "kernels.h"
#include "param_epi.h"
#include "transformer.h"

namespace mfmg {

namespace {

inline int cdivl(long a, long b) { return (int)((a + b - 1) / b); }

// ------------------------------------------------------------------------------------
// Tokens: input ids and next-token labels from [batch][seq + 1] sequences.
// Out-of-range ids gather a zero row; out-of-range labels make the loss NaN.
// ------------------------------------------------------------------------------------
__global__ void split_tokens_kernel(const int* __restrict__ tok, int B, int S, int V, int* ids,
                                    int* labels) {
  const int n = blockIdx.x * 256 + threadIdx.x;
  if (n >= B * S) return;
  const int b = n / S, s = n % S;
  const int a = tok[b * (S + 1) + s];
  const int y = tok[b * (S + 1) + s + 1];
  ids[n] = (a >= 0 && a < V) ? a : -1;
  labels[n] = (y >= 0 && y < V) ? y : -1;
}

// h[n] = E[ids[n]] (and the tangent rows).
__global__ void gather_rows_kernel(const int* __restrict__ ids, int N, int d,
                                   const float* __restrict__ E, const float* __restrict__ Ed,
                                   float* h, float* hd) {
  const long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= (long)N * d) return;
  const int n = (int)(e / d), j = (int)(e % d);
  const int v = ids[n];
  h[e] = v >= 0 ? E[(long)v * d + j] : 0.0f;
  if (hd) hd[e] = v >= 0 ? Ed[(long)v * d + j] : 0.0f;
}

// ------------------------------------------------------------------------------------
// LayerNorm forward, one wavefront per row: xh = (x - mean) rstd,
// y = g xh + b.  Tangent: xhd = rstd (xd - mean(xd) - xh mean(xh xd)),
// yd = g xhd + gd xh + bd.  Saves xh, rstd, c = mean(xh xd) and xhd for the
// backward.
// ------------------------------------------------------------------------------------
constexpr int LN_MAXPL = 16;  // d <= 64 * 16

__global__ void __launch_bounds__(256) ln_fwd_kernel(LnArgs a) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.N) return;
  const int d = a.d;
  const float* x = a.x + (long)row * d;
  float xv[LN_MAXPL], xdv[LN_MAXPL];
  float s = 0.f;
  int cnt = 0;
  for (int j = lane, k = 0; j < d; j += 64, ++k) {
    xv[k] = x[j];
    s += xv[k];
    cnt = k + 1;
  }
  const float mean = wave_sum(s) / d;
  float v = 0.f;
  for (int k = 0; k < cnt; ++k) {
    xv[k] -= mean;
    v += xv[k] * xv[k];
  }
  const float rstd = rsqrtf(wave_sum(v) / d + a.eps);
  for (int k = 0; k < cnt; ++k) xv[k] *= rstd;  // xh
  float c = 0.f, md = 0.f;
  if (a.dual) {
    const float* xd = a.xd + (long)row * d;
    for (int j = lane, k = 0; j < d; j += 64, ++k) {
      xdv[k] = xd[j];
      md += xdv[k];
      c += xv[k] * xdv[k];
    }
    md = wave_sum(md) / d;
    c = wave_sum(c) / d;
  }
  for (int j = lane, k = 0; j < d; j += 64, ++k) {
    const long o = (long)row * d + j;
    a.xh[o] = xv[k];
    a.y[o] = a.g[j] * xv[k] + a.b[j];
    if (a.dual) {
      const float xhd = rstd * (xdv[k] - md - xv[k] * c);
      a.xhd[o] = xhd;
      a.yd[o] = a.g[j] * xhd + a.gd[j] * xv[k] + a.bd[j];
    }
  }
  if (lane == 0) {
    a.rstd[row] = rstd;
    if (a.dual) a.c[row] = c;
  }
}

// ------------------------------------------------------------------------------------
// LayerNorm backward, one wavefront per row, with the residual add:
//   q = g dy, A = q - mean(q) - xh mean(xh q), dx = rstd A, dh_out = dh_in + dx.
// Tangent (w.r.t. x through xh and rstd, g and dy): with rstd' = -rstd^2 c,
//   qd = gd dy + g dyd,
//   Ad = qd - mean(qd) - xhd mean(xh q) - xh (mean(xhd q) + mean(xh qd)),
//   dxd = rstd' A + rstd Ad.
// The column sums of dy xh, dy and their tangents (dyd xh + dy xhd, dyd), the
// gradients of g and b, come from ln_colsum_kernel.
// ------------------------------------------------------------------------------------
__global__ void __launch_bounds__(256) ln_bwd_kernel(LnBwdArgs a) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.N) return;
  const int d = a.d;
  const long base = (long)row * d;
  const float rstd = a.rstd[row];
  float xh[LN_MAXPL], dy[LN_MAXPL], q[LN_MAXPL];
  float mq = 0.f, mxq = 0.f;
  for (int j = lane, k = 0; j < d; j += 64, ++k) {
    xh[k] = a.xh[base + j];
    dy[k] = a.dy[base + j];
    q[k] = a.g[j] * dy[k];
    mq += q[k];
    mxq += xh[k] * q[k];
  }
  mq = wave_sum(mq) / d;
  mxq = wave_sum(mxq) / d;
  float xhd[LN_MAXPL], qd[LN_MAXPL];
  float mqd = 0.f, mxdq = 0.f, mxqd = 0.f;
  if (a.dual) {
    for (int j = lane, k = 0; j < d; j += 64, ++k) {
      xhd[k] = a.xhd[base + j];
      qd[k] = a.gd[j] * dy[k] + a.g[j] * a.dyd[base + j];
      mqd += qd[k];
      mxdq += xhd[k] * q[k];
      mxqd += xh[k] * qd[k];
    }
    mqd = wave_sum(mqd) / d;
    mxdq = wave_sum(mxdq) / d;
    mxqd = wave_sum(mxqd) / d;
  }
  const float rstdd = a.dual ? -rstd * rstd * a.c[row] : 0.f;
  for (int j = lane, k = 0; j < d; j += 64, ++k) {
    const float A = q[k] - mq - xh[k] * mxq;
    a.dh_out[base + j] = (a.dh_in ? a.dh_in[base + j] : 0.f) + rstd * A;
    if (a.dual) {
      const float Ad = qd[k] - mqd - xhd[k] * mxq - xh[k] * (mxdq + mxqd);
      a.dhd_out[base + j] = (a.dhd_in ? a.dhd_in[base + j] : 0.f) + rstdd * A + rstd * Ad;
    }
  }
}

// The same two kernels for d a multiple of 256: lane l holds columns
// 256 k + 4 l .. +3 and moves 16 bytes per access.
constexpr int LN_MAXV = LN_MAX_D / 256;

__device__ __forceinline__ f32x4 ldv(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
__device__ __forceinline__ void stv(float* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
__device__ __forceinline__ float hsum(f32x4 v) { return (v[0] + v[1]) + (v[2] + v[3]); }

__global__ void __launch_bounds__(256) ln_fwd_vec_kernel(LnArgs a) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.N) return;
  const int d = a.d, nv = d >> 8;
  const long base = (long)row * d;
  f32x4 xv[LN_MAXV], xdv[LN_MAXV];
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < LN_MAXV; ++k)
    if (k < nv) {
      xv[k] = ldv(a.x + base + 256 * k + 4 * lane);
      s += hsum(xv[k]);
    }
  const float mean = wave_sum(s) / d;
  float v = 0.f;
#pragma unroll
  for (int k = 0; k < LN_MAXV; ++k)
    if (k < nv) {
      xv[k] -= mean;
      v += hsum(xv[k] * xv[k]);
    }
  const float rstd = rsqrtf(wave_sum(v) / d + a.eps);
  float c = 0.f, md = 0.f;
#pragma unroll
  for (int k = 0; k < LN_MAXV; ++k)
    if (k < nv) {
      xv[k] *= rstd;  // xh
      if (a.dual) {
        xdv[k] = ldv(a.xd + base + 256 * k + 4 * lane);
        md += hsum(xdv[k]);
        c += hsum(xv[k] * xdv[k]);
      }
    }
  if (a.dual) {
    md = wave_sum(md) / d;
    c = wave_sum(c) / d;
  }
#pragma unroll
  for (int k = 0; k < LN_MAXV; ++k)
    if (k < nv) {
      const int j = 256 * k + 4 * lane;
      const f32x4 g = ldv(a.g + j);
      stv(a.xh + base + j, xv[k]);
      const f32x4 yv = g * xv[k] + ldv(a.b + j);
      if (a.yb)
        store4(a.yb + (long)row * a.ldb + j, yv[0], yv[1], yv[2], yv[3]);
      else
        stv(a.y + base + j, yv);
      if (a.dual) {
        const f32x4 xhd = rstd * (xdv[k] - md - xv[k] * c);
        stv(a.xhd + base + j, xhd);
        const f32x4 ydv = g * xhd + ldv(a.gd + j) * xv[k] + ldv(a.bd + j);
        if (a.ydb)
          store4(a.ydb + (long)row * a.ldb + j, ydv[0], ydv[1], ydv[2], ydv[3]);
        else
          stv(a.yd + base + j, ydv);
      }
    }
  if (lane == 0) {
    a.rstd[row] = rstd;
    if (a.dual) a.c[row] = c;
  }
}

__global__ void __launch_bounds__(256) ln_bwd_vec_kernel(LnBwdArgs a) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.N) return;
  const int d = a.d, nv = d >> 8;
  const long base = (long)row * d;
  const float rstd = a.rstd[row];
  f32x4 xh[LN_MAXV], q[LN_MAXV], xhd[LN_MAXV], qd[LN_MAXV];
  float mq = 0.f, mxq = 0.f, mqd = 0.f, mxdq = 0.f, mxqd = 0.f;
#pragma unroll
  for (int k = 0; k < LN_MAXV; ++k)
    if (k < nv) {
      const int j = 256 * k + 4 * lane;
      xh[k] = ldv(a.xh + base + j);
      const f32x4 dy = ldv(a.dy + base + j), g = ldv(a.g + j);
      q[k] = g * dy;
      mq += hsum(q[k]);
      mxq += hsum(xh[k] * q[k]);
      if (a.dual) {
        xhd[k] = ldv(a.xhd + base + j);
        qd[k] = ldv(a.gd + j) * dy + g * ldv(a.dyd + base + j);
        mqd += hsum(qd[k]);
        mxdq += hsum(xhd[k] * q[k]);
        mxqd += hsum(xh[k] * qd[k]);
      }
    }
  mq = wave_sum(mq) / d;
  mxq = wave_sum(mxq) / d;
  if (a.dual) {
    mqd = wave_sum(mqd) / d;
    mxdq = wave_sum(mxdq) / d;
    mxqd = wave_sum(mxqd) / d;
  }
  const float rstdd = a.dual ? -rstd * rstd * a.c[row] : 0.f;
#pragma unroll
  for (int k = 0; k < LN_MAXV; ++k)
    if (k < nv) {
      const int j = 256 * k + 4 * lane;
      const f32x4 A = q[k] - mq - xh[k] * mxq;
      const f32x4 hin = a.dh_in ? ldv(a.dh_in + base + j) : f32x4{0.f, 0.f, 0.f, 0.f};
      const f32x4 ho = hin + rstd * A;
      stv(a.dh_out + base + j, ho);
      if (a.hb) store4(a.hb + (long)row * a.ldb + j, ho[0], ho[1], ho[2], ho[3]);
      if (a.dual) {
        const f32x4 Ad = qd[k] - mqd - xhd[k] * mxq - xh[k] * (mxdq + mxqd);
        const f32x4 hdin = a.dhd_in ? ldv(a.dhd_in + base + j) : f32x4{0.f, 0.f, 0.f, 0.f};
        const f32x4 hdo = hdin + rstdd * A + rstd * Ad;
        stv(a.dhd_out + base + j, hdo);
        if (a.hdb) store4(a.hdb + (long)row * a.ldb + j, hdo[0], hdo[1], hdo[2], hdo[3]);
      }
    }
}

// Column sums over a chunk of LN_CHUNK rows: partial[chunk][4][d] = sums of
// dy xh, dy, dyd xh + dy xhd, dyd.  Block: 64 columns x 4 row phases; each
// phase sums every fourth row of the chunk, then the four are added in order.
__global__ void __launch_bounds__(256) ln_colsum_kernel(LnBwdArgs a) {
  __shared__ float red[4][4][64];
  const int c = threadIdx.x & 63, ph = threadIdx.x >> 6;
  const int j = blockIdx.x * 64 + c;
  const int r0 = blockIdx.y * LN_CHUNK;
  const int r1 = min(a.N, r0 + LN_CHUNK);
  float sg = 0.f, sb = 0.f, sgd = 0.f, sbd = 0.f;
  if (j < a.d) {
    for (int r = r0 + ph; r < r1; r += 4) {
      const long o = (long)r * a.d + j;
      const float dy = a.dy[o], xh = a.xh[o];
      sg += dy * xh;
      sb += dy;
      if (a.dual) {
        const float dyd = a.dyd[o];
        sgd += dyd * xh + dy * a.xhd[o];
        sbd += dyd;
      }
    }
  }
  red[ph][0][c] = sg;
  red[ph][1][c] = sb;
  red[ph][2][c] = sgd;
  red[ph][3][c] = sbd;
  __syncthreads();
  if (ph == 0 && j < a.d) {
    float* P = a.partial + (long)blockIdx.y * 4 * a.d;
#pragma unroll
    for (int k = 0; k < 4; ++k) P[k * a.d + j] = ((red[0][k][c] + red[1][k][c]) + red[2][k][c]) + red[3][k][c];
  }
}

// Column sums of the chunk partials in a fixed order (phase p of 16 sums chunks
// p, p + 16, ...; the phases are added in order), then the parameter epilogue
// on g (offset g_off) and b (offset b_off).  16 columns per block.
template <typename T>
__global__ void __launch_bounds__(256) ln_param_kernel(const float* __restrict__ partial,
                                                       int nparts, int d, long g_off, long b_off,
                                                       ParamArgs<T> P, float* out_g,
                                                       float* out_b) {
  __shared__ float red[16][4][16];
  const int c = threadIdx.x & 15, ph = threadIdx.x >> 4;
  const int j = blockIdx.x * 16 + c;
  float s[4] = {0.f, 0.f, 0.f, 0.f};
  if (j < d) {
    for (int p = ph; p < nparts; p += 16) {
      const float* Pp = partial + (long)p * 4 * d;
#pragma unroll
      for (int k = 0; k < 4; ++k) s[k] += Pp[k * d + j];
    }
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) red[ph][k][c] = s[k];
  __syncthreads();
  if (ph != 0 || j >= d) return;
  float t[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    t[k] = red[0][k][c];
    for (int q = 1; q < 16; ++q) t[k] += red[q][k][c];
  }
  const float cg = param_elem(P, g_off + j, t[0], t[2]);
  const float cb = param_elem(P, b_off + j, t[1], t[3]);
  if (out_g) out_g[j] = cg;
  if (out_b) out_b[j] = cb;
}

// ------------------------------------------------------------------------------------
// RoPE.  cos/sin table [seq][dh/2] in double precision, rounded to float.
// Rotate-half pairing (j, j + dh/2): q'_j = q_j c - q_{j+h} s,
// q'_{j+h} = q_{j+h} c + q_j s, with angle s * base^(-2j/dh).  Linear, so the
// tangent uses the same rotation; the backward applies the transpose.
// ------------------------------------------------------------------------------------
__global__ void rope_table_kernel(int S, int dh, double base, float* cs, float* sn) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  const int half = dh / 2;
  if (e >= S * half) return;
  const int s = e / half, j = e % half;
  const double ang = (double)s * pow(base, -2.0 * j / dh);
  cs[e] = (float)cos(ang);
  sn[e] = (float)sin(ang);
}

// qkv [N][3d] (columns q heads | k heads | v heads) -> per-head Q, K (rotated), V.
__global__ void rope_split_kernel(RopeArgs a) {
  const long e = (long)blockIdx.x * 256 + threadIdx.x;
  const int d = a.H * a.dh, half = a.dh / 2;
  if (e >= (long)a.N * d) return;
  const int n = (int)(e / d), c = (int)(e % d);
  const int h = c / a.dh, j = c % a.dh;
  const int b = n / a.S, s = n % a.S;
  const long src = (long)n * 3 * d;
  const long dst = ((long)(b * a.H + h) * a.S + s) * a.dh + j;
  const int jp = j < half ? j + half : j - half;
  const float cs = a.cs[s * half + (j % half)], sn = a.sn[s * half + (j % half)];
  const float sg = j < half ? -sn : sn;
  for (int t = 0; t < (a.dual ? 2 : 1); ++t) {
    const float* q = t == 0 ? a.qkv : a.qkvd;
    const float vq = q[src + h * a.dh + j] * cs + sg * q[src + h * a.dh + jp];
    const float vk = q[src + d + h * a.dh + j] * cs + sg * q[src + d + h * a.dh + jp];
    const float vv = q[src + 2 * d + h * a.dh + j];
    bf16_t* Qb = t == 0 ? a.Qb : a.Qdb;
    if (Qb) {
      Qb[dst] = f2bf(vq);
      (t == 0 ? a.Kb : a.Kdb)[dst] = f2bf(vk);
      (t == 0 ? a.Vb : a.Vdb)[dst] = f2bf(vv);
    } else {
      (t == 0 ? a.Q : a.Qd)[dst] = vq;
      (t == 0 ? a.K : a.Kd)[dst] = vk;
      (t == 0 ? a.V : a.Vd)[dst] = vv;
    }
  }
}

// Per-head dQ, dK (rotated frame), dV -> dqkv [N][3d] in the unrotated frame.
__global__ void rope_merge_kernel(RopeArgs a) {
  const long e = (long)blockIdx.x * 256 + threadIdx.x;
  const int d = a.H * a.dh, half = a.dh / 2;
  if (e >= (long)a.N * d) return;
  const int n = (int)(e / d), c = (int)(e % d);
  const int h = c / a.dh, j = c % a.dh;
  const int b = n / a.S, s = n % a.S;
  const long dst = (long)n * 3 * d;
  const long src = ((long)(b * a.H + h) * a.S + s) * a.dh;
  const int jp = j < half ? j + half : j - half;
  const float cs = a.cs[s * half + (j % half)], sn = a.sn[s * half + (j % half)];
  const float sg = j < half ? sn : -sn;  // transpose of the rotation
  for (int t = 0; t < (a.dual ? 2 : 1); ++t) {
    const float* Q = t == 0 ? a.Q : a.Qd;
    const float* K = t == 0 ? a.K : a.Kd;
    const float* Vv = t == 0 ? a.V : a.Vd;
    const float vq = Q[src + j] * cs + sg * Q[src + jp];
    const float vk = K[src + j] * cs + sg * K[src + jp];
    const float vv = Vv[src + j];
    bf16_t* ob = t == 0 ? a.ob : a.odb;
    if (ob) {
      const long o = (long)n * a.ldb + h * a.dh + j;
      ob[o] = f2bf(vq);
      ob[o + d] = f2bf(vk);
      ob[o + 2 * d] = f2bf(vv);
    } else {
      float* q = t == 0 ? a.qkv_out : a.qkvd_out;
      q[dst + h * a.dh + j] = vq;
      q[dst + d + h * a.dh + j] = vk;
      q[dst + 2 * d + h * a.dh + j] = vv;
    }
  }
}

// ------------------------------------------------------------------------------------
// Causal softmax over keys 0..q of each query row q, one wavefront per row.
// Tangent: Pd = P (Sd - <P, Sd>).  Scores arrive already scaled.
// ------------------------------------------------------------------------------------
__global__ void __launch_bounds__(256) softmax_fwd_kernel(SoftmaxArgs a) {
  const long row = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.rows) return;
  const int S = a.S;
  const int q = (int)(row % S);
  const long base = row * S;
  float mx = -INFINITY;
  for (int k = lane; k <= q; k += 64) mx = fmaxf(mx, a.Sc[base + k]);
  mx = wave_max(mx);
  float se = 0.f;
  for (int k = lane; k <= q; k += 64) se += expf(a.Sc[base + k] - mx);
  se = wave_sum(se);
  const float inv = 1.0f / se;
  float sd = 0.f;
  if (a.dual) {
    for (int k = lane; k <= q; k += 64) sd += expf(a.Sc[base + k] - mx) * inv * a.Scd[base + k];
    sd = wave_sum(sd);
  }
  for (int k = lane; k < S; k += 64) {
    const float p = k <= q ? expf(a.Sc[base + k] - mx) * inv : 0.0f;
    a.P[base + k] = p;
    if (a.dual) a.Pd[base + k] = k <= q ? p * (a.Scd[base + k] - sd) : 0.0f;
  }
}

// dS = scale P (dP - r), r = <P, dP>; tangent with rd = <Pd, dP> + <P, dPd>:
// dSd = scale (Pd (dP - r) + P (dPd - rd)).
__global__ void __launch_bounds__(256) softmax_bwd_kernel(SoftmaxArgs a) {
  const long row = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.rows) return;
  const int S = a.S;
  const long base = row * S;
  float r = 0.f, rd = 0.f;
  for (int k = lane; k < S; k += 64) {
    r += a.P[base + k] * a.dP[base + k];
    if (a.dual) rd += a.Pd[base + k] * a.dP[base + k] + a.P[base + k] * a.dPd[base + k];
  }
  r = wave_sum(r);
  if (a.dual) rd = wave_sum(rd);
  for (int k = lane; k < S; k += 64) {
    const float p = a.P[base + k], g = a.dP[base + k];
    a.dS[base + k] = a.scale * p * (g - r);
    if (a.dual)
      a.dSd[base + k] = a.scale * (a.Pd[base + k] * (g - r) + p * (a.dPd[base + k] - rd));
  }
}

// ------------------------------------------------------------------------------------
// Embedding gradient.  The token ids of a batch are sorted (bitonic sort of
// (id, position) pairs in one workgroup) and the sorted positions cut into
// segments of at most EMB_SEG positions of one id.  One wave sums each
// segment's rows, and each vocabulary row then adds its segments' sums in
// order: a deterministic scatter-add whose work is spread evenly even for the
// Zipf-hot ids.
// ------------------------------------------------------------------------------------
__global__ void __launch_bounds__(1024) sort_tokens_kernel(const int* __restrict__ ids, int N,
                                                           int V, TokenSegs ts) {
  extern __shared__ unsigned long long key[];
  int P2 = 1;
  while (P2 < N) P2 <<= 1;
  int* scan = reinterpret_cast<int*>(key + P2);   // [1024] per-thread segment counts
  __shared__ int n_valid;
  const int t = threadIdx.x;
  for (int i = t; i < P2; i += blockDim.x) {
    const unsigned long long id = i < N ? (unsigned long long)(unsigned)(ids[i] < 0 ? V : ids[i])
                                        : 0xffffffffull;
    key[i] = (id << 32) | (unsigned)i;
  }
  for (int v = t; v < V; v += blockDim.x) ts.tok2seg[v] = -1;
  if (t == 0) n_valid = 0;
  __syncthreads();
  for (int k = 2; k <= P2; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = t; i < P2; i += blockDim.x) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const bool up = (i & k) == 0;
          const unsigned long long x = key[i], y = key[ixj];
          if ((x > y) == up) {
            key[i] = y;
            key[ixj] = x;
          }
        }
      }
      __syncthreads();
    }
  }
  for (int i = t; i < N; i += blockDim.x) ts.perm[i] = (int)(key[i] & 0xffffffffu);
  // Segment heads: the first sorted index of a run of one id, and every
  // multiple of EMB_SEG inside a run.  Ids >= V (ignored positions) sort last.
  auto tok = [&](int i) { return (unsigned)(key[i] >> 32); };
  auto head = [&](int i) {
    return i < N && tok(i) < (unsigned)V &&
           (i == 0 || tok(i - 1) != tok(i) || i % EMB_SEG == 0);
  };
  const int C = (P2 + 1023) / 1024;   // sorted indices per thread
  int cnt = 0;
  for (int c = 0; c < C; ++c) {
    const int i = t * C + c;
    if (head(i)) ++cnt;
    if (i < N && tok(i) < (unsigned)V && (i + 1 == N || tok(i + 1) >= (unsigned)V)) n_valid = i + 1;
  }
  scan[t] = cnt;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {   // inclusive scan of the counts
    const int add = t >= off ? scan[t - off] : 0;
    __syncthreads();
    scan[t] += add;
    __syncthreads();
  }
  int idx = scan[t] - cnt;
  for (int c = 0; c < C; ++c) {
    const int i = t * C + c;
    if (head(i)) {
      ts.seg_start[idx] = i;
      ts.seg_tok[idx] = (int)tok(i);
      if (i == 0 || tok(i - 1) != tok(i)) ts.tok2seg[tok(i)] = idx;
      ++idx;
    }
  }
  if (t == 0) {
    ts.nseg[0] = scan[1023];
    ts.seg_start[scan[1023]] = n_valid;   // end of the last segment
  }
}

// Sum of dh (and dhd) over the positions of one segment per wave:
// part[s][0][:] and part[s][1][:].
__global__ void __launch_bounds__(256) embed_seg_kernel(EmbedGradArgs a) {
  const int sg = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (sg >= a.ts.nseg[0]) return;
  const int p0 = a.ts.seg_start[sg], p1 = a.ts.seg_start[sg + 1];
  const int d = a.d;
  const bool vec = (d & 3) == 0;
  for (int j = lane * 4; j < d; j += 256) {
    const int cnt = min(4, d - j);
    float g[4] = {0.f, 0.f, 0.f, 0.f}, h[4] = {0.f, 0.f, 0.f, 0.f};
    for (int p = p0; p < p1; ++p) {
      const long off = (long)a.ts.perm[p] * d + j;
      if (vec) {
        const float4 x = *reinterpret_cast<const float4*>(a.dh + off);
        g[0] += x.x; g[1] += x.y; g[2] += x.z; g[3] += x.w;
        if (a.dhd) {
          const float4 y = *reinterpret_cast<const float4*>(a.dhd + off);
          h[0] += y.x; h[1] += y.y; h[2] += y.z; h[3] += y.w;
        }
      } else {
        for (int k = 0; k < cnt; ++k) {
          g[k] += a.dh[off + k];
          if (a.dhd) h[k] += a.dhd[off + k];
        }
      }
    }
    float* out = a.part + (long)sg * 2 * d + j;
    for (int k = 0; k < cnt; ++k) {
      out[k] = g[k];
      out[d + k] = h[k];
    }
  }
}

// g[v][j] = sum over positions n with ids[n] == v of dh[n][j] (tangent too),
// added up from the token's segment sums in order, then the parameter
// epilogue over every vocabulary row (rows without occurrences get g = 0).
template <typename T>
__global__ void __launch_bounds__(256) embed_grad_kernel(EmbedGradArgs a, ParamArgs<T> P) {
  const long e4 = ((long)blockIdx.x * 256 + threadIdx.x) * 4;  // 4 consecutive j
  const int d = a.d;
  if (e4 >= (long)a.V * d) return;
  const int v = (int)(e4 / d), j = (int)(e4 % d);
  float g[4] = {0.f, 0.f, 0.f, 0.f}, hv[4] = {0.f, 0.f, 0.f, 0.f}, cv[4];
  const int cnt = min(4, d - j);
  const int s0 = a.ts.tok2seg[v];
  if (s0 >= 0) {
    const int ns = a.ts.nseg[0];
    for (int sg = s0; sg < ns && a.ts.seg_tok[sg] == v; ++sg) {
      const float* in = a.part + (long)sg * 2 * d + j;
      for (int k = 0; k < cnt; ++k) {
        g[k] += in[k];
        hv[k] += in[d + k];
      }
    }
  }
  param_apply(P, a.emb_off + (long)v * d + j, cnt, g, hv, cv);
  if (a.outE)
    for (int k = 0; k < cnt; ++k) a.outE[(long)v * d + j + k] = cv[k];
}

// ------------------------------------------------------------------------------------
// Loss-weighting meta-model u = w2 . tanh(e W1 + b1) + b2 (alpha = sigmoid(u)):
// the hidden layer is a gemm_nt product; these are its output row and VJP.
// ------------------------------------------------------------------------------------
__global__ void __launch_bounds__(256) meta_out_kernel(const float* __restrict__ hid, int rows,
                                                       int hdim, const float* __restrict__ w2,
                                                       const float* __restrict__ b2, float* u) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  float s = 0.f;
  for (int j = lane; j < hdim; j += 64) s += hid[(long)row * hdim + j] * w2[j];
  s = wave_sum(s);
  if (lane == 0) u[row] = s + b2[0];
}

// dhid[n][j] = ubar_n w2_j (1 - hid^2); per-block partials of
// sum_n ubar_n hid[n][j] (-> d w2), sum_n dhid[n][j] (-> d b1), sum_n ubar_n (-> d b2).
__global__ void __launch_bounds__(256) meta_vjp_rows_kernel(const float* __restrict__ hid,
                                                            const float* __restrict__ ubar,
                                                            int rows, int hdim,
                                                            const float* __restrict__ w2,
                                                            float* dhid, float* partial,
                                                            int rows_per_block) {
  // thread t handles column j = t of the block's row range (hdim <= 256)
  const int j = threadIdx.x;
  const int r0 = blockIdx.x * rows_per_block;
  const int r1 = min(rows, r0 + rows_per_block);
  float sw = 0.f, sb = 0.f, su = 0.f;
  if (j < hdim) {
    for (int n = r0; n < r1; ++n) {
      const float h = hid[(long)n * hdim + j];
      const float ub = ubar[n];
      const float dh = ub * w2[j] * (1.0f - h * h);
      dhid[(long)n * hdim + j] = dh;
      sw += ub * h;
      sb += dh;
      su += ub;
    }
    float* Pp = partial + (long)blockIdx.x * (2 * hdim + 1);
    Pp[j] = sw;
    Pp[hdim + j] = sb;
    if (j == 0) Pp[2 * hdim] = su;
  }
}

__global__ void meta_vjp_reduce_kernel(const float* __restrict__ partial, int nparts, int hdim,
                                       float* d_w2, float* d_b1, float* d_b2) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j > hdim) return;
  if (j == hdim) {
    float s = 0.f;
    for (int p = 0; p < nparts; ++p) s += partial[(long)p * (2 * hdim + 1) + 2 * hdim];
    d_b2[0] = s;
    return;
  }
  float sw = 0.f, sb = 0.f;
  for (int p = 0; p < nparts; ++p) {
    sw += partial[(long)p * (2 * hdim + 1) + j];
    sb += partial[(long)p * (2 * hdim + 1) + hdim + j];
  }
  d_w2[j] = sw;
  d_b1[j] = sb;
}

}  // namespace

hipError_t split_tokens(const int* tok, int B, int S, int V, int* ids, int* labels,
                        hipStream_t s) {
  hipLaunchKernelGGL(split_tokens_kernel, dim3(cdivl((long)B * S, 256)), dim3(256), 0, s, tok, B,
                     S, V, ids, labels);
  return hipGetLastError();
}

hipError_t gather_rows(const int* ids, int N, int d, const float* E, const float* Ed, float* h,
                       float* hd, hipStream_t s) {
  hipLaunchKernelGGL(gather_rows_kernel, dim3(cdivl((long)N * d, 256)), dim3(256), 0, s, ids, N, d,
                     E, Ed, h, hd);
  return hipGetLastError();
}

hipError_t ln_fwd(const LnArgs& a, hipStream_t s) {
  if ((a.yb || a.ydb) && (a.d % 256 || a.ldb % 4)) return hipErrorInvalidValue;
  if (a.d % 256 == 0)
    hipLaunchKernelGGL(ln_fwd_vec_kernel, dim3(cdivl(a.N, 4)), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(ln_fwd_kernel, dim3(cdivl(a.N, 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

int ln_bwd_parts(int N) { return cdivl(N, LN_CHUNK); }

template <typename T>
hipError_t ln_bwd(const LnBwdArgs& a, long g_off, long b_off, const ParamArgs<T>& P,
                  float* out_g, float* out_b, hipStream_t s) {
  if (a.N <= 0) return hipSuccess;
  if ((a.hb || a.hdb) && (a.d % 256 || a.ldb % 4)) return hipErrorInvalidValue;
  if (a.d % 256 == 0)
    hipLaunchKernelGGL(ln_bwd_vec_kernel, dim3(cdivl(a.N, 4)), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(ln_bwd_kernel, dim3(cdivl(a.N, 4)), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(ln_colsum_kernel, dim3(cdivl(a.d, 64), ln_bwd_parts(a.N)), dim3(256), 0, s,
                     a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(ln_param_kernel<T>, dim3(cdivl(a.d, 16)), dim3(256), 0, s, a.partial,
                     ln_bwd_parts(a.N), a.d, g_off, b_off, P, out_g, out_b);
  return hipGetLastError();
}

hipError_t rope_table(int S, int dh, double base, float* cs, float* sn, hipStream_t s) {
  hipLaunchKernelGGL(rope_table_kernel, dim3(cdivl((long)S * dh / 2, 256)), dim3(256), 0, s, S, dh,
                     base, cs, sn);
  return hipGetLastError();
}

hipError_t rope_split(const RopeArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(rope_split_kernel, dim3(cdivl((long)a.N * a.H * a.dh, 256)), dim3(256), 0, s,
                     a);
  return hipGetLastError();
}

hipError_t rope_merge(const RopeArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(rope_merge_kernel, dim3(cdivl((long)a.N * a.H * a.dh, 256)), dim3(256), 0, s,
                     a);
  return hipGetLastError();
}

hipError_t softmax_fwd(const SoftmaxArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(softmax_fwd_kernel, dim3(cdivl(a.rows, 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t softmax_bwd(const SoftmaxArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(softmax_bwd_kernel, dim3(cdivl(a.rows, 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

bool sort_tokens_fits(int N) { return N >= 1 && N <= TOKEN_SORT_MAX; }

int embed_segments_max(int N) { return N + (N + EMB_SEG - 1) / EMB_SEG; }

hipError_t sort_tokens(const int* ids, int N, int V, const TokenSegs& ts, hipStream_t s) {
  if (!sort_tokens_fits(N)) return hipErrorInvalidValue;
  int P2 = 1;
  while (P2 < N) P2 <<= 1;
  hipLaunchKernelGGL(sort_tokens_kernel, dim3(1), dim3(1024),
                     P2 * sizeof(unsigned long long) + 1024 * sizeof(int), s, ids, N, V, ts);
  return hipGetLastError();
}

template <typename T>
hipError_t embed_grad(const EmbedGradArgs& a, const ParamArgs<T>& P, hipStream_t s) {
  hipLaunchKernelGGL(embed_seg_kernel, dim3(cdivl(embed_segments_max(a.N), 4)), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(embed_grad_kernel<T>, dim3(cdivl((long)a.V * a.d / 4 + 1, 256)), dim3(256), 0,
                     s, a, P);
  return hipGetLastError();
}

hipError_t meta_out(const float* hid, int rows, int hdim, const float* w2, const float* b2,
                    float* u, hipStream_t s) {
  hipLaunchKernelGGL(meta_out_kernel, dim3(cdivl(rows, 4)), dim3(256), 0, s, hid, rows, hdim, w2,
                     b2, u);
  return hipGetLastError();
}

int meta_vjp_parts(int rows) { return cdivl(rows, META_ROWS_PER_BLOCK); }

hipError_t meta_vjp(const float* hid, const float* ubar, int rows, int hdim, const float* w2,
                    float* dhid, float* partial, float* d_w2, float* d_b1, float* d_b2,
                    hipStream_t s) {
  const int parts = meta_vjp_parts(rows);
  hipLaunchKernelGGL(meta_vjp_rows_kernel, dim3(parts), dim3(256), 0, s, hid, ubar, rows, hdim, w2,
                     dhid, partial, META_ROWS_PER_BLOCK);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(meta_vjp_reduce_kernel, dim3(cdivl(hdim + 1, 256)), dim3(256), 0, s, partial,
                     parts, hdim, d_w2, d_b1, d_b2);
  return hipGetLastError();
}

template hipError_t ln_bwd<bf16_t>(const LnBwdArgs&, long, long, const ParamArgs<bf16_t>&, float*, float*, hipStream_t);
template hipError_t ln_bwd<float>(const LnBwdArgs&, long, long, const ParamArgs<float>&, float*, float*, hipStream_t);
template hipError_t embed_grad<bf16_t>(const EmbedGradArgs&, const ParamArgs<bf16_t>&, hipStream_t);
template hipError_t embed_grad<float>(const EmbedGradArgs&, const ParamArgs<float>&, hipStream_t);

}  // namespace mfmg
