// Fused causal dual attention for head dimension 64 with bf16 operands.
//
// Attention of one head, with scores S = s Q K^T (s = 1/sqrt(64)), causal
// mask, P = softmax(S) by rows and O = P V, and its tangent along (Qd, Kd, Vd)
// (the forward-mode half of the forward-over-reverse HVP, Section 2.2):
//   Sd = s (Qd K^T + Q Kd^T),  Pd = P (Sd - c),  c = rowsum(P Sd),
//   Od = Pd V + P Vd = (P Sd) V - c O + P Vd.
// The forward walks the key blocks of a query block once, keeping a running
// row maximum m, the partial sums l = sum exp(S - m) and sum exp(S - m) Sd,
// and three accumulators (for P V, (P Sd) V and P Vd) rescaled whenever m
// grows.  It saves lse = m + log l and c per query row; nothing of size S^2
// is stored.  The backward recomputes P and Pd from them:
//   dP = dO V^T,  dPd = dOd V^T + dO Vd^T,
//   r = rowsum(P dP) = <dO, O>,  rd = rowsum(Pd dP + P dPd) = <dOd, O> + <dO, Od>,
//   dS = s P (dP - r),  dSd = s (Pd (dP - r) + P (dPd - rd)),
//   dQ = dS K,  dQd = dSd K + dS Kd,  dK = dS^T Q,  dKd = dSd^T Q + dS^T Qd,
//   dV = P^T dO,  dVd = Pd^T dO + P^T dOd,
// in two passes: one per query block (dQ, dQd; it also writes r and rd) and
// one per key block (dK, dKd, dV, dVd), so every output has one writer and
// the sums run in a fixed order.
//
// Tiles of 64 queries x 64 keys; four waves per workgroup, each owning 16
// rows.  Products use v_mfma_f32_16x16x32_bf16 in the NT form (both operands
// with the contraction index contiguous): a lane holds row lane%16, elements
// 8 (lane/16) .. +7 of a 32-deep slice, and the accumulator holds rows
// 4 (lane/16) + 0..3 of column lane%16.  Probabilities and score cotangents
// go through a per-wave LDS tile to move from the accumulator layout to the
// operand layout.
#include "transformer.h"

namespace mfmg {

namespace {

constexpr int AB = 64;       // queries or keys per block
constexpr int DH = 64;       // head dimension
constexpr int LP = DH + 8;   // LDS row pitch in bf16 elements (144 bytes)

__device__ __forceinline__ f32x4 mma(const bf16x8& a, const bf16x8& b, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 ld8(const bf16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

// 64 x 64 tile of a row-major bf16 matrix (leading dimension ld) into LDS.
__device__ __forceinline__ void stage(bf16_t* lds, const bf16_t* __restrict__ g, long ld, int tid) {
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = tid + 256 * k, r = i >> 3, ch = i & 7;
    *reinterpret_cast<uint4*>(lds + r * LP + ch * 8) =
        *reinterpret_cast<const uint4*>(g + (long)r * ld + ch * 8);
  }
}

// Operand fragment c (0, 1) of row `row` of an LDS tile.
__device__ __forceinline__ bf16x8 frag(const bf16_t* lds, int row, int lg, int c) {
  return ld8(lds + row * LP + 8 * lg + 32 * c);
}

__device__ __forceinline__ float max16(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float sum16(float v) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// ---------------------------------------------------------------- forward
template <bool DUAL>
__global__ void __launch_bounds__(256) attn_fwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t sK[AB * LP], sKd[AB * LP], sVT[DH * LP],
      sVdT[DH * LP];
  __shared__ __attribute__((aligned(16))) bf16_t sP[4][16 * LP], sPd[4][16 * LP];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int S = a.S, nqb = S / AB;
  const int qb = nqb - 1 - (int)blockIdx.x;  // longest rows first
  const int bh = blockIdx.y;
  const long hb = (long)bh * S * DH, tb = (long)bh * DH * S;
  const int q0 = qb * AB + w * 16;
  bf16x8 qf[2], qdf[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    qf[c] = ld8(a.Q + hb + (long)(q0 + lr) * DH + 8 * lg + 32 * c);
    if (DUAL) qdf[c] = ld8(a.Qd + hb + (long)(q0 + lr) * DH + 8 * lg + 32 * c);
  }
  float m[4], l[4], cs[4];
  f32x4 o[4], o2[4], o3[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m[i] = -INFINITY; l[i] = 0.f; cs[i] = 0.f;
    o[i] = zero4(); o2[i] = zero4(); o3[i] = zero4();
  }
  const float sc = a.scale;
  for (int kb = 0; kb <= qb; ++kb) {
    __syncthreads();
    stage(sK, a.K + hb + (long)kb * AB * DH, DH, tid);
    stage(sVT, a.VT + tb + kb * AB, S, tid);
    if (DUAL) {
      stage(sKd, a.Kd + hb + (long)kb * AB * DH, DH, tid);
      stage(sVdT, a.VdT + tb + kb * AB, S, tid);
    }
    __syncthreads();
    f32x4 s[4], sd[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      s[n] = zero4(); sd[n] = zero4();
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const bf16x8 kf = frag(sK, n * 16 + lr, lg, c);
        s[n] = mma(qf[c], kf, s[n]);
        if (DUAL) {
          sd[n] = mma(qdf[c], kf, sd[n]);
          sd[n] = mma(qf[c], frag(sKd, n * 16 + lr, lg, c), sd[n]);
        }
      }
    }
    const bool diag = kb == qb;
    float al[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int qrow = w * 16 + 4 * lg + r;  // within the block
      float mx = -INFINITY;
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        float v = s[n][r] * sc;
        if (diag && n * 16 + lr > qrow) v = -INFINITY;
        s[n][r] = v;
        mx = fmaxf(mx, v);
      }
      mx = max16(mx);
      const float mn = fmaxf(m[r], mx);
      al[r] = __expf(m[r] - mn);
      m[r] = mn;
      float ls = 0.f, lc = 0.f;
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        const float p = __expf(s[n][r] - mn);
        ls += p;
        sP[w][(4 * lg + r) * LP + n * 16 + lr] = f2bf(p);
        if (DUAL) {
          const float t = p * sd[n][r] * sc;
          lc += t;
          sPd[w][(4 * lg + r) * LP + n * 16 + lr] = f2bf(t);
        }
      }
      l[r] = l[r] * al[r] + ls;
      if (DUAL) cs[r] = cs[r] * al[r] + lc;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        o[e][r] *= al[r];
        if (DUAL) { o2[e][r] *= al[r]; o3[e][r] *= al[r]; }
      }
    __syncthreads();
    bf16x8 pf[2], pdf[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      pf[c] = frag(sP[w], lr, lg, c);
      if (DUAL) pdf[c] = frag(sPd[w], lr, lg, c);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const bf16x8 vf = frag(sVT, e * 16 + lr, lg, c);
        o[e] = mma(pf[c], vf, o[e]);
        if (DUAL) {
          o2[e] = mma(pdf[c], vf, o2[e]);
          o3[e] = mma(pf[c], frag(sVdT, e * 16 + lr, lg, c), o3[e]);
        }
      }
  }
  const int bs = bh / a.H, h = bh % a.H;
  const long tok0 = (long)bs * S + q0 + 4 * lg;  // token of accumulator row 0
  float inv[4], cc[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float lt = sum16(l[r]);
    inv[r] = 1.0f / lt;
    cc[r] = DUAL ? sum16(cs[r]) * inv[r] : 0.f;
    if (lr == 0) {
      a.lse[(long)bh * S + q0 + 4 * lg + r] = m[r] + __logf(lt);
      if (DUAL) a.cst[(long)bh * S + q0 + 4 * lg + r] = cc[r];
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int col = h * DH + e * 16 + lr;
    float ov[4], odv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      ov[r] = o[e][r] * inv[r];
      a.O[(tok0 + r) * a.ldO + col] = f2bf(ov[r]);
      if (DUAL) {
        odv[r] = (o2[e][r] + o3[e][r]) * inv[r] - cc[r] * ov[r];
        a.Od[(tok0 + r) * a.ldO + col] = f2bf(odv[r]);
      }
    }
    store4(a.OT + (long)col * a.ldOT + tok0, ov[0], ov[1], ov[2], ov[3]);
    if (DUAL) store4(a.OdT + (long)col * a.ldOT + tok0, odv[0], odv[1], odv[2], odv[3]);
  }
}

// ---------------------------------------------------------------- backward: dQ
template <bool DUAL>
__global__ void __launch_bounds__(256) attn_bwd_dq_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t sK[AB * LP], sKd[AB * LP], sV[AB * LP],
      sVd[AB * LP], sKT[DH * LP], sKdT[DH * LP];
  __shared__ __attribute__((aligned(16))) bf16_t sS[4][16 * LP], sSd[4][16 * LP];
  __shared__ float sR[4][16], sRd[4][16];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int S = a.S, nqb = S / AB;
  const int qb = nqb - 1 - (int)blockIdx.x;
  const int bh = blockIdx.y;
  const int bs = bh / a.H, h = bh % a.H;
  const long hb = (long)bh * S * DH, tb = (long)bh * DH * S;
  const int q0 = qb * AB + w * 16;
  bf16x8 qf[2], qdf[2], gf[2], gdf[2];
  float r0 = 0.f, r1 = 0.f;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const long off = hb + (long)(q0 + lr) * DH + 8 * lg + 32 * c;
    qf[c] = ld8(a.Q + off);
    gf[c] = ld8(a.dO + off);
    const long ooff = ((long)bs * S + q0 + lr) * a.ldO + h * DH + 8 * lg + 32 * c;
    const bf16x8 of = ld8(a.O + ooff);
    if (DUAL) {
      qdf[c] = ld8(a.Qd + off);
      gdf[c] = ld8(a.dOd + off);
      const bf16x8 odf = ld8(a.Od + ooff);
#pragma unroll
      for (int k = 0; k < 8; ++k)
        r1 += (float)gdf[c][k] * (float)of[k] + (float)gf[c][k] * (float)odf[k];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) r0 += (float)gf[c][k] * (float)of[k];
  }
  r0 += __shfl_xor(r0, 16, 64);
  r0 += __shfl_xor(r0, 32, 64);
  if (DUAL) {
    r1 += __shfl_xor(r1, 16, 64);
    r1 += __shfl_xor(r1, 32, 64);
  }
  if (lg == 0) {
    sR[w][lr] = r0;
    sRd[w][lr] = r1;
    a.r[(long)bh * S + q0 + lr] = r0;
    if (DUAL) a.rd[(long)bh * S + q0 + lr] = r1;
  }
  __syncthreads();
  float rr[4], rrd[4], lse[4], cst[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    rr[r] = sR[w][4 * lg + r];
    rrd[r] = sRd[w][4 * lg + r];
    lse[r] = a.lse[(long)bh * S + q0 + 4 * lg + r];
    cst[r] = DUAL ? a.cst[(long)bh * S + q0 + 4 * lg + r] : 0.f;
  }
  f32x4 dq[4], dqd[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) { dq[e] = zero4(); dqd[e] = zero4(); }
  const float sc = a.scale;
  for (int kb = 0; kb <= qb; ++kb) {
    __syncthreads();
    stage(sK, a.K + hb + (long)kb * AB * DH, DH, tid);
    stage(sV, a.V + hb + (long)kb * AB * DH, DH, tid);
    stage(sKT, a.KT + tb + kb * AB, S, tid);
    if (DUAL) {
      stage(sKd, a.Kd + hb + (long)kb * AB * DH, DH, tid);
      stage(sVd, a.Vd + hb + (long)kb * AB * DH, DH, tid);
      stage(sKdT, a.KdT + tb + kb * AB, S, tid);
    }
    __syncthreads();
    const bool diag = kb == qb;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      f32x4 s = zero4(), sd = zero4(), dp = zero4(), dpd = zero4();
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const bf16x8 kf = frag(sK, n * 16 + lr, lg, c), vf = frag(sV, n * 16 + lr, lg, c);
        s = mma(qf[c], kf, s);
        dp = mma(gf[c], vf, dp);
        if (DUAL) {
          sd = mma(qdf[c], kf, sd);
          sd = mma(qf[c], frag(sKd, n * 16 + lr, lg, c), sd);
          dpd = mma(gdf[c], vf, dpd);
          dpd = mma(gf[c], frag(sVd, n * 16 + lr, lg, c), dpd);
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool ok = !diag || n * 16 + lr <= w * 16 + 4 * lg + r;
        const float p = ok ? __expf(s[r] * sc - lse[r]) : 0.f;
        const float g = dp[r] - rr[r];
        sS[w][(4 * lg + r) * LP + n * 16 + lr] = f2bf(sc * p * g);
        if (DUAL) {
          const float pd = p * (sd[r] * sc - cst[r]);
          sSd[w][(4 * lg + r) * LP + n * 16 + lr] = f2bf(sc * (pd * g + p * (dpd[r] - rrd[r])));
        }
      }
    }
    __syncthreads();
    bf16x8 df[2], ddf[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      df[c] = frag(sS[w], lr, lg, c);
      if (DUAL) ddf[c] = frag(sSd[w], lr, lg, c);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const bf16x8 kt = frag(sKT, e * 16 + lr, lg, c);
        dq[e] = mma(df[c], kt, dq[e]);
        if (DUAL) {
          dqd[e] = mma(ddf[c], kt, dqd[e]);
          dqd[e] = mma(df[c], frag(sKdT, e * 16 + lr, lg, c), dqd[e]);
        }
      }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const long off = hb + (long)(q0 + 4 * lg + r) * DH + e * 16 + lr;
      a.dQ[off] = dq[e][r];
      if (DUAL) a.dQd[off] = dqd[e][r];
    }
}

// ---------------------------------------------------------------- backward: dK, dV
template <bool DUAL>
__global__ void __launch_bounds__(256) attn_bwd_dkv_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t sQ[AB * LP], sQd[AB * LP], sG[AB * LP],
      sGd[AB * LP], sQT[DH * LP], sQdT[DH * LP], sGT[DH * LP], sGdT[DH * LP];
  __shared__ __attribute__((aligned(16))) bf16_t sP[4][16 * LP], sPd[4][16 * LP],
      sS[4][16 * LP], sSd[4][16 * LP];
  __shared__ float sL[AB], sC[AB], sR[AB], sRd[AB];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int S = a.S, nqb = S / AB;
  const int kb = blockIdx.x;  // key block 0 has the most query blocks
  const int bh = blockIdx.y;
  const long hb = (long)bh * S * DH, tb = (long)bh * DH * S;
  const int k0 = kb * AB + w * 16;
  bf16x8 kf[2], kdf[2], vf[2], vdf[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const long off = hb + (long)(k0 + lr) * DH + 8 * lg + 32 * c;
    kf[c] = ld8(a.K + off);
    vf[c] = ld8(a.V + off);
    if (DUAL) {
      kdf[c] = ld8(a.Kd + off);
      vdf[c] = ld8(a.Vd + off);
    }
  }
  f32x4 dk[4], dkd[4], dv[4], dvd[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) { dk[e] = zero4(); dkd[e] = zero4(); dv[e] = zero4(); dvd[e] = zero4(); }
  const float sc = a.scale;
  for (int qb = kb; qb < nqb; ++qb) {
    __syncthreads();
    stage(sQ, a.Q + hb + (long)qb * AB * DH, DH, tid);
    stage(sG, a.dO + hb + (long)qb * AB * DH, DH, tid);
    stage(sQT, a.QT + tb + qb * AB, S, tid);
    stage(sGT, a.dOT + tb + qb * AB, S, tid);
    if (DUAL) {
      stage(sQd, a.Qd + hb + (long)qb * AB * DH, DH, tid);
      stage(sGd, a.dOd + hb + (long)qb * AB * DH, DH, tid);
      stage(sQdT, a.QdT + tb + qb * AB, S, tid);
      stage(sGdT, a.dOdT + tb + qb * AB, S, tid);
    }
    if (tid < AB) {
      const long i = (long)bh * S + qb * AB + tid;
      sL[tid] = a.lse[i];
      sR[tid] = a.r[i];
      if (DUAL) {
        sC[tid] = a.cst[i];
        sRd[tid] = a.rd[i];
      }
    }
    __syncthreads();
    const bool diag = kb == qb;
#pragma unroll
    for (int n = 0; n < 4; ++n) {  // 16 queries n*16 .. of the block
      f32x4 s = zero4(), sd = zero4(), dp = zero4(), dpd = zero4();
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const bf16x8 qq = frag(sQ, n * 16 + lr, lg, c), gg = frag(sG, n * 16 + lr, lg, c);
        s = mma(kf[c], qq, s);
        dp = mma(vf[c], gg, dp);
        if (DUAL) {
          sd = mma(kdf[c], qq, sd);
          sd = mma(kf[c], frag(sQd, n * 16 + lr, lg, c), sd);
          dpd = mma(vdf[c], gg, dpd);
          dpd = mma(vf[c], frag(sGd, n * 16 + lr, lg, c), dpd);
        }
      }
      const int ql = n * 16 + lr;
      const float L = sL[ql], R = sR[ql];
      const float C = DUAL ? sC[ql] : 0.f, Rd = DUAL ? sRd[ql] : 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {  // key w*16 + 4*lg + r of the block
        const bool ok = !diag || w * 16 + 4 * lg + r <= ql;
        const float p = ok ? __expf(s[r] * sc - L) : 0.f;
        const float g = dp[r] - R;
        const int at = (4 * lg + r) * LP + ql;
        sP[w][at] = f2bf(p);
        sS[w][at] = f2bf(sc * p * g);
        if (DUAL) {
          const float pd = p * (sd[r] * sc - C);
          sPd[w][at] = f2bf(pd);
          sSd[w][at] = f2bf(sc * (pd * g + p * (dpd[r] - Rd)));
        }
      }
    }
    __syncthreads();
    bf16x8 pf[2], pdf[2], df[2], ddf[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      pf[c] = frag(sP[w], lr, lg, c);
      df[c] = frag(sS[w], lr, lg, c);
      if (DUAL) {
        pdf[c] = frag(sPd[w], lr, lg, c);
        ddf[c] = frag(sSd[w], lr, lg, c);
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const bf16x8 gt = frag(sGT, e * 16 + lr, lg, c), qt = frag(sQT, e * 16 + lr, lg, c);
        dv[e] = mma(pf[c], gt, dv[e]);
        dk[e] = mma(df[c], qt, dk[e]);
        if (DUAL) {
          dvd[e] = mma(pdf[c], gt, dvd[e]);
          dvd[e] = mma(pf[c], frag(sGdT, e * 16 + lr, lg, c), dvd[e]);
          dkd[e] = mma(ddf[c], qt, dkd[e]);
          dkd[e] = mma(df[c], frag(sQdT, e * 16 + lr, lg, c), dkd[e]);
        }
      }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const long off = hb + (long)(k0 + 4 * lg + r) * DH + e * 16 + lr;
      a.dK[off] = dk[e][r];
      a.dV[off] = dv[e][r];
      if (DUAL) {
        a.dKd[off] = dkd[e][r];
        a.dVd[off] = dvd[e][r];
      }
    }
}

}  // namespace

bool attn_fused_supported(int S, int dh) { return dh == DH && S >= AB && S % AB == 0; }

hipError_t attn_fwd(const AttnArgs& a, hipStream_t s) {
  if (!attn_fused_supported(a.S, a.dh) || a.BH < 1 || a.H < 1 || a.BH % a.H) return hipErrorInvalidValue;
  const dim3 g(a.S / AB, a.BH);
  if (a.dual)
    hipLaunchKernelGGL(attn_fwd_kernel<true>, g, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<false>, g, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t attn_bwd(const AttnArgs& a, hipStream_t s) {
  if (!attn_fused_supported(a.S, a.dh) || a.BH < 1 || a.H < 1 || a.BH % a.H) return hipErrorInvalidValue;
  const dim3 g(a.S / AB, a.BH);
  if (a.dual) {
    hipLaunchKernelGGL(attn_bwd_dq_kernel<true>, g, dim3(256), 0, s, a);
    hipLaunchKernelGGL(attn_bwd_dkv_kernel<true>, g, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL(attn_bwd_dq_kernel<false>, g, dim3(256), 0, s, a);
    hipLaunchKernelGGL(attn_bwd_dkv_kernel<false>, g, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace mfmg
