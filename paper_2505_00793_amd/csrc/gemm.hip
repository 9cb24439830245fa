// Dual NT GEMM for gfx950 with fused epilogues.
//
// One kernel template computes a matrix product and, optionally, its tangent:
//   C1 = A B^T,   C2 = Ad B^T + A Bd^T
// which covers every product of a forward-over-reverse pass through an MLP
// layer (Section 2.2 and Section 3: the JVP of the gradient map):
//   dual forward          Z  = A W,       Zd  = Ad W + A Wd
//   dual backward-data    dA = dZ W^T,    dAd = dZd W^T + dZ Wd^T
//   dual backward-weight  G  = A^T dZ,    Gd  = Ad^T dZ + A^T dZd   (= H v)
// All operands are stored with the contraction index contiguous (the
// producers write both layouts), so tiles go from HBM to LDS with 16-byte
// loads and from LDS to the MFMA units with 16-byte reads and no transposes.
// Tiles of A, Ad, B, Bd are staged together in LDS, so each HBM read of a
// weight tile serves the primal and the tangent product.
//
// Matrix cores: v_mfma_f32_16x16x32_bf16 (bf16 operands) or
// v_mfma_f32_16x16x4_f32 (float32 operands), 64-lane wavefronts, 4 waves per
// workgroup in a 2 x 2 arrangement, double-buffered LDS, one barrier per
// 32-deep k step.
#include "kernels.h"
#include "param_epi.h"

namespace mfmg {

namespace {

constexpr int BK = 32;

__device__ __forceinline__ void mma(f32x4& acc, const bf16x8& a, const bf16x8& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x4& acc, const f32x4& a, const f32x4& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], acc, 0, 0, 0);
}

template <typename T> struct Frag;
template <> struct Frag<bf16_t> { typedef bf16x8 type; };
template <> struct Frag<float> { typedef f32x4 type; };

// 16 bytes of row gr starting at column gk, zero outside [0,M) x [0,K).
template <typename T>
__device__ __forceinline__ uint4 load_chunk(const T* __restrict__ src, int gr, int gk, int M,
                                            int K, int ld) {
  constexpr int VE = Elem<T>::VE;
  if (gr < M && gk + VE <= K) return *reinterpret_cast<const uint4*>(src + (long)gr * ld + gk);
  union {
    uint4 v;
    T e[VE];
  } u;
  u.v = make_uint4(0, 0, 0, 0);
  if (gr < M) {
#pragma unroll
    for (int e = 0; e < VE; ++e)
      if (gk + e < K) u.e[e] = src[(long)gr * ld + gk + e];
  }
  return u.v;
}

template <typename T, int FLAGS, int BM, int BN, class Epi>
__global__ void __launch_bounds__(256) gemm_nt(GemmOperands<T> op, Epi epi) {
  constexpr int VE = Elem<T>::VE;
  constexpr int LDL = BK + VE;  // padded LDS row, in elements
  constexpr bool HC1 = (FLAGS & G_C1) != 0;
  constexpr bool HAD = (FLAGS & G_AD) != 0;
  constexpr bool HBD = (FLAGS & G_BD) != 0;
  constexpr int NAS = HAD ? 2 : 1;
  constexpr int NBS = HBD ? 2 : 1;
  constexpr int STAGE = (NAS * BM + NBS * BN) * LDL;
  constexpr int WTM = BM / 2, WTN = BN / 2;
  constexpr int TM = WTM / 16, TN = WTN / 16;
  constexpr int CPR = BK / VE;           // 16-byte chunks per tile row
  constexpr int ACH = BM * CPR / 256;    // chunks per thread, A-side tile
  constexpr int BCH = BN * CPR / 256;    // chunks per thread, B-side tile
  constexpr int NCH = BK / (4 * VE);     // 16-byte fragment reads per k step
  static_assert(ACH >= 1 && BCH >= 1 && (BM * CPR) % 256 == 0 && (BN * CPR) % 256 == 0, "tile");
  typedef typename Frag<T>::type frag_t;

  __shared__ __attribute__((aligned(16))) T smem[2 * STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Tile order.  Workgroup ids are dispatched round-robin over the 8 XCDs; give
  // each XCD a contiguous range of tiles, then walk tiles in groups of 8 tile
  // rows so that neighbouring tiles share A and B panels in that XCD's L2.
  const int tiles_m = (op.M + BM - 1) / BM;
  const int tiles_n = (op.N + BN - 1) / BN;
  const int nt = tiles_m * tiles_n;
  int pid = blockIdx.x;
  if ((nt & 7) == 0) pid = (pid & 7) * (nt >> 3) + (pid >> 3);
  constexpr int GM = 8;
  const int group = pid / (GM * tiles_n);
  const int first_m = group * GM;
  const int gsz = min(tiles_m - first_m, GM);
  const int within = pid - group * GM * tiles_n;
  const int tm = first_m + within % gsz;
  const int tn = within / gsz;
  const int m0 = tm * BM, n0 = tn * BN;

  uint4 ra[NAS][ACH], rb[NBS][BCH];

  auto gload = [&](int k0) {
#pragma unroll
    for (int s = 0; s < NAS; ++s) {
      const T* src = s == 0 ? op.A : op.Ad;
#pragma unroll
      for (int c = 0; c < ACH; ++c) {
        int ch = tid + c * 256;
        ra[s][c] = load_chunk<T>(src, m0 + ch / CPR, k0 + (ch % CPR) * VE, op.M, op.K, op.lda);
      }
    }
#pragma unroll
    for (int s = 0; s < NBS; ++s) {
      const T* src = s == 0 ? op.B : op.Bd;
#pragma unroll
      for (int c = 0; c < BCH; ++c) {
        int ch = tid + c * 256;
        rb[s][c] = load_chunk<T>(src, n0 + ch / CPR, k0 + (ch % CPR) * VE, op.N, op.K, op.ldb);
      }
    }
  };
  auto sstore = [&](int buf) {
    T* base = smem + buf * STAGE;
#pragma unroll
    for (int s = 0; s < NAS; ++s)
#pragma unroll
      for (int c = 0; c < ACH; ++c) {
        int ch = tid + c * 256;
        *reinterpret_cast<uint4*>(base + (s * BM + ch / CPR) * LDL + (ch % CPR) * VE) = ra[s][c];
      }
#pragma unroll
    for (int s = 0; s < NBS; ++s)
#pragma unroll
      for (int c = 0; c < BCH; ++c) {
        int ch = tid + c * 256;
        *reinterpret_cast<uint4*>(base + (NAS * BM + s * BN + ch / CPR) * LDL + (ch % CPR) * VE) =
            rb[s][c];
      }
  };

  f32x4 acc1[TM][TN], acc2[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      acc1[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      acc2[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

  const int nk = (op.K + BK - 1) / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
    const T* As = smem + buf * STAGE;
    const T* Ads = As + BM * LDL;
    const T* Bs = As + NAS * BM * LDL;
    const T* Bds = Bs + BN * LDL;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int kof = (lane >> 4) * VE + c * 4 * VE;
      frag_t a[TM], ad[TM], b[TN], bd[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * WTM + i * 16 + (lane & 15);
        a[i] = *reinterpret_cast<const frag_t*>(As + r * LDL + kof);
        if constexpr (HAD) ad[i] = *reinterpret_cast<const frag_t*>(Ads + r * LDL + kof);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * WTN + j * 16 + (lane & 15);
        b[j] = *reinterpret_cast<const frag_t*>(Bs + r * LDL + kof);
        if constexpr (HBD) bd[j] = *reinterpret_cast<const frag_t*>(Bds + r * LDL + kof);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          if constexpr (HC1) mma(acc1[i][j], a[i], b[j]);
          if constexpr (HAD) mma(acc2[i][j], ad[i], b[j]);
          if constexpr (HBD) mma(acc2[i][j], a[i], bd[j]);
        }
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // C layout of a 16x16 MFMA tile: lane holds rows 4*(lane/16) + 0..3 of
  // column lane%16.
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int mr = m0 + wm * WTM + i * 16 + (lane >> 4) * 4;
      const int nc = n0 + wn * WTN + j * 16 + (lane & 15);
      epi(mr, nc, acc1[i][j], acc2[i][j]);
    }
}

// ------------------------------------------------------------------------------------
// Epilogues
// ------------------------------------------------------------------------------------
template <typename T>
struct ActFwdOp {
  EpiActFwd<T> e;
  __device__ __forceinline__ void operator()(int m0, int n, const f32x4& c1, const f32x4& c2) const {
    if (n >= e.N) return;
    const float b = e.bias ? e.bias[n] : 0.0f;
    const float bd = (e.dual && e.bias_d) ? e.bias_d[n] : 0.0f;
    float a[4], ad[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + r;
      const float z = c1[r] + b;
      const float zd = c2[r] + bd;
      a[r] = 0.0f;
      ad[r] = 0.0f;
      if (m < e.M) {
        e.Z[(long)m * e.N + n] = z;
        if (e.dual) e.Zd[(long)m * e.N + n] = zd;
        if (!e.last) {
          a[r] = act_f(e.act, z);
          e.Ao[(long)m * e.ldA + n] = Elem<T>::from_float(a[r]);
          if (e.dual) {
            float d1, d2;
            act_d12(e.act, z, d1, d2);
            ad[r] = d1 * zd;
            e.Ado[(long)m * e.ldA + n] = Elem<T>::from_float(ad[r]);
          }
        }
      }
    }
    if (e.last) return;
    if (m0 + 3 < e.M) {
      store4(e.AoT + (long)n * e.ldAT + m0, a[0], a[1], a[2], a[3]);
      if (e.dual) store4(e.AdoT + (long)n * e.ldAT + m0, ad[0], ad[1], ad[2], ad[3]);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (m0 + r < e.M) {
          e.AoT[(long)n * e.ldAT + m0 + r] = Elem<T>::from_float(a[r]);
          if (e.dual) e.AdoT[(long)n * e.ldAT + m0 + r] = Elem<T>::from_float(ad[r]);
        }
    }
  }
};

template <typename T>
struct ActBwdOp {
  EpiActBwd<T> e;
  __device__ __forceinline__ void operator()(int m0, int n, const f32x4& c1, const f32x4& c2) const {
    if (n >= e.N) return;
    float dz[4], dzd[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + r;
      dz[r] = 0.0f;
      dzd[r] = 0.0f;
      if (m < e.M) {
        float d1, d2;
        act_d12(e.act, e.Zp[(long)m * e.N + n], d1, d2);
        dz[r] = c1[r] * d1;
        e.dZ[(long)m * e.ld + n] = Elem<T>::from_float(dz[r]);
        if (e.dual) {
          dzd[r] = c2[r] * d1 + c1[r] * d2 * e.Zdp[(long)m * e.N + n];
          e.dZd[(long)m * e.ld + n] = Elem<T>::from_float(dzd[r]);
        }
      }
    }
    if (m0 + 3 < e.M) {
      store4(e.dZT + (long)n * e.ldT + m0, dz[0], dz[1], dz[2], dz[3]);
      if (e.dual) store4(e.dZdT + (long)n * e.ldT + m0, dzd[0], dzd[1], dzd[2], dzd[3]);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (m0 + r < e.M) {
          e.dZT[(long)n * e.ldT + m0 + r] = Elem<T>::from_float(dz[r]);
          if (e.dual) e.dZdT[(long)n * e.ldT + m0 + r] = Elem<T>::from_float(dzd[r]);
        }
    }
  }
};

template <typename T>
struct ParamOp {
  ParamArgs<T> P;
  __device__ __forceinline__ void operator()(int m0, int n, const f32x4& c1, const f32x4& c2) const {
    if (n >= P.nout) return;
    float cv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + r;
      cv[r] = 0.0f;
      if (m < P.nin) {
        const long idx = P.w_off + (long)m * P.nout + n;
        cv[r] = param_elem(P, idx, c1[r], c2[r]);
        if (P.outW) P.outW[(long)m * P.ldW + n] = Elem<T>::from_float(cv[r]);
      }
    }
    if (!P.outWT) return;
    if (m0 + 3 < P.nin) {
      store4(P.outWT + (long)n * P.ldWT + m0, cv[0], cv[1], cv[2], cv[3]);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (m0 + r < P.nin) P.outWT[(long)n * P.ldWT + m0 + r] = Elem<T>::from_float(cv[r]);
    }
  }
};

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

template <typename T, int FLAGS, int BM, int BN, class Epi>
hipError_t launch(const GemmOperands<T>& op, const Epi& epi, hipStream_t s) {
  const int tiles = cdiv(op.M, BM) * cdiv(op.N, BN);
  hipLaunchKernelGGL((gemm_nt<T, FLAGS, BM, BN, Epi>), dim3(tiles), dim3(256), 0, s, op, epi);
  return hipGetLastError();
}

template <typename T, int FLAGS, class Epi>
hipError_t launch_sized(const GemmOperands<T>& op, const Epi& epi, hipStream_t s) {
  if (op.M <= 0 || op.N <= 0) return hipSuccess;
  if constexpr (sizeof(T) == 2) {
    // 128 x 128 tiles once they alone fill most of the 256 compute units.
    if (cdiv(op.M, 128) * cdiv(op.N, 128) >= 192) return launch<T, FLAGS, 128, 128>(op, epi, s);
  }
  return launch<T, FLAGS, 64, 64>(op, epi, s);
}

template <typename T, class Epi>
hipError_t dispatch(const GemmOperands<T>& op, int flags, const Epi& epi, hipStream_t s) {
  switch (flags) {
    case G_C1: return launch_sized<T, G_C1>(op, epi, s);
    case G_C1 | G_BD: return launch_sized<T, G_C1 | G_BD>(op, epi, s);
    case G_C1 | G_AD | G_BD: return launch_sized<T, G_C1 | G_AD | G_BD>(op, epi, s);
    case G_AD | G_BD: return launch_sized<T, G_AD | G_BD>(op, epi, s);
    case G_BD: return launch_sized<T, G_BD>(op, epi, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

template <typename T>
hipError_t gemm_act_fwd(const GemmOperands<T>& op, int flags, const EpiActFwd<T>& epi,
                        hipStream_t s) {
  return dispatch(op, flags, ActFwdOp<T>{epi}, s);
}
template <typename T>
hipError_t gemm_act_bwd(const GemmOperands<T>& op, int flags, const EpiActBwd<T>& epi,
                        hipStream_t s) {
  return dispatch(op, flags, ActBwdOp<T>{epi}, s);
}
template <typename T>
hipError_t gemm_param(const GemmOperands<T>& op, int flags, const ParamArgs<T>& P,
                      hipStream_t s) {
  return dispatch(op, flags, ParamOp<T>{P}, s);
}

template hipError_t gemm_act_fwd<bf16_t>(const GemmOperands<bf16_t>&, int, const EpiActFwd<bf16_t>&, hipStream_t);
template hipError_t gemm_act_fwd<float>(const GemmOperands<float>&, int, const EpiActFwd<float>&, hipStream_t);
template hipError_t gemm_act_bwd<bf16_t>(const GemmOperands<bf16_t>&, int, const EpiActBwd<bf16_t>&, hipStream_t);
template hipError_t gemm_act_bwd<float>(const GemmOperands<float>&, int, const EpiActBwd<float>&, hipStream_t);
template hipError_t gemm_param<bf16_t>(const GemmOperands<bf16_t>&, int, const ParamArgs<bf16_t>&, hipStream_t);
template hipError_t gemm_param<float>(const GemmOperands<float>&, int, const ParamArgs<float>&, hipStream_t);

}  // namespace mfmg
