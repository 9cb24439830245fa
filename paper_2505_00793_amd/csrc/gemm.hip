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
// v_mfma_f32_16x16x4_f32 (float32 operands), 64-lane wavefronts, four
// computing waves per workgroup in a 2 x 2 arrangement.  Two main loops:
//   gemm_nt_ws  bf16 operands with k, leading dimensions and strides multiples
//               of 8: a 2- to 4-stage LDS ring of 64-deep k steps filled by
//               buffer_load ... lds from four loader waves while four waves
//               multiply (512 threads);
//   gemm_nt     everything else (float32, ragged k): register-staged,
//               double-buffered LDS, 256 threads.
// Both end in the same staged epilogue.  Backward-weight products with few
// output tiles and a long k can run split-K (batched partial products into a
// caller workspace, then an ordered sum with the epilogue).
#include <type_traits>

#include "kernels.h"
#include "param_epi.h"

namespace mfmg {

namespace {


// 16 bytes of LDS read with an explicit ds_read_b128.  The compiler makes every
// LDS read it emits in a wave with global-to-LDS loads in flight wait for all of
// them (it cannot tell which LDS bytes they write); this one does not, so the
// caller must know that the bytes it reads have landed, and must wait with
// lds_read_wait() before using the value.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x4 lds_read16(const void* p) {
  const unsigned a = (unsigned)reinterpret_cast<uintptr_t>(p);   // LDS offset: low 32 bits
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a) : "memory");
  return v;
}
__device__ __forceinline__ void lds_read_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Sum of 8 bfloat16 values (packed in 4 dwords) in float32, pairwise in a fixed order.
__device__ __forceinline__ float sum8(const u32x4& u) {
  float x[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(u[i] << 16);
    x[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
  }
  return ((x[0] + x[1]) + (x[2] + x[3])) + ((x[4] + x[5]) + (x[6] + x[7]));
}

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

// 16 bytes of row gr starting at column gk of an operand with M >= 1 rows of
// K >= 1 elements.  Every lane loads, from indices clamped into the operand:
// with KVEC (K a multiple of the chunk width, so that a chunk lies wholly
// inside or outside K) one 16-byte load, else single elements; the parts
// outside [0,M) x [0,K) are zeroed by mask_chunk when the chunk is stored.
// With no branch around a load the compiler never waits for all loads in
// flight to merge the registers of two paths, and with the form a template
// parameter it cannot fold the 16-byte load into the element loads.
template <typename T, bool KVEC>
__device__ __forceinline__ uint4 load_chunk(const T* __restrict__ src, int gr, int gk, int M,
                                            int K, int ld) {
  constexpr int VE = Elem<T>::VE;
  const long row = (long)min(gr, M - 1) * ld;
  if constexpr (KVEC) return *reinterpret_cast<const uint4*>(src + row + min(gk, K - VE));
  union {
    uint4 v;
    T e[VE];
  } u;
#pragma unroll
  for (int e = 0; e < VE; ++e) u.e[e] = src[row + min(gk + e, K - 1)];
  return u.v;
}
template <typename T, bool KVEC>
__device__ __forceinline__ uint4 mask_chunk(const uint4& v, int gr, int gk, int M, int K) {
  constexpr int VE = Elem<T>::VE;
  if constexpr (KVEC) return gr < M && gk < K ? v : make_uint4(0, 0, 0, 0);
  union {
    uint4 v;
    T e[VE];
  } u;
  u.v = v;
  const T z = T(0);
#pragma unroll
  for (int e = 0; e < VE; ++e) u.e[e] = gr < M && gk + e < K ? u.e[e] : z;
  return u.v;
}
// Sum of a chunk's elements, in order.
template <typename T>
__device__ __forceinline__ float chunk_sum(const uint4& v) {
  constexpr int VE = Elem<T>::VE;
  union {
    uint4 v;
    T e[VE];
  } u;
  u.v = v;
  float s = 0.0f;
#pragma unroll
  for (int e = 0; e < VE; ++e) s += Elem<T>::to_float(u.e[e]);
  return s;
}

// ------------------------------------------------------------------------------------
// Epilogues.  row(m, n, cnt, c1, c2, t1, t2): cnt (1..4) consecutive columns
// n.. of row m; writes the row-major outputs and returns in t1/t2 the values
// of the outputs also stored transposed.  trans(k, n, m, cnt, v): stores cnt
// consecutive rows m.. of column n into transposed output k.
// ------------------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void store_row4(T* p, long off, int cnt, const float* v) {
  if (cnt == 4 && (off & 3) == 0) {
    store4(p + off, v[0], v[1], v[2], v[3]);
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (k < cnt) p[off + k] = Elem<T>::from_float(v[k]);
  }
}

template <typename T>
struct ActFwdOp {
  EpiActFwd<T> e;
  int M, N;
  static constexpr bool PRELOAD = false;
  typedef int In;
  __device__ int n_trans() const { return e.last ? 0 : (e.dual ? 2 : 1); }
  __device__ __forceinline__ void row(int bz, int m, int n, int cnt, const float* c1,
                                      const float* c2, float* t1, float* t2) const {
    const bool vec = cnt == 4 && (e.N & 3) == 0;
    float b[4] = {0.f, 0.f, 0.f, 0.f}, bd[4] = {0.f, 0.f, 0.f, 0.f};
    if (e.bias) ld4(e.bias, n, cnt, cnt == 4, b);
    if (e.dual && e.bias_d) ld4(e.bias_d, n, cnt, cnt == 4, bd);
    float z[4], zd[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      z[k] = c1[k] + b[k];
      zd[k] = c2[k] + bd[k];
    }
    if (e.Z) st4(e.Z, (long)m * e.N + n, cnt, vec, z);
    if (e.dual && e.Zd) st4(e.Zd, (long)m * e.N + n, cnt, vec, zd);
    if (e.last) return;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      t1[k] = act_f(e.act, z[k]);
      if (e.dual) {
        float d1, d2;
        act_d12(e.act, z[k], d1, d2);
        t2[k] = d1 * zd[k];
      }
    }
    store_row4(e.Ao, (long)m * e.ldA + n, cnt, t1);
    if (e.dual) store_row4(e.Ado, (long)m * e.ldA + n, cnt, t2);
  }
  __device__ __forceinline__ void trans(int k, int bz, int n, int m, int cnt,
                                        const float* v) const {
    store_row4(k == 0 ? e.AoT : e.AdoT, (long)n * e.ldAT + m, cnt, v);
  }
};

template <typename T>
struct ActBwdOp {
  EpiActBwd<T> e;
  int M, N;
  // the walk of an interior tile loads every row's z (zd) before the first row's stores
  static constexpr bool PRELOAD = true;
  struct In {
    float z[4], zd[4];
  };
  __device__ int n_trans() const { return e.dual ? 2 : 1; }
  __device__ bool aligned() const { return (e.N & 3) == 0; }
  // 4 consecutive activations a[m][n..n+3] (n a multiple of 4) as floats
  __device__ __forceinline__ void ld_act4(long idx, float* out) const {
    if constexpr (sizeof(T) == 2) {
      const uint2 v = *reinterpret_cast<const uint2*>(e.Ap + idx);
      out[0] = bf2f((bf16_t)(v.x & 0xffffu)); out[1] = bf2f((bf16_t)(v.x >> 16));
      out[2] = bf2f((bf16_t)(v.y & 0xffffu)); out[3] = bf2f((bf16_t)(v.y >> 16));
    } else {
      ld4v(reinterpret_cast<const float*>(e.Ap), idx, out);
    }
  }
  template <int NIT>
  __device__ __forceinline__ void load_rows(int bz, int m, int dm, int n, In (&in)[NIT]) const {
    if (!e.Zp) {   // ReLU: the sign of the activation
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        ld_act4((long)(m + it * dm) * e.ldAp + n, in[it].z);
        in[it].zd[0] = in[it].zd[1] = in[it].zd[2] = in[it].zd[3] = 0.f;
      }
      return;
    }
#pragma unroll
    for (int it = 0; it < NIT; ++it) ld4v(e.Zp, (long)(m + it * dm) * e.N + n, in[it].z);
    if (e.dual) {
#pragma unroll
      for (int it = 0; it < NIT; ++it) ld4v(e.Zdp, (long)(m + it * dm) * e.N + n, in[it].zd);
    }
  }
  // Any tile: indices clamped into the M x N output (the values past its edges
  // are loaded but never used); 16-byte loads when N is a multiple of 4.
  template <int NIT>
  __device__ __forceinline__ void load_rows_clamped(int bz, int m, int dm, int n,
                                                    In (&in)[NIT]) const {
    if (aligned() && (N & 3) == 0) {
      const int nc = min(n, N - 4);
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const long r = min(m + it * dm, M - 1);
        if (!e.Zp) {
          ld_act4(r * e.ldAp + nc, in[it].z);
          in[it].zd[0] = in[it].zd[1] = in[it].zd[2] = in[it].zd[3] = 0.f;
        } else {
          ld4v(e.Zp, r * e.N + nc, in[it].z);
          if (e.dual) ld4v(e.Zdp, r * e.N + nc, in[it].zd);
          else in[it].zd[0] = in[it].zd[1] = in[it].zd[2] = in[it].zd[3] = 0.f;
        }
      }
      return;
    }
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const long r = min(m + it * dm, M - 1);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int nk = min(n + k, N - 1);
        if (!e.Zp) {   // ReLU: the sign of the activation
          in[it].z[k] = Elem<T>::to_float(e.Ap[r * e.ldAp + nk]);
          in[it].zd[k] = 0.f;
        } else {
          in[it].z[k] = e.Zp[r * e.N + nk];
          in[it].zd[k] = e.dual ? e.Zdp[r * e.N + nk] : 0.f;
        }
      }
    }
  }
  __device__ __forceinline__ void row_in(int bz, int m, int n, int cnt, const In& in,
                                         const float* c1, const float* c2, float* t1,
                                         float* t2) const {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float d1, d2;
      act_d12(e.act, in.z[k], d1, d2);
      t1[k] = c1[k] * d1;
      t2[k] = e.dual ? c2[k] * d1 + c1[k] * d2 * in.zd[k] : 0.0f;
    }
    store_row4(e.dZ, (long)m * e.ld + n, cnt, t1);
    if (e.dual) store_row4(e.dZd, (long)m * e.ld + n, cnt, t2);
  }
  __device__ __forceinline__ void row(int bz, int m, int n, int cnt, const float* c1,
                                      const float* c2, float* t1, float* t2) const {
    const bool vec = cnt == 4 && (e.N & 3) == 0;
    In in;
    in.zd[0] = in.zd[1] = in.zd[2] = in.zd[3] = 0.f;
    if (e.Zp) {
      ld4(e.Zp, (long)m * e.N + n, cnt, vec, in.z);
      if (e.dual) ld4(e.Zdp, (long)m * e.N + n, cnt, vec, in.zd);
    } else {   // ReLU: the sign of the activation
#pragma unroll
      for (int k = 0; k < 4; ++k)
        in.z[k] = k < cnt ? Elem<T>::to_float(e.Ap[(long)m * e.ldAp + n + k]) : 0.f;
    }
    row_in(bz, m, n, cnt, in, c1, c2, t1, t2);
  }
  __device__ __forceinline__ void trans(int k, int bz, int n, int m, int cnt,
                                        const float* v) const {
    store_row4(k == 0 ? e.dZT : e.dZdT, (long)n * e.ldT + m, cnt, v);
  }
};

template <typename T>
struct ParamOp {
  ParamArgs<T> P;
  int M, N;
  // the walk loads every row's inputs before the first row's arithmetic
  static constexpr bool PRELOAD = true;
  typedef ParamIn In;
  __device__ int n_trans() const { return P.outWT ? 1 : 0; }
  __device__ bool aligned() const { return (P.nout & 3) == 0 && (P.w_off & 3) == 0; }
  template <int NIT>
  __device__ __forceinline__ void load_rows(int bz, int m, int dm, int n, ParamIn (&in)[NIT]) const {
    const float* src[3];
    param_sources(P, src);
#pragma unroll
    for (int s = 0; s < 3; ++s)
      if (src[s]) {
#pragma unroll
        for (int it = 0; it < NIT; ++it)
          ld4v(src[s], P.w_off + (long)(m + it * dm) * P.nout + n, in[it].x[s]);
      }
  }
  template <int NIT>
  __device__ __forceinline__ void load_rows_clamped(int bz, int m, int dm, int n,
                                                    ParamIn (&in)[NIT]) const {
    const float* src[3];
    param_sources(P, src);
    const bool al = aligned() && (N & 3) == 0;
    const int nc = min(n, N - 4);
#pragma unroll
    for (int s = 0; s < 3; ++s)
      if (src[s]) {
#pragma unroll
        for (int it = 0; it < NIT; ++it) {
          const long r = P.w_off + (long)min(m + it * dm, M - 1) * P.nout;
          if (al) {
            ld4v(src[s], r + nc, in[it].x[s]);
          } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) in[it].x[s][k] = src[s][r + min(n + k, N - 1)];
          }
        }
      }
  }
  __device__ __forceinline__ void load(int bz, int m, int n, int cnt, ParamIn& in) const {
    param_load(P, P.w_off + (long)m * P.nout + n, cnt, in);
  }
  __device__ __forceinline__ void row_in(int bz, int m, int n, int cnt, const ParamIn& in,
                                         const float* c1, const float* c2, float* t1,
                                         float* t2) const {
    param_finish(P, P.w_off + (long)m * P.nout + n, cnt, in, c1, c2, t1);
    if (P.outW) store_row4(P.outW, (long)m * P.ldW + n, cnt, t1);
  }
  __device__ __forceinline__ void row(int bz, int m, int n, int cnt, const float* c1,
                                      const float* c2, float* t1, float* t2) const {
    ParamIn in;
    load(bz, m, n, cnt, in);
    row_in(bz, m, n, cnt, in, c1, c2, t1, t2);
  }
  __device__ __forceinline__ void trans(int k, int bz, int n, int m, int cnt,
                                        const float* v) const {
    store_row4(P.outWT, (long)n * P.ldWT + m, cnt, v);
  }
  __device__ bool fuse_bias() const { return P.fuse_bias != 0 && P.b_off >= 0; }
  // bias entry n: its inputs (loaded ahead), then the update from its gradient g
  // (and H v entry hv)
  __device__ __forceinline__ void bias_load(int n, ParamIn& in) const {
    param_load(P, P.b_off + n, 1, in);
  }
  __device__ __forceinline__ void bias_finish(int n, const ParamIn& in, float g, float hv) const {
    float g4[4] = {g, 0.f, 0.f, 0.f}, h4[4] = {hv, 0.f, 0.f, 0.f}, cv[4];
    param_finish(P, P.b_off + n, 1, in, g4, h4, cv);
    if (P.outb) P.outb[n] = cv[0];
  }
};

template <class E> struct IsParamOp : std::false_type {};
template <typename T> struct IsParamOp<ParamOp<T>> : std::true_type {};
template <class E> struct IsActFwdOp : std::false_type {};
template <typename T> struct IsActFwdOp<ActFwdOp<T>> : std::true_type {};

struct StoreOp {
  EpiStore e;
  int M, N;
  static constexpr bool PRELOAD = false;
  typedef int In;
  __device__ int n_trans() const { return 0; }
  __device__ __forceinline__ void row(int bz, int m, int n, int cnt, const float* c1,
                                      const float* c2, float* t1, float* t2) const {
    const long off = bz * e.sC + (long)m * e.ldc + n;
    const bool vec = cnt == 4 && (off & 3) == 0;
    float v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = e.scale * c1[k];
    st4(e.C, off, cnt, vec, v);
    if (e.dual) {
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] = e.scale * c2[k];
      st4(e.Cd, off, cnt, vec, v);
    }
  }
  __device__ __forceinline__ void trans(int, int, int, int, int, const float*) const {}
};

struct ResidOp {
  EpiResid e;
  int M, N;
  static constexpr bool PRELOAD = false;
  typedef int In;
  __device__ int n_trans() const { return 0; }
  __device__ __forceinline__ void row(int bz, int m, int n, int cnt, const float* c1,
                                      const float* c2, float* t1, float* t2) const {
    const long off = (long)m * e.N + n;
    const bool vec = cnt == 4 && (e.N & 3) == 0;
    float h[4];
    ld4(e.H, off, cnt, vec, h);
#pragma unroll
    for (int k = 0; k < 4; ++k) h[k] += c1[k];
    st4(e.Ho, off, cnt, vec, h);
    if (e.dual) {
      ld4(e.Hd, off, cnt, vec, h);
#pragma unroll
      for (int k = 0; k < 4; ++k) h[k] += c2[k];
      st4(e.Hdo, off, cnt, vec, h);
    }
  }
  __device__ __forceinline__ void trans(int, int, int, int, int, const float*) const {}
};

template <typename T>
struct HeadMergeOp {
  EpiHeadMerge<T> e;
  int M, N;
  static constexpr bool PRELOAD = false;
  typedef int In;
  __device__ int n_trans() const { return e.dual ? 2 : 1; }
  __device__ __forceinline__ void row(int bz, int m, int n, int cnt, const float* c1,
                                      const float* c2, float* t1, float* t2) const {
    const long r = (long)(bz / e.heads) * e.seq + m;
    const int c = (bz % e.heads) * e.dh + n;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      t1[k] = c1[k];
      t2[k] = c2[k];
    }
    store_row4(e.O, r * e.ldO + c, cnt, t1);
    if (e.dual) store_row4(e.Od, r * e.ldO + c, cnt, t2);
  }
  __device__ __forceinline__ void trans(int k, int bz, int n, int m, int cnt,
                                        const float* v) const {
    const long r = (long)(bz / e.heads) * e.seq + m;
    const long c = (bz % e.heads) * e.dh + n;
    store_row4(k == 0 ? e.OT : e.OdT, c * e.ldOT + r, cnt, v);
  }
};

template <typename T>
struct HeadSplitOp {
  EpiHeadSplit<T> e;
  int M, N;
  static constexpr bool PRELOAD = false;
  typedef int In;
  __device__ int n_trans() const { return e.dual ? 2 : 1; }
  __device__ __forceinline__ void row(int bz, int m, int n, int cnt, const float* c1,
                                      const float* c2, float* t1, float* t2) const {
    const int b = m / e.seq, s = m % e.seq;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      t1[k] = c1[k];
      t2[k] = c2[k];
    }
    // cnt columns n.. lie in one head (dh is a multiple of 4)
    const int h = n / e.dh, j = n % e.dh;
    const long off = ((long)(b * e.heads + h) * e.seq + s) * e.ldh + j;
    store_row4(e.Oh, off, cnt, t1);
    if (e.dual) store_row4(e.Odh, off, cnt, t2);
  }
  __device__ __forceinline__ void trans(int k, int bz, int n, int m, int cnt,
                                        const float* v) const {
    // cnt rows m.. lie in one sequence (seq is a multiple of 4)
    const int b = m / e.seq, s = m % e.seq;
    const int h = n / e.dh, j = n % e.dh;
    const long off = ((long)(b * e.heads + h) * e.dh + j) * e.ldhT + s;
    store_row4(k == 0 ? e.OhT : e.OdhT, off, cnt, v);
  }
};

// Staged epilogue geometry: the accumulator tile goes to LDS one wave-row
// (BM/2 rows) at a time, then all 256 threads walk it in row-major order with
// 16-byte global accesses, and (for outputs that are also needed in the
// transposed layout) a second walk writes contiguous runs of the transpose.
template <int BN>
struct Stage {
  static constexpr int SLD = BN + 4;  // padded LDS row stride, floats
};

// NPASS: the tile is staged in NPASS slabs of BM / NPASS rows.
template <int FLAGS, int BM, int BN, int NPASS>
struct EpiSmem {
  static constexpr int NS = (FLAGS & (G_AD | G_BD)) ? 2 : 1;  // staged accumulators
  static constexpr int BYTES = NS * (BM / NPASS) * Stage<BN>::SLD * 4;
};

// LDS of the register-staged main loop: double-buffered tiles, rows padded by
// one 16-byte chunk.
template <typename T, int FLAGS, int BM, int BN, int BK>
struct Smem {
  static constexpr int VE = Elem<T>::VE;
  static constexpr int LDL = BK + VE;
  static constexpr int NAS = (FLAGS & G_AD) ? 2 : 1;
  static constexpr int NBS = (FLAGS & G_BD) ? 2 : 1;
  static constexpr int STAGE = (NAS * BM + NBS * BN) * LDL;  // elements
  static constexpr int PIPE_BYTES = 2 * STAGE * (int)sizeof(T);
  static constexpr int EPI_BYTES = EpiSmem<FLAGS, BM, BN, BM == 64 ? 1 : 2>::BYTES;
  static constexpr int BYTES = PIPE_BYTES > EPI_BYTES ? PIPE_BYTES : EPI_BYTES;
};

// Tile order.  Workgroup ids are dispatched round-robin over the 8 XCDs; give
// each XCD a contiguous range of tiles, then walk tiles in groups of 8 tile
// rows so that neighbouring tiles share A and B panels in that XCD's L2.
template <int BM, int BN>
__device__ __forceinline__ void tile_origin(int M, int N, int& m0, int& n0, int pid) {
  const int tiles_m = (M + BM - 1) / BM;
  const int tiles_n = (N + BN - 1) / BN;
  const int nt = tiles_m * tiles_n;
  if ((nt & 7) == 0) pid = (pid & 7) * (nt >> 3) + (pid >> 3);
  constexpr int GM = 8;
  const int group = pid / (GM * tiles_n);
  const int first_m = group * GM;
  const int gsz = min(tiles_m - first_m, GM);
  const int within = pid - group * GM * tiles_n;
  m0 = (first_m + within % gsz) * BM;
  n0 = (within / gsz) * BN;
}
template <int BM, int BN>
__device__ __forceinline__ void tile_origin(int M, int N, int& m0, int& n0) {
  tile_origin<BM, BN>(M, N, m0, n0, (int)blockIdx.x);
}

// Position of element (row, col) in the epilogue staging buffer: rows padded
// to SLD floats, and 4-float column groups XOR-swizzled by row bits 4..5 so
// that the transposed walk (16 lanes reading one column at rows 4 t + k) hits
// 16 different banks; 4-float groups stay contiguous for the row walk.
template <int SLD>
__device__ __forceinline__ int stage_idx(int row, int col) {
  return row * SLD + (col ^ (((row >> 4) & 3) << 2));
}

// Accumulators of the four computing waves (WN = 2: a 2 x 2 arrangement; WN = 1:
// four waves stacked along m, for 16-column tiles; each TM x TN tiles of 16 x 16)
// -> LDS staging buffer, the wave's rows from rbase.  C layout of a 16x16 MFMA
// tile: lane holds rows 4*(lane/16) + 0..3 of column lane%16.  Called by the
// waves whose rows fall in the slab.
template <int FLAGS, int BM, int BN, int RP, int WN = 2>
__device__ __forceinline__ void stage_tile(const f32x4 (&acc1)[BM * WN / 64][BN / (16 * WN)],
                                           const f32x4 (&acc2)[BM * WN / 64][BN / (16 * WN)],
                                           float* S1, float* S2, int rbase) {
  constexpr bool HC1 = (FLAGS & G_C1) != 0;
  constexpr bool HC2 = (FLAGS & (G_AD | G_BD)) != 0;
  constexpr int WTN = BN / WN;
  constexpr int TM = BM * WN / 64, TN = BN / (16 * WN);
  constexpr int SLD = Stage<BN>::SLD;
  const int lane = threadIdx.x & 63;
  const int wn = (threadIdx.x >> 6) % WN;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int c = wn * WTN + j * 16 + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int rl = rbase + i * 16 + (lane >> 4) * 4 + r;
        S1[stage_idx<SLD>(rl, c)] = HC1 ? acc1[i][j][r] : 0.0f;
        if constexpr (HC2) S2[stage_idx<SLD>(rl, c)] = acc2[i][j][r];
      }
    }
}

// Epilogue walk over a staged slab of RP rows (tile rows mr0 .. mr0 + RP - 1) by
// all NT threads: a row-major walk with 16-byte accesses calls epi.row, then
// (for outputs also needed transposed) a walk down the columns writes
// contiguous runs of the transpose.  Ends with the LDS free again.
template <int FLAGS, int BN, int RP, int NT, class Epi>
__device__ __forceinline__ void walk_tile(float* S1, float* S2, int mr0, int n0, int bz,
                                          const Epi& epi) {
  constexpr bool HC2 = (FLAGS & (G_AD | G_BD)) != 0;
  constexpr int SLD = Stage<BN>::SLD;
  const int tid = threadIdx.x;
  const int nT = epi.n_trans();
  bool walked = false;
  if constexpr (Epi::PRELOAD && NT == 512) {
    // Interior tile, aligned rows: every row's global inputs are requested with
    // unconditional 16-byte loads before the first row's arithmetic, so a
    // thread keeps all of them in flight at once.
    if (mr0 + RP <= epi.M && n0 + BN <= epi.N && epi.aligned()) {
      constexpr int TPR = BN / 4;
      constexpr int RPI = NT / TPR;
      constexpr int NIT = RP / RPI;
      static_assert(RP % RPI == 0, "rows per thread");
      const int c = (tid % TPR) * 4;
      const int n = n0 + c;
      typename Epi::In in[NIT];
      epi.template load_rows<NIT>(bz, mr0 + tid / TPR, RPI, n, in);
#pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const int rr = tid / TPR + it * RPI;
        float c1[4], c2[4], t1[4], t2[4];
        const int si = stage_idx<SLD>(rr, c);
        const float4 x1 = *reinterpret_cast<const float4*>(S1 + si);
        c1[0] = x1.x; c1[1] = x1.y; c1[2] = x1.z; c1[3] = x1.w;
        if constexpr (HC2) {
          const float4 x2 = *reinterpret_cast<const float4*>(S2 + si);
          c2[0] = x2.x; c2[1] = x2.y; c2[2] = x2.z; c2[3] = x2.w;
        } else {
          c2[0] = c2[1] = c2[2] = c2[3] = 0.0f;
        }
        epi.row_in(bz, mr0 + rr, n, 4, in[it], c1, c2, t1, t2);
        if (nT > 0) *reinterpret_cast<float4*>(S1 + si) = make_float4(t1[0], t1[1], t1[2], t1[3]);
        if (nT > 1) *reinterpret_cast<float4*>(S2 + si) = make_float4(t2[0], t2[1], t2[2], t2[3]);
      }
      walked = true;
    }
  }
  if constexpr (Epi::PRELOAD && NT == 256) {
    // Any tile: every row's inputs first (single elements from clamped indices,
    // no branch around a load), then the rows inside the output.
    constexpr int TPR = BN / 4;
    constexpr int RPI = NT / TPR;
    constexpr int NIT = RP / RPI;
    static_assert(RP % RPI == 0, "rows per thread");
    const int c = (tid % TPR) * 4;
    const int n = n0 + c;
    typename Epi::In in[NIT];
    epi.template load_rows_clamped<NIT>(bz, mr0 + tid / TPR, RPI, n, in);
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int rr = tid / TPR + it * RPI;
      const int m = mr0 + rr;
      if (m < epi.M && n < epi.N) {
        float c1[4], c2[4], t1[4], t2[4];
        const int si = stage_idx<SLD>(rr, c);
        const float4 x1 = *reinterpret_cast<const float4*>(S1 + si);
        c1[0] = x1.x; c1[1] = x1.y; c1[2] = x1.z; c1[3] = x1.w;
        if constexpr (HC2) {
          const float4 x2 = *reinterpret_cast<const float4*>(S2 + si);
          c2[0] = x2.x; c2[1] = x2.y; c2[2] = x2.z; c2[3] = x2.w;
        } else {
          c2[0] = c2[1] = c2[2] = c2[3] = 0.0f;
        }
        epi.row_in(bz, m, n, min(4, epi.N - n), in[it], c1, c2, t1, t2);
        if (nT > 0) *reinterpret_cast<float4*>(S1 + si) = make_float4(t1[0], t1[1], t1[2], t1[3]);
        if (nT > 1) *reinterpret_cast<float4*>(S2 + si) = make_float4(t2[0], t2[1], t2[2], t2[3]);
      }
    }
    walked = true;
  }
  if (!walked) {
    constexpr int TPR = BN / 4;        // threads per row, 4 columns each
    constexpr int RPI = NT / TPR;      // rows per iteration
    const int c = (tid % TPR) * 4;
    const int n = n0 + c;
    for (int rr = tid / TPR; rr < RP; rr += RPI) {
      const int m = mr0 + rr;
      if (m < epi.M && n < epi.N) {
        float c1[4], c2[4], t1[4], t2[4];
        const int si = stage_idx<SLD>(rr, c);
        const float4 x1 = *reinterpret_cast<const float4*>(S1 + si);
        c1[0] = x1.x; c1[1] = x1.y; c1[2] = x1.z; c1[3] = x1.w;
        if constexpr (HC2) {
          const float4 x2 = *reinterpret_cast<const float4*>(S2 + si);
          c2[0] = x2.x; c2[1] = x2.y; c2[2] = x2.z; c2[3] = x2.w;
        } else {
          c2[0] = c2[1] = c2[2] = c2[3] = 0.0f;
        }
        epi.row(bz, m, n, min(4, epi.N - n), c1, c2, t1, t2);
        if (nT > 0) *reinterpret_cast<float4*>(S1 + si) = make_float4(t1[0], t1[1], t1[2], t1[3]);
        if (nT > 1) *reinterpret_cast<float4*>(S2 + si) = make_float4(t2[0], t2[1], t2[2], t2[3]);
      }
    }
  }
  if (nT > 0) {
    __syncthreads();
    constexpr int TPC = RP / 4;        // threads per transposed row, 4 rows of C each
    constexpr int CPI = NT / TPC;
    const int r4 = (tid % TPC) * 4;
    const int m = mr0 + r4;
    for (int cc = tid / TPC; cc < BN; cc += CPI) {
      const int n = n0 + cc;
      if (n < epi.N && m < epi.M) {
        const int cnt = min(4, epi.M - m);
        float v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = S1[stage_idx<SLD>(r4 + k, cc)];
        epi.trans(0, bz, n, m, cnt, v);
        if (nT > 1) {
#pragma unroll
          for (int k = 0; k < 4; ++k) v[k] = S2[stage_idx<SLD>(r4 + k, cc)];
          epi.trans(1, bz, n, m, cnt, v);
        }
      }
    }
  }
  __syncthreads();
}

// Epilogue of the 256-thread kernels.  A 64-row tile is staged whole (it fits in
// the LDS of the main loop) and walked in one pass, so a thread requests the
// epilogue inputs of all its rows at once; a 128-row tile goes one wave row
// (BM / 2 rows) at a time in half the LDS.  The caller guarantees that no wave
// still reads or writes smem.
template <int FLAGS, int BM, int BN, int WN, class Epi>
__device__ __forceinline__ void run_epilogue(const f32x4 (&acc1)[BM * WN / 64][BN / (16 * WN)],
                                             const f32x4 (&acc2)[BM * WN / 64][BN / (16 * WN)],
                                             char* smem_raw, int m0, int n0, int bz,
                                             const Epi& epi) {
  const int wm = (threadIdx.x >> 6) / WN;
  if constexpr (BM == 64) {
    float* S1 = reinterpret_cast<float*>(smem_raw);
    float* S2 = S1 + BM * Stage<BN>::SLD;
    stage_tile<FLAGS, BM, BN, BM, WN>(acc1, acc2, S1, S2, wm * (BM * WN / 4));
    __syncthreads();
    walk_tile<FLAGS, BN, BM, 256>(S1, S2, m0, n0, bz, epi);
  } else {
    constexpr int RP = BM / 2;
    float* S1 = reinterpret_cast<float*>(smem_raw);
    float* S2 = S1 + RP * Stage<BN>::SLD;
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      if (wm == pass) stage_tile<FLAGS, BM, BN, RP, WN>(acc1, acc2, S1, S2, 0);
      __syncthreads();
      walk_tile<FLAGS, BN, RP, 256>(S1, S2, m0 + pass * RP, n0, bz, epi);
    }
  }
}

// ------------------------------------------------------------------------------------
// Main loop, register-staged: each thread loads its 16-byte chunks of the next
// k step into registers while the current one is multiplied, then stores them
// to the other LDS buffer.  Handles any K, leading dimension and element type.
// ------------------------------------------------------------------------------------
// KVEC: K is a multiple of the 16-byte chunk width (see load_chunk).
template <typename T, int FLAGS, int BM, int BN, int BK, class Epi, bool KVEC>
__global__ void __launch_bounds__(256) gemm_nt(GemmOperands<T> op, Epi epi) {
  typedef Smem<T, FLAGS, BM, BN, BK> SM;
  constexpr int VE = Elem<T>::VE;
  constexpr int LDL = SM::LDL;
  constexpr bool HC1 = (FLAGS & G_C1) != 0;
  constexpr bool HAD = (FLAGS & G_AD) != 0;
  constexpr bool HBD = (FLAGS & G_BD) != 0;
  constexpr int NAS = SM::NAS;
  constexpr int NBS = SM::NBS;
  constexpr int STAGE = SM::STAGE;
  // 2 x 2 waves over the tile, or 4 x 1 (stacked along m) for 16-column tiles
  constexpr int WN = BN >= 32 ? 2 : 1, WM = 4 / WN;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 16, TN = WTN / 16;
  constexpr int CPR = BK / VE;           // 16-byte chunks per tile row
  constexpr int ACH = BM * CPR / 256;    // chunks per thread, A-side tile
  constexpr int BCH = BN * CPR / 256;    // chunks per thread, B-side tile
  constexpr int NCH = BK / (4 * VE);     // 16-byte fragment reads per k step
  static_assert(ACH >= 1 && BCH >= 1 && (BM * CPR) % 256 == 0 && (BN * CPR) % 256 == 0, "tile");
  typedef typename Frag<T>::type frag_t;

  __shared__ __attribute__((aligned(16))) char smem_raw[SM::BYTES];
  T* smem = reinterpret_cast<T*>(smem_raw);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  int m0, n0;
  tile_origin<BM, BN>(op.M, op.N, m0, n0);
  const int bz = blockIdx.y;
  if (bz > 0) {
    op.A += bz * op.sA;
    if (op.Ad) op.Ad += bz * op.sA;
    op.B += bz * op.sB;
    if (op.Bd) op.Bd += bz * op.sB;
  }

  uint4 ra[NAS][ACH], rb[NBS][BCH];

  // Parameter epilogues with fused bias: as in the direct-to-LDS kernel, the
  // tiles of a tile column share out its BN bias entries; each B (and Bd) chunk
  // of a row in this tile's share is added up as it is stored to LDS, in k
  // order, and the CPR threads of a row then combine their sums in lane order.
  constexpr bool BIAS = IsParamOp<Epi>::value;
  int br0 = 0, bnr = 0;
  float bsum[BCH], bdsum[BCH];
  ParamIn bin[BCH];
  if constexpr (BIAS) {
    if (bz == 0 && epi.fuse_bias()) {
      const int tiles_m = (op.M + BM - 1) / BM;
      const int rpt = (BN + tiles_m - 1) / tiles_m;   // bias rows per tile
      br0 = (m0 / BM) * rpt;
      bnr = max(0, min(BN, br0 + rpt) - br0);
    }
#pragma unroll
    for (int c = 0; c < BCH; ++c) {
      bsum[c] = bdsum[c] = 0.0f;
      const int rr = (tid + c * 256) / CPR;
      if (rr >= br0 && rr < br0 + bnr && tid % CPR == 0 && n0 + rr < op.N)
        epi.bias_load(n0 + rr, bin[c]);
    }
  }

  auto gload = [&](int k0) {
#pragma unroll
    for (int s = 0; s < NAS; ++s) {
      const T* src = s == 0 ? op.A : op.Ad;
#pragma unroll
      for (int c = 0; c < ACH; ++c) {
        int ch = tid + c * 256;
        ra[s][c] = load_chunk<T, KVEC>(src, m0 + ch / CPR, k0 + (ch % CPR) * VE, op.M, op.K,
                                       op.lda);
      }
    }
#pragma unroll
    for (int s = 0; s < NBS; ++s) {
      const T* src = s == 0 ? op.B : op.Bd;
#pragma unroll
      for (int c = 0; c < BCH; ++c) {
        int ch = tid + c * 256;
        rb[s][c] = load_chunk<T, KVEC>(src, n0 + ch / CPR, k0 + (ch % CPR) * VE, op.N, op.K,
                                       op.ldb);
      }
    }
  };
  auto sstore = [&](int buf, int k0) {
    T* base = smem + buf * STAGE;
#pragma unroll
    for (int s = 0; s < NAS; ++s)
#pragma unroll
      for (int c = 0; c < ACH; ++c) {
        int ch = tid + c * 256;
        *reinterpret_cast<uint4*>(base + (s * BM + ch / CPR) * LDL + (ch % CPR) * VE) =
            mask_chunk<T, KVEC>(ra[s][c], m0 + ch / CPR, k0 + (ch % CPR) * VE, op.M, op.K);
      }
#pragma unroll
    for (int s = 0; s < NBS; ++s)
#pragma unroll
      for (int c = 0; c < BCH; ++c) {
        int ch = tid + c * 256;
        const uint4 v =
            mask_chunk<T, KVEC>(rb[s][c], n0 + ch / CPR, k0 + (ch % CPR) * VE, op.N, op.K);
        *reinterpret_cast<uint4*>(base + (NAS * BM + s * BN + ch / CPR) * LDL + (ch % CPR) * VE) =
            v;
        if constexpr (BIAS) {
          if (bnr > 0) {
            if (s == 0) bsum[c] += chunk_sum<T>(v);
            else bdsum[c] += chunk_sum<T>(v);
          }
        }
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
  if (op.K > 0) gload(0);   // with K = 0 every chunk is masked to zero
  sstore(0, 0);
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
    if (kt + 1 < nk) sstore(buf ^ 1, (kt + 1) * BK);
    __syncthreads();
  }
  if constexpr (BIAS) {
    if (bnr > 0) {   // uniform: every lane of the block takes part in the shuffles
#pragma unroll
      for (int c = 0; c < BCH; ++c) {
        for (int o = 1; o < CPR; o <<= 1) {
          bsum[c] += __shfl_xor(bsum[c], o, 64);
          bdsum[c] += __shfl_xor(bdsum[c], o, 64);
        }
        const int rr = (tid + c * 256) / CPR;
        if (rr >= br0 && rr < br0 + bnr && tid % CPR == 0 && n0 + rr < op.N)
          epi.bias_finish(n0 + rr, bin[c], bsum[c], bdsum[c]);
      }
    }
  }
  run_epilogue<FLAGS, BM, BN, WN>(acc1, acc2, smem_raw, m0, n0, bz, epi);
}

// ------------------------------------------------------------------------------------
// Direct-to-LDS tile loads (bfloat16).  Tiles go from HBM to LDS with
// buffer_load_dwordx4 ... lds, which needs no registers, so NST k steps are in
// flight at once (NST - 1 loading while one is multiplied).  Each load
// instruction fills 1 KB of LDS, lane l at byte 16 l; a lane picks which
// 16-byte chunk of which row it fetches so that the tile lands row-major with
// the chunk index XOR-swizzled by the row (conflict-free fragment reads, no
// padding).  Rows past M or N and chunks past K read zero: the buffer
// descriptor's range check turns an offset at or above num_records into a zero
// load, and such lanes are given the offset 2^31.  Requires K, the leading
// dimensions and the batch strides to be multiples of 8 elements, 16-byte
// aligned operands, and each operand to span less than 2^31 bytes.
// ------------------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;

// Chunk swizzle by row.  For the fragment reads below (16 consecutive rows, one
// logical chunk per 16 lanes) both forms were measured free of LDS bank
// conflicts on gfx950 with the SQ_LDS_BANK_CONFLICT counter, while mixing
// row bit 3 into either leaves half of the LDS cycles in conflict.
template <int CPR>
__device__ __forceinline__ int chunk_swizzle(int r) {
  static_assert(CPR == 8 || CPR == 4, "16-byte chunks per row");
  if constexpr (CPR == 8) return r & 7;    // 128-byte rows
  else return (r >> 1) & 3;                // 64-byte rows
}

// s_waitcnt vmcnt(N) lgkmcnt(0), leaving expcnt free (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vm_lgkm() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}
// Workgroup barrier that orders LDS accesses only: the explicit waitcnt before
// it decides which global-to-LDS loads have landed.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int FLAGS, int BM, int BN, int BK, int NST, int NPASS>
struct DmaSmem {
  static constexpr bool LA = (FLAGS & (G_C1 | G_BD)) != 0;  // tiles loaded
  static constexpr bool LAD = (FLAGS & G_AD) != 0;
  static constexpr bool LB = (FLAGS & (G_C1 | G_AD)) != 0;
  static constexpr bool LBD = (FLAGS & G_BD) != 0;
  static constexpr int ROWB = BK * 2;                         // bytes per tile row
  static constexpr int OFF_AD = (LA ? BM : 0) * ROWB;
  static constexpr int OFF_B = OFF_AD + (LAD ? BM : 0) * ROWB;
  static constexpr int OFF_BD = OFF_B + (LB ? BN : 0) * ROWB;
  static constexpr int STAGE_BYTES = OFF_BD + (LBD ? BN : 0) * ROWB;
  static constexpr int NOPS = (LA ? 1 : 0) + (LAD ? 1 : 0) + (LB ? 1 : 0) + (LBD ? 1 : 0);
  static constexpr int CPR = BK / 8;
  static constexpr int LPW = STAGE_BYTES / 1024 / 4;         // load instructions per wave
  static constexpr int PIPE_BYTES = NST * STAGE_BYTES;
  static constexpr int EPI_BYTES = EpiSmem<FLAGS, BM, BN, NPASS>::BYTES;
  static constexpr int BYTES = PIPE_BYTES > EPI_BYTES ? PIPE_BYTES : EPI_BYTES;
};

// Per-lane state for one operand tile: which rows this lane fetches.
template <int ROWS, int CPR>
struct DmaTile {
  static constexpr int RPB = 64 / CPR;         // tile rows per 1 KB load
  static constexpr int BPW = ROWS / RPB / 4;   // loads per wave per k step
  static_assert(BPW >= 1 && ROWS % (4 * RPB) == 0, "tile rows");
  __amdgpu_buffer_rsrc_t rsrc;
  unsigned row_off[BPW];   // byte offset of the lane's row plus its chunk, or 2^31
  int kq;                  // element offset of the lane's chunk within a k step

  // w: index 0..3 of this wave among the four that load the tile
  __device__ __forceinline__ void init(const bf16_t* base, int rows, int ld, int K, int row0,
                                       int w) {
    const unsigned bytes = rows > 0 ? (unsigned)(((long)(rows - 1) * ld + K) * 2) : 0u;
    rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(base), 0, (int)bytes, 0x00020000);
    const int lane = threadIdx.x & 63;
    const int p = lane % CPR;
#pragma unroll
    for (int c = 0; c < BPW; ++c) {
      const int r = (c * 4 + w) * RPB + lane / CPR;
      const int q = p ^ chunk_swizzle<CPR>(r);
      const int gr = row0 + r;
      row_off[c] = gr < rows ? (unsigned)((long)gr * ld + q * 8) * 2u : 0x80000000u;
      kq = q * 8;   // the same for every c: the swizzle reads row bits that c does not change
    }
  }
  // Issue the loads of k step k0 into the tile at dst (LDS).
  __device__ __forceinline__ void issue(char* dst, int k0, int K, int w) const {
    const bool kin = k0 + kq < K;
#pragma unroll
    for (int c = 0; c < BPW; ++c) {
      const unsigned off = (kin && row_off[c] != 0x80000000u) ? row_off[c] + (unsigned)k0 * 2u
                                                             : 0x80000000u;
      char* d = dst + (c * 4 + w) * RPB * (CPR * 16);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t*)d, 16, off, 0, 0, 0);
    }
  }
};

// ------------------------------------------------------------------------------------
// Main loop, warp-specialised (bfloat16, 512 threads).  A wave that issues a
// global load stalls until the compute unit's load unit takes it (about 16
// cycles per 1 KB load, one unit per compute unit), and in-order issue holds
// back its MFMAs meanwhile.  Here waves 4..7 only issue the direct-to-LDS loads
// and waves 0..3 only read fragments and multiply, so each SIMD has one wave
// that keeps its matrix core busy while the other waits on the load unit.  The
// eight waves meet at one barrier per k step and all of them walk the epilogue.
// ------------------------------------------------------------------------------------
template <int FLAGS, int BM, int BN, int BK, int NST, class Epi>
__device__ __forceinline__ void gemm_ws_tile(const GemmOperands<bf16_t>& op, const Epi& epi,
                                             int pid, int bz, char* smem) {
  typedef DmaSmem<FLAGS, BM, BN, BK, NST, 1> SM;
  constexpr bool HC1 = (FLAGS & G_C1) != 0;
  constexpr bool HAD = (FLAGS & G_AD) != 0;
  constexpr bool HBD = (FLAGS & G_BD) != 0;
  constexpr int CPR = SM::CPR;
  constexpr int ROWB = SM::ROWB;
  constexpr int WTM = BM / 2, WTN = BN / 2;
  constexpr int TM = WTM / 16, TN = WTN / 16;
  constexpr int NCH = CPR / 4;
  static_assert(NST >= 2 && SM::LPW * (NST - 2) < 64, "pipeline depth");

  float* S1 = reinterpret_cast<float*>(smem);
  float* S2 = S1 + BM * Stage<BN>::SLD;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int m0, n0;
  tile_origin<BM, BN>(op.M, op.N, m0, n0, pid);
  const int K = op.K;
  const int nk = (K + BK - 1) / BK;

  // The two roles run separate loops, so their registers do not add up; both
  // pass the same barriers: one per k step, one when the LDS turns into the
  // staging buffer and one when the staged tile is complete.
  if (wave >= 4) {
    const int pw = wave - 4;
    DmaTile<BM, CPR> tA, tAd;
    DmaTile<BN, CPR> tB, tBd;
    if constexpr (SM::LA) tA.init(op.A + bz * op.sA, op.M, op.lda, K, m0, pw);
    if constexpr (SM::LAD) tAd.init(op.Ad + bz * op.sA, op.M, op.lda, K, m0, pw);
    if constexpr (SM::LB) tB.init(op.B + bz * op.sB, op.N, op.ldb, K, n0, pw);
    if constexpr (SM::LBD) tBd.init(op.Bd + bz * op.sB, op.N, op.ldb, K, n0, pw);
    auto issue = [&](int kt) {
      char* st = smem + (kt % NST) * SM::STAGE_BYTES;
      const int k0 = kt * BK;
      if constexpr (SM::LA) tA.issue(st, k0, K, pw);
      if constexpr (SM::LAD) tAd.issue(st + SM::OFF_AD, k0, K, pw);
      if constexpr (SM::LB) tB.issue(st + SM::OFF_B, k0, K, pw);
      if constexpr (SM::LBD) tBd.issue(st + SM::OFF_BD, k0, K, pw);
    };
    // Parameter epilogues with fused bias: every tile of a tile column stages
    // the same B rows (dZ^T, and Bd = the tangent) over all of k, so the column's
    // BN bias entries are shared out among its tiles_m tiles.  While the
    // computing waves multiply step kt, loader threads add up this tile's share
    // of the B and Bd rows, btpr threads per row, each over its 16-byte chunks
    // in their order in LDS; the btpr partial sums of a row are then combined in
    // lane order.  The entries' epilogue inputs are loaded before the loop.
    constexpr bool BIAS = IsParamOp<Epi>::value && (SM::LB || SM::LBD);
    const int lt = tid - 256;
    bool bias_w = false;
    int brow = 0, btpr = 1, bcpt = CPR;
    float bsum = 0.0f, bdsum = 0.0f;
    typename Epi::In bin;
    if constexpr (BIAS) {
      if (bz == 0 && epi.fuse_bias()) {
        const int tiles_m = (op.M + BM - 1) / BM;
        const int rpt = (BN + tiles_m - 1) / tiles_m;        // bias rows per tile
        const int r0 = (m0 / BM) * rpt, nr = min(BN, r0 + rpt) - r0;
        if (nr > 0) {
          btpr = CPR;
          while (btpr > 1 && nr * btpr > 256) btpr >>= 1;
          bcpt = CPR / btpr;
          brow = r0 + lt / btpr;
          bias_w = lt < nr * btpr;
          if (bias_w && lt % btpr == 0 && n0 + brow < op.N) epi.bias_load(n0 + brow, bin);
        }
      }
    }
#pragma unroll
    for (int s = 0; s < NST - 1; ++s) issue(s);
    for (int kt = 0; kt < nk; ++kt) {
      wait_vm_lgkm<SM::LPW * (NST - 2)>();   // this wave's loads of step kt have landed
      lds_barrier();                         // ... and every other wave's
      issue(kt + NST - 1);                   // past the last step: zero loads into a dead stage
      if constexpr (BIAS) {
        if (bias_w) {
          // stage kt has landed (the wait and barrier above); the loads in
          // flight write other stages
          const char* st = smem + (kt % NST) * SM::STAGE_BYTES;
          const int c0 = (lt % btpr) * bcpt;
          for (int c = 0; c < bcpt; ++c) {
            const int off = brow * ROWB + (c0 + c) * 16;
            // a product without a B tile (tangent only: an Adam reverse, whose
            // epilogue reads no gradient) sums Bd alone
            u32x4 u = {0u, 0u, 0u, 0u}, ud = {0u, 0u, 0u, 0u};
            if constexpr (SM::LB) u = lds_read16(st + SM::OFF_B + off);
            if constexpr (SM::LBD) ud = lds_read16(st + SM::OFF_BD + off);
            lds_read_wait();
            if constexpr (SM::LB) bsum += sum8(u);
            if constexpr (SM::LBD) bdsum += sum8(ud);
          }
        }
      }
    }
    if constexpr (BIAS) {
      // every lane takes part in the shuffles (idle ones add zeros to each other)
      for (int o = 1; o < btpr; o <<= 1) {
        bsum += __shfl_xor(bsum, o, 64);
        bdsum += __shfl_xor(bdsum, o, 64);
      }
      if (bias_w && lt % btpr == 0 && n0 + brow < op.N) epi.bias_finish(n0 + brow, bin, bsum, bdsum);
    }
    wait_vm_lgkm<0>();
    lds_barrier();
    lds_barrier();
  } else {
    const int wm = wave >> 1, wn = wave & 1;
    f32x4 acc1[TM][TN], acc2[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        acc1[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        acc2[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    // lane reads row (lane % 16) of a 16-row slab, logical chunk lane / 16 + 4 c
    const int sw = chunk_swizzle<CPR>(lane & 15);
    int foff[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) foff[c] = (lane & 15) * ROWB + (((lane >> 4) + 4 * c) ^ sw) * 16;
    for (int kt = 0; kt < nk; ++kt) {
      wait_vm_lgkm<0>();   // reads of step kt - 1 done: its stage may be refilled
      lds_barrier();       // every load of step kt has landed
      const char* st = smem + (kt % NST) * SM::STAGE_BYTES;
      const char* As = st;
      const char* Ads = st + SM::OFF_AD;
      const char* Bs = st + SM::OFF_B;
      const char* Bds = st + SM::OFF_BD;
      // Fragments of NF chunks are read before the first chunk's MFMAs, so the
      // later chunks' LDS reads overlap them: all chunks of the step for two
      // operand tiles, one at a time for the dual products (registers).
      constexpr int NF = SM::NOPS <= 2 ? NCH : 1;
#pragma unroll
      for (int c0 = 0; c0 < NCH; c0 += NF) {
        bf16x8 a[NF][TM], ad[NF][TM], b[NF][TN], bd[NF][TN];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const int r0 = (wm * WTM + i * 16) * ROWB + foff[c0 + f];
            if constexpr (SM::LA) a[f][i] = *reinterpret_cast<const bf16x8*>(As + r0);
            if constexpr (HAD) ad[f][i] = *reinterpret_cast<const bf16x8*>(Ads + r0);
          }
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int r0 = (wn * WTN + j * 16) * ROWB + foff[c0 + f];
            if constexpr (SM::LB) b[f][j] = *reinterpret_cast<const bf16x8*>(Bs + r0);
            if constexpr (HBD) bd[f][j] = *reinterpret_cast<const bf16x8*>(Bds + r0);
          }
        }
#pragma unroll
        for (int f = 0; f < NF; ++f)
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
              if constexpr (HC1) mma(acc1[i][j], a[f][i], b[f][j]);
              if constexpr (HAD) mma(acc2[i][j], ad[f][i], b[f][j]);
              if constexpr (HBD) mma(acc2[i][j], a[f][i], bd[f][j]);
            }
      }
    }
    wait_vm_lgkm<0>();
    lds_barrier();         // the trailing zero loads have landed: LDS is free
    stage_tile<FLAGS, BM, BN, BM>(acc1, acc2, S1, S2, wm * WTM);
    wait_vm_lgkm<0>();     // the staging writes are complete before other waves read them
    lds_barrier();
  }
  walk_tile<FLAGS, BN, BM, 512>(S1, S2, m0, n0, bz, epi);
}

template <int FLAGS, int BM, int BN, int BK, int NST, class Epi>
__global__ void __launch_bounds__(512) gemm_nt_ws(GemmOperands<bf16_t> op, Epi epi) {
  __shared__ __attribute__((aligned(1024))) char smem[DmaSmem<FLAGS, BM, BN, BK, NST, 1>::BYTES];
  gemm_ws_tile<FLAGS, BM, BN, BK, NST, Epi>(op, epi, (int)blockIdx.x, (int)blockIdx.y, smem);
}

// Two independent products in one launch, for products too small to fill the
// chip alone (at most two workgroups per compute unit between them): a layer's
// backward-weight product (parameter epilogue) and its backward-data product
// (activation epilogue).  Workgroup ids alternate between runs of G1 tiles of
// the first product and G2 of the second, so both run at once.
template <int F1, int BM1, int BN1, int NST1, class E1, int F2, int BM2, int BN2, int NST2,
          class E2>
__global__ void __launch_bounds__(512) gemm_pair_ws(GemmOperands<bf16_t> op1, E1 epi1, int t1,
                                                    int g1, GemmOperands<bf16_t> op2, E2 epi2,
                                                    int t2, int g2) {
  constexpr int B1 = DmaSmem<F1, BM1, BN1, 64, NST1, 1>::BYTES;
  constexpr int B2 = DmaSmem<F2, BM2, BN2, 64, NST2, 1>::BYTES;
  __shared__ __attribute__((aligned(1024))) char smem[B1 > B2 ? B1 : B2];
  const int b = (int)blockIdx.x;
  const int period = g1 + g2;
  const int cyc = min(t1 / g1, t2 / g2);
  int which, j;
  if (b < cyc * period) {
    const int q = b / period, r = b % period;
    which = r < g1 ? 0 : 1;
    j = which == 0 ? q * g1 + r : q * g2 + (r - g1);
  } else {
    const int r = b - cyc * period;
    const int rest1 = t1 - cyc * g1;
    which = r < rest1 ? 0 : 1;
    j = which == 0 ? cyc * g1 + r : cyc * g2 + (r - rest1);
  }
  if (which == 0)
    gemm_ws_tile<F1, BM1, BN1, 64, NST1, E1>(op1, epi1, j, 0, smem);
  else
    gemm_ws_tile<F2, BM2, BN2, 64, NST2, E2>(op2, epi2, j, 0, smem);
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// k depth per LDS stage of the register-staged loop: 64 keeps more MFMA work in
// flight per prefetch; the dual backward-weight kernels (short k = batch rows,
// heavy epilogue) use 32 so that their double-buffered tiles stay at 80 KB.
template <int FLAGS, class Epi>
struct KDepth {
  static constexpr int value = 64;
};
template <typename T>
struct KDepth<G_C1 | G_AD | G_BD, ParamOp<T>> {
  static constexpr int value = 32;
};
template <typename T>
struct KDepth<G_AD | G_BD, ParamOp<T>> {
  static constexpr int value = 32;
};
template <typename T>
struct KDepth<G_C1 | G_BD, ParamOp<T>> {
  static constexpr int value = 32;
};
template <typename T>
struct KDepth<G_BD, ParamOp<T>> {
  static constexpr int value = 32;
};

// Direct-to-LDS pipeline shape.  The k depth is 64 (128-byte rows): each 1 KB
// load then covers 8 whole 128-byte lines, where 64-byte rows make it touch 16
// half lines and halve the load unit's throughput.  Stages: as many 32 KB
// (two tiles), 48 KB (three) or 64 KB (four) stages as fit in 144 KB.
template <int FLAGS>
struct DmaShape {
  static constexpr int NOPS = ((FLAGS & (G_C1 | G_BD)) ? 1 : 0) + ((FLAGS & G_AD) ? 1 : 0) +
                              ((FLAGS & (G_C1 | G_AD)) ? 1 : 0) + ((FLAGS & G_BD) ? 1 : 0);
  static constexpr int BK = 64;
  static constexpr int NST = NOPS <= 2 ? 4 : NOPS == 3 ? 3 : 2;
};

// Pipeline depth of the small tiles (64 x 64, 64 x 32), whose products are
// bound by load latency rather than by delivery: as many stages as fit in an
// LDS budget per workgroup (144 KB with one workgroup per compute unit, 72 KB
// with two), 2 to 8.
template <int FLAGS, int BM, int BN, int BUDGET>
struct DmaDepth {
  static constexpr int STAGE = DmaSmem<FLAGS, BM, BN, 64, 2, 1>::STAGE_BYTES;
  static constexpr int N0 = BUDGET / STAGE;
  static constexpr int NST = BM > 64 ? DmaShape<FLAGS>::NST : N0 < 2 ? 2 : N0 > 8 ? 8 : N0;
};

template <typename T>
bool dma_operand_ok(const T* p, int rows, int ld, int K, long stride) {
  if (!p) return true;
  if ((reinterpret_cast<uintptr_t>(p) & 15) || (ld & 7) || (stride & 7)) return false;
  return rows <= 0 || ((long)(rows - 1) * ld + K) * (long)sizeof(T) < (1L << 31);
}

template <typename T>
bool dma_ok(const GemmOperands<T>& op) {
  if (sizeof(T) != 2 || (op.K & 7)) return false;
  return dma_operand_ok(op.A, op.M, op.lda, op.K, op.sA) &&
         dma_operand_ok(op.Ad, op.M, op.lda, op.K, op.sA) &&
         dma_operand_ok(op.B, op.N, op.ldb, op.K, op.sB) &&
         dma_operand_ok(op.Bd, op.N, op.ldb, op.K, op.sB);
}

template <typename T, int FLAGS, int BM, int BN, class Epi>
hipError_t launch(const GemmOperands<T>& op, const Epi& epi, hipStream_t s) {
  const int tiles = cdiv(op.M, BM) * cdiv(op.N, BN);
  if constexpr (sizeof(T) == 2) {
    typedef DmaShape<FLAGS> DS;
    if (dma_ok(op)) {
      if constexpr (BM == 64) {
        if (tiles * op.batch <= 256) {   // one workgroup per compute unit: a deeper ring
          constexpr int NST = DmaDepth<FLAGS, BM, BN, 147456>::NST;
          hipLaunchKernelGGL((gemm_nt_ws<FLAGS, BM, BN, DS::BK, NST, Epi>), dim3(tiles, op.batch),
                             dim3(512), 0, s, op, epi);
          return hipGetLastError();
        }
      }
      hipLaunchKernelGGL((gemm_nt_ws<FLAGS, BM, BN, DS::BK, DS::NST, Epi>), dim3(tiles, op.batch),
                         dim3(512), 0, s, op, epi);
      return hipGetLastError();
    }
  }
  if constexpr (BN >= 64 || BN == 16) {
    constexpr int BK = BN == 16 ? 64 : KDepth<FLAGS, Epi>::value;
    if (op.K % Elem<T>::VE == 0)
      hipLaunchKernelGGL((gemm_nt<T, FLAGS, BM, BN, BK, Epi, true>), dim3(tiles, op.batch),
                         dim3(256), 0, s, op, epi);
    else
      hipLaunchKernelGGL((gemm_nt<T, FLAGS, BM, BN, BK, Epi, false>), dim3(tiles, op.batch),
                         dim3(256), 0, s, op, epi);
    return hipGetLastError();
  }
  return hipErrorInvalidValue;
}

// ------------------------------------------------------------------------------------
// Split-K for backward-weight products with few output tiles and a long k (the
// token dimension of a transformer's weight gradients, and of its meta-model's):
// S batched products over k slices (128 x 128 tiles for bf16 operands, 64 x 64
// for float32) write float32 partial sums C1, C2 to the workspace, then a second
// kernel adds the S slices in order and applies the epilogue (row-major
// outputs through epi.row, transposed ones through epi.trans).
// ------------------------------------------------------------------------------------
int splitk_count(int M, int N, int K) {
  const int tiles = cdiv(M, 128) * cdiv(N, 128);
  if (M <= 0 || N <= 0 || tiles >= 192 || K < 1024) return 1;
  int S = (256 + tiles - 1) / tiles;
  if (S > 8) S = 8;
  if (S > K / 256) S = K / 256;
  while (S > 1 && K % (S * 64) != 0) --S;
  return S;
}

// Float32 products with at most 8 output tiles of 64 x 64 and a long k (say a
// 784-deep first layer with 128 x 256 outputs: 8 workgroups would each walk all
// of k), or at most 2 tiles and k >= 256 (a 10-wide output layer over 128 rows):
// up to 8 k slices, each at least 64 deep and a multiple of 4.
int splitk_count_small(int M, int N, int K) {
  const int tiles = cdiv(M, 64) * cdiv(N, 64);
  if (M <= 0 || N <= 0 || tiles > 8 || K < (tiles <= 2 ? 256 : 512)) return 1;
  if (N <= 16 && K <= 4096) return 1;   // 64 x 16 tiles instead (launch_sized)
  int S = 8;
  while (S > 1 && (K % S != 0 || (K / S) % 4 != 0 || K / S < 64)) --S;
  return S;
}

// One workgroup per 16 x 64 output tile, one thread per 4 columns of a row;
// the transposed outputs go through an LDS copy of the tile.
template <class Epi>
__global__ void __launch_bounds__(256) splitk_epilogue(const float* __restrict__ P1,
                                                       const float* __restrict__ P2, int S, int M,
                                                       int N, Epi epi) {
  __shared__ float T1[16][68], T2[16][68];
  const int tiles_n = (N + 63) / 64;
  const int m0 = (blockIdx.x / tiles_n) * 16, n0 = (blockIdx.x % tiles_n) * 64;
  const int r = threadIdx.x >> 4, c = (threadIdx.x & 15) * 4;
  const int m = m0 + r, n = n0 + c;
  const int cn = min(4, N - n);
  const long MN = (long)M * N;
  float c1[4] = {0.f, 0.f, 0.f, 0.f}, c2[4] = {0.f, 0.f, 0.f, 0.f};
  float t1[4] = {0.f, 0.f, 0.f, 0.f}, t2[4] = {0.f, 0.f, 0.f, 0.f};
  if (m < M && cn > 0) {
    constexpr int SMAX = 8;   // the most slices a split-K launch makes
    if (cn == 4 && (N & 3) == 0 && S <= SMAX) {
      // every slice's 16 bytes requested before the first is added; the sum
      // keeps the slice order
      float4 x[SMAX], y[SMAX];
#pragma unroll
      for (int sp = 0; sp < SMAX; ++sp)
        if (sp < S) {
          const long off = sp * MN + (long)m * N + n;
          x[sp] = *reinterpret_cast<const float4*>(P1 + off);
          if (P2) y[sp] = *reinterpret_cast<const float4*>(P2 + off);
        }
#pragma unroll
      for (int sp = 0; sp < SMAX; ++sp)
        if (sp < S) {
          c1[0] += x[sp].x; c1[1] += x[sp].y; c1[2] += x[sp].z; c1[3] += x[sp].w;
          if (P2) {
            c2[0] += y[sp].x; c2[1] += y[sp].y; c2[2] += y[sp].z; c2[3] += y[sp].w;
          }
        }
    } else {
      for (int sp = 0; sp < S; ++sp) {
        const long off = sp * MN + (long)m * N + n;
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (k < cn) {
            c1[k] += P1[off + k];
            if (P2) c2[k] += P2[off + k];
          }
      }
    }
    epi.row(0, m, n, cn, c1, c2, t1, t2);
  }
  const int nT = epi.n_trans();
  if (nT == 0) return;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    T1[r][c + k] = t1[k];
    T2[r][c + k] = t2[k];
  }
  __syncthreads();
  // thread: column cc of the tile, rows 4 q .. 4 q + 3
  const int cc = threadIdx.x >> 2, q = threadIdx.x & 3;
  const int nn = n0 + cc, mm = m0 + 4 * q;
  const int cm = min(4, M - mm);
  if (nn >= N || cm <= 0) return;
  float v[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) v[k] = T1[4 * q + k][cc];
  epi.trans(0, 0, nn, mm, cm, v);
  if (nT > 1) {
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = T2[4 * q + k][cc];
    epi.trans(1, 0, nn, mm, cm, v);
  }
}

template <typename T, int FLAGS, class Epi>
hipError_t launch_splitk(const GemmOperands<T>& op, const Epi& epi, int S, hipStream_t s) {
  constexpr bool HC2 = (FLAGS & (G_AD | G_BD)) != 0;
  const long MN = (long)op.M * op.N;
  GemmOperands<T> p = op;
  p.K = op.K / S;
  p.batch = S;
  p.sA = p.K;
  p.sB = p.K;
  p.ws = nullptr;
  p.ws_floats = 0;
  EpiStore e;
  e.C = op.ws; e.Cd = op.ws + S * MN; e.ldc = op.N; e.sC = MN; e.scale = 1.0f;
  e.M = op.M; e.N = op.N; e.dual = HC2 ? 1 : 0;
  hipError_t r;
  if constexpr (sizeof(T) == 2)
    r = launch<T, FLAGS, 128, 128>(p, StoreOp{e, op.M, op.N}, s);
  else
    r = launch<T, FLAGS, 64, 64>(p, StoreOp{e, op.M, op.N}, s);
  if (r != hipSuccess) return r;
  const int nb = cdiv(op.M, 16) * cdiv(op.N, 64);
  hipLaunchKernelGGL((splitk_epilogue<Epi>), dim3(nb), dim3(256), 0, s, op.ws,
                     HC2 ? op.ws + S * MN : nullptr, S, op.M, op.N, epi);
  return hipGetLastError();
}

template <typename T, int FLAGS, class Epi>
hipError_t launch_sized(const GemmOperands<T>& op, const Epi& epi, hipStream_t s) {
  if (op.M <= 0 || op.N <= 0) return hipSuccess;
  if constexpr (IsParamOp<Epi>::value) {
    if (op.ws && op.batch == 1) {
      const int S = splitk_count(op.M, op.N, op.K);
      if (S > 1 && op.ws_floats >= 2L * S * op.M * op.N)
        return launch_splitk<T, FLAGS>(op, epi, S, s);
    }
  }
  if constexpr (sizeof(T) == 4) {
    // at most 16 output columns: 64 x 16 tiles, a quarter of a 64 x 64 tile's
    // MFMA work (k at most 4096; longer narrow products split k above); also
    // short-k products with few 64 x 64 tiles, whose time is their epilogue:
    // four times the workgroups, each with a quarter of the outputs
    if (op.N <= 16 && op.K <= 4096) return launch<T, FLAGS, 64, 16>(op, epi, s);
    if (op.K <= 128 && cdiv(op.M, 64) * cdiv(op.N, 64) * op.batch < 64)
      return launch<T, FLAGS, 64, 16>(op, epi, s);
  }
  if constexpr (sizeof(T) == 4 && IsActFwdOp<Epi>::value) {
    if (op.ws && op.batch == 1) {
      const int S = splitk_count_small(op.M, op.N, op.K);
      if (S > 1 && op.ws_floats >= 2L * S * op.M * op.N)
        return launch_splitk<T, FLAGS>(op, epi, S, s);
    }
  }
  if constexpr (sizeof(T) == 2) {
    // 128 x 128 tiles once they alone fill most of the 256 compute units, else
    // 128 x 64 on the direct-to-LDS path (each compute unit then loads 128 + 64
    // rows per k step for 8192 outputs against 2 x 128 for two 64 x 64 tiles),
    // else 64 x 64, or 64 x 32 on the direct-to-LDS path when 64 x 64 tiles
    // would still leave compute units idle (512 x 1024 products: 256
    // workgroups instead of 128).
    if (cdiv(op.M, 128) * cdiv(op.N, 128) * op.batch >= 192)
      return launch<T, FLAGS, 128, 128>(op, epi, s);
    if (cdiv(op.M, 128) * cdiv(op.N, 64) * op.batch >= 192 && dma_ok(op))
      return launch<T, FLAGS, 128, 64>(op, epi, s);
    if (cdiv(op.M, 64) * cdiv(op.N, 64) * op.batch < 192 && dma_ok(op))
      return launch<T, FLAGS, 64, 32>(op, epi, s);
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

// The tile launch_sized picks for a bf16 product on the direct-to-LDS path:
// 0 = 128 x 128, 1 = 128 x 64, 2 = 64 x 64, 3 = 64 x 32; -1 when it would not take
// that path (float32, ragged k or strides, several batches, split-K).
template <typename T>
int dma_tile_kind(const GemmOperands<T>& o) {
  if (sizeof(T) != 2 || o.batch != 1 || o.M <= 0 || o.N <= 0 || !dma_ok(o)) return -1;
  if (o.ws && splitk_count(o.M, o.N, o.K) > 1) return -1;
  if (cdiv(o.M, 128) * cdiv(o.N, 128) >= 192) return 0;
  if (cdiv(o.M, 128) * cdiv(o.N, 64) >= 192) return 1;
  if (cdiv(o.M, 64) * cdiv(o.N, 64) >= 192) return 2;
  return 3;
}

template <int F1, int BM1, int BN1, class E1, int F2, int BM2, int BN2, class E2>
hipError_t launch_pair(const GemmOperands<bf16_t>& o1, const E1& e1,
                       const GemmOperands<bf16_t>& o2, const E2& e2, hipStream_t s) {
  const int t1 = cdiv(o1.M, BM1) * cdiv(o1.N, BN1);
  const int t2 = cdiv(o2.M, BM2) * cdiv(o2.N, BN2);
  // runs of 8 tiles of the smaller product and about 8 x the ratio of the larger
  int g1 = 8, g2 = 8;
  if (t2 >= t1) g2 = 8 * max(1, (t2 + t1 / 2) / max(t1, 1));
  else g1 = 8 * max(1, (t1 + t2 / 2) / max(t2, 1));
  // at most two workgroups per compute unit: 72 KB rings
  hipLaunchKernelGGL((gemm_pair_ws<F1, BM1, BN1, DmaDepth<F1, BM1, BN1, 73728>::NST, E1, F2, BM2,
                                   BN2, DmaDepth<F2, BM2, BN2, 73728>::NST, E2>),
                     dim3(t1 + t2), dim3(512), 0, s, o1, e1, t1, g1, o2, e2, t2, g2);
  return hipGetLastError();
}

template <int FW, int FD, typename T>
hipError_t pair_by_tiles(int kw, int kd, const GemmOperands<bf16_t>& ow, const ParamOp<T>& ew,
                         const GemmOperands<bf16_t>& od, const ActBwdOp<T>& ed, hipStream_t s) {
  if (kw == 2 && kd == 2)
    return launch_pair<FW, 64, 64, ParamOp<T>, FD, 64, 64, ActBwdOp<T>>(ow, ew, od, ed, s);
  if (kw == 2 && kd == 3)
    return launch_pair<FW, 64, 64, ParamOp<T>, FD, 64, 32, ActBwdOp<T>>(ow, ew, od, ed, s);
  if (kw == 3 && kd == 2)
    return launch_pair<FW, 64, 32, ParamOp<T>, FD, 64, 64, ActBwdOp<T>>(ow, ew, od, ed, s);
  return launch_pair<FW, 64, 32, ParamOp<T>, FD, 64, 32, ActBwdOp<T>>(ow, ew, od, ed, s);
}

}  // namespace

template <typename T>
bool gemm_pairs(const GemmOperands<T>& opw, int flags_w, const GemmOperands<T>& opd,
                int flags_d) {
  // products on 64 x 64 or 64 x 32 tiles (two workgroups fit on a compute unit)
  // that together need at most two workgroups per compute unit
  const int kw = dma_tile_kind(opw), kd = dma_tile_kind(opd);
  if (kw < 2 || kd < 2) return false;
  const bool flags_ok = (flags_w == G_C1 && flags_d == G_C1) ||
                        (flags_w == (G_C1 | G_AD | G_BD) && flags_d == (G_C1 | G_AD | G_BD)) ||
                        (flags_w == (G_AD | G_BD) && flags_d == (G_C1 | G_AD | G_BD));
  const int tw = kw == 2 ? cdiv(opw.M, 64) * cdiv(opw.N, 64) : cdiv(opw.M, 64) * cdiv(opw.N, 32);
  const int td = kd == 2 ? cdiv(opd.M, 64) * cdiv(opd.N, 64) : cdiv(opd.M, 64) * cdiv(opd.N, 32);
  return flags_ok && tw + td <= 512;
}

template <typename T>
hipError_t gemm_param_and_act_bwd(const GemmOperands<T>& opw, int flags_w, const ParamArgs<T>& P,
                                  const GemmOperands<T>& opd, int flags_d,
                                  const EpiActBwd<T>& e, hipStream_t s) {
  if constexpr (sizeof(T) == 2) {
    if (gemm_pairs(opw, flags_w, opd, flags_d)) {
      const int kw = dma_tile_kind(opw), kd = dma_tile_kind(opd);
      {
        const ParamOp<T> ew{P, P.nin, P.nout};
        const ActBwdOp<T> ed{e, e.M, e.N};
        if (flags_w == G_C1 && flags_d == G_C1)
          return pair_by_tiles<G_C1, G_C1, T>(kw, kd, opw, ew, opd, ed, s);
        if (flags_w == (G_C1 | G_AD | G_BD) && flags_d == (G_C1 | G_AD | G_BD))
          return pair_by_tiles<G_C1 | G_AD | G_BD, G_C1 | G_AD | G_BD, T>(kw, kd, opw, ew, opd, ed, s);
        if (flags_w == (G_AD | G_BD) && flags_d == (G_C1 | G_AD | G_BD))
          return pair_by_tiles<G_AD | G_BD, G_C1 | G_AD | G_BD, T>(kw, kd, opw, ew, opd, ed, s);
      }
    }
  }
  hipError_t r = gemm_param<T>(opw, flags_w, P, s);
  if (r != hipSuccess) return r;
  return gemm_act_bwd<T>(opd, flags_d, e, s);
}

// Both tile kernels sum the bias entries of a parameter epilogue; split-K
// launches and batched products do not.
template <typename T>
bool gemm_fuses_bias(const GemmOperands<T>& op, int flags) {
  if (flags == 0 || op.batch != 1 || op.M <= 0 || op.N <= 0) return false;
  return !(op.ws && splitk_count(op.M, op.N, op.K) > 1);
}
template bool gemm_fuses_bias<bf16_t>(const GemmOperands<bf16_t>&, int);
template bool gemm_fuses_bias<float>(const GemmOperands<float>&, int);

long gemm_splitk_floats(int M, int N, int K) {
  const int S = splitk_count(M, N, K);
  return S > 1 ? 2L * S * M * N : 0;
}

long gemm_splitk_fwd_f32_floats(int M, int N, int K) {
  const int S = splitk_count_small(M, N, K);
  return S > 1 ? 2L * S * M * N : 0;
}

template <typename T>
hipError_t gemm_act_fwd(const GemmOperands<T>& op, int flags, const EpiActFwd<T>& epi,
                        hipStream_t s) {
  return dispatch(op, flags, ActFwdOp<T>{epi, epi.M, epi.N}, s);
}
template <typename T>
hipError_t gemm_act_bwd(const GemmOperands<T>& op, int flags, const EpiActBwd<T>& epi,
                        hipStream_t s) {
  return dispatch(op, flags, ActBwdOp<T>{epi, epi.M, epi.N}, s);
}
template <typename T>
hipError_t gemm_param(const GemmOperands<T>& op, int flags, const ParamArgs<T>& P,
                      hipStream_t s) {
  return dispatch(op, flags, ParamOp<T>{P, P.nin, P.nout}, s);
}

template <typename T>
hipError_t gemm_store(const GemmOperands<T>& op, int flags, const EpiStore& e, hipStream_t s) {
  return dispatch(op, flags, StoreOp{e, e.M, e.N}, s);
}
template <typename T>
hipError_t gemm_resid(const GemmOperands<T>& op, int flags, const EpiResid& e, hipStream_t s) {
  return dispatch(op, flags, ResidOp{e, e.M, e.N}, s);
}
template <typename T>
hipError_t gemm_head_merge(const GemmOperands<T>& op, int flags, const EpiHeadMerge<T>& e,
                           hipStream_t s) {
  return dispatch(op, flags, HeadMergeOp<T>{e, e.M, e.N}, s);
}
template <typename T>
hipError_t gemm_head_split(const GemmOperands<T>& op, int flags, const EpiHeadSplit<T>& e,
                           hipStream_t s) {
  return dispatch(op, flags, HeadSplitOp<T>{e, e.M, e.N}, s);
}

template hipError_t gemm_store<bf16_t>(const GemmOperands<bf16_t>&, int, const EpiStore&, hipStream_t);
template hipError_t gemm_store<float>(const GemmOperands<float>&, int, const EpiStore&, hipStream_t);
template hipError_t gemm_resid<bf16_t>(const GemmOperands<bf16_t>&, int, const EpiResid&, hipStream_t);
template hipError_t gemm_resid<float>(const GemmOperands<float>&, int, const EpiResid&, hipStream_t);
template hipError_t gemm_head_merge<bf16_t>(const GemmOperands<bf16_t>&, int, const EpiHeadMerge<bf16_t>&, hipStream_t);
template hipError_t gemm_head_merge<float>(const GemmOperands<float>&, int, const EpiHeadMerge<float>&, hipStream_t);
template hipError_t gemm_head_split<bf16_t>(const GemmOperands<bf16_t>&, int, const EpiHeadSplit<bf16_t>&, hipStream_t);
template hipError_t gemm_head_split<float>(const GemmOperands<float>&, int, const EpiHeadSplit<float>&, hipStream_t);
template hipError_t gemm_act_fwd<bf16_t>(const GemmOperands<bf16_t>&, int, const EpiActFwd<bf16_t>&, hipStream_t);
template hipError_t gemm_act_fwd<float>(const GemmOperands<float>&, int, const EpiActFwd<float>&, hipStream_t);
template hipError_t gemm_act_bwd<bf16_t>(const GemmOperands<bf16_t>&, int, const EpiActBwd<bf16_t>&, hipStream_t);
template hipError_t gemm_act_bwd<float>(const GemmOperands<float>&, int, const EpiActBwd<float>&, hipStream_t);
template hipError_t gemm_param<bf16_t>(const GemmOperands<bf16_t>&, int, const ParamArgs<bf16_t>&, hipStream_t);
template hipError_t gemm_param<float>(const GemmOperands<float>&, int, const ParamArgs<float>&, hipStream_t);

template bool gemm_pairs<bf16_t>(const GemmOperands<bf16_t>&, int, const GemmOperands<bf16_t>&, int);
template bool gemm_pairs<float>(const GemmOperands<float>&, int, const GemmOperands<float>&, int);
template hipError_t gemm_param_and_act_bwd<bf16_t>(const GemmOperands<bf16_t>&, int, const ParamArgs<bf16_t>&, const GemmOperands<bf16_t>&, int, const EpiActBwd<bf16_t>&, hipStream_t);
template hipError_t gemm_param_and_act_bwd<float>(const GemmOperands<float>&, int, const ParamArgs<float>&, const GemmOperands<float>&, int, const EpiActBwd<float>&, hipStream_t);

}  // namespace mfmg
