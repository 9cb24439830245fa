// Internal interfaces between the C ABI front end (api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"
#include "mfmg.h"

namespace mfmg {

// ------------------------------------------------------------------------------------
// Dual NT GEMM: every operand is stored with its contraction index contiguous.
//   C1[m][n] = sum_k A[m][k] B[n][k]                      (flag G_C1)
//   C2[m][n] = sum_k Ad[m][k] B[n][k] + A[m][k] Bd[n][k]  (flags G_AD, G_BD)
// (A, Ad): M x K with leading dimension lda; (B, Bd): N x K with ldb.  Leading
// dimensions are multiples of 16 bytes and base pointers are 16-byte aligned.
// ------------------------------------------------------------------------------------
enum GemmFlags { G_C1 = 1, G_AD = 2, G_BD = 4 };

template <typename T>
struct GemmOperands {
  const T* A;
  const T* Ad;
  const T* B;
  const T* Bd;
  int lda, ldb;
  int M, N, K;
  int batch = 1;      // independent products (grid.y); operand z starts at A + z * sA
  long sA = 0, sB = 0;
  // Optional float32 workspace for split-K (products with few output tiles and
  // a long k): null, or ws_floats >= gemm_splitk_floats(M, N, K).
  float* ws = nullptr;
  long ws_floats = 0;
};

// Workspace (floats) that the backward-weight product of an M x N output over K
// uses for split-K when given it; 0 when it runs without (bf16 operands, one
// batch).
long gemm_splitk_floats(int M, int N, int K);
// Workspace (floats) that a float32 forward product (activation epilogue) of an
// M x N output over K uses for split-K when given it (few output tiles, long k);
// 0 when it runs without.
long gemm_splitk_fwd_f32_floats(int M, int N, int K);
// Whether the parameter GEMM of op / flags (B = dZ^T, Bd = its tangent) sums the
// bias gradients of P.fuse_bias itself (either tile kernel; not split-K or
// batched launches).
template <typename T>
bool gemm_fuses_bias(const GemmOperands<T>& op, int flags);

// Forward of one layer: z = C1 + b, zd = C2 + bd (tangent), a = act(z),
// ad = act'(z) zd.  Hidden layers store z (and zd) in float32 for the
// backward (not with ReLU: Z and Zd null, the backward reads the sign of a) and
// a (ad) as operands in both layouts; the output layer stores the logits z (and
// zd) only.
template <typename T>
struct EpiActFwd {
  const float* bias;     // [N] or null
  const float* bias_d;   // [N] or null (tangent of the bias)
  int act, last, dual;
  int M, N;
  float* Z;              // [M][N]
  float* Zd;             // [M][N] (dual)
  T* Ao;  T* AoT;        // [M][ldA], [N][ldAT]
  T* Ado; T* AdoT;       // (dual)
  int ldA, ldAT;
};

// Backward-data of one layer: C1 = dA of the previous layer's output, C2 its
// tangent.  dz = dA * act'(z), dzd = dAd * act'(z) + dA * act''(z) * zd, stored
// as operands in both layouts.  For ReLU, act'(z) = [z > 0] = [a > 0] and
// act'' = 0, so the previous layer's activation operand rows Ap can stand in for
// its pre-activations (Zp and Zdp null).
template <typename T>
struct EpiActBwd {
  const float* Zp;       // [M][N] pre-activations of the previous layer, or null
  const float* Zdp;      // [M][N] their tangents (dual), or null
  const T* Ap;           // ReLU without Zp: activations of the previous layer [M][ldAp]
  int ldAp;
  int act, dual;
  int M, N;
  T* dZ;  T* dZT;        // [M][ld], [N][ldT]
  T* dZd; T* dZdT;
  int ld, ldT;
};

// What the per-parameter epilogue does with (g, hv) = (C1, C2) of a
// backward-weight GEMM (and of the bias reduction).
// Plain float32 store of scale * C1 (and scale * C2): C[z * sC + m * ldc + n].
struct EpiStore {
  float* C;
  float* Cd;
  int ldc;
  long sC;
  float scale;
  int M, N, dual;
};

// Residual stream update: Ho = H + C1, Hdo = Hd + C2 (float32 [M][N]).
struct EpiResid {
  const float* H;
  const float* Hd;
  float* Ho;
  float* Hdo;
  int M, N, dual;
};

// Attention output of head z = b * heads + h (rows = query positions s,
// columns = head dims j) written as operands in token-major layout:
// O[(b * seq + s) * ldO + h * dh + j] and the transpose OT[(h * dh + j) * ldOT + b * seq + s].
template <typename T>
struct EpiHeadMerge {
  T* O; T* OT; T* Od; T* OdT;
  int ldO, ldOT;
  int seq, heads, dh;
  int M, N, dual;
};

// The inverse: a token-major [tokens][heads * dh] result written per head,
// Oh[((b * heads + h) * seq + s) * ldh + j] and OhT[((b * heads + h) * dh + j) * ldhT + s].
template <typename T>
struct EpiHeadSplit {
  T* Oh; T* OhT; T* Odh; T* OdhT;
  int ldh, ldhT;
  int seq, heads, dh;
  int M, N, dual;
};

enum ParamMode {
  P_UPD_SGD_PP = 0,     // theta' = theta - exp(eta) g
  P_UPD_SGD_FIXED = 1,  // theta' = theta - lr g
  P_UPD_ADAM = 2,       // Adam with bias correction, per-layer lr, decoupled decay
  P_SEED_SGD_PP = 3,    // tb = g (= dV/dtheta_T); v = -exp(eta) tb
  P_SEED_SGD_FIXED = 4, // tb = g; v = -lr tb
  P_SEED_ADAM = 5,      // tb = g
  P_REV_SGD_PP = 6,     // eb (+)= -exp(eta) g tb; tb += hv; v = -exp(eta) tb
  P_REV_SGD_FIXED = 7,  // tb += hv; v = -lr tb
  P_REV_ADAM = 8,       // tb += hv
  P_HVP = 9,            // grad_out = g; hvp_out = hv
  P_STORE_G = 10        // grad_out = g
};

template <typename T>
struct ParamArgs {
  int mode;
  int layer, n_layers;
  int nin, nout;
  long w_off, b_off;       // offsets of W_l and b_l in the flat theta layout
  // update
  const float* theta;      // theta_t
  float* theta_next;
  const float* eta;
  float lr;
  const float* m_in; const float* v_in;
  float* m_out; float* v_out; float* g_save;
  float b1, b2, eps, k1, k2;  // k1 = 1 - b1^t, k2 = 1 - b2^t
  float* grad_out;
  // reverse
  float* thetabar;
  float* etabar;
  int first;
  float* hvp_out;
  // operand copies written by the epilogue (new theta for P_UPD_*, the next
  // tangent for P_SEED_SGD_* and P_REV_SGD_*); each may be null
  T* outW; T* outWT; float* outb;
  int ldW, ldWT;
  // set by the host when the backward-weight GEMM also finishes the bias
  // entries (the tiles of each tile column share out the column's entries and
  // sum the rows of dZ^T they stage; see gemm_fuses_bias), so that no separate
  // reduction runs
  int fuse_bias;
};

template <typename T>
struct LossArgs {
  int loss;                 // 0 MSE, 1 CE, 2 MSE after the M-step map (mean over outputs)
  int map_M;                // M of that map
  int rows, C, dual;
  float inv_n;
  const float* Z;           // [rows][C] outputs
  const float* Zd;          // [rows][C] their tangents (dual)
  const int* labels;        // CE
  const float* targets;     // MSE [rows][C]
  const float* alpha_logits;  // per-row weight logits, or null (weights 1)
  T* d; T* dT;              // dL/dz in both layouts [rows][ld], [C][ldT]
  T* dd; T* ddT;            // its tangent (dual)
  int ld, ldT;
  int pad_to;               // columns C .. pad_to - 1 of d (dd) are written as zero
  int direct_t;             // set by loss_head: the kernel also writes dT (ddT) itself
  float* loss_rows;         // l_n (unweighted), or null
  float* mvp_rows;          // (1/N) ldot_n, or null
  float* deta_rows;         // sigmoid'(eta_n) (1/N) ldot_n, or null
};

template <typename T>
hipError_t gemm_act_fwd(const GemmOperands<T>& op, int flags, const EpiActFwd<T>& epi,
                        hipStream_t s);
template <typename T>
hipError_t gemm_act_bwd(const GemmOperands<T>& op, int flags, const EpiActBwd<T>& epi,
                        hipStream_t s);
template <typename T>
hipError_t gemm_param(const GemmOperands<T>& op, int flags, const ParamArgs<T>& P,
                      hipStream_t s);
// A layer's backward-weight product (with the parameter epilogue) and its
// backward-data product (with the activation epilogue), which are independent:
// one launch running both when they are small (bf16 operands on 64-row tiles,
// at most two workgroups per compute unit together), else the two launches
// above in that order.
template <typename T>
bool gemm_pairs(const GemmOperands<T>& opw, int flags_w, const GemmOperands<T>& opd, int flags_d);
template <typename T>
hipError_t gemm_param_and_act_bwd(const GemmOperands<T>& opw, int flags_w, const ParamArgs<T>& P,
                                  const GemmOperands<T>& opd, int flags_d,
                                  const EpiActBwd<T>& e, hipStream_t s);
template <typename T>
hipError_t gemm_store(const GemmOperands<T>& op, int flags, const EpiStore& e, hipStream_t s);
template <typename T>
hipError_t gemm_resid(const GemmOperands<T>& op, int flags, const EpiResid& e, hipStream_t s);
template <typename T>
hipError_t gemm_head_merge(const GemmOperands<T>& op, int flags, const EpiHeadMerge<T>& e,
                           hipStream_t s);
template <typename T>
hipError_t gemm_head_split(const GemmOperands<T>& op, int flags, const EpiHeadSplit<T>& e,
                           hipStream_t s);

// float32 matrix [rows][cols] (leading dim lds) -> operand copies dst [rows][ldd]
// and dstT [cols][lddT] (either may be null).
template <typename T>
hipError_t convert_matrix(const float* src, int rows, int cols, int lds, T* dst, int ldd,
                          T* dstT, int lddT, hipStream_t s, int batch = 1, long s_src = 0,
                          long s_dst = 0, long s_dstT = 0);

// The same for up to CONV_MAX_JOBS matrices of one shape and layout in one
// launch (job k: src[k] -> dst[k], dstT[k]; src[k] non-null).
constexpr int CONV_MAX_JOBS = 6;
template <typename T>
struct ConvJobs {
  int n = 0;
  const float* src[CONV_MAX_JOBS] = {};
  T* dst[CONV_MAX_JOBS] = {};
  T* dstT[CONV_MAX_JOBS] = {};
};
// Transposed copies of bf16 matrices: up to TR_MAX_JOBS of one shape, each a
// batch of matrices at strides s_src / s_dst (rows, leading dimensions and
// strides multiples of 8; cols may be ragged when ld >= cols rounded up to 8).
constexpr int TR_MAX_JOBS = 6;
struct TrJobs {
  int n = 0;
  const bf16_t* src[TR_MAX_JOBS];
  bf16_t* dst[TR_MAX_JOBS];
};
hipError_t transpose_bf16_jobs(const TrJobs& J, int batch, int rows, int cols, int ld, int ldT,
                               long s_src, long s_dst, hipStream_t s);
// One or two matrices (a1/t1 may be null).
hipError_t transpose_bf16(const bf16_t* a0, const bf16_t* a1, int rows, int cols, int ld,
                          bf16_t* t0, bf16_t* t1, int ldT, hipStream_t s);
template <typename T>
hipError_t convert_matrices(const ConvJobs<T>& J, int rows, int cols, int lds, int ldd, int lddT,
                            hipStream_t s, int batch = 1, long s_src = 0, long s_dst = 0,
                            long s_dstT = 0);

// Column sums over rows of dZT [nout][ld] (and dZdT) -> per-parameter epilogue
// on the bias entries of layer P.layer.
template <typename T>
hipError_t bias_reduce(const T* dZT, const T* dZdT, int ld, int rows, const ParamArgs<T>& P,
                       hipStream_t s);

template <typename T>
hipError_t loss_head(const LossArgs<T>& a, hipStream_t s);

// loss_out = (1/N) sum_n alpha_n l_n (alpha from logits, or 1).
hipError_t loss_reduce(const float* loss_rows, const float* alpha_logits, int rows, float inv_n,
                       float* loss_out, hipStream_t s);

// Adam's reverse step before the dual pass (see adam_vjp in elementwise.hip).
template <typename T>
struct AdamVjpArgs {
  int layer, n_layers, nin, nout;
  long w_off, b_off;
  int first;                     // adjoints of m and v are zero (i = T-1)
  float b1, b2, eps, k1, k2;
  const float* eta;
  const float* theta; const float* m; const float* v; const float* g;   // step i state
  float* thetabar; float* mbar; float* vbar;                            // in/out
  T* vW; T* vWT; float* vb; int ldW, ldWT;                              // tangent out
};
// The Adam reverse of layers 0 .. L-1 of one step in one launch.  partial:
// [blocks][2] (eta_l partial, omega partial); layer l owns blocks
// part_off[l] .. part_off[l + 1] - 1, which must be its 16 x 64 tiles of W plus
// its bias blocks of 256 entries.
template <typename T>
hipError_t adam_vjp(const AdamVjpArgs<T>* a, int L, const int* part_off, float* partial,
                    hipStream_t s);

// d_eta[layer] (+)= sum partial[l][.][0]; d_eta[L] (+)= sum of all partial[.][1].
hipError_t adam_reduce(const float* partial, const int* block_offsets, int n_layers, int first,
                       float* d_eta, hipStream_t s);

// Linear regression, SGD with per-parameter log learning rates, squared loss:
// the whole meta-gradient in one workgroup.  xs, ys: host arrays of T device
// pointers; scratch: (T + 1) * d floats of device memory.
hipError_t linreg_meta_grad(const float* theta0, const float* eta, const float* const* xs,
                            const float* const* ys, int T, int rows, int d, const float* vx,
                            const float* vy, int vrows, float* d_eta, float* val_loss,
                            float* scratch, hipStream_t s);
bool linreg_fits(int T, int rows, int vrows, int d);

// Fill / copy float arrays with kernels (no memset or memcpy nodes, so the
// calls stay safe inside captured HIP graphs).
hipError_t fill(float* p, long n, float v, hipStream_t s);

// Zero columns c0 .. c1 - 1 (c1 <= ld) of up to ZC_MAX_JOBS bf16 matrices in one
// launch (a fill kernel, no memset node).
constexpr int ZC_MAX_JOBS = 48;
struct ZeroColJobs {
  int n;
  uint16_t* p[ZC_MAX_JOBS];
  int rows[ZC_MAX_JOBS], ld[ZC_MAX_JOBS], c0[ZC_MAX_JOBS], c1[ZC_MAX_JOBS];
};
hipError_t zero_cols(const ZeroColJobs& J, hipStream_t s);
hipError_t copy(const float* src, float* dst, long n, hipStream_t s);

// *count (device) = number of NaN or infinite entries of x[0..n).
hipError_t count_nonfinite(const float* x, long n, unsigned long long* count, hipStream_t s);

// Kernel timing (api.hip).
void timing_begin(int cls, hipStream_t s);
void timing_end(int cls, hipStream_t s);

}  // namespace mfmg
