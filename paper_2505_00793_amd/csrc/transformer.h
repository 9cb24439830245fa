// Interfaces of the decoder-block dual kernels (transformer.hip).
#pragma once

#include "kernels.h"

namespace mfmg {

constexpr int LN_CHUNK = 64;  // rows per partial column sum of the LayerNorm backward
constexpr int LN_MAX_D = 1024;
constexpr int TOKEN_SORT_MAX = 8192;
constexpr int EMB_SEG = 32;   // positions per embedding-gradient segment
constexpr int META_ROWS_PER_BLOCK = 128;
constexpr int META_MAX_HIDDEN = 256;

struct LnArgs {
  const float* x;  const float* xd;          // [N][d] input (and tangent)
  const float* g;  const float* b;           // gain, bias [d]
  const float* gd; const float* bd;          // their tangents
  float* y;  float* yd;                      // [N][d] output (and tangent)
  float* xh; float* xhd;                     // normalised input (and tangent), saved
  float* rstd; float* c;                     // [N] 1/sigma and mean(xh xd), saved
  bf16_t* yb; bf16_t* ydb;                   // if set (d a multiple of 256): y, yd as bf16
  int ldb;                                   //   rows [N][ldb] instead of the float32 ones
  int N, d, dual;
  float eps;
};

struct LnBwdArgs {
  const float* dy; const float* dyd;         // [N][d] cotangent of y (and tangent)
  const float* xh; const float* xhd;
  const float* rstd; const float* c;
  const float* g;  const float* gd;
  const float* dh_in; const float* dhd_in;   // residual-stream gradient entering
  float* dh_out; float* dhd_out;             // dh_in + dx (may alias dh_in)
  float* partial;                            // [ln_bwd_parts(N)][4][d] column-sum partials
  bf16_t* hb; bf16_t* hdb;                   // if set (d a multiple of 256): also bf16 rows
  int ldb;                                   //   [N][ldb] of dh_out, dhd_out
  int N, d, dual;
};

struct RopeArgs {
  const float* qkv; const float* qkvd;       // split: [N][3d] in
  float* Q; float* K; float* V;              // per-head [B*H][S][dh]
  float* Qd; float* Kd; float* Vd;
  bf16_t* Qb; bf16_t* Kb; bf16_t* Vb;        // split: if set, bf16 per-head rows instead
  bf16_t* Qdb; bf16_t* Kdb; bf16_t* Vdb;
  float* qkv_out; float* qkvd_out;           // merge: [N][3d] out
  bf16_t* ob; bf16_t* odb; int ldb;          // merge: if set, bf16 rows [N][ldb] instead
  const float* cs; const float* sn;          // [S][dh/2]
  int N, S, H, dh, dual;
};

struct SoftmaxArgs {
  const float* Sc; const float* Scd;         // scores (scaled) [rows][S]
  float* P; float* Pd;                       // probabilities (and tangent)
  const float* dP; const float* dPd;         // backward: cotangent of P
  float* dS; float* dSd;                     // backward: scale * cotangent of the scores
  long rows;
  int S, dual;
  float scale;
};

// Fused causal attention of head dimension 64 over bf16 operands (forward and
// backward, primal or dual).  Per-head operands are rows [B*H][S][64] and
// transposes [B*H][64][S]; S is a multiple of 64.
struct AttnArgs {
  const bf16_t *Q, *K, *V, *QT, *KT, *VT;         // per-head operands
  const bf16_t *Qd, *Kd, *Vd, *QdT, *KdT, *VdT;   // their tangents (dual)
  bf16_t *O, *OT, *Od, *OdT;                      // token-major [N][ldO], transposed [d][ldOT]
  int ldO, ldOT;
  float *lse, *cst;                               // [B*H][S] saved by the forward: m + log l, <P, Sd>
  const bf16_t *dO, *dOT, *dOd, *dOdT;            // per-head cotangent of O (and its tangent)
  float *r, *rd;                                  // [B*H][S] <dO, O>, <dOd, O> + <dO, Od>
  float *dQ, *dK, *dV, *dQd, *dKd, *dVd;          // fp32 per-head rows [B*H][S][64]
  int S, H, BH, dh, dual;
  float scale;
};

// Token positions sorted by id are cut into segments: maximal runs of one id,
// split further at every multiple of EMB_SEG in the sorted order, so that a
// segment holds at most EMB_SEG positions of one token.
struct TokenSegs {
  int* perm;       // [N] positions in ascending (id, position) order
  int* seg_start;  // [embed_segments_max(N) + 1] first sorted index of each segment; sentinel
  int* seg_tok;    // [embed_segments_max(N)] token id of each segment
  int* nseg;       // [1] number of segments
  int* tok2seg;    // [V] first segment of each token, -1 if absent
};

struct EmbedGradArgs {
  const float* dh; const float* dhd;         // [N][d] gradient at the embedding output
  TokenSegs ts;
  float* part;                               // [embed_segments_max(N)][2][d] segment sums
  long emb_off;
  float* outE;                               // operand copy of the new rows (fp32 [V][d]) or null
  int V, d, N;
};

hipError_t split_tokens(const int* tok, int B, int S, int V, int* ids, int* labels,
                        hipStream_t s);
hipError_t gather_rows(const int* ids, int N, int d, const float* E, const float* Ed, float* h,
                       float* hd, hipStream_t s);
hipError_t ln_fwd(const LnArgs& a, hipStream_t s);
int ln_bwd_parts(int N);
template <typename T>
hipError_t ln_bwd(const LnBwdArgs& a, long g_off, long b_off, const ParamArgs<T>& P,
                  float* out_g, float* out_b, hipStream_t s);
hipError_t rope_table(int S, int dh, double base, float* cs, float* sn, hipStream_t s);
hipError_t rope_split(const RopeArgs& a, hipStream_t s);
hipError_t rope_merge(const RopeArgs& a, hipStream_t s);
hipError_t softmax_fwd(const SoftmaxArgs& a, hipStream_t s);
hipError_t softmax_bwd(const SoftmaxArgs& a, hipStream_t s);
bool attn_fused_supported(int S, int dh);
hipError_t attn_fwd(const AttnArgs& a, hipStream_t s);
hipError_t attn_bwd(const AttnArgs& a, hipStream_t s);  // dQ pass (writes r, rd), then dK/dV pass
bool sort_tokens_fits(int N);
int embed_segments_max(int N);
hipError_t sort_tokens(const int* ids, int N, int V, const TokenSegs& ts, hipStream_t s);
template <typename T>
hipError_t embed_grad(const EmbedGradArgs& a, const ParamArgs<T>& P, hipStream_t s);
hipError_t meta_out(const float* hid, int rows, int hdim, const float* w2, const float* b2,
                    float* u, hipStream_t s);
int meta_vjp_parts(int rows);
hipError_t meta_vjp(const float* hid, const float* ubar, int rows, int hdim, const float* w2,
                    float* dhid, float* partial, float* d_w2, float* d_b1, float* d_b2,
                    hipStream_t s);

}  // namespace mfmg
