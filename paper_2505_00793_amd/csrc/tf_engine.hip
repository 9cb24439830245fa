// Transformer meta-gradient engine: a decoder-only pre-LayerNorm transformer
// with RoPE (the Chinchilla-style inner models of Section 5), next-token
// cross-entropy weighted per token by alpha = sigmoid(u), u from a two-layer
// meta-model on the initial token embeddings (adaptive loss weighting,
// Section 5.2), trained by SGD with a fixed learning rate.
//
// Every pass is a dual pass when a tangent operand set is given: the forward
// carries (h, hd) through LayerNorm, the QKV product, RoPE, causal attention,
// the output projection, the GELU MLP and the unembedding; the backward
// carries the cotangents and their tangents back to the parameters, whose
// epilogue applies the update (unroll), the seed (validation pass) or the
// reverse accumulation bar theta += H v, v' = -lr bar theta (Section 3,
// eq. bptt_recur with eq. vhp_to_hvp); the loss head's per-token loss
// tangent gives the mixed product that flows into the meta-model
// (eq. vmp_to_mvp).  All activations of one inner step are kept (dynamic
// memory, independent of T); checkpoints hold the operand copies of theta_t.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include <initializer_list>
#include <type_traits>

#include "kernels.h"
#include "tf_engine.h"
#include "transformer.h"

namespace mfmg {

namespace {

inline long rup(long x, long m) { return (x + m - 1) / m * m; }

struct Carver {
  char* base;
  size_t off = 0;
  template <typename T>
  T* take(size_t n) {
    off = (size_t)rup((long)off, 256);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
};

constexpr int MAXB = 16;

struct Lay {
  int d, H, dh, F, V, S, Bt, Bv, L, mh, VE, fused, remat;
  float eps, lr;
  double base;
  long emb, ln1g[MAXB], ln1b[MAXB], wqkv[MAXB], wo[MAXB], ln2g[MAXB], ln2b[MAXB], w1[MAXB],
      w2[MAXB], lnfg, lnfb, unemb, n;
  long ld(long x) const { return rup(x, VE); }
  int maxB() const { return std::max(Bt, Bv); }
  // per-block matrices: 0 wqkv d->3d, 1 wo d->d, 2 w1 d->F, 3 w2 F->d
  int in(int m) const { return m == 3 ? F : d; }
  int out(int m) const { return m == 0 ? 3 * d : m == 2 ? F : d; }
  long woff(int b, int m) const { return m == 0 ? wqkv[b] : m == 1 ? wo[b] : m == 2 ? w1[b] : w2[b]; }
};

Lay make_lay(const mfmg_problem_desc& D) {
  Lay y;
  y.d = D.d_model;
  y.H = D.n_heads;
  y.dh = D.d_model / D.n_heads;
  y.F = D.d_ff;
  y.V = D.vocab;
  y.S = D.seq;
  y.Bt = D.rows;
  y.Bv = D.val_rows;
  y.L = D.n_blocks;
  y.mh = D.meta_hidden;
  y.VE = D.precision == MFMG_PREC_BF16 ? 8 : 4;
  y.fused = D.fused_attention;
  y.remat = D.block_remat;
  y.eps = D.ln_eps;
  y.lr = D.sgd_lr;
  y.base = D.rope_base;
  long o = 0;
  const long d = y.d;
  y.emb = o;
  o += (long)y.V * d;
  for (int b = 0; b < y.L; ++b) {
    y.ln1g[b] = o; o += d;
    y.ln1b[b] = o; o += d;
    y.wqkv[b] = o; o += d * 3 * d;
    y.wo[b] = o; o += d * d;
    y.ln2g[b] = o; o += d;
    y.ln2b[b] = o; o += d;
    y.w1[b] = o; o += d * y.F;
    y.w2[b] = o; o += (long)y.F * d;
  }
  y.lnfg = o; o += d;
  y.lnfb = o; o += d;
  y.unemb = o; o += d * y.V;
  y.n = o;
  return y;
}

template <typename T>
struct Ops {  // operand copies of a parameter vector (theta_t or a tangent)
  T* W[MAXB][4];
  T* WT[MAXB][4];
  float* ln[MAXB][4];  // ln1 g, ln1 b, ln2 g, ln2 b
  float* lnf[2];
  T* U;
  T* UT;
  float* emb;
};

template <typename T>
void carve_ops(const Lay& y, Carver& c, Ops<T>& o) {
  for (int b = 0; b < y.L; ++b) {
    for (int m = 0; m < 4; ++m) {
      o.W[b][m] = c.take<T>((size_t)y.in(m) * y.ld(y.out(m)));
      o.WT[b][m] = c.take<T>((size_t)y.out(m) * y.ld(y.in(m)));
    }
    for (int k = 0; k < 4; ++k) o.ln[b][k] = c.take<float>(y.d);
  }
  o.lnf[0] = c.take<float>(y.d);
  o.lnf[1] = c.take<float>(y.d);
  o.U = c.take<T>((size_t)y.d * y.ld(y.V));
  o.UT = c.take<T>((size_t)y.V * y.ld(y.d));
  o.emb = c.take<float>((size_t)y.V * y.d);
}

// Sorted token positions and their segments for N tokens over a vocabulary of V.
TokenSegs carve_segs(Carver& c, long N, int V) {
  const long nsm = embed_segments_max((int)N);
  TokenSegs t;
  t.perm = c.take<int>(N);
  t.seg_start = c.take<int>(nsm + 1);
  t.seg_tok = c.take<int>(nsm);
  t.nseg = c.take<int>(1);
  t.tok2seg = c.take<int>(V);
  return t;
}

template <typename T>
struct Act {  // one inner step at up to maxB sequences (the dynamic memory)
  int *ids, *labels;
  float *h[2 * MAXB + 1], *hd[2 * MAXB + 1];
  float *xh1[MAXB], *xhd1[MAXB], *rs1[MAXB], *c1[MAXB];
  float *xh2[MAXB], *xhd2[MAXB], *rs2[MAXB], *c2[MAXB];
  float *xhf, *xhdf, *rsf, *cf;
  T *a1[MAXB], *a1T[MAXB], *a1d[MAXB], *a1dT[MAXB];
  T *a2[MAXB], *a2T[MAXB], *a2d[MAXB], *a2dT[MAXB];
  T *Q[MAXB], *QT[MAXB], *K[MAXB], *KT[MAXB], *Vv[MAXB], *VT[MAXB];
  T *Qd[MAXB], *QdT[MAXB], *Kd[MAXB], *KdT[MAXB], *Vd[MAXB], *VdT[MAXB];
  float *P32[MAXB], *Pd32[MAXB];                 // materialised attention only
  T *Pb[MAXB], *PbT[MAXB], *Pdb[MAXB], *PdbT[MAXB];
  float *lse[MAXB], *cst[MAXB], *ar, *ard;       // fused attention only: per query row
  T *O[MAXB], *OT[MAXB], *Od[MAXB], *OdT[MAXB];
  float *Z1[MAXB], *Z1d[MAXB];
  T *A1[MAXB], *A1T[MAXB], *A1d[MAXB], *A1dT[MAXB];
  T *af, *afT, *afd, *afdT;
  float *logits, *logitsd;
  float *y32, *yd32, *qkv32, *qkvd32;
  float *Qh, *Kh, *Vh, *Qdh, *Kdh, *Vdh;
  float *S32, *Sd32, *dS32, *dSd32;
  T *dS, *dST, *dSd, *dSdT;
  T *dz, *dzT, *dzd, *dzdT;
  float *dh, *dhd;
  T *dhb, *dhbT, *dhdb, *dhdbT;
  T *dZ1, *dZ1T, *dZ1d, *dZ1dT;
  T *dOh, *dOhT, *dOdh, *dOdhT;
  float *lnpart;
  TokenSegs ts;
  float* epart;
  float* skws;   // split-K workspace of the weight-gradient products
  long skws_n;
  float* loss_rows;
  float *cs, *sn;
};

template <typename T>
void carve_act(const Lay& y, Carver& c, Act<T>& a) {
  const long N = (long)y.maxB() * y.S, d = y.d, F = y.F, S = y.S;
  const long BH = (long)y.maxB() * y.H;
  const long hrow = (long)S * y.ld(y.dh), hcol = (long)y.dh * y.ld(S);  // per-head operand sizes
  auto F32 = [&](long n) { return c.take<float>(n); };
  auto OPT = [&](long n) { return c.take<T>(n); };
  a.ids = c.take<int>(N);
  a.labels = c.take<int>(N);
  // The residual stream: h[2b] enters block b, h[2b + 1] is its middle (after
  // attention), h[2L] enters the final LayerNorm.  With block rematerialisation
  // the block inputs are kept and one buffer holds every block's middle.
  for (int k = 0; k <= 2 * y.L; ++k) {
    if (y.remat && (k & 1) && k > 1) {
      a.h[k] = a.h[1];
      a.hd[k] = a.hd[1];
      continue;
    }
    a.h[k] = F32(N * d);
    a.hd[k] = F32(N * d);
  }
  // Per-block activations: one set per block, or with block rematerialisation
  // one set that every block's (re)computed forward fills in turn.
  for (int b = 0; b < y.L; ++b) {
    if (y.remat && b > 0) {
      a.xh1[b] = a.xh1[0]; a.xhd1[b] = a.xhd1[0]; a.rs1[b] = a.rs1[0]; a.c1[b] = a.c1[0];
      a.xh2[b] = a.xh2[0]; a.xhd2[b] = a.xhd2[0]; a.rs2[b] = a.rs2[0]; a.c2[b] = a.c2[0];
      a.a1[b] = a.a1[0]; a.a1T[b] = a.a1T[0]; a.a1d[b] = a.a1d[0]; a.a1dT[b] = a.a1dT[0];
      a.a2[b] = a.a2[0]; a.a2T[b] = a.a2T[0]; a.a2d[b] = a.a2d[0]; a.a2dT[b] = a.a2dT[0];
      a.Q[b] = a.Q[0]; a.QT[b] = a.QT[0]; a.K[b] = a.K[0]; a.KT[b] = a.KT[0];
      a.Vv[b] = a.Vv[0]; a.VT[b] = a.VT[0];
      a.Qd[b] = a.Qd[0]; a.QdT[b] = a.QdT[0]; a.Kd[b] = a.Kd[0]; a.KdT[b] = a.KdT[0];
      a.Vd[b] = a.Vd[0]; a.VdT[b] = a.VdT[0];
      a.P32[b] = a.P32[0]; a.Pd32[b] = a.Pd32[0];
      a.Pb[b] = a.Pb[0]; a.PbT[b] = a.PbT[0]; a.Pdb[b] = a.Pdb[0]; a.PdbT[b] = a.PdbT[0];
      a.lse[b] = a.lse[0]; a.cst[b] = a.cst[0];
      a.O[b] = a.O[0]; a.OT[b] = a.OT[0]; a.Od[b] = a.Od[0]; a.OdT[b] = a.OdT[0];
      a.Z1[b] = a.Z1[0]; a.Z1d[b] = a.Z1d[0];
      a.A1[b] = a.A1[0]; a.A1T[b] = a.A1T[0]; a.A1d[b] = a.A1d[0]; a.A1dT[b] = a.A1dT[0];
      continue;
    }
    a.xh1[b] = F32(N * d); a.xhd1[b] = F32(N * d); a.rs1[b] = F32(N); a.c1[b] = F32(N);
    a.xh2[b] = F32(N * d); a.xhd2[b] = F32(N * d); a.rs2[b] = F32(N); a.c2[b] = F32(N);
    a.a1[b] = OPT(N * y.ld(d)); a.a1T[b] = OPT(d * y.ld(N));
    a.a1d[b] = OPT(N * y.ld(d)); a.a1dT[b] = OPT(d * y.ld(N));
    a.a2[b] = OPT(N * y.ld(d)); a.a2T[b] = OPT(d * y.ld(N));
    a.a2d[b] = OPT(N * y.ld(d)); a.a2dT[b] = OPT(d * y.ld(N));
    a.Q[b] = OPT(BH * hrow); a.QT[b] = OPT(BH * hcol);
    a.K[b] = OPT(BH * hrow); a.KT[b] = OPT(BH * hcol);
    a.Vv[b] = OPT(BH * hrow); a.VT[b] = OPT(BH * hcol);
    a.Qd[b] = OPT(BH * hrow); a.QdT[b] = OPT(BH * hcol);
    a.Kd[b] = OPT(BH * hrow); a.KdT[b] = OPT(BH * hcol);
    a.Vd[b] = OPT(BH * hrow); a.VdT[b] = OPT(BH * hcol);
    if (y.fused) {
      a.P32[b] = a.Pd32[b] = nullptr;
      a.Pb[b] = a.PbT[b] = a.Pdb[b] = a.PdbT[b] = nullptr;
      a.lse[b] = F32(BH * S); a.cst[b] = F32(BH * S);
    } else {
      a.P32[b] = F32(BH * S * S); a.Pd32[b] = F32(BH * S * S);
      a.Pb[b] = OPT(BH * S * y.ld(S)); a.PbT[b] = OPT(BH * S * y.ld(S));
      a.Pdb[b] = OPT(BH * S * y.ld(S)); a.PdbT[b] = OPT(BH * S * y.ld(S));
      a.lse[b] = a.cst[b] = nullptr;
    }
    a.O[b] = OPT(N * y.ld(d)); a.OT[b] = OPT(d * y.ld(N));
    a.Od[b] = OPT(N * y.ld(d)); a.OdT[b] = OPT(d * y.ld(N));
    a.Z1[b] = F32(N * F); a.Z1d[b] = F32(N * F);
    a.A1[b] = OPT(N * y.ld(F)); a.A1T[b] = OPT(F * y.ld(N));
    a.A1d[b] = OPT(N * y.ld(F)); a.A1dT[b] = OPT(F * y.ld(N));
  }
  a.xhf = F32(N * d); a.xhdf = F32(N * d); a.rsf = F32(N); a.cf = F32(N);
  a.af = OPT(N * y.ld(d)); a.afT = OPT(d * y.ld(N));
  a.afd = OPT(N * y.ld(d)); a.afdT = OPT(d * y.ld(N));
  a.logits = F32(N * y.V); a.logitsd = F32(N * y.V);
  a.y32 = F32(N * std::max(d, F)); a.yd32 = F32(N * std::max(d, F));
  a.qkv32 = F32(N * 3 * d); a.qkvd32 = F32(N * 3 * d);
  a.Qh = F32(N * d); a.Kh = F32(N * d); a.Vh = F32(N * d);
  a.Qdh = F32(N * d); a.Kdh = F32(N * d); a.Vdh = F32(N * d);
  if (y.fused) {
    a.S32 = a.Sd32 = a.dS32 = a.dSd32 = nullptr;
    a.dS = a.dST = a.dSd = a.dSdT = nullptr;
    a.ar = F32(BH * S); a.ard = F32(BH * S);
  } else {
    a.S32 = F32(BH * S * S); a.Sd32 = F32(BH * S * S);
    a.dS32 = F32(BH * S * S); a.dSd32 = F32(BH * S * S);
    a.dS = OPT(BH * S * y.ld(S)); a.dST = OPT(BH * S * y.ld(S));
    a.dSd = OPT(BH * S * y.ld(S)); a.dSdT = OPT(BH * S * y.ld(S));
    a.ar = a.ard = nullptr;
  }
  a.dz = OPT(N * y.ld(y.V)); a.dzT = OPT((long)y.V * y.ld(N));
  a.dzd = OPT(N * y.ld(y.V)); a.dzdT = OPT((long)y.V * y.ld(N));
  a.dh = F32(N * d); a.dhd = F32(N * d);
  a.dhb = OPT(N * y.ld(d)); a.dhbT = OPT(d * y.ld(N));
  a.dhdb = OPT(N * y.ld(d)); a.dhdbT = OPT(d * y.ld(N));
  const long FQ = std::max(F, 3 * d);  // also holds the dqkv operands
  a.dZ1 = OPT(N * y.ld(FQ)); a.dZ1T = OPT(FQ * y.ld(N));
  a.dZ1d = OPT(N * y.ld(FQ)); a.dZ1dT = OPT(FQ * y.ld(N));
  a.dOh = OPT(BH * hrow); a.dOhT = OPT(BH * hcol);
  a.dOdh = OPT(BH * hrow); a.dOdhT = OPT(BH * hcol);
  a.lnpart = F32((long)ln_bwd_parts((int)N) * 4 * d);
  const long nsm = embed_segments_max((int)N);
  a.ts = carve_segs(c, N, y.V);
  a.epart = F32(nsm * 2 * d);
  a.skws_n = std::max({gemm_splitk_floats(F, d, (int)N), gemm_splitk_floats(d, F, (int)N),
                       gemm_splitk_floats(d, d, (int)N), gemm_splitk_floats(d, 3 * d, (int)N),
                       gemm_splitk_floats(d, y.V, (int)N)});
  a.skws = F32(a.skws_n);
  a.loss_rows = F32(N);
  a.cs = F32((long)S * y.dh / 2);
  a.sn = F32((long)S * y.dh / 2);
}

// Meta-model buffers for R token rows.
struct Meta {
  float *E, *ET, *W1T, *Z, *Hh, *HT, *u, *ubar, *dhid, *dhidT, *part;
  long rows;
};

void carve_meta(const Lay& y, Carver& c, Meta& m, long rows, bool vjp) {
  const long d = y.d, h = y.mh;
  const long ldr = rup(rows, 4);
  m.rows = rows;
  m.E = c.take<float>(rows * d);
  m.ET = vjp ? c.take<float>(d * ldr) : nullptr;
  m.W1T = c.take<float>(h * rup(d, 4));
  m.Z = c.take<float>(rows * h);
  m.Hh = c.take<float>(rows * h);
  m.HT = c.take<float>(h * ldr);
  m.u = c.take<float>(rows);
  m.ubar = vjp ? c.take<float>(rows) : nullptr;
  m.dhid = vjp ? c.take<float>(rows * h) : nullptr;
  m.dhidT = vjp ? c.take<float>(h * ldr) : nullptr;
  m.part = vjp ? c.take<float>((long)meta_vjp_parts((int)rows) * (2 * h + 1)) : nullptr;
}

template <typename T>
struct MetaPlanT {
  std::vector<Ops<T>> slot;
  std::vector<TokenSegs> segs;  // the training batches' sorted tokens, one per step
  Ops<T> v[2];
  float *run[2], *thetabar;
  Meta meta;
  Act<T> act;
  size_t st, dy, total;
};

template <typename T>
void plan_meta_t(const Lay& y, int T_, char* base, MetaPlanT<T>& p) {
  Carver c{base};
  p.slot.resize(T_ + 1);
  for (int t = 0; t <= T_; ++t) carve_ops(y, c, p.slot[t]);
  carve_ops(y, c, p.v[0]);
  carve_ops(y, c, p.v[1]);
  p.run[0] = c.take<float>(y.n);
  p.run[1] = c.take<float>(y.n);
  p.thetabar = c.take<float>(y.n);
  p.segs.resize(T_);
  for (int t = 0; t < T_; ++t) p.segs[t] = carve_segs(c, (long)y.Bt * y.S, y.V);
  carve_meta(y, c, p.meta, (long)T_ * y.Bt * y.S, true);
  p.st = c.off;
  carve_act(y, c, p.act);
  p.dy = c.off - p.st;
  p.total = c.off;
}

template <typename T>
struct StepPlanT {
  Ops<T> th, v;
  Meta meta;
  Act<T> act;
  size_t total;
};

template <typename T>
void plan_step_t(const Lay& y, char* base, StepPlanT<T>& p) {
  Carver c{base};
  carve_ops(y, c, p.th);
  carve_ops(y, c, p.v);
  carve_meta(y, c, p.meta, (long)y.Bt * y.S, false);
  carve_act(y, c, p.act);
  p.total = c.off;
}

#define HC(expr)                          \
  do {                                    \
    hipError_t e_ = (expr);               \
    if (e_ != hipSuccess) return e_;      \
  } while (0)

template <typename T>
struct TfEng {
  const Lay& y;
  const float* eta;
  hipStream_t s;

  // ---------------------------------------------------------------- helpers
  GemmOperands<T> op(const T* A, const T* Ad, const T* B, const T* Bd, int lda, int ldb, int M,
                     int N, int K) const {
    GemmOperands<T> o;
    o.A = A; o.Ad = Ad; o.B = B; o.Bd = Bd;
    o.lda = lda; o.ldb = ldb;
    o.M = M; o.N = N; o.K = K;
    return o;
  }
  // the split-K workspace for a weight-gradient product
  GemmOperands<T> wsk(GemmOperands<T> o, const Act<T>& a) const {
    o.ws = a.skws;
    o.ws_floats = a.skws_n;
    return o;
  }
  // Operands of block b's fused attention (bf16 only: the option is rejected
  // for float32 operands before any plan is made).
  AttnArgs attn_args(int b, int Bn, bool dual, const Act<T>& a) const {
    AttnArgs t;
    std::memset(&t, 0, sizeof(t));
    if constexpr (std::is_same<T, bf16_t>::value) {
      t.Q = a.Q[b]; t.K = a.K[b]; t.V = a.Vv[b]; t.QT = a.QT[b]; t.KT = a.KT[b]; t.VT = a.VT[b];
      if (dual) {
        t.Qd = a.Qd[b]; t.Kd = a.Kd[b]; t.Vd = a.Vd[b];
        t.QdT = a.QdT[b]; t.KdT = a.KdT[b]; t.VdT = a.VdT[b];
      }
      t.O = a.O[b]; t.OT = a.OT[b];
      t.Od = dual ? a.Od[b] : nullptr; t.OdT = dual ? a.OdT[b] : nullptr;
      t.dO = a.dOh; t.dOT = a.dOhT;
      t.dOd = dual ? a.dOdh : nullptr; t.dOdT = dual ? a.dOdhT : nullptr;
    }
    t.ldO = (int)y.ld(y.d);
    t.ldOT = (int)y.ld((long)Bn * y.S);
    t.lse = a.lse[b]; t.cst = a.cst[b]; t.r = a.ar; t.rd = a.ard;
    t.dQ = a.Qh; t.dK = a.Kh; t.dV = a.Vh; t.dQd = a.Qdh; t.dKd = a.Kdh; t.dVd = a.Vdh;
    t.S = y.S; t.H = y.H; t.BH = Bn * y.H; t.dh = y.dh; t.dual = dual;
    t.scale = 1.0f / std::sqrt((float)y.dh);
    return t;
  }
  static int fl(bool dual, bool ad = true) {
    return G_C1 | (dual ? (G_BD | (ad ? G_AD : 0)) : 0);
  }
  // Up to six matrices of one shape in one launch; jobs with a null source are skipped.
  struct Job {
    const float* src;
    T* dst;
    T* dstT;
  };
  hipError_t convs(std::initializer_list<Job> js, int rows, int cols, int batch = 1, long ss = 0,
                   long sd = 0, long sdT = 0) const {
    ConvJobs<T> J;
    for (const Job& j : js) {
      if (!j.src) continue;
      if (J.n == CONV_MAX_JOBS) return hipErrorInvalidValue;
      J.src[J.n] = j.src; J.dst[J.n] = j.dst; J.dstT[J.n] = j.dstT;
      ++J.n;
    }
    return convert_matrices<T>(J, rows, cols, cols, (int)y.ld(cols), (int)y.ld(rows), s, batch, ss,
                               sd, sdT);
  }
  // With bf16 operands, d a multiple of 256 and N (tokens) a multiple of 8 the
  // LayerNorm kernels write the bf16 operand rows themselves and a bf16
  // transpose makes the transposed copies; otherwise float32 rows are converted
  // to both layouts.
  bool ln_direct(int N) const {
    return std::is_same<T, bf16_t>::value && y.d % 256 == 0 && N % 8 == 0;
  }
  // A LayerNorm's output (and tangent) as operand rows [N][ld(d)] and transposes [d][ld(N)].
  hipError_t ln_operands(LnArgs ln, T* row, T* rowd, T* tr, T* trd) const {
    const bool dual = ln.dual;
    ln.yb = ln.ydb = nullptr;
    ln.ldb = 0;
    if constexpr (std::is_same<T, bf16_t>::value) {
      if (ln_direct(ln.N)) {
        ln.yb = row; ln.ydb = dual ? rowd : nullptr; ln.ldb = (int)y.ld(y.d);
        HC(ln_fwd(ln, s));
        return transpose_bf16(row, dual ? rowd : nullptr, ln.N, y.d, (int)y.ld(y.d), tr,
                              dual ? trd : nullptr, (int)y.ld(ln.N), s);
      }
    }
    HC(ln_fwd(ln, s));
    return convs({{ln.y, row, tr}, {dual ? ln.yd : nullptr, rowd, trd}}, ln.N, y.d);
  }
  // The residual-stream gradient dh (and tangent) as operands dhb, dhbT, right
  // after the LayerNorm backward that produced it.
  hipError_t dh_operands(int N, bool dual, const Act<T>& a) const {
    if constexpr (std::is_same<T, bf16_t>::value) {
      if (ln_direct(N))
        return transpose_bf16(a.dhb, dual ? a.dhdb : nullptr, N, y.d, (int)y.ld(y.d), a.dhbT,
                              dual ? a.dhdbT : nullptr, (int)y.ld(N), s);
    }
    return convs({{a.dh, a.dhb, a.dhbT}, {dual ? a.dhd : nullptr, a.dhdb, a.dhdbT}}, N, y.d);
  }
  hipError_t store(const GemmOperands<T>& o, int flags, float* C, float* Cd, int ldc, long sC,
                   float scale, bool dual) const {
    EpiStore e;
    e.C = C; e.Cd = Cd; e.ldc = ldc; e.sC = sC; e.scale = scale;
    e.M = o.M; e.N = o.N; e.dual = dual;
    return gemm_store<T>(o, flags, e, s);
  }

  hipError_t to_ops(const float* th, const Ops<T>& o) const {
    for (int b = 0; b < y.L; ++b) {
      for (int m = 0; m < 4; ++m)
        HC(convert_matrix<T>(th + y.woff(b, m), y.in(m), y.out(m), y.out(m), o.W[b][m],
                             (int)y.ld(y.out(m)), o.WT[b][m], (int)y.ld(y.in(m)), s));
      const long offs[4] = {y.ln1g[b], y.ln1b[b], y.ln2g[b], y.ln2b[b]};
      for (int k = 0; k < 4; ++k) HC(copy(th + offs[k], o.ln[b][k], y.d, s));
    }
    HC(copy(th + y.lnfg, o.lnf[0], y.d, s));
    HC(copy(th + y.lnfb, o.lnf[1], y.d, s));
    HC(convert_matrix<T>(th + y.unemb, y.d, y.V, y.V, o.U, (int)y.ld(y.V), o.UT, (int)y.ld(y.d), s));
    HC(copy(th + y.emb, o.emb, (long)y.V * y.d, s));
    return hipSuccess;
  }

  // ------------------------------------------------------------ meta-model
  // u = w2 . tanh(E W1 + b1) + b2 for the gathered embedding rows m.E.
  hipError_t meta_fwd(Meta& m, long rows) const {
    const int d = y.d, h = y.mh;
    const float* W1 = eta;
    const float* b1 = eta + (long)d * h;
    const float* w2 = b1 + h;
    const float* b2 = w2 + h;
    HC(convert_matrix<float>(W1, d, h, h, nullptr, 0, m.W1T, (int)rup(d, 4), s));
    GemmOperands<float> o;
    o.A = m.E; o.Ad = nullptr; o.B = m.W1T; o.Bd = nullptr;
    o.lda = d; o.ldb = (int)rup(d, 4);
    o.M = (int)rows; o.N = h; o.K = d;
    EpiActFwd<float> e;
    e.bias = b1; e.bias_d = nullptr; e.act = ACT_TANH; e.last = 0; e.dual = 0;
    e.M = (int)rows; e.N = h; e.Z = m.Z; e.Zd = nullptr;
    e.Ao = m.Hh; e.AoT = m.HT; e.Ado = nullptr; e.AdoT = nullptr;
    e.ldA = h; e.ldAT = (int)rup(rows, 4);
    HC(gemm_act_fwd<float>(o, G_C1, e, s));
    return meta_out(m.Hh, (int)rows, h, w2, b2, m.u, s);
  }

  // d eta of the meta-model from ubar (cotangents of u) over all rows.
  hipError_t meta_vjp_all(Meta& m, float* d_eta, const Act<T>& a) const {
    const int d = y.d, h = y.mh;
    const long rows = m.rows;
    const float* w2 = eta + (long)d * h + h;
    float* dW1 = d_eta;
    float* db1 = d_eta + (long)d * h;
    float* dw2 = db1 + h;
    float* db2 = dw2 + h;
    HC(meta_vjp(m.Hh, m.ubar, (int)rows, h, w2, m.dhid, m.part, dw2, db1, db2, s));
    HC(convert_matrix<float>(m.E, (int)rows, d, d, nullptr, 0, m.ET, (int)rup(rows, 4), s));
    HC(convert_matrix<float>(m.dhid, (int)rows, h, h, nullptr, 0, m.dhidT, (int)rup(rows, 4), s));
    GemmOperands<float> o;
    o.A = m.ET; o.Ad = nullptr; o.B = m.dhidT; o.Bd = nullptr;
    o.lda = o.ldb = (int)rup(rows, 4);
    o.M = d; o.N = h; o.K = (int)rows;
    o.ws = a.skws;  // split-K over the T x tokens rows
    o.ws_floats = a.skws_n;
    ParamArgs<float> P;
    std::memset(&P, 0, sizeof(P));
    P.mode = P_STORE_G;
    P.nin = d; P.nout = h; P.w_off = 0; P.b_off = -1;
    P.grad_out = dW1;
    return gemm_param<float>(o, G_C1, P, s);
  }

  // ------------------------------------------------------------ forward
  // Forward (dual when v) of Bn sequences through the decoder up to the logits.
  hipError_t forward(const Ops<T>& th, const Ops<T>* v, int Bn, const Act<T>& a) const {
    const bool dual = v != nullptr;
    const int d = y.d, N = Bn * y.S;
    HC(gather_rows(a.ids, N, d, th.emb, dual ? v->emb : nullptr, a.h[0], dual ? a.hd[0] : nullptr, s));
    for (int b = 0; b < y.L; ++b) HC(block_forward(th, v, Bn, b, true, a));
    // final LayerNorm -> af, logits = af U
    LnArgs ln;
    ln.x = a.h[2 * y.L]; ln.xd = a.hd[2 * y.L];
    ln.g = th.lnf[0]; ln.b = th.lnf[1];
    ln.gd = dual ? v->lnf[0] : nullptr; ln.bd = dual ? v->lnf[1] : nullptr;
    ln.y = a.y32; ln.yd = a.yd32; ln.xh = a.xhf; ln.xhd = a.xhdf; ln.rstd = a.rsf; ln.c = a.cf;
    ln.N = N; ln.d = d; ln.dual = dual; ln.eps = y.eps;
    HC(ln_operands(ln, a.af, a.afd, a.afT, a.afdT));
    HC(store(op(a.af, dual ? a.afd : nullptr, th.UT, dual ? v->UT : nullptr, (int)y.ld(d),
                (int)y.ld(d), N, y.V, d),
             fl(dual), a.logits, a.logitsd, y.V, 0, 1.0f, dual));
    return hipSuccess;
  }

  // Block b's forward from its input h[2b] (and tangent): everything its
  // backward reads, and with `output` also the block's output h[2b + 2] (the
  // rematerialising pass before the block's backward skips that last product).
  hipError_t block_forward(const Ops<T>& th, const Ops<T>* v, int Bn, int b, bool output,
                           const Act<T>& a) const {
    const bool dual = v != nullptr;
    const int d = y.d, S = y.S, H = y.H, dh = y.dh, F = y.F;
    const int N = Bn * S, BH = Bn * H;
    const long hrow = (long)S * y.ld(dh), hcol = (long)dh * y.ld(S), pS = (long)S * y.ld(S);
    const float scale = 1.0f / std::sqrt((float)dh);
    {
      // LayerNorm 1 -> a1
      LnArgs ln;
      ln.x = a.h[2 * b]; ln.xd = a.hd[2 * b];
      ln.g = th.ln[b][0]; ln.b = th.ln[b][1];
      ln.gd = dual ? v->ln[b][0] : nullptr; ln.bd = dual ? v->ln[b][1] : nullptr;
      ln.y = a.y32; ln.yd = a.yd32; ln.xh = a.xh1[b]; ln.xhd = a.xhd1[b];
      ln.rstd = a.rs1[b]; ln.c = a.c1[b]; ln.N = N; ln.d = d; ln.dual = dual; ln.eps = y.eps;
      HC(ln_operands(ln, a.a1[b], a.a1d[b], a.a1T[b], a.a1dT[b]));
      // qkv = a1 Wqkv
      HC(store(op(a.a1[b], dual ? a.a1d[b] : nullptr, th.WT[b][0], dual ? v->WT[b][0] : nullptr,
                  (int)y.ld(d), (int)y.ld(d), N, 3 * d, d),
               fl(dual), a.qkv32, a.qkvd32, 3 * d, 0, 1.0f, dual));
      RopeArgs r;
      std::memset(&r, 0, sizeof(r));
      r.qkv = a.qkv32; r.qkvd = a.qkvd32;
      r.Q = a.Qh; r.K = a.Kh; r.V = a.Vh; r.Qd = a.Qdh; r.Kd = a.Kdh; r.Vd = a.Vdh;
      r.cs = a.cs; r.sn = a.sn; r.N = N; r.S = S; r.H = H; r.dh = dh; r.dual = dual;
      // per-head operands: bf16 rows straight from the split and batched bf16
      // transposes (S a multiple of 8), or float32 per-head rows converted
      bool qdirect = false;
      if constexpr (std::is_same<T, bf16_t>::value) {
        if (S % 8 == 0) {
          qdirect = true;
          r.Qb = a.Q[b]; r.Kb = a.K[b]; r.Vb = a.Vv[b];
          if (dual) { r.Qdb = a.Qd[b]; r.Kdb = a.Kd[b]; r.Vdb = a.Vd[b]; }
        }
      }
      HC(rope_split(r, s));
      const long sh = (long)S * dh;
      if (qdirect) {
        if constexpr (std::is_same<T, bf16_t>::value) {
          TrJobs J;
          auto add = [&](const bf16_t* src, bf16_t* dst) {
            J.src[J.n] = src; J.dst[J.n] = dst; ++J.n;
          };
          add(a.Q[b], a.QT[b]); add(a.K[b], a.KT[b]); add(a.Vv[b], a.VT[b]);
          if (dual) { add(a.Qd[b], a.QdT[b]); add(a.Kd[b], a.KdT[b]); add(a.Vd[b], a.VdT[b]); }
          HC(transpose_bf16_jobs(J, BH, S, dh, (int)y.ld(dh), (int)y.ld(S), hrow, hcol, s));
        }
      } else {
        HC(convs({{a.Qh, a.Q[b], a.QT[b]}, {a.Kh, a.K[b], a.KT[b]}, {a.Vh, a.Vv[b], a.VT[b]},
                  {dual ? a.Qdh : nullptr, a.Qd[b], a.QdT[b]},
                  {dual ? a.Kdh : nullptr, a.Kd[b], a.KdT[b]},
                  {dual ? a.Vdh : nullptr, a.Vd[b], a.VdT[b]}},
                 S, dh, BH, sh, hrow, hcol));
      }
      if (y.fused) {
        HC(attn_fwd(attn_args(b, Bn, dual, a), s));
      } else {
        // scores S = scale Q K^T (per head), softmax
        {
          GemmOperands<T> o = op(a.Q[b], dual ? a.Qd[b] : nullptr, a.K[b], dual ? a.Kd[b] : nullptr,
                                 (int)y.ld(dh), (int)y.ld(dh), S, S, dh);
          o.batch = BH; o.sA = hrow; o.sB = hrow;
          HC(store(o, fl(dual), a.S32, a.Sd32, S, (long)S * S, scale, dual));
        }
        SoftmaxArgs sm;
        std::memset(&sm, 0, sizeof(sm));
        sm.Sc = a.S32; sm.Scd = a.Sd32; sm.P = a.P32[b]; sm.Pd = a.Pd32[b];
        sm.rows = (long)BH * S; sm.S = S; sm.dual = dual;
        HC(softmax_fwd(sm, s));
        HC(convs({{a.P32[b], a.Pb[b], a.PbT[b]}, {dual ? a.Pd32[b] : nullptr, a.Pdb[b], a.PdbT[b]}},
                 S, S, BH, (long)S * S, pS, pS));
        // O = P V (per head) -> token-major operands
        {
          GemmOperands<T> o = op(a.Pb[b], dual ? a.Pdb[b] : nullptr, a.VT[b], dual ? a.VdT[b] : nullptr,
                                 (int)y.ld(S), (int)y.ld(S), S, dh, S);
          o.batch = BH; o.sA = pS; o.sB = hcol;
          EpiHeadMerge<T> e;
          e.O = a.O[b]; e.OT = a.OT[b]; e.Od = a.Od[b]; e.OdT = a.OdT[b];
          e.ldO = (int)y.ld(d); e.ldOT = (int)y.ld(N);
          e.seq = S; e.heads = H; e.dh = dh; e.M = S; e.N = dh; e.dual = dual;
          HC(gemm_head_merge<T>(o, fl(dual), e, s));
        }
      }
      // h_mid = h + O Wo
      {
        EpiResid e;
        e.H = a.h[2 * b]; e.Hd = a.hd[2 * b]; e.Ho = a.h[2 * b + 1]; e.Hdo = a.hd[2 * b + 1];
        e.M = N; e.N = d; e.dual = dual;
        HC(gemm_resid<T>(op(a.O[b], dual ? a.Od[b] : nullptr, th.WT[b][1], dual ? v->WT[b][1] : nullptr,
                            (int)y.ld(d), (int)y.ld(d), N, d, d),
                         fl(dual), e, s));
      }
      // LayerNorm 2 -> a2
      ln.x = a.h[2 * b + 1]; ln.xd = a.hd[2 * b + 1];
      ln.g = th.ln[b][2]; ln.b = th.ln[b][3];
      ln.gd = dual ? v->ln[b][2] : nullptr; ln.bd = dual ? v->ln[b][3] : nullptr;
      ln.xh = a.xh2[b]; ln.xhd = a.xhd2[b]; ln.rstd = a.rs2[b]; ln.c = a.c2[b];
      HC(ln_operands(ln, a.a2[b], a.a2d[b], a.a2T[b], a.a2dT[b]));
      // A1 = GELU(a2 W1)
      {
        EpiActFwd<T> e;
        e.bias = nullptr; e.bias_d = nullptr; e.act = ACT_GELU; e.last = 0; e.dual = dual;
        e.M = N; e.N = F; e.Z = a.Z1[b]; e.Zd = a.Z1d[b];
        e.Ao = a.A1[b]; e.AoT = a.A1T[b]; e.Ado = a.A1d[b]; e.AdoT = a.A1dT[b];
        e.ldA = (int)y.ld(F); e.ldAT = (int)y.ld(N);
        HC(gemm_act_fwd<T>(op(a.a2[b], dual ? a.a2d[b] : nullptr, th.WT[b][2], dual ? v->WT[b][2] : nullptr,
                              (int)y.ld(d), (int)y.ld(d), N, F, d),
                           fl(dual), e, s));
      }
      // h_out = h_mid + A1 W2
      if (output) {
        EpiResid e;
        e.H = a.h[2 * b + 1]; e.Hd = a.hd[2 * b + 1]; e.Ho = a.h[2 * b + 2]; e.Hdo = a.hd[2 * b + 2];
        e.M = N; e.N = d; e.dual = dual;
        HC(gemm_resid<T>(op(a.A1[b], dual ? a.A1d[b] : nullptr, th.WT[b][3], dual ? v->WT[b][3] : nullptr,
                            (int)y.ld(F), (int)y.ld(F), N, d, F),
                         fl(dual), e, s));
      }
    }
    return hipSuccess;
  }

  hipError_t head(int Bn, bool dual, const float* u, float* mvp, float* ubar,
                  const Act<T>& a) const {
    const int N = Bn * y.S;
    LossArgs<T> la;
    la.loss = MFMG_LOSS_CE; la.rows = N; la.C = y.V; la.dual = dual; la.inv_n = 1.0f / N;
    la.Z = a.logits; la.Zd = a.logitsd; la.labels = a.labels; la.targets = nullptr;
    la.alpha_logits = u;
    la.d = a.dz; la.dT = a.dzT; la.dd = a.dzd; la.ddT = a.dzdT;
    la.ld = (int)y.ld(y.V); la.ldT = (int)y.ld(N); la.pad_to = y.V;
    la.loss_rows = a.loss_rows; la.mvp_rows = mvp; la.deta_rows = ubar;
    return loss_head<T>(la, s);
  }

  // ------------------------------------------------------------ backward
  // out: operand copies to write from the parameter epilogue (or null).
  // segs: where the batch's sorted tokens go (null: the step workspace's);
  // sorted: they are already there (the same batch was sorted by an earlier pass).
  hipError_t backward(const Ops<T>& th, const Ops<T>* v, int Bn, ParamArgs<T> P,
                      const Ops<T>* out, const Act<T>& a, const TokenSegs* segs = nullptr,
                      bool sorted = false) const {
    const bool dual = v != nullptr;
    const int d = y.d, S = y.S, H = y.H, dh = y.dh, F = y.F;
    const int N = Bn * S, BH = Bn * H;
    const long hrow = (long)S * y.ld(dh), hcol = (long)dh * y.ld(S), pS = (long)S * y.ld(S);
    const float scale = 1.0f / std::sqrt((float)dh);
    auto matP = [&](long woff, int nin, int nout, T* oW, T* oWT) {
      ParamArgs<T> Q = P;
      Q.nin = nin; Q.nout = nout; Q.w_off = woff; Q.b_off = -1;
      Q.ldW = (int)y.ld(nout); Q.ldWT = (int)y.ld(nin);
      Q.outW = oW; Q.outWT = oWT; Q.outb = nullptr;
      return Q;
    };
    auto ln_bwd_call = [&](const float* dy, const float* dyd, const float* xh, const float* xhd,
                           const float* rs, const float* c, const float* g, const float* gd,
                           const float* dh_in, const float* dhd_in, long goff, long boff,
                           float* og, float* ob) {
      LnBwdArgs l;
      l.dy = dy; l.dyd = dyd; l.xh = xh; l.xhd = xhd; l.rstd = rs; l.c = c; l.g = g; l.gd = gd;
      l.dh_in = dh_in; l.dhd_in = dhd_in; l.dh_out = a.dh; l.dhd_out = a.dhd;
      l.partial = a.lnpart; l.N = N; l.d = d; l.dual = dual;
      l.hb = l.hdb = nullptr;
      l.ldb = 0;
      if constexpr (std::is_same<T, bf16_t>::value) {
        if (ln_direct(N)) {
          l.hb = a.dhb; l.hdb = dual ? a.dhdb : nullptr; l.ldb = (int)y.ld(d);
        }
      }
      return ln_bwd<T>(l, goff, boff, P, og, ob, s);
    };
    // unembedding
    HC(gemm_param<T>(wsk(op(a.afT, dual ? a.afdT : nullptr, a.dzT, dual ? a.dzdT : nullptr,
                        (int)y.ld(N), (int)y.ld(N), d, y.V, N), a),
                     fl(dual), matP(y.unemb, d, y.V, out ? out->U : nullptr, out ? out->UT : nullptr), s));
    HC(store(op(a.dz, dual ? a.dzd : nullptr, th.U, dual ? v->U : nullptr, (int)y.ld(y.V),
                (int)y.ld(y.V), N, d, y.V),
             fl(dual), a.y32, a.yd32, d, 0, 1.0f, dual));
    HC(ln_bwd_call(a.y32, a.yd32, a.xhf, a.xhdf, a.rsf, a.cf, th.lnf[0], dual ? v->lnf[0] : nullptr,
                   nullptr, nullptr, y.lnfg, y.lnfb, out ? out->lnf[0] : nullptr,
                   out ? out->lnf[1] : nullptr));
    for (int b = y.L - 1; b >= 0; --b) {
      // block rematerialisation: the shared buffers hold the last block's
      // activations from the forward; every other block is recomputed from its
      // input h[2b] before its backward
      if (y.remat && b < y.L - 1) HC(block_forward(th, v, Bn, b, false, a));
      // ---- MLP: h_out = h_mid + GELU(a2 W1) W2
      HC(dh_operands(N, dual, a));
      HC(gemm_param<T>(wsk(op(a.A1T[b], dual ? a.A1dT[b] : nullptr, a.dhbT, dual ? a.dhdbT : nullptr,
                          (int)y.ld(N), (int)y.ld(N), F, d, N), a),
                       fl(dual), matP(y.w2[b], F, d, out ? out->W[b][3] : nullptr, out ? out->WT[b][3] : nullptr), s));
      {
        EpiActBwd<T> e;
        e.Zp = a.Z1[b]; e.Zdp = a.Z1d[b]; e.Ap = nullptr; e.ldAp = 0;
        e.act = ACT_GELU; e.dual = dual; e.M = N; e.N = F;
        e.dZ = a.dZ1; e.dZT = a.dZ1T; e.dZd = a.dZ1d; e.dZdT = a.dZ1dT;
        e.ld = (int)y.ld(F); e.ldT = (int)y.ld(N);
        HC(gemm_act_bwd<T>(op(a.dhb, dual ? a.dhdb : nullptr, th.W[b][3], dual ? v->W[b][3] : nullptr,
                              (int)y.ld(d), (int)y.ld(d), N, F, d),
                           fl(dual), e, s));
      }
      HC(gemm_param<T>(wsk(op(a.a2T[b], dual ? a.a2dT[b] : nullptr, a.dZ1T, dual ? a.dZ1dT : nullptr,
                          (int)y.ld(N), (int)y.ld(N), d, F, N), a),
                       fl(dual), matP(y.w1[b], d, F, out ? out->W[b][2] : nullptr, out ? out->WT[b][2] : nullptr), s));
      HC(store(op(a.dZ1, dual ? a.dZ1d : nullptr, th.W[b][2], dual ? v->W[b][2] : nullptr,
                  (int)y.ld(F), (int)y.ld(F), N, d, F),
               fl(dual), a.y32, a.yd32, d, 0, 1.0f, dual));
      HC(ln_bwd_call(a.y32, a.yd32, a.xh2[b], a.xhd2[b], a.rs2[b], a.c2[b], th.ln[b][2],
                     dual ? v->ln[b][2] : nullptr, a.dh, dual ? a.dhd : nullptr, y.ln2g[b], y.ln2b[b],
                     out ? out->ln[b][2] : nullptr, out ? out->ln[b][3] : nullptr));
      // ---- attention: h_mid = h + Attn(LN1(h)) Wo
      HC(dh_operands(N, dual, a));
      HC(gemm_param<T>(wsk(op(a.OT[b], dual ? a.OdT[b] : nullptr, a.dhbT, dual ? a.dhdbT : nullptr,
                          (int)y.ld(N), (int)y.ld(N), d, d, N), a),
                       fl(dual), matP(y.wo[b], d, d, out ? out->W[b][1] : nullptr, out ? out->WT[b][1] : nullptr), s));
      {
        EpiHeadSplit<T> e;
        e.Oh = a.dOh; e.OhT = a.dOhT; e.Odh = a.dOdh; e.OdhT = a.dOdhT;
        e.ldh = (int)y.ld(dh); e.ldhT = (int)y.ld(S);
        e.seq = S; e.heads = H; e.dh = dh; e.M = N; e.N = d; e.dual = dual;
        HC(gemm_head_split<T>(op(a.dhb, dual ? a.dhdb : nullptr, th.W[b][1], dual ? v->W[b][1] : nullptr,
                                 (int)y.ld(d), (int)y.ld(d), N, d, d),
                              fl(dual), e, s));
      }
      if (y.fused) {
        HC(attn_bwd(attn_args(b, Bn, dual, a), s));
      } else {
        {  // dP = dO V^T
          GemmOperands<T> o = op(a.dOh, dual ? a.dOdh : nullptr, a.Vv[b], dual ? a.Vd[b] : nullptr,
                                 (int)y.ld(dh), (int)y.ld(dh), S, S, dh);
          o.batch = BH; o.sA = hrow; o.sB = hrow;
          HC(store(o, fl(dual), a.S32, a.Sd32, S, (long)S * S, 1.0f, dual));
        }
        {  // dV = P^T dO
          GemmOperands<T> o = op(a.PbT[b], dual ? a.PdbT[b] : nullptr, a.dOhT, dual ? a.dOdhT : nullptr,
                                 (int)y.ld(S), (int)y.ld(S), S, dh, S);
          o.batch = BH; o.sA = pS; o.sB = hcol;
          HC(store(o, fl(dual), a.Vh, a.Vdh, dh, (long)S * dh, 1.0f, dual));
        }
        SoftmaxArgs sm;
        std::memset(&sm, 0, sizeof(sm));
        sm.P = a.P32[b]; sm.Pd = a.Pd32[b]; sm.dP = a.S32; sm.dPd = a.Sd32;
        sm.dS = a.dS32; sm.dSd = a.dSd32; sm.rows = (long)BH * S; sm.S = S; sm.dual = dual;
        sm.scale = scale;
        HC(softmax_bwd(sm, s));
        HC(convs({{a.dS32, a.dS, a.dST}, {dual ? a.dSd32 : nullptr, a.dSd, a.dSdT}}, S, S, BH,
                 (long)S * S, pS, pS));
        {  // dQ = dS K
          GemmOperands<T> o = op(a.dS, dual ? a.dSd : nullptr, a.KT[b], dual ? a.KdT[b] : nullptr,
                                 (int)y.ld(S), (int)y.ld(S), S, dh, S);
          o.batch = BH; o.sA = pS; o.sB = hcol;
          HC(store(o, fl(dual), a.Qh, a.Qdh, dh, (long)S * dh, 1.0f, dual));
        }
        {  // dK = dS^T Q
          GemmOperands<T> o = op(a.dST, dual ? a.dSdT : nullptr, a.QT[b], dual ? a.QdT[b] : nullptr,
                                 (int)y.ld(S), (int)y.ld(S), S, dh, S);
          o.batch = BH; o.sA = pS; o.sB = hcol;
          HC(store(o, fl(dual), a.Kh, a.Kdh, dh, (long)S * dh, 1.0f, dual));
        }
      }
      RopeArgs r;
      std::memset(&r, 0, sizeof(r));
      r.Q = a.Qh; r.K = a.Kh; r.V = a.Vh; r.Qd = a.Qdh; r.Kd = a.Kdh; r.Vd = a.Vdh;
      r.qkv_out = a.qkv32; r.qkvd_out = a.qkvd32;
      r.cs = a.cs; r.sn = a.sn; r.N = N; r.S = S; r.H = H; r.dh = dh; r.dual = dual;
      // dqkv operands in the dZ1 buffers (sized for max(F, 3d)): bf16 rows
      // straight from the merge and a bf16 transpose, or float32 rows converted
      bool direct = false;
      if constexpr (std::is_same<T, bf16_t>::value) {
        if (N % 8 == 0) {
          direct = true;
          r.ob = a.dZ1; r.odb = dual ? a.dZ1d : nullptr; r.ldb = (int)y.ld(3 * d);
        }
      }
      HC(rope_merge(r, s));
      if (direct) {
        if constexpr (std::is_same<T, bf16_t>::value)
          HC(transpose_bf16(a.dZ1, dual ? a.dZ1d : nullptr, N, 3 * d, (int)y.ld(3 * d), a.dZ1T,
                            dual ? a.dZ1dT : nullptr, (int)y.ld(N), s));
      } else {
        HC(convs({{a.qkv32, a.dZ1, a.dZ1T}, {dual ? a.qkvd32 : nullptr, a.dZ1d, a.dZ1dT}}, N,
                 3 * d));
      }
      HC(gemm_param<T>(wsk(op(a.a1T[b], dual ? a.a1dT[b] : nullptr, a.dZ1T, dual ? a.dZ1dT : nullptr,
                          (int)y.ld(N), (int)y.ld(N), d, 3 * d, N), a),
                       fl(dual), matP(y.wqkv[b], d, 3 * d, out ? out->W[b][0] : nullptr, out ? out->WT[b][0] : nullptr), s));
      HC(store(op(a.dZ1, dual ? a.dZ1d : nullptr, th.W[b][0], dual ? v->W[b][0] : nullptr,
                  (int)y.ld(3 * d), (int)y.ld(3 * d), N, d, 3 * d),
               fl(dual), a.y32, a.yd32, d, 0, 1.0f, dual));
      HC(ln_bwd_call(a.y32, a.yd32, a.xh1[b], a.xhd1[b], a.rs1[b], a.c1[b], th.ln[b][0],
                     dual ? v->ln[b][0] : nullptr, a.dh, dual ? a.dhd : nullptr, y.ln1g[b], y.ln1b[b],
                     out ? out->ln[b][0] : nullptr, out ? out->ln[b][1] : nullptr));
    }
    // embedding rows
    const TokenSegs& ts = segs ? *segs : a.ts;
    if (!(segs && sorted)) HC(sort_tokens(a.ids, N, y.V, ts, s));
    EmbedGradArgs eg;
    eg.dh = a.dh; eg.dhd = dual ? a.dhd : nullptr; eg.ts = ts; eg.part = a.epart;
    eg.emb_off = y.emb; eg.outE = out ? out->emb : nullptr;
    eg.V = y.V; eg.d = d; eg.N = N;
    return embed_grad<T>(eg, P, s);
  }
};

template <typename T>
ParamArgs<T> pbase(const Lay& y, int mode, const float* eta) {
  ParamArgs<T> P;
  std::memset(&P, 0, sizeof(P));
  P.mode = mode;
  P.eta = eta;
  P.lr = y.lr;
  P.k1 = P.k2 = 1.0f;
  return P;
}

template <typename T>
hipError_t run_meta_t(const Lay& y, const float* theta0, const float* eta,
                      const mfmg_batch* batches, int T_, const mfmg_batch* val, float* d_eta,
                      float* val_loss, char* ws, hipStream_t s) {
  MetaPlanT<T> p;
  plan_meta_t(y, T_, ws, p);
  TfEng<T> E{y, eta, s};
  const Act<T>& a = p.act;
  const int Nt = y.Bt * y.S;
  HC(rope_table(y.S, y.dh, y.base, a.cs, a.sn, s));
  HC(E.to_ops(theta0, p.slot[0]));
  // meta-model inputs: rows of the initial embedding table at every step's tokens
  for (int t = 0; t < T_; ++t) {
    HC(split_tokens(static_cast<const int*>(batches[t].x), y.Bt, y.S, y.V, a.ids, a.labels, s));
    HC(gather_rows(a.ids, Nt, y.d, theta0 + y.emb, nullptr, p.meta.E + (long)t * Nt * y.d, nullptr, s));
  }
  HC(E.meta_fwd(p.meta, (long)T_ * Nt));
  // forward unroll
  for (int t = 0; t < T_; ++t) {
    HC(split_tokens(static_cast<const int*>(batches[t].x), y.Bt, y.S, y.V, a.ids, a.labels, s));
    HC(E.forward(p.slot[t], nullptr, y.Bt, a));
    HC(E.head(y.Bt, false, p.meta.u + (long)t * Nt, nullptr, nullptr, a));
    ParamArgs<T> P = pbase<T>(y, P_UPD_SGD_FIXED, eta);
    P.theta = t == 0 ? theta0 : p.run[(t - 1) & 1];
    P.theta_next = p.run[t & 1];
    HC(E.backward(p.slot[t], nullptr, y.Bt, P, &p.slot[t + 1], a, &p.segs[t], false));
  }
  // outer loss and seed
  {
    const int Nv = y.Bv * y.S;
    HC(split_tokens(static_cast<const int*>(val->x), y.Bv, y.S, y.V, a.ids, a.labels, s));
    HC(E.forward(p.slot[T_], nullptr, y.Bv, a));
    HC(E.head(y.Bv, false, nullptr, nullptr, nullptr, a));
    if (val_loss) HC(loss_reduce(a.loss_rows, nullptr, Nv, 1.0f / Nv, val_loss, s));
    ParamArgs<T> P = pbase<T>(y, P_SEED_SGD_FIXED, eta);
    P.thetabar = p.thetabar;
    HC(E.backward(p.slot[T_], nullptr, y.Bv, P, &p.v[0], a));
  }
  // reverse sweep
  int vc = 0;
  for (int i = T_ - 1; i >= 0; --i) {
    HC(split_tokens(static_cast<const int*>(batches[i].x), y.Bt, y.S, y.V, a.ids, a.labels, s));
    HC(E.forward(p.slot[i], &p.v[vc], y.Bt, a));
    HC(E.head(y.Bt, true, p.meta.u + (long)i * Nt, nullptr, p.meta.ubar + (long)i * Nt, a));
    ParamArgs<T> P = pbase<T>(y, P_REV_SGD_FIXED, eta);
    P.thetabar = p.thetabar;
    HC(E.backward(p.slot[i], &p.v[vc], y.Bt, P, i > 0 ? &p.v[vc ^ 1] : nullptr, a, &p.segs[i],
                  true));
    vc ^= 1;
  }
  return E.meta_vjp_all(p.meta, d_eta, p.act);
}

template <typename T>
hipError_t meta_alpha_step(const Lay& y, TfEng<T>& E, const float* theta, Meta& m,
                           const Act<T>& a) {
  const int N = y.Bt * y.S;
  HC(gather_rows(a.ids, N, y.d, theta + y.emb, nullptr, m.E, nullptr, E.s));
  return E.meta_fwd(m, N);
}

template <typename T>
hipError_t run_inner_t(const Lay& y, const float* theta, const float* eta, const mfmg_batch* b,
                       float* theta_next, float* grad_out, float* loss_out, char* ws,
                       hipStream_t s) {
  StepPlanT<T> p;
  plan_step_t(y, ws, p);
  TfEng<T> E{y, eta, s};
  const Act<T>& a = p.act;
  const int N = y.Bt * y.S;
  HC(rope_table(y.S, y.dh, y.base, a.cs, a.sn, s));
  HC(E.to_ops(theta, p.th));
  HC(split_tokens(static_cast<const int*>(b->x), y.Bt, y.S, y.V, a.ids, a.labels, s));
  HC(meta_alpha_step(y, E, theta, p.meta, a));
  HC(E.forward(p.th, nullptr, y.Bt, a));
  HC(E.head(y.Bt, false, p.meta.u, nullptr, nullptr, a));
  if (loss_out) HC(loss_reduce(a.loss_rows, p.meta.u, N, 1.0f / N, loss_out, s));
  ParamArgs<T> P = pbase<T>(y, P_UPD_SGD_FIXED, eta);
  P.theta = theta;
  P.theta_next = theta_next;
  P.grad_out = grad_out;
  return E.backward(p.th, nullptr, y.Bt, P, nullptr, a);
}

template <typename T>
hipError_t run_hvp_t(const Lay& y, const float* theta, const float* eta, const mfmg_batch* b,
                     const float* v, float* grad_out, float* hvp_out, float* mvp_out, char* ws,
                     hipStream_t s) {
  StepPlanT<T> p;
  plan_step_t(y, ws, p);
  TfEng<T> E{y, eta, s};
  const Act<T>& a = p.act;
  HC(rope_table(y.S, y.dh, y.base, a.cs, a.sn, s));
  HC(E.to_ops(theta, p.th));
  HC(E.to_ops(v, p.v));
  HC(split_tokens(static_cast<const int*>(b->x), y.Bt, y.S, y.V, a.ids, a.labels, s));
  HC(meta_alpha_step(y, E, theta, p.meta, a));
  HC(E.forward(p.th, &p.v, y.Bt, a));
  HC(E.head(y.Bt, true, p.meta.u, mvp_out, nullptr, a));
  ParamArgs<T> P = pbase<T>(y, P_HVP, eta);
  P.grad_out = grad_out;
  P.hvp_out = hvp_out;
  return E.backward(p.th, &p.v, y.Bt, P, nullptr, a);
}

}  // namespace

const char* tf_validate(const mfmg_problem_desc& D) {
  if (D.meta != MFMG_META_TOKEN_WEIGHT_MLP)
    return "transformer problems are implemented with the token-weight meta-model";
  if (D.optimizer != MFMG_OPT_SGD) return "transformer problems are implemented for SGD";
  if (D.loss != MFMG_LOSS_CE) return "transformer problems use next-token cross-entropy";
  if (D.precision != MFMG_PREC_FP32 && D.precision != MFMG_PREC_BF16) return "unknown precision";
  if (D.n_blocks < 1 || D.n_blocks > MAXB) return "n_blocks outside [1, 16]";
  if (D.n_heads < 1 || D.d_model < 8 || D.d_model % D.n_heads) return "bad d_model / n_heads";
  const int dh = D.d_model / D.n_heads;
  if (D.d_model % 8 || dh % 8 || D.d_ff % 8 || D.d_model > LN_MAX_D)
    return "d_model, d_ff and the head dim must be multiples of 8 (d_model <= 1024)";
  if (D.vocab < 2 || D.vocab > (1 << 24)) return "vocab outside [2, 2^24]";
  if (D.seq < 4 || D.seq % 4) return "seq must be a positive multiple of 4";
  if (D.rows < 1 || D.val_rows < 1) return "rows and val_rows must be >= 1";
  if (!sort_tokens_fits(D.rows * D.seq) || !sort_tokens_fits(D.val_rows * D.seq))
    return "rows * seq (and val_rows * seq) must be <= 8192 tokens";
  if (D.meta_hidden < 8 || D.meta_hidden % 8 || D.meta_hidden > META_MAX_HIDDEN)
    return "meta_hidden must be a multiple of 8 in [8, 256]";
  if (!(D.ln_eps > 0.f) || !(D.rope_base > 0.f) || !std::isfinite(D.sgd_lr))
    return "ln_eps and rope_base must be > 0, sgd_lr finite";
  if (D.fused_attention != 0 && D.fused_attention != 1) return "fused_attention must be 0 or 1";
  if (D.block_remat != 0 && D.block_remat != 1) return "block_remat must be 0 or 1";
  if (D.fused_attention &&
      (D.precision != MFMG_PREC_BF16 || !attn_fused_supported(D.seq, dh)))
    return "fused attention needs bf16 operands, head dim 64 and seq a multiple of 64";
  return nullptr;
}

long tf_n_theta(const mfmg_problem_desc& d) { return make_lay(d).n; }

long tf_n_eta(const mfmg_problem_desc& d) {
  return (long)d.d_model * d.meta_hidden + 2L * d.meta_hidden + 1;
}

size_t tf_meta_ws(const mfmg_problem_desc& d, int T, size_t* st, size_t* dy) {
  const Lay y = make_lay(d);
  if (d.precision == MFMG_PREC_BF16) {
    MetaPlanT<bf16_t> p;
    plan_meta_t(y, T, nullptr, p);
    *st = p.st; *dy = p.dy;
    return p.total;
  }
  MetaPlanT<float> p;
  plan_meta_t(y, T, nullptr, p);
  *st = p.st; *dy = p.dy;
  return p.total;
}

size_t tf_step_ws(const mfmg_problem_desc& d) {
  const Lay y = make_lay(d);
  if (d.precision == MFMG_PREC_BF16) {
    StepPlanT<bf16_t> p;
    plan_step_t(y, nullptr, p);
    return p.total;
  }
  StepPlanT<float> p;
  plan_step_t(y, nullptr, p);
  return p.total;
}

hipError_t tf_run_meta(const mfmg_problem_desc& d, const float* theta0, const float* eta,
                       const mfmg_batch* batches, int T, const mfmg_batch* val, float* d_eta,
                       float* val_loss, char* ws, hipStream_t s) {
  const Lay y = make_lay(d);
  if (d.precision == MFMG_PREC_BF16)
    return run_meta_t<bf16_t>(y, theta0, eta, batches, T, val, d_eta, val_loss, ws, s);
  return run_meta_t<float>(y, theta0, eta, batches, T, val, d_eta, val_loss, ws, s);
}

hipError_t tf_run_inner(const mfmg_problem_desc& d, const float* theta, const float* eta,
                        const mfmg_batch* b, float* theta_next, float* grad_out, float* loss_out,
                        char* ws, hipStream_t s) {
  const Lay y = make_lay(d);
  if (d.precision == MFMG_PREC_BF16)
    return run_inner_t<bf16_t>(y, theta, eta, b, theta_next, grad_out, loss_out, ws, s);
  return run_inner_t<float>(y, theta, eta, b, theta_next, grad_out, loss_out, ws, s);
}

hipError_t tf_run_hvp(const mfmg_problem_desc& d, const float* theta, const float* eta,
                      const mfmg_batch* b, const float* v, float* grad_out, float* hvp_out,
                      float* mvp_out, char* ws, hipStream_t s) {
  const Lay y = make_lay(d);
  if (d.precision == MFMG_PREC_BF16)
    return run_hvp_t<bf16_t>(y, theta, eta, b, v, grad_out, hvp_out, mvp_out, ws, s);
  return run_hvp_t<float>(y, theta, eta, b, v, grad_out, hvp_out, mvp_out, ws, s);
}

}  // namespace mfmg
