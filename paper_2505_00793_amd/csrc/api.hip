// C ABI front end: argument validation, workspace planning and the
// orchestration of the meta-gradient (Algorithm 2 with per-inner-step
// checkpointing, Section 4) on one HIP stream.
//
// meta_grad on an MLP:
//   prologue        theta_0 -> operand copies (slot 0)
//   forward unroll  t = 0..T-1: forward, loss head, backward-data, and
//                   backward-weight GEMMs whose epilogue applies the inner
//                   update and writes slot t+1 (theta_{t+1} operand copies;
//                   Adam also m, v and the inner gradient g_t)
//   seed            forward/backward of V at theta_T: bar theta_T = dV/dtheta_T
//                   (eq. dVdmeta), and for SGD the first tangent v
//   reverse sweep   i = T-1..0: (Adam: optimiser VJP -> tangent v) dual
//                   forward, dual loss head, dual backward whose weight
//                   epilogue adds H v to bar theta and accumulates d eta
//                   (eq. bptt_recur with eq. vhp_to_hvp / eq. vmp_to_mvp)
// No host synchronisation happens inside a call.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "kernels.h"
#include "mfmg.h"
#include "tf_engine.h"

using namespace mfmg;

namespace {

thread_local std::string g_err;

mfmg_status fail(mfmg_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define HIPCHK(expr)                                                                 \
  do {                                                                               \
    hipError_t e_ = (expr);                                                          \
    if (e_ != hipSuccess) return fail(MFMG_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

inline long rup(long x, long m) { return (x + m - 1) / m * m; }

// Bump allocator over the caller's workspace; with base == nullptr it measures.
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

}  // namespace

struct mfmg_problem {
  mfmg_problem_desc d;
  bool tf;  // transformer kind (tf_engine)
  int L;
  int w[MFMG_MAX_LAYERS + 1];
  long w_off[MFMG_MAX_LAYERS];
  long b_off[MFMG_MAX_LAYERS];
  long n_theta;
  int VE;  // operand elements per 16 bytes
  long ld(long x) const { return rup(x, VE); }
  bool bf16() const { return d.precision == MFMG_PREC_BF16; }
  bool adam() const { return d.optimizer == MFMG_OPT_ADAM; }
  bool linreg_path(int T) const {
    return L == 1 && w[1] == 1 && !d.has_bias && d.loss == MFMG_LOSS_MSE &&
           d.optimizer == MFMG_OPT_SGD && d.meta == MFMG_META_LOGLR_PER_PARAM &&
           d.precision == MFMG_PREC_FP32 && linreg_fits(T, d.rows, d.val_rows, w[0]);
  }
  int maxR() const { return d.rows > d.val_rows ? d.rows : d.val_rows; }
  // Contraction of the last layer's backward-data product (over its outputs):
  // with bf16 operands the width rounded up to 8, so that the product takes the
  // direct-to-LDS path; the loss head writes the padding columns of dZ as zero
  // and zero_last_pads clears those of the W copies.
  int k_last() const {
    const int c = w[L];
    return bf16() && L >= 2 && c % 8 != 0 ? (c + 7) / 8 * 8 : c;
  }
};

namespace {

// ------------------------------------------------------------------------------------
// Workspace layout
// ------------------------------------------------------------------------------------
template <typename T>
struct OperandSet {  // operand copies of one parameter vector (theta_t or a tangent)
  T* W[MFMG_MAX_LAYERS];   // [in][ld(out)]  (B operand of backward-data)
  T* WT[MFMG_MAX_LAYERS];  // [out][ld(in)]  (B operand of forward)
  float* b[MFMG_MAX_LAYERS];
};

template <typename T>
struct Act {  // one inner step's activations, up to R rows (the dynamic memory)
  T* X;
  T* XT;
  float* Z[MFMG_MAX_LAYERS];
  float* Zd[MFMG_MAX_LAYERS];
  T* A[MFMG_MAX_LAYERS];
  T* AT[MFMG_MAX_LAYERS];
  T* Ad[MFMG_MAX_LAYERS];
  T* AdT[MFMG_MAX_LAYERS];
  T* dZ[2];
  T* dZT[2];
  T* dZd[2];
  T* dZdT[2];
  float* loss_rows;
  float* skws;   // split-K partial sums of the float32 forward products (or null)
  long skws_n;
};

template <typename T>
void carve_opset(const mfmg_problem* p, Carver& c, OperandSet<T>& o) {
  for (int l = 0; l < p->L; ++l) {
    const int nin = p->w[l], nout = p->w[l + 1];
    o.W[l] = c.take<T>((size_t)nin * p->ld(nout));
    o.WT[l] = c.take<T>((size_t)nout * p->ld(nin));
    o.b[l] = p->d.has_bias ? c.take<float>(nout) : nullptr;
  }
}

template <typename T>
void carve_act(const mfmg_problem* p, Carver& c, Act<T>& a, int R, bool dual) {
  const int L = p->L;
  a.X = c.take<T>((size_t)R * p->ld(p->w[0]));
  a.XT = c.take<T>((size_t)p->w[0] * p->ld(R));
  int maxw = 1;
  // ReLU hidden layers keep no pre-activations: the backward reads the sign of
  // their activations instead
  const bool relu = p->d.act == MFMG_ACT_RELU;
  for (int l = 0; l < L; ++l) {
    const int nout = p->w[l + 1];
    if (nout > maxw) maxw = nout;
    const bool keep_z = !relu || l == L - 1;
    a.Z[l] = keep_z ? c.take<float>((size_t)R * nout) : nullptr;
    a.Zd[l] = (dual && keep_z) ? c.take<float>((size_t)R * nout) : nullptr;
    a.A[l] = a.AT[l] = a.Ad[l] = a.AdT[l] = nullptr;
    if (l < L - 1) {
      a.A[l] = c.take<T>((size_t)R * p->ld(nout));
      a.AT[l] = c.take<T>((size_t)nout * p->ld(R));
      if (dual) {
        a.Ad[l] = c.take<T>((size_t)R * p->ld(nout));
        a.AdT[l] = c.take<T>((size_t)nout * p->ld(R));
      }
    }
  }
  for (int k = 0; k < 2; ++k) {
    a.dZ[k] = c.take<T>((size_t)R * p->ld(maxw));
    a.dZT[k] = c.take<T>((size_t)maxw * p->ld(R));
    a.dZd[k] = dual ? c.take<T>((size_t)R * p->ld(maxw)) : nullptr;
    a.dZdT[k] = dual ? c.take<T>((size_t)maxw * p->ld(R)) : nullptr;
  }
  a.loss_rows = c.take<float>(R);
  // float32 forward products with few output tiles and a long k run split-K
  long ws = 0;
  if (!p->bf16()) {
    for (int l = 0; l < L; ++l) {
      ws = std::max(ws, gemm_splitk_fwd_f32_floats(p->d.rows, p->w[l + 1], p->w[l]));
      ws = std::max(ws, gemm_splitk_fwd_f32_floats(p->d.val_rows, p->w[l + 1], p->w[l]));
    }
  }
  a.skws_n = ws;
  a.skws = ws > 0 ? c.take<float>(ws) : nullptr;
}

template <typename T>
struct MetaPlan {
  int seg;                          // 0, or the segment length k of recomputed checkpoints
  std::vector<OperandSet<T>> slot;  // T + 1 operand checkpoints, or a ring of k + 1
  std::vector<float*> ck;           // segments: theta_{s k} (float32), s = 1 .. ceil(T/k) - 1
  std::vector<float*> ckm, ckv;     // segments, Adam: m_{s k}, v_{s k}
  float* run[2];                    // SGD: theta_{t+1} (float32), ping-pong
  float* thetabar;
  OperandSet<T> v[2];               // tangent operand copies, ping-pong
  // Adam checkpoints: theta_t, m_t, v_t (t = 0..T) and g_t (t < T); with
  // segments a ring of k + 1 states and k gradients (see the *_at helpers)
  std::vector<float*> th, m, vv, g;
  float* mbar;
  float* vbar;
  float* partial;
  int part_off[MFMG_MAX_LAYERS + 1];
  Act<T> act;
  float* linreg_scratch;
  size_t static_bytes, dynamic_bytes, total;
};

// Blocks of the Adam reverse kernel for layer l: 16 x 64 tiles of W, then 256
// bias entries per block (the kernel's launcher checks the count against this).
int adam_blocks(const mfmg_problem* p, int l) {
  const long tiles = (long)((p->w[l] + 15) / 16) * ((p->w[l + 1] + 63) / 64);
  return (int)(tiles + (p->d.has_bias ? (p->w[l + 1] + 255) / 256 : 0));
}

// Segment length of the recomputed checkpoints for T inner steps (0: every
// step's state is kept).
int seg_of(const mfmg_problem* p, int T) {
  const int k = p->d.ckpt_segment;
  return (k > 0 && k < T) ? k : 0;
}

template <typename T>
void plan_meta(const mfmg_problem* p, int T_, char* base, MetaPlan<T>& mp) {
  Carver c{base};
  mp.linreg_scratch = nullptr;
  if (p->linreg_path(T_)) {
    mp.linreg_scratch = c.take<float>((size_t)(T_ + 1) * p->w[0]);
    mp.static_bytes = c.off;
    mp.dynamic_bytes = 0;
    mp.total = c.off;
    return;
  }
  const size_t n = p->n_theta;
  mp.seg = seg_of(p, T_);
  const int nslot = mp.seg ? mp.seg + 1 : T_ + 1;
  mp.slot.resize(nslot);
  for (int t = 0; t < nslot; ++t) carve_opset(p, c, mp.slot[t]);
  mp.ck.clear();
  mp.ckm.clear();
  mp.ckv.clear();
  if (mp.seg) {
    const int nseg = (T_ + mp.seg - 1) / mp.seg;
    mp.ck.assign(nseg, nullptr);
    for (int q = 1; q < nseg; ++q) mp.ck[q] = c.take<float>(n);
    if (p->adam()) {
      mp.ckm.assign(nseg, nullptr);
      mp.ckv.assign(nseg, nullptr);
      for (int q = 1; q < nseg; ++q) {
        mp.ckm[q] = c.take<float>(n);
        mp.ckv[q] = c.take<float>(n);
      }
    }
  }
  mp.run[0] = mp.run[1] = nullptr;
  if (!p->adam()) {
    mp.run[0] = c.take<float>(n);
    mp.run[1] = c.take<float>(n);
  }
  mp.thetabar = c.take<float>(n);
  carve_opset(p, c, mp.v[0]);
  if (!p->adam()) carve_opset(p, c, mp.v[1]);
  mp.mbar = mp.vbar = mp.partial = nullptr;
  if (p->adam()) {
    // states t = 0..T (theta_0 is the caller's), or a ring of k + 1 states and
    // k gradients with segments
    const int ns = mp.seg ? mp.seg + 1 : T_ + 1;
    const int ng = mp.seg ? mp.seg : T_;
    mp.th.assign(ns, nullptr);
    mp.m.assign(ns, nullptr);
    mp.vv.assign(ns, nullptr);
    mp.g.assign(ng, nullptr);
    for (int t = mp.seg ? 0 : 1; t < ns; ++t) mp.th[t] = c.take<float>(n);
    for (int t = 0; t < ns; ++t) {
      mp.m[t] = c.take<float>(n);
      mp.vv[t] = c.take<float>(n);
    }
    for (int t = 0; t < ng; ++t) mp.g[t] = c.take<float>(n);
    mp.mbar = c.take<float>(n);
    mp.vbar = c.take<float>(n);
    int off = 0;
    for (int l = 0; l < p->L; ++l) {
      mp.part_off[l] = off;
      off += adam_blocks(p, l);
    }
    mp.part_off[p->L] = off;
    mp.partial = c.take<float>(2 * (size_t)off);
  }
  mp.static_bytes = c.off;
  carve_act(p, c, mp.act, p->maxR(), true);
  mp.dynamic_bytes = c.off - mp.static_bytes;
  mp.total = c.off;
}

template <typename T>
struct StepPlan {
  OperandSet<T> th;
  OperandSet<T> v;
  Act<T> act;
  size_t total;
};

template <typename T>
void plan_step(const mfmg_problem* p, char* base, StepPlan<T>& sp) {
  Carver c{base};
  carve_opset(p, c, sp.th);
  carve_opset(p, c, sp.v);
  carve_act(p, c, sp.act, p->maxR(), true);
  sp.total = c.off;
}

size_t meta_ws_bytes(const mfmg_problem* p, int T, size_t* st, size_t* dy) {
  if (p->bf16()) {
    MetaPlan<bf16_t> mp;
    plan_meta(p, T, nullptr, mp);
    *st = mp.static_bytes;
    *dy = mp.dynamic_bytes;
    return mp.total;
  }
  MetaPlan<float> mp;
  plan_meta(p, T, nullptr, mp);
  *st = mp.static_bytes;
  *dy = mp.dynamic_bytes;
  return mp.total;
}

size_t step_ws_bytes(const mfmg_problem* p) {
  if (p->bf16()) {
    StepPlan<bf16_t> sp;
    plan_step(p, nullptr, sp);
    return sp.total;
  }
  StepPlan<float> sp;
  plan_step(p, nullptr, sp);
  return sp.total;
}

// ------------------------------------------------------------------------------------
// Engine: one pass of each kind over the MLP
// ------------------------------------------------------------------------------------
struct TimingScope {
  int cls;
  hipStream_t s;
  TimingScope(int c, hipStream_t st) : cls(c), s(st) { timing_begin(cls, s); }
  ~TimingScope() { timing_end(cls, s); }
};

template <typename T>
struct Eng {
  const mfmg_problem* p;
  hipStream_t s;

  mfmg_status to_ops(const float* theta, const OperandSet<T>& o) {
    for (int l = 0; l < p->L; ++l) {
      const int nin = p->w[l], nout = p->w[l + 1];
      TimingScope ts(7, s);
      HIPCHK(convert_matrix<T>(theta + p->w_off[l], nin, nout, nout, o.W[l], (int)p->ld(nout),
                               o.WT[l], (int)p->ld(nin), s));
      if (p->d.has_bias) HIPCHK(copy(theta + p->b_off[l], o.b[l], nout, s));
    }
    return MFMG_OK;
  }

  mfmg_status load_x(const float* x, int R, const Act<T>& a) {
    TimingScope ts(7, s);
    HIPCHK(convert_matrix<T>(x, R, p->w[0], p->w[0], a.X, (int)p->ld(p->w[0]), a.XT,
                             (int)p->ld(R), s));
    return MFMG_OK;
  }

  mfmg_status forward(const OperandSet<T>& th, const OperandSet<T>* v, int R, const Act<T>& a) {
    const bool dual = v != nullptr;
    for (int l = 0; l < p->L; ++l) {
      const int nin = p->w[l], nout = p->w[l + 1];
      GemmOperands<T> op;
      op.A = l == 0 ? a.X : a.A[l - 1];
      op.Ad = (dual && l > 0) ? a.Ad[l - 1] : nullptr;
      op.B = th.WT[l];
      op.Bd = dual ? v->WT[l] : nullptr;
      op.lda = op.ldb = (int)p->ld(nin);
      op.M = R;
      op.N = nout;
      op.K = nin;
      op.ws = a.skws;
      op.ws_floats = a.skws_n;
      const int flags = G_C1 | (dual ? (G_BD | (l > 0 ? G_AD : 0)) : 0);
      EpiActFwd<T> e;
      e.bias = th.b[l];
      e.bias_d = dual ? v->b[l] : nullptr;
      e.act = p->d.act;
      e.last = l == p->L - 1;
      e.dual = dual;
      e.M = R;
      e.N = nout;
      e.Z = a.Z[l];
      e.Zd = a.Zd[l];
      e.Ao = a.A[l];
      e.AoT = a.AT[l];
      e.Ado = a.Ad[l];
      e.AdoT = a.AdT[l];
      e.ldA = (int)p->ld(nout);
      e.ldAT = (int)p->ld(R);
      TimingScope ts(dual ? 3 : 0, s);
      HIPCHK(gemm_act_fwd<T>(op, flags, e, s));
    }
    return MFMG_OK;
  }

  mfmg_status head(const mfmg_batch& b, int R, bool dual, const float* alpha_logits,
                   float* mvp_rows, float* deta_rows, const Act<T>& a) {
    const int C = p->w[p->L];
    LossArgs<T> la;
    la.loss = p->d.loss;
    la.map_M = p->d.map_steps;
    la.rows = R;
    la.C = C;
    la.dual = dual;
    la.inv_n = 1.0f / (float)R;
    la.Z = a.Z[p->L - 1];
    la.Zd = a.Zd[p->L - 1];
    la.labels = p->d.loss == MFMG_LOSS_CE ? static_cast<const int*>(b.y) : nullptr;
    la.targets = p->d.loss != MFMG_LOSS_CE ? static_cast<const float*>(b.y) : nullptr;
    la.alpha_logits = alpha_logits;
    la.d = a.dZ[0];
    la.dT = a.dZT[0];
    la.dd = a.dZd[0];
    la.ddT = a.dZdT[0];
    la.ld = (int)p->ld(C);
    la.ldT = (int)p->ld(R);
    la.pad_to = p->k_last();
    la.loss_rows = a.loss_rows;
    la.mvp_rows = mvp_rows;
    la.deta_rows = deta_rows;
    TimingScope ts(6, s);
    HIPCHK(loss_head<T>(la, s));
    return MFMG_OK;
  }

  // Backward over layers L-1..0.  set_out(P, l) fills the operand-copy outputs.
  template <class F>
  mfmg_status backward(const OperandSet<T>& th, const OperandSet<T>* v, int R, bool need_c1,
                       ParamArgs<T> P, F set_out, const Act<T>& a) {
    const bool dual = v != nullptr;
    int cur = 0;
    for (int l = p->L - 1; l >= 0; --l) {
      const int nin = p->w[l], nout = p->w[l + 1];
      P.layer = l;
      P.n_layers = p->L;
      P.nin = nin;
      P.nout = nout;
      P.w_off = p->w_off[l];
      P.b_off = p->b_off[l];
      P.ldW = (int)p->ld(nout);
      P.ldWT = (int)p->ld(nin);
      set_out(P, l);
      // backward-weight product G = A^T dZ (and its tangent), parameter epilogue
      GemmOperands<T> opw;
      opw.A = l == 0 ? a.XT : a.AT[l - 1];
      opw.Ad = (dual && l > 0) ? a.AdT[l - 1] : nullptr;
      opw.B = a.dZT[cur];
      opw.Bd = dual ? a.dZdT[cur] : nullptr;
      opw.lda = opw.ldb = (int)p->ld(R);
      opw.M = nin;
      opw.N = nout;
      opw.K = R;
      const int flags_w = (need_c1 ? G_C1 : 0) | (dual ? (G_BD | (l > 0 ? G_AD : 0)) : 0);
      // backward-data product dA = dZ W^T (and its tangent), activation epilogue
      GemmOperands<T> opd;
      EpiActBwd<T> e;
      const int flags_d = G_C1 | (dual ? (G_AD | G_BD) : 0);
      if (l > 0) {
        opd.A = a.dZ[cur];
        opd.Ad = dual ? a.dZd[cur] : nullptr;
        opd.B = th.W[l];
        opd.Bd = dual ? v->W[l] : nullptr;
        opd.lda = opd.ldb = (int)p->ld(nout);
        opd.M = R;
        opd.N = nin;
        opd.K = l == p->L - 1 ? p->k_last() : nout;
        e.Zp = a.Z[l - 1];
        e.Zdp = a.Zd[l - 1];
        e.Ap = a.A[l - 1];
        e.ldAp = (int)p->ld(nin);
        e.act = p->d.act;
        e.dual = dual;
        e.M = R;
        e.N = nin;
        e.dZ = a.dZ[cur ^ 1];
        e.dZT = a.dZT[cur ^ 1];
        e.dZd = a.dZd[cur ^ 1];
        e.dZdT = a.dZdT[cur ^ 1];
        e.ld = (int)p->ld(nin);
        e.ldT = (int)p->ld(R);
      }
      // the bias entries: summed by the backward-weight GEMM itself unless it
      // runs split-K, else by a reduction over dZ^T
      P.fuse_bias = p->d.has_bias && gemm_fuses_bias<T>(opw, flags_w) ? 1 : 0;
      // the two products are independent: small ones share one launch
      const bool paired = l > 0 && gemm_pairs<T>(opw, flags_w, opd, flags_d);
      if (paired) {
        TimingScope ts(dual ? 8 : 2, s);
        HIPCHK(gemm_param_and_act_bwd<T>(opw, flags_w, P, opd, flags_d, e, s));
      } else {
        TimingScope ts(dual ? (flags_w == (G_C1 | G_AD | G_BD) ? 8 : 5) : 2, s);
        HIPCHK(gemm_param<T>(opw, flags_w, P, s));
      }
      if (p->d.has_bias && !P.fuse_bias) {
        TimingScope ts(7, s);
        HIPCHK(bias_reduce<T>(a.dZT[cur], dual ? a.dZdT[cur] : nullptr, (int)p->ld(R), R, P, s));
      }
      if (l > 0) {
        if (!paired) {
          TimingScope ts(dual ? 4 : 1, s);
          HIPCHK(gemm_act_bwd<T>(opd, flags_d, e, s));
        }
        cur ^= 1;
      }
    }
    return MFMG_OK;
  }
};

#define TRY(expr)                        \
  do {                                   \
    mfmg_status st_ = (expr);            \
    if (st_ != MFMG_OK) return st_;      \
  } while (0)

// Columns w[L] .. k_last() - 1 of the last layer's W copies (the B operand of
// its backward-data product) set to zero in every operand set of a call;
// nothing else writes there, so they stay zero for the whole call.
template <typename T>
mfmg_status zero_last_pads(const mfmg_problem* p, const std::vector<const OperandSet<T>*>& sets,
                           hipStream_t s) {
  const int l = p->L - 1, nout = p->w[p->L], kp = p->k_last();
  if (kp == nout) return MFMG_OK;
  ZeroColJobs J;
  J.n = 0;
  for (const OperandSet<T>* o : sets) {
    if (!o || !o->W[l]) continue;
    if (J.n == ZC_MAX_JOBS) {
      HIPCHK(zero_cols(J, s));
      J.n = 0;
    }
    J.p[J.n] = reinterpret_cast<uint16_t*>(o->W[l]);
    J.rows[J.n] = p->w[l];
    J.ld[J.n] = (int)p->ld(nout);
    J.c0[J.n] = nout;
    J.c1[J.n] = kp;
    ++J.n;
  }
  if (J.n) HIPCHK(zero_cols(J, s));
  return MFMG_OK;
}

template <typename T>
ParamArgs<T> param_base(const mfmg_problem* p, int mode, const float* eta) {
  ParamArgs<T> P;
  std::memset(&P, 0, sizeof(P));
  P.mode = mode;
  P.eta = eta;
  P.lr = p->d.sgd_lr;
  P.b1 = p->d.adam_b1;
  P.b2 = p->d.adam_b2;
  P.eps = p->d.adam_eps;
  P.k1 = P.k2 = 1.0f;
  return P;
}

void bias_corr(const mfmg_problem* p, int step, float* k1, float* k2) {
  *k1 = (float)(1.0 - std::pow((double)p->d.adam_b1, step + 1));
  *k2 = (float)(1.0 - std::pow((double)p->d.adam_b2, step + 1));
}

int mode_of(const mfmg_problem* p, int phase) {  // phase 0 update, 1 seed, 2 reverse
  if (p->adam()) return phase == 0 ? P_UPD_ADAM : phase == 1 ? P_SEED_ADAM : P_REV_ADAM;
  if (p->d.meta == MFMG_META_LOGLR_PER_PARAM)
    return phase == 0 ? P_UPD_SGD_PP : phase == 1 ? P_SEED_SGD_PP : P_REV_SGD_PP;
  return phase == 0 ? P_UPD_SGD_FIXED : phase == 1 ? P_SEED_SGD_FIXED : P_REV_SGD_FIXED;
}

template <typename T>
mfmg_status run_meta(const mfmg_problem* p, const float* theta0, const float* opt0,
                     const float* eta, const mfmg_batch* batches, int T_, const mfmg_batch* val,
                     float* d_eta, float* val_loss, char* ws, hipStream_t s) {
  MetaPlan<T> mp;
  plan_meta(p, T_, ws, mp);
  Eng<T> E{p, s};
  const Act<T>& a = mp.act;
  {
    std::vector<const OperandSet<T>*> sets;
    for (const OperandSet<T>& o : mp.slot) sets.push_back(&o);
    sets.push_back(&mp.v[0]);
    if (!p->adam()) sets.push_back(&mp.v[1]);
    TRY(zero_last_pads<T>(p, sets, s));
  }
  const bool adam = p->adam();
  const bool wlog = p->d.meta == MFMG_META_EXAMPLE_WEIGHT_LOGITS;
  const bool maml = p->d.meta == MFMG_META_MAML;
  const int R = p->d.rows;
  const long n = p->n_theta;
  if (maml) theta0 = eta;   // the meta-parameters are the starting point

  // Operand checkpoint of theta_t: slot t, or with segments the ring entry
  // t mod (k + 1), which holds one segment's states plus theta_T at once.
  // Adam's float32 states (theta_t, m_t, v_t) use the same ring, its saved
  // gradients g_t the ring t mod k.
  const int k = mp.seg;
  auto sl = [&](int t) -> const OperandSet<T>& { return mp.slot[k ? t % (k + 1) : t]; };
  auto st_of = [&](int t) { return k ? t % (k + 1) : t; };
  auto th_at = [&](int t) -> float* {
    return t == 0 ? const_cast<float*>(theta0) : mp.th[st_of(t)];
  };
  auto g_at = [&](int t) -> float* { return mp.g[k ? t % k : t]; };
  // Adam: m_0, v_0 into state t (the optimiser state at the start)
  auto adam_init = [&](int t) -> mfmg_status {
    if (opt0) {
      HIPCHK(copy(opt0, mp.m[st_of(t)], n, s));
      HIPCHK(copy(opt0 + n, mp.vv[st_of(t)], n, s));
    } else {
      HIPCHK(fill(mp.m[st_of(t)], n, 0.0f, s));
      HIPCHK(fill(mp.vv[st_of(t)], n, 0.0f, s));
    }
    return MFMG_OK;
  };

  // prologue
  TRY(E.to_ops(theta0, sl(0)));
  if (adam) TRY(adam_init(0));

  // One forward inner step t from the float32 theta_t at th: the update writes
  // theta_{t+1} to th_next and its operand copies to checkpoint t + 1.
  auto fwd_step = [&](int t, const float* th, float* th_next) -> mfmg_status {
    TRY(E.load_x(static_cast<const float*>(batches[t].x), R, a));
    TRY(E.forward(sl(t), nullptr, R, a));
    const float* alpha = wlog ? eta + (long)t * R : nullptr;
    TRY(E.head(batches[t], R, false, alpha, nullptr, nullptr, a));
    ParamArgs<T> P = param_base<T>(p, mode_of(p, 0), eta);
    if (adam) {
      P.theta = th_at(t);
      P.theta_next = th_at(t + 1);
      P.m_in = mp.m[st_of(t)];
      P.v_in = mp.vv[st_of(t)];
      P.m_out = mp.m[st_of(t + 1)];
      P.v_out = mp.vv[st_of(t + 1)];
      P.g_save = g_at(t);
      bias_corr(p, t, &P.k1, &P.k2);
    } else {
      P.theta = th;
      P.theta_next = th_next;
    }
    const OperandSet<T>& nxt = sl(t + 1);
    TRY(E.backward(sl(t), nullptr, R, true, P,
                   [&](ParamArgs<T>& Q, int l) {
                     Q.outW = nxt.W[l];
                     Q.outWT = nxt.WT[l];
                     Q.outb = nxt.b[l];
                   },
                   a));
    return MFMG_OK;
  };
  // SGD keeps theta in the run ping-pong; with segments theta at a segment
  // start goes to its float32 checkpoint instead.
  auto other = [&](const float* th) { return th == mp.run[0] ? mp.run[1] : mp.run[0]; };

  // forward unroll with checkpoints (with segments, Adam copies the state at
  // each segment start out of the ring)
  {
    const float* th = theta0;
    for (int t = 0; t < T_; ++t) {
      float* nx = nullptr;
      if (!adam) nx = (k && (t + 1) % k == 0 && t + 1 < T_) ? mp.ck[(t + 1) / k] : other(th);
      TRY(fwd_step(t, th, nx));
      th = nx;
      if (adam && k && (t + 1) % k == 0 && t + 1 < T_) {
        const int q = (t + 1) / k, r = st_of(t + 1);
        HIPCHK(copy(mp.th[r], mp.ck[q], n, s));
        HIPCHK(copy(mp.m[r], mp.ckm[q], n, s));
        HIPCHK(copy(mp.vv[r], mp.ckv[q], n, s));
      }
    }
  }

  // outer loss V at theta_T and its gradient: the seed of the reverse sweep
  {
    const int Rv = p->d.val_rows;
    TRY(E.load_x(static_cast<const float*>(val->x), Rv, a));
    TRY(E.forward(sl(T_), nullptr, Rv, a));
    TRY(E.head(*val, Rv, false, nullptr, nullptr, nullptr, a));
    if (val_loss) HIPCHK(loss_reduce(a.loss_rows, nullptr, Rv, 1.0f / (float)Rv, val_loss, s));
    ParamArgs<T> P = param_base<T>(p, mode_of(p, 1), eta);
    P.thetabar = mp.thetabar;
    const OperandSet<T>& v0 = mp.v[0];
    TRY(E.backward(sl(T_), nullptr, Rv, true, P,
                   [&](ParamArgs<T>& Q, int l) {
                     if (!adam) {
                       Q.outW = v0.W[l];
                       Q.outWT = v0.WT[l];
                       Q.outb = v0.b[l];
                     }
                   },
                   a));
  }

  // reverse sweep
  int vc = 0;
  for (int i = T_ - 1; i >= 0; --i) {
    const bool first = i == T_ - 1;
    // entering a segment other than the last: recompute theta_{s0} .. theta_i
    // from the segment's float32 checkpoint (the same kernels on the same
    // inputs, so the operand copies are bit-identical to the unroll's)
    if (k && (i + 1) % k == 0 && i + 1 < T_) {
      const int s0 = i + 1 - k;
      if (adam) {
        // the segment's start state back into the ring, then its steps s0..i
        // (step i too: its inner gradient is read before the dual pass)
        if (s0 == 0) {
          TRY(adam_init(0));
        } else {
          const int r = st_of(s0), q = s0 / k;
          HIPCHK(copy(mp.ck[q], mp.th[r], n, s));
          HIPCHK(copy(mp.ckm[q], mp.m[r], n, s));
          HIPCHK(copy(mp.ckv[q], mp.vv[r], n, s));
        }
        TRY(E.to_ops(th_at(s0), sl(s0)));
        for (int t = s0; t <= i; ++t) TRY(fwd_step(t, nullptr, nullptr));
      } else {
        const float* th = s0 == 0 ? theta0 : mp.ck[s0 / k];
        TRY(E.to_ops(th, sl(s0)));
        for (int t = s0; t < i; ++t) {
          float* nx = other(th);
          TRY(fwd_step(t, th, nx));
          th = nx;
        }
      }
    }
    if (adam) {
      float k1, k2;
      bias_corr(p, i, &k1, &k2);
      AdamVjpArgs<T> AL[MFMG_MAX_LAYERS];
      for (int l = 0; l < p->L; ++l) {
        AdamVjpArgs<T>& A = AL[l];
        A.layer = l;
        A.n_layers = p->L;
        A.nin = p->w[l];
        A.nout = p->w[l + 1];
        A.w_off = p->w_off[l];
        A.b_off = p->b_off[l];
        A.first = first;
        A.b1 = p->d.adam_b1;
        A.b2 = p->d.adam_b2;
        A.eps = p->d.adam_eps;
        A.k1 = k1;
        A.k2 = k2;
        A.eta = eta;
        A.theta = th_at(i);
        A.m = mp.m[st_of(i)];
        A.v = mp.vv[st_of(i)];
        A.g = g_at(i);
        A.thetabar = mp.thetabar;
        A.mbar = mp.mbar;
        A.vbar = mp.vbar;
        A.vW = mp.v[0].W[l];
        A.vWT = mp.v[0].WT[l];
        A.vb = mp.v[0].b[l];
        A.ldW = (int)p->ld(A.nout);
        A.ldWT = (int)p->ld(A.nin);
      }
      TimingScope ts(7, s);
      HIPCHK(adam_vjp<T>(AL, p->L, mp.part_off, mp.partial, s));
      HIPCHK(adam_reduce(mp.partial, mp.part_off, p->L, first, d_eta, s));
    }
    TRY(E.load_x(static_cast<const float*>(batches[i].x), R, a));
    TRY(E.forward(sl(i), &mp.v[vc], R, a));
    const float* alpha = wlog ? eta + (long)i * R : nullptr;
    TRY(E.head(batches[i], R, true, alpha, nullptr, wlog ? d_eta + (long)i * R : nullptr, a));
    ParamArgs<T> P = param_base<T>(p, mode_of(p, 2), eta);
    P.thetabar = mp.thetabar;
    P.etabar = d_eta;
    P.first = first;
    const OperandSet<T>& vn = mp.v[vc ^ 1];
    const bool write_next = !adam && i > 0;
    TRY(E.backward(sl(i), &mp.v[vc], R, !adam, P,
                   [&](ParamArgs<T>& Q, int l) {
                     if (write_next) {
                       Q.outW = vn.W[l];
                       Q.outWT = vn.WT[l];
                       Q.outb = vn.b[l];
                     }
                   },
                   a));
    if (!adam) vc ^= 1;
  }
  // MAML: nothing else depends on eta = theta_0, so dV/deta = bar theta_0
  if (maml) HIPCHK(copy(mp.thetabar, d_eta, n, s));
  return MFMG_OK;
}

template <typename T>
mfmg_status run_inner_step(const mfmg_problem* p, const float* theta, const float* opt,
                           const float* eta, const mfmg_batch* b, int step, float* theta_next,
                           float* opt_next, float* grad_out, float* loss_out, char* ws,
                           hipStream_t s) {
  StepPlan<T> sp;
  plan_step(p, ws, sp);
  Eng<T> E{p, s};
  TRY(zero_last_pads<T>(p, {&sp.th}, s));
  const int R = (int)b->rows;
  const long n = p->n_theta;
  const float* alpha =
      p->d.meta == MFMG_META_EXAMPLE_WEIGHT_LOGITS ? eta + (long)step * p->d.rows : nullptr;
  TRY(E.to_ops(theta, sp.th));
  TRY(E.load_x(static_cast<const float*>(b->x), R, sp.act));
  TRY(E.forward(sp.th, nullptr, R, sp.act));
  TRY(E.head(*b, R, false, alpha, nullptr, nullptr, sp.act));
  if (loss_out) HIPCHK(loss_reduce(sp.act.loss_rows, alpha, R, 1.0f / (float)R, loss_out, s));
  ParamArgs<T> P = param_base<T>(p, mode_of(p, 0), eta);
  P.theta = theta;
  P.theta_next = theta_next;
  P.grad_out = grad_out;
  if (p->adam()) {
    P.m_in = opt;
    P.v_in = opt ? opt + n : nullptr;
    P.m_out = opt_next;
    P.v_out = opt_next + n;
    bias_corr(p, step, &P.k1, &P.k2);
  }
  TRY(E.backward(sp.th, nullptr, R, true, P, [](ParamArgs<T>&, int) {}, sp.act));
  return MFMG_OK;
}

template <typename T>
mfmg_status run_hvp(const mfmg_problem* p, const float* theta, const float* eta,
                    const mfmg_batch* b, int step, const float* v, float* grad_out,
                    float* hvp_out, float* mvp_out, char* ws, hipStream_t s) {
  StepPlan<T> sp;
  plan_step(p, ws, sp);
  Eng<T> E{p, s};
  TRY(zero_last_pads<T>(p, {&sp.th, &sp.v}, s));
  const int R = (int)b->rows;
  const float* alpha =
      p->d.meta == MFMG_META_EXAMPLE_WEIGHT_LOGITS ? eta + (long)step * p->d.rows : nullptr;
  TRY(E.to_ops(theta, sp.th));
  TRY(E.to_ops(v, sp.v));
  TRY(E.load_x(static_cast<const float*>(b->x), R, sp.act));
  TRY(E.forward(sp.th, &sp.v, R, sp.act));
  TRY(E.head(*b, R, true, alpha, mvp_out, nullptr, sp.act));
  ParamArgs<T> P = param_base<T>(p, P_HVP, eta);
  P.grad_out = grad_out;
  P.hvp_out = hvp_out;
  TRY(E.backward(sp.th, &sp.v, R, true, P, [](ParamArgs<T>&, int) {}, sp.act));
  return MFMG_OK;
}

// ------------------------------------------------------------------------------------
// Validation helpers
// ------------------------------------------------------------------------------------
long n_eta_of(const mfmg_problem* p, int T) {
  if (p->tf) return tf_n_eta(p->d);
  switch (p->d.meta) {
    case MFMG_META_LOGLR_PER_PARAM: return p->n_theta;
    case MFMG_META_MAML: return p->n_theta;
    case MFMG_META_LOGLR_PER_LAYER_WD: return p->L + 1;
    case MFMG_META_EXAMPLE_WEIGHT_LOGITS: return (long)T * p->d.rows;
    default: return 0;
  }
}

bool aligned(const void* ptr, size_t a) { return (reinterpret_cast<uintptr_t>(ptr) % a) == 0; }

mfmg_status check_batch(const mfmg_problem* p, const mfmg_batch* b, int rows, const char* what,
                        int idx) {
  if (!b) return fail(MFMG_ERR_INVALID_ARGUMENT, "%s[%d]: null batch", what, idx);
  if (!b->x || (!b->y && !p->tf))
    return fail(MFMG_ERR_INVALID_ARGUMENT, "%s[%d]: null x or y", what, idx);
  if (b->rows != rows)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "%s[%d]: rows %lld, expected %d", what, idx,
                (long long)b->rows, rows);
  if (!aligned(b->x, 4) || (b->y && !aligned(b->y, 4)))
    return fail(MFMG_ERR_INVALID_ARGUMENT, "%s[%d]: x/y not 4-byte aligned", what, idx);
  return MFMG_OK;
}

mfmg_status check_align16(std::initializer_list<const void*> ptrs) {
  for (const void* q : ptrs)
    if (q && !aligned(q, 16))
      return fail(MFMG_ERR_INVALID_ARGUMENT, "parameter-shaped arrays must be 16-byte aligned");
  return MFMG_OK;
}

mfmg_status check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (ws_bytes < need)
    return fail(MFMG_ERR_WORKSPACE, "workspace of %zu bytes, %zu required", ws_bytes, need);
  if (need > 0 && !ws) return fail(MFMG_ERR_INVALID_ARGUMENT, "null workspace");
  if (ws && !aligned(ws, 256)) return fail(MFMG_ERR_INVALID_ARGUMENT, "workspace not 256-byte aligned");
  return MFMG_OK;
}

}  // namespace

// ------------------------------------------------------------------------------------
// Kernel timing
// ------------------------------------------------------------------------------------
namespace mfmg {
namespace {
std::mutex g_tm;
bool g_timing = false;
struct Rec {
  int cls;
  hipEvent_t a, b;
};
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_pool;
thread_local hipEvent_t g_open = nullptr;

hipEvent_t get_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

void timing_begin(int cls, hipStream_t s) {
  (void)cls;
  std::lock_guard<std::mutex> g(g_tm);
  if (!g_timing) return;
  g_open = get_event();
  if (g_open && hipEventRecord(g_open, s) != hipSuccess) {  // no record: time nothing
    g_pool.push_back(g_open);
    g_open = nullptr;
  }
}

void timing_end(int cls, hipStream_t s) {
  std::lock_guard<std::mutex> g(g_tm);
  if (!g_timing || !g_open) return;
  hipEvent_t e = get_event();
  if (e && hipEventRecord(e, s) == hipSuccess) {
    g_recs.push_back(Rec{cls, g_open, e});
  } else {
    if (e) g_pool.push_back(e);
    g_pool.push_back(g_open);
  }
  g_open = nullptr;
}
}  // namespace mfmg

// ------------------------------------------------------------------------------------
// C ABI
// ------------------------------------------------------------------------------------
extern "C" {

const char* mfmg_status_string(mfmg_status s) {
  switch (s) {
    case MFMG_OK: return "MFMG_OK";
    case MFMG_ERR_INVALID_ARGUMENT: return "MFMG_ERR_INVALID_ARGUMENT";
    case MFMG_ERR_UNSUPPORTED: return "MFMG_ERR_UNSUPPORTED";
    case MFMG_ERR_WORKSPACE: return "MFMG_ERR_WORKSPACE";
    case MFMG_ERR_HIP: return "MFMG_ERR_HIP";
    case MFMG_ERR_NUMERIC: return "MFMG_ERR_NUMERIC";
  }
  return "MFMG_UNKNOWN_STATUS";
}

const char* mfmg_last_error_message(void) { return g_err.c_str(); }

mfmg_status mfmg_problem_create(const mfmg_problem_desc* desc, mfmg_problem_t* out) {
  if (!desc || !out) return fail(MFMG_ERR_INVALID_ARGUMENT, "null desc or out");
  *out = nullptr;
  const mfmg_problem_desc& d = *desc;
  if (d.kind == MFMG_KIND_TRANSFORMER) {
    if (const char* msg = tf_validate(d)) return fail(MFMG_ERR_UNSUPPORTED, "%s", msg);
    mfmg_problem* p = new (std::nothrow) mfmg_problem;
    if (!p) return fail(MFMG_ERR_INVALID_ARGUMENT, "out of host memory");
    std::memset(p, 0, sizeof(*p));
    p->d = d;
    p->tf = true;
    p->VE = d.precision == MFMG_PREC_BF16 ? 8 : 4;
    p->n_theta = tf_n_theta(d);
    *out = p;
    return MFMG_OK;
  }
  if (d.kind != MFMG_KIND_MLP) return fail(MFMG_ERR_INVALID_ARGUMENT, "unknown kind %d", d.kind);
  if (d.n_layers < 1 || d.n_layers > MFMG_MAX_LAYERS)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "n_layers %d outside [1, %d]", d.n_layers,
                MFMG_MAX_LAYERS);
  for (int l = 0; l <= d.n_layers; ++l)
    if (d.widths[l] < 1 || d.widths[l] > (1 << 20))
      return fail(MFMG_ERR_INVALID_ARGUMENT, "widths[%d] = %d outside [1, 2^20]", l, d.widths[l]);
  if (d.act < MFMG_ACT_TANH || d.act > MFMG_ACT_NONE)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "unknown activation %d", d.act);
  if (d.loss != MFMG_LOSS_MSE && d.loss != MFMG_LOSS_CE && d.loss != MFMG_LOSS_MAPMSE)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "unknown loss %d", d.loss);
  if (d.loss == MFMG_LOSS_MAPMSE && (d.map_steps < 1 || d.map_steps > 1024))
    return fail(MFMG_ERR_INVALID_ARGUMENT, "map_steps = %d outside [1, 1024]", d.map_steps);
  if (d.ckpt_segment < 0 || d.ckpt_segment > (1 << 20))
    return fail(MFMG_ERR_INVALID_ARGUMENT, "ckpt_segment = %d outside [0, 2^20]",
                d.ckpt_segment);
  if (d.fused_attention != 0 || d.block_remat != 0)
    return fail(MFMG_ERR_INVALID_ARGUMENT,
                "fused_attention and block_remat apply to transformer problems");
  if (d.optimizer != MFMG_OPT_SGD && d.optimizer != MFMG_OPT_ADAM)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "unknown optimizer %d", d.optimizer);
  if (d.precision != MFMG_PREC_FP32 && d.precision != MFMG_PREC_BF16)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "unknown precision %d", d.precision);
  if (d.has_bias != 0 && d.has_bias != 1)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "has_bias must be 0 or 1");
  if (d.rows < 1 || d.val_rows < 1 || d.rows > (1 << 20) || d.val_rows > (1 << 20))
    return fail(MFMG_ERR_INVALID_ARGUMENT, "rows %d / val_rows %d outside [1, 2^20]", d.rows,
                d.val_rows);
  if (d.loss == MFMG_LOSS_CE && d.widths[d.n_layers] < 2)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "cross-entropy needs at least 2 classes");
  switch (d.meta) {
    case MFMG_META_LOGLR_PER_PARAM:
      if (d.optimizer != MFMG_OPT_SGD)
        return fail(MFMG_ERR_UNSUPPORTED, "per-parameter log-lr is implemented for SGD");
      break;
    case MFMG_META_LOGLR_PER_LAYER_WD:
      if (d.optimizer != MFMG_OPT_ADAM)
        return fail(MFMG_ERR_UNSUPPORTED, "per-layer log-lr + weight decay is implemented for Adam");
      break;
    case MFMG_META_EXAMPLE_WEIGHT_LOGITS:
      if (d.optimizer != MFMG_OPT_SGD)
        return fail(MFMG_ERR_UNSUPPORTED, "example loss weights are implemented for SGD");
      if (!std::isfinite(d.sgd_lr))
        return fail(MFMG_ERR_INVALID_ARGUMENT, "sgd_lr must be finite");
      break;
    case MFMG_META_TOKEN_WEIGHT_MLP:
      return fail(MFMG_ERR_UNSUPPORTED, "token-weight meta-MLP needs the transformer kind");
    case MFMG_META_MAML:
      if (d.optimizer != MFMG_OPT_SGD)
        return fail(MFMG_ERR_UNSUPPORTED, "MAML is implemented for SGD");
      if (!std::isfinite(d.sgd_lr))
        return fail(MFMG_ERR_INVALID_ARGUMENT, "sgd_lr must be finite");
      break;
    default:
      return fail(MFMG_ERR_INVALID_ARGUMENT, "unknown meta kind %d", d.meta);
  }
  if (d.optimizer == MFMG_OPT_ADAM) {
    if (!(d.adam_b1 >= 0.f && d.adam_b1 < 1.f) || !(d.adam_b2 >= 0.f && d.adam_b2 < 1.f) ||
        !(d.adam_eps > 0.f))
      return fail(MFMG_ERR_INVALID_ARGUMENT, "Adam needs b1, b2 in [0, 1) and eps > 0");
  }
  mfmg_problem* p = new (std::nothrow) mfmg_problem;
  if (!p) return fail(MFMG_ERR_INVALID_ARGUMENT, "out of host memory");
  p->d = d;
  p->tf = false;
  p->L = d.n_layers;
  p->VE = d.precision == MFMG_PREC_BF16 ? 8 : 4;
  long off = 0;
  for (int l = 0; l <= p->L; ++l) p->w[l] = d.widths[l];
  for (int l = 0; l < p->L; ++l) {
    p->w_off[l] = off;
    off += (long)p->w[l] * p->w[l + 1];
    p->b_off[l] = -1;
    if (d.has_bias) {
      p->b_off[l] = off;
      off += p->w[l + 1];
    }
  }
  p->n_theta = off;
  const long maxR = p->maxR();
  for (int l = 0; l <= p->L; ++l) {
    if ((long)p->w[l] * rup(maxR, 8) >= (1L << 31) || (long)p->w[l] * rup(p->w[l], 8) >= (1L << 31)) {
      delete p;
      return fail(MFMG_ERR_UNSUPPORTED, "a matrix exceeds 2^31 elements");
    }
  }
  *out = p;
  return MFMG_OK;
}

void mfmg_problem_destroy(mfmg_problem_t p) { delete p; }

mfmg_status mfmg_query_sizes(mfmg_problem_t p, int T, mfmg_sizes* out) {
  if (!p || !out) return fail(MFMG_ERR_INVALID_ARGUMENT, "null problem or out");
  if (T < 1) return fail(MFMG_ERR_INVALID_ARGUMENT, "T = %d, must be >= 1", T);
  out->n_theta = p->n_theta;
  out->n_opt_state = p->adam() ? 2 * p->n_theta : 0;
  out->n_eta = n_eta_of(p, T);
  size_t st = 0, dy = 0;
  if (p->tf) {
    out->workspace_bytes = tf_meta_ws(p->d, T, &st, &dy);
    out->static_bytes = st;
    out->dynamic_bytes = dy;
    out->step_workspace_bytes = tf_step_ws(p->d);
    return MFMG_OK;
  }
  out->workspace_bytes = meta_ws_bytes(p, T, &st, &dy);
  out->static_bytes = st;
  out->dynamic_bytes = dy;
  out->step_workspace_bytes = step_ws_bytes(p);
  return MFMG_OK;
}

mfmg_status mfmg_inner_step(mfmg_problem_t p, const float* theta, const float* opt_state,
                            const float* eta, const mfmg_batch* batch, int step_index,
                            float* theta_next, float* opt_state_next, float* grad_out,
                            float* loss_out, void* ws, size_t ws_bytes, void* stream) {
  if (!p) return fail(MFMG_ERR_INVALID_ARGUMENT, "null problem");
  if (!theta || !eta || !theta_next)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "null theta, eta or theta_next");
  if (p->adam() && !opt_state_next)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "Adam needs opt_state_next");
  if (step_index < 0) return fail(MFMG_ERR_INVALID_ARGUMENT, "negative step_index");
  if (!batch) return fail(MFMG_ERR_INVALID_ARGUMENT, "null batch");
  if (batch->rows != p->d.rows)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "batch rows %lld, expected %d", (long long)batch->rows,
                p->d.rows);
  TRY(check_batch(p, batch, p->d.rows, "batch", 0));
  TRY(check_align16({theta, opt_state, eta, theta_next, opt_state_next, grad_out}));
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (p->tf) {
    TRY(check_ws(ws, ws_bytes, tf_step_ws(p->d)));
    HIPCHK(tf_run_inner(p->d, theta, eta, batch, theta_next, grad_out, loss_out, (char*)ws, s));
    return MFMG_OK;
  }
  TRY(check_ws(ws, ws_bytes, step_ws_bytes(p)));
  if (p->bf16())
    return run_inner_step<bf16_t>(p, theta, opt_state, eta, batch, step_index, theta_next,
                                  opt_state_next, grad_out, loss_out, (char*)ws, s);
  return run_inner_step<float>(p, theta, opt_state, eta, batch, step_index, theta_next,
                               opt_state_next, grad_out, loss_out, (char*)ws, s);
}

mfmg_status mfmg_hvp_fwd_over_rev(mfmg_problem_t p, const float* theta, const float* eta,
                                  const mfmg_batch* batch, int step_index, const float* v,
                                  float* grad_out, float* hvp_out, float* mvp_out, void* ws,
                                  size_t ws_bytes, void* stream) {
  if (!p) return fail(MFMG_ERR_INVALID_ARGUMENT, "null problem");
  if (!theta || !eta || !v || !hvp_out)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "null theta, eta, v or hvp_out");
  if (step_index < 0) return fail(MFMG_ERR_INVALID_ARGUMENT, "negative step_index");
  TRY(check_batch(p, batch, p->d.rows, "batch", 0));
  TRY(check_align16({theta, eta, v, grad_out, hvp_out}));
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (p->tf) {
    TRY(check_ws(ws, ws_bytes, tf_step_ws(p->d)));
    HIPCHK(tf_run_hvp(p->d, theta, eta, batch, v, grad_out, hvp_out, mvp_out, (char*)ws, s));
    return MFMG_OK;
  }
  TRY(check_ws(ws, ws_bytes, step_ws_bytes(p)));
  if (p->bf16())
    return run_hvp<bf16_t>(p, theta, eta, batch, step_index, v, grad_out, hvp_out, mvp_out,
                           (char*)ws, s);
  return run_hvp<float>(p, theta, eta, batch, step_index, v, grad_out, hvp_out, mvp_out,
                        (char*)ws, s);
}

}  // extern "C"

namespace {

// Host-side checks of mfmg_meta_grad's arguments (all but the workspace);
// *need = the workspace bytes the call uses.
mfmg_status check_meta_args(mfmg_problem_t p, const float* theta0, const float* opt_state0,
                            const float* eta, const mfmg_batch* train_batches, int T,
                            const mfmg_batch* val_batch, const float* d_eta_out, size_t* need) {
  if (!p) return fail(MFMG_ERR_INVALID_ARGUMENT, "null problem");
  if (T < 1) return fail(MFMG_ERR_INVALID_ARGUMENT, "T = %d, must be >= 1", T);
  if ((!theta0 && p->d.meta != MFMG_META_MAML) || !eta || !d_eta_out)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "null theta0, eta or d_eta_out");
  if (!train_batches) return fail(MFMG_ERR_INVALID_ARGUMENT, "null train_batches");
  for (int t = 0; t < T; ++t) TRY(check_batch(p, &train_batches[t], p->d.rows, "train_batches", t));
  TRY(check_batch(p, val_batch, p->d.val_rows, "val_batch", 0));
  TRY(check_align16({theta0, opt_state0, eta, d_eta_out}));
  size_t st = 0, dy = 0;
  *need = p->tf ? tf_meta_ws(p->d, T, &st, &dy) : meta_ws_bytes(p, T, &st, &dy);
  return MFMG_OK;
}

// The meta-gradient on validated arguments and a workspace of at least `need` bytes.
mfmg_status meta_grad_run(mfmg_problem_t p, const float* theta0, const float* opt_state0,
                          const float* eta, const mfmg_batch* train_batches, int T,
                          const mfmg_batch* val_batch, float* d_eta_out, float* val_loss_out,
                          size_t* peak_bytes_out, size_t need, void* ws, void* stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (p->tf) {
    if (peak_bytes_out) {
      const long n_eta = tf_n_eta(p->d);
      size_t b = need + 4 * (size_t)p->n_theta + 8 * (size_t)n_eta + (val_loss_out ? 4 : 0);
      b += (size_t)(T * p->d.rows + p->d.val_rows) * (p->d.seq + 1) * 4;
      *peak_bytes_out = b;
    }
    HIPCHK(tf_run_meta(p->d, theta0, eta, train_batches, T, val_batch, d_eta_out, val_loss_out,
                       (char*)ws, s));
    return MFMG_OK;
  }
  if (peak_bytes_out) {
    const long n_eta = n_eta_of(p, T);
    const size_t ybytes = 4 * (size_t)(p->d.loss == MFMG_LOSS_CE ? 1 : p->w[p->L]);
    size_t b = need + 4 * (size_t)p->n_theta + 8 * (size_t)n_eta;
    if (opt_state0) b += 8 * (size_t)p->n_theta;
    if (val_loss_out) b += 4;
    b += (size_t)T * p->d.rows * (4 * (size_t)p->w[0] + ybytes);
    b += (size_t)p->d.val_rows * (4 * (size_t)p->w[0] + ybytes);
    *peak_bytes_out = b;
  }
  if (p->linreg_path(T)) {
    std::vector<const float*> xs(T), ys(T);
    for (int t = 0; t < T; ++t) {
      xs[t] = static_cast<const float*>(train_batches[t].x);
      ys[t] = static_cast<const float*>(train_batches[t].y);
    }
    MetaPlan<float> mp;
    plan_meta(p, T, (char*)ws, mp);
    TimingScope ts(7, s);
    HIPCHK(linreg_meta_grad(theta0, eta, xs.data(), ys.data(), T, p->d.rows, p->w[0],
                            static_cast<const float*>(val_batch->x),
                            static_cast<const float*>(val_batch->y), p->d.val_rows, d_eta_out,
                            val_loss_out, mp.linreg_scratch, s));
    return MFMG_OK;
  }
  if (p->bf16())
    return run_meta<bf16_t>(p, theta0, opt_state0, eta, train_batches, T, val_batch, d_eta_out,
                            val_loss_out, (char*)ws, s);
  return run_meta<float>(p, theta0, opt_state0, eta, train_batches, T, val_batch, d_eta_out,
                         val_loss_out, (char*)ws, s);
}

// Scratch of mfmg_meta_grad_noalloc: device memory of the code object, one copy
// per GPU, held until the process ends.  In host code `scratch` names a
// host-side stand-in; its device address on the current GPU comes from
// hipGetSymbolAddress, once per device, and only that address is used.
static __device__ __align__(256) unsigned char scratch[MFMG_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

mfmg_status scratch_of_current_device(void** out) {
  int dev = -1;
  HIPCHK(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(MFMG_ERR_UNSUPPORTED, "device index %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    HIPCHK(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    if (!ptr || !aligned(ptr, 256))
      return fail(MFMG_ERR_HIP, "no 256-byte-aligned address for the static scratch");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return MFMG_OK;
}

}  // namespace

extern "C" {

mfmg_status mfmg_meta_grad(mfmg_problem_t p, const float* theta0, const float* opt_state0,
                           const float* eta, const mfmg_batch* train_batches, int T,
                           const mfmg_batch* val_batch, float* d_eta_out, float* val_loss_out,
                           size_t* peak_bytes_out, void* ws, size_t ws_bytes, void* stream) {
  size_t need = 0;
  TRY(check_meta_args(p, theta0, opt_state0, eta, train_batches, T, val_batch, d_eta_out, &need));
  TRY(check_ws(ws, ws_bytes, need));
  return meta_grad_run(p, theta0, opt_state0, eta, train_batches, T, val_batch, d_eta_out,
                       val_loss_out, peak_bytes_out, need, ws, stream);
}

mfmg_status mfmg_meta_grad_noalloc(mfmg_problem_t p, const float* theta0,
                                   const float* opt_state0, const float* eta,
                                   const mfmg_batch* train_batches, int T,
                                   const mfmg_batch* val_batch, float* d_eta_out,
                                   float* val_loss_out, size_t* peak_bytes_out, void* stream) {
  size_t need = 0;
  TRY(check_meta_args(p, theta0, opt_state0, eta, train_batches, T, val_batch, d_eta_out, &need));
  if (need > (size_t)MFMG_NOALLOC_SCRATCH_BYTES)
    return fail(MFMG_ERR_WORKSPACE,
                "this problem needs %zu bytes of scratch at T = %d; the static scratch of "
                "mfmg_meta_grad_noalloc holds %zu (use mfmg_meta_grad with a workspace)",
                need, T, (size_t)MFMG_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  TRY(scratch_of_current_device(&ws));
  return meta_grad_run(p, theta0, opt_state0, eta, train_batches, T, val_batch, d_eta_out,
                       val_loss_out, peak_bytes_out, need, ws, stream);
}

mfmg_status mfmg_check_finite(const float* x, size_t n, size_t* count_out, void* ws,
                              size_t ws_bytes, void* stream) {
  if (!x && n) return fail(MFMG_ERR_INVALID_ARGUMENT, "null x");
  if (x && !aligned(x, 4)) return fail(MFMG_ERR_INVALID_ARGUMENT, "x not 4-byte aligned");
  TRY(check_ws(ws, ws_bytes, 256));
  if (!ws) return fail(MFMG_ERR_INVALID_ARGUMENT, "null workspace");
  hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned long long* cnt = static_cast<unsigned long long*>(ws);
  HIPCHK(count_nonfinite(x, (long)n, cnt, s));
  unsigned long long h = 0;
  HIPCHK(hipMemcpyAsync(&h, cnt, sizeof(h), hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  if (count_out) *count_out = (size_t)h;
  if (h) return fail(MFMG_ERR_NUMERIC, "%llu of %zu values are NaN or infinite", h, n);
  return MFMG_OK;
}

mfmg_status mfmg_timing_enable(int enable) {
  std::lock_guard<std::mutex> g(mfmg::g_tm);
  mfmg::g_timing = enable != 0;
  return MFMG_OK;
}

mfmg_status mfmg_timing_read(int cls, int* launches, double* total_ms) {
  if (cls < 0 || cls >= MFMG_NUM_KERNEL_CLASSES || !launches || !total_ms)
    return fail(MFMG_ERR_INVALID_ARGUMENT, "bad kernel class or null output");
  std::lock_guard<std::mutex> g(mfmg::g_tm);
  int n = 0;
  double ms = 0.0;
  std::vector<mfmg::Rec> keep;
  for (auto& r : mfmg::g_recs) {
    if (r.cls != cls) {
      keep.push_back(r);
      continue;
    }
    float e = 0.0f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&e, r.a, r.b) != hipSuccess)
      return fail(MFMG_ERR_HIP, "timing events failed");
    ms += e;
    ++n;
    mfmg::g_pool.push_back(r.a);
    mfmg::g_pool.push_back(r.b);
  }
  mfmg::g_recs.swap(keep);
  *launches = n;
  *total_ms = ms;
  return MFMG_OK;
}

}  // extern "C"
