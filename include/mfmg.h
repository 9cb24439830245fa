/*
 * mfmg.h -- C ABI of the MixFlow-MG meta-gradient library for MI355X (gfx950).
 *
 * The library computes the truncated-BPTT meta-gradient dV/deta of the bilevel
 * problem (Section 2.1, eq. bilevel_opt_problem and eq. bptt_bilevel):
 *
 *   (theta_{i+1}, upsilon_{i+1}) = Upsilon(dL(theta_i, eta, x_i)/dtheta_i,
 *                                          theta_i, upsilon_i, eta),  i = 0..T-1
 *   V = V(theta_T, val)
 *
 * with the inner gradient an explicit argument of the update (Section 3,
 * eq. reparam).  The reverse sweep follows the one-step recurrence of
 * Section 3 (eq. bptt_recur) seeded by eq. dVdmeta; every Hessian-vector and
 * mixed-derivative product it needs is formed forward-over-reverse
 * (Section 2.2; Section 3, eq. vhp_to_hvp and eq. vmp_to_mvp): a tangent on
 * theta rides through the inner gradient computation.
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 *  - Pointers marked (dev) are device memory on the current HIP device, owned
 *    by the caller.  Pointers marked (host) are host memory.
 *  - The library never allocates or frees device memory inside a call.  All
 *    scratch comes from the caller's workspace `ws` of `ws_bytes` bytes, whose
 *    required size mfmg_query_sizes reports.  `ws` must be 256-byte aligned.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued
 *    asynchronously on it; outputs are valid once the stream has reached the
 *    end of the call.
 *  - All arguments are validated on the host before anything is enqueued.  On
 *    MFMG_ERR_INVALID_ARGUMENT, MFMG_ERR_UNSUPPORTED and MFMG_ERR_WORKSPACE
 *    nothing has been enqueued and no output has been written;
 *    mfmg_last_error_message() describes the failure.  MFMG_ERR_HIP means a
 *    launch failed part-way: outputs are undefined.  Errors of the device
 *    execution itself surface at the caller's next synchronisation.
 *  - Inputs are never modified; outputs are fully overwritten.
 *  - Arrays in the theta, opt_state or eta layout (and v, grad_out, hvp_out,
 *    d_eta_out) must be 16-byte aligned; batch arrays 4-byte aligned.
 *  - Calls on the same workspace must not overlap in time; distinct
 *    workspaces may be used concurrently on distinct streams.
 *
 * Parameter layout (flat float32 arrays)
 * --------------------------------------
 *  MLP: for each layer l = 0..n_layers-1, W_l row-major [widths[l]][widths[l+1]]
 *  followed by b_l [widths[l+1]] when has_bias.  Linear regression is the
 *  one-layer, bias-free, identity-activation MLP with squared loss.
 *  opt_state (Adam): [m | v], each n_theta floats in the theta layout.
 *  eta, by meta-parameter kind:
 *   MFMG_META_LOGLR_PER_PARAM      n_theta log learning rates, theta layout;
 *                                  update theta' = theta - exp(eta) * g.
 *   MFMG_META_LOGLR_PER_LAYER_WD   n_layers log learning rates then one raw
 *                                  decoupled weight decay omega (Adam).
 *   MFMG_META_EXAMPLE_WEIGHT_LOGITS [T][rows] logits; example n of inner step
 *                                  t has loss weight sigmoid(eta[t][n]).
 *   MFMG_META_MAML                 n_theta floats, theta layout: the starting
 *                                  point theta_0 itself (MAML, the task list of
 *                                  Section 5.2); SGD with the fixed rate sgd_lr,
 *                                  unweighted loss.  dV/deta = bar theta_0;
 *                                  mfmg_meta_grad ignores its theta0 argument
 *                                  (which may be null).  MLP kind only.
 *  Transformer (MFMG_KIND_TRANSFORMER; d = d_model, F = d_ff, V = vocab; every
 *  matrix row-major [in][out], applied as x W): the token embedding E [V][d];
 *  then for each block b = 0..n_blocks-1: ln1 gain [d], ln1 bias [d],
 *  W_qkv [d][3d] (output columns q | k | v, head h owning columns h*d/H ..
 *  (h+1)*d/H - 1 of each), W_o [d][d], ln2 gain [d], ln2 bias [d], W_1 [d][F],
 *  W_2 [F][d]; then the final LayerNorm gain [d] and bias [d] and the
 *  unembedding U [d][V].  No linear biases.  Each block is pre-LayerNorm:
 *  h += Attn(LN1(h)) W_o, h += GELU(LN2(h) W_1) W_2, with causal softmax
 *  attention scaled by 1/sqrt(d/H) and rotary position embeddings on q and k
 *  (rotate-half pairing of head dims j and j + d/(2H), angle pos *
 *  rope_base^(-2j/(d/H))); GELU is the exact erf form; logits = LNf(h) U.
 *   MFMG_META_TOKEN_WEIGHT_MLP (transformer only): eta = [W1 [d][meta_hidden] |
 *                                  b1 [meta_hidden] | w2 [meta_hidden] | b2],
 *                                  d*meta_hidden + 2*meta_hidden + 1 floats.
 *                                  Token (b, s) of inner step t has loss weight
 *                                  sigmoid(tanh(e W1 + b1) . w2 + b2), where e is
 *                                  row tokens[b][s] of the embedding E of the
 *                                  theta_0 passed in, held constant (for the
 *                                  single-step calls: of the theta passed in).
 *  The inner loss is L = (1/N) sum_n alpha_n l_n over the N rows of a batch,
 *  alpha_n = 1 unless the loss is weighted; the outer loss V is the unweighted
 *  mean over the validation rows.  l_n is softmax cross-entropy (CE) or the
 *  squared error sum_j (z_nj - y_nj)^2 (MSE), or for MAPMSE the mean over the
 *  outputs j of (y_M,nj - y_nj)^2, where y_0 = z and y_i = i (2 + sin y_{i-1})^
 *  cos(y_{i-1}) elementwise for i = 1..M (the map of Section 3.2, eq.
 *  motivational_example; with one D x D layer and MAML this is the paper's
 *  motivating example).  MAPMSE targets are float32 like MSE ones.
 *
 * Batches (mfmg_batch)
 * --------------------
 *  MLP: x (dev) float32 [rows][widths[0]] row-major; y (dev) int32 class
 *  labels [rows] for CE or float32 targets [rows][widths[n_layers]] for MSE
 *  and MAPMSE.
 *  Transformer: x (dev) int32 tokens [rows][seq + 1] row-major, ids in
 *  [0, vocab); sequence b predicts tokens[b][1..seq] from tokens[b][0..seq-1],
 *  so a batch has N = rows * seq loss rows (the mvp_out rows of
 *  mfmg_hvp_fwd_over_rev are ordered b * seq + s).  y is unused (may be NULL).
 */
#ifndef MFMG_H_
#define MFMG_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MFMG_OK = 0,
  MFMG_ERR_INVALID_ARGUMENT = 1, /* a null/misaligned pointer, a bad size or shape */
  MFMG_ERR_UNSUPPORTED = 2,      /* a valid combination the library does not implement */
  MFMG_ERR_WORKSPACE = 3,        /* ws_bytes smaller than mfmg_query_sizes reports */
  MFMG_ERR_HIP = 4,              /* a HIP runtime call failed while enqueueing */
  MFMG_ERR_NUMERIC = 5           /* mfmg_check_finite found a NaN or an infinity */
} mfmg_status;

enum { MFMG_KIND_MLP = 0, MFMG_KIND_TRANSFORMER = 1 };
enum { MFMG_ACT_TANH = 0, MFMG_ACT_GELU = 1, MFMG_ACT_RELU = 2, MFMG_ACT_NONE = 3 };
enum { MFMG_LOSS_MSE = 0, MFMG_LOSS_CE = 1, MFMG_LOSS_MAPMSE = 2 };
enum { MFMG_OPT_SGD = 0, MFMG_OPT_ADAM = 1 };
enum {
  MFMG_META_LOGLR_PER_PARAM = 0,
  MFMG_META_LOGLR_PER_LAYER_WD = 1,
  MFMG_META_EXAMPLE_WEIGHT_LOGITS = 2,
  MFMG_META_TOKEN_WEIGHT_MLP = 3,
  MFMG_META_MAML = 4
};
/* FP32: float32 GEMM operands.  BF16: bfloat16 GEMM operands (round to nearest
 * even) with float32 accumulation; parameters, optimiser state, adjoints and
 * all elementwise arithmetic stay float32 in both modes. */
enum { MFMG_PREC_FP32 = 0, MFMG_PREC_BF16 = 1 };

#define MFMG_MAX_LAYERS 16

/* Problem description.  Fields a kind does not use are ignored. */
typedef struct {
  int kind;                            /* MFMG_KIND_* */
  int n_layers;                        /* MLP: number of weight matrices, 1..MFMG_MAX_LAYERS */
  int widths[MFMG_MAX_LAYERS + 1];     /* MLP: widths[0] inputs .. widths[n_layers] outputs */
  int act;                             /* hidden activation, MFMG_ACT_* */
  int loss;                            /* MFMG_LOSS_* */
  int optimizer;                       /* MFMG_OPT_* */
  int meta;                            /* MFMG_META_* */
  int precision;                       /* MFMG_PREC_* */
  int has_bias;                        /* MLP: 0 or 1 */
  int rows;                            /* rows of every training batch */
  int val_rows;                        /* rows of the validation batch */
  float sgd_lr;                        /* fixed inner learning rate (weighted-loss metas) */
  float adam_b1, adam_b2, adam_eps;    /* Adam constants */
  /* Transformer kind only (see "Parameter layout"): model width, heads,
   * feed-forward width, vocabulary, tokens per sequence, blocks, width of the
   * token-weight meta-model's hidden layer, LayerNorm epsilon, RoPE base.
   * Supported: d_model, d_ff and d_model / n_heads multiples of 8, d_model <=
   * 1024; seq a multiple of 4; rows * seq and val_rows * seq <= 8192 tokens;
   * meta_hidden a multiple of 8 in [8, 256]; SGD with the fixed rate sgd_lr,
   * cross-entropy, MFMG_META_TOKEN_WEIGHT_MLP. */
  int d_model, n_heads, d_ff, vocab, seq, n_blocks, meta_hidden;
  float ln_eps, rope_base;
  int map_steps;                       /* MFMG_LOSS_MAPMSE: M, 1..1024 */
  /* Static-memory reduction (MLP kind): 0 keeps the checkpoint of every
   * theta_t (memory linear in T).  k >= 1 keeps float32 theta (and Adam's m
   * and v) only at t = k, 2k, .. and a ring of k + 1 states (operand copies;
   * for Adam also float32 theta, m, v and k saved inner gradients), and
   * recomputes each segment's states (the same kernels on the same inputs, so
   * the result is bit-identical) when the reverse sweep enters it: static
   * memory ~ (T/k + k) parameter copies, one extra forward inner step per
   * recomputed state (Adam: per state of the segment, since the gradient of
   * its last step is read before that step's dual pass).  A two-level form of
   * the rematerialisation schedules the appendix on static device memory
   * proposes (whose logarithmic form needs a recursive schedule).  Ignored
   * when k >= T. */
  int ckpt_segment;
  /* Transformer kind only.  0 materialises each block's attention
   * probabilities P and their tangent (B*H*S^2 per block, kept from the
   * forward for the backward).  1 runs fused causal attention: the forward
   * keeps running row maxima and sums over key blocks and saves two floats per
   * query row (log-sum-exp and <P, Sd>); the backward recomputes P and its
   * tangent per tile, so attention adds O(B*H*S) to dynamic memory instead of
   * O(B*H*S^2).  Same quantities as 0 (Section 2.2, the dual products of
   * softmax attention); requires MFMG_PREC_BF16, head dimension
   * d_model / n_heads = 64 and seq a multiple of 64. */
  int fused_attention;
  /* Transformer kind only: block rematerialisation (Section 4, "Block
   * rematerialisation").  0 keeps every block's activations (and tangents) of
   * one inner step from its forward for its backward, so dynamic memory grows
   * with n_blocks.  1 keeps only the residual stream entering each block (and
   * its tangent) and recomputes the block's forward, with the tangent in dual
   * passes, at the start of that block's backward: one buffer set serves all
   * blocks, dynamic memory is flat in n_blocks up to the block inputs
   * (2 * 4 * rows * seq * d_model bytes per block), and each backward does one
   * more block forward per block (its last residual product excepted).  The
   * recomputation repeats the same kernels on the same inputs, so results are
   * bit-identical to 0. */
  int block_remat;
} mfmg_problem_desc;

typedef struct mfmg_problem* mfmg_problem_t;

/* Sizes, in elements (n_*) and bytes (*_bytes). */
typedef struct {
  size_t n_theta;              /* floats in theta */
  size_t n_opt_state;          /* floats in opt_state (0 for SGD) */
  size_t n_eta;                /* floats in eta (depends on T for EXAMPLE_WEIGHT_LOGITS) */
  size_t workspace_bytes;      /* workspace mfmg_meta_grad needs at this T */
  size_t static_bytes;         /* part of it that lives through the whole call
                                  (theta checkpoints, adjoints, tangents) */
  size_t dynamic_bytes;        /* part of it reused by every inner step
                                  (one step's activations); independent of T */
  size_t step_workspace_bytes; /* workspace mfmg_inner_step / mfmg_hvp_fwd_over_rev need */
} mfmg_sizes;

typedef struct {
  const void* x;  /* (dev) see "Batches" above */
  const void* y;  /* (dev) see "Batches" above */
  int64_t rows;   /* must equal desc.rows (training) or desc.val_rows (validation) */
} mfmg_batch;

/* Validates `desc` and creates an immutable problem handle.  The handle holds
 * host memory only and may be shared by threads.  INVALID_ARGUMENT for a bad
 * description, UNSUPPORTED for a valid one the library does not implement. */
mfmg_status mfmg_problem_create(const mfmg_problem_desc* desc, mfmg_problem_t* out);

/* Releases a handle (NULL is ignored). */
void mfmg_problem_destroy(mfmg_problem_t problem);

/* Host-only size query for T inner steps (T >= 1).  No device work. */
mfmg_status mfmg_query_sizes(mfmg_problem_t problem, int T, mfmg_sizes* out);

/* One inner update (Section 2.1, eq. bptt_bilevel; Section 3, eq. reparam):
 * g = dL(theta, eta, batch)/dtheta, then (theta_next, opt_state_next) =
 * Upsilon(g, theta, opt_state, eta) with Adam's bias correction taken at update
 * count step_index + 1.  step_index (0-based) also selects the loss weights of
 * EXAMPLE_WEIGHT_LOGITS.
 *   theta (dev, n_theta), opt_state (dev, n_opt_state; NULL = zeros; must be
 *   NULL-or-valid for Adam, ignored for SGD), eta (dev, n_eta),
 *   theta_next (dev, n_theta), opt_state_next (dev, n_opt_state; required for
 *   Adam, ignored for SGD), grad_out (dev, n_theta, nullable), loss_out (dev,
 *   1 float, nullable: L of this batch).
 *   ws: at least step_workspace_bytes.  Outputs must not alias inputs. */
mfmg_status mfmg_inner_step(mfmg_problem_t problem, const float* theta, const float* opt_state,
                            const float* eta, const mfmg_batch* batch, int step_index,
                            float* theta_next, float* opt_state_next, float* grad_out,
                            float* loss_out, void* ws, size_t ws_bytes, void* stream);

/* One forward-over-reverse pass (Section 2.2; Section 3, eq. vhp_to_hvp and
 * eq. vmp_to_mvp; the JVP-of-gradient rule of the fwdrev_grad transformation,
 * Section 3.1): with the tangent v on theta,
 *   grad_out = dL/dtheta                                   (dev, n_theta, nullable)
 *   hvp_out  = (d^2 L / dtheta^2) v                        (dev, n_theta)
 *   mvp_out  = (d^2 L / dalpha_n dtheta) v, one float per loss row n
 *              (= (1/N) <grad l_n, v>)                     (dev, rows floats, nullable)
 * at theta (dev, n_theta) on one batch; eta and step_index select the loss
 * weights alpha as in mfmg_inner_step.  v (dev, n_theta).
 * ws: at least step_workspace_bytes. */
mfmg_status mfmg_hvp_fwd_over_rev(mfmg_problem_t problem, const float* theta, const float* eta,
                                  const mfmg_batch* batch, int step_index, const float* v,
                                  float* grad_out, float* hvp_out, float* mvp_out, void* ws,
                                  size_t ws_bytes, void* stream);

/* The meta-gradient dV/deta through T inner steps (Algorithm 2, mixed-mode
 * truncated BPTT), with per-inner-step checkpointing of theta_t (Section 4):
 * the forward unroll stores theta_t (and Adam's state and inner gradients,
 * Section 4 "saving inner gradients"); the reverse sweep i = T-1..0 recomputes
 * step i from its checkpoint with a tangent, accumulating d eta.
 *   theta0 (dev, n_theta), opt_state0 (dev, n_opt_state or NULL = zeros),
 *   eta (dev, n_eta at this T), train_batches (host array of T descriptors
 *   whose x/y are dev), val_batch (host descriptor, dev x/y),
 *   d_eta_out (dev, n_eta), val_loss_out (dev, 1 float, nullable: V),
 *   peak_bytes_out (host, nullable): bytes of device memory the call touches
 *   at its peak: caller-visible inputs and outputs plus the workspace it uses.
 * ws: at least workspace_bytes of mfmg_query_sizes(problem, T). */
mfmg_status mfmg_meta_grad(mfmg_problem_t problem, const float* theta0, const float* opt_state0,
                           const float* eta, const mfmg_batch* train_batches, int T,
                           const mfmg_batch* val_batch, float* d_eta_out, float* val_loss_out,
                           size_t* peak_bytes_out, void* ws, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * computation and outputs as mfmg_meta_grad, with the workspace taken from a
 * static scratch array inside the library instead of a caller buffer.  No
 * device memory is allocated or freed by the call.  Each GPU the library runs
 * on holds one MFMG_NOALLOC_SCRATCH_BYTES array from the first use of the
 * library on it until the process ends; its address is looked up on the
 * first call per device (a HIP runtime query, no allocation).
 *   Limit: problems whose mfmg_query_sizes(problem, T).workspace_bytes exceeds
 *   MFMG_NOALLOC_SCRATCH_BYTES are rejected with MFMG_ERR_WORKSPACE before
 *   anything is enqueued (small MLPs and transformers; not the 8 x 4096 one).
 *   Every call on one GPU shares its array, whose contents persist between
 *   calls: calls that overlap in time on one GPU (on different streams or
 *   threads) race and give undefined results.  Arguments and outputs as for
 *   mfmg_meta_grad. */
#define MFMG_NOALLOC_SCRATCH_BYTES (64u * 1024u * 1024u)
mfmg_status mfmg_meta_grad_noalloc(mfmg_problem_t problem, const float* theta0,
                                   const float* opt_state0, const float* eta,
                                   const mfmg_batch* train_batches, int T,
                                   const mfmg_batch* val_batch, float* d_eta_out,
                                   float* val_loss_out, size_t* peak_bytes_out, void* stream);

/* Non-finite check of a result, e.g. d_eta_out of mfmg_meta_grad (whose
 * calls never inspect their outputs: that would need a host synchronisation
 * inside the call).  Counts the NaN and infinite entries of x (dev, n floats)
 * into the caller's workspace ws (dev, >= 256 bytes, 256-byte aligned), copies
 * the count to the host and waits for `stream`: unlike every other entry point
 * this one synchronises.  count_out (host, nullable) receives the count.
 * Returns MFMG_ERR_NUMERIC when the count is not zero, MFMG_ERR_HIP when the
 * stream reports an error (including one left by earlier work on it). */
mfmg_status mfmg_check_finite(const float* x, size_t n, size_t* count_out, void* ws,
                              size_t ws_bytes, void* stream);

/* Static string naming a status. */
const char* mfmg_status_string(mfmg_status status);

/* Thread-local description of the last non-OK status returned on this thread. */
const char* mfmg_last_error_message(void);

/* Kernel timing instrumentation.  While enabled, every launch of the kernel
 * classes below is bracketed by HIP events on its stream; mfmg_timing_read
 * (after the caller has synchronised the stream) returns the number of
 * launches and their summed duration, then clears that class.  Classes:
 *   0 forward GEMM, 1 backward-data GEMM, 2 backward-weight GEMM (with update),
 *   3 dual forward GEMM, 4 dual backward-data GEMM, 5 dual backward-weight GEMM
 *   (with reverse accumulation) computing fewer than three products (first
 *   layer, or no primal gradient), 6 loss head, 7 other elementwise kernels,
 *   8 dual backward-weight GEMM computing all three products G = A^T dZ and
 *   G' = A'^T dZ + A^T dZ' (hidden layers).  Timing covers MLP problems. */
#define MFMG_NUM_KERNEL_CLASSES 9
mfmg_status mfmg_timing_enable(int enable);
mfmg_status mfmg_timing_read(int kernel_class, int* launches, double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* MFMG_H_ */
