"""Seeded synthetic workloads for the meta-gradient path.

This module holds problem shapes, hyperparameters, the flat parameter layout
and seeded input draws.  It holds none of the method's arithmetic: no loss,
no gradient, no update rule.  Both the float64 oracle and the GPU path read
their inputs from here, so that both see bit-identical float32 arrays.

Problem statement (Section 2.1, eq. bptt_bilevel): T inner steps
(theta_{i+1}, upsilon_{i+1}) = Phi(theta_i, upsilon_i, eta, x_i) on training
batches x_0..x_{T-1}, then the outer loss V(theta_T, val).  The paper names no
dataset (it uses next-token prediction on language data, Section 5); every
array here is a seeded synthetic stand-in with the shape and distribution
listed per workload.

Seeds: np.random.SeedSequence(250500793, spawn_key=(cfg_id,)), children in the
order [theta0, eta0, train, val, extra].  The train child spawns one
generator per inner step, so batch t does not depend on T.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

ROOT_SEED = 250500793

# enum values shared with include/mfmg.h (plain integers, no arithmetic)
ACT_TANH, ACT_GELU, ACT_RELU, ACT_NONE = 0, 1, 2, 3
LOSS_MSE, LOSS_CE = 0, 1
# squared error after the M-step map y_i = i (2 + sin y_{i-1})^cos y_{i-1} of Section 3.2
# (eq. motivational_example), averaged over the outputs
LOSS_MAPMSE = 2
OPT_SGD, OPT_ADAM = 0, 1
META_LOGLR_PER_PARAM, META_LOGLR_PER_LAYER_WD, META_EXAMPLE_WEIGHT_LOGITS, META_TOKEN_WEIGHT_MLP = 0, 1, 2, 3
META_MAML = 4   # eta is the initial parameter vector theta_0 (SGD, fixed inner lr)
PREC_FP32, PREC_BF16 = 0, 1
KIND_MLP, KIND_TRANSFORMER = 0, 1

ACT_NAMES = {ACT_TANH: "tanh", ACT_GELU: "gelu", ACT_RELU: "relu", ACT_NONE: "none"}


@dataclasses.dataclass(frozen=True)
class Config:
    """One bilevel problem: inner model, inner loss, inner optimiser, meta-parameters."""

    name: str
    cfg_id: int
    kind: int = KIND_MLP
    widths: Tuple[int, ...] = ()          # MLP: widths[0] = input dim, widths[-1] = outputs
    act: int = ACT_RELU
    loss: int = LOSS_CE
    optimizer: int = OPT_SGD
    meta: int = META_LOGLR_PER_PARAM
    precision: int = PREC_FP32
    has_bias: bool = True
    rows: int = 128                        # training rows per inner step (sequences for the transformer)
    val_rows: int = 128
    T: int = 4
    init: str = "he"                       # "xavier" | "he" | "normal0.1" | "normal0.02"
    sgd_lr: float = 0.1                    # fixed inner learning rate (META_EXAMPLE_WEIGHT_LOGITS / TOKEN)
    adam_b1: float = 0.9
    adam_b2: float = 0.999
    adam_eps: float = 1e-8
    loglr_init: float = math.log(0.01)
    wd_init: float = 1e-4
    map_steps: int = 0                     # M of the toy map (LOSS_MAPMSE)
    ckpt_segment: int = 0                  # GPU static-memory segments (0: keep every step)
    fused_attention: int = 0               # transformer, bf16: fused causal attention (no S^2 buffers)
    block_remat: int = 0                   # transformer: recompute each block in its backward
    # transformer
    d_model: int = 0
    n_heads: int = 0
    d_ff: int = 0
    vocab: int = 0
    seq: int = 0
    n_blocks: int = 0
    meta_hidden: int = 0
    ln_eps: float = 1e-5
    rope_base: float = 10000.0
    zipf_s: float = 1.1

    def with_(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)

    @property
    def n_layers(self) -> int:
        return len(self.widths) - 1

    @property
    def n_out(self) -> int:
        return self.vocab if self.kind == KIND_TRANSFORMER else self.widths[-1]


# --------------------------------------------------------------------------------------
# The five workloads (sizes, activations, losses and meta-parameters of each).
# --------------------------------------------------------------------------------------
C1 = Config(name="c1_linreg", cfg_id=1, widths=(64, 1), act=ACT_NONE, loss=LOSS_MSE,
            optimizer=OPT_SGD, meta=META_LOGLR_PER_PARAM, precision=PREC_FP32, has_bias=False,
            rows=256, val_rows=256, T=4, init="normal0.1")
C2 = Config(name="c2_mlp_tanh_lossweights", cfg_id=2, widths=(784, 256, 10), act=ACT_TANH,
            loss=LOSS_CE, optimizer=OPT_SGD, meta=META_EXAMPLE_WEIGHT_LOGITS,
            precision=PREC_FP32, rows=128, val_rows=512, T=8, init="xavier", sgd_lr=0.1)
C3 = Config(name="c3_mlp_gelu_adam", cfg_id=3, widths=(1024, 1024, 1024, 1024, 100), act=ACT_GELU,
            loss=LOSS_CE, optimizer=OPT_ADAM, meta=META_LOGLR_PER_LAYER_WD, precision=PREC_BF16,
            rows=512, val_rows=1024, T=16, init="he", loglr_init=math.log(1e-3), wd_init=1e-4)
C4 = Config(name="c4_transformer_tokenweights", cfg_id=4, kind=KIND_TRANSFORMER, loss=LOSS_CE,
            optimizer=OPT_SGD, meta=META_TOKEN_WEIGHT_MLP, precision=PREC_BF16, has_bias=False,
            rows=16, val_rows=16, T=8, init="normal0.02", sgd_lr=0.1, act=ACT_GELU,
            d_model=512, n_heads=8, d_ff=2048, vocab=8192, seq=256, n_blocks=4, meta_hidden=128)
C5 = Config(name="c5_mlp_relu_8x4096", cfg_id=5, widths=(4096,) * 8 + (1000,), act=ACT_RELU,
            loss=LOSS_CE, optimizer=OPT_SGD, meta=META_LOGLR_PER_PARAM, precision=PREC_BF16,
            rows=1024, val_rows=1024, T=8, init="he")
C5_TS = (4, 8, 16, 32)

CONFIGS: Dict[str, Config] = {c.name: c for c in (C1, C2, C3, C4, C5)}

# MAML on the config-5 network: eta = theta_0, SGD at a fixed rate
MAML5 = C5.with_(name="maml_mlp_relu_8x4096", cfg_id=6, meta=META_MAML, sgd_lr=0.05)

# The paper's motivating example (Section 3.2): y_0 = x w with x of B x D and
# w of D x D, M map steps, mean squared error against standard normal targets,
# MAML (w_0 = eta), T = 2 inner SGD steps at rate 1e-3, B = 1024, D = 4096.
TOY = Config(name="toy_mstep_map", cfg_id=7, widths=(4096, 4096), act=ACT_NONE,
             loss=LOSS_MAPMSE, optimizer=OPT_SGD, meta=META_MAML, precision=PREC_FP32,
             has_bias=False, rows=1024, val_rows=1024, T=2, init="normal1", sgd_lr=1e-3,
             map_steps=8)
TOY_MS = (1, 2, 4, 8, 16, 32, 64)

# Long contexts on the config-4 decoder (the paper sweeps sequence lengths up to
# 8192): 8192 tokens per batch as S x (8192 / S) sequences, T = 2.
C4_LONG_S = (2048, 4096, 8192)

TOY_SMALL_BASE = Config(name="toy", cfg_id=0, act=ACT_NONE, loss=LOSS_MAPMSE, optimizer=OPT_SGD,
                        meta=META_MAML, precision=PREC_FP32, has_bias=False, T=2,
                        init="normal0.1")

# Reduced variants for parity tests: same structure, sizes the oracle finishes in
# seconds, each spanning several GEMM tiles plus a ragged tail.
SMALL: Dict[str, Config] = {
    "c1_small": C1.with_(name="c1_small", cfg_id=101, rows=100, val_rows=77, T=3, widths=(37, 1)),
    # batches too large to stage in LDS (read from global memory), rows past 256
    "c1_wide": C1.with_(name="c1_wide", cfg_id=127, rows=1000, val_rows=700, T=3, widths=(130, 1)),
    # checkpoints too many for LDS ((T + 1) d > 4096), staged batches
    "c1_long": C1.with_(name="c1_long", cfg_id=128, rows=120, val_rows=128, T=33, widths=(131, 1)),
    # 16-byte loads (d % 4 == 0) whose steps wrap rows; the validation batch is unstaged
    "c1_vec": C1.with_(name="c1_vec", cfg_id=129, rows=150, val_rows=200, T=4, widths=(100, 1)),
    # batches held in registers (d <= 64, d % 4 == 0, at most 256 rows): partial
    # 16-lane rows (9 of 16 groups) and partial row slots in training and validation
    "c1_reg": C1.with_(name="c1_reg", cfg_id=134, rows=200, val_rows=250, T=5, widths=(36, 1)),
    # registers with the checkpoints in global memory ((T + 1) d > 4096)
    "c1_reg_long": C1.with_(name="c1_reg_long", cfg_id=135, rows=40, val_rows=24, T=64,
                            widths=(64, 1)),
    "c2_small": C2.with_(name="c2_small", cfg_id=102, widths=(150, 70, 13), rows=70, val_rows=90, T=3),
    # a float32 first layer with a long contraction and few output tiles: the
    # training forward products run split-K (8 slices of 76), the validation
    # ones (more tiles) do not
    "c2_splitk": C2.with_(name="c2_splitk", cfg_id=126, widths=(608, 72, 10), rows=36,
                          val_rows=300, T=3),
    # a float32 output layer over few rows: 90 x 20 outputs (2 tiles of 64 x 64; wider
    # than the 16 columns of the narrow tiles) contracting over 320, split into 5 k
    # slices of 64 (ragged rows in the last tile)
    "c2_narrow": C2.with_(name="c2_narrow", cfg_id=136, widths=(96, 320, 20), rows=90,
                          val_rows=70, T=3),
    "c3_small": C3.with_(name="c3_small", cfg_id=103, widths=(136, 200, 72, 10), rows=150,
                         val_rows=96, T=4),
    "c5_small": C5.with_(name="c5_small", cfg_id=105, widths=(200, 300, 260, 37), rows=130,
                         val_rows=70, T=3),
    # a tall first layer: its backward-weight product has more tile rows (65 of
    # 64) than bias entries per tile column (24), so each tile sums at most one
    # bias row and some none
    "c5_tall": C5.with_(name="c5_tall", cfg_id=133, widths=(4104, 24, 10), rows=64, val_rows=40,
                        T=2),
    # 50 steps: more operand sets (51 checkpoints + 2 tangents) than one launch of
    # the padding-zeroing kernel takes; the 37-wide output layer contracts over 40
    "c5_small_long": C5.with_(name="c5_small_long", cfg_id=132, widths=(200, 300, 260, 37),
                              rows=130, val_rows=70, T=50),
    "c5_tanh_fp32": C5.with_(name="c5_tanh_fp32", cfg_id=106, widths=(40, 50, 7), act=ACT_TANH,
                             precision=PREC_FP32, rows=33, val_rows=20, T=3),
    "c5_gelu_fp32": C5.with_(name="c5_gelu_fp32", cfg_id=107, widths=(40, 50, 30, 7), act=ACT_GELU,
                             precision=PREC_FP32, rows=33, val_rows=20, T=3),
    "c3_fp32": C3.with_(name="c3_fp32", cfg_id=108, widths=(40, 48, 9), precision=PREC_FP32,
                        rows=36, val_rows=25, T=3, loglr_init=math.log(1e-2)),
    # large enough that every layer's products use the 128 x 128 bf16 tiles
    "c5_mid": C5.with_(name="c5_mid", cfg_id=109, widths=(2048, 2048, 2048, 64), rows=2048,
                       val_rows=512, T=2),
    # every dimension a multiple of 8 but not of the tile sizes: ragged row,
    # column and k tails on the direct-to-LDS GEMM path (64 and 128 tiles)
    "c5_r8": C5.with_(name="c5_r8", cfg_id=110, widths=(200, 264, 136, 40), rows=200,
                      val_rows=136, T=3),
    "c5_mid_r8": C5.with_(name="c5_mid_r8", cfg_id=111, widths=(1544, 2056, 1032, 40), rows=1544,
                          val_rows=520, T=2),
    # MAML: eta is theta_0 (fixed-rate SGD inside)
    "c5_maml_fp32": C5.with_(name="c5_maml_fp32", cfg_id=114, widths=(40, 50, 30, 7),
                             act=ACT_TANH, precision=PREC_FP32, meta=META_MAML, sgd_lr=0.1,
                             has_bias=True, rows=33, val_rows=20, T=3),
    "c5_maml": C5.with_(name="c5_maml", cfg_id=115, widths=(200, 264, 136, 40), meta=META_MAML,
                        sgd_lr=0.1, rows=200, val_rows=136, T=3),
    "c5_maml_r8_fp32": C5.with_(name="c5_maml_r8_fp32", cfg_id=116, widths=(200, 264, 136, 40),
                                meta=META_MAML, sgd_lr=0.1, precision=PREC_FP32, rows=200,
                                val_rows=136, T=3),
    # the motivating example (one D x D layer, the M-step map, MAML), small
    "toy_small": TOY_SMALL_BASE.with_(name="toy_small", cfg_id=117, widths=(64, 48), rows=24,
                                      val_rows=16, map_steps=3, sgd_lr=0.05),
    "toy_mid": TOY_SMALL_BASE.with_(name="toy_mid", cfg_id=118, widths=(200, 136), rows=100,
                                    val_rows=40, map_steps=2, sgd_lr=0.02),
    # more 128 x 128 output tiles than compute units (two tiles for some
    # persistent workgroups), ragged rows, columns and k
    "c5_rag2": C5.with_(name="c5_rag2", cfg_id=112, widths=(2056, 2312, 40), rows=520,
                        val_rows=264, T=2),
    "c4_small": C4.with_(name="c4_small", cfg_id=104, d_model=64, n_heads=4, d_ff=128, vocab=97,
                         seq=24, rows=3, val_rows=2, n_blocks=2, meta_hidden=16, T=2),
    # a long context (2 x 1024 tokens): attention of 1024 x 1024 per head
    "c4_long": C4.with_(name="c4_long", cfg_id=119, d_model=64, n_heads=2, d_ff=128, vocab=97,
                        seq=1024, rows=2, val_rows=1, n_blocks=1, meta_hidden=16, T=2),
    # enough tokens (8 x 160) for the split-K weight gradients, an odd vocabulary
    "c4_mid": C4.with_(name="c4_mid", cfg_id=113, d_model=128, n_heads=4, d_ff=256, vocab=301,
                       seq=160, rows=8, val_rows=4, n_blocks=2, meta_hidden=32, T=2),
    # fused attention (head dim 64, bf16): three 64-query blocks per sequence,
    # so diagonal and off-diagonal key blocks; and a 1024-token context
    "c4_fused": C4.with_(name="c4_fused", cfg_id=120, d_model=128, n_heads=2, d_ff=256, vocab=97,
                         seq=192, rows=3, val_rows=2, n_blocks=2, meta_hidden=16, T=2,
                         fused_attention=1),
    "c4_fused64": C4.with_(name="c4_fused64", cfg_id=125, d_model=128, n_heads=2, d_ff=256,
                           vocab=97, seq=64, rows=4, val_rows=2, n_blocks=2, meta_hidden=16,
                           T=2, fused_attention=1),
    "c4_fused128": C4.with_(name="c4_fused128", cfg_id=122, d_model=128, n_heads=2, d_ff=256,
                            vocab=97, seq=128, rows=3, val_rows=2, n_blocks=2, meta_hidden=16,
                            T=2, fused_attention=1),
    # d = 256: the 16-byte LayerNorm kernels writing bf16 operand rows directly
    # (2 x 16 tokens), and with 3 x 12 tokens (not a multiple of 8) their float32 path
    "c4_d256": C4.with_(name="c4_d256", cfg_id=123, d_model=256, n_heads=4, d_ff=512, vocab=97,
                        seq=16, rows=2, val_rows=2, n_blocks=1, meta_hidden=16, T=2),
    "c4_d256_n12": C4.with_(name="c4_d256_n12", cfg_id=124, d_model=256, n_heads=4, d_ff=512,
                            vocab=97, seq=12, rows=3, val_rows=2, n_blocks=1, meta_hidden=16,
                            T=2),
    "c4_long_fused": C4.with_(name="c4_long_fused", cfg_id=121, d_model=128, n_heads=2, d_ff=256,
                              vocab=97, seq=1024, rows=2, val_rows=1, n_blocks=1, meta_hidden=16,
                              T=2, fused_attention=1),
}


# Full-width slices of the 8 x 4096 network: its 4096-wide layers and 1024-row
# batches with bf16 operands, but two or three weight matrices instead of eight.
# Rounding alone moves their meta-gradients by well under 2e-2 (the deep network
# amplifies one bf16 ulp of an activation into percent-level changes), so every
# full-size product shape is gated at the plain bf16 tolerance on these.
SLICES: Dict[str, Config] = {
    "c5_slice2": C5.with_(name="c5_slice2", cfg_id=130, widths=(4096, 4096, 1000)),
    "c5_slice3": C5.with_(name="c5_slice3", cfg_id=131, widths=(4096, 4096, 4096, 1000)),
}


def get(name: str) -> Config:
    """A workload by name: the five configurations, their reduced variants, the
    full-width slices, MAML on config 5 and the motivating example."""
    for table in (CONFIGS, SMALL, SLICES, {MAML5.name: MAML5, TOY.name: TOY}):
        if name in table:
            return table[name]
    raise KeyError(name)


# --------------------------------------------------------------------------------------
# Flat parameter layout (the ABI's theta layout).
# --------------------------------------------------------------------------------------
def theta_layout(cfg: Config) -> List[Tuple[str, int, Tuple[int, ...]]]:
    """(name, offset, shape) of every tensor packed in the flat theta array.

    MLP: per layer l, W_l row-major [in][out], then b_l [out] if has_bias.
    Transformer: emb [V][d]; per block: ln1_g, ln1_b [d], wqkv [d][3d], wo [d][d],
    ln2_g, ln2_b [d], w1 [d][ff], w2 [ff][d]; then lnf_g, lnf_b [d]; unemb [d][V].
    """
    out: List[Tuple[str, int, Tuple[int, ...]]] = []
    off = 0

    def add(name, shape):
        nonlocal off
        out.append((name, off, tuple(shape)))
        off += int(np.prod(shape))

    if cfg.kind == KIND_MLP:
        for l in range(cfg.n_layers):
            add(f"W{l}", (cfg.widths[l], cfg.widths[l + 1]))
            if cfg.has_bias:
                add(f"b{l}", (cfg.widths[l + 1],))
    else:
        d, ff, V = cfg.d_model, cfg.d_ff, cfg.vocab
        add("emb", (V, d))
        for b in range(cfg.n_blocks):
            add(f"ln1_g{b}", (d,))
            add(f"ln1_b{b}", (d,))
            add(f"wqkv{b}", (d, 3 * d))
            add(f"wo{b}", (d, d))
            add(f"ln2_g{b}", (d,))
            add(f"ln2_b{b}", (d,))
            add(f"w1{b}", (d, ff))
            add(f"w2{b}", (ff, d))
        add("lnf_g", (d,))
        add("lnf_b", (d,))
        add("unemb", (d, V))
    return out


def n_theta(cfg: Config) -> int:
    lay = theta_layout(cfg)
    name, off, shape = lay[-1]
    return off + int(np.prod(shape))


def meta_layout(cfg: Config) -> List[Tuple[str, int, Tuple[int, ...]]]:
    """Layout of the flat eta array."""
    if cfg.meta in (META_LOGLR_PER_PARAM, META_MAML):
        return theta_layout(cfg)
    if cfg.meta == META_LOGLR_PER_LAYER_WD:
        return [(f"loglr{l}", l, ()) for l in range(cfg.n_layers)] + [("wd", cfg.n_layers, ())]
    if cfg.meta == META_EXAMPLE_WEIGHT_LOGITS:
        return [("logits", 0, (cfg.T, cfg.rows))]
    if cfg.meta == META_TOKEN_WEIGHT_MLP:
        d, h = cfg.d_model, cfg.meta_hidden
        return [("mW1", 0, (d, h)), ("mb1", d * h, (h,)), ("mw2", d * h + h, (h, 1)),
                ("mb2", d * h + 2 * h, (1,))]
    raise ValueError(cfg.meta)


def n_eta(cfg: Config) -> int:
    if cfg.meta in (META_LOGLR_PER_PARAM, META_MAML):
        return n_theta(cfg)
    if cfg.meta == META_LOGLR_PER_LAYER_WD:
        return cfg.n_layers + 1
    if cfg.meta == META_EXAMPLE_WEIGHT_LOGITS:
        return cfg.T * cfg.rows
    d, h = cfg.d_model, cfg.meta_hidden
    return d * h + h + h + 1


def n_opt_state(cfg: Config) -> int:
    return 2 * n_theta(cfg) if cfg.optimizer == OPT_ADAM else 0


# --------------------------------------------------------------------------------------
# Seeded draws.
# --------------------------------------------------------------------------------------
def _children(cfg: Config):
    ss = np.random.SeedSequence(ROOT_SEED, spawn_key=(cfg.cfg_id,))
    return ss.spawn(5)


def _init_std(cfg: Config, shape) -> float:
    if cfg.init == "normal0.1":
        return 0.1
    if cfg.init == "normal0.02":
        return 0.02
    if cfg.init == "normal1":
        return 1.0
    fan_in, fan_out = shape[0], shape[1]
    if cfg.init == "xavier":
        return math.sqrt(2.0 / (fan_in + fan_out))
    if cfg.init == "he":
        return math.sqrt(2.0 / fan_in)
    raise ValueError(cfg.init)


def make_theta0(cfg: Config) -> np.ndarray:
    rng = np.random.default_rng(_children(cfg)[0])
    theta = np.zeros(n_theta(cfg), dtype=np.float32)
    for name, off, shape in theta_layout(cfg):
        size = int(np.prod(shape))
        if cfg.kind == KIND_TRANSFORMER and name.startswith(("ln1_g", "ln2_g", "lnf_g")):
            theta[off:off + size] = 1.0
        elif len(shape) == 2 or name == "emb":
            std = _init_std(cfg, shape)
            theta[off:off + size] = (std * rng.standard_normal(size)).astype(np.float32)
        # biases and LayerNorm betas stay 0
    return theta


def make_eta(cfg: Config) -> np.ndarray:
    if cfg.meta == META_MAML:
        return make_theta0(cfg)
    if cfg.meta == META_LOGLR_PER_PARAM:
        return np.full(n_theta(cfg), cfg.loglr_init, dtype=np.float32)
    if cfg.meta == META_LOGLR_PER_LAYER_WD:
        e = np.full(cfg.n_layers + 1, cfg.loglr_init, dtype=np.float32)
        e[-1] = cfg.wd_init
        return e
    if cfg.meta == META_EXAMPLE_WEIGHT_LOGITS:
        return np.zeros(cfg.T * cfg.rows, dtype=np.float32)
    # token-weight meta-MLP: Xavier-normal weights, zero biases
    rng = np.random.default_rng(_children(cfg)[1])
    eta = np.zeros(n_eta(cfg), dtype=np.float32)
    for name, off, shape in meta_layout(cfg):
        size = int(np.prod(shape))
        if len(shape) == 2:
            std = math.sqrt(2.0 / (shape[0] + shape[1]))
            eta[off:off + size] = (std * rng.standard_normal(size)).astype(np.float32)
    return eta


def _zipf_tokens(rng, cfg: Config, shape) -> np.ndarray:
    k = np.arange(1, cfg.vocab + 1, dtype=np.float64)
    p = k ** (-cfg.zipf_s)
    p /= p.sum()
    return rng.choice(cfg.vocab, size=shape, p=p).astype(np.int32)


def _wstar(cfg: Config) -> np.ndarray:
    rng = np.random.default_rng(_children(cfg)[4])
    return rng.standard_normal(cfg.widths[0])


def _draw_batch(cfg: Config, rng, rows: int):
    if cfg.kind == KIND_TRANSFORMER:
        return _zipf_tokens(rng, cfg, (rows, cfg.seq + 1)), None
    x = rng.standard_normal((rows, cfg.widths[0])).astype(np.float32)
    if cfg.loss == LOSS_MAPMSE:   # the toy task: standard normal inputs and targets
        return x, rng.standard_normal((rows, cfg.widths[-1])).astype(np.float32)
    if cfg.loss == LOSS_MSE:
        noise = rng.standard_normal((rows, cfg.widths[-1]))
        y = (x.astype(np.float64) @ _wstar(cfg).reshape(-1, 1) + 0.1 * noise).astype(np.float32)
        if cfg.widths[-1] != 1:
            raise ValueError("MSE workloads have one output")
    else:
        y = rng.integers(0, cfg.widths[-1], size=rows).astype(np.int32)
    return x, y


def make_train_batch(cfg: Config, t: int):
    """Training batch x_t (0-based inner step t)."""
    child = _children(cfg)[2]
    rng = np.random.default_rng(child.spawn(t + 1)[t])
    return _draw_batch(cfg, rng, cfg.rows)


def make_val_batch(cfg: Config):
    rng = np.random.default_rng(_children(cfg)[3])
    return _draw_batch(cfg, rng, cfg.val_rows)


def make_inputs(cfg: Config, T: Optional[int] = None) -> dict:
    """All inputs of one meta-gradient: theta0, eta, T training batches, val batch."""
    T = cfg.T if T is None else T
    batches = [make_train_batch(cfg, t) for t in range(T)]
    vx, vy = make_val_batch(cfg)
    return {
        # with MAML the starting point is eta; theta0 is then unused (zeros)
        "theta0": (np.zeros(n_theta(cfg), dtype=np.float32) if cfg.meta == META_MAML
                   else make_theta0(cfg)),
        "eta": make_eta(cfg),
        "opt_state0": (np.zeros(n_opt_state(cfg), dtype=np.float32)
                       if cfg.optimizer == OPT_ADAM else None),
        "train_x": [b[0] for b in batches],
        "train_y": [b[1] for b in batches],
        "val_x": vx,
        "val_y": vy,
        "T": T,
    }


def random_direction(n: int, seed: int) -> np.ndarray:
    """Seeded float32 N(0,1) vector, e.g. a tangent v for HVP tests."""
    return np.random.default_rng(np.random.SeedSequence(ROOT_SEED, spawn_key=(9000 + seed,))) \
        .standard_normal(n).astype(np.float32)
