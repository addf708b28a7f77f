"""Seeded synthetic inputs with the shapes of P4Q's LLaVA workloads.

This module only *draws* inputs. It holds none of the method's arithmetic (no
quantizer, no scoring, no selection, no GEMM), so both the CPU oracle and the
HIP path can be fed from it without sharing any of the computation under test.

Shapes follow the paper's evaluation setting (Sec. 4.1 and Table 1): LLaVA-1.5
feeds 576 visual tokens to the LLM, LLaVA-NeXT feeds 2880 (five AnyRes tiles of
576, row-newline tokens excluded), retained budgets are 64 / 192 / 320 / 640,
the 7B decoder has hidden 4096 and MLP 11008, and the 13B decoder 5120 / 13824.
The benchmarks themselves (MMMU, GQA, ...) are not used; only their shapes are.

Value recipe (identical for every config):
  * visual features: N(0, 1), then 8 outlier channels (drawn once per config,
    without replacement, shared by all tokens and samples) scaled by 20;
  * text tokens: N(0, 1);
  * query concepts (stand-in for the mean subword embedding of noun j,
    Sec. 3.2): C_j = fp16(0.5 * (text_{2j} + text_{2j+1})), summed in fp32;
  * weights: N(0, 0.02^2), one independent stream per linear;
  * inputs of o_proj / down_proj (stand-ins for the attention output and the
    gated MLP activation): drawn like the visual features, each with its own
    outlier channels;
  * RMSNorm weight of the fused prologue (stand-in, with calibration's
    diagonal scales folded in): 1 + 0.1 N(0, 1);
  * CLS-to-patch attention (stand-in for the vision tower's final-layer
    attention that the Visual Saliency stage reads, Sec. 3.2): per image
    tile of 576 patches and per head (16 heads), a softmax of N(0, 3^2)
    logits over the tile's patches, averaged over the heads; the tiles'
    weights are concatenated (one global ranking over all tiles).
All values are drawn in float32 with numpy's PCG64 and cast to fp16 with
round-to-nearest-even.  The seed of every tensor is
SeedSequence([42, config_id, tensor_id, sample]); 42 echoes the paper's seed.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

SEED = 42

# tensor ids of the seed tree
_T_VIS, _T_TEXT, _T_OUTLIER, _T_OPROJ_IN, _T_DOWN_IN = 0, 1, 2, 3, 4
_T_OPROJ_OUTLIER, _T_DOWN_OUTLIER = 5, 6
_T_CLS = 7               # CLS-to-patch attention stand-in
_T_NORM = 8              # RMSNorm weight (with folded diagonal scales) stand-in
_T_WEIGHT0 = 16          # weights use tensor ids 16 + linear index
_T_GEMV_IN = 32          # decode-step activations

N_OUTLIER = 8
OUTLIER_SCALE = 20.0
WEIGHT_STD = 0.02


@dataclass(frozen=True)
class Linear:
    """One linear layer: y[M, n_out] = x[M, k_in] @ W[n_out, k_in]^T."""
    name: str
    n_out: int
    k_in: int
    # which activation feeds it: "x" (selector output), "attn" (o_proj stand-in)
    # or "mlp" (down_proj stand-in)
    source: str


@dataclass(frozen=True)
class Config:
    cfg_id: int
    name: str
    B: int            # images (samples)
    N: int            # visual tokens per sample
    d: int            # LLM hidden size (= projector output width)
    K: int            # retained visual tokens per sample
    T: int            # text tokens per sample
    J: int            # query concepts per sample
    linears: Tuple[Linear, ...]
    out_dtype: str    # "fp16" | "bf16"
    in_dtype: str = "fp16"
    gemv_M: Tuple[int, ...] = ()

    @property
    def M(self) -> int:
        """Rows of the pruned sequence that the linears run on."""
        return self.B * (self.K + self.T)

    def linear_ops(self) -> int:
        """2*M*n_out*k_in summed over the layer's linears."""
        return sum(2 * self.M * l.n_out * l.k_in for l in self.linears)


def decoder_linears(h: int, f: int) -> Tuple[Linear, ...]:
    """The seven linears of one LLaMA-family decoder layer."""
    return (
        Linear("q_proj", h, h, "x"),
        Linear("k_proj", h, h, "x"),
        Linear("v_proj", h, h, "x"),
        Linear("o_proj", h, h, "attn"),
        Linear("gate_proj", f, h, "x"),
        Linear("up_proj", f, h, "x"),
        Linear("down_proj", h, f, "mlp"),
    )


CONFIGS: Dict[str, Config] = {
    "tiny": Config(0, "tiny-576x4096-k64", B=1, N=576, d=4096, K=64, T=32, J=4,
                   linears=(Linear("proj", 4096, 4096, "x"),), out_dtype="fp16"),
    "llava15_7b": Config(1, "llava1.5-7b-layer", B=1, N=576, d=4096, K=192, T=64, J=4,
                         linears=decoder_linears(4096, 11008), out_dtype="bf16"),
    "next7b_b1_k320": Config(2, "llava-next-7b-b1-k320", B=1, N=2880, d=4096, K=320, T=64,
                             J=4, linears=decoder_linears(4096, 11008), out_dtype="bf16"),
    "next7b_b1_k640": Config(2, "llava-next-7b-b1-k640", B=1, N=2880, d=4096, K=640, T=64,
                             J=4, linears=decoder_linears(4096, 11008), out_dtype="bf16"),
    "next7b_b16": Config(3, "llava-next-7b-b16", B=16, N=2880, d=4096, K=640, T=64, J=4,
                         linears=decoder_linears(4096, 11008), out_dtype="bf16"),
    "stress13b_b8": Config(4, "13b-shape-b8", B=8, N=2880, d=5120, K=640, T=64, J=4,
                           linears=decoder_linears(5120, 13824), out_dtype="bf16",
                           gemv_M=(1, 4, 16)),
}


def _rng(cfg_id: int, tensor_id: int, sample: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([SEED, cfg_id, tensor_id, sample])))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Encode float32 values as bfloat16 bit patterns (round to nearest even).

    Input encoding only (used to hand bf16 tensors to both sides)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def encode(x32: np.ndarray, dtype: str) -> np.ndarray:
    """fp32 -> storage array: float16 array, or uint16 bf16 bit patterns."""
    if dtype == "fp16":
        return x32.astype(np.float16)
    if dtype == "bf16":
        return f32_to_bf16_bits(x32)
    raise ValueError(dtype)


def outlier_channels(cfg_id: int, tensor_id: int, d: int) -> np.ndarray:
    return np.sort(_rng(cfg_id, tensor_id).choice(d, size=N_OUTLIER, replace=False))


def outlier_features(cfg_id: int, tensor_id: int, outlier_tid: int, rows: int, d: int,
                     sample: int = 0, dtype: str = "fp16") -> np.ndarray:
    """rows x d features: N(0,1) with 8 shared outlier channels scaled x20."""
    x = _rng(cfg_id, tensor_id, sample).standard_normal((rows, d), dtype=np.float32)
    x[:, outlier_channels(cfg_id, outlier_tid, d)] *= np.float32(OUTLIER_SCALE)
    return encode(x, dtype)


def visual_features(cfg: Config, sample: int) -> np.ndarray:
    """[N, d] projector-output stand-in for one image."""
    return outlier_features(cfg.cfg_id, _T_VIS, _T_OUTLIER, cfg.N, cfg.d, sample, cfg.in_dtype)


def text_tokens(cfg: Config, sample: int) -> np.ndarray:
    """[T, d] text-token embeddings stand-in for one question."""
    x = _rng(cfg.cfg_id, _T_TEXT, sample).standard_normal((cfg.T, cfg.d), dtype=np.float32)
    return encode(x, cfg.in_dtype)


def concepts_from_text(text_f32: np.ndarray, J: int, dtype: str) -> np.ndarray:
    """[J, d] concept rows: mean of two consecutive text rows, summed in fp32."""
    assert text_f32.shape[0] >= 2 * J, "need two text rows per concept"
    c = (text_f32[0:2 * J:2] + text_f32[1:2 * J:2]) * np.float32(0.5)
    return encode(c.astype(np.float32), dtype)


def to_f32(a: np.ndarray, dtype: str) -> np.ndarray:
    """Decode a storage array (fp16, or bf16 bit patterns) to float32 exactly."""
    if dtype == "fp16":
        return a.astype(np.float32)
    return (a.astype(np.uint32) << 16).view(np.float32)


CLS_HEADS = 16
CLS_LOGIT_STD = 3.0
PATCHES_PER_TILE = 576


def cls_attention(cfg_id: int, N: int, sample: int = 0) -> np.ndarray:
    """[N] fp32 head-averaged CLS-to-patch attention weights of one image.

    Input synthesis only: softmax over each tile's patches of seeded logits,
    computed in float64 and rounded to fp32."""
    g = _rng(cfg_id, _T_CLS, sample)
    out = np.empty(N, dtype=np.float64)
    for t0 in range(0, N, PATCHES_PER_TILE):
        n = min(PATCHES_PER_TILE, N - t0)
        z = g.standard_normal((CLS_HEADS, n)) * CLS_LOGIT_STD
        z -= z.max(axis=1, keepdims=True)
        e = np.exp(z)
        out[t0:t0 + n] = (e / e.sum(axis=1, keepdims=True)).mean(axis=0)
    return out.astype(np.float32)


@dataclass
class SelectorInputs:
    vis: np.ndarray        # [B, N, d]
    concepts: np.ndarray   # [B, J, d]
    text: np.ndarray       # [B, T, d]
    dtype: str


def selector_inputs(cfg: Config, samples: Optional[List[int]] = None) -> SelectorInputs:
    samples = list(range(cfg.B)) if samples is None else samples
    vis, con, txt = [], [], []
    for b in samples:
        vis.append(visual_features(cfg, b))
        t = text_tokens(cfg, b)
        txt.append(t)
        con.append(concepts_from_text(to_f32(t, cfg.in_dtype), cfg.J, cfg.in_dtype))
    return SelectorInputs(np.stack(vis), np.stack(con), np.stack(txt), cfg.in_dtype)


def weight(cfg: Config, li: int, dtype: str = "fp16") -> np.ndarray:
    """[n_out, k_in] weight of linear li: N(0, 0.02^2)."""
    lin = cfg.linears[li]
    w = _rng(cfg.cfg_id, _T_WEIGHT0 + li).standard_normal((lin.n_out, lin.k_in),
                                                          dtype=np.float32)
    w *= np.float32(WEIGHT_STD)
    return encode(w, dtype)


def attn_standin(cfg: Config, rows: Optional[int] = None) -> np.ndarray:
    """[M, d] input of o_proj (attention-output stand-in)."""
    rows = cfg.M if rows is None else rows
    return outlier_features(cfg.cfg_id, _T_OPROJ_IN, _T_OPROJ_OUTLIER, rows, cfg.d, 0,
                            cfg.in_dtype)


def mlp_standin(cfg: Config, rows: Optional[int] = None) -> np.ndarray:
    """[M, f] input of down_proj (gated-MLP-activation stand-in)."""
    rows = cfg.M if rows is None else rows
    f = [l.k_in for l in cfg.linears if l.source == "mlp"]
    width = f[0] if f else cfg.d
    return outlier_features(cfg.cfg_id, _T_DOWN_IN, _T_DOWN_OUTLIER, rows, width, 0,
                            cfg.in_dtype)


def norm_weight(cfg: Config, d: Optional[int] = None) -> np.ndarray:
    """[d] RMSNorm weight stand-in (the per-channel slot into which the
    calibration's diagonal scales fold): 1 + 0.1 N(0, 1), storage dtype."""
    d = cfg.d if d is None else d
    g = _rng(cfg.cfg_id, _T_NORM).standard_normal(d, dtype=np.float32)
    return encode(np.float32(1.0) + np.float32(0.1) * g, cfg.in_dtype)


def gemv_activations(cfg: Config, M: int, k_in: int) -> np.ndarray:
    """[M, k_in] decode-step activations with the same outlier recipe."""
    return outlier_features(cfg.cfg_id, _T_GEMV_IN + M, _T_OUTLIER, M, k_in, 0, cfg.in_dtype)


def random_features(seed: int, rows: int, cols: int, dtype: str = "fp16",
                    outliers: int = N_OUTLIER, scale: float = OUTLIER_SCALE,
                    std: float = 1.0) -> np.ndarray:
    """Free-form seeded features for edge-case tests: N(0, std^2) with outliers."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED, 1000, seed])))
    x = g.standard_normal((rows, cols), dtype=np.float32) * np.float32(std)
    if outliers and cols >= outliers:
        ch = g.choice(cols, size=outliers, replace=False)
        x[:, ch] *= np.float32(scale)
    return encode(x, dtype)


@dataclass
class CalibProblem:
    """Inputs of one calibration step of one linear (see calib_problem)."""
    x: np.ndarray          # [M, K] storage dtype: block input rows of the pruned sequence
    w: np.ndarray          # [N, K] storage dtype: the frozen full-precision weight
    target: np.ndarray     # [M, N] float32: the full-precision layer output
    sigma: np.ndarray      # [K] float32 > 0: diagonal channel scales
    clip_a: float          # activation clipping factor
    clip_w: np.ndarray     # [N] float32: weight clipping factors
    dtype: str


def calib_problem(seed: int, M: int, N: int, K: int, dtype: str = "fp16",
                  clip_a: float = 0.9, w_std: float = WEIGHT_STD) -> CalibProblem:
    """Seeded stand-in for one calibration step on a pruned sequence
    (Sec. 3.3, Appendix B.3: block inputs captured after the selector, frozen
    weights, learnable diagonal scales and clipping factors mid-optimization).

    * x: the activation recipe above (N(0, 1), 8 outlier channels x20);
    * w: N(0, w_std^2);
    * sigma: exp(0.3 N(0, 1)), times 20^0.3 on x's outlier channels (the
      direction in which scales initialized from activation and weight ranges
      start: outlier channels are divided down);
    * clip_w: U(0.75, 1) per output channel;
    * target: x @ w^T in float64 from the stored values, rounded to fp32.
    No quantizer, gradient or calibration arithmetic happens here."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED, 2000, seed])))
    x32 = g.standard_normal((M, K), dtype=np.float32)
    ch = g.choice(K, size=min(N_OUTLIER, K), replace=False)
    x32[:, ch] *= np.float32(OUTLIER_SCALE)
    w32 = g.standard_normal((N, K), dtype=np.float32) * np.float32(w_std)
    sigma = np.exp(np.float32(0.3) * g.standard_normal(K, dtype=np.float32)).astype(np.float32)
    sigma[ch] *= np.float32(OUTLIER_SCALE ** 0.3)
    clip_w = g.uniform(0.75, 1.0, N).astype(np.float32)
    x = encode(x32, dtype)
    w = encode(w32, dtype)
    xf, wf = to_f32(x, dtype).astype(np.float64), to_f32(w, dtype).astype(np.float64)
    target = (xf @ wf.T).astype(np.float32)
    return CalibProblem(x, w, target, sigma.astype(np.float32), float(clip_a), clip_w, dtype)


@dataclass
class CalibBlockProblem:
    x: np.ndarray          # [M, d] block input (storage dtype)
    weights: dict          # "qkv" [3d, d], "o" [d, d], "gu" [2f, d], "down" [d, f]
    gamma1: np.ndarray     # [d]
    gamma2: np.ndarray     # [d]
    sigma: dict            # per group: fp32 [input width]
    clip_a: dict           # per group: float
    clip_w: dict           # per group: fp32 [output width]
    H: int
    dtype: str


def calib_block_problem(seed: int, M: int, d: int, f: int, H: int,
                        dtype: str = "fp16") -> CalibBlockProblem:
    """Seeded stand-in for one block-level calibration step (Sec. 3.3,
    Appendix B.3) on a pruned sequence of M tokens: a decoder block of
    hidden size d, MLP width f and H heads.

    * x: the activation recipe (N(0, 1), 8 outlier channels x20);
    * weights: N(0, 0.02^2) for q|k|v, o, gate|up, down;
    * gamma1, gamma2: 1 + 0.1 N(0, 1) (RMSNorm weights);
    * sigma: exp(0.3 N(0, 1)) per input channel of each linear group, times
      20^0.3 on x's outlier channels for the q|k|v group (whose input keeps
      the block input's outlier channels through the RMSNorm);
    * clip_a: 0.9, 0.95, 0.85, 0.9 (q|k|v, o, gate|up, down); clip_w:
      U(0.75, 1) per output channel.
    The target (the full-precision block's output) is not drawn: it is the
    block computed without quantization.  No block arithmetic happens here."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED, 3000, seed])))
    x32 = g.standard_normal((M, d), dtype=np.float32)
    ch = g.choice(d, size=min(N_OUTLIER, d), replace=False)
    x32[:, ch] *= np.float32(OUTLIER_SCALE)
    shapes = {"qkv": (3 * d, d), "o": (d, d), "gu": (2 * f, d), "down": (d, f)}
    weights = {k: encode(g.standard_normal(s, dtype=np.float32) * np.float32(WEIGHT_STD), dtype)
               for k, s in shapes.items()}
    gam = [encode((1.0 + 0.1 * g.standard_normal(d)).astype(np.float32), dtype) for _ in range(2)]
    sigma, clip_w = {}, {}
    for k, (n_out, k_in) in shapes.items():
        s_ = np.exp(np.float32(0.3) * g.standard_normal(k_in, dtype=np.float32)).astype(np.float32)
        if k == "qkv":
            s_[ch] *= np.float32(OUTLIER_SCALE ** 0.3)
        sigma[k] = s_
        clip_w[k] = g.uniform(0.75, 1.0, n_out).astype(np.float32)
    clip_a = {"qkv": 0.9, "o": 0.95, "gu": 0.85, "down": 0.9}
    return CalibBlockProblem(encode(x32, dtype), weights, gam[0], gam[1], sigma, clip_a, clip_w,
                             H, dtype)
