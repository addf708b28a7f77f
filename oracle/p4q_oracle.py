"""P4Q CPU oracle -- TEST INFRASTRUCTURE, not part of the product.

A plain, slow, obviously-correct CPU implementation of what the P4Q hot path
computes, written from the paper's definitions.  Only the test-suite, the
smoke check and the benchmark's CPU-baseline leg may import or call it; the
HIP library never does, and this module shares no code with it.

Conventions
-----------
* fl32(.) is IEEE binary32 with round-to-nearest-even.  NumPy float32 array
  arithmetic (x / s, a * b) is exactly that on x86-64 (SSE, no fast-math); the
  self-tests pin it against exact rational arithmetic.
* rne(.) rounds half to even (``np.rint``).
* Integers (codes, dot products, accumulators) are exact: int64 or Python int.
* fp16 data are numpy float16; bf16 data are uint16 bit patterns.

Paper anchors (P4Q, "Co-designing Token Pruning and Quantization for VLM
Acceleration"):
* Sec. 3.2, Eq. (p4q_progressive_selection): the selector ranks visual tokens
  by CosSim between fake-quantized copies of the projector features and of the
  query-concept embeddings; the original FP16 rows go forward.
* Sec. 3.2 (Query Relevance paragraph): per-concept ranking, each concept keeps
  its highest-scoring tokens within its quota.
* Appendix A (experimental details) and Appendix B.3 (PTQ calibration
  details): W4A4 = symmetric round-to-nearest, per-output-channel 4-bit
  weights, per-token 4-bit activations, group size -1, activation clip 1.0.
* Appendix B.3: after calibration the weights are quantized with RTN for W4A4
  inference -- an integer GEMM on codes followed by dequantization.
* Sec. 3.2 (Visual Saliency and Visual Diversity paragraphs, budget ratios
  alpha = 0.3, beta = 0.2, gamma = 0.5): the full selector -- CLS-attention
  top-k over the tokens left after Query Relevance, then max-min completion
  on the cosines of the fake-quantized copies.
* Sec. 3.3, Eq. (p4q_pruning_aware_calibration) and Appendix B.3: block-wise
  calibration minimizes the per-sample mean squared error between the
  W4A4 fake-quantized and the full-precision outputs on the pruned sequence,
  over diagonal channel scales and weight / activation clipping factors.

Readings where the paper is silent (the same readings as the kernels):
* code range [-8, 7], scale = fl32(fl32(c*absmax)/7); ties round half to even;
  x/s is a correctly rounded fp32 division; an all-zero row has scale 0;
* the selector's fake quant uses the same per-token 4-bit quantizer (clip 1);
* cosine similarity is taken on the real-valued fake-quantized vectors, which
  equals the cosine of the integer codes exactly (the scales cancel);
* equal scores are broken by the lower token index;
* the Query-Relevance budget is split evenly across concepts (remainder to the
  earliest), concepts are processed in order, already-kept tokens are skipped;
* retained rows are emitted in ascending index order, text rows after them;
* stage budgets are floor(alpha K), floor(beta K) and the rest, in exact
  integer arithmetic; equal CLS weights and equal max-cosines go to the lower
  index; a zero code vector has cosine 0 with everything; with an empty
  retained set the diversity stage starts from the most salient token;
* epilogue y = out_rne(fl32(fl32(float(acc) * s_a[m]) * s_w[n])).
* calibration (O7), one linear at a time: the diagonal scales divide the
  activation channels and multiply the weight input channels; the clipping
  factor multiplies the row maximum before the division by 7 (one factor for
  activations, one per output channel for weights); rounding passes
  gradients straight through, the clamp only where the rounded quotient is
  in [-8, 7], the row maximum to its lowest-index element; the loss is the
  squared error summed over the M x N outputs divided by M N.
"""
from __future__ import annotations

from fractions import Fraction
from typing import List, Sequence, Tuple

import numpy as np

QMIN, QMAX = -8, 7          # two's-complement int4
QDIV = np.float32(7.0)      # symmetric range divisor (2^(4-1) - 1)


# --------------------------------------------------------------------------
# storage helpers (dtype decoding / encoding)
# --------------------------------------------------------------------------
def as_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    """Decode fp16 (float16 array) or bf16 (uint16 bit patterns) exactly;
    "fp32" passes float32 rows through."""
    if dtype == "fp32":
        return np.asarray(x, dtype=np.float32)
    if dtype == "fp16":
        return np.asarray(x, dtype=np.float16).astype(np.float32)
    if dtype == "bf16":
        u = np.asarray(x, dtype=np.uint16).astype(np.uint32) << 16
        return u.view(np.float32)
    raise ValueError(f"unknown dtype {dtype}")


def f32_to_bf16_rne(y: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even) -> uint16 bits.

    Finite inputs only (the epilogue never produces NaN).  Overflow past the
    largest bf16 carries into the exponent and yields +-inf, as IEEE rounding
    does."""
    u = np.ascontiguousarray(y, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    return ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)


def round_out(y32: np.ndarray, out_dtype: str) -> np.ndarray:
    """Final RNE rounding of the fp32 epilogue value to the output dtype."""
    if out_dtype == "fp16":
        return y32.astype(np.float16)          # IEEE RNE conversion
    if out_dtype == "bf16":
        return f32_to_bf16_rne(y32)
    raise ValueError(out_dtype)


# --------------------------------------------------------------------------
# O1: the symmetric 4-bit round-to-nearest quantizer (per row)
# --------------------------------------------------------------------------
def quantize_rows(x: np.ndarray, dtype: str = "fp16", clip: float = 1.0
                  ) -> Tuple[np.ndarray, np.ndarray]:
    """Per-row symmetric int4 RTN quantization (Appendix A / B.3 W4A4 setting).

    For every row (a token for activations, an output channel for weights):
      a      = max_k |x_k|                       (exact)
      s      = fl32(fl32(clip * a) / 7)
      code_k = clamp(rne(fl32(x_k / s)), -8, 7)   (s > 0)
      code_k = 0, s = 0                           (s == 0)
    Returns (codes int8 [..., L], scales float32 [...]).
    """
    xf = as_f32(x, dtype)
    lead = xf.shape[:-1]
    rows = xf.reshape(-1, xf.shape[-1])
    codes = np.zeros(rows.shape, dtype=np.int8)
    scales = np.zeros(rows.shape[0], dtype=np.float32)
    c = np.float32(clip)
    for r in range(rows.shape[0]):
        row = rows[r]
        if not np.all(np.isfinite(row)):
            raise ValueError("non-finite input row")
        a = np.max(np.abs(row))                       # exact in fp32
        s = np.float32(np.float32(c * a) / QDIV)      # two fp32 roundings
        scales[r] = s
        if s == 0:
            continue
        q = row / s                                   # correctly rounded fp32
        codes[r] = np.clip(np.rint(q), QMIN, QMAX).astype(np.int8)
    return codes.reshape(xf.shape), scales.reshape(lead)


def dequantize_rows(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """The fake-quantized copy s * code, exactly, in float64."""
    return codes.astype(np.float64) * scales.astype(np.float64)[..., None]


# --------------------------------------------------------------------------
# O2: nibble packing (low nibble = even k)
# --------------------------------------------------------------------------
def pack_int4(codes: np.ndarray) -> np.ndarray:
    """byte_t = (code_{2t} & 0xF) | ((code_{2t+1} & 0xF) << 4)."""
    c = np.asarray(codes, dtype=np.int16)
    assert c.shape[-1] % 2 == 0
    lo = c[..., 0::2] & 0xF
    hi = c[..., 1::2] & 0xF
    return (lo | (hi << 4)).astype(np.uint8)


def unpack_int4(packed: np.ndarray) -> np.ndarray:
    """Inverse of pack_int4: sign-extend each nibble back to int8."""
    p = np.asarray(packed, dtype=np.int16)
    lo = p & 0xF
    hi = (p >> 4) & 0xF
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    out = np.empty(p.shape[:-1] + (p.shape[-1] * 2,), dtype=np.int8)
    out[..., 0::2] = lo
    out[..., 1::2] = hi
    return out


def quant_act(x: np.ndarray, dtype: str = "fp16", clip: float = 1.0
              ) -> Tuple[np.ndarray, np.ndarray]:
    """Per-token activation quantize + pack: (packed uint8 [M, L/2], scales [M])."""
    codes, scales = quantize_rows(x, dtype, clip)
    return pack_int4(codes), scales


# --------------------------------------------------------------------------
# O3: quantization-aware Query-Relevance selection (Sec. 3.2)
# --------------------------------------------------------------------------
def concept_dots(cv: np.ndarray, cq: np.ndarray) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Exact integer statistics of the fake-quantized copies.

    D[i, j] = sum_k cv[i,k] * cq[j,k],  Nv[i] = sum_k cv[i,k]^2,
    Nq[j] = sum_k cq[j,k]^2.  With v~_i = s_v cv_i and q~_j = s_q cq_j,
    CosSim(q~_j, v~_i) = D[i,j] / sqrt(Nv[i] * Nq[j]) exactly (scales cancel).
    """
    cv64 = cv.astype(np.int64)
    cq64 = cq.astype(np.int64)
    D = cv64 @ cq64.T
    Nv = np.sum(cv64 * cv64, axis=1)
    Nq = np.sum(cq64 * cq64, axis=1)
    return D, Nv, Nq


def signed_cos2(D: int, Nv: int, Nq: int) -> Fraction:
    """sgn(cos) * cos^2 as an exact rational; 0 when a vector is all-zero.

    x -> x|x| is strictly increasing, so it orders tokens exactly as the
    cosine does while staying rational."""
    den = int(Nv) * int(Nq)
    if den == 0:
        return Fraction(0)
    D = int(D)
    return Fraction(D * abs(D), den)


def concept_order(D: np.ndarray, Nv: np.ndarray, Nq: np.ndarray, j: int) -> List[int]:
    """Token indices in concept j's ranking: higher cosine first, equal
    cosines by lower index."""
    N = D.shape[0]
    keys = [signed_cos2(D[i, j], Nv[i], Nq[j]) for i in range(N)]
    return sorted(range(N), key=lambda i: (-keys[i], i))


def concept_quotas(K: int, J: int) -> List[int]:
    """Even split of the Query-Relevance budget, remainder to the first concepts."""
    return [K // J + (1 if j < K % J else 0) for j in range(J)]


def select_query_relevance(cv: np.ndarray, cq: np.ndarray, K: int) -> np.ndarray:
    """Concept-wise top-K on the fake-quantized copies; returns sorted indices."""
    D, Nv, Nq = concept_dots(cv, cq)
    J = cq.shape[0]
    kept: List[int] = []
    in_set = set()
    for j, quota in enumerate(concept_quotas(K, J)):
        taken = 0
        for i in concept_order(D, Nv, Nq, j):
            if taken == quota:
                break
            if i in in_set:
                continue
            kept.append(i)
            in_set.add(i)
            taken += 1
    return np.array(sorted(kept), dtype=np.int32)


def select(vis: np.ndarray, concepts: np.ndarray, text: np.ndarray, K: int,
           dtype: str = "fp16", clip: float = 1.0):
    """The hot-path selector for one sample (Query Relevance holds all of K).

    vis [N, d], concepts [J, d], text [T, d] (storage arrays of `dtype`).
    Returns (idx int32 [K] ascending, tokens [K+T, d] storage dtype,
             D int64 [N, J], Nv int64 [N]).
    The fake-quantized copies decide *which* rows are kept; the rows that go
    forward are the original, unquantized ones.
    """
    N = vis.shape[0]
    if not (1 <= K <= N):
        raise ValueError("need 1 <= K <= N")
    cv, _ = quantize_rows(vis, dtype, clip)
    cq, _ = quantize_rows(concepts, dtype, clip)
    idx = select_query_relevance(cv, cq, K)
    tokens = np.concatenate([np.asarray(vis)[idx], np.asarray(text)], axis=0)
    D, Nv, _ = concept_dots(cv, cq)
    return idx, tokens, D, Nv


def select_batch(vis: np.ndarray, concepts: np.ndarray, text: np.ndarray, K: int,
                 dtype: str = "fp16", clip: float = 1.0):
    """select() for every sample of a batch [B, ...]."""
    outs = [select(vis[b], concepts[b], text[b], K, dtype, clip) for b in range(vis.shape[0])]
    idx = np.stack([o[0] for o in outs])
    tok = np.stack([o[1] for o in outs])
    D = np.stack([o[2] for o in outs])
    Nv = np.stack([o[3] for o in outs])
    return idx, tok, D, Nv


# --------------------------------------------------------------------------
# O3': the full progressive selector (Sec. 3.2, Eq. p4q_progressive_selection):
#      Query Relevance, then Visual Saliency over the tokens left, then Visual
#      Diversity completion, with budget ratios alpha, beta, gamma.
# --------------------------------------------------------------------------
def stage_budgets(K: int, alpha: Tuple[int, int] = (3, 10),
                  beta: Tuple[int, int] = (2, 10)) -> Tuple[int, int, int]:
    """Token budgets of the three stages: floor(alpha K), floor(beta K) and the
    rest, in exact integer arithmetic (the paper's defaults alpha = 0.3,
    beta = 0.2, gamma = 0.5 give (192, 128, 320) at K = 640)."""
    kq = K * alpha[0] // alpha[1]
    ks = K * beta[0] // beta[1]
    return kq, ks, K - kq - ks


def saliency_topk(a_cls: np.ndarray, kept: Sequence[int], k: int) -> List[int]:
    """Visual Saliency: among the tokens not kept by the earlier stage, the k
    with the largest head-averaged CLS-to-patch attention weight A_i^cls
    (equal weights: lower index first).  Returns them best first."""
    taken = set(int(i) for i in kept)
    remaining = [i for i in range(len(a_cls)) if i not in taken]
    order = sorted(remaining, key=lambda i: (-float(a_cls[i]), i))
    return order[:k]


def diversity_greedy(cv: np.ndarray, kept: Sequence[int], k: int,
                     a_cls: np.ndarray) -> List[int]:
    """Visual Diversity completion, k picks.  For every candidate left, the
    maximum cosine similarity to the retained set is computed; the candidate
    whose maximum is lowest is retained (equal maxima: lower index); the
    retained set grows by it and the maxima are recomputed.

    Cosines are those of the fake-quantized copies: cos(i, t) =
    D_it / sqrt(Nv_i Nv_t) with D = cv cv^T, exactly (scales cancel), and 0
    when either code vector is all zero.  They are compared through the exact
    rational sgn(cos) cos^2.  With an empty retained set the first pick is the
    most salient token (the paper leaves this case open)."""
    # Gram matrix of the codes as a float64 matmul: every product is an
    # integer of magnitude <= 64 and every partial sum an integer of magnitude
    # <= 64 d < 2^53, so the result is exact whatever the summation order
    cvf = cv.astype(np.float64)
    G = (cvf @ cvf.T).astype(np.int64)
    Nv = np.diag(G)
    S = [int(i) for i in kept]
    in_s = set(S)
    picks: List[int] = []
    if k > 0 and not S:
        seed = saliency_topk(a_cls, [], 1)[0]
        S.append(seed)
        in_s.add(seed)
        picks.append(seed)
        k -= 1
    cand = [i for i in range(cv.shape[0]) if i not in in_s]
    m = {i: max(signed_cos2(G[i, t], Nv[i], Nv[t]) for t in S) for i in cand}
    for _ in range(k):
        best = min(cand, key=lambda i: (m[i], i))
        picks.append(best)
        S.append(best)
        cand.remove(best)
        del m[best]
        for i in cand:
            c = signed_cos2(G[i, best], Nv[i], Nv[best])
            if c > m[i]:
                m[i] = c
    return picks


def select_full(vis: np.ndarray, concepts: np.ndarray, a_cls: np.ndarray,
                text: np.ndarray, K: int, kq: int, ks: int,
                dtype: str = "fp16", clip: float = 1.0):
    """The three-stage selector for one sample: kq tokens by Query Relevance,
    ks by Visual Saliency over the rest, K - kq - ks by Visual Diversity.

    vis [N, d], concepts [J, d], a_cls [N] (fp32 head-averaged CLS-to-patch
    attention), text [T, d].  Returns (idx int32 [K] ascending, tokens
    [K+T, d] storage dtype, (query picks sorted, saliency picks best first,
    diversity picks in pick order))."""
    N = vis.shape[0]
    if not (1 <= K <= N) or kq < 0 or ks < 0 or kq + ks > K:
        raise ValueError("need 1 <= K <= N and 0 <= kq, ks with kq + ks <= K")
    cv, _ = quantize_rows(vis, dtype, clip)
    cq, _ = quantize_rows(concepts, dtype, clip)
    q_picks = [int(i) for i in select_query_relevance(cv, cq, kq)] if kq else []
    s_picks = saliency_topk(a_cls, q_picks, ks)
    d_picks = diversity_greedy(cv, q_picks + s_picks, K - kq - ks, a_cls)
    idx = np.array(sorted(q_picks + s_picks + d_picks), dtype=np.int32)
    tokens = np.concatenate([np.asarray(vis)[idx], np.asarray(text)], axis=0)
    return idx, tokens, (q_picks, s_picks, d_picks)


# --------------------------------------------------------------------------
# O5: the fused decoder prologue -- RMSNorm with its per-channel weight (the
#     slot into which calibration's diagonal scales fold, Appendix B.3), then
#     the per-token quantizer, without materializing the normalized row
# --------------------------------------------------------------------------
def rmsnorm_quant(x: np.ndarray, gamma: np.ndarray, eps: float = 1e-5,
                  dtype: str = "fp16", clip: float = 1.0
                  ) -> Tuple[np.ndarray, np.ndarray]:
    """Per-token Q4 of RMSNorm(x) * gamma.

    RMSNorm(x)_k = x_k / rms(x) with rms(x) = sqrt(mean_k x_k^2 + eps).  A
    positive factor per row does not change Q4's codes in exact arithmetic
    and multiplies its scale, so the prologue quantizes the row
    u = x * gamma (fp32; exact, since both factors are 16-bit floats) and
    moves 1/rms(x) into the scale:
        codes = Q4(u; clip).codes
        scale = fl32(Q4(u; clip).scale * (1 / rms(x)))
    with 1/rms(x) in float64 from the float64 sum of squares.

    x [M, d] and gamma [d] in storage dtype.  Returns (packed codes uint8
    [M, d/2], scales float32 [M])."""
    xf = as_f32(x, dtype)
    gf = as_f32(gamma, dtype)
    u = (xf * gf[None, :]).astype(np.float32)
    if not np.all(np.isfinite(u)):
        raise ValueError("non-finite x * gamma")
    codes, su = quantize_rows(u, "fp32", clip)
    x64 = xf.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):      # zero rows at eps = 0
        inv_rms = 1.0 / np.sqrt(np.sum(x64 * x64, axis=1) / x64.shape[1] + float(eps))
        scales = (su.astype(np.float64) * inv_rms).astype(np.float32)
    scales[su == 0] = 0.0
    return pack_int4(codes), scales


# --------------------------------------------------------------------------
# O6: FP16-KV attention prefill on the pruned sequence -- the decoder step
#     after the q/k/v linears (Appendix B.3: W4A4 with the key and value
#     caches kept in FP16)
# --------------------------------------------------------------------------
def attention_prefill(q: np.ndarray, k: np.ndarray, v: np.ndarray, causal: bool = True,
                      dtype: str = "fp16") -> np.ndarray:
    """Scaled dot-product attention of one sequence, all heads.

    q, k, v [L, H, D] in storage dtype.  For token t and head h:
        S[t, j] = <q_t, k_j> / sqrt(D)   over the allowed keys j (j <= t when
                                          causal, every j otherwise)
        P[t, :] = softmax(S[t, :]),  O[t] = sum_j P[t, j] v_j
    in float64, then rounded to the storage dtype (nearest, ties to even).
    Returns O [L, H, D] in storage dtype."""
    qf, kf, vf = (as_f32(a, dtype).astype(np.float64) for a in (q, k, v))
    L, H, D = qf.shape
    out = np.empty((L, H, D), dtype=np.float64)
    allowed = np.tril(np.ones((L, L), dtype=bool)) if causal else np.ones((L, L), dtype=bool)
    for h in range(H):
        S = (qf[:, h, :] @ kf[:, h, :].T) / np.sqrt(D)
        S = np.where(allowed, S, -np.inf)
        S = S - S.max(axis=1, keepdims=True)
        P = np.exp(S)
        P = P / P.sum(axis=1, keepdims=True)
        out[:, h, :] = P @ vf[:, h, :]
    if dtype == "fp16":
        return out.astype(np.float16)
    return f32_to_bf16_rne(out.astype(np.float32))


# --------------------------------------------------------------------------
# O4: the W4A4 linear (integer GEMM on codes + dequant epilogue)
# --------------------------------------------------------------------------
def int_gemm(a_codes: np.ndarray, w_codes: np.ndarray) -> np.ndarray:
    """acc[m, n] = sum_k A[m, k] * W[n, k], exact.

    Computed as a float64 matmul of the codes: every product is an integer of
    magnitude <= 64 and every partial sum an integer below 2^24, so each one is
    exactly representable and the result is exact whatever the summation
    order."""
    acc = a_codes.astype(np.float64) @ w_codes.astype(np.float64).T
    return acc.astype(np.int64)


def epilogue(acc: np.ndarray, a_scales: np.ndarray, w_scales: np.ndarray,
             out_dtype: str) -> np.ndarray:
    """y = out_rne(fl32(fl32(float(acc) * s_a[m]) * s_w[n]))."""
    t = acc.astype(np.float32) * a_scales.astype(np.float32)[:, None]
    t = t.astype(np.float32)
    y = t * w_scales.astype(np.float32)[None, :]
    return round_out(y.astype(np.float32), out_dtype)


def w4a4_linear(a_packed: np.ndarray, a_scales: np.ndarray, w_packed: np.ndarray,
                w_scales: np.ndarray, out_dtype: str):
    """W4A4 linear on packed operands. Returns (acc int64 [M, N], y [M, N])."""
    acc = int_gemm(unpack_int4(a_packed), unpack_int4(w_packed))
    return acc, epilogue(acc, a_scales, w_scales, out_dtype)


def w4a4_linear_entry(a_packed: np.ndarray, a_scales: np.ndarray, w_packed: np.ndarray,
                      w_scales: np.ndarray, m: int, n: int, out_dtype: str):
    """One output element (m, n) computed on its own, for sampled full-size checks."""
    a = unpack_int4(a_packed[m]).astype(np.int64)
    w = unpack_int4(w_packed[n]).astype(np.int64)
    acc = int(np.dot(a, w))
    y = epilogue(np.array([[acc]], dtype=np.int64), a_scales[m:m + 1], w_scales[n:n + 1],
                 out_dtype)
    return acc, y[0, 0]


# --------------------------------------------------------------------------
# O7: pruning-aware calibration mechanics (Sec. 3.3, Eq.
#     p4q_pruning_aware_calibration; Appendix B.3) -- the reconstruction
#     objective of one W4A4 fake-quantized linear on a pruned sequence and its
#     gradients with respect to the learnable diagonal channel scales and the
#     activation / weight clipping factors
# --------------------------------------------------------------------------
def quant_rows_scaled(z: np.ndarray, sigma: np.ndarray, divide: bool, clip,
                      dtype: str = "fp16"):
    """Q4 of the channel-transformed rows z'.

    z' = fl32(z / sigma_k) (divide=True: activations, whose channels the
    diagonal scales divide) or fl32(z * sigma_k) (divide=False: weights, whose
    input channels they multiply), each a correctly rounded fp32 operation.
    clip is one factor for every row or one per row.  Returns (codes int8
    [R, L], scales fp32 [R], absmax fp32 [R] = max_k |z'_k|, kstar int64 [R] =
    the lowest k attaining it, z' fp32 [R, L])."""
    zf = as_f32(z, dtype)
    sig = np.asarray(sigma, dtype=np.float32)
    zp = (zf / sig[None, :]) if divide else (zf * sig[None, :])
    zp = zp.astype(np.float32)
    if not np.all(np.isfinite(zp)):
        raise ValueError("non-finite transformed row")
    R = zp.shape[0]
    clips = np.broadcast_to(np.asarray(clip, dtype=np.float32), (R,))
    codes = np.zeros(zp.shape, dtype=np.int8)
    scales = np.zeros(R, dtype=np.float32)
    absmax = np.zeros(R, dtype=np.float32)
    kstar = np.zeros(R, dtype=np.int64)
    for r in range(R):
        c, s = quantize_rows(zp[r:r + 1], "fp32", float(clips[r]))
        codes[r], scales[r] = c[0], s[0]
        mag = np.abs(zp[r])
        absmax[r] = mag.max()
        kstar[r] = int(np.flatnonzero(mag == absmax[r])[0])
    return codes, scales, absmax, kstar, zp


def fq_row_backward(zp: np.ndarray, s: float, clip: float, codes: np.ndarray,
                    absmax: float, kstar: int, g: np.ndarray, absolute: bool = False):
    """Gradient of one fake-quantized row F(z') = s * clamp(rne(z'/s), -8, 7),
    s = clip * max|z'| / 7, given the upstream gradient g = dL/dF.

    Rounding passes gradients straight through; the clamp passes them only
    where the rounded quotient rho = rne(fl32(z'/s)) lies in [-8, 7]
    ("inside"); the maximum passes its share to the lowest index attaining it.
    With g_s = dL/ds = sum_k g_k (code_k - inside_k z'_k / s):
        dL/dz'_k  = inside_k g_k + [k = kstar] g_s (clip / 7) sign(z'_k)
        dL/dclip  = g_s * absmax / 7
    A row with s = 0 has no gradient.  With absolute=True (g >= 0) every
    factor is taken in magnitude (the linear error-propagation form).
    Returns (dz' float64 [L], dclip)."""
    if s == 0:
        return np.zeros(zp.shape, dtype=np.float64), 0.0
    ab = np.abs if absolute else (lambda v: v)
    rho = np.rint(zp / np.float32(s))                  # the quotient's fp32 rounding decides
    inside = ((rho >= QMIN) & (rho <= QMAX)).astype(np.float64)
    z64 = zp.astype(np.float64)
    g_s = float(np.sum(g * ab(codes.astype(np.float64) - inside * z64 / float(s))))
    dz = g * inside
    sign = 1.0 if absolute else float(np.sign(z64[kstar]))
    dz[kstar] += g_s * (float(clip) / 7.0) * sign
    return dz, g_s * float(absmax) / 7.0


def _calib_backward(P1, P2, scale, q, absolute=False):
    """The backward pass of calib_linear from its two contraction operands
    P1 [M, N] (the residual times sW[n]) and P2 [M, N] (times sA[m]).

    With absolute=False this is the gradient.  With absolute=True every
    quantity is replaced by its magnitude and every sum by a sum of
    magnitudes (P1, P2 are then non-negative arrays): the result bounds, per
    output component, how far an error of size P1 / P2 in the operands can
    move it (linear propagation)."""
    ab = np.abs if absolute else (lambda v: v)
    cA, cW = q["a_codes"].astype(np.float64), q["w_codes"].astype(np.float64)
    gA = scale * (P1 @ ab(cW))                           # dL/d(sA cA)  [M, K]
    gW = scale * (P2.T @ ab(cA))                         # dL/d(sW cW)  [N, K]

    def side(g, zp, s, clip, codes, absmax, kstar):
        """fq_row_backward over every row of one side."""
        R = zp.shape[0]
        dz = np.zeros(zp.shape, dtype=np.float64)
        dclip = np.zeros(R, dtype=np.float64)
        clip = np.broadcast_to(np.asarray(clip, dtype=np.float32), (R,))
        for r in range(R):
            dz[r], dclip[r] = fq_row_backward(zp[r], s[r], clip[r], codes[r], absmax[r],
                                              kstar[r], g[r], absolute)
        return dz, dclip

    dxp, dca = side(gA, q["xp"], q["a_scales"], q["clip_a"], q["a_codes"], q["a_absmax"],
                    q["a_kstar"])
    dwp, dcw = side(gW, q["wp"], q["w_scales"], q["clip_w"], q["w_codes"], q["w_absmax"],
                    q["w_kstar"])
    s64 = q["sigma"].astype(np.float64)
    grad_sigma = (np.sum(dxp * ab(-q["x64"] / (s64 * s64)[None, :]), axis=0)
                  + np.sum(dwp * ab(q["w64"]), axis=0))
    return grad_sigma, float(np.sum(dca)), dcw


def calib_linear(x: np.ndarray, w: np.ndarray, target: np.ndarray, sigma: np.ndarray,
                 clip_a: float, clip_w: np.ndarray, dtype: str = "fp16",
                 operands: str = "fp64", bounds: bool = False) -> dict:
    """Reconstruction loss of one W4A4 fake-quantized linear and its gradients.

    x [M, K] (the pruned sequence's input rows) and w [N, K] in storage
    dtype; target [M, N] fp32 is the full-precision layer output; sigma [K]
    > 0 the diagonal channel scales; clip_a the activation clipping factor
    (one per layer: tokens vary at run time); clip_w [N] the per-output-
    channel weight clipping factors.

      X' = X diag(sigma)^-1 and W' = W diag(sigma) (the product is unchanged
      in exact arithmetic, which lets calibration fold sigma into the model);
      (cA, sA) = Q4 rows of X' with clip_a; (cW, sW) = Q4 rows of W' with
      clip_w[n]; the fake-quantized output is Yq = (sA cA)(sW cW)^T, i.e.
      Yq[m, n] = sA[m] sW[n] acc[m, n] with the exact integer acc;
      loss = ||Yq - target||_F^2 / (M N)    (the per-sample term of the
      calibration objective, m = M rows of width d = N).

    Gradients (rounding passed straight through, see fq_row_backward), with
    G = 2 (Yq - target) / (M N):
      dL/d(sA cA) = G (sW cW),   dL/d(sW cW) = G^T (sA cA);
      d sigma_k  = sum_m dX'[m, k] (-X[m, k] / sigma_k^2) + sum_n dW'[n, k] W[n, k];
      d clip_a   = sum over rows m of their dclip;  d clip_w[n] = row n's dclip.

    operands="fp64": everything after the quantizer in float64 -- the plain
    definition.
    operands="bf16": the two contractions take bf16 operands, as a mixed-
    precision calibration runs them: R = fl32(fl32(fl32(acc sA[m]) sW[n]) -
    target), and the operands are bf16(fl32(R sW[n])) and bf16(fl32(R sA[m]))
    (nearest, ties to even); the loss is sum R^2 / (M N); the codes and
    the rest stay exact / float64.  A diagnostic of that arithmetic only.

    bounds=True (with operands="fp64") also returns, per output, a bound on
    how far an evaluation that rounds the residual in fp32, the contraction
    operands to bf16 and accumulates in fp32 can lie from the float64 result:
      * operand error, per entry: |P^ - R sW| <= sW (1.01 * 2^-8 |R|
        + 4 u (|Yq| + |R|)) with u = 2^-24 (the fp32 residual is within
        3 u (|Yq| + |R|) of R; bf16 rounding is 2^-8 relative, fl32 of the
        product 2^-24), and likewise with sA for the other operand;
      * this error propagated linearly through the backward pass in
        magnitude form (_calib_backward with absolute=True);
      * plus (gamma_N + gamma_M + gamma_K + 2^-20) times the magnitude form
        of the whole backward pass, gamma_n = n u / (1 - n u) being the
        worst-case relative error of an fp32 sum of n terms (the two
        contractions, the row and the column sums) and 2^-20 covering the
        fp32 rounding of the few per-element products.
    The loss bound is sum (2 |R| e + e^2) / (M N) + gamma_{MN} loss with
    e = 3 u (|Yq| + |R|).

    Returns a dict with loss, grad_sigma [K], grad_clip_a, grad_clip_w [N]
    (float64), the quantizer outputs of both sides and, with bounds, the
    matching bound_* entries."""
    M, K = x.shape
    N = w.shape[0]
    sig = np.asarray(sigma, dtype=np.float32)
    cw_clip = np.asarray(clip_w, dtype=np.float32).reshape(N)
    cA, sA, aA, kA, xp = quant_rows_scaled(x, sig, True, np.float32(clip_a), dtype)
    cW, sW, aW, kW, wp = quant_rows_scaled(w, sig, False, cw_clip, dtype)
    acc = int_gemm(cA, cW).astype(np.float64)
    T = np.asarray(target, dtype=np.float32)
    Y = sA.astype(np.float64)[:, None] * sW.astype(np.float64)[None, :] * acc
    if operands == "fp64":
        R = Y - T
        P1 = R * sW.astype(np.float64)[None, :]
        P2 = R * sA.astype(np.float64)[:, None]
    elif operands == "bf16":
        y32 = (acc.astype(np.float32) * sA[:, None]).astype(np.float32)
        y32 = (y32 * sW[None, :]).astype(np.float32)
        R32 = (y32 - T).astype(np.float32)
        P1 = as_f32(f32_to_bf16_rne((R32 * sW[None, :]).astype(np.float32)), "bf16")
        P2 = as_f32(f32_to_bf16_rne((R32 * sA[:, None]).astype(np.float32)), "bf16")
        R = R32.astype(np.float64)
        P1 = P1.astype(np.float64)
        P2 = P2.astype(np.float64)
    else:
        raise ValueError(operands)
    scale = 2.0 / (M * N)
    loss = float(np.sum(R * R)) / (M * N)
    q = {"a_codes": cA, "a_scales": sA, "a_absmax": aA, "a_kstar": kA, "xp": xp,
         "clip_a": np.float32(clip_a), "w_codes": cW, "w_scales": sW, "w_absmax": aW,
         "w_kstar": kW, "wp": wp, "clip_w": cw_clip, "sigma": sig,
         "x64": as_f32(x, dtype).astype(np.float64), "w64": as_f32(w, dtype).astype(np.float64)}
    grad_sigma, dclip_a, dclip_w = _calib_backward(P1, P2, scale, q)
    out = {"loss": loss, "grad_sigma": grad_sigma, "grad_clip_a": dclip_a,
           "grad_clip_w": dclip_w, "a_codes": cA, "a_scales": sA, "a_absmax": aA,
           "a_kstar": kA, "w_codes": cW, "w_scales": sW, "w_absmax": aW, "w_kstar": kW}
    if bounds:
        if operands != "fp64":
            raise ValueError("bounds are taken around the float64 result")
        u = 2.0 ** -24
        gam = lambda n: n * u / (1.0 - n * u)
        absR, absY = np.abs(R), np.abs(Y)
        e = 4.0 * u * (absY + absR)
        E1 = (1.01 * 2.0 ** -8 * absR + e) * sW.astype(np.float64)[None, :]
        E2 = (1.01 * 2.0 ** -8 * absR + e) * sA.astype(np.float64)[:, None]
        bs, bca, bcw = _calib_backward(E1, E2, scale, q, absolute=True)
        ms, mca, mcw = _calib_backward(np.abs(P1), np.abs(P2), scale, q, absolute=True)
        g = gam(N) + gam(M) + gam(K) + 2.0 ** -20
        out["bound_grad_sigma"] = bs + g * ms
        out["bound_grad_clip_a"] = bca + g * mca
        out["bound_grad_clip_w"] = bcw + g * mcw
        eR = 3.0 * u * (absY + absR)
        out["bound_loss"] = float(np.sum(2.0 * absR * eR + eR * eR)) / (M * N) + gam(M * N) * loss
    return out


# --------------------------------------------------------------------------
# O8: pruning-aware calibration of a whole decoder block (Sec. 3.3, Eq.
#     p4q_pruning_aware_calibration: the per-sample MSE between the W4A4
#     fake-quantized block and the full-precision block on the pruned
#     sequence; Appendix B.3: block by block, diagonal scales and weight /
#     activation clipping factors learned, K and V kept in FP16)
# --------------------------------------------------------------------------
BLOCK_GROUPS = ("qkv", "o", "gu", "down")     # the block's four fake-quantized linear groups


def _r16(v: np.ndarray, dtype: str) -> np.ndarray:
    """Round real values to the block's storage dtype (nearest, ties to
    even); returned as float64 holding the 16-bit values exactly."""
    if dtype == "fp16":
        return np.asarray(v, dtype=np.float64).astype(np.float16).astype(np.float64)
    return as_f32(f32_to_bf16_rne(np.asarray(v, dtype=np.float64).astype(np.float32)),
                  "bf16").astype(np.float64)


def _store16(v64: np.ndarray, dtype: str) -> np.ndarray:
    """float64 values that are exact 16-bit numbers -> storage array."""
    if dtype == "fp16":
        return v64.astype(np.float16)
    return f32_to_bf16_rne(v64.astype(np.float32))


def _rope_tables(M: int, D: int, base: float):
    """cos / sin of position p times theta_i = base^(-2i/D), i < D/2,
    positions 0..M-1 (the pruned sequence re-indexed consecutively)."""
    i = np.arange(D // 2, dtype=np.float64)
    theta = base ** (-2.0 * i / D)
    ang = np.arange(M, dtype=np.float64)[:, None] * theta[None, :]
    return np.cos(ang), np.sin(ang)


def _rope(z: np.ndarray, cos: np.ndarray, sin: np.ndarray, inverse: bool = False) -> np.ndarray:
    """Rotary embedding of z [M, H, D] (rotate-half pairing of channel i
    with i + D/2); inverse=True applies the transposed rotation (its
    backward)."""
    h = z.shape[2] // 2
    a, b = z[:, :, :h], z[:, :, h:]
    c, s = cos[:, None, :], sin[:, None, :]
    if inverse:
        s = -s
    return np.concatenate([a * c - b * s, b * c + a * s], axis=2)


def _rmsnorm(x: np.ndarray, g: np.ndarray, eps: float, fp32: bool = False):
    """n = x * gamma / sqrt(mean(x^2) + eps) in real arithmetic; returns (n,
    r = 1/rms per row).  fp32: r and the two products rounded to fp32."""
    r = 1.0 / np.sqrt(np.mean(x * x, axis=1) + eps)
    if fp32:
        r = r.astype(np.float32)
        n = (x.astype(np.float32) * r[:, None]).astype(np.float32) * g.astype(np.float32)[None, :]
        return n.astype(np.float64), r.astype(np.float64)
    return x * r[:, None] * g[None, :], r


def _rmsnorm_backward(x, g, r, dn):
    """dL/dx of n = x gamma r(x):  r gamma dn - x r^3 / d sum_j x_j gamma_j dn_j."""
    d = x.shape[1]
    s = np.sum(x * g[None, :] * dn, axis=1)
    return r[:, None] * g[None, :] * dn - x * (r ** 3 * s / d)[:, None]


def _attention(q, k, v, fp32: bool = False):
    """Causal softmax attention per head in real arithmetic: q, k, v [M, H,
    D] -> (O [M, H, D], P [H, M, M]).  fp32: scores, weights and products
    in fp32."""
    M, H, D = q.shape
    causal = np.tril(np.ones((M, M), dtype=bool))
    P = np.empty((H, M, M), dtype=np.float64)
    O = np.empty((M, H, D), dtype=np.float64)
    t = np.float32 if fp32 else np.float64
    for hh in range(H):
        S = (q[:, hh, :].astype(t) @ k[:, hh, :].T.astype(t)) * t(1.0 / np.sqrt(D))
        S = np.where(causal, S, -np.inf).astype(t)
        E = np.exp(S - S.max(axis=1, keepdims=True)).astype(t)
        Ph = (E / E.sum(axis=1, keepdims=True)).astype(t)
        P[hh] = Ph
        O[:, hh, :] = Ph @ v[:, hh, :].astype(t)
    return O, P


def _attention_backward(q, k, v, P, dO):
    """(dq, dk, dv) of O = P v, P = softmax(q k^T / sqrt(D)):
    dv = P^T dO, dP = dO v^T, dS = P (dP - rowsum(P dP)), dq = dS k / sqrt(D),
    dk = dS^T q / sqrt(D)."""
    M, H, D = q.shape
    dq, dk, dv = (np.empty((M, H, D)) for _ in range(3))
    for hh in range(H):
        dv[:, hh, :] = P[hh].T @ dO[:, hh, :]
        dP = dO[:, hh, :] @ v[:, hh, :].T
        dS = P[hh] * (dP - np.sum(P[hh] * dP, axis=1, keepdims=True))
        dq[:, hh, :] = dS @ k[:, hh, :] / np.sqrt(D)
        dk[:, hh, :] = dS.T @ q[:, hh, :] / np.sqrt(D)
    return dq, dk, dv


def _silu_mul_backward(g, u, da):
    """(dg, du) of a = SiLU(g) u = g sig(g) u, sig the logistic function:
    dSiLU/dg = sig(g) (1 + g (1 - sig(g)))."""
    sg = 1.0 / (1.0 + np.exp(-g))
    return da * u * sg * (1.0 + g * (1.0 - sg)), da * g * sg


def _fq_linear(X16, W16, sigma, clip_a, clip_w, dtype):
    """The W4A4 fake-quantized linear of calib_linear, applied in a block:
    X' = X / sigma and W' = W * sigma quantized per row (clip_a, clip_w[n]),
    Y = out_rne(fl32(fl32(acc sA) sW)) in the storage dtype (the epilogue of
    the W4A4 linear).  Returns (Y as float64 values, the quantizer state)."""
    cA, sA, aA, kA, xp = quant_rows_scaled(X16, sigma, True, np.float32(clip_a), dtype)
    cW, sW, aW, kW, wp = quant_rows_scaled(W16, sigma, False, clip_w, dtype)
    acc = int_gemm(cA, cW)
    y = as_f32(epilogue(acc, sA, sW, dtype), dtype).astype(np.float64)
    q = {"a_codes": cA, "a_scales": sA, "a_absmax": aA, "a_kstar": kA, "xp": xp,
         "clip_a": np.float32(clip_a), "w_codes": cW, "w_scales": sW, "w_absmax": aW,
         "w_kstar": kW, "wp": wp, "clip_w": np.asarray(clip_w, dtype=np.float32),
         "sigma": np.asarray(sigma, dtype=np.float32),
         "x64": as_f32(X16, dtype).astype(np.float64), "w64": as_f32(W16, dtype).astype(np.float64)}
    return y, q


def _fq_linear_backward(q, G):
    """Gradients of a fake-quantized linear from G = dL/dY (rounding of the
    output passed straight through): (dL/dX [M, K], dL/dsigma [K],
    dL/dclip_a, dL/dclip_w [N]).  Per row as fq_row_backward; X' = X / sigma
    gives dX = dX' / sigma."""
    cA, cW = q["a_codes"].astype(np.float64), q["w_codes"].astype(np.float64)
    sA, sW = q["a_scales"].astype(np.float64), q["w_scales"].astype(np.float64)
    gA = G @ (sW[:, None] * cW)                      # dL/d(sA cA)  [M, K]
    gW = G.T @ (sA[:, None] * cA)                    # dL/d(sW cW)  [N, K]
    M, N = G.shape
    dxp = np.zeros(q["xp"].shape, dtype=np.float64)
    dwp = np.zeros(q["wp"].shape, dtype=np.float64)
    dclip_a = 0.0
    dclip_w = np.zeros(N, dtype=np.float64)
    q["a_dclip_rows"] = np.zeros(M, dtype=np.float64)
    for m in range(M):
        dxp[m], dc = fq_row_backward(q["xp"][m], q["a_scales"][m], q["clip_a"], q["a_codes"][m],
                                     q["a_absmax"][m], q["a_kstar"][m], gA[m])
        dclip_a += dc
        q["a_dclip_rows"][m] = dc
    for n in range(N):
        dwp[n], dclip_w[n] = fq_row_backward(q["wp"][n], q["w_scales"][n], q["clip_w"][n],
                                             q["w_codes"][n], q["w_absmax"][n], q["w_kstar"][n],
                                             gW[n])
    s64 = q["sigma"].astype(np.float64)
    dsigma = (np.sum(dxp * (-q["x64"] / (s64 * s64)[None, :]), axis=0)
              + np.sum(dwp * q["w64"], axis=0))
    return dxp / s64[None, :], dsigma, dclip_a, dclip_w


def calib_block(x: np.ndarray, weights: dict, gamma1: np.ndarray, gamma2: np.ndarray,
                H: int, target: np.ndarray = None, sigma: dict = None, clip_a: dict = None,
                clip_w: dict = None, eps: float = 1e-5, rope_base: float = 10000.0,
                dtype: str = "fp16", quantize: bool = True, bounds: bool = False,
                fp32_ops: bool = False) -> dict:
    """One decoder block on one pruned sequence, full precision or W4A4
    fake-quantized, and for the latter the calibration loss and gradients.

    x [M, d] is the block input (storage dtype); weights holds "qkv" [3d, d]
    (q, k, v rows concatenated), "o" [d, d], "gu" [2f, d] (gate then up) and
    "down" [d, f]; gamma1, gamma2 [d] the RMSNorm weights; H heads of D =
    d / H.  The block (LLaMA-family decoder, intermediates held in the
    storage dtype between operations, each rounded once, nearest even):
        n1 = RMSNorm(x) gamma1;  q|k|v = L_qkv(n1);  q, k <- RoPE(q), RoPE(k)
        O = softmax(q k^T / sqrt(D), causal) v   (per head, real arithmetic)
        h = x + L_o(O);  n2 = RMSNorm(h) gamma2;  g|u = L_gu(n2)
        a = SiLU(g) u;   out = h + L_down(a)
    With quantize=False every L is the plain linear (X W^T, rounded): the
    full-precision block whose output is the calibration target.  With
    quantize=True every L is the W4A4 fake-quantized linear of calib_linear
    with its group's diagonal scales sigma[g] (dividing the input channels,
    multiplying the weights' input channels), activation clipping factor
    clip_a[g] and per-output-channel weight clipping factors clip_w[g];
    loss = ||out - target||^2 / (M d) (the per-sample term of the calibration
    objective), and its gradients with respect to every sigma, clip_a and
    clip_w (rounding of codes and of intermediates passed straight through,
    clamp and row maxima as in fq_row_backward), by the chain rule through
    the full-precision attention, RMSNorm and SiLU-gated MLP.

    Returns {"out": out (storage dtype)} and, with quantize and target,
    "loss", "grad_sigma"[g], "grad_clip_a"[g], "grad_clip_w"[g] (float64) and
    "state"[g], each group's quantizer state (codes, scales, row maxima and
    their indices, transformed rows) for inspection.  With bounds, also
    "mag_grad_sigma"[g], "mag_grad_clip_a"[g] and "mag_grad_clip_w"[g]: for
    every gradient component the sum of the magnitudes of its terms given
    the group's upstream gradient (calib_linear's magnitude form), the scale
    against which a rounded evaluation of the component is measured.

    fp32_ops=True evaluates RMSNorm, attention and the SiLU-gated product
    with fp32 arithmetic instead of real arithmetic (every rounding of the
    definition unchanged).  It is a probe of how sensitive each result is to
    the precision those operations are evaluated in -- some components are
    ill-conditioned -- and never the reference, which is fp32_ops=False."""
    r16 = lambda v: _r16(v, dtype)
    X = as_f32(x, dtype).astype(np.float64)
    M, d = X.shape
    D = d // H
    g1 = as_f32(gamma1, dtype).astype(np.float64)
    g2 = as_f32(gamma2, dtype).astype(np.float64)

    def lin(name, A16):
        if not quantize:
            W = as_f32(weights[name], dtype).astype(np.float64)
            return r16(A16 @ W.T), None
        return _fq_linear(_store16(A16, dtype), weights[name], sigma[name], clip_a[name],
                          clip_w[name], dtype)

    # ---- forward
    n1f, r1 = _rmsnorm(X, g1, eps, fp32_ops)
    n1 = r16(n1f)
    qkv, c_qkv = lin("qkv", n1)
    cos, sin = _rope_tables(M, D, rope_base)
    q = r16(_rope(qkv[:, :d].reshape(M, H, D), cos, sin))
    k = r16(_rope(qkv[:, d:2 * d].reshape(M, H, D), cos, sin))
    v = qkv[:, 2 * d:].reshape(M, H, D)
    O, P = _attention(q, k, v, fp32_ops)
    O = r16(O).reshape(M, d)
    o, c_o = lin("o", O)
    h = r16(X + o)
    n2f, r2 = _rmsnorm(h, g2, eps, fp32_ops)
    n2 = r16(n2f)
    gu, c_gu = lin("gu", n2)
    f = gu.shape[1] // 2
    gg, uu = gu[:, :f], gu[:, f:]
    sig_g = 1.0 / (1.0 + np.exp(-gg))
    if fp32_ops:
        g32 = gg.astype(np.float32)
        a = r16(((g32 / (np.float32(1) + np.exp(-g32))) * uu.astype(np.float32)).astype(np.float64))
    else:
        a = r16(gg * sig_g * uu)
    y, c_down = lin("down", a)
    out = r16(h + y)
    res = {"out": _store16(out, dtype)}
    if not quantize or target is None:
        return res

    # ---- loss and backward (straight through every rounding)
    T = np.asarray(target, dtype=np.float64)
    R = out - T
    res["loss"] = float(np.sum(R * R)) / (M * d)
    dout = 2.0 * R / (M * d)
    grads = {}

    mags = {}

    def back(name, cache, G):
        dX, ds, dca, dcw = _fq_linear_backward(cache, G)
        grads[name] = (ds, dca, dcw)
        if bounds:
            # the sums of magnitudes of each component's terms, given this
            # group's upstream gradient (the backward pass in magnitude form)
            aG = np.abs(G)
            mags[name] = _calib_backward(aG * cache["w_scales"].astype(np.float64)[None, :],
                                         aG * cache["a_scales"].astype(np.float64)[:, None],
                                         1.0, cache, absolute=True)
        return dX

    da = back("down", c_down, dout)
    dg, du = _silu_mul_backward(gg, uu, da)
    dn2 = back("gu", c_gu, np.concatenate([dg, du], axis=1))
    dh = dout + _rmsnorm_backward(h, g2, r2, dn2)
    dO = back("o", c_o, dh).reshape(M, H, D)
    dq, dk, dv = _attention_backward(q, k, v, P, dO)
    dq = _rope(dq, cos, sin, inverse=True)
    dk = _rope(dk, cos, sin, inverse=True)
    back("qkv", c_qkv, np.concatenate([dq.reshape(M, d), dk.reshape(M, d), dv.reshape(M, d)],
                                      axis=1))
    res["state"] = {"qkv": c_qkv, "o": c_o, "gu": c_gu, "down": c_down}
    if bounds:
        res["mag_grad_sigma"] = {g: mags[g][0] for g in BLOCK_GROUPS}
        res["mag_grad_clip_a"] = {g: mags[g][1] for g in BLOCK_GROUPS}
        res["mag_grad_clip_w"] = {g: mags[g][2] for g in BLOCK_GROUPS}
    res["grad_sigma"] = {g: grads[g][0] for g in BLOCK_GROUPS}
    res["grad_clip_a"] = {g: grads[g][1] for g in BLOCK_GROUPS}
    res["grad_clip_w"] = {g: grads[g][2] for g in BLOCK_GROUPS}
    return res
