/*
 * p4q.h -- C ABI of the P4Q hot path on MI355X (gfx950).
 *
 * P4Q (co-designed visual-token pruning and W4A4 quantization) has two
 * data-parallel steps on its inference path:
 *   1. a quantization-aware visual-token selector placed before the LLM
 *      (Sec. 3.2, Eq. p4q_progressive_selection): projector features and
 *      query-concept embeddings are fake-quantized, visual tokens are ranked
 *      per concept by the cosine similarity of those copies, the top tokens
 *      within each concept's quota are kept, and the ORIGINAL feature rows of
 *      the kept tokens are forwarded with the text tokens;
 *   2. the W4A4 linear layers of the LLM on that pruned sequence (Appendix A
 *      and B.3: symmetric round-to-nearest, per-output-channel 4-bit weights,
 *      per-token 4-bit activations, no groups, activation clip 1.0).
 *
 * Conventions shared by every entry point
 *   - Every call is asynchronous and ordered on the caller's `stream`.
 *     Argument checks run on the host before any HIP call; a failing check
 *     returns a status and enqueues nothing.  A launch failure returns
 *     P4Q_ERR_HIP.  No call synchronizes the device.
 *   - All pointers are device pointers owned by the caller.  The library
 *     keeps no pointer after it returns and allocates no device memory.
 *   - Matrices are row-major.  fp16 / bf16 tensors are IEEE binary16 /
 *     bfloat16 bit patterns.
 *   - The 4-bit quantizer Q4(x; c) of a row x (Appendix A, B.3):
 *         a = max_k |x_k|,  s = fl32(fl32(c * a) / 7),
 *         code_k = clamp(rne(fl32(x_k / s)), -8, 7)  (correctly rounded
 *         division, ties to even);  s == 0  =>  all codes 0.
 *     Packed codes hold two's-complement nibbles, the even k in the low
 *     nibble: byte t = (code[2t] & 0xF) | (code[2t+1] & 0xF) << 4.
 *   - The last error message of the calling thread is p4q_last_error().
 */
#ifndef P4Q_H
#define P4Q_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum p4q_status {
    P4Q_OK = 0,
    P4Q_ERR_INVALID_ARG = 1,   /* null pointer, bad size, misalignment, bad clip */
    P4Q_ERR_UNSUPPORTED = 2,   /* valid request outside what the kernels handle */
    P4Q_ERR_WORKSPACE = 3,     /* workspace missing or too small */
    P4Q_ERR_HIP = 4            /* a HIP launch or runtime call failed */
} p4q_status;

typedef enum p4q_dtype {
    P4Q_FP16 = 0,
    P4Q_BF16 = 1,
    /* Not dtypes: they widen the enumeration's range to every int, so that
     * any value a caller passes is a valid p4q_dtype for the implementation
     * (C++), and one other than the two above is rejected with
     * P4Q_ERR_UNSUPPORTED instead of being undefined behaviour. */
    P4Q_DTYPE_RANGE_MIN_ = -0x7FFFFFFF - 1,
    P4Q_DTYPE_RANGE_MAX_ = 0x7FFFFFFF
} p4q_dtype;

/* Library version string, e.g. "p4q 0.1.0 gfx950". */
const char *p4q_version(void);

/* Human-readable name of a status code. */
const char *p4q_status_string(int status);

/* Message describing the last failing call on this thread ("" if none). */
const char *p4q_last_error(void);

/* ------------------------------------------------------------------------
 * Quantization-aware visual-token selection (Sec. 3.2, Query Relevance).
 *
 * For each sample b < B:
 *   - cv_i = Q4(vis[b][i]; clip) and cq_j = Q4(concepts[b][j]; clip) are the
 *     fake-quantized copies (only their integer codes are needed: with
 *     v~ = s_v cv and q~ = s_q cq, CosSim(q~_j, v~_i) = D_ij / sqrt(Nv_i Nq_j)
 *     with D_ij = <cv_i, cq_j> and Nv_i = |cv_i|^2, exactly);
 *   - concept j ranks tokens by that cosine, higher first, equal cosines by
 *     lower token index (a zero code vector has cosine 0);
 *   - quotas k_j = floor(K/J) + (j < K mod J); for j = 0..J-1 in order, the
 *     first k_j tokens of concept j's ranking not already kept are kept
 *     (the Query-Relevance stage holding the whole budget);
 *   - idx_out[b][0..K) = kept token indices in ascending order;
 *   - tokens_out[b] = [vis[b][idx_out[b][0]], ..., vis[b][idx_out[b][K-1]],
 *                      text[b][0], ..., text[b][T-1]]  (bitwise copies of the
 *     original rows: the quantized copies are never materialized).
 *
 * Layouts:  vis [B, N, d], concepts [B, J, d], text [B, T, d] (dtype dt),
 *           idx_out int32 [B, K], tokens_out [B, K + T, d] (dtype dt).
 * Workspace: at least p4q_select_workspace_bytes(B, N, d, J) bytes, 256-byte
 *   aligned.  Its first B*N*(J+1) int32 hold, per token, D_i0 .. D_i(J-1)
 *   then Nv_i (layout [B][N][J+1]); the rest is internal.
 * Limits: 1 <= K <= N <= 8192, 1 <= J <= 8 (J <= 4 when d > 8192), T >= 0
 *   (text may be NULL iff T == 0), d % 32 == 0, 32 <= d <= 16384, clip in
 *   [2^-16, 1]; pointers 16-byte aligned.
 * Errors: P4Q_ERR_INVALID_ARG / P4Q_ERR_UNSUPPORTED / P4Q_ERR_WORKSPACE as
 *   above; nothing is enqueued on error.
 * ---------------------------------------------------------------------- */
size_t p4q_select_workspace_bytes(int B, int N, int d, int J);

int p4q_select(p4q_dtype dt, int B, int N, int d,
               const void *vis, const void *concepts, int J,
               const void *text, int T, int K, float clip,
               int32_t *idx_out, void *tokens_out,
               void *ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * p4q_select without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  It computes exactly what p4q_select
 * computes, with the same arguments, checks and results, and calls no
 * allocating routine.
 *
 * Its workspace is a static device array of P4Q_SELECT_SCRATCH_BYTES (8 MiB)
 * that every device the library runs on holds until the process ends.  A
 * call needs p4q_select_workspace_bytes(B, N, d, J) bytes of it (2.4 MB for
 * 16 images of 2880 tokens, d = 4096, J = 4); a larger request returns
 * P4Q_ERR_WORKSPACE and enqueues nothing.  No part of the array is read
 * before the same call has written it, so nothing needs clearing between
 * calls.  Calls on one device share the array: calls that overlap in time on
 * one device (concurrent streams, or host threads) race and must not be
 * issued.  The first call on a device looks up the array's device address
 * (with the stream's device current) and may fail with P4Q_ERR_HIP.
 * ---------------------------------------------------------------------- */
#define P4Q_SELECT_SCRATCH_BYTES (8u << 20)

int p4q_select_noalloc(p4q_dtype dt, int B, int N, int d,
                       const void *vis, const void *concepts, int J,
                       const void *text, int T, int K, float clip,
                       int32_t *idx_out, void *tokens_out, hipStream_t stream);

/* ------------------------------------------------------------------------
 * The three-stage quantization-aware selector (Sec. 3.2, Eq.
 * p4q_progressive_selection: Query Relevance, Visual Saliency, Visual
 * Diversity, with budgets kq + ks + kd = K).
 *
 * For each sample b < B, with the fake-quantized codes cv_i, cq_j of
 * p4q_select:
 *   1. Query Relevance keeps kq tokens, exactly as p4q_select with K = kq;
 *   2. Visual Saliency keeps, among the tokens not kept by stage 1, the ks
 *      with the largest cls_attn[b][i] (the vision tower's last-layer
 *      CLS-to-patch attention averaged over heads; equal weights: lower
 *      index first);
 *   3. Visual Diversity runs kd = K - kq - ks greedy steps; each keeps the
 *      remaining token whose largest cosine similarity to the tokens kept so
 *      far is smallest (equal values: lower index first), with
 *      cos(i, t) = <cv_i, cv_t> / sqrt(Nv_i Nv_t) (0 when either code vector
 *      is zero), compared exactly.  If stages 1-2 keep nothing, the first
 *      step keeps the most salient token (largest cls_attn, lower index
 *      first).
 *   idx_out[b][0..K) = all kept tokens, ascending; tokens_out as p4q_select.
 *   stages_out (may be NULL), int32 [B, K]: stage 1's tokens ascending, then
 *   stage 2's ascending, then stage 3's in the order they were kept.
 *
 * Layouts: as p4q_select; cls_attn fp32 [B, N], finite values.
 * Workspace: at least p4q_select_full_workspace_bytes(B, N, d, J, K) bytes,
 *   256-byte aligned; it holds the B code Gram matrices (B * N^2 int32).  Its
 *   first B*N*(J+1) int32 hold D and Nv as for p4q_select.
 * Limits: as p4q_select, plus d <= 8192 and 0 <= kq, 0 <= ks, kq + ks <= K;
 *   cls_attn 4-byte aligned, stages_out 4-byte aligned when given.
 * ---------------------------------------------------------------------- */
size_t p4q_select_full_workspace_bytes(int B, int N, int d, int J, int K);

/* The default budget split of Sec. 3.2 (alpha, beta, gamma) = (0.3, 0.2,
 * 0.5): kq = floor(3K/10), ks = floor(2K/10), kd = K - kq - ks.  Host-only;
 * P4Q_ERR_INVALID_ARG for K < 0 or a NULL output. */
int p4q_select_budgets(int K, int *kq, int *ks, int *kd);

int p4q_select_full(p4q_dtype dt, int B, int N, int d,
                    const void *vis, const void *concepts, int J,
                    const float *cls_attn, const void *text, int T,
                    int K, int kq, int ks, float clip,
                    int32_t *idx_out, int32_t *stages_out, void *tokens_out,
                    void *ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Per-row activation quantization + packing (Appendix A / B.3: per-token
 * int4 activations; the same call quantizes weight rows per output channel).
 *
 *   (codes[m], scales[m]) = Q4(x[m, 0..K_in); clip)   for m < M
 *
 * Layouts: x [M, ldx] (dtype dt, only the first K_in columns are read),
 *          codes uint8 [M, K_in/2] packed (see above), scales fp32 [M].
 * Limits: M >= 1, K_in % 32 == 0, 32 <= K_in <= 65536, ldx >= K_in,
 *   ldx % 8 == 0, clip in [2^-16, 1]; x and codes 16-byte aligned, scales
 *   4-byte aligned.
 * ---------------------------------------------------------------------- */
int p4q_quant_act(p4q_dtype dt, int M, int K_in, const void *x, int64_t ldx,
                  float clip, uint8_t *codes, float *scales, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Fused decoder prologue: per-token int4 quantization of RMSNorm(x) * gamma
 * without materializing the normalized rows (Appendix A / B.3: per-token
 * symmetric RTN activations; gamma is the RMSNorm weight, the per-channel
 * slot into which calibration's diagonal scales fold before RTN).
 *
 *   u[m][k]   = x[m][k] * gamma[k]                 (fp32, exact)
 *   codes[m]  = Q4(u[m]; clip).codes               (packed as above)
 *   scales[m] = fl32(Q4(u[m]; clip).scale / rms(x[m])),
 *   rms(x[m]) = sqrt(sum_k x[m][k]^2 / d + eps)     (fp32; summation order
 *               unspecified, so scales agree with an exact rms to ~1e-6)
 * Q4 is invariant under a positive factor per row, so these are the codes
 * and scale of RMSNorm(x[m]) * gamma; scales[m] = 0 when u[m] is all zero.
 *
 * Layouts: x [M, ldx] (dtype dt, first d columns read), gamma [d] (dtype
 *   dt), codes uint8 [M, d/2], scales fp32 [M].
 * Limits: M >= 1, d % 32 == 0, 32 <= d <= 16384, ldx >= d, ldx % 8 == 0,
 *   eps in [0, 1], clip in [2^-16, 1]; products x * gamma finite; x, gamma
 *   and codes 16-byte aligned, scales 4-byte aligned.
 * ---------------------------------------------------------------------- */
int p4q_rmsnorm_quant(p4q_dtype dt, int M, int d, const void *x, int64_t ldx,
                      const void *gamma, float eps, float clip,
                      uint8_t *codes, float *scales, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Attention prefill on the pruned sequence (Appendix B.3: W4A4 linears with
 * the key and value caches kept in FP16; this is the step after the q/k/v
 * linears of a decoder layer).
 *
 * For sample b < B, head h < H and token t < L:
 *   S[t, j] = <q[b,t,h,:], k[b,j,h,:]> / sqrt(D) over j <= t (causal = 1)
 *             or every j < L (causal = 0),
 *   out[b,t,h,:] = sum_j softmax_j(S[t, :]) v[b,j,h,:].
 * fp32 scores, softmax and accumulation; the softmax weights are rounded to
 * the input dtype before they multiply v (so outputs agree with an exact
 * evaluation to about 2^-10 (fp16) / 2^-7 (bf16) of max|v|); out is rounded
 * to the input dtype (nearest, ties to even).
 *
 * Layouts: element (b, t, h, d) of q, k and v is at ptr[(b L + t) ld + h D
 *   + d] -- so q, k, v can point into one fused q|k|v projection output
 *   with ld = 3 H D -- and of out at out[(b L + t) ld_out + h D + d].
 * Limits: D == 128; ld >= H D, ld % 8 == 0; ld_out >= H D, ld_out % 4 == 0;
 *   q, k, v 16-byte aligned, out 8-byte aligned; causal is 0 or 1.
 * ---------------------------------------------------------------------- */
int p4q_attention_prefill(p4q_dtype dt, int B, int L, int H, int D,
                          const void *q, const void *k, const void *v, int64_t ld,
                          void *out, int64_t ld_out, int causal, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Channel-scaled per-row quantizer (Sec. 3.3 and Appendix B.3: the diagonal
 * channel scales and clipping factors that calibration learns, applied
 * before RTN; also the folded-weight quantization after calibration).
 *
 *   z'[r][k] = fl32(z[r][k] / sigma[k])   (divide = 1: activation channels)
 *            = fl32(z[r][k] * sigma[k])   (divide = 0: weight input channels)
 *   (codes[r], scales[r]) = Q4(z'[r]; c_r),  c_r = clip_rows[r] or clip
 *   absmax[r] = max_k |z'[r][k]|,  kstar[r] = the lowest k attaining it
 *
 * Layouts: z [R, ldz] of dt; sigma fp32 [K] (> 0, z' finite); codes uint8
 *   [R, K/2] packed as p4q_quant_act's; scales, absmax fp32 [R]; kstar int32
 *   [R].  absmax and kstar may be NULL; clip_rows may be NULL (then clip,
 *   in (0, 1], serves every row; given, its entries should lie in (0, 1]).
 * Limits: R >= 1, K % 32 == 0, K <= 16384, ldz >= K and ldz % 8 == 0; z,
 *   sigma and codes 16-byte aligned.
 * ---------------------------------------------------------------------- */
int p4q_quant_scaled(p4q_dtype dt, int R, int K, const void *z, int64_t ldz,
                     const float *sigma, int divide, float clip,
                     const float *clip_rows, uint8_t *codes, float *scales,
                     float *absmax, int32_t *kstar, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Pruning-aware calibration step of one W4A4 linear (Sec. 3.3, Eq.
 * p4q_pruning_aware_calibration: the per-sample mean squared error between
 * the fake-quantized and the full-precision outputs on the pruned sequence;
 * Appendix B.3: diagonal channel scales and weight / activation clipping
 * factors are the learnable parameters).
 *
 *   X' = X / sigma, W' = W * sigma (per channel, as p4q_quant_scaled);
 *   (cA, sA) = Q4 rows of X' with clip_a; (cW, sW) = Q4 rows of W' with
 *   clip_w[n]; acc = cA cW^T (exact int32, int8 MFMA);
 *   R[m][n] = fl32(fl32(fl32(acc sA[m]) sW[n]) - target[m][n]);
 *   loss = sum R^2 / (M N)
 * and the gradients of loss with respect to sigma, clip_a and clip_w:
 * rounding passes gradients straight through, the clamp only where the
 * rounded quotient lies in [-8, 7], a row's maximum to its lowest-index
 * element.  The two contractions of the backward pass take bf16 operands
 * bf16(R sW[n]) and bf16(R sA[m]) (nearest even) against the exact codes,
 * with fp32 accumulation; every reduction after them is fp32 per tile and
 * float64 across tiles.
 *
 * Layouts: x [M, ldx] and w [N, ldw] of dt (the block input rows of the
 *   pruned sequence; the frozen weight); target fp32 [M, ldt] (the
 *   full-precision layer output); sigma fp32 [K] > 0; clip_w fp32 [N] in
 *   (0, 1]; outputs loss fp32 [1], grad_sigma fp32 [K], grad_clip_a fp32
 *   [1], grad_clip_w fp32 [N].
 * Workspace: p4q_calib_linear_workspace_bytes(M, N, K) bytes, 256-byte
 *   aligned, caller-owned; nothing of it is read before being written.
 * Limits: M >= 1, N % 64 == 0, K % 128 == 0, K <= 16384, M N and N K
 *   < 2^31; ldx, ldw >= K and multiples of 8; ldt >= N, multiple of 4;
 *   clip_a in (0, 1]; x, w, target, sigma 16-byte aligned.
 * The scatter of the row maxima's shares uses float64 atomics: results can
 *   differ between runs in the last bits of float64 sums, far below the
 *   fp32 outputs' precision.
 * ---------------------------------------------------------------------- */
size_t p4q_calib_linear_workspace_bytes(int M, int N, int K);

int p4q_calib_linear_grad(p4q_dtype dt, int M, int N, int K,
                          const void *x, int64_t ldx, const void *w, int64_t ldw,
                          const float *target, int64_t ldt, const float *sigma,
                          float clip_a, const float *clip_w, float *loss,
                          float *grad_sigma, float *grad_clip_a,
                          float *grad_clip_w, void *ws, size_t ws_bytes,
                          hipStream_t stream);

/* ------------------------------------------------------------------------
 * Pruning-aware calibration step of a whole decoder block (Sec. 3.3, Eq.
 * p4q_pruning_aware_calibration: calibration proceeds block by block, each
 * block's W4A4 fake-quantized output reconstructing the full-precision
 * block's output on the pruned sequence by mean squared error; Appendix
 * B.3: diagonal scales and weight / activation clipping factors learned,
 * keys and values in FP16).
 *
 * The block (LLaMA-family decoder, intermediates rounded once to fp16,
 * nearest even, between operations; H heads of D = d / H):
 *   n1 = RMSNorm(x) gamma1 (eps);   q|k|v = L_qkv(n1);
 *   q, k <- RoPE (channel i < D/2 paired with i + D/2, angle p theta_i,
 *           theta_i = rope_base^(-2i/D), p = the token's position 0..M-1);
 *   O = softmax(q k^T / sqrt(D), causal) v per head (fp32 arithmetic);
 *   h = x + L_o(O);  n2 = RMSNorm(h) gamma2;  g|u = L_gu(n2);
 *   a = SiLU(g) u;   out = h + L_down(a);
 *   loss = sum (out - target)^2 / (M d),
 * where every L is the W4A4 fake-quantized linear of p4q_calib_linear_grad
 * with its group's diagonal scales (dividing the input channels,
 * multiplying the weights' input channels), activation clipping factor and
 * per-output-channel weight clipping factors; its output is the W4A4
 * epilogue's out_rne(fl32(fl32(acc sA) sW)).  Returns the loss and its
 * gradients with respect to every group's sigma, clip_a and clip_w (rounding
 * of codes and of intermediates passed straight through, the clamp and the
 * row maxima as in p4q_calib_linear_grad), chained through the
 * full-precision attention, RMSNorm and SiLU-gated MLP; each group's
 * backward contractions take bf16 operands with fp32 accumulation.
 *
 * Groups, in this order: q|k|v (N = 3d, input width d), o (d, d), gate|up
 * (2f, d), down (d, f).
 * Layouts: x fp16 [M, d] (the block input on the pruned sequence); target
 *   fp32 [M, ldt] (the full-precision block's output); w_qkv fp16 [3d, d]
 *   (q, k, v rows), w_o [d, d], w_gu [2f, d] (gate rows, then up rows),
 *   w_down [d, f]; gamma1, gamma2 fp16 [d];
 *   sigma fp32 [3d + f] = [qkv: d | o: d | gate|up: d | down: f];
 *   clip_a: HOST array of 4 floats in (0, 1], one per group;
 *   clip_w fp32 [5d + 2f] = [qkv: 3d | o: d | gate|up: 2f | down: d];
 *   outputs loss fp32 [1], grad_sigma [3d + f], grad_clip_a [4] and
 *   grad_clip_w [5d + 2f] in the same layouts (device).
 * Workspace: p4q_calib_block_workspace_bytes(M, d, f, H) bytes, 256-byte
 *   aligned; nothing of it is read before being written.
 * Limits: dt == P4Q_FP16; 1 <= M <= 4096; d, f multiples of 128, <= 16384;
 *   d % H == 0 with D = d / H even; M * 2f < 2^31 and 3d * d, 2f * d < 2^31;
 *   ldt >= d; eps in [0, 1]; rope_base > 1; pointers 16-byte aligned.
 * ---------------------------------------------------------------------- */
size_t p4q_calib_block_workspace_bytes(int M, int d, int f, int H);

int p4q_calib_block_grad(p4q_dtype dt, int M, int d, int f, int H, const void *x,
                         const float *target, int64_t ldt, const void *w_qkv,
                         const void *w_o, const void *w_gu, const void *w_down,
                         const void *gamma1, const void *gamma2, float eps, float rope_base,
                         const float *sigma, const float *clip_a, const float *clip_w,
                         float *loss, float *grad_sigma, float *grad_clip_a,
                         float *grad_clip_w, void *ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * W4A4 linear (Appendix B.3: RTN int4 weights and activations for W4A4
 * inference): an integer GEMM on the codes and a dequant epilogue.
 *
 *   acc[m][n] = sum_k A[m][k] * W[n][k]                (exact int32)
 *   y[m][n]   = out_rne(fl32(fl32(float(acc) * a_scales[m]) * w_scales[n]))
 *
 * Layouts: a_codes uint8 [M, K_in/2] and w_codes uint8 [N_out, K_in/2]
 *   packed as above (both K-contiguous); a_scales fp32 [M]; w_scales fp32
 *   [N_out]; y [M, ldy] of out_dt; acc_out int32 [M, N_out] or NULL (when
 *   given, the raw accumulators are stored too).
 * Workspace (optional): p4q_w4a4_linear_workspace_bytes(M, N_out, K_in)
 *   bytes, 16-byte aligned.  It is nonzero for M < 1024 when the output
 *   tiles do not divide evenly over the CUs: given that much, the call
 *   splits K of the tiles past the last whole round across work-groups,
 *   which meet in the workspace (exact int32 partial sums; the last to
 *   arrive writes the tile), or, below 128 x 128 tiles, sums the slices in
 *   a second kernel.  With ws NULL, smaller or misaligned the call runs
 *   unsplit.  The results are identical either way (integer sums).  The
 *   first 4096 bytes hold per-tile arrival counters: they must be zero
 *   before the first call that uses the workspace (allocate it
 *   zero-filled), and every call leaves them zero.  Calls that share a
 *   workspace must not overlap.  The size depends on the current device
 *   (its number of compute units): query it with that device current.
 * Limits: M >= 1, N_out >= 1, K_in % 32 == 0, 32 <= K_in <= 131072,
 *   ldy >= N_out; code pointers 16-byte aligned, y 4-byte aligned.
 * ---------------------------------------------------------------------- */
size_t p4q_w4a4_linear_workspace_bytes(int M, int N_out, int K_in);

int p4q_w4a4_linear(int M, int N_out, int K_in,
                    const uint8_t *a_codes, const float *a_scales,
                    const uint8_t *w_codes, const float *w_scales,
                    p4q_dtype out_dt, void *y, int64_t ldy, int32_t *acc_out,
                    void *ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Diagnostics: microbenchmarks of the device's own ceilings, against which
 * the kernels above are reported beside the published peaks.  They are not
 * part of the method.
 *
 * p4q_diag_mfma_i8: `blocks` work-groups of 256 threads; every wavefront
 *   issues iters x 16 independent v_mfma_i32_16x16x64_i8 on pseudo-random
 *   operands, i.e. blocks * 4 * iters * 16 * 32768 integer operations.
 *   out int32 [blocks * 256] receives a checksum per thread.
 * p4q_diag_stream_read: reads the `bytes` (a multiple of 16) at src with
 *   `blocks` work-groups of 256 threads, 16 bytes per load;
 *   out uint32 [blocks * 256] receives a checksum per thread.
 * Limits: blocks in [1, 2^20], iters in [1, 2^20]; src 16-byte aligned,
 *   out 4-byte aligned.
 * ---------------------------------------------------------------------- */
int p4q_diag_mfma_i8(int blocks, int iters, int32_t *out, hipStream_t stream);

int p4q_diag_stream_read(const void *src, size_t bytes, int blocks, uint32_t *out,
                         hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* P4Q_H */
