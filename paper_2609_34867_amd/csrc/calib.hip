// Pruning-aware calibration mechanics (P4Q Sec. 3.3, Eq.
// p4q_pruning_aware_calibration; Appendix B.3): the reconstruction loss of one
// W4A4 fake-quantized linear on a pruned sequence and its gradients with
// respect to the learnable diagonal channel scales sigma and the activation /
// weight clipping factors.  Rounding passes gradients straight through; the
// clamp passes them where the rounded quotient lies in [-8, 7]; a row's
// maximum passes its share to its lowest-index element.
//
// One step, stream-ordered:
//   1. k_quant_scaled (x2): X' = fl32(X / sigma), W' = fl32(W * sigma); per
//      row Q4 with its clipping factor -> packed codes, scale, row maximum,
//      the maximum's lowest index, and one bit per value telling whether the
//      rounded quotient lay inside [-8, 7] (the activation side also keeps
//      X' in fp32).
//   2. k_codes_bf16t (x2): the codes transposed to bf16 [K][rows], the
//      contraction operands of the backward products (int4 codes are exact
//      in bf16).
//   3. The W4A4 GEMM (int8 MFMA) -> acc[M][N] int32.
//   4. k_calib_residual: R = fl32(fl32(fl32(acc sA) sW) - T); the bf16
//      operands P1 = bf16(R sW) [M][N] and P2^T = bf16(R sA) [N][Mp]; partial
//      sums of R^2.
//   5. k_calib_bwd (x2, bf16 MFMA, fp32 accumulation): dL/dXq ~ P1 Cw and
//      dL/dWq ~ P2^T Ca are never stored.  The epilogue takes each element's
//      code and inside bit from step 1 (the quantizer's own decisions, so no
//      division happens here) and reduces its tile to per-row sums of
//      g (code - inside z'/s) and per-column sums of g inside z'.  Both are
//      linear in g, so the contraction is split freely across work-groups,
//      each writing its own partial slot.
//   6. k_calib_rows: per row g_s (deterministic sum of the slots), the clip
//      gradients, and the row maximum's share g_s clip absmax / 7, added to
//      its column with float64 atomics.
//   7. k_calib_cols: with colX / colW the per-column totals of both sides,
//      d sigma_k = (2 / (M N)) (colW_k - colX_k) / sigma_k (the product
//      X W^T is unchanged when sigma divides one side and multiplies the
//      other); the loss and the activation clip gradient.
// The factor 2 / (M N) of the mean squared error is applied once, at the end.
#include "p4q_internal.h"
#include "q4_device.h"

#include <algorithm>

namespace p4q {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void *lds_ptr_t;

constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t bf16_rne(float v) {
    const uint32_t u = __float_as_uint(v);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

template <bool BF16>
__device__ __forceinline__ float half_to_f32(uint16_t h) {
    if constexpr (BF16) return __uint_as_float((uint32_t)h << 16);
    else return (float)__builtin_bit_cast(_Float16, h);
}

// z' of one stored value: correctly rounded fp32 division (activations) or
// product (weights)
template <bool DIV>
__device__ __forceinline__ float transform(float z, float sg) {
    if constexpr (DIV) return z / sg;
    else return __fmul_rn(z, sg);
}


__device__ __forceinline__ double block_sum(double v, double *red) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    const int t = threadIdx.x;
    if ((t & 63) == 0) red[t >> 6] = v;
    __syncthreads();
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) s += red[w];
    return s;
}

// ---------------------------------------------------------------------------
// 1. Transformed per-row quantizer.  One 256-thread work-group per row; the
//    transformed row stays in registers (CH chunks of 8 values per thread,
//    K <= 2048 CH).  The row maximum is a float maximum (non-negative
//    floats order as their bit patterns); its lowest index is searched for
//    afterwards, only by the threads that hold the maximum.
// ---------------------------------------------------------------------------
template <int CH, bool BF16, bool DIV>
__global__ __launch_bounds__(kThreads) void k_quant_scaled(
    const uint8_t *__restrict__ z, int64_t ldz_bytes, int nchunk, const float *__restrict__ sigma,
    float clip, const float *__restrict__ clip_rows, uint8_t *__restrict__ codes,
    int64_t ldc_bytes, float *__restrict__ scales, float *__restrict__ absmax,
    int32_t *__restrict__ kstar, float *__restrict__ zprime, uint8_t *__restrict__ inside) {
    __shared__ uint32_t s_red[kThreads / 64];
    const int row = blockIdx.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const uint4 *src = reinterpret_cast<const uint4 *>(z + (int64_t)row * ldz_bytes);
    const float4 *sg4 = reinterpret_cast<const float4 *>(sigma);

    float zp[CH][8];
    float am = 0.0f;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int q = t + kThreads * c;
        if (q < nchunk) {
            const uint4 v = load_nt(src + q);
            const float4 s0 = sg4[2 * q], s1 = sg4[2 * q + 1];
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
            const float sg[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                zp[c][2 * i] = transform<DIV>(lo_f32<BF16>(w[i]), sg[2 * i]);
                zp[c][2 * i + 1] = transform<DIV>(hi_f32<BF16>(w[i]), sg[2 * i + 1]);
            }
            if (zprime) {
                float4 *zo = reinterpret_cast<float4 *>(zprime + (int64_t)row * (8 * nchunk) + 8 * q);
                zo[0] = make_float4(zp[c][0], zp[c][1], zp[c][2], zp[c][3]);
                zo[1] = make_float4(zp[c][4], zp[c][5], zp[c][6], zp[c][7]);
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) am = __builtin_fmaxf(am, __builtin_fabsf(zp[c][e]));
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) zp[c][e] = 0.0f;
        }
    }
    const uint32_t mw = wave_max_u32(__float_as_uint(am));
    if (lane == 0) s_red[wave] = mw;
    __syncthreads();
    const uint32_t abits = max(max(s_red[0], s_red[1]), max(s_red[2], s_red[3]));
    const float a = __uint_as_float(abits);
    const float cl = clip_rows ? clip_rows[row] : clip;
    const float s = __fmul_rn(cl, a) / 7.0f;
    if (kstar) {                                             // block-uniform
        // lowest k with |z'_k| = a: only threads holding the maximum look
        uint32_t nk = 0u;                                    // ~k, maximised
        if (__float_as_uint(am) == abits) {
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                const int q = t + kThreads * c;
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (q < nchunk && __float_as_uint(__builtin_fabsf(zp[c][e])) == abits)
                        nk = max(nk, ~(uint32_t)(8 * q + e));
            }
        }
        const uint32_t wk = wave_max_u32(nk);
        __syncthreads();                                     // every read of s_red above is done
        if (lane == 0) s_red[wave] = wk;
        __syncthreads();
        if (t == 0) kstar[row] = (int32_t)~max(max(s_red[0], s_red[1]), max(s_red[2], s_red[3]));
    }
    if (t == 0) {
        scales[row] = s;
        if (absmax) absmax[row] = a;
    }

    uint32_t *dst = reinterpret_cast<uint32_t *>(codes + (int64_t)row * ldc_bytes);
    const bool tiny = !(s >= kTinyScale);
    const float r = tiny ? 0.0f : 1.0f / s;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int q = t + kThreads * c;
        uint32_t packed = 0u, ins = 0xFFu;
        if (s != 0.0f) {
            uint32_t w[8];
            float fm = 0.0f;
            ins = 0u;
            if (!tiny) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float tq = __builtin_fmaf(zp[c][e], r, kRneMagic);
                    const float qq = tq - kRneMagic;
                    fm = __builtin_fmaxf(fm, __builtin_fabsf(__builtin_fmaf(zp[c][e], r, -qq)));
                    const float tc = __builtin_amdgcn_fmed3f(tq, kRneMagic - 8.0f, kRneMagic + 7.0f);
                    ins |= (uint32_t)(tc == tq) << e;
                    w[e] = __float_as_uint(tc);
                }
            }
            // a value within 2^-19 of a rounding boundary somewhere in the
            // wave (or a tiny scale): this chunk by exact division
            if (tiny || __any(fm > kNearHalf)) {
                ins = 0u;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float rq = __builtin_rintf(zp[c][e] / s);
                    const float cq = __builtin_amdgcn_fmed3f(rq, -8.0f, 7.0f);
                    ins |= (uint32_t)(cq == rq) << e;
                    w[e] = (uint32_t)(int)cq;
                }
            }
            packed = pack_nibbles(w);
        }
        if (q < nchunk) {
            dst[q] = packed;
            if (inside) inside[(int64_t)row * nchunk + q] = (uint8_t)ins;
        }
    }
}

template <int CH, bool BF16, bool DIV>
hipError_t launch_qs(int R, int nchunk, const void *z, int64_t ldz_bytes, const float *sigma,
                     float clip, const float *clip_rows, uint8_t *codes, int64_t ldc_bytes,
                     float *scales, float *absmax, int32_t *kstar, float *zprime,
                     uint8_t *inside, hipStream_t stream) {
    hipLaunchKernelGGL((k_quant_scaled<CH, BF16, DIV>), dim3(R), dim3(kThreads), 0, stream,
                       static_cast<const uint8_t *>(z), ldz_bytes, nchunk, sigma, clip, clip_rows,
                       codes, ldc_bytes, scales, absmax, kstar, zprime, inside);
    return hipGetLastError();
}

template <bool BF16, bool DIV>
hipError_t launch_qs_typed(int R, int K, const void *z, int64_t ldz, const float *sigma,
                           float clip, const float *clip_rows, uint8_t *codes, float *scales,
                           float *absmax, int32_t *kstar, hipStream_t stream,
                           float *zprime = nullptr, uint8_t *inside = nullptr) {
    const int nchunk = K / 8;
    const int per = (nchunk + kThreads - 1) / kThreads;      // <= 8 (K <= 16384)
#define P4Q_QS(N)                                                                          \
    return launch_qs<N, BF16, DIV>(R, nchunk, z, ldz * 2, sigma, clip, clip_rows, codes,  \
                                   K / 2, scales, absmax, kstar, zprime, inside, stream)
    if (per <= 1) P4Q_QS(1);
    if (per <= 2) P4Q_QS(2);
    if (per <= 4) P4Q_QS(4);
    if (per <= 6) P4Q_QS(6);
    P4Q_QS(8);
#undef P4Q_QS
}

// ---------------------------------------------------------------------------
// 2. Packed codes [R][K/2] -> bf16 [K][ldo], rows R..ldo-1 of the output's
//    columns zero.  64 (rows) x 128 (k) tiles through LDS as int8.
// ---------------------------------------------------------------------------
constexpr int kT8Stride = 132;        // bytes per LDS row: rows 32 apart land 32 banks apart

__global__ __launch_bounds__(kThreads) void k_codes_bf16t(const uint8_t *__restrict__ codes,
                                                          int R, int Kb,
                                                          uint16_t *__restrict__ out,
                                                          int64_t ldo) {
    __shared__ __attribute__((aligned(16))) uint8_t s8[64 * kT8Stride];
    const int t = threadIdx.x;
    const int r0 = blockIdx.x * 64, k0 = blockIdx.y * 128;
    {
        const int rl = t >> 2, c = t & 3, r = r0 + rl;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (r < R) v = *reinterpret_cast<const uint4 *>(codes + (int64_t)r * Kb + k0 / 2 + 16 * c);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
        uint32_t *d = reinterpret_cast<uint32_t *>(s8 + rl * kT8Stride + 32 * c);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            // nibbles k = 8i .. 8i+7 -> sign-extended bytes, k order
            uint32_t o[2] = {0u, 0u};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int nib = (int)((w[i] >> (4 * e)) & 0xFu);
                const uint32_t b = (uint32_t)(uint8_t)(int8_t)((nib ^ 8) - 8);
                o[e >> 2] |= b << (8 * (e & 3));
            }
            d[2 * i] = o[0];
            d[2 * i + 1] = o[1];
        }
    }
    __syncthreads();
    {
        const int kl = t >> 1, h = t & 1;
        uint32_t pk[16];
#pragma unroll
        for (int e = 0; e < 32; e += 2) {
            const float a = (float)(int8_t)s8[(32 * h + e) * kT8Stride + kl];
            const float b = (float)(int8_t)s8[(32 * h + e + 1) * kT8Stride + kl];
            pk[e >> 1] = (__float_as_uint(a) >> 16) | (__float_as_uint(b) & 0xFFFF0000u);
        }
        uint4 *dst = reinterpret_cast<uint4 *>(out + (int64_t)(k0 + kl) * ldo + r0 + 32 * h);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            dst[q] = make_uint4(pk[4 * q], pk[4 * q + 1], pk[4 * q + 2], pk[4 * q + 3]);
    }
}

// Wide variant for the weight codes (many rows): a 256-row x 128-k tile, so
// each half-wavefront writes 512 consecutive bytes of one output row.  The
// int8 tile sits in LDS as [row][32 words of 4 k]; word q of row r is stored
// at slot q ^ g(r), g(r) = ((r >> 3) ^ ((r & 7) << 2)) & 31, so the 32 lanes
// that read rows 8 rc + j (rc = 0 .. 31) at one word hit 32 distinct banks.
constexpr int kTWide = 256;

__device__ __forceinline__ int wide_swz(int r) { return ((r >> 3) ^ ((r & 7) << 2)) & 31; }

__global__ __launch_bounds__(kThreads) void k_codes_bf16t_wide(const uint8_t *__restrict__ codes,
                                                               int R, int Kb,
                                                               uint16_t *__restrict__ out,
                                                               int64_t ldo) {
    __shared__ uint32_t s32[kTWide * 32];
    const int t = threadIdx.x;
    const int r0 = blockIdx.x * kTWide, k0 = blockIdx.y * 128;
#pragma unroll
    for (int p = 0; p < kTWide / 64; ++p) {
        const int rl = 64 * p + (t >> 2), c = t & 3, r = r0 + rl;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (r < R) v = *reinterpret_cast<const uint4 *>(codes + (int64_t)r * Kb + k0 / 2 + 16 * c);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
        const int g = wide_swz(rl);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            // nibbles k = 32 c + 8 i .. +7 -> sign-extended bytes, k order:
            // words 8 c + 2 i and 8 c + 2 i + 1
            uint32_t o[2] = {0u, 0u};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int nib = (int)((w[i] >> (4 * e)) & 0xFu);
                const uint32_t b = (uint32_t)(uint8_t)(int8_t)((nib ^ 8) - 8);
                o[e >> 2] |= b << (8 * (e & 3));
            }
            s32[rl * 32 + ((8 * c + 2 * i) ^ g)] = o[0];
            s32[rl * 32 + ((8 * c + 2 * i + 1) ^ g)] = o[1];
        }
    }
    __syncthreads();
    // thread (rc, kq): rows 8 rc .. 8 rc + 7, k words kq, kq + 8, kq + 16, kq + 24
    const int rc = t & 31, kq = t >> 5;
    const bool in = r0 + 8 * rc < R;                         // R is a multiple of 8
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int kw = kq + 8 * i;
        uint32_t wv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) wv[j] = s32[(8 * rc + j) * 32 + (kw ^ ((rc ^ (j << 2)) & 31))];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            uint32_t pk[4];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const float a = (float)(int8_t)(uint8_t)(wv[2 * m] >> (8 * e));
                const float b = (float)(int8_t)(uint8_t)(wv[2 * m + 1] >> (8 * e));
                pk[m] = (__float_as_uint(a) >> 16) | (__float_as_uint(b) & 0xFFFF0000u);
            }
            if (in)
                *reinterpret_cast<uint4 *>(out + (int64_t)(k0 + 4 * kw + e) * ldo + r0 + 8 * rc) =
                    make_uint4(pk[0], pk[1], pk[2], pk[3]);
        }
    }
}

// ---------------------------------------------------------------------------
// 4. Residual, bf16 contraction operands and loss partials.  64 x 64 tiles;
//    grid (N / 64, Mp / 64).  The grid also clears the float64 scatter
//    targets of k_calib_rows.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_calib_residual(
    const int32_t *__restrict__ acc, const float *__restrict__ sa, const float *__restrict__ sw,
    const float *__restrict__ T, int64_t ldt, int M, int N, int Mp, uint16_t *__restrict__ P1,
    uint16_t *__restrict__ P2T, double *__restrict__ loss_part, double *__restrict__ corr,
    int ncorr) {
    __shared__ __attribute__((aligned(16))) uint16_t tr[64 * 72];   // [n][m] bf16(R sA)
    __shared__ double red[kThreads / 64];
    const int t = threadIdx.x;
    const int n0 = blockIdx.x * 64, m0 = blockIdx.y * 64;
    const int bid = blockIdx.y * gridDim.x + blockIdx.x;
    const int nb = gridDim.x * gridDim.y;
    for (int i = bid * kThreads + t; i < ncorr; i += nb * kThreads) corr[i] = 0.0;

    const int cn = 4 * (t & 15);
    const float4 swv = *reinterpret_cast<const float4 *>(sw + n0 + cn);
    const float swa[4] = {swv.x, swv.y, swv.z, swv.w};
    double l2 = 0.0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int ml = (t >> 4) + 16 * i, m = m0 + ml;
        if (m < M) {
            const int4 a = *reinterpret_cast<const int4 *>(acc + (int64_t)m * N + n0 + cn);
            const float4 tv = *reinterpret_cast<const float4 *>(T + (int64_t)m * ldt + n0 + cn);
            const int av[4] = {a.x, a.y, a.z, a.w};
            const float ta[4] = {tv.x, tv.y, tv.z, tv.w};
            const float s = sa[m];
            uint32_t p[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float y = __fmul_rn(__fmul_rn((float)av[e], s), swa[e]);
                const float r = __fsub_rn(y, ta[e]);
                l2 += (double)r * (double)r;
                p[e] = bf16_rne(__fmul_rn(r, swa[e]));
                tr[(cn + e) * 72 + ml] = (uint16_t)bf16_rne(__fmul_rn(r, s));
            }
            *reinterpret_cast<uint2 *>(P1 + (int64_t)m * N + n0 + cn) =
                make_uint2(p[0] | (p[1] << 16), p[2] | (p[3] << 16));
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) tr[(cn + e) * 72 + ml] = 0;
        }
    }
    __syncthreads();
    {
        const int nl = t >> 2, c = t & 3;
        const uint4 *sp = reinterpret_cast<const uint4 *>(tr + nl * 72 + 16 * c);
        uint4 *dp = reinterpret_cast<uint4 *>(P2T + (int64_t)(n0 + nl) * Mp + m0 + 16 * c);
        dp[0] = sp[0];
        dp[1] = sp[1];
    }
    const double s = block_sum(l2, red);
    if (t == 0) loss_part[bid] = s;
}

// ---------------------------------------------------------------------------
// 5. Backward contraction O[i][k] = sum_j P[i][j] C[k][j] (bf16 operands,
//    fp32 accumulation on v_mfma_f32_32x32x16_bf16) with the fused reduction
//    epilogue.  128 x 128 tiles, 4 wavefronts of 64 (i) x 64 (k), each 2 x 2
//    MFMA tiles with C as the first operand, so that a lane's accumulators
//    hold four consecutive k of one i; 64 j per stage, two LDS stages filled
//    by buffer_load ... lds (rows past I read as zeros).  LDS rows are 128
//    bytes; 16-byte chunk c of row r sits at chunk c ^ ((r >> 1) & 7), so the
//    16 rows one fragment read touches hit distinct banks.
//    grid (Kd / 128, ceil(I / 128), splits); split z covers j in
//    [z js, min(J, (z + 1) js)).  Outputs: rowpart[(kt splits + z) I + i],
//    colpart[(it splits + z) Kd + k], and when gpart is given the values
//    inside ? g : 0 themselves at gpart[(z I + i) Kd + k] (the direct part of
//    the gradient with respect to the transformed input, per split).
// ---------------------------------------------------------------------------
constexpr int BB = 128;
constexpr int BJ = 64;
constexpr int kHalfStage = BB * BJ * 2;        // 16 KB: one operand
constexpr int kStage = 2 * kHalfStage;
// epilogue LDS rows (bytes); strides chosen so that the 32 rows a half-wave
// reads at one column offset fall in distinct banks
constexpr int kZStride = 264;                  // 128 16-bit values + 8
constexpr int kCStride = 68;                   // 64 bytes of packed codes + 4
constexpr int kBStride = 20;                   // 16 bytes of inside bits + 4
constexpr int kOffC = BB * kZStride;
constexpr int kOffB = kOffC + BB * kCStride;
constexpr int kOffS = kOffB + BB * kBStride;
static_assert(kOffS + 10 * BB * 4 <= 2 * kStage, "epilogue LDS");

__device__ __forceinline__ v4i buffer_rsrc(const void *base, uint32_t bytes) {
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    return v4i{(int)(uint32_t)b, (int)((b >> 32) & 0xFFFFu), (int)bytes, 0x00020000};
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16(v4i desc, uint32_t voffset, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                 :
                 : "v"(voffset), "s"(desc), "s"(lds)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ v16f mfma_bf16(uint4 a, uint4 b, v16f c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, a),
                                                   __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
}

// Epilogue per element (g = the contraction's value at (i, k), z' the
// transformed input, code and inside bit as the quantizer decided them,
// f = z'/s - code, taken only where inside):
//   row sum i    += g (code - inside z'/s) = inside ? -g f : g code
//   column sum k += inside ? g z' : 0
template <bool BF16, bool DIV>
__global__ __launch_bounds__(kThreads, 2) void k_calib_bwd(
    const uint16_t *__restrict__ P, int64_t ldp, const uint16_t *__restrict__ C, int64_t ldc,
    int I, int J, int js, const uint16_t *__restrict__ Z, int64_t ldz,
    const float *__restrict__ zprime, const uint8_t *__restrict__ codes,
    const uint8_t *__restrict__ inside, const float *__restrict__ sigma,
    const float *__restrict__ srow, int Kd, float *__restrict__ rowpart,
    float *__restrict__ colpart, float *__restrict__ gpart) {
    __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * kStage];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int wi = wave >> 1, wk = wave & 1;
    const int kt = blockIdx.x, it = blockIdx.y, split = blockIdx.z, nsplit = gridDim.z;
    const int i0 = it * BB, k0 = kt * BB;
    const int jb = split * js;
    const int nst = max(0, min(J - jb, js)) / BJ;

    const v4i dP = buffer_rsrc(P + (int64_t)i0 * ldp, (uint32_t)(min(I - i0, BB) * ldp * 2));
    const v4i dC = buffer_rsrc(C + (int64_t)k0 * ldc, (uint32_t)(BB * ldc * 2));
    // DMA: one 1 KB instruction fills 8 LDS rows; lane L -> row +L/8, slot
    // L%8, which holds chunk (L%8) ^ ((row >> 1) & 7).  Wave w copies rows
    // [32w, 32w + 32) of both operands.
    uint32_t voP[4], voC[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) {
        const int row = 32 * wave + 8 * n + (lane >> 3);
        const uint32_t lc = (uint32_t)((lane & 7) ^ ((row >> 1) & 7));
        voP[n] = (uint32_t)(row * ldp * 2) + lc * 16u;
        voC[n] = (uint32_t)(row * ldc * 2) + lc * 16u;
    }
    const uint32_t lds0 = (uint32_t)(size_t)(lds_ptr_t)smem +
                          (uint32_t)__builtin_amdgcn_readfirstlane(wave) * 32u * 128u;
    auto issue = [&](int slot, int st) __attribute__((always_inline)) {
        const uint32_t jo = (uint32_t)(jb + st * BJ) * 2u;
#pragma unroll
        for (int n = 0; n < 4; ++n) {
            lds_dma16(dP, voP[n] + jo, lds0 + slot * kStage + n * 1024);
            lds_dma16(dC, voC[n] + jo, lds0 + slot * kStage + kHalfStage + n * 1024);
        }
    };

    // acc[kx][iy]: rows k = wk*64 + 32kx + 8(r/4) + 4(l/32) + r%4, column
    // i = wi*64 + 32iy + l%32
    v16f acc[2][2];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[x][y][e] = 0.0f;

    const int r32 = lane & 31, g2 = lane >> 5;
    uint32_t fp[2], fc[2];
#pragma unroll
    for (int x = 0; x < 2; ++x) {
        fp[x] = (uint32_t)((wi * 64 + 32 * x + r32) * 128);
        fc[x] = (uint32_t)(kHalfStage + (wk * 64 + 32 * x + r32) * 128);
    }
    const uint32_t swz = (uint32_t)((r32 >> 1) & 7);    // (row >> 1) & 7 of every fragment row

    // the epilogue's inputs, fetched now so that their latency overlaps the
    // first stage's: weight tile (16-bit), packed codes, inside bits, row
    // scale and sigma
    const int64_t cb = Kd / 2, ib = Kd / 8;                  // row bytes of codes, inside bits
    uint4 zpre[DIV ? 1 : 8], cpre[2], bpre = make_uint4(0u, 0u, 0u, 0u);
    float spre = 0.0f, gpre = 0.0f;
    if constexpr (!DIV) {
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const int idx = t + kThreads * c, r = idx >> 4, q = idx & 15, i = i0 + r;
            zpre[c] = (i < I) ? *reinterpret_cast<const uint4 *>(Z + (int64_t)i * ldz + k0 + 8 * q)
                              : make_uint4(0u, 0u, 0u, 0u);
        }
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        const int idx = t + kThreads * c, r = idx >> 2, q = idx & 3, i = i0 + r;
        cpre[c] = (i < I) ? *reinterpret_cast<const uint4 *>(codes + (int64_t)i * cb + k0 / 2 + 16 * q)
                          : make_uint4(0u, 0u, 0u, 0u);
    }
    if (t < BB) {
        const int i = i0 + t;
        if (i < I) {
            bpre = *reinterpret_cast<const uint4 *>(inside + (int64_t)i * ib + k0 / 8);
            spre = srow[i];
        }
        gpre = sigma[k0 + t];
    }

    if (nst > 0) issue(0, 0);
    for (int st = 0; st < nst; ++st) {
        // stage st has landed from every wave, and every wave is done with
        // stage st - 1, whose slot the next DMA overwrites
        asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
        if (st + 1 < nst) issue((st + 1) & 1, st + 1);
        const uint8_t *base = smem + (st & 1) * kStage;
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
            const uint32_t ch = (((uint32_t)(2 * s4 + g2)) ^ swz) * 16u;
            uint4 a[2], b[2];
#pragma unroll
            for (int x = 0; x < 2; ++x) {
                a[x] = *reinterpret_cast<const uint4 *>(base + fc[x] + ch);
                b[x] = *reinterpret_cast<const uint4 *>(base + fp[x] + ch);
            }
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y) acc[x][y] = mfma_bf16(a[x], b[y], acc[x][y]);
        }
    }

    // ---- epilogue: the tile's inputs, codes and inside bits to LDS ----
    __syncthreads();
    float *s_r = reinterpret_cast<float *>(smem + kOffS);    // 1 / (s P)
    float *s_p = s_r + BB;                                   // P = 1, or 2^64 for s < 2^-100
    float *s_m = s_p + BB;                                   // 1, or 0 (zero row / past I)
    float *s_g = s_m + BB;                                   // sigma of the tile's columns
    float *rowred = s_g + BB;                                // [2][128]
    float *colred = rowred + 2 * BB;                         // [2][128]
    if constexpr (!DIV) {
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            const int idx = t + kThreads * c, r = idx >> 4, q = idx & 15;
            uint2 *d = reinterpret_cast<uint2 *>(smem + r * kZStride + 16 * q);
            d[0] = make_uint2(zpre[c].x, zpre[c].y);
            d[1] = make_uint2(zpre[c].z, zpre[c].w);
        }
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        const int idx = t + kThreads * c, r = idx >> 2, q = idx & 3;
        uint32_t *d = reinterpret_cast<uint32_t *>(smem + kOffC + r * kCStride + 16 * q);
        d[0] = cpre[c].x; d[1] = cpre[c].y; d[2] = cpre[c].z; d[3] = cpre[c].w;
    }
    if (t < BB) {
        uint32_t *d = reinterpret_cast<uint32_t *>(smem + kOffB + t * kBStride);
        d[0] = bpre.x; d[1] = bpre.y; d[2] = bpre.z; d[3] = bpre.w;
        const float s = spre;
        const bool tiny = s < 0x1p-100f;
        const float pw = tiny ? 0x1p64f : 1.0f;
        s_r[t] = (s != 0.0f) ? 1.0f / (s * pw) : 0.0f;
        s_p[t] = pw;
        s_m[t] = (s != 0.0f) ? 1.0f : 0.0f;
        s_g[t] = gpre;
    }
    __syncthreads();

    float rowv[2] = {0.0f, 0.0f};
    float colv[32];
#pragma unroll
    for (int v = 0; v < 32; ++v) colv[v] = 0.0f;
    float rs[2], pw[2], gm[2];
#pragma unroll
    for (int y = 0; y < 2; ++y) {
        const int il = wi * 64 + 32 * y + r32;
        rs[y] = s_r[il];
        pw[y] = s_p[il];
        gm[y] = s_m[il];
    }
    const int ish = 4 * g2;                   // bit of k = kb within its inside byte
#pragma unroll
    for (int x = 0; x < 2; ++x) {
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
            const int kb = wk * 64 + 32 * x + 8 * rg + 4 * g2;      // 4 consecutive k
            const float4 sg = *reinterpret_cast<const float4 *>(s_g + kb);
            const float sgv[4] = {sg.x, sg.y, sg.z, sg.w};
#pragma unroll
            for (int y = 0; y < 2; ++y) {
                const int il = wi * 64 + 32 * y + r32;
                float zp[4];
                if constexpr (DIV) {
                    const float4 v = *reinterpret_cast<const float4 *>(
                        zprime + (int64_t)min(i0 + il, I - 1) * Kd + k0 + kb);
                    zp[0] = v.x; zp[1] = v.y; zp[2] = v.z; zp[3] = v.w;
                } else {
                    const uint2 v = *reinterpret_cast<const uint2 *>(smem + il * kZStride + 2 * kb);
                    zp[0] = __fmul_rn(half_to_f32<BF16>((uint16_t)(v.x & 0xFFFFu)), sgv[0]);
                    zp[1] = __fmul_rn(half_to_f32<BF16>((uint16_t)(v.x >> 16)), sgv[1]);
                    zp[2] = __fmul_rn(half_to_f32<BF16>((uint16_t)(v.y & 0xFFFFu)), sgv[2]);
                    zp[3] = __fmul_rn(half_to_f32<BF16>((uint16_t)(v.y >> 16)), sgv[3]);
                }
                const uint32_t cw = *reinterpret_cast<const uint16_t *>(
                    smem + kOffC + il * kCStride + kb / 2);
                const uint32_t bw = (uint32_t)smem[kOffB + il * kBStride + kb / 8] >> ish;
                float gi[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float g = acc[x][y][4 * rg + e] * gm[y];
                    const float q = (float)(((int)(cw << (28 - 4 * e))) >> 28);
                    const bool in = (bw >> e) & 1u;
                    const float f = __builtin_fmaf(zp[e] * pw[y], rs[y], -q);
                    rowv[y] = __builtin_fmaf(g, in ? -f : q, rowv[y]);
                    colv[16 * x + 4 * rg + e] = __builtin_fmaf(in ? g : 0.0f, zp[e],
                                                               colv[16 * x + 4 * rg + e]);
                    gi[e] = in ? g : 0.0f;
                }
                if (gpart != nullptr && i0 + il < I)
                    *reinterpret_cast<float4 *>(gpart + ((int64_t)split * I + i0 + il) * Kd + k0 + kb) =
                        make_float4(gi[0], gi[1], gi[2], gi[3]);
            }
        }
    }
    // columns: the 32 values of each half-wave summed over its 32 lanes (the
    // i direction) by a halving exchange; lane l ends with value index l % 32
#pragma unroll
    for (int m = 16; m >= 1; m >>= 1) {
        const bool up = (lane & m) != 0;
#pragma unroll
        for (int v = 0; v < m; ++v) {
            // the asm keeps the two selects on values: a select between two
            // elements of the array would otherwise become an indexed access
            float lo = colv[v], hi = colv[v + m];
            asm volatile("" : "+v"(lo), "+v"(hi));
            const float send = up ? lo : hi;
            const float keep = up ? hi : lo;
            colv[v] = keep + __shfl_xor(send, m);
        }
    }
    {
        const int v = r32, x = v >> 4, rg = (v >> 2) & 3, e = v & 3;
        colred[wi * BB + wk * 64 + 32 * x + 8 * rg + 4 * g2 + e] = colv[0];
    }
#pragma unroll
    for (int y = 0; y < 2; ++y) {
        const float r = rowv[y] + __shfl_xor(rowv[y], 32);
        if (g2 == 0) rowred[wk * BB + wi * 64 + 32 * y + r32] = r;
    }
    __syncthreads();
    if (t < BB) {
        if (i0 + t < I)
            rowpart[((int64_t)kt * nsplit + split) * I + i0 + t] = rowred[t] + rowred[BB + t];
    } else {
        const int k = t - BB;
        colpart[((int64_t)it * nsplit + split) * Kd + k0 + k] = colred[k] + colred[BB + k];
    }
}

// ---------------------------------------------------------------------------
// 6-7. Finishing sums over the partial slots, in a fixed order: RB rows (or
//    columns) per 256-thread block, the slots dealt round-robin to 256 / RB
//    groups of RB threads, each thread keeping four loads in flight.
// ---------------------------------------------------------------------------
template <int G>
__device__ __forceinline__ double slot_sum(const float *__restrict__ p, int n, int64_t stride,
                                           int g) {
    double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
    int s = g;
    for (; s + 3 * G < n; s += 4 * G) {
        a0 += (double)p[(int64_t)s * stride];
        a1 += (double)p[(int64_t)(s + G) * stride];
        a2 += (double)p[(int64_t)(s + 2 * G) * stride];
        a3 += (double)p[(int64_t)(s + 3 * G) * stride];
    }
    for (; s < n; s += G) a0 += (double)p[(int64_t)s * stride];
    return (a0 + a1) + (a2 + a3);
}

// groups' partial sums -> the total for row / column t (valid in t < RB)
template <int RB>
__device__ __forceinline__ double group_total(double v, double *part) {
    const int t = threadIdx.x;
    part[t] = v;
    __syncthreads();
    double s = 0.0;
    if (t < RB)
        for (int g = 0; g < kThreads / RB; ++g) s += part[RB * g + t];
    return s;
}

constexpr int kRowsA = 16;     // activation rows per block (their slots are many)
constexpr int kRowsW = 64;     // weight rows, columns per block

// 6. Rows: g_s, the clip gradients, and the row maximum's share scattered
//    to its column.  Blocks [0, nbA) hold activation rows, the rest weight
//    rows.
__global__ __launch_bounds__(kThreads) void k_calib_rows(
    const float *__restrict__ rowA, int nsA, int M, const float *__restrict__ sA,
    const float *__restrict__ aA, const int32_t *__restrict__ kA, float clip_a,
    const float *__restrict__ rowW, int nsW, int N, const float *__restrict__ sW,
    const float *__restrict__ aW, const int32_t *__restrict__ kW,
    const float *__restrict__ clip_w, int nbA, double scale, double *__restrict__ corrA,
    double *__restrict__ corrW, double *__restrict__ dclipa_part,
    float *__restrict__ grad_clip_w) {
    __shared__ double part[kThreads];
    const int t = threadIdx.x;
    if ((int)blockIdx.x < nbA) {
        const int m = blockIdx.x * kRowsA + (t % kRowsA);
        const double gs = group_total<kRowsA>(
            m < M ? slot_sum<kThreads / kRowsA>(rowA + m, nsA, M, t / kRowsA) : 0.0, part);
        if (t < 64) {
            double v = 0.0;
            if (t < kRowsA && m < M) {
                const double a = (double)aA[m];
                if (sA[m] != 0.0f) atomicAdd(&corrA[kA[m]], gs * (double)clip_a * a / 7.0);
                v = gs * a / 7.0;
            }
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
            if (t == 0) dclipa_part[blockIdx.x] = v;
        }
    } else {
        const int n = (blockIdx.x - nbA) * kRowsW + (t % kRowsW);
        const double gs = group_total<kRowsW>(
            n < N ? slot_sum<kThreads / kRowsW>(rowW + n, nsW, N, t / kRowsW) : 0.0, part);
        if (t < kRowsW && n < N) {
            const double a = (double)aW[n];
            if (sW[n] != 0.0f) atomicAdd(&corrW[kW[n]], gs * (double)clip_w[n] * a / 7.0);
            grad_clip_w[n] = (float)(scale * gs * a / 7.0);
        }
    }
}

// 7. Columns: d sigma; block 0 also reduces the loss and d clip_a.
__global__ __launch_bounds__(kThreads) void k_calib_cols(
    const float *__restrict__ colA, int nslA, const float *__restrict__ colW, int nslW,
    const double *__restrict__ corrA, const double *__restrict__ corrW,
    const float *__restrict__ sigma, int K, double scale, float *__restrict__ grad_sigma,
    const double *__restrict__ loss_part, int nloss, double inv_mn, float *__restrict__ loss,
    const double *__restrict__ dclipa_part, int nbA, float *__restrict__ grad_clip_a) {
    __shared__ double part[kThreads];
    __shared__ double red[kThreads / 64];
    const int t = threadIdx.x, c = t % kRowsW, g = t / kRowsW;
    const int k = blockIdx.x * kRowsW + c;      // K % 64 == 0
    const double cx = group_total<kRowsW>(slot_sum<kThreads / kRowsW>(colA + k, nslA, K, g), part);
    __syncthreads();
    const double cw = group_total<kRowsW>(slot_sum<kThreads / kRowsW>(colW + k, nslW, K, g), part);
    if (t < kRowsW)
        grad_sigma[k] = (float)(scale * ((cw + corrW[k]) - (cx + corrA[k])) / (double)sigma[k]);
    if (blockIdx.x == 0) {
        double l = 0.0;
        for (int i = t; i < nloss; i += kThreads) l += loss_part[i];
        l = block_sum(l, red);
        __syncthreads();
        double cl = 0.0;
        for (int i = t; i < nbA; i += kThreads) cl += dclipa_part[i];
        cl = block_sum(cl, red);
        if (t == 0) {
            loss[0] = (float)(l * inv_mn);
            grad_clip_a[0] = (float)(scale * cl);
        }
    }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
inline size_t up256(size_t b) { return (b + 255) & ~(size_t)255; }

struct CalibPlan {
    int Mp, nsA, jsA, nsW, jsW, nbA, nloss, tilesMA, tilesNW;
};

CalibPlan calib_plan(int M, int N, int K) {
    CalibPlan p;
    p.Mp = (M + 63) / 64 * 64;
    const int kt = K / BB;
    p.tilesMA = (M + BB - 1) / BB;
    p.tilesNW = (N + BB - 1) / BB;
    auto splits = [](int tiles, int J, int &ns, int &js) {
        // about two work-groups per CU of 256, at least 4 stages per split
        int want = (512 + tiles - 1) / tiles;
        want = std::max(1, std::min(want, J / (4 * BJ)));
        js = ((J + want - 1) / want + BJ - 1) / BJ * BJ;
        ns = (J + js - 1) / js;
    };
    splits(p.tilesMA * kt, N, p.nsA, p.jsA);
    splits(p.tilesNW * kt, p.Mp, p.nsW, p.jsW);
    p.nbA = (M + kRowsA - 1) / kRowsA;
    p.nloss = (N / 64) * (p.Mp / 64);
    return p;
}

struct CalibWs {
    uint8_t *codesA, *codesW;
    float *sA, *aA, *sW, *aW;
    int32_t *kA, *kW;
    uint16_t *CaT, *CwT, *P1, *P2T;
    float *xprime;
    uint8_t *insA, *insW;
    int32_t *acc;
    double *loss_part, *corr, *dclipa_part;
    float *rowA, *colA, *rowW, *colW;
};

size_t calib_carve(const CalibPlan &p, int M, int N, int K, uint8_t *base, CalibWs *w) {
    size_t off = 0;
    auto take = [&](size_t bytes) {
        uint8_t *q = base ? base + off : nullptr;
        off += up256(bytes);
        return q;
    };
    const int kt = K / BB;
    CalibWs c;
    c.codesA = take((size_t)M * K / 2);
    c.codesW = take((size_t)N * K / 2);
    c.sA = reinterpret_cast<float *>(take((size_t)M * 4));
    c.aA = reinterpret_cast<float *>(take((size_t)M * 4));
    c.kA = reinterpret_cast<int32_t *>(take((size_t)M * 4));
    c.sW = reinterpret_cast<float *>(take((size_t)N * 4));
    c.aW = reinterpret_cast<float *>(take((size_t)N * 4));
    c.kW = reinterpret_cast<int32_t *>(take((size_t)N * 4));
    c.xprime = reinterpret_cast<float *>(take((size_t)M * K * 4));
    c.insA = take((size_t)M * K / 8);
    c.insW = take((size_t)N * K / 8);
    c.CaT = reinterpret_cast<uint16_t *>(take((size_t)K * p.Mp * 2));
    c.CwT = reinterpret_cast<uint16_t *>(take((size_t)K * N * 2));
    c.acc = reinterpret_cast<int32_t *>(take((size_t)M * N * 4));
    c.P1 = reinterpret_cast<uint16_t *>(take((size_t)M * N * 2));
    c.P2T = reinterpret_cast<uint16_t *>(take((size_t)N * p.Mp * 2));
    c.loss_part = reinterpret_cast<double *>(take((size_t)p.nloss * 8));
    c.corr = reinterpret_cast<double *>(take((size_t)2 * K * 8));
    c.dclipa_part = reinterpret_cast<double *>(take((size_t)p.nbA * 8));
    c.rowA = reinterpret_cast<float *>(take((size_t)kt * p.nsA * M * 4));
    c.colA = reinterpret_cast<float *>(take((size_t)p.tilesMA * p.nsA * K * 4));
    c.rowW = reinterpret_cast<float *>(take((size_t)kt * p.nsW * N * 4));
    c.colW = reinterpret_cast<float *>(take((size_t)p.tilesNW * p.nsW * K * 4));
    if (w) *w = c;
    return off;
}

template <bool BF16>
hipError_t calib_typed(int M, int N, int K, const void *x, int64_t ldx, const void *w,
                       int64_t ldw, const float *target, int64_t ldt, const float *sigma,
                       float clip_a, const float *clip_w, float *loss, float *grad_sigma,
                       float *grad_clip_a, float *grad_clip_w, void *ws, hipStream_t stream) {
    const CalibPlan p = calib_plan(M, N, K);
    CalibWs c;
    calib_carve(p, M, N, K, static_cast<uint8_t *>(ws), &c);
    hipError_t e;
    // 1. transformed quantizers
    if ((e = launch_qs_typed<BF16, true>(M, K, x, ldx, sigma, clip_a, nullptr, c.codesA, c.sA,
                                         c.aA, c.kA, stream, c.xprime, c.insA)) != hipSuccess)
        return e;
    if ((e = launch_qs_typed<BF16, false>(N, K, w, ldw, sigma, 1.0f, clip_w, c.codesW, c.sW,
                                          c.aW, c.kW, stream, nullptr, c.insW)) != hipSuccess)
        return e;
    // 2. transposed bf16 codes
    hipLaunchKernelGGL(k_codes_bf16t, dim3(p.Mp / 64, K / 128), dim3(kThreads), 0, stream,
                       c.codesA, M, K / 2, c.CaT, (int64_t)p.Mp);
    if (N >= 2048)
        hipLaunchKernelGGL(k_codes_bf16t_wide, dim3((N + kTWide - 1) / kTWide, K / 128),
                           dim3(kThreads), 0, stream, c.codesW, N, K / 2, c.CwT, (int64_t)N);
    else
        hipLaunchKernelGGL(k_codes_bf16t, dim3(N / 64, K / 128), dim3(kThreads), 0, stream,
                           c.codesW, N, K / 2, c.CwT, (int64_t)N);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // 3. forward W4A4 GEMM (its bf16 output lands in P1, rewritten below)
    if ((e = launch_w4a4_gemm(M, N, K, c.codesA, c.sA, c.codesW, c.sW, P4Q_BF16, c.P1, N, c.acc,
                              nullptr, 0, stream)) != hipSuccess)
        return e;
    // 4. residual
    hipLaunchKernelGGL(k_calib_residual, dim3(N / 64, p.Mp / 64), dim3(kThreads), 0, stream,
                       c.acc, c.sA, c.sW, target, ldt, M, N, p.Mp, c.P1, c.P2T, c.loss_part,
                       c.corr, 2 * K);
    // 5. backward contractions with fused reductions
    hipLaunchKernelGGL((k_calib_bwd<BF16, true>), dim3(K / BB, p.tilesMA, p.nsA),
                       dim3(kThreads), 0, stream, c.P1, (int64_t)N, c.CwT, (int64_t)N, M, N,
                       p.jsA, static_cast<const uint16_t *>(x), ldx, c.xprime, c.codesA, c.insA,
                       sigma, c.sA, K, c.rowA, c.colA, nullptr);
    hipLaunchKernelGGL((k_calib_bwd<BF16, false>), dim3(K / BB, p.tilesNW, p.nsW),
                       dim3(kThreads), 0, stream, c.P2T, (int64_t)p.Mp, c.CaT, (int64_t)p.Mp, N,
                       p.Mp, p.jsW, static_cast<const uint16_t *>(w), ldw, c.xprime, c.codesW,
                       c.insW, sigma, c.sW, K, c.rowW, c.colW, nullptr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // 6-7. finish
    const double scale = 2.0 / ((double)M * (double)N);
    const int nbW = (N + kRowsW - 1) / kRowsW;
    hipLaunchKernelGGL(k_calib_rows, dim3(p.nbA + nbW), dim3(kThreads), 0, stream, c.rowA,
                       (K / BB) * p.nsA, M, c.sA, c.aA, c.kA, clip_a, c.rowW, (K / BB) * p.nsW,
                       N, c.sW, c.aW, c.kW, clip_w, p.nbA, scale, c.corr, c.corr + K,
                       c.dclipa_part, grad_clip_w);
    hipLaunchKernelGGL(k_calib_cols, dim3(K / kRowsW), dim3(kThreads), 0,
                       stream, c.colA, p.tilesMA * p.nsA, c.colW, p.tilesNW * p.nsW, c.corr,
                       c.corr + K, sigma, K, scale, grad_sigma, c.loss_part, p.nloss,
                       1.0 / ((double)M * (double)N), loss, c.dclipa_part, p.nbA, grad_clip_a);
    return hipGetLastError();
}


// ===========================================================================
// Block-level calibration: one decoder block on a pruned sequence (Sec. 3.3,
// Eq. p4q_pruning_aware_calibration; Appendix B.3).  The four linear groups
// (q|k|v, o, gate|up, down) run as above (transformed quantizers, int8 MFMA
// forward, bf16 backward contractions with fused reductions); between them
// the block's full-precision operations run in fp32 on 16-bit intermediates:
//   n1 = RMSNorm(x) g1; q|k|v = L(n1); RoPE(q), RoPE(k); O = attention;
//   h = x + L(O); n2 = RMSNorm(h) g2; g|u = L(n2); a = SiLU(g) u;
//   out = h + L(a); loss = ||out - T||^2 / (M d)
// and the backward pass chains the groups' input gradients through them.
// Every intermediate is rounded once to fp16 (nearest even) as the FP16
// model holds it; rounding passes gradients straight through.
// ===========================================================================
__device__ __forceinline__ float f16v(uint16_t h) { return half_to_f32<false>(h); }
__device__ __forceinline__ uint16_t to_f16(float v) {
    return __builtin_bit_cast(uint16_t, (_Float16)v);
}

// sum over the 256 threads of a block (fp32 partials summed in double)
__device__ __forceinline__ double block_sum_f(double v, double *red) {
    const double s = block_sum(v, red);
    __syncthreads();
    return s;
}

// RMSNorm of row m: out = fp16(x r gamma), r = 1 / sqrt(mean(x^2) + eps)
__global__ __launch_bounds__(kThreads) void k_blk_rmsnorm(const uint16_t *__restrict__ x, int d,
                                                         const uint16_t *__restrict__ gamma,
                                                         float eps, uint16_t *__restrict__ out,
                                                         float *__restrict__ rinv) {
    __shared__ double red[kThreads / 64];
    const int m = blockIdx.x, t = threadIdx.x;
    const uint16_t *xr = x + (int64_t)m * d;
    double ss = 0.0;
    for (int k = t; k < d; k += kThreads) {
        const float v = f16v(xr[k]);
        ss += (double)v * v;
    }
    ss = block_sum_f(ss, red);
    const float r = (float)(1.0 / sqrt(ss / d + (double)eps));
    if (t == 0) rinv[m] = r;
    for (int k = t; k < d; k += kThreads)
        out[(int64_t)m * d + k] = to_f16(__fmul_rn(__fmul_rn(f16v(xr[k]), r), f16v(gamma[k])));
}

// dL/dx of n = x r gamma plus the residual path's gradient dres:
//   dx = dres + r gamma dn - x r^3 / d sum_j x_j gamma_j dn_j
__global__ __launch_bounds__(kThreads) void k_blk_rmsnorm_bwd(
    const uint16_t *__restrict__ x, const uint16_t *__restrict__ gamma,
    const float *__restrict__ rinv, const float *__restrict__ dn, const float *__restrict__ dres,
    int d, float *__restrict__ dx) {
    __shared__ double red[kThreads / 64];
    const int m = blockIdx.x, t = threadIdx.x;
    const int64_t o = (int64_t)m * d;
    double s = 0.0;
    for (int k = t; k < d; k += kThreads) s += (double)f16v(x[o + k]) * f16v(gamma[k]) * dn[o + k];
    s = block_sum_f(s, red);
    const double r = rinv[m];
    const float c = (float)(r * r * r * s / d);
    for (int k = t; k < d; k += kThreads)
        dx[o + k] = dres[o + k] + (float)r * f16v(gamma[k]) * dn[o + k] - f16v(x[o + k]) * c;
}

// cos / sin of position p times theta_i = base^(-2i/D) for p < M, i < D/2,
// computed in double and rounded to fp32: tab[p][i] = (cos, sin)
__global__ __launch_bounds__(kThreads) void k_blk_rope_table(int M, int D, double base,
                                                            float2 *__restrict__ tab) {
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int half = D / 2;
    if (idx >= (int64_t)M * half) return;
    const int i = (int)(idx % half), m = (int)(idx / half);
    const double ang = (double)m * pow(base, -2.0 * i / D);
    tab[idx] = make_float2((float)cos(ang), (float)sin(ang));
}

// Rotary embedding of q and k (columns [0, 2 d) of the fused q|k|v rows):
// channel i < D/2 of a head pairs with i + D/2, angle p theta_i (the table
// above).  forward: in place on the fp16 values; backward (BWD): the
// transposed rotation in place on the fp32 gradients.
template <bool BWD, typename T>
__global__ __launch_bounds__(kThreads) void k_blk_rope(T *__restrict__ z, int64_t ld, int M,
                                                      int H, int D, const float2 *__restrict__ tab) {
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int half = D / 2;
    const int64_t total = (int64_t)M * 2 * H * half;
    if (idx >= total) return;
    const int i = (int)(idx % half);
    const int hh = (int)((idx / half) % (2 * H));           // q heads, then k heads
    const int m = (int)(idx / ((int64_t)half * 2 * H));
    const float2 cs = tab[(int64_t)m * half + i];
    const float c = cs.x, s = cs.y;
    T *row = z + (int64_t)m * ld + (int64_t)hh * D;
    if constexpr (BWD) {
        const float a = row[i], b = row[i + half];
        row[i] = a * c + b * s;
        row[i + half] = b * c - a * s;
    } else {
        const float a = f16v(row[i]), b = f16v(row[i + half]);
        row[i] = to_f16(__fmul_rn(a, c) - __fmul_rn(b, s));
        row[i + half] = to_f16(__fmul_rn(b, c) + __fmul_rn(a, s));
    }
}

template <typename T> __device__ __forceinline__ float ldv(const T *p, int64_t i);
template <> __device__ __forceinline__ float ldv<float>(const float *p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ float ldv<uint16_t>(const uint16_t *p, int64_t i) {
    return f16v(p[i]);
}

// Batched strided GEMM with fp32 accumulation (the attention products of
// one block): C[b](i, j) = alpha sum_k A[b](i, k) B[b](k, j); A element
// (i, k) at A + b sAb + i sAi + k sAk, B (k, j) at B + b sBb + k sBk + j sBj,
// C (i, j) at C + b sCb + i sCi + j.  64 x 64 tiles, 32 k per stage, 256
// threads with 4 x 4 outputs each; the next stage's elements are loaded into
// registers while the current stage is multiplied.  band: 0 all k; 1 only
// k <= i (A is lower triangular: P or dS); 2 only k >= i (A is upper
// triangular: P^T or dS^T); 3 full k, tiles strictly above the diagonal
// (j > i everywhere) skipped (their entries are never read).
constexpr int GB = 64, GK = 32;
template <typename TA, typename TB, bool C16>
__global__ __launch_bounds__(kThreads) void k_blk_bgemm(
    const TA *__restrict__ A, int64_t sAb, int64_t sAi, int64_t sAk, const TB *__restrict__ B,
    int64_t sBb, int64_t sBk, int64_t sBj, void *__restrict__ Cv, int64_t sCb, int64_t sCi, int I,
    int J, int K, float alpha, int band) {
    __shared__ float As[GK][GB + 1];
    __shared__ float Bs[GK][GB + 1];
    const int t = threadIdx.x, tx = t & 15, ty = t >> 4;
    const int i0 = blockIdx.y * GB, j0 = blockIdx.x * GB, b = blockIdx.z;
    if (band == 3 && j0 > i0 + GB - 1) return;
    A += b * sAb;
    B += b * sBb;
    int kbeg = 0, kend = K;
    if (band == 1) kend = min(K, i0 + GB);
    if (band == 2) kbeg = i0;
    float acc[4][4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = 0.0f;
    const bool a_kfast = (sAk == 1), b_jfast = (sBj == 1);
    // this thread's 8 elements of each stage: A (kk, ii), B (kb, jj)
    int akk[8], aii[8], bkk[8], bjj[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int e = t + kThreads * q;
        akk[q] = a_kfast ? (e & 31) : (e >> 6);
        aii[q] = a_kfast ? (e >> 5) : (e & 63);
        bkk[q] = b_jfast ? (e >> 6) : (e & 31);
        bjj[q] = b_jfast ? (e & 63) : (e >> 5);
    }
    float ra[8], rb[8];
    auto load = [&](int k0) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int i = i0 + aii[q], k = k0 + akk[q];
            ra[q] = (i < I && k < kend) ? ldv<TA>(A, (int64_t)i * sAi + (int64_t)k * sAk) : 0.0f;
            const int j = j0 + bjj[q], kq = k0 + bkk[q];
            rb[q] = (j < J && kq < kend) ? ldv<TB>(B, (int64_t)kq * sBk + (int64_t)j * sBj) : 0.0f;
        }
    };
    if (kbeg < kend) load(kbeg);
    for (int k0 = kbeg; k0 < kend; k0 += GK) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            As[akk[q]][aii[q]] = ra[q];
            Bs[bkk[q]][bjj[q]] = rb[q];
        }
        __syncthreads();
        if (k0 + GK < kend) load(k0 + GK);          // in flight during this stage
#pragma unroll 8
        for (int kk = 0; kk < GK; ++kk) {
            float a[4], bv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) a[r] = As[kk][ty + 16 * r];
#pragma unroll
            for (int c = 0; c < 4; ++c) bv[c] = Bs[kk][tx + 16 * c];
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int c = 0; c < 4; ++c) acc[r][c] = __builtin_fmaf(a[r], bv[c], acc[r][c]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int i = i0 + ty + 16 * r;
        if (i >= I) continue;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int j = j0 + tx + 16 * c;
            if (j >= J) continue;
            const int64_t o = b * sCb + (int64_t)i * sCi + j;
            if constexpr (C16) static_cast<uint16_t *>(Cv)[o] = to_f16(alpha * acc[r][c]);
            else static_cast<float *>(Cv)[o] = alpha * acc[r][c];
        }
    }
}

// Causal softmax of every row of S [H][M][M] (already scaled) in place: P
// over j <= i, zeros beyond.  One wavefront per row.
__global__ __launch_bounds__(kThreads) void k_blk_softmax(float *__restrict__ S, int M, int rows) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (row >= rows) return;
    const int i = row % M;
    float *p = S + (int64_t)row * M;
    float mx = -INFINITY;
    for (int j = lane; j <= i; j += 64) mx = fmaxf(mx, p[j]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    double sum = 0.0;
    for (int j = lane; j <= i; j += 64) sum += (double)expf(p[j] - mx);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    const float inv = (float)(1.0 / sum);
    for (int j = lane; j < M; j += 64) p[j] = (j <= i) ? expf(p[j] - mx) * inv : 0.0f;
}

// dS = P (dP - sum_l P dP) over j <= i, zeros beyond; dP [H][M][M] in place
__global__ __launch_bounds__(kThreads) void k_blk_softmax_bwd(const float *__restrict__ P,
                                                             float *__restrict__ dP, int M,
                                                             int rows) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (row >= rows) return;
    const int i = row % M;
    const float *p = P + (int64_t)row * M;
    float *g = dP + (int64_t)row * M;
    double s = 0.0;
    for (int j = lane; j <= i; j += 64) s += (double)p[j] * g[j];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    const float sf = (float)s;
    for (int j = lane; j < M; j += 64) g[j] = (j <= i) ? p[j] * (g[j] - sf) : 0.0f;
}

// out = fp16(a + b), elementwise
__global__ __launch_bounds__(kThreads) void k_blk_add16(const uint16_t *__restrict__ a,
                                                       const uint16_t *__restrict__ b,
                                                       uint16_t *__restrict__ out, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n) out[i] = to_f16(f16v(a[i]) + f16v(b[i]));
}

// a = fp16(SiLU(g) u) from the fused gate|up rows [M][2f]
__global__ __launch_bounds__(kThreads) void k_blk_silu_mul(const uint16_t *__restrict__ gu, int M,
                                                          int f, uint16_t *__restrict__ a) {
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (idx >= (int64_t)M * f) return;
    const int64_t m = idx / f, k = idx % f;
    const float g = f16v(gu[m * 2 * f + k]), u = f16v(gu[m * 2 * f + f + k]);
    a[idx] = to_f16(__fmul_rn(g / (1.0f + expf(-g)), u));
}

// (dg, du) of a = g sig(g) u: dg = da u sig (1 + g (1 - sig)), du = da g sig
__global__ __launch_bounds__(kThreads) void k_blk_silu_mul_bwd(const float *__restrict__ da,
                                                              const uint16_t *__restrict__ gu,
                                                              int M, int f,
                                                              float *__restrict__ dgu) {
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (idx >= (int64_t)M * f) return;
    const int64_t m = idx / f, k = idx % f;
    const float g = f16v(gu[m * 2 * f + k]), u = f16v(gu[m * 2 * f + f + k]);
    const float sg = 1.0f / (1.0f + expf(-g));
    const float d = da[idx];
    dgu[m * 2 * f + k] = d * u * sg * (1.0f + g * (1.0f - sg));
    dgu[m * 2 * f + f + k] = d * g * sg;
}

// block output out = fp16(h + y), residual against the fp32 target, the
// upstream gradient 2 (out - T) / (M d) and per-block partial sums of the
// squared residual
__global__ __launch_bounds__(kThreads) void k_blk_out(const uint16_t *__restrict__ h,
                                                     const uint16_t *__restrict__ y,
                                                     const float *__restrict__ T, int64_t ldt,
                                                     int M, int d, float g_scale,
                                                     float *__restrict__ dout,
                                                     double *__restrict__ loss_part) {
    __shared__ double red[kThreads / 64];
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    double l2 = 0.0;
    if (idx < (int64_t)M * d) {
        const int64_t m = idx / d, k = idx % d;
        const float out = f16v(to_f16(f16v(h[idx]) + f16v(y[idx])));
        const float r = out - T[m * ldt + k];
        l2 = (double)r * r;
        dout[idx] = r * g_scale;
    }
    const double s = block_sum(l2, red);
    if (threadIdx.x == 0) loss_part[blockIdx.x] = s;
}

// The bf16 contraction operands of a linear group's backward pass from its
// upstream gradient G [M][N] (fp32): P1 = bf16(G sW[n]) [M][N], P2^T =
// bf16(G sA[m]) [N][Mp] (rows m >= M zero).  64 x 64 tiles, grid (N / 64,
// Mp / 64); the grid also clears the float64 scatter targets.
__global__ __launch_bounds__(kThreads) void k_blk_upstream(
    const float *__restrict__ G, int64_t ldg, const float *__restrict__ sa,
    const float *__restrict__ sw, int M, int N, int Mp, uint16_t *__restrict__ P1,
    uint16_t *__restrict__ P2T, double *__restrict__ corr, int ncorr) {
    __shared__ __attribute__((aligned(16))) uint16_t tr[64 * 72];
    const int t = threadIdx.x;
    const int n0 = blockIdx.x * 64, m0 = blockIdx.y * 64;
    const int bid = blockIdx.y * gridDim.x + blockIdx.x;
    const int nb = gridDim.x * gridDim.y;
    for (int i = bid * kThreads + t; i < ncorr; i += nb * kThreads) corr[i] = 0.0;
    const int cn = 4 * (t & 15);
    const float4 swv = *reinterpret_cast<const float4 *>(sw + n0 + cn);
    const float swa[4] = {swv.x, swv.y, swv.z, swv.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int ml = (t >> 4) + 16 * i, m = m0 + ml;
        if (m < M) {
            const float4 gv = *reinterpret_cast<const float4 *>(G + (int64_t)m * ldg + n0 + cn);
            const float ga[4] = {gv.x, gv.y, gv.z, gv.w};
            const float s = sa[m];
            uint32_t p[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                p[e] = bf16_rne(__fmul_rn(ga[e], swa[e]));
                tr[(cn + e) * 72 + ml] = (uint16_t)bf16_rne(__fmul_rn(ga[e], s));
            }
            *reinterpret_cast<uint2 *>(P1 + (int64_t)m * N + n0 + cn) =
                make_uint2(p[0] | (p[1] << 16), p[2] | (p[3] << 16));
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) tr[(cn + e) * 72 + ml] = 0;
        }
    }
    __syncthreads();
    const int nl = t >> 2, c = t & 3;
    const uint4 *sp = reinterpret_cast<const uint4 *>(tr + nl * 72 + 16 * c);
    uint4 *dp = reinterpret_cast<uint4 *>(P2T + (int64_t)(n0 + nl) * Mp + m0 + 16 * c);
    dp[0] = sp[0];
    dp[1] = sp[1];
}

// The gradient with respect to a linear group's input X (X' = X / sigma):
//   dX[m][k] = (sum_z gpart[z][m][k] + [k = kstar_m] g_s[m] clip / 7
//               sign(X'[m][k])) / sigma_k,
// g_s[m] = the row's slot sums (its share through the scale).  Grid
// (ceil(K / 1024), M): each thread handles 4 consecutive k of row m (K % 4
// == 0) and every block re-sums its row's slots.
__global__ __launch_bounds__(kThreads) void k_blk_input_grad(
    const float *__restrict__ gpart, int ns, const float *__restrict__ rowpart, int nslots,
    const float *__restrict__ xprime, const int32_t *__restrict__ kstar,
    const float *__restrict__ scales, float clip, const float *__restrict__ sigma, int M, int K,
    float *__restrict__ dX) {
    __shared__ double red[kThreads / 64];
    const int m = blockIdx.y, t = threadIdx.x;
    double gs = 0.0;
    for (int s2 = t; s2 < nslots; s2 += kThreads) gs += (double)rowpart[(int64_t)s2 * M + m];
    gs = block_sum_f(gs, red);
    const int k = 4 * (blockIdx.x * kThreads + t);
    if (k >= K) return;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int z = 0; z < ns; ++z) {
        const float4 g = *reinterpret_cast<const float4 *>(gpart + ((int64_t)z * M + m) * K + k);
        v.x += g.x; v.y += g.y; v.z += g.z; v.w += g.w;
    }
    float o[4] = {v.x, v.y, v.z, v.w};
    const int ks = kstar[m];
    if (scales[m] != 0.0f && ks >= k && ks < k + 4) {
        const float xp = xprime[(int64_t)m * K + ks];
        const double share = gs * (double)clip / 7.0 * (xp > 0.0f ? 1.0 : (xp < 0.0f ? -1.0 : 0.0));
        o[ks - k] = (float)((double)o[ks - k] + share);
    }
    const float4 sg = *reinterpret_cast<const float4 *>(sigma + k);
    *reinterpret_cast<float4 *>(dX + (int64_t)m * K + k) =
        make_float4(o[0] / sg.x, o[1] / sg.y, o[2] / sg.z, o[3] / sg.w);
}

// ---------------------------------------------------------------------------
// Block-level calibration, host side
// ---------------------------------------------------------------------------
enum { kGQkv = 0, kGO = 1, kGGu = 2, kGDown = 3 };

struct BlockGroup {
    int N, K;
    bool dx;                // the chain needs the gradient with respect to its input
    CalibPlan p;
    CalibWs c;
    float *gpart;
};

struct BlockWs {
    BlockGroup g[4];
    uint16_t *n1, *qkv, *O, *o_out, *h, *n2, *gu, *a, *y;
    float *r1, *r2, *P, *dP, *dout, *da, *dgu, *dn2, *dh, *dO, *dqkv, *dummy;
    float2 *rope;
    double *loss_part;
    int nloss;
    void *gemm_ws;          // split-K workspace of the forward GEMMs
    size_t gemm_ws_bytes;
};

void block_groups(int d, int f, BlockGroup *g) {
    const int N[4] = {3 * d, d, 2 * f, d}, K[4] = {d, d, d, f};
    for (int i = 0; i < 4; ++i) {
        g[i].N = N[i];
        g[i].K = K[i];
        g[i].dx = (i != kGQkv);
    }
}

size_t block_carve(int M, int d, int f, int H, uint8_t *base, BlockWs *w) {
    size_t off = 0;
    auto take = [&](size_t bytes) {
        uint8_t *q = base ? base + off : nullptr;
        off += up256(bytes);
        return q;
    };
    BlockWs b;
    block_groups(d, f, b.g);
    for (int i = 0; i < 4; ++i) {
        BlockGroup &g = b.g[i];
        g.p = calib_plan(M, g.N, g.K);
        const size_t cb = calib_carve(g.p, M, g.N, g.K, nullptr, nullptr);
        uint8_t *cbase = take(cb);
        calib_carve(g.p, M, g.N, g.K, cbase, &g.c);
        g.gpart = g.dx ? reinterpret_cast<float *>(take((size_t)g.p.nsA * M * g.K * 4)) : nullptr;
    }
    const size_t Md = (size_t)M * d, Mf = (size_t)M * f, HMM = (size_t)H * M * M;
    auto h16 = [&](size_t n) { return reinterpret_cast<uint16_t *>(take(n * 2)); };
    auto f32 = [&](size_t n) { return reinterpret_cast<float *>(take(n * 4)); };
    b.n1 = h16(Md); b.qkv = h16(3 * Md); b.O = h16(Md); b.o_out = h16(Md); b.h = h16(Md);
    b.n2 = h16(Md); b.gu = h16(2 * Mf); b.a = h16(Mf); b.y = h16(Md);
    b.r1 = f32(M); b.r2 = f32(M); b.P = f32(HMM); b.dP = f32(HMM); b.dout = f32(Md);
    b.da = f32(Mf); b.dgu = f32(2 * Mf); b.dn2 = f32(Md); b.dh = f32(Md); b.dO = f32(Md);
    b.dqkv = f32(3 * Md); b.dummy = f32(64);
    b.rope = reinterpret_cast<float2 *>(take((size_t)M * (d / H / 2) * 8));
    b.gemm_ws_bytes = 0;
    for (int i = 0; i < 4; ++i)
        b.gemm_ws_bytes = std::max(b.gemm_ws_bytes, gemm_workspace_bytes(M, b.g[i].N, b.g[i].K));
    b.gemm_ws = b.gemm_ws_bytes ? take(b.gemm_ws_bytes) : nullptr;
    b.nloss = (int)((Md + kThreads - 1) / kThreads);
    b.loss_part = reinterpret_cast<double *>(take((size_t)b.nloss * 8));
    if (w) *w = b;
    return off;
}

// forward of one fake-quantized group: quantizers, transposed codes, the
// W4A4 GEMM into y (fp16, row stride ldy)
hipError_t group_forward(BlockGroup &g, int M, const uint16_t *X, const void *W,
                         const float *sigma, float clip_a, const float *clip_w, uint16_t *y,
                         int64_t ldy, void *gemm_ws, size_t gemm_ws_bytes, hipStream_t stream) {
    CalibWs &c = g.c;
    const int N = g.N, K = g.K;
    hipError_t e;
    if ((e = launch_qs_typed<false, true>(M, K, X, K, sigma, clip_a, nullptr, c.codesA, c.sA, c.aA,
                                          c.kA, stream, c.xprime, c.insA)) != hipSuccess)
        return e;
    if ((e = launch_qs_typed<false, false>(N, K, W, K, sigma, 1.0f, clip_w, c.codesW, c.sW, c.aW,
                                           c.kW, stream, nullptr, c.insW)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_codes_bf16t, dim3(g.p.Mp / 64, K / 128), dim3(kThreads), 0, stream,
                       c.codesA, M, K / 2, c.CaT, (int64_t)g.p.Mp);
    if (N >= 2048)
        hipLaunchKernelGGL(k_codes_bf16t_wide, dim3((N + kTWide - 1) / kTWide, K / 128),
                           dim3(kThreads), 0, stream, c.codesW, N, K / 2, c.CwT, (int64_t)N);
    else
        hipLaunchKernelGGL(k_codes_bf16t, dim3(N / 64, K / 128), dim3(kThreads), 0, stream,
                           c.codesW, N, K / 2, c.CwT, (int64_t)N);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_w4a4_gemm(M, N, K, c.codesA, c.sA, c.codesW, c.sW, P4Q_FP16, y, ldy, nullptr,
                            gemm_ws, gemm_ws_bytes, stream);
}

// backward of one group from its upstream gradient G [M][N] (fp32, row
// stride ldg): sigma / clip gradients into the given slices and, when the
// group has one, the gradient with respect to its input into dX [M][K]
hipError_t group_backward(BlockGroup &g, int M, const float *G, int64_t ldg, const uint16_t *X,
                          const void *W, const float *sigma, float clip_a, const float *clip_w,
                          float *grad_sigma, float *grad_clip_a, float *grad_clip_w, float *dX,
                          const double *loss_part, int nloss, double inv_md, float *loss,
                          hipStream_t stream) {
    CalibWs &c = g.c;
    const CalibPlan &p = g.p;
    const int N = g.N, K = g.K;
    hipLaunchKernelGGL(k_blk_upstream, dim3(N / 64, p.Mp / 64), dim3(kThreads), 0, stream, G, ldg,
                       c.sA, c.sW, M, N, p.Mp, c.P1, c.P2T, c.corr, 2 * K);
    hipLaunchKernelGGL((k_calib_bwd<false, true>), dim3(K / BB, p.tilesMA, p.nsA),
                       dim3(kThreads), 0, stream, c.P1, (int64_t)N, c.CwT, (int64_t)N, M, N, p.jsA,
                       X, (int64_t)K, c.xprime, c.codesA, c.insA, sigma, c.sA, K, c.rowA, c.colA,
                       dX ? g.gpart : nullptr);
    hipLaunchKernelGGL((k_calib_bwd<false, false>), dim3(K / BB, p.tilesNW, p.nsW),
                       dim3(kThreads), 0, stream, c.P2T, (int64_t)p.Mp, c.CaT, (int64_t)p.Mp, N,
                       p.Mp, p.jsW, static_cast<const uint16_t *>(W), (int64_t)K, c.xprime,
                       c.codesW, c.insW, sigma, c.sW, K, c.rowW, c.colW, nullptr);
    const int nbW = (N + kRowsW - 1) / kRowsW;
    hipLaunchKernelGGL(k_calib_rows, dim3(p.nbA + nbW), dim3(kThreads), 0, stream, c.rowA,
                       (K / BB) * p.nsA, M, c.sA, c.aA, c.kA, clip_a, c.rowW, (K / BB) * p.nsW, N,
                       c.sW, c.aW, c.kW, clip_w, p.nbA, 1.0, c.corr, c.corr + K, c.dclipa_part,
                       grad_clip_w);
    hipLaunchKernelGGL(k_calib_cols, dim3(K / kRowsW), dim3(kThreads), 0, stream, c.colA,
                       p.tilesMA * p.nsA, c.colW, p.tilesNW * p.nsW, c.corr, c.corr + K, sigma, K,
                       1.0, grad_sigma, loss_part, nloss, inv_md, loss, c.dclipa_part, p.nbA,
                       grad_clip_a);
    if (dX)
        hipLaunchKernelGGL(k_blk_input_grad, dim3((K + 4 * kThreads - 1) / (4 * kThreads), M),
                           dim3(kThreads), 0, stream, g.gpart, p.nsA, c.rowA, (K / BB) * p.nsA,
                           c.xprime, c.kA, c.sA, clip_a, sigma, M, K, dX);
    return hipGetLastError();
}

// C[b] = alpha A[b] B[b] over a grid of 64 x 64 tiles (see k_blk_bgemm)
template <typename TA, typename TB, bool C16>
void bgemm(const TA *A, int64_t sAb, int64_t sAi, int64_t sAk, const TB *B, int64_t sBb,
           int64_t sBk, int64_t sBj, void *C, int64_t sCb, int64_t sCi, int I, int J, int K,
           int batch, float alpha, int band, hipStream_t stream) {
    hipLaunchKernelGGL((k_blk_bgemm<TA, TB, C16>), dim3((J + GB - 1) / GB, (I + GB - 1) / GB, batch),
                       dim3(kThreads), 0, stream, A, sAb, sAi, sAk, B, sBb, sBk, sBj, C, sCb, sCi,
                       I, J, K, alpha, band);
}

hipError_t calib_block_run(int M, int d, int f, int H, const uint16_t *x, const float *target,
                           int64_t ldt, const void *const w[4], const uint16_t *gamma1,
                           const uint16_t *gamma2, float eps, float rope_base,
                           const float *sigma, const float clip_a[4], const float *clip_w,
                           float *loss, float *grad_sigma, float *grad_clip_a,
                           float *grad_clip_w, void *ws, hipStream_t stream) {
    BlockWs b;
    block_carve(M, d, f, H, static_cast<uint8_t *>(ws), &b);
    const int D = d / H;
    const int64_t ld3 = 3 * (int64_t)d;
    const float isd = (float)(1.0 / sqrt((double)D));
    // parameter slices: sigma [qkv d | o d | gu d | down f], clip_w [3d | d | 2f | d]
    const float *sg[4] = {sigma, sigma + d, sigma + 2 * d, sigma + 3 * d};
    float *gsg[4] = {grad_sigma, grad_sigma + d, grad_sigma + 2 * d, grad_sigma + 3 * d};
    const int64_t cwo[4] = {0, 3 * (int64_t)d, 4 * (int64_t)d, 4 * (int64_t)d + 2 * (int64_t)f};
    hipError_t e;
    const int64_t Md = (int64_t)M * d, Mf = (int64_t)M * f;
    const unsigned ebl = (unsigned)((Md + kThreads - 1) / kThreads);
    const int rows = H * M;

    // ---- forward
    // the forward GEMMs' split-K arrival counters live in this call's workspace
    if ((e = gemm_workspace_clear(b.gemm_ws, b.gemm_ws_bytes, stream)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_blk_rmsnorm, dim3(M), dim3(kThreads), 0, stream, x, d, gamma1, eps, b.n1,
                       b.r1);
    if ((e = group_forward(b.g[kGQkv], M, b.n1, w[kGQkv], sg[kGQkv], clip_a[kGQkv],
                           clip_w + cwo[kGQkv], b.qkv, ld3, b.gemm_ws, b.gemm_ws_bytes, stream)) != hipSuccess)
        return e;
    const int64_t nrope = (int64_t)M * 2 * H * (D / 2);
    const int64_t ntab = (int64_t)M * (D / 2);
    hipLaunchKernelGGL(k_blk_rope_table, dim3((unsigned)((ntab + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, stream, M, D, (double)rope_base, b.rope);
    hipLaunchKernelGGL((k_blk_rope<false, uint16_t>), dim3((unsigned)((nrope + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, stream, b.qkv, ld3, M, H, D, (const float2 *)b.rope);
    // S = q k^T / sqrt(D) (causal tiles only), P = softmax, O = P v
    bgemm<uint16_t, uint16_t, false>(b.qkv, D, ld3, 1, b.qkv + d, D, 1, ld3, b.P, (int64_t)M * M, M,
                                     M, M, D, H, isd, 3, stream);
    hipLaunchKernelGGL(k_blk_softmax, dim3((rows + 3) / 4), dim3(kThreads), 0, stream, b.P, M, rows);
    bgemm<float, uint16_t, true>(b.P, (int64_t)M * M, M, 1, b.qkv + 2 * d, D, ld3, 1, b.O, D, d, M,
                                 D, M, H, 1.0f, 1, stream);
    if ((e = group_forward(b.g[kGO], M, b.O, w[kGO], sg[kGO], clip_a[kGO], clip_w + cwo[kGO],
                           b.o_out, d, b.gemm_ws, b.gemm_ws_bytes, stream)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_blk_add16, dim3(ebl), dim3(kThreads), 0, stream, x, b.o_out, b.h, Md);
    hipLaunchKernelGGL(k_blk_rmsnorm, dim3(M), dim3(kThreads), 0, stream, b.h, d, gamma2, eps, b.n2,
                       b.r2);
    if ((e = group_forward(b.g[kGGu], M, b.n2, w[kGGu], sg[kGGu], clip_a[kGGu],
                           clip_w + cwo[kGGu], b.gu, 2 * (int64_t)f, b.gemm_ws, b.gemm_ws_bytes,
                           stream)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_blk_silu_mul, dim3((unsigned)((Mf + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, stream, b.gu, M, f, b.a);
    if ((e = group_forward(b.g[kGDown], M, b.a, w[kGDown], sg[kGDown], clip_a[kGDown],
                           clip_w + cwo[kGDown], b.y, d, b.gemm_ws, b.gemm_ws_bytes, stream)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_blk_out, dim3(ebl), dim3(kThreads), 0, stream, b.h, b.y, target, ldt, M, d,
                       (float)(2.0 / ((double)M * d)), b.dout, b.loss_part);

    // ---- backward (the down group also reduces the loss)
    const double inv_md = 1.0 / ((double)M * d);
    if ((e = group_backward(b.g[kGDown], M, b.dout, d, b.a, w[kGDown], sg[kGDown], clip_a[kGDown],
                            clip_w + cwo[kGDown], gsg[kGDown], grad_clip_a + kGDown,
                            grad_clip_w + cwo[kGDown],
                            b.da, b.loss_part, b.nloss, inv_md, loss, stream)) != hipSuccess)
        return e;
    hipLaunchKernelGGL(k_blk_silu_mul_bwd, dim3((unsigned)((Mf + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, stream, b.da, b.gu, M, f, b.dgu);
    if ((e = group_backward(b.g[kGGu], M, b.dgu, 2 * (int64_t)f, b.n2, w[kGGu], sg[kGGu],
                            clip_a[kGGu], clip_w + cwo[kGGu], gsg[kGGu], grad_clip_a + kGGu,
                            grad_clip_w + cwo[kGGu], b.dn2, nullptr, 0, 0.0, b.dummy, stream)) !=
        hipSuccess)
        return e;
    hipLaunchKernelGGL(k_blk_rmsnorm_bwd, dim3(M), dim3(kThreads), 0, stream, b.h, gamma2, b.r2,
                       b.dn2, b.dout, d, b.dh);
    if ((e = group_backward(b.g[kGO], M, b.dh, d, b.O, w[kGO], sg[kGO], clip_a[kGO],
                            clip_w + cwo[kGO], gsg[kGO], grad_clip_a + kGO, grad_clip_w + cwo[kGO],
                            b.dO, nullptr, 0, 0.0, b.dummy, stream)) != hipSuccess)
        return e;
    // dP = dO v^T (causal tiles), dS = P (dP - rowsum(P dP)); dq = dS k / sqrt(D),
    // dk = dS^T q / sqrt(D), dv = P^T dO, into the fused d(q|k|v) rows
    bgemm<float, uint16_t, false>(b.dO, D, d, 1, b.qkv + 2 * d, D, 1, ld3, b.dP, (int64_t)M * M, M,
                                  M, M, D, H, 1.0f, 3, stream);
    hipLaunchKernelGGL(k_blk_softmax_bwd, dim3((rows + 3) / 4), dim3(kThreads), 0, stream, b.P,
                       b.dP, M, rows);
    bgemm<float, uint16_t, false>(b.dP, (int64_t)M * M, M, 1, b.qkv + d, D, ld3, 1, b.dqkv, D, ld3,
                                  M, D, M, H, isd, 1, stream);
    bgemm<float, uint16_t, false>(b.dP, (int64_t)M * M, 1, M, b.qkv, D, ld3, 1, b.dqkv + d, D, ld3,
                                  M, D, M, H, isd, 2, stream);
    bgemm<float, float, false>(b.P, (int64_t)M * M, 1, M, b.dO, D, d, 1, b.dqkv + 2 * d, D, ld3, M,
                               D, M, H, 1.0f, 2, stream);
    hipLaunchKernelGGL((k_blk_rope<true, float>), dim3((unsigned)((nrope + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, stream, b.dqkv, ld3, M, H, D, (const float2 *)b.rope);
    return group_backward(b.g[kGQkv], M, b.dqkv, ld3, b.n1, w[kGQkv], sg[kGQkv], clip_a[kGQkv],
                          clip_w + cwo[kGQkv], gsg[kGQkv], grad_clip_a + kGQkv,
                          grad_clip_w + cwo[kGQkv], nullptr, nullptr, 0, 0.0, b.dummy, stream);
}

}  // namespace

hipError_t launch_quant_scaled(p4q_dtype dt, int R, int K, const void *z, int64_t ldz,
                               const float *sigma, int divide, float clip, const float *clip_rows,
                               uint8_t *codes, float *scales, float *absmax, int32_t *kstar,
                               hipStream_t stream) {
    if (dt == P4Q_BF16)
        return divide ? launch_qs_typed<true, true>(R, K, z, ldz, sigma, clip, clip_rows, codes,
                                                    scales, absmax, kstar, stream)
                      : launch_qs_typed<true, false>(R, K, z, ldz, sigma, clip, clip_rows, codes,
                                                     scales, absmax, kstar, stream);
    return divide ? launch_qs_typed<false, true>(R, K, z, ldz, sigma, clip, clip_rows, codes,
                                                 scales, absmax, kstar, stream)
                  : launch_qs_typed<false, false>(R, K, z, ldz, sigma, clip, clip_rows, codes,
                                                  scales, absmax, kstar, stream);
}

size_t calib_linear_workspace_bytes(int M, int N, int K) {
    return calib_carve(calib_plan(M, N, K), M, N, K, nullptr, nullptr);
}

hipError_t launch_calib_linear(p4q_dtype dt, int M, int N, int K, const void *x, int64_t ldx,
                               const void *w, int64_t ldw, const float *target, int64_t ldt,
                               const float *sigma, float clip_a, const float *clip_w,
                               float *loss, float *grad_sigma, float *grad_clip_a,
                               float *grad_clip_w, void *ws, hipStream_t stream) {
    if (dt == P4Q_BF16)
        return calib_typed<true>(M, N, K, x, ldx, w, ldw, target, ldt, sigma, clip_a, clip_w,
                                 loss, grad_sigma, grad_clip_a, grad_clip_w, ws, stream);
    return calib_typed<false>(M, N, K, x, ldx, w, ldw, target, ldt, sigma, clip_a, clip_w, loss,
                              grad_sigma, grad_clip_a, grad_clip_w, ws, stream);
}

size_t calib_block_workspace_bytes(int M, int d, int f, int H) {
    return block_carve(M, d, f, H, nullptr, nullptr);
}

hipError_t launch_calib_block(int M, int d, int f, int H, const void *x, const float *target,
                              int64_t ldt, const void *w_qkv, const void *w_o, const void *w_gu,
                              const void *w_down, const void *gamma1, const void *gamma2,
                              float eps, float rope_base, const float *sigma, const float *clip_a,
                              const float *clip_w, float *loss, float *grad_sigma,
                              float *grad_clip_a, float *grad_clip_w, void *ws,
                              hipStream_t stream) {
    const void *const w[4] = {w_qkv, w_o, w_gu, w_down};
    return calib_block_run(M, d, f, H, static_cast<const uint16_t *>(x), target, ldt, w,
                           static_cast<const uint16_t *>(gamma1), static_cast<const uint16_t *>(gamma2),
                           eps, rope_base, sigma, clip_a, clip_w, loss, grad_sigma, grad_clip_a,
                           grad_clip_w, ws, stream);
}

}  // namespace p4q
