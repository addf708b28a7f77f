// W4A4 linear: int4 x int4 GEMM with int32 accumulation on gfx950 int8 MFMA,
// then the dequant epilogue (P4Q Appendix B.3: RTN W4A4 inference; Appendix A:
// per-token activation scales, per-output-channel weight scales).
//
//   acc[m][n] = sum_k A[m][k] W[n][k]
//   y[m][n]   = out_rne(fl32(fl32(float(acc) * sa[m]) * sw[n]))
//
// Operands stay packed (two int4 per byte) in HBM and in LDS.  After an LDS
// read, a 32-bit word p of eight nibbles becomes two words of four int8:
//   hi = p & 0xF0F0F0F0         -> 16 * (odd-k codes)
//   lo = (p << 4) & 0xF0F0F0F0  -> 16 * (even-k codes)
// Both operands are unpacked the same way, so the MFMA sees the same
// permutation of k on both sides and accumulates 256 * acc exactly
// (|256 * acc| <= 256 * 64 * K_in < 2^31 for K_in <= 131072); an arithmetic
// shift by 8 recovers acc.
#include "p4q_internal.h"

namespace p4q {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128;
constexpr int BKB = 64;            // packed bytes of k per stage (128 k values)
constexpr int kThreads = 256;      // 4 wavefronts, 2 x 2, each 64 x 64

// LDS tile: rows of 64 bytes = four 16-byte chunks; the chunk index is XORed
// with (row >> 1) & 3 so that the 16 rows one MFMA fragment reads hit
// distinct banks.
__device__ __forceinline__ int lds_off(int row, int c) {
    return row * BKB + ((c ^ ((row >> 1) & 3)) << 4);
}

__device__ __forceinline__ uint32_t nib_lo(uint32_t p) { return (p << 4) & 0xF0F0F0F0u; }
__device__ __forceinline__ uint32_t nib_hi(uint32_t p) { return p & 0xF0F0F0F0u; }

template <bool BF16OUT>
__device__ __forceinline__ void store_out(void *y, int64_t off, float v) {
    if constexpr (BF16OUT) {
        uint32_t u = __float_as_uint(v);
        u = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
        static_cast<uint16_t *>(y)[off] = (uint16_t)u;
    } else {
        // Materialize the fp32 product first: otherwise the backend folds the
        // multiply and the conversion into v_fma_mixlo_f16, rounding once
        // instead of the two roundings (fp32, then fp16) the epilogue defines.
        asm volatile("" : "+v"(v));
        static_cast<_Float16 *>(y)[off] = (_Float16)v;
    }
}

template <bool BF16OUT>
__global__ __launch_bounds__(kThreads) void k_w4a4_gemm(const uint8_t *__restrict__ A,
                                                        const float *__restrict__ sa,
                                                        const uint8_t *__restrict__ W,
                                                        const float *__restrict__ sw, int M,
                                                        int N, int Kb, void *__restrict__ y,
                                                        int64_t ldy,
                                                        int32_t *__restrict__ acc_out) {
    __shared__ __attribute__((aligned(16))) uint8_t sA[2][BM * BKB];
    __shared__ __attribute__((aligned(16))) uint8_t sB[2][BN * BKB];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int ktiles = (Kb + BKB - 1) / BKB;

    int lrow[2], lc[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int q = t + kThreads * i;
        lrow[i] = q >> 2;
        lc[i] = q & 3;
    }
    uint4 ra[2], rb[2];
    auto gload = [&](int kt) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int kbyte = kt * BKB + lc[i] * 16;
            const int ar = m0 + lrow[i], br = n0 + lrow[i];
            ra[i] = (ar < M && kbyte < Kb)
                        ? *reinterpret_cast<const uint4 *>(A + (int64_t)ar * Kb + kbyte)
                        : make_uint4(0, 0, 0, 0);
            rb[i] = (br < N && kbyte < Kb)
                        ? *reinterpret_cast<const uint4 *>(W + (int64_t)br * Kb + kbyte)
                        : make_uint4(0, 0, 0, 0);
        }
    };
    auto sstore = [&](int st) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            *reinterpret_cast<uint4 *>(&sA[st][lds_off(lrow[i], lc[i])]) = ra[i];
            *reinterpret_cast<uint4 *>(&sB[st][lds_off(lrow[i], lc[i])]) = rb[i];
        }
    };

    v4i acc[4][4];
#pragma unroll
    for (int f = 0; f < 4; ++f)
#pragma unroll
        for (int g = 0; g < 4; ++g) acc[f][g] = v4i{0, 0, 0, 0};

    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < ktiles; ++kt) {
        const int st = kt & 1;
        if (kt + 1 < ktiles) gload(kt + 1);
        v4i a0[4], a1[4], b0[4], b1[4];
#pragma unroll
        for (int f = 0; f < 4; ++f) {
            const int c = lane >> 4;
            const int ar = wm * 64 + f * 16 + (lane & 15);
            const uint4 pa = *reinterpret_cast<const uint4 *>(&sA[st][lds_off(ar, c)]);
            a0[f] = v4i{(int)nib_lo(pa.x), (int)nib_hi(pa.x), (int)nib_lo(pa.y), (int)nib_hi(pa.y)};
            a1[f] = v4i{(int)nib_lo(pa.z), (int)nib_hi(pa.z), (int)nib_lo(pa.w), (int)nib_hi(pa.w)};
            const int br = wn * 64 + f * 16 + (lane & 15);
            const uint4 pb = *reinterpret_cast<const uint4 *>(&sB[st][lds_off(br, c)]);
            b0[f] = v4i{(int)nib_lo(pb.x), (int)nib_hi(pb.x), (int)nib_lo(pb.y), (int)nib_hi(pb.y)};
            b1[f] = v4i{(int)nib_lo(pb.z), (int)nib_hi(pb.z), (int)nib_lo(pb.w), (int)nib_hi(pb.w)};
        }
#pragma unroll
        for (int f = 0; f < 4; ++f)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                acc[f][g] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a0[f], b0[g], acc[f][g], 0, 0, 0);
#pragma unroll
        for (int f = 0; f < 4; ++f)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                acc[f][g] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a1[f], b1[g], acc[f][g], 0, 0, 0);
        if (kt + 1 < ktiles) sstore(st ^ 1);
        __syncthreads();
    }

    // epilogue: lane holds rows 4*(lane>>4)+e, column lane&15 of each 16x16 tile
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const int n = n0 + wn * 64 + g * 16 + (lane & 15);
        const float swn = (n < N) ? sw[n] : 0.0f;
#pragma unroll
        for (int f = 0; f < 4; ++f) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int m = m0 + wm * 64 + f * 16 + 4 * (lane >> 4) + e;
                if (m < M && n < N) {
                    const int v = acc[f][g][e] >> 8;
                    const float t1 = __fmul_rn((float)v, sa[m]);
                    store_out<BF16OUT>(y, (int64_t)m * ldy + n, __fmul_rn(t1, swn));
                    if (acc_out) acc_out[(int64_t)m * N + n] = v;
                }
            }
        }
    }
}

}  // namespace

size_t gemm_workspace_bytes(int, int, int) { return 0; }

hipError_t launch_w4a4_gemm(int M, int N, int K, const uint8_t *a, const float *sa,
                            const uint8_t *w, const float *sw, p4q_dtype out_dt, void *y,
                            int64_t ldy, int32_t *acc_out, void *, size_t, hipStream_t stream) {
    const dim3 grid((N + BN - 1) / BN, (M + BM - 1) / BM);
    if (out_dt == P4Q_BF16)
        hipLaunchKernelGGL(k_w4a4_gemm<true>, grid, dim3(kThreads), 0, stream, a, sa, w, sw, M, N,
                           K / 2, y, ldy, acc_out);
    else
        hipLaunchKernelGGL(k_w4a4_gemm<false>, grid, dim3(kThreads), 0, stream, a, sa, w, sw, M,
                           N, K / 2, y, ldy, acc_out);
    return hipGetLastError();
}

}  // namespace p4q
