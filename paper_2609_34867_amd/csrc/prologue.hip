// Fused decoder prologue: per-token int4 quantization of RMSNorm(x) * gamma
// (P4Q Appendix B.3: per-token symmetric RTN activations; gamma is the
// per-channel slot into which calibration's diagonal scales fold).
//
// The normalized row is never formed.  Q4's codes are unchanged by a positive
// factor per row (in exact arithmetic) and its scale is multiplied by it, so
// the kernel quantizes u = x * gamma -- exact in fp32, both factors being
// 16-bit floats -- and multiplies the scale by 1/rms(x):
//   codes = Q4(u; c).codes,  scale = fl32(Q4(u; c).scale * (1 / rms(x))),
//   rms(x) = sqrt(sum_k x_k^2 / d + eps).
// The codes follow the same fp32 steps as the plain quantizer (bit-exact);
// the sum of squares is an fp32 tree sum, so the scale carries its rounding.
//
// One 256-thread work-group per row, as the plain quantize-and-pack kernel:
// thread t owns 16-byte chunks t, t+256, ..., the row stays in registers
// (as fp32 u) between the reductions and the quantize pass: one HBM read of
// x (2 bytes per element), gamma from cache, 0.5 bytes per element written.
#include "p4q_internal.h"
#include "q4_device.h"

namespace p4q {
namespace {

constexpr int kThreads = 256;

template <int CH, bool BF16, bool CLIP1>
__global__ __launch_bounds__(kThreads) void k_rmsnorm_quant(const uint8_t *__restrict__ x,
                                                            int64_t ldx_bytes,
                                                            const uint4 *__restrict__ gamma,
                                                            int nchunk, int d, float eps, float clip,
                                                            uint8_t *__restrict__ codes,
                                                            int64_t ldc_bytes,
                                                            float *__restrict__ scales) {
    __shared__ uint32_t s_max[kThreads / 64];
    __shared__ float s_ss[kThreads / 64];
    const int row = blockIdx.x;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const uint4 *src = reinterpret_cast<const uint4 *>(x + (int64_t)row * ldx_bytes);
    uint32_t *dst = reinterpret_cast<uint32_t *>(codes + (int64_t)row * ldc_bytes);

    uint4 v[CH], g[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int q = t + kThreads * c;
        v[c] = (q < nchunk) ? load_nt(src + q) : make_uint4(0, 0, 0, 0);
        g[c] = (q < nchunk) ? gamma[q] : make_uint4(0, 0, 0, 0);
    }
    float u[CH][8];
    float am = 0.0f, ss = 0.0f;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const uint32_t xw[4] = {v[c].x, v[c].y, v[c].z, v[c].w};
        const uint32_t gw[4] = {g[c].x, g[c].y, g[c].z, g[c].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float x0 = lo_f32<BF16>(xw[i]), x1 = hi_f32<BF16>(xw[i]);
            u[c][2 * i] = x0 * lo_f32<BF16>(gw[i]);          // exact
            u[c][2 * i + 1] = x1 * hi_f32<BF16>(gw[i]);
            am = __builtin_fmaxf(am, __builtin_fmaxf(__builtin_fabsf(u[c][2 * i]), __builtin_fabsf(u[c][2 * i + 1])));
            ss = __builtin_fmaf(x0, x0, ss);
            ss = __builtin_fmaf(x1, x1, ss);
        }
    }
    // block max of |u| (non-negative floats order as their bit patterns) and
    // block sum of x^2
    const uint32_t mw = wave_max_u32(__float_as_uint(am));
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
    if (lane == 0) { s_max[wave] = mw; s_ss[wave] = ss; }
    __syncthreads();
    const float a = __uint_as_float(max(max(s_max[0], s_max[1]), max(s_max[2], s_max[3])));
    const float sumsq = (s_ss[0] + s_ss[1]) + (s_ss[2] + s_ss[3]);
    const float s = row_scale<CLIP1>(a, clip);
    if (t == 0) {
        const float rinv = 1.0f / __builtin_sqrtf(sumsq / (float)d + eps);
        scales[row] = (s == 0.0f) ? 0.0f : s * rinv;
    }

    uint32_t packed[CH];
    if (s == 0.0f) {                                        // all-zero u
#pragma unroll
        for (int c = 0; c < CH; ++c) packed[c] = 0u;
    } else {
        const bool tiny = !(s >= kTinyScale);
        const float r = tiny ? 0.0f : 1.0f / s;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            uint32_t w[8];
            uint32_t near = 0;
            if (!tiny) {
#pragma unroll
                for (int k = 0; k < 8; ++k) w[k] = q4_fast<CLIP1>(u[c][k], r, near);
                packed[c] = pack_nibbles(w);
            }
            // rare (wave-uniform): a value within 2^-19 of a rounding boundary,
            // or a tiny scale -> this chunk by exact division
            if (tiny || __any((int)near)) {
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    float uk = u[c][k];
                    asm volatile("" : "+v"(uk));
                    w[k] = q4_exact(uk, s);
                }
                packed[c] = pack_nibbles(w);
            }
        }
    }
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int q = t + kThreads * c;
        if (q < nchunk) dst[q] = packed[c];
    }
}

template <int CH, bool BF16, bool CLIP1>
hipError_t launch_ch(int M, int d, const void *x, int64_t ldx, const void *gamma, float eps,
                     float clip, uint8_t *codes, float *scales, hipStream_t stream) {
    hipLaunchKernelGGL((k_rmsnorm_quant<CH, BF16, CLIP1>), dim3(M), dim3(kThreads), 0, stream,
                       static_cast<const uint8_t *>(x), ldx * 2, static_cast<const uint4 *>(gamma), d / 8,
                       d, eps, clip, codes, (int64_t)(d / 2), scales);
    return hipGetLastError();
}

template <bool BF16, bool CLIP1>
hipError_t launch_typed(int M, int d, const void *x, int64_t ldx, const void *gamma, float eps,
                        float clip, uint8_t *codes, float *scales, hipStream_t stream) {
    const int per = (d / 8 + kThreads - 1) / kThreads;      // d <= 16384: at most 8
#define P4Q_RQ(N) return launch_ch<N, BF16, CLIP1>(M, d, x, ldx, gamma, eps, clip, codes, scales, stream)
    if (per <= 1) P4Q_RQ(1);
    if (per <= 2) P4Q_RQ(2);
    if (per <= 3) P4Q_RQ(3);
    if (per <= 4) P4Q_RQ(4);
    if (per <= 6) P4Q_RQ(6);
    P4Q_RQ(8);
#undef P4Q_RQ
}

}  // namespace

hipError_t launch_rmsnorm_quant(p4q_dtype dt, int M, int d, const void *x, int64_t ldx,
                                const void *gamma, float eps, float clip, uint8_t *codes,
                                float *scales, hipStream_t stream) {
    const bool clip1 = (clip == 1.0f);
    if (dt == P4Q_BF16)
        return clip1 ? launch_typed<true, true>(M, d, x, ldx, gamma, eps, clip, codes, scales, stream)
                     : launch_typed<true, false>(M, d, x, ldx, gamma, eps, clip, codes, scales, stream);
    return clip1 ? launch_typed<false, true>(M, d, x, ldx, gamma, eps, clip, codes, scales, stream)
                 : launch_typed<false, false>(M, d, x, ldx, gamma, eps, clip, codes, scales, stream);
}

}  // namespace p4q
