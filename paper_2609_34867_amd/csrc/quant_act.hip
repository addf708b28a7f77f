// Fused per-row quantize + pack (P4Q Appendix A / B.3: per-token int4
// activations; per-output-channel int4 weights use the same call).
//
// One wavefront per row.  A row of K_in 16-bit values is read as 16-byte
// chunks (8 values); lane l owns chunks l, l+64, l+128, ... so every load and
// store instruction touches a contiguous span across the wavefront.  The row
// stays in registers between the absmax pass and the quantize pass (one HBM
// read, 2.5 bytes moved per element).  Rows longer than 32 chunks per lane use
// a two-pass variant that re-reads the row (the re-read hits L2/MALL).
#include "p4q_internal.h"
#include "q4_device.h"

namespace p4q {
namespace {

constexpr int kRowsPerBlock = 4;   // 4 wavefronts of 64 lanes

template <int CH, bool BF16, bool CLIP1>
__global__ __launch_bounds__(256) void k_quant_act(const uint8_t *__restrict__ x, int64_t ldx_bytes,
                                                   int M, int nchunk, float clip,
                                                   uint8_t *__restrict__ codes, int64_t ldc_bytes,
                                                   float *__restrict__ scales) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    if (row >= M) return;                                   // wave-uniform
    const uint4 *src = reinterpret_cast<const uint4 *>(x + (int64_t)row * ldx_bytes);
    uint32_t *dst = reinterpret_cast<uint32_t *>(codes + (int64_t)row * ldc_bytes);

    uint4 v[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int q = lane + 64 * c;
        v[c] = (q < nchunk) ? load_nt(src + q) : make_uint4(0, 0, 0, 0);
    }
    uint32_t m2 = 0;
#pragma unroll
    for (int c = 0; c < CH; ++c) m2 = absmax_chunk(m2, v[c]);
    const uint32_t mbits = wave_max_u32(max(m2 & 0xFFFFu, m2 >> 16));
    const float s = row_scale<CLIP1>(mag_to_f32<BF16>(mbits), clip);
    if (lane == 0) scales[row] = s;
    if (s == 0.0f) {                                        // all-zero row
#pragma unroll
        for (int c = 0; c < CH; ++c)
            if (lane + 64 * c < nchunk) dst[lane + 64 * c] = 0u;
        return;
    }
    uint32_t packed[CH];
    uint32_t near = 0;
    const bool tiny = !(s >= kTinyScale);
    if (!tiny) {
        const float r = 1.0f / s;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            uint32_t w[8];
            q4_chunk_fast<BF16, CLIP1>(v[c], r, w, near);
            packed[c] = nibbles8(w);
        }
    }
    if (tiny || __any((int)near)) {                          // wave-uniform, rare
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            uint32_t w[8];
            q4_chunk_exact<BF16>(v[c], s, w);
            packed[c] = nibbles8(w);
        }
    }
#pragma unroll
    for (int c = 0; c < CH; ++c)
        if (lane + 64 * c < nchunk) dst[lane + 64 * c] = packed[c];
}

// Two-pass variant for long rows: absmax sweep, then quantize sweep.
template <bool BF16, bool CLIP1>
__global__ __launch_bounds__(256) void k_quant_act_long(const uint8_t *__restrict__ x,
                                                        int64_t ldx_bytes, int M, int nchunk,
                                                        float clip, uint8_t *__restrict__ codes,
                                                        int64_t ldc_bytes,
                                                        float *__restrict__ scales) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    if (row >= M) return;
    const uint4 *src = reinterpret_cast<const uint4 *>(x + (int64_t)row * ldx_bytes);
    uint32_t *dst = reinterpret_cast<uint32_t *>(codes + (int64_t)row * ldc_bytes);
    uint32_t m2 = 0;
    for (int q = lane; q < nchunk; q += 64) m2 = absmax_chunk(m2, src[q]);
    const uint32_t mbits = wave_max_u32(max(m2 & 0xFFFFu, m2 >> 16));
    const float s = row_scale<CLIP1>(mag_to_f32<BF16>(mbits), clip);
    if (lane == 0) scales[row] = s;
    const bool tiny = !(s >= kTinyScale);
    const float r = tiny ? 0.0f : 1.0f / s;
    for (int q0 = 0; q0 < nchunk; q0 += 64) {
        const int q = q0 + lane;
        const uint4 v = (q < nchunk) ? src[q] : make_uint4(0, 0, 0, 0);
        uint32_t w[8];
        uint32_t near = 0;
        if (s == 0.0f) {
#pragma unroll
            for (int i = 0; i < 8; ++i) w[i] = 0;
        } else if (!tiny) {
            q4_chunk_fast<BF16, CLIP1>(v, r, w, near);
        }
        if (s != 0.0f && (tiny || __any((int)near))) q4_chunk_exact<BF16>(v, s, w);
        if (q < nchunk) dst[q] = nibbles8(w);
    }
}

template <int CH, bool BF16, bool CLIP1>
hipError_t launch_ch(int M, int nchunk, const void *x, int64_t ldx_bytes, float clip,
                     uint8_t *codes, int64_t ldc_bytes, float *scales, hipStream_t stream) {
    const dim3 grid((M + kRowsPerBlock - 1) / kRowsPerBlock);
    hipLaunchKernelGGL((k_quant_act<CH, BF16, CLIP1>), grid, dim3(256), 0, stream,
                       static_cast<const uint8_t *>(x), ldx_bytes, M, nchunk, clip, codes,
                       ldc_bytes, scales);
    return hipGetLastError();
}

template <bool BF16, bool CLIP1>
hipError_t launch_typed(int M, int K_in, const void *x, int64_t ldx, float clip, uint8_t *codes,
                        float *scales, hipStream_t stream) {
    const int nchunk = K_in / 8;
    const int per_lane = (nchunk + 63) / 64;
    const int64_t ldx_bytes = ldx * 2;
    const int64_t ldc_bytes = K_in / 2;
    if (per_lane <= 1) return launch_ch<1, BF16, CLIP1>(M, nchunk, x, ldx_bytes, clip, codes, ldc_bytes, scales, stream);
    if (per_lane <= 2) return launch_ch<2, BF16, CLIP1>(M, nchunk, x, ldx_bytes, clip, codes, ldc_bytes, scales, stream);
    if (per_lane <= 4) return launch_ch<4, BF16, CLIP1>(M, nchunk, x, ldx_bytes, clip, codes, ldc_bytes, scales, stream);
    if (per_lane <= 8) return launch_ch<8, BF16, CLIP1>(M, nchunk, x, ldx_bytes, clip, codes, ldc_bytes, scales, stream);
    if (per_lane <= 10) return launch_ch<10, BF16, CLIP1>(M, nchunk, x, ldx_bytes, clip, codes, ldc_bytes, scales, stream);
    if (per_lane <= 16) return launch_ch<16, BF16, CLIP1>(M, nchunk, x, ldx_bytes, clip, codes, ldc_bytes, scales, stream);
    if (per_lane <= 22) return launch_ch<22, BF16, CLIP1>(M, nchunk, x, ldx_bytes, clip, codes, ldc_bytes, scales, stream);
    if (per_lane <= 28) return launch_ch<28, BF16, CLIP1>(M, nchunk, x, ldx_bytes, clip, codes, ldc_bytes, scales, stream);
    if (per_lane <= 32) return launch_ch<32, BF16, CLIP1>(M, nchunk, x, ldx_bytes, clip, codes, ldc_bytes, scales, stream);
    const dim3 grid((M + kRowsPerBlock - 1) / kRowsPerBlock);
    hipLaunchKernelGGL((k_quant_act_long<BF16, CLIP1>), grid, dim3(256), 0, stream,
                       static_cast<const uint8_t *>(x), ldx_bytes, M, nchunk, clip, codes,
                       ldc_bytes, scales);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_quant_act(p4q_dtype dt, int M, int K_in, const void *x, int64_t ldx, float clip,
                            uint8_t *codes, float *scales, hipStream_t stream) {
    const bool clip1 = (clip == 1.0f);
    if (dt == P4Q_BF16)
        return clip1 ? launch_typed<true, true>(M, K_in, x, ldx, clip, codes, scales, stream)
                     : launch_typed<true, false>(M, K_in, x, ldx, clip, codes, scales, stream);
    return clip1 ? launch_typed<false, true>(M, K_in, x, ldx, clip, codes, scales, stream)
                 : launch_typed<false, false>(M, K_in, x, ldx, clip, codes, scales, stream);
}

}  // namespace p4q
