// Fused per-row quantize + pack (P4Q Appendix A / B.3: per-token int4
// activations; per-output-channel int4 weights use the same call).
//
// One 256-thread work-group per row.  A row of K_in 16-bit values is read as
// 16-byte chunks (8 values); thread t owns chunks t, t+256, ... so every load
// and store instruction of a wavefront touches a contiguous span.  The row
// stays in registers between the absmax pass and the quantize pass (one HBM
// read, 2.5 bytes moved per element); at most 32 chunks per thread
// (K_in <= 65536) keep the register count, and so the occupancy, bounded.
#include "p4q_internal.h"
#include "q4_device.h"

namespace p4q {
namespace {

constexpr int kThreads = 256;      // one work-group (4 wavefronts) per row

template <bool BF16>
__device__ __forceinline__ uint32_t chunk_exact(uint4 v, float s) {
    uint32_t c[8];
    q4_chunk_exact<BF16>(v, s, c);
    return pack_nibbles(c);
}

template <int CH, bool BF16, bool CLIP1>
__global__ __launch_bounds__(kThreads) void k_quant_act(const uint8_t *__restrict__ x,
                                                        int64_t ldx_bytes, int nchunk, float clip,
                                                        uint8_t *__restrict__ codes,
                                                        int64_t ldc_bytes,
                                                        float *__restrict__ scales) {
    __shared__ uint32_t s_max[kThreads / 64];
    const int row = blockIdx.x;
    const int t = threadIdx.x;
    const uint4 *src = reinterpret_cast<const uint4 *>(x + (int64_t)row * ldx_bytes);
    uint32_t *dst = reinterpret_cast<uint32_t *>(codes + (int64_t)row * ldc_bytes);

    // chunk q = t + 256 c: each load and store instruction of a wavefront
    // covers a contiguous span of the row
    uint4 v[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int q = t + kThreads * c;
        v[c] = (q < nchunk) ? load_nt(src + q) : make_uint4(0, 0, 0, 0);
    }
    const uint32_t mw = wave_max_u32(lane_absmax_bits<CH, BF16>(v));
    if ((t & 63) == 0) s_max[t >> 6] = mw;
    __syncthreads();
    const uint32_t mbits = max(max(s_max[0], s_max[1]), max(s_max[2], s_max[3]));
    const float s = row_scale<CLIP1>(mag_to_f32<BF16>(mbits), clip);
    if (t == 0) scales[row] = s;

    uint32_t packed[CH];
    if (s == 0.0f) {                                        // all-zero row
#pragma unroll
        for (int c = 0; c < CH; ++c) packed[c] = 0u;
    } else {
        const bool tiny = !(s >= kTinyScale);
        const float r = tiny ? 0.0f : 1.0f / s;
        const float rhi = __fmul_rn(r, 1.0f + 0x1p-20f), rlo = __fmul_rn(r, 1.0f - 0x1p-20f);
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            uint32_t w[8];
            uint32_t dif = 0u;
            if (!tiny) {
                q4_chunk_bracket<BF16, CLIP1>(v[c], rhi, rlo, w, dif);
                packed[c] = pack_nibbles(w);
            }
            // rare: in some lane a bracket of this chunk straddles a
            // rounding boundary (or the scale is tiny): recompute this chunk
            // by exact division (wave-uniform branch)
            if (tiny || __any(dif != 0u)) {
                uint4 vc = v[c];
                asm volatile("" : "+v"(vc.x), "+v"(vc.y), "+v"(vc.z), "+v"(vc.w));
                packed[c] = chunk_exact<BF16>(vc, s);
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
hipError_t launch_ch(int M, int nchunk, const void *x, int64_t ldx_bytes, float clip,
                     uint8_t *codes, int64_t ldc_bytes, float *scales, hipStream_t stream) {
    hipLaunchKernelGGL((k_quant_act<CH, BF16, CLIP1>), dim3(M), dim3(kThreads), 0, stream,
                       static_cast<const uint8_t *>(x), ldx_bytes, nchunk, clip, codes, ldc_bytes,
                       scales);
    return hipGetLastError();
}

template <bool BF16, bool CLIP1>
hipError_t launch_typed(int M, int K_in, const void *x, int64_t ldx, float clip, uint8_t *codes,
                        float *scales, hipStream_t stream) {
    const int nchunk = K_in / 8;                    // <= 8192 (K_in <= 65536)
    const int per = (nchunk + kThreads - 1) / kThreads;
    const int64_t ldx_bytes = ldx * 2;
    const int64_t ldc_bytes = K_in / 2;
#define P4Q_QA(N) return launch_ch<N, BF16, CLIP1>(M, nchunk, x, ldx_bytes, clip, codes, ldc_bytes, scales, stream)
    if (per <= 1) P4Q_QA(1);
    if (per <= 2) P4Q_QA(2);
    if (per <= 3) P4Q_QA(3);
    if (per <= 4) P4Q_QA(4);
    if (per <= 6) P4Q_QA(6);
    if (per <= 8) P4Q_QA(8);
    if (per <= 12) P4Q_QA(12);
    if (per <= 16) P4Q_QA(16);
    if (per <= 24) P4Q_QA(24);
    P4Q_QA(32);
#undef P4Q_QA
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
