// Attention prefill on the pruned sequence with FP16 (or BF16) Q, K, V --
// the decoder step after the q/k/v linears (P4Q Appendix B.3: W4A4 with the
// key and value caches kept in FP16):
//     O[t, h] = sum_j softmax_j(<q_t, k_j> / sqrt(D)) v_j,  j <= t when causal.
//
// One work-group of 4 wavefronts per (128 queries, head, sample); each
// wavefront owns 32 queries and walks the key tiles of 32 keys:
//  * S^T = K Q^T on v_mfma_f32_32x32x16 (K from LDS, Q^T held in registers):
//    lane l ends up with query l%32 and 16 of the tile's keys, so the
//    softmax statistics of a query need its 16 registers and one exchange
//    with lane l^32;
//  * online softmax in fp32 (running max m, running sum, rescale of the
//    output accumulators), exponentials as exp2 with log2(e)/sqrt(D) folded;
//  * O^T += V^T P^T: P^T is the softmax of S^T converted to 16 bits, used as
//    the MFMA's B operand straight from the S^T registers.  The key order it
//    implies (register r of lane group g holds key 8(r/4) + 4g + r%4) is
//    matched by storing V^T in LDS with the tile's keys permuted the same
//    way, so every operand read is one 16-byte LDS read.
// Output layout of the 32x32 MFMA: register r of lane l holds row
// 8(r/4) + 4(l/32) + r%4, column l%32.
#include "p4q_internal.h"

namespace p4q {
namespace {

typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kD = 128;                 // head dimension
constexpr int kQW = 32;                 // queries per wavefront
constexpr int kQB = 4 * kQW;            // queries per work-group
constexpr int kKT = 32;                 // keys per tile
constexpr int kKStride = kD * 2 + 16;   // bytes per K row in LDS (padded)
constexpr int kVStride = kKT * 2 + 16;  // bytes per V^T row in LDS (padded)

// position of key k (0..31) of a tile inside a V^T row: PV step k / 16, lane
// group (k % 16 / 4) % 2, element 4 (k % 16 / 8) + k % 4
__device__ __forceinline__ int vpos(int k) {
    const int r = k & 15;
    return (k & 16) + 8 * ((r >> 2) & 1) + 4 * (r >> 3) + (r & 3);
}

template <bool BF16>
__device__ __forceinline__ v16f mfma(uint4 a, uint4 b, v16f c) {
    if constexpr (BF16)
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(v8h, a), __builtin_bit_cast(v8h, b), c, 0, 0, 0);
}

template <bool BF16>
__device__ __forceinline__ uint32_t to16(float x) {
    if constexpr (BF16) {
        const uint32_t u = __float_as_uint(x);
        return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;      // finite values: nearest-even
    } else {
        return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)x);
    }
}

template <bool BF16>
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
    return to16<BF16>(lo) | (to16<BF16>(hi) << 16);
}

template <bool BF16, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void k_attention(const uint16_t *__restrict__ q,
                                                      const uint16_t *__restrict__ k,
                                                      const uint16_t *__restrict__ v, int64_t ld,
                                                      int L, uint16_t *__restrict__ o, int64_t ldo,
                                                      float c2) {
    __shared__ __attribute__((aligned(16))) uint8_t sK[kKT * kKStride];
    __shared__ __attribute__((aligned(16))) uint8_t sV[kD * kVStride];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 5, c32 = lane & 31;
    const int nqt = (L + kQB - 1) / kQB;
    const int qt = CAUSAL ? nqt - 1 - (int)blockIdx.x : (int)blockIdx.x;   // longest rows first
    const int h = blockIdx.y, b = blockIdx.z;
    const int q0 = qt * kQB;
    const int64_t base = (int64_t)b * L * ld + (int64_t)h * kD;

    // this lane's query and its Q^T operands (8 k-steps of 16 d)
    const int tq = q0 + kQW * wave + c32;
    uint4 qf[8];
#pragma unroll
    for (int s = 0; s < 8; ++s)
        qf[s] = (tq < L) ? *reinterpret_cast<const uint4 *>(q + base + (int64_t)tq * ld + 16 * s + 8 * g)
                         : make_uint4(0, 0, 0, 0);

    v16f acc[4];
#pragma unroll
    for (int db = 0; db < 4; ++db) acc[db] = v16f{};
    float m = -__builtin_huge_valf(), lsum = 0.0f;

    const int kend = CAUSAL ? min(L, q0 + kQB) : L;
    const int ntiles = (kend + kKT - 1) / kKT;
    for (int kt = 0; kt < ntiles; ++kt) {
        const int k0 = kt * kKT;
        // stage K (row-major, padded) and V^T (keys permuted) of the tile
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int idx = tid + 256 * i, key = idx >> 4, ch = idx & 15;
            const int kk = k0 + key;
            uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
            if (kk < L) {
                kv = *reinterpret_cast<const uint4 *>(k + base + (int64_t)kk * ld + 8 * ch);
                vv = *reinterpret_cast<const uint4 *>(v + base + (int64_t)kk * ld + 8 * ch);
            }
            *reinterpret_cast<uint4 *>(sK + key * kKStride + 16 * ch) = kv;
            const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
            const int p = vpos(key);
#pragma unroll
            for (int e = 0; e < 8; ++e)
                *reinterpret_cast<uint16_t *>(sV + (8 * ch + e) * kVStride + 2 * p) =
                    (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
        }
        __syncthreads();

        // S^T = K Q^T: lane holds query c32, keys 8(r/4) + 4g + r%4
        v16f st = v16f{};
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            const uint4 ka = *reinterpret_cast<const uint4 *>(sK + c32 * kKStride + 32 * s + 16 * g);
            st = mfma<BF16>(ka, qf[s], st);
        }
        // mask and tile maximum
        float tmax = -__builtin_huge_valf();
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int kk = k0 + 8 * (r >> 2) + 4 * g + (r & 3);
            const bool ok = kk < L && (!CAUSAL || kk <= tq);
            st[r] = ok ? st[r] : -__builtin_huge_valf();
            tmax = __builtin_fmaxf(tmax, st[r]);
        }
        tmax = __builtin_fmaxf(tmax, __shfl_xor(tmax, 32));
        const float mnew = __builtin_fmaxf(m, tmax);
        // all keys so far masked (only for rows past L): keep everything at 0
        const float mref = (mnew == -__builtin_huge_valf()) ? 0.0f : mnew;
        const float alpha = __builtin_amdgcn_exp2f((m - mref) * c2);
        m = mnew;
        float psum = 0.0f;
        uint32_t pw[8];
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
            const float p0 = __builtin_amdgcn_exp2f((st[r] - mref) * c2);
            const float p1 = __builtin_amdgcn_exp2f((st[r + 1] - mref) * c2);
            psum += p0 + p1;
            pw[r >> 1] = pack2<BF16>(p0, p1);
        }
        psum += __shfl_xor(psum, 32);
        lsum = lsum * alpha + psum;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[db][r] *= alpha;
        // O^T += V^T P^T (two steps of 16 keys)
        const uint4 pb0 = make_uint4(pw[0], pw[1], pw[2], pw[3]);
        const uint4 pb1 = make_uint4(pw[4], pw[5], pw[6], pw[7]);
#pragma unroll
        for (int db = 0; db < 4; ++db) {
            const uint8_t *vrow = sV + (32 * db + c32) * kVStride;
            const uint4 va0 = *reinterpret_cast<const uint4 *>(vrow + 16 * g);
            const uint4 va1 = *reinterpret_cast<const uint4 *>(vrow + 32 + 16 * g);
            acc[db] = mfma<BF16>(va0, pb0, acc[db]);
            acc[db] = mfma<BF16>(va1, pb1, acc[db]);
        }
    }

    // O[tq][d] = acc / lsum; register r of d-block db holds d = 32 db + 8(r/4) + 4g + r%4
    if (tq < L) {
        const float inv = 1.0f / lsum;
        uint16_t *orow = o + (int64_t)b * L * ldo + (int64_t)tq * ldo + (int64_t)h * kD;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int d = 32 * db + 8 * j + 4 * g;
                const uint2 w = make_uint2(pack2<BF16>(acc[db][4 * j] * inv, acc[db][4 * j + 1] * inv),
                                           pack2<BF16>(acc[db][4 * j + 2] * inv, acc[db][4 * j + 3] * inv));
                *reinterpret_cast<uint2 *>(orow + d) = w;
            }
    }
}

}  // namespace

hipError_t launch_attention(p4q_dtype dt, int B, int L, int H, const void *q, const void *k,
                            const void *v, int64_t ld, void *o, int64_t ldo, int causal,
                            hipStream_t stream) {
    const dim3 grid((L + kQB - 1) / kQB, H, B);
    const float c2 = 1.4426950408889634f / __builtin_sqrtf((float)kD);   // log2(e) / sqrt(D)
    const uint16_t *qq = static_cast<const uint16_t *>(q), *kk = static_cast<const uint16_t *>(k),
                   *vv = static_cast<const uint16_t *>(v);
    uint16_t *oo = static_cast<uint16_t *>(o);
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, grid, dim3(256), 0, stream, qq, kk, vv, ld, L, oo, ldo, c2);
        return hipGetLastError();
    };
    if (dt == P4Q_BF16) return causal ? go(k_attention<true, true>) : go(k_attention<true, false>);
    return causal ? go(k_attention<false, true>) : go(k_attention<false, false>);
}

}  // namespace p4q
