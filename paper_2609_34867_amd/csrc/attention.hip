// Attention prefill on the pruned sequence with FP16 (or BF16) Q, K, V --
// the decoder step after the q/k/v linears (P4Q Appendix B.3: W4A4 with the
// key and value caches kept in FP16):
//     O[t, h] = sum_j softmax_j(<q_t, k_j> / sqrt(D)) v_j,  j <= t when causal.
//
// One work-group of 4 wavefronts per (128 queries, head, sample); each
// wavefront owns 32 queries and walks the key tiles of 64 keys:
//  * S^T = K Q^T on v_mfma_f32_32x32x16 (K from LDS, Q^T held in registers):
//    lane l ends up with query l%32 and 16 keys of each 32-key half, so the
//    softmax statistics of a query need its registers and one exchange with
//    lane l^32;
//  * online softmax in fp32 with exp2 (log2(e)/sqrt(D) folded in); the
//    running maximum is raised only when a tile exceeds it by more than 2^8
//    in exp2 units, so the output accumulators are rescaled rarely (the
//    weights stay below 2^8, well inside the 16-bit range);
//  * O^T += V^T P^T: P^T is the softmax of S^T converted to 16 bits, used as
//    the MFMA's B operand straight from the S^T registers.  The key order it
//    implies (register r of lane group g holds key 8(r/4) + 4g + r%4 of a
//    32-key half) is matched by storing V^T in LDS with the keys permuted
//    the same way, so every operand read is one 16-byte LDS read;
//  * K and V^T are double-buffered in LDS; the next tile's global loads are
//    issued before the current tile's MFMAs (one barrier per tile); the two
//    32-key halves of a tile go through S^T, softmax and P V one after the
//    other, which keeps the register count at two wavefronts per SIMD.
// Output layout of the 32x32 MFMA: register r of lane l holds row
// 8(r/4) + 4(l/32) + r%4, column l%32.
#include "p4q_internal.h"

#include <type_traits>

namespace p4q {
namespace {

typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kD = 128;                 // head dimension
constexpr int kQW = 32;                 // queries per wavefront
constexpr int kQB = 4 * kQW;            // queries per work-group
constexpr int kKT = 64;                 // keys per tile
constexpr int kKStride = kD * 2 + 16;   // bytes per K row in LDS (padded)
constexpr int kVStride = kKT * 2 + 16;  // bytes per V^T row in LDS (padded)
constexpr int kKBytes = kKT * kKStride;
constexpr int kVBytes = kD * kVStride;
constexpr float kRescale = 8.0f;        // raise the running max past this margin (exp2 units)

// position of key k (0..63) of a tile inside a V^T row: 32-key half k / 32,
// PV step (k % 32) / 16, lane group (k % 16 / 4) % 2, element
// 4 (k % 16 / 8) + k % 4.  Four consecutive keys 4a..4a+3 stay consecutive.
__device__ __forceinline__ int vpos(int k) {
    const int r = k & 15;
    return (k & 48) + 8 * ((r >> 2) & 1) + 4 * (r >> 3) + (r & 3);
}

template <bool BF16>
__device__ __forceinline__ v16f mfma(uint4 a, uint4 b, v16f c) {
    if constexpr (BF16)
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(v8h, a), __builtin_bit_cast(v8h, b), c, 0, 0, 0);
}

// two fp32 -> two 16-bit values (nearest, ties to even), low half first
template <bool BF16>
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
    if constexpr (BF16) {
        const __bf16 a = (__bf16)lo, b = (__bf16)hi;
        return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
    } else {
        const _Float16 a = (_Float16)lo, b = (_Float16)hi;
        return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
    }
}

// the low (hi = false) or high 16-bit halves of four words, as two words
// [w0, w1 | w2, w3]
__device__ __forceinline__ uint2 gather_halves(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3, bool hi) {
    const uint32_t sel = hi ? 0x07060302u : 0x05040100u;
    return make_uint2(__builtin_amdgcn_perm(w1, w0, sel), __builtin_amdgcn_perm(w3, w2, sel));
}

template <bool BF16, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void k_attention(const uint16_t *__restrict__ q,
                                                      const uint16_t *__restrict__ k,
                                                      const uint16_t *__restrict__ v, int64_t ld,
                                                      int L, uint16_t *__restrict__ o, int64_t ldo,
                                                      float c2) {
    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * (kKBytes + kVBytes)];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 5, c32 = lane & 31;
    const int nqt = (L + kQB - 1) / kQB;
    // query tiles in the slowest grid dimension, longest (causal) first: all
    // the heaviest work-groups are dispatched before any lighter one
    const int qt = CAUSAL ? nqt - 1 - (int)blockIdx.z : (int)blockIdx.z;
    const int h = blockIdx.x, b = blockIdx.y;
    const int q0 = qt * kQB;
    const int64_t base = (int64_t)b * L * ld + (int64_t)h * kD;

    // this lane's query and its Q^T operands (8 k-steps of 16 d)
    const int qw0 = q0 + kQW * wave;                      // first query of the wavefront
    const int tq = qw0 + c32;
    uint4 qf[8];
#pragma unroll
    for (int s = 0; s < 8; ++s)
        qf[s] = (tq < L) ? *reinterpret_cast<const uint4 *>(q + base + (int64_t)tq * ld + 16 * s + 8 * g)
                         : make_uint4(0, 0, 0, 0);

    // staging of a tile: K by thread (ka, kc) = (tid / 16, tid % 16): keys
    // 4ka..4ka+3, d 8kc..8kc+7, so 16 lanes store one 256-byte row; V by
    // thread (va, vc) = (tid % 16, tid / 16): keys 4va..4va+3, d 8vc..8vc+7, so
    // the 8-byte V^T stores of 32 lanes fill two rows 32 banks apart
    const int ka = tid >> 4, kc = tid & 15, va = tid & 15, vc = tid >> 4;
    // range-checked buffers over this sample's rows of the head: rows past L
    // read as zeros, so the tile loads need no branches
    const uint32_t span = (uint32_t)((int64_t)L * ld * 2);
    const __amdgpu_buffer_rsrc_t kres = __builtin_amdgcn_make_buffer_rsrc((void *)(k + base), 0, (int)span, 0x00020000);
    const __amdgpu_buffer_rsrc_t vres = __builtin_amdgcn_make_buffer_rsrc((void *)(v + base), 0, (int)span, 0x00020000);
    const uint32_t ld2 = (uint32_t)(ld * 2);
    auto load_tile = [&](int k0, uint4 *kr, uint4 *vr) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t ko = (uint32_t)(k0 + 4 * ka + j) * ld2 + 16u * kc;
            const uint32_t vo = (uint32_t)(k0 + 4 * va + j) * ld2 + 16u * vc;
            kr[j] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(kres, ko, 0, 0));
            vr[j] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(vres, vo, 0, 0));
        }
    };
    const int vp0 = 2 * vpos(4 * va);
    auto store_tile = [&](int buf, const uint4 *kr, const uint4 *vr) {
        uint8_t *sK = smem + buf * (kKBytes + kVBytes);
        uint8_t *sV = sK + kKBytes;
#pragma unroll
        for (int j = 0; j < 4; ++j) *reinterpret_cast<uint4 *>(sK + (4 * ka + j) * kKStride + 16 * kc) = kr[j];
        // V^T row d = 8 vc + i takes word i/2, half i%2 of the four keys
        const uint32_t w[4][4] = {{vr[0].x, vr[0].y, vr[0].z, vr[0].w}, {vr[1].x, vr[1].y, vr[1].z, vr[1].w},
                                  {vr[2].x, vr[2].y, vr[2].z, vr[2].w}, {vr[3].x, vr[3].y, vr[3].z, vr[3].w}};
#pragma unroll
        for (int i = 0; i < 8; ++i)
            *reinterpret_cast<uint2 *>(sV + (8 * vc + i) * kVStride + vp0) =
                gather_halves(w[0][i >> 1], w[1][i >> 1], w[2][i >> 1], w[3][i >> 1], i & 1);
    };

    v16f acc[4];
#pragma unroll
    for (int db = 0; db < 4; ++db) acc[db] = v16f{};
    float m = -__builtin_huge_valf(), lsum = 0.0f;

    const int kend = CAUSAL ? min(L, q0 + kQB) : L;
    const int ntiles = (kend + kKT - 1) / kKT;
    // lanes l and l ^ 32 hold the two halves of a query's keys: their
    // combination through a permlane swap (no LDS round trip)
    auto xmax32 = [](float x) __attribute__((always_inline)) {
        const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        return __builtin_fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
    };
    auto xsum32 = [](float x) __attribute__((always_inline)) {
        const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        return __uint_as_float(p[0]) + __uint_as_float(p[1]);
    };
    // One tile of 64 keys from LDS buffer kt & 1, both 32-key halves at once:
    // their S^T products are two independent MFMA chains, and one softmax
    // update (one max, one rescale decision, one sum) covers the 64 keys.
    // TWO = false: only the first half has keys at or before this
    // wavefront's last query (causal diagonal); the second is skipped (its
    // weights would all be 0, leaving m, lsum and O unchanged).
    auto tile_keys = [&](int kt, auto two_c) __attribute__((always_inline)) {
        constexpr bool TWO = decltype(two_c)::value;
        constexpr int NH = TWO ? 2 : 1;
        const uint8_t *sK = smem + (kt & 1) * (kKBytes + kVBytes);
        const uint8_t *sV = sK + kKBytes;
        const int k0 = kt * kKT;
        // S^T = K Q^T: lane holds query c32, keys k0 + 32 hf + 8(r/4) + 4g + r%4
        v16f st[NH];
#pragma unroll
        for (int hf = 0; hf < NH; ++hf) st[hf] = v16f{};
#pragma unroll
        for (int s = 0; s < 8; ++s)
#pragma unroll
            for (int hf = 0; hf < NH; ++hf) {
                const uint4 kf = *reinterpret_cast<const uint4 *>(sK + (32 * hf + c32) * kKStride + 32 * s + 16 * g);
                st[hf] = mfma<BF16>(kf, qf[s], st[hf]);
            }
        // mask (only where the tile reaches the diagonal or the end)
        float tmax = -__builtin_huge_valf();
#pragma unroll
        for (int hf = 0; hf < NH; ++hf) {
            const int kh = k0 + 32 * hf;
            const bool need_mask = (kh + 32 > L) || (CAUSAL && kh + 31 > qw0);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                if (need_mask) {
                    const int kk = kh + 8 * (r >> 2) + 4 * g + (r & 3);
                    const bool ok = kk < L && (!CAUSAL || kk <= tq);
                    st[hf][r] = ok ? st[hf][r] : -__builtin_huge_valf();
                }
                tmax = __builtin_fmaxf(tmax, st[hf][r]);
            }
        }
        tmax = xmax32(tmax);
        // raise the running max only past the margin (wave-uniform rescale)
        const bool raise = (tmax - m) * c2 > kRescale || m == -__builtin_huge_valf();
        if (__any((int)raise)) {
            const float mnew = raise ? tmax : m;
            const float mref = (mnew == -__builtin_huge_valf()) ? 0.0f : mnew;
            const float alpha = (m == -__builtin_huge_valf()) ? 0.0f : __builtin_amdgcn_exp2f((m - mref) * c2);
            m = mnew;
            lsum *= alpha;
#pragma unroll
            for (int db = 0; db < 4; ++db)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[db][r] *= alpha;
        }
        const float mc = (m == -__builtin_huge_valf()) ? 0.0f : m * c2;
        float psum = 0.0f;
        uint4 pb[NH][2];
#pragma unroll
        for (int hf = 0; hf < NH; ++hf) {
            uint32_t pw[8];
#pragma unroll
            for (int r = 0; r < 16; r += 2) {
                const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(st[hf][r], c2, -mc));
                const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(st[hf][r + 1], c2, -mc));
                psum += p0 + p1;
                pw[r >> 1] = pack2<BF16>(p0, p1);
            }
            pb[hf][0] = make_uint4(pw[0], pw[1], pw[2], pw[3]);
            pb[hf][1] = make_uint4(pw[4], pw[5], pw[6], pw[7]);
        }
        lsum += xsum32(psum);
        // O^T += V^T P^T (two steps of 16 keys per half)
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
            for (int hf = 0; hf < NH; ++hf) {
                const uint8_t *vrow = sV + (32 * db + c32) * kVStride + 64 * hf + 16 * g;
                acc[db] = mfma<BF16>(*reinterpret_cast<const uint4 *>(vrow), pb[hf][0], acc[db]);
                acc[db] = mfma<BF16>(*reinterpret_cast<const uint4 *>(vrow + 32), pb[hf][1], acc[db]);
            }
    };
    auto tile = [&](int kt) __attribute__((always_inline)) {
        const int k0 = kt * kKT;
        // halves past this wavefront's last query hold only masked keys
        if (!CAUSAL || k0 + 32 <= qw0 + kQW - 1) tile_keys(kt, std::true_type{});
        else if (k0 <= qw0 + kQW - 1) tile_keys(kt, std::false_type{});
    };
    // the next tile's global loads are in flight while this tile computes
    uint4 kr[4], vr[4];
    load_tile(0, kr, vr);
    store_tile(0, kr, vr);
    __syncthreads();
    for (int kt = 0; kt < ntiles; ++kt) {                  // block-uniform
        if (kt + 1 < ntiles) load_tile((kt + 1) * kKT, kr, vr);
        tile(kt);
        if (kt + 1 < ntiles) store_tile((kt + 1) & 1, kr, vr);
        __syncthreads();
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
    const dim3 grid(H, B, (L + kQB - 1) / kQB);
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
