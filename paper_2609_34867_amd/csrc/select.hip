// Quantization-aware visual-token selection (P4Q Sec. 3.2, Query Relevance
// with the whole budget), three kernels on one stream:
//
//  1. k_select_score: one pass over the visual features.  Each block first
//     fake-quantizes its sample's J concept rows (Q4, clip c) into packed
//     int4 codes in LDS.  Then each wavefront holds one token row in
//     registers, takes its absmax, quantizes it on-chip (the fake-quantized
//     copy is never written), and forms the exact integer statistics
//     D_ij = <cv_i, cq_j> and Nv_i = |cv_i|^2 with 8-wide int4 dot products
//     against the concept codes.  It also turns (D_ij, Nv_i) into an exact
//     integer order key (see exact_key).
//  2. k_select_topk: one workgroup per sample.  For each concept in order it
//     radix-selects the quota's largest (key, -index) composites among tokens
//     not yet kept, then writes the kept indices in ascending order.
//  3. k_select_gather: copies the ORIGINAL rows of the kept tokens, then the
//     text rows, into the pruned sequence with 16-byte vector copies.
#include "p4q_internal.h"

#include <algorithm>
#include "q4_device.h"
#include "wave_ops.h"

namespace p4q {
namespace {

// ---------------------------------------------------------------------------
// Exact order key.  Concept j ranks token i by cos = D / sqrt(Nv * Nq); for a
// fixed concept this orders like x = sgn(D) D^2 / Nv (x = 0 when Nv = 0).
// Distinct values of x differ by at least 1/Nv_max^2, and Nv <= 64 d, so with
// 2^LS >= (64 d)^2 the map x -> sgn(x) floor(|x| 2^LS) is strictly increasing
// on the values that occur: comparing keys is comparing cosines exactly.
// Both floor steps use an fp64 quotient (exact operands, result < 2^53) and
// an integer remainder check that removes its possible off-by-one.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int64_t exact_key(int32_t D, int32_t Nv, int LS) {
    if (Nv <= 0 || D == 0) return 0;
    const uint64_t n = (uint64_t)((int64_t)D * (int64_t)D);     // < 2^40
    const uint64_t q = (uint64_t)Nv;                             // <= 2^20
    uint64_t q0 = (uint64_t)((double)n / (double)q);
    int64_t r = (int64_t)n - (int64_t)(q0 * q);
    if (r < 0) { q0 -= 1; r += (int64_t)q; }
    if (r >= (int64_t)q) { q0 += 1; r -= (int64_t)q; }
    uint64_t q1 = (uint64_t)(__builtin_ldexp((double)r, LS) / (double)q);
    int64_t r2 = (int64_t)(((uint64_t)r << LS) - q1 * q);
    if (r2 < 0) { q1 -= 1; r2 += (int64_t)q; }
    if (r2 >= (int64_t)q) { q1 += 1; }
    const int64_t mag = (int64_t)((q0 << LS) + q1);
    return D > 0 ? mag : -mag;
}

// ---------------------------------------------------------------------------
// 1. fake-quant + score.  Grid (row blocks, B); 4 wavefronts per block, each
//    wavefront walks `rows_per_wave` consecutive tokens of sample blockIdx.y.
// ---------------------------------------------------------------------------
constexpr int kMaxJ = 8;

// Butterfly reduce-scatter of 8 per-lane partial sums: afterwards lane l holds
// the wavefront total of value ((l>>5)&1)*4 + ((l>>4)&1)*2 + ((l>>3)&1), i.e.
// value v sits in lanes 8v .. 8v+7.  The halves of the wavefront (32 lanes)
// and of each half (16 lanes) trade values with permlane swaps; within a row
// of 16, DPP mirrors and quad swaps finish the sums.  No LDS round trip.
__device__ __forceinline__ int reduce8(const int *v, int lane) {
    const bool b3 = lane & 8;
    int w[4], x[2];
#pragma unroll
    for (int k = 0; k < 4; ++k) {          // lanes < 32: value k, lanes >= 32: value k + 4
        const auto p = __builtin_amdgcn_permlane32_swap(v[k], v[k + 4], false, false);
        w[k] = p[0] + p[1];
    }
#pragma unroll
    for (int k = 0; k < 2; ++k) {          // 16-lane rows 0, 2: w[k]; rows 1, 3: w[k + 2]
        const auto p = __builtin_amdgcn_permlane16_swap(w[k], w[k + 2], false, false);
        x[k] = p[0] + p[1];
    }
    // lane i of a row keeps x[b3] and takes the partner's from lane 15 - i
    // (which has the other b3); the 8 lanes sharing b3 then cover the row
    int y = (b3 ? x[1] : x[0]) +
            __builtin_amdgcn_update_dpp(0, b3 ? x[0] : x[1], 0x140, 0xF, 0xF, false);  // row_mirror
    y += __builtin_amdgcn_update_dpp(0, y, 0x141, 0xF, 0xF, false);                    // row_half_mirror
    y += __builtin_amdgcn_update_dpp(0, y, 0x4E, 0xF, 0xF, false);                     // quad [2,3,0,1]
    y += __builtin_amdgcn_update_dpp(0, y, 0xB1, 0xF, 0xF, false);                     // quad [1,0,3,2]
    return y;
}

typedef int v4i_t __attribute__((ext_vector_type(4)));

// Range-checked 16-byte load: offsets at or past `bytes` read as zeros.
__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2));
}

// Q4 codes of one row held as CH 16-byte chunks per lane (lane l: chunks
// l, l + 64, ...; zeros past the row end), packed 8 per word in value order.
// absmax through the wavefront (no LDS), then the bracketed fast path with a
// per-chunk exact fallback.  Every lane of the wavefront must be active.
template <int CH, bool BF16, bool CLIP1>
__device__ __forceinline__ void q4_row_packed(const uint4 *v, float clip, uint32_t *cv) {
    const uint32_t mbits = wave_max_u32(lane_absmax_bits<CH, BF16>(v));
    const float s = row_scale<CLIP1>(mag_to_f32<BF16>(mbits), clip);
#pragma unroll
    for (int c = 0; c < CH; ++c) cv[c] = 0u;
    if (s != 0.0f) {
        const bool tiny = !(s >= kTinyScale);
        const float rc = tiny ? 0.0f : 1.0f / s;
        // bracketed fast path (q4_chunk_bracket), exact division per chunk
        // where a bracket straddles a rounding boundary
        const float rhi = __fmul_rn(rc, 1.0f + 0x1p-20f), rlo = __fmul_rn(rc, 1.0f - 0x1p-20f);
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            uint32_t w[8];
            uint32_t dif = 0u;    // nonzero: a bracket of this chunk straddles a boundary
            if (!tiny) q4_chunk_bracket<BF16, CLIP1>(v[c], rhi, rlo, w, dif);
            // wave-uniform and rare: some lane holds a value of this chunk
            // next to a rounding boundary (exact fp16 ratios such as x = a/2
            // land on ties), or the scale is tiny.  Only this chunk is
            // recomputed by exact division.
            if (tiny || __any(dif != 0u)) {
                uint4 vc = v[c];
                // opaque copy: keeps the exact path's fp16 -> fp32 conversions
                // from being hoisted into (and paid on) the fast path
                asm volatile("" : "+v"(vc.x), "+v"(vc.y), "+v"(vc.z), "+v"(vc.w));
                q4_chunk_exact<BF16>(vc, s, w);
            }
            cv[c] = pack_nibbles(w);
        }
    }
}

constexpr int kRowsPerWave = 8;   // rows per batch (sums gathered for one key per lane)

// Work-group size of the score pass: 16 wavefronts (one work-group per CU)
// while a wavefront fits in 128 registers, else 8.
template <int CH>
constexpr int score_waves() { return CH <= 8 ? 16 : 8; }

template <int CH, int JMAX, bool BF16, bool CLIP1>
__global__ __launch_bounds__(64 * score_waves<CH>()) void k_select_score(
    const uint8_t *__restrict__ vis, int N, int d, int J, float clip, int LS, int rpb,
    const uint8_t *__restrict__ concepts, int32_t *__restrict__ stats,
    int64_t *__restrict__ keys, uint32_t *__restrict__ vcodes) {
    extern __shared__ uint32_t s_cc[];       // [JMAX][64*CH] packed int4, zero-padded
    __shared__ uint32_t s_next;              // next unclaimed row of this block
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63;
    // wave-uniform (keeps the row buffer descriptor in SGPRs)
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nchunk = d / 8;
    constexpr int kChunks = 64 * CH;
    // this block's rows [row_begin, row_begin + nrb) of sample b
    const int row_begin = min(blockIdx.x * rpb, N);
    const int nrb = min(rpb, N - row_begin);

    uint32_t coff[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int q = lane + 64 * c;
        coff[c] = (q < nchunk) ? (uint32_t)q * 16u : 0x80000000u;
    }
    if (threadIdx.x == 0) s_next = 0;
    // this sample's concept codes into LDS, one concept row per wavefront, by
    // the same quantizer as the visual rows; absent concepts and chunks past
    // the row end are zeros, so the dot products below need no guards
    if (wave < JMAX) {                                       // wave-uniform
        const int j = wave;
        uint32_t cq[CH];
#pragma unroll
        for (int c = 0; c < CH; ++c) cq[c] = 0u;
        if (j < J) {
            const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
                (void *)(concepts + ((int64_t)b * J + j) * d * 2), 0, d * 2, 0x00020000);
            uint4 v[CH];
#pragma unroll
            for (int c = 0; c < CH; ++c) v[c] = buf_load16(rc, coff[c]);
            q4_row_packed<CH, BF16, CLIP1>(v, clip, cq);
        }
#pragma unroll
        for (int c = 0; c < CH; ++c) s_cc[j * kChunks + lane + 64 * c] = cq[c];
    }
    __syncthreads();

    // Rows are claimed one at a time from the block's range through an LDS
    // counter, so every wavefront works until the range is used up: the
    // sequencer favours older wavefronts, and a fixed share per wavefront
    // would leave the whole block waiting on its youngest ones.
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(vis + ((int64_t)b * N + row_begin) * d * 2), 0, nrb * d * 2, 0x00020000);
    auto load_row = [&](int i, uint4 *v) __attribute__((always_inline)) {    // row row_begin + i
#pragma unroll
        for (int c = 0; c < CH; ++c) v[c] = buf_load16(rv, coff[c] + (uint32_t)(i * d * 2));
    };
    auto claim = [&]() __attribute__((always_inline)) {
        uint32_t i = 0;
        if (lane == 0) i = atomicAdd(&s_next, 1u);
        return (int)__builtin_amdgcn_readfirstlane(i);
    };

    // one-row prefetch only for short rows; wide rows rely on occupancy
    constexpr bool kPrefetch = CH <= 4;
    uint4 nxt[kPrefetch ? CH : 1];
    int cur = claim();
    if constexpr (kPrefetch) {
        if (cur < nrb) load_row(cur, nxt);
    }
    // batch of up to 8 rows: lane 8v + r collects value v (D_v, or Nv at
    // v = J) of the batch's row r; lane r of rowid holds that row
    int myval = 0, mynv = 0, rowid = 0, n = 0;
    while (cur < nrb) {                                      // wave-uniform
        // keeps the concept-code LDS reads inside the loop (hoisting them
        // would cost JMAX * 2 * CH registers and halve the occupancy)
        asm volatile("" ::: "memory");
        const int nx = claim();                              // the row after this one
        uint4 v[CH];
        if constexpr (kPrefetch) {
#pragma unroll
            for (int c = 0; c < CH; ++c) v[c] = nxt[c];
            if (nx < nrb) load_row(nx, nxt);                 // prefetch next token
        } else {
            load_row(cur, v);
        }
        uint32_t cv[CH];                                     // packed int4 codes, 8 per chunk
        q4_row_packed<CH, BF16, CLIP1>(v, clip, cv);
        // packed int4 copy of the codes, when asked for (the Gram matrix of
        // the diversity stage is computed from it)
        if (vcodes) {
            uint32_t *vrow = vcodes + ((int64_t)b * N + row_begin + cur) * (d / 8);
#pragma unroll
            for (int c = 0; c < CH; ++c)
                if (lane + 64 * c < nchunk) vrow[lane + 64 * c] = cv[c];
        }

        int nv = 0;
        int dj[JMAX];
#pragma unroll
        for (int j = 0; j < JMAX; ++j) dj[j] = 0;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            nv = __builtin_amdgcn_sdot8((int)cv[c], (int)cv[c], nv, false);
#pragma unroll
            for (int j = 0; j < JMAX; ++j)
                dj[j] = __builtin_amdgcn_sdot8((int)cv[c], (int)s_cc[j * kChunks + lane + 64 * c],
                                               dj[j], false);
        }
        int part[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) part[j] = (j < JMAX) ? dj[j] : 0;
        if (JMAX < 8) part[JMAX < 8 ? J : 0] = nv;           // slot J holds Nv
        const int tot = reduce8(part, lane);                 // value (lane >> 3) of this row
        if ((lane & 7) == n) myval = tot;
        if (JMAX == 8) {
            int p2[8] = {nv, 0, 0, 0, 0, 0, 0, 0};
            const int nvt = reduce8(p2, lane);               // Nv in lanes 0..7
            if ((lane & 7) == n) mynv = nvt;
        }
        if (lane == n) rowid = cur;
        ++n;
        cur = nx;
        if (n == kRowsPerWave || cur >= nrb) {               // wave-uniform
            // one stats word and one key per lane
            const int r = lane & 7, vslot = lane >> 3;
            const int nv_r = (JMAX == 8) ? __shfl(mynv, r) : __shfl(myval, 8 * J + r);
            const int i = row_begin + __shfl(rowid, r);
            if (r < n) {
                int32_t *st = stats + ((int64_t)b * N + i) * (J + 1);
                if (vslot < J) {
                    st[vslot] = myval;
                    keys[((int64_t)b * J + vslot) * N + i] = exact_key(myval, nv_r, LS);
                } else if (vslot == J) {
                    st[J] = myval;
                }
                if (JMAX == 8 && vslot == 0) st[J] = nv_r;
            }
            n = 0;
        }
    }
}

// ---------------------------------------------------------------------------
// 2. top-K.  One 1024-thread workgroup per sample; thread t owns tokens
//    t*E .. t*E+E-1 (E <= 8), so the final compaction is an ordered scan.
//    Per concept: candidates = tokens not yet kept.  Each exact key k is
//    mapped to an order-preserving 67-bit code V = [s | e | m]: s = 1 for
//    k >= 0, e = bit length of |k| (6 bits), m = |k| without its leading one,
//    left-aligned to 60 bits; negative keys take the bitwise complement of
//    (e, m) with s = 0.  The composite X = V * 2^13 + (8191 - i) is unique, so
//    "the quota largest X" is exactly "the quota best tokens, lower index first
//    on equal cosine".  MSD radix select with 11-bit digits from the top of X:
//    the first digit is sign + exponent + 4 mantissa bits, which spreads the
//    typical scores (most near zero) over many buckets; the select stops as
//    soon as the boundary bucket is taken whole; when it holds at most 128
//    candidates, by ranking them against each other on the whole composite;
//    or, when every candidate left in it carries the same key (a tie), by one
//    ordered scan that keeps the lowest indices.
// ---------------------------------------------------------------------------
constexpr int kTkThreads = 1024;
constexpr int kDigit = 11;
constexpr int kBins = 1 << kDigit;
constexpr int kLoBits = 16;          // low word of X: 3 mantissa bits + 13 index bits
constexpr int kXBits = 80;           // 1 + 6 + 60 + 13

struct Composite {
    uint64_t hi;      // X >> 16
    uint32_t lo;      // X & 0xFFFF
};

// a boundary-bucket candidate listed for the final ranking (one 16-byte read)
struct __attribute__((aligned(16))) Ranked {
    int64_t key;
    uint32_t idx, pad;
};
constexpr int kRankMax = kTkThreads / 8;   // largest boundary bucket ranked directly

__device__ __forceinline__ Composite make_composite(int64_t k, int i) {
    const uint64_t u = (uint64_t)(k < 0 ? -k : k);
    uint64_t e = 0, m = 0;                       // 6-bit exponent, 60-bit mantissa
    if (u) {
        const int lz = __clzll((long long)u);
        e = (uint64_t)(64 - lz);                 // 1 .. 61
        m = ((u << lz) << 1) >> 4;               // drop the leading one, keep 60 bits
    }
    uint64_t em_hi = (e << 57) | (m >> 3);       // 63 bits: e(6) m(57 top)
    uint32_t em_lo = (uint32_t)(m & 7);          // 3 low mantissa bits
    if (k < 0) {                                 // s = 0, complement (e, m)
        em_hi = ~em_hi & ((1ull << 63) - 1);
        em_lo = ~em_lo & 7u;
    } else {
        em_hi |= 1ull << 63;                     // s = 1
    }
    return Composite{em_hi, (em_lo << 13) | (uint32_t)(8191 - i)};
}

// bits [lo, lo + w) of X (w <= 11)
__device__ __forceinline__ uint32_t comp_digit(const Composite &x, int lo, int w) {
    const uint32_t mask = (1u << w) - 1u;
    if (lo >= kLoBits) return (uint32_t)(x.hi >> (lo - kLoBits)) & mask;
    const uint64_t v = (x.hi << (kLoBits - lo)) | (uint64_t)(x.lo >> lo);
    return (uint32_t)v & mask;
}

// The top 11 bits of X (sign, exponent, 4 mantissa bits) straight from the
// key, without building the composite.
__device__ __forceinline__ uint32_t top_digit(int64_t k) {
    const uint64_t u = (uint64_t)(k < 0 ? -k : k);
    uint32_t em = 0;                             // e (6 bits) and 4 mantissa bits
    if (u) {
        const int lz = __clzll((long long)u);
        em = ((uint32_t)(64 - lz) << 4) | (uint32_t)(((u << lz) << 1) >> 60);
    }
    return (k < 0) ? (~em & 0x3FFu) : (0x400u | em);
}

// Order-preserving integer key of an fp32 value (finite inputs): larger
// values give larger keys, -0 and +0 the same key.
__device__ __forceinline__ int64_t f32_order_key(float a) {
    const uint32_t u = __float_as_uint(a);
    return (u >> 31) ? -(int64_t)(u & 0x7FFFFFFFu) : (int64_t)u;
}

// FKEYS: `keys` holds one fp32 score per token ([B][N], J == 1) instead of
// exact int64 keys ([B][J][N]).  Tokens listed in pre[b * pre_stride + 0 ..
// npre) are kept beforehand: they are never candidates and are not written.
// idx_out[b * out_stride + 0 .. K) = the K newly kept tokens, ascending.
template <int E, bool FKEYS>
__global__ __launch_bounds__(kTkThreads) void k_select_topk(const void *__restrict__ keys_,
                                                            int N, int J, int K,
                                                            const int32_t *__restrict__ pre,
                                                            int npre, int pre_stride,
                                                            int32_t *__restrict__ idx_out,
                                                            int out_stride) {
    __shared__ __attribute__((aligned(16))) uint32_t hist[kBins];
    __shared__ __attribute__((aligned(16))) uint32_t wtot[kTkThreads / 64];
    __shared__ uint32_t sh_bucket, sh_gt, sh_eq;
    __shared__ unsigned long long sh_hmin, sh_hmax;      // key bits of X above the index
    __shared__ uint32_t sh_cnt;                          // candidates listed for ranking
    __shared__ Ranked s_rk[kRankMax];
    __shared__ uint32_t s_rk_keep[kRankMax];
    __shared__ uint32_t sh_lmin, sh_lmax;

    const int b = blockIdx.x;
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    for (int q = t; q < kBins; q += kTkThreads) hist[q] = 0;
    if (t == 0) { sh_hmin = ~0ull; sh_hmax = 0; sh_lmin = ~0u; sh_lmax = 0; sh_cnt = 0; }
    __syncthreads();
    // tokens kept beforehand: bitmap in the (still unused) histogram
    uint32_t prekept = 0;
    if (npre > 0) {                                          // block-uniform
        const int32_t *pb = pre + (int64_t)b * pre_stride;
        for (int q = t; q < npre; q += kTkThreads) {
            const int i = pb[q];
            if ((unsigned)i < (unsigned)N) atomicOr(&hist[i >> 5], 1u << (i & 31));
        }
        __syncthreads();
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int i = t * E + e;
            if (i < N && ((hist[i >> 5] >> (i & 31)) & 1u)) prekept |= 1u << e;
        }
        __syncthreads();
        for (int q = t; q < (N + 31) / 32; q += kTkThreads) hist[q] = 0;
        __syncthreads();
    }
    uint32_t kept = prekept;

    // thread t owns tokens t*E .. t*E+E-1; keys of the next concept are loaded
    // while the current one is selected
    int64_t kn[E];
    auto load_keys = [&](int j) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int i = t * E + e;
            if constexpr (FKEYS) {
                const float *kf = static_cast<const float *>(keys_) + (int64_t)b * N;
                kn[e] = (i < N) ? f32_order_key(kf[i]) : 0;
            } else {
                const int64_t *kj = static_cast<const int64_t *>(keys_) + ((int64_t)b * J + j) * N;
                kn[e] = (i < N) ? kj[i] : 0;
            }
        }
    };
    // prefetch of the next concept's keys only while registers allow it
    constexpr bool kPrefetch = E <= 6;
    load_keys(0);
    for (int j = 0; j < J; ++j) {
        const uint32_t quota = (uint32_t)(K / J + (j < K % J ? 1 : 0));
        if (!kPrefetch && j > 0) load_keys(j);
        int64_t kc[E];                                       // this concept's keys
        uint32_t cont = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int i = t * E + e;
            kc[e] = kn[e];
            if (i < N && !((kept >> e) & 1u)) cont |= 1u << e;
        }
        if (kPrefetch && j + 1 < J) load_keys(j + 1);
        if (quota == 0) continue;                            // block-uniform
        // The first digit comes straight from the key; the full composites
        // are built only if the select goes past the first digit without
        // reaching the direct ranking.
        uint32_t dg1[E];
#pragma unroll
        for (int e = 0; e < E; ++e) dg1[e] = top_digit(kc[e]);
        Composite x[E];
        bool have_x = false;                                 // block-uniform
        uint32_t need = quota;
        int pos = kXBits;
        while (true) {
            const int w = min(kDigit, pos);
            const int lo = pos - w;
            const bool first = (pos == kXBits);
            auto digit = [&](int e) __attribute__((always_inline)) {
                return first ? dg1[e] : comp_digit(x[e], lo, w);
            };
#pragma unroll
            for (int e = 0; e < E; ++e)
                if ((cont >> e) & 1u) atomicAdd(&hist[digit(e)], 1u);
            __syncthreads();
            // reverse-order inclusive scan: thread t covers bins kBins-1-2t, kBins-2-2t
            const int b0 = kBins - 1 - 2 * t, b1 = kBins - 2 - 2 * t;
            const uint32_t c0 = hist[b0], c1 = hist[b1];
            hist[b0] = 0;
            hist[b1] = 0;
            const uint32_t inc = wave_inclusive_scan(c0 + c1);
            if (lane == 63) wtot[wave] = inc;
            __syncthreads();
            const uint32_t excl = inc - (c0 + c1) + waves_before(wtot, wave);
            if (excl < need && need <= excl + c0) { sh_bucket = b0; sh_gt = excl; sh_eq = c0; }
            const uint32_t e1 = excl + c0;
            if (e1 < need && need <= e1 + c1) { sh_bucket = b1; sh_gt = e1; sh_eq = c1; }
            __syncthreads();
            const uint32_t bucket = sh_bucket, gt = sh_gt, eq = sh_eq;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                if ((cont >> e) & 1u) {
                    const uint32_t dg = digit(e);
                    if (dg > bucket) { kept |= 1u << e; cont &= ~(1u << e); }
                    else if (dg < bucket) { cont &= ~(1u << e); }
                }
            }
            need -= gt;
            if (eq == need || lo == 0) { kept |= cont; break; }   // block-uniform
            if (eq <= (uint32_t)kRankMax) {                      // block-uniform
                // Few candidates left in the boundary bucket: list them (one
                // LDS atomic per wavefront) and rank each against all the
                // others by (key, lower index first), the order of the
                // composite (so the ranks are 0 .. eq - 1), 8 threads per
                // candidate; the `need` best are kept.  Two barriers instead
                // of a tie check and further digit passes.
                uint32_t slot[E];
                uint64_t bal[E];
                uint32_t wsum = 0;
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    bal[e] = __ballot((cont >> e) & 1u);
                    wsum += (uint32_t)__popcll(bal[e]);
                }
                if (wsum) {                                      // wavefront-uniform
                    uint32_t base = 0;
                    if (lane == 0) base = atomicAdd(&sh_cnt, wsum);
                    base = (uint32_t)__shfl((int)base, 0);
#pragma unroll
                    for (int e = 0; e < E; ++e) {
                        const uint32_t below = __builtin_amdgcn_mbcnt_hi(
                            (uint32_t)(bal[e] >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal[e], 0u));
                        slot[e] = base + below;
                        if ((cont >> e) & 1u) s_rk[slot[e]] = Ranked{kc[e], (uint32_t)(t * E + e), 0u};
                        base += (uint32_t)__popcll(bal[e]);
                    }
                }
                __syncthreads();
                {
                    const uint32_t ci = (uint32_t)t >> 3, sub = (uint32_t)t & 7u;
                    uint32_t rank = 0;
                    if (ci < eq) {
                        const Ranked me = s_rk[ci];
#pragma unroll 4
                        for (uint32_t c = sub; c < eq; c += 8) {
                            const Ranked o = s_rk[c];
                            rank += (o.key > me.key || (o.key == me.key && o.idx < me.idx)) ? 1u : 0u;
                        }
                    }
                    rank += (uint32_t)__shfl_xor((int)rank, 1);
                    rank += (uint32_t)__shfl_xor((int)rank, 2);
                    rank += (uint32_t)__shfl_xor((int)rank, 4);
                    if (ci < eq && sub == 0) s_rk_keep[ci] = (rank < need) ? 1u : 0u;
                }
                __syncthreads();
#pragma unroll
                for (int e = 0; e < E; ++e)
                    if (((cont >> e) & 1u) && s_rk_keep[slot[e]]) kept |= 1u << e;
                // the list is next written after further barriers
                if (t == 0) sh_cnt = 0;
                break;
            }
            if (!have_x) {
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    // opaque copy: keeps the composites inside this rarely
                    // taken branch instead of being computed for every concept
                    int64_t k = kc[e];
                    asm volatile("" : "+v"(k));
                    x[e] = make_composite(k, t * E + e);
                }
                have_x = true;
            }
            // key part of X of the candidates left: hi (67 - 3 bits) and the
            // 3 key bits of lo
            unsigned long long hmin = ~0ull, hmax = 0;
            uint32_t lmin = ~0u, lmax = 0;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                if ((cont >> e) & 1u) {
                    hmin = min(hmin, (unsigned long long)x[e].hi);
                    hmax = max(hmax, (unsigned long long)x[e].hi);
                    lmin = min(lmin, x[e].lo >> 13);
                    lmax = max(lmax, x[e].lo >> 13);
                }
            }
            // Still ambiguous.  If every remaining candidate has the same key
            // (a tie in cosine), the lower indices win: take the `need` first
            // candidates in token order with one ordered scan instead of
            // walking the remaining digits down to the index bits.
            if (cont) {
                atomicMin(&sh_hmin, hmin);
                atomicMax(&sh_hmax, hmax);
                atomicMin(&sh_lmin, lmin);
                atomicMax(&sh_lmax, lmax);
            }
            __syncthreads();
            const bool tied = (sh_hmin == sh_hmax) && (sh_lmin == sh_lmax);
            __syncthreads();
            if (t == 0) { sh_hmin = ~0ull; sh_hmax = 0; sh_lmin = ~0u; sh_lmax = 0; }
            if (tied) {                                          // block-uniform
                const uint32_t c = __builtin_popcount(cont);
                const uint32_t ic = wave_inclusive_scan(c);
                if (lane == 63) wtot[wave] = ic;
                __syncthreads();
                uint32_t rank = ic - c + waves_before(wtot, wave);
#pragma unroll
                for (int e = 0; e < E; ++e)
                    if ((cont >> e) & 1u) {
                        if (rank < need) kept |= 1u << e;
                        ++rank;
                    }
                __syncthreads();                                 // wtot reused below
                break;
            }
            pos = lo;
        }
    }

    // ordered compaction of the newly kept set
    kept &= ~prekept;
    const uint32_t cnt = __builtin_popcount(kept);
    const uint32_t inc = wave_inclusive_scan(cnt);
    __syncthreads();
    if (lane == 63) wtot[wave] = inc;
    __syncthreads();
    uint32_t opos = inc - cnt + waves_before(wtot, wave);
    int32_t *out = idx_out + (int64_t)b * out_stride;
#pragma unroll
    for (int e = 0; e < E; ++e)
        if (((kept >> e) & 1u) && opos < (uint32_t)K) out[opos++] = t * E + e;
}

// ---------------------------------------------------------------------------
// 3. gather: one wavefront per output row; all of a row's 16-byte loads are
//    issued before its stores (up to 8 KB in flight per wavefront)
// ---------------------------------------------------------------------------
constexpr int kGatherMaxCh = 16;      // chunks per lane held in registers (d <= 8192)

__global__ __launch_bounds__(256) void k_select_gather(const uint4 *__restrict__ vis,
                                                       const uint4 *__restrict__ text,
                                                       const int32_t *__restrict__ idx, int B,
                                                       int N, int K, int T, int dchunks,
                                                       uint4 *__restrict__ out) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int L = K + T;
    if (row >= (int64_t)B * L) return;
    const int b = (int)(row / L), r = (int)(row % L);
    const int src_tok = (r < K) ? idx[(int64_t)b * K + r] : 0;
    uint4 *dst = out + row * dchunks;
    if (r < K && (unsigned)src_tok >= (unsigned)N) {      // never taken for a valid selection
        for (int q = lane; q < dchunks; q += 64) dst[q] = make_uint4(0, 0, 0, 0);
        return;
    }
    const uint4 *src = (r < K) ? vis + ((int64_t)b * N + src_tok) * dchunks
                               : text + ((int64_t)b * T + (r - K)) * dchunks;
    for (int q0 = 0; q0 < dchunks; q0 += 64 * kGatherMaxCh) {
        uint4 v[kGatherMaxCh];
#pragma unroll
        for (int c = 0; c < kGatherMaxCh; ++c) {
            const int q = q0 + lane + 64 * c;
            if (q < dchunks) v[c] = load_nt(src + q);
        }
#pragma unroll
        for (int c = 0; c < kGatherMaxCh; ++c) {
            const int q = q0 + lane + 64 * c;
            if (q < dchunks) dst[q] = v[c];
        }
    }
}

template <int CH, int JMAX, bool BF16, bool CLIP1>
hipError_t launch_score(int B, int N, int d, int J, float clip, int LS, const void *vis,
                        const void *concepts, const SelectWorkspace &ws, hipStream_t stream) {
    constexpr int kWaves = score_waves<CH>();
    const size_t lds = (size_t)JMAX * 64 * CH * 4;
    // Blocks per sample: together one block per CU for the batch (the
    // blocks hold the whole CU), at least 2 rows per wavefront.
    const int cus = device_cus();
    const int per_sample = (int)std::max<int64_t>(
        1, std::min<int64_t>(((int64_t)cus + B - 1) / B, ((int64_t)N + 2 * kWaves - 1) / (2 * kWaves)));
    const int rpb = (N + per_sample - 1) / per_sample;
    const dim3 grid((N + rpb - 1) / rpb, B);
    hipLaunchKernelGGL((k_select_score<CH, JMAX, BF16, CLIP1>), grid, dim3(64 * kWaves), lds, stream,
                       static_cast<const uint8_t *>(vis), N, d, J, clip, LS, rpb,
                       static_cast<const uint8_t *>(concepts), ws.stats, ws.keys, ws.vcodes);
    return hipGetLastError();
}

template <int CH, bool BF16, bool CLIP1>
hipError_t launch_score_j(int B, int N, int d, int J, float clip, int LS, const void *vis,
                          const void *concepts, const SelectWorkspace &ws, hipStream_t stream) {
    if (J <= 4) return launch_score<CH, 4, BF16, CLIP1>(B, N, d, J, clip, LS, vis, concepts, ws, stream);
    return launch_score<CH, 8, BF16, CLIP1>(B, N, d, J, clip, LS, vis, concepts, ws, stream);
}

template <bool BF16, bool CLIP1>
hipError_t launch_score_typed(int B, int N, int d, int J, float clip, int LS, const void *vis,
                              const void *concepts, const SelectWorkspace &ws, hipStream_t stream) {
    const int per_lane = (d / 8 + 63) / 64;
    if (per_lane <= 1) return launch_score_j<1, BF16, CLIP1>(B, N, d, J, clip, LS, vis, concepts, ws, stream);
    if (per_lane <= 2) return launch_score_j<2, BF16, CLIP1>(B, N, d, J, clip, LS, vis, concepts, ws, stream);
    if (per_lane <= 4) return launch_score_j<4, BF16, CLIP1>(B, N, d, J, clip, LS, vis, concepts, ws, stream);
    if (per_lane <= 8) return launch_score_j<8, BF16, CLIP1>(B, N, d, J, clip, LS, vis, concepts, ws, stream);
    if (per_lane <= 10) return launch_score_j<10, BF16, CLIP1>(B, N, d, J, clip, LS, vis, concepts, ws, stream);
    if (per_lane <= 16) return launch_score_j<16, BF16, CLIP1>(B, N, d, J, clip, LS, vis, concepts, ws, stream);
    return launch_score<32, 4, BF16, CLIP1>(B, N, d, J, clip, LS, vis, concepts, ws, stream);
}

template <bool FKEYS>
hipError_t launch_topk(int B, int N, int J, int K, const void *keys, const int32_t *pre, int npre,
                       int pre_stride, int32_t *idx_out, int out_stride, hipStream_t stream) {
    switch ((N + kTkThreads - 1) / kTkThreads) {    // tokens per thread, N <= 8192
#define P4Q_TK(E)                                                                                  \
    case E:                                                                                       \
        hipLaunchKernelGGL((k_select_topk<E, FKEYS>), dim3(B), dim3(kTkThreads), 0, stream, keys, N, \
                           J, K, pre, npre, pre_stride, idx_out, out_stride);                     \
        break;
        P4Q_TK(1) P4Q_TK(2) P4Q_TK(3) P4Q_TK(4) P4Q_TK(5) P4Q_TK(6) P4Q_TK(7) P4Q_TK(8)
#undef P4Q_TK
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <bool BF16, bool CLIP1>
hipError_t launch_codes_and_scores(int B, int N, int d, int J, float clip, const void *vis,
                                   const void *concepts, const SelectWorkspace &ws,
                                   hipStream_t stream) {
    // 2^LS >= (64 d)^2: LS = 2 * ceil(log2(64 d))
    int lg = 0;
    while ((1ll << lg) < 64ll * d) ++lg;
    const int LS = 2 * lg;
    return launch_score_typed<BF16, CLIP1>(B, N, d, J, clip, LS, vis, concepts, ws, stream);
}

hipError_t launch_gather(int B, int N, int d, const void *vis, const void *text, int T, int K,
                         const int32_t *idx, void *tokens_out, hipStream_t stream) {
    const int64_t rows = (int64_t)B * (K + T);
    hipLaunchKernelGGL(k_select_gather, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream,
                       static_cast<const uint4 *>(vis), static_cast<const uint4 *>(text), idx,
                       B, N, K, T, d / 8, static_cast<uint4 *>(tokens_out));
    return hipGetLastError();
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

size_t select_workspace_bytes(int B, int N, int d, int J) {
    return align256((size_t)B * N * (J + 1) * 4) + align256((size_t)B * J * N * 8);
}

SelectWorkspace select_workspace_carve(void *ws, int B, int N, int d, int J) {
    uint8_t *p = static_cast<uint8_t *>(ws);
    SelectWorkspace w;
    w.stats = reinterpret_cast<int32_t *>(p);
    p += align256((size_t)B * N * (J + 1) * 4);
    w.keys = reinterpret_cast<int64_t *>(p);
    return w;
}

hipError_t launch_select(p4q_dtype dt, int B, int N, int d, const void *vis, const void *concepts,
                         int J, const void *text, int T, int K, float clip, int32_t *idx_out,
                         void *tokens_out, const SelectWorkspace &ws, hipStream_t stream) {
    const bool bf16 = (dt == P4Q_BF16);
    const bool clip1 = (clip == 1.0f);
    hipError_t e;
    if (bf16) e = clip1 ? launch_codes_and_scores<true, true>(B, N, d, J, clip, vis, concepts, ws, stream)
                        : launch_codes_and_scores<true, false>(B, N, d, J, clip, vis, concepts, ws, stream);
    else e = clip1 ? launch_codes_and_scores<false, true>(B, N, d, J, clip, vis, concepts, ws, stream)
                   : launch_codes_and_scores<false, false>(B, N, d, J, clip, vis, concepts, ws, stream);
    if (e != hipSuccess) return e;
    if ((e = launch_topk<false>(B, N, J, K, ws.keys, nullptr, 0, 0, idx_out, K, stream)) != hipSuccess)
        return e;
    return launch_gather(B, N, d, vis, text, T, K, idx_out, tokens_out, stream);
}

size_t select_full_workspace_bytes(int B, int N, int d, int J, int K) {
    return select_workspace_bytes(B, N, d, J) + align256((size_t)B * N * (d / 2)) +
           align256((size_t)B * N * N * 4) + align256((size_t)kDivInitPlanes * B * N * 8) +
           align256((size_t)kDivInitPlanes * B * N * 4) + align256((size_t)B * K * 4);
}

SelectFullWorkspace select_full_workspace_carve(void *ws, int B, int N, int d, int J, int K) {
    SelectFullWorkspace w;
    w.sel = select_workspace_carve(ws, B, N, d, J);
    uint8_t *p = static_cast<uint8_t *>(ws) + select_workspace_bytes(B, N, d, J);
    w.sel.vcodes = reinterpret_cast<uint32_t *>(p);
    p += align256((size_t)B * N * (d / 2));
    w.gram = reinterpret_cast<int32_t *>(p);
    p += align256((size_t)B * N * N * 4);
    w.mp = reinterpret_cast<int64_t *>(p);
    p += align256((size_t)kDivInitPlanes * B * N * 8);
    w.mq = reinterpret_cast<int32_t *>(p);
    p += align256((size_t)kDivInitPlanes * B * N * 4);
    w.stages = reinterpret_cast<int32_t *>(p);
    return w;
}

hipError_t launch_select_full(p4q_dtype dt, int B, int N, int d, const void *vis,
                              const void *concepts, int J, const float *cls_attn,
                              const void *text, int T, int K, int kq, int ks, float clip,
                              int32_t *idx_out, int32_t *stages_out, void *tokens_out,
                              const SelectFullWorkspace &ws, hipStream_t stream) {
    const bool bf16 = (dt == P4Q_BF16);
    const bool clip1 = (clip == 1.0f);
    const int kd = K - kq - ks;
    int32_t *stages = stages_out ? stages_out : ws.stages;
    hipError_t e;
    // codes of the fake-quantized copies (packed, for the Gram matrix) and the
    // exact Query-Relevance keys, in one pass over the features
    if (bf16) e = clip1 ? launch_codes_and_scores<true, true>(B, N, d, J, clip, vis, concepts, ws.sel, stream)
                        : launch_codes_and_scores<true, false>(B, N, d, J, clip, vis, concepts, ws.sel, stream);
    else e = clip1 ? launch_codes_and_scores<false, true>(B, N, d, J, clip, vis, concepts, ws.sel, stream)
                   : launch_codes_and_scores<false, false>(B, N, d, J, clip, vis, concepts, ws.sel, stream);
    if (e != hipSuccess) return e;
    // Query Relevance: kq tokens -> stages[b][0, kq)
    if (kq > 0 && (e = launch_topk<false>(B, N, J, kq, ws.sel.keys, nullptr, 0, 0, stages, K, stream)) != hipSuccess)
        return e;
    // Visual Saliency over the tokens left: ks tokens -> stages[b][kq, kq + ks)
    if (ks > 0 && (e = launch_topk<true>(B, N, 1, ks, cls_attn, stages, kq, K, stages + kq, K, stream)) != hipSuccess)
        return e;
    // Visual Diversity: kd greedy picks -> stages[b][kq + ks, K); idx_out = all K, ascending
    if (kd > 0 && (e = launch_code_gram(B, N, d, reinterpret_cast<const uint8_t *>(ws.sel.vcodes), ws.gram,
                                        stream)) != hipSuccess)
        return e;
    if ((e = launch_diversity(B, N, K, kq + ks, kd, ws.gram, cls_attn, ws.mp, ws.mq, stages, idx_out,
                              stream)) != hipSuccess)
        return e;
    return launch_gather(B, N, d, vis, text, T, K, idx_out, tokens_out, stream);
}

}  // namespace p4q
