// Quantization-aware visual-token selection (P4Q Sec. 3.2, Query Relevance
// with the whole budget), four kernels on one stream:
//
//  1. k_concept_codes: fake-quantize the J concept rows of each sample to
//     int8 codes (Q4, clip c).
//  2. k_select_score: one pass over the visual features.  Each wavefront
//     holds one token row in registers, takes its absmax, quantizes it
//     on-chip (the fake-quantized copy is never written), and forms the exact
//     integer statistics D_ij = <cv_i, cq_j> and Nv_i = |cv_i|^2 with packed
//     int8 dot products against concept codes staged in LDS.  It also turns
//     (D_ij, Nv_i) into an exact integer order key (see exact_key).
//  3. k_select_topk: one workgroup per sample.  For each concept in order it
//     radix-selects the quota's largest (key, -index) composites among tokens
//     not yet kept, then writes the kept indices in ascending order.
//  4. k_select_gather: copies the ORIGINAL rows of the kept tokens, then the
//     text rows, into the pruned sequence with 16-byte vector copies.
#include "p4q_internal.h"
#include "q4_device.h"

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
// 1. concept codes: one wavefront per concept row, int8 codes out
// ---------------------------------------------------------------------------
template <bool BF16, bool CLIP1>
__global__ __launch_bounds__(256) void k_concept_codes(const uint8_t *__restrict__ con, int rows,
                                                       int d, float clip,
                                                       int8_t *__restrict__ ccodes) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    const int nchunk = d / 8;
    const uint4 *src = reinterpret_cast<const uint4 *>(con + (int64_t)row * d * 2);
    uint2 *dst = reinterpret_cast<uint2 *>(ccodes + (int64_t)row * d);
    uint32_t m2 = 0;
    for (int q = lane; q < nchunk; q += 64) m2 = absmax_chunk(m2, src[q]);
    const uint32_t mbits = wave_max_u32(max(m2 & 0xFFFFu, m2 >> 16));
    const float s = row_scale<CLIP1>(mag_to_f32<BF16>(mbits), clip);
    const bool tiny = !(s >= kTinyScale);
    const float r = tiny ? 0.0f : 1.0f / s;
    for (int q0 = 0; q0 < nchunk; q0 += 64) {
        const int q = q0 + lane;
        const uint4 v = (q < nchunk) ? src[q] : make_uint4(0, 0, 0, 0);
        uint32_t w[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        uint32_t near = 0;
        if (s != 0.0f && !tiny) q4_chunk_fast<BF16, CLIP1>(v, r, w, near);
        if (s != 0.0f && (tiny || __any((int)near))) q4_chunk_exact<BF16>(v, s, w);
        if (q < nchunk) dst[q] = make_uint2(bytes4(w[0], w[1], w[2], w[3]),
                                            bytes4(w[4], w[5], w[6], w[7]));
    }
}

// ---------------------------------------------------------------------------
// 2. fake-quant + score.  Grid (row blocks, B); 4 wavefronts per block, each
//    wavefront walks `rows_per_wave` consecutive tokens of sample blockIdx.y.
// ---------------------------------------------------------------------------
constexpr int kMaxJ = 8;

// Butterfly reduce-scatter of 8 per-lane partial sums: afterwards lane l holds
// the wavefront total of value ((l>>5)&1)*4 + ((l>>4)&1)*2 + ((l>>3)&1), i.e.
// value v sits in lanes 8v .. 8v+7.  10 shuffles instead of 48.
__device__ __forceinline__ int reduce8(const int *v, int lane) {
    const bool b5 = lane & 32, b4 = lane & 16, b3 = lane & 8;
    int w[4], x[2];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int send = b5 ? v[k] : v[k + 4];
        const int keep = b5 ? v[k + 4] : v[k];
        w[k] = keep + __shfl_xor(send, 32);
    }
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int send = b4 ? w[k] : w[k + 2];
        const int keep = b4 ? w[k + 2] : w[k];
        x[k] = keep + __shfl_xor(send, 16);
    }
    int y = (b3 ? x[1] : x[0]) + __shfl_xor(b3 ? x[0] : x[1], 8);
    y += __shfl_xor(y, 4);
    y += __shfl_xor(y, 2);
    y += __shfl_xor(y, 1);
    return y;
}

template <int CH, bool BF16, bool CLIP1>
__global__ __launch_bounds__(256) void k_select_score(const uint8_t *__restrict__ vis, int N, int d,
                                                      int J, float clip, int rows_per_wave,
                                                      int LS,
                                                      const int8_t *__restrict__ ccodes,
                                                      int32_t *__restrict__ stats,
                                                      int64_t *__restrict__ keys) {
    extern __shared__ uint2 s_cc[];          // [J][d/8] uint2 (8 int8 codes each)
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int nchunk = d / 8;

    // stage this sample's concept codes in LDS
    {
        const uint4 *g = reinterpret_cast<const uint4 *>(ccodes + (int64_t)b * J * d);
        uint4 *l = reinterpret_cast<uint4 *>(s_cc);
        const int n16 = J * d / 16;
        for (int q = threadIdx.x; q < n16; q += 256) l[q] = g[q];
    }
    __syncthreads();

    const int row0 = (blockIdx.x * 4 + wave) * rows_per_wave;
    const int row_end = min(row0 + rows_per_wave, N);
    const uint8_t *vb = vis + (int64_t)b * N * d * 2;

    uint4 nxt[CH];
    auto load_row = [&](int i, uint4 *v) {
        const uint4 *src = reinterpret_cast<const uint4 *>(vb + (int64_t)i * d * 2);
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int q = lane + 64 * c;
            v[c] = (q < nchunk) ? load_nt(src + q) : make_uint4(0, 0, 0, 0);
        }
    };
    if (row0 < row_end) load_row(row0, nxt);

    for (int i = row0; i < row_end; ++i) {
        uint4 v[CH];
#pragma unroll
        for (int c = 0; c < CH; ++c) v[c] = nxt[c];
        if (i + 1 < row_end) load_row(i + 1, nxt);          // prefetch next token

        uint32_t m2 = 0;
#pragma unroll
        for (int c = 0; c < CH; ++c) m2 = absmax_chunk(m2, v[c]);
        const uint32_t mbits = wave_max_u32(max(m2 & 0xFFFFu, m2 >> 16));
        const float s = row_scale<CLIP1>(mag_to_f32<BF16>(mbits), clip);

        uint2 cv[CH];                                        // int8 codes, 8 per chunk
        if (s == 0.0f) {
#pragma unroll
            for (int c = 0; c < CH; ++c) cv[c] = make_uint2(0, 0);
        } else {
            uint32_t near = 0;
            const bool tiny = !(s >= kTinyScale);
            if (!tiny) {
                const float r = 1.0f / s;
#pragma unroll
                for (int c = 0; c < CH; ++c) {
                    uint32_t w[8];
                    q4_chunk_fast<BF16, CLIP1>(v[c], r, w, near);
                    cv[c] = make_uint2(bytes4(w[0], w[1], w[2], w[3]), bytes4(w[4], w[5], w[6], w[7]));
                }
            }
            if (tiny || __any((int)near)) {
#pragma unroll
                for (int c = 0; c < CH; ++c) {
                    uint32_t w[8];
                    q4_chunk_exact<BF16>(v[c], s, w);
                    cv[c] = make_uint2(bytes4(w[0], w[1], w[2], w[3]), bytes4(w[4], w[5], w[6], w[7]));
                }
            }
        }

        int part[8];                                         // D_0..D_{J-1}, Nv at [J]
        int nv = 0;
        int dj[kMaxJ] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int q = lane + 64 * c;
            if (q < nchunk) {
                nv = __builtin_amdgcn_sdot4((int)cv[c].x, (int)cv[c].x, nv, false);
                nv = __builtin_amdgcn_sdot4((int)cv[c].y, (int)cv[c].y, nv, false);
#pragma unroll
                for (int j = 0; j < kMaxJ; ++j) {
                    if (j < J) {
                        const uint2 cc = s_cc[j * nchunk + q];
                        dj[j] = __builtin_amdgcn_sdot4((int)cv[c].x, (int)cc.x, dj[j], false);
                        dj[j] = __builtin_amdgcn_sdot4((int)cv[c].y, (int)cc.y, dj[j], false);
                    }
                }
            }
        }
        // slot J holds Nv (J <= 7 here); J == 8 handled with a second reduction
#pragma unroll
        for (int j = 0; j < kMaxJ; ++j) part[j] = (j < J) ? dj[j] : (j == J ? nv : 0);
        const int tot = reduce8(part, lane);
        int nv_tot;
        if (J < kMaxJ) {
            nv_tot = __shfl(tot, 8 * J);
        } else {
            int p2[8] = {nv, 0, 0, 0, 0, 0, 0, 0};
            nv_tot = __shfl(reduce8(p2, lane), 0);
        }
        const int slot = lane >> 3;                          // value held by this lane
        if ((lane & 7) == 0) {
            int32_t *st = stats + ((int64_t)b * N + i) * (J + 1);
            if (slot < J) {
                st[slot] = tot;
                keys[((int64_t)b * J + slot) * N + i] = exact_key(tot, nv_tot, LS);
            } else if (slot == J) {
                st[J] = nv_tot;
            }
        }
        if (J == kMaxJ && lane == 0) stats[((int64_t)b * N + i) * (J + 1) + J] = nv_tot;
    }
}

// ---------------------------------------------------------------------------
// 3. top-K.  One 1024-thread workgroup per sample; thread t owns tokens
//    t*E .. t*E+E-1 (E <= 8), so the final compaction is an ordered scan.
//    Per concept: candidates = tokens not yet kept; the composite
//    X = (key ^ 2^63) * 2^13 + (8191 - i) is unique, so "the quota largest X"
//    is exactly "the quota best tokens, lower index first on equal cosine".
//    MSD radix select with 11-bit digits, starting at the highest bit where
//    candidates differ, stopping as soon as the boundary bucket is taken whole.
// ---------------------------------------------------------------------------
constexpr int kTkThreads = 1024;
constexpr int kTkMaxE = 8;
constexpr int kDigit = 11;
constexpr int kBins = 1 << kDigit;
constexpr int kIdxBits = 13;

__device__ __forceinline__ uint32_t comp_digit(uint64_t hk, uint32_t lo13, int lo, int w) {
    const uint32_t mask = (1u << w) - 1u;
    if (lo >= kIdxBits) return (uint32_t)(hk >> (lo - kIdxBits)) & mask;
    const uint64_t x = (hk << (kIdxBits - lo)) | (uint64_t)(lo13 >> lo);
    return (uint32_t)x & mask;
}

__global__ __launch_bounds__(kTkThreads) void k_select_topk(const int64_t *__restrict__ keys,
                                                            int N, int J, int K,
                                                            int32_t *__restrict__ idx_out) {
    __shared__ uint32_t hist[kBins];
    __shared__ uint32_t wtot[kTkThreads / 64];
    __shared__ uint64_t rmin[kTkThreads / 64], rmax[kTkThreads / 64];
    __shared__ uint32_t sh_bucket, sh_gt, sh_eq;

    const int b = blockIdx.x;
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int E = (N + kTkThreads - 1) / kTkThreads;
    for (int q = t; q < kBins; q += kTkThreads) hist[q] = 0;
    uint32_t kept = 0;

    for (int j = 0; j < J; ++j) {
        const uint32_t quota = (uint32_t)(K / J + (j < K % J ? 1 : 0));
        if (quota == 0) continue;
        const int64_t *kj = keys + ((int64_t)b * J + j) * N;
        uint64_t hk[kTkMaxE];
        uint32_t cont = 0;
        uint64_t mn = ~0ull, mx = 0;
#pragma unroll
        for (int e = 0; e < kTkMaxE; ++e) {
            const int i = t * E + e;
            hk[e] = 0;
            if (e < E && i < N && !((kept >> e) & 1u)) {
                hk[e] = (uint64_t)kj[i] ^ (1ull << 63);
                cont |= 1u << e;
                mn = min(mn, hk[e]);
                mx = max(mx, hk[e]);
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            mn = min(mn, (uint64_t)__shfl_xor((unsigned long long)mn, o));
            mx = max(mx, (uint64_t)__shfl_xor((unsigned long long)mx, o));
        }
        if (lane == 0) { rmin[wave] = mn; rmax[wave] = mx; }
        __syncthreads();
        mn = rmin[0];
        mx = rmax[0];
        for (int w = 1; w < kTkThreads / 64; ++w) { mn = min(mn, rmin[w]); mx = max(mx, rmax[w]); }
        int pos = (mn != mx) ? kIdxBits + 64 - __clzll((long long)(mn ^ mx)) : kIdxBits;

        uint32_t need = quota;
        while (true) {
            const int w = min(kDigit, pos);
            const int lo = pos - w;
#pragma unroll
            for (int e = 0; e < kTkMaxE; ++e)
                if ((cont >> e) & 1u)
                    atomicAdd(&hist[comp_digit(hk[e], (uint32_t)(8191 - (t * E + e)), lo, w)], 1u);
            __syncthreads();
            // reverse-order inclusive scan: thread t covers bins kBins-1-2t, kBins-2-2t
            const int b0 = kBins - 1 - 2 * t, b1 = kBins - 2 - 2 * t;
            const uint32_t c0 = hist[b0], c1 = hist[b1];
            hist[b0] = 0;
            hist[b1] = 0;
            uint32_t inc = c0 + c1;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t up = (uint32_t)__shfl_up((int)inc, o);
                if (lane >= o) inc += up;
            }
            if (lane == 63) wtot[wave] = inc;
            __syncthreads();
            uint32_t excl = inc - (c0 + c1);
            for (int w2 = 0; w2 < wave; ++w2) excl += wtot[w2];
            if (excl < need && need <= excl + c0) { sh_bucket = b0; sh_gt = excl; sh_eq = c0; }
            const uint32_t e1 = excl + c0;
            if (e1 < need && need <= e1 + c1) { sh_bucket = b1; sh_gt = e1; sh_eq = c1; }
            __syncthreads();
            const uint32_t bucket = sh_bucket, gt = sh_gt, eq = sh_eq;
#pragma unroll
            for (int e = 0; e < kTkMaxE; ++e) {
                if ((cont >> e) & 1u) {
                    const uint32_t dg = comp_digit(hk[e], (uint32_t)(8191 - (t * E + e)), lo, w);
                    if (dg > bucket) { kept |= 1u << e; cont &= ~(1u << e); }
                    else if (dg < bucket) { cont &= ~(1u << e); }
                }
            }
            need -= gt;
            if (eq == need || lo == 0) { kept |= cont; break; }   // block-uniform
            pos = lo;
        }
    }

    // ordered compaction of the kept set
    const uint32_t cnt = __builtin_popcount(kept);
    uint32_t inc = cnt;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t up = (uint32_t)__shfl_up((int)inc, o);
        if (lane >= o) inc += up;
    }
    __syncthreads();
    if (lane == 63) wtot[wave] = inc;
    __syncthreads();
    uint32_t pos = inc - cnt;
    for (int w2 = 0; w2 < wave; ++w2) pos += wtot[w2];
    int32_t *out = idx_out + (int64_t)b * K;
#pragma unroll
    for (int e = 0; e < kTkMaxE; ++e)
        if (((kept >> e) & 1u) && pos < (uint32_t)K) out[pos++] = t * E + e;
}

// ---------------------------------------------------------------------------
// 4. gather: one wavefront per output row, 16-byte copies
// ---------------------------------------------------------------------------
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
    for (int q = lane; q < dchunks; q += 64) dst[q] = src[q];
}

template <int CH, bool BF16, bool CLIP1>
hipError_t launch_score(int B, int N, int d, int J, float clip, int LS, const void *vis,
                        const SelectWorkspace &ws, hipStream_t stream) {
    constexpr int kRowsPerWave = 16;
    const dim3 grid((N + 4 * kRowsPerWave - 1) / (4 * kRowsPerWave), B);
    const size_t lds = (size_t)J * d;
    hipLaunchKernelGGL((k_select_score<CH, BF16, CLIP1>), grid, dim3(256), lds, stream,
                       static_cast<const uint8_t *>(vis), N, d, J, clip, kRowsPerWave, LS,
                       ws.ccodes, ws.stats, ws.keys);
    return hipGetLastError();
}

template <bool BF16, bool CLIP1>
hipError_t launch_score_typed(int B, int N, int d, int J, float clip, int LS, const void *vis,
                              const SelectWorkspace &ws, hipStream_t stream) {
    const int per_lane = (d / 8 + 63) / 64;
    if (per_lane <= 1) return launch_score<1, BF16, CLIP1>(B, N, d, J, clip, LS, vis, ws, stream);
    if (per_lane <= 2) return launch_score<2, BF16, CLIP1>(B, N, d, J, clip, LS, vis, ws, stream);
    if (per_lane <= 4) return launch_score<4, BF16, CLIP1>(B, N, d, J, clip, LS, vis, ws, stream);
    if (per_lane <= 8) return launch_score<8, BF16, CLIP1>(B, N, d, J, clip, LS, vis, ws, stream);
    if (per_lane <= 10) return launch_score<10, BF16, CLIP1>(B, N, d, J, clip, LS, vis, ws, stream);
    if (per_lane <= 16) return launch_score<16, BF16, CLIP1>(B, N, d, J, clip, LS, vis, ws, stream);
    return launch_score<32, BF16, CLIP1>(B, N, d, J, clip, LS, vis, ws, stream);
}

template <bool BF16, bool CLIP1>
hipError_t launch_concepts(int rows, int d, float clip, const void *con, int8_t *cc,
                           hipStream_t stream) {
    hipLaunchKernelGGL((k_concept_codes<BF16, CLIP1>), dim3((rows + 3) / 4), dim3(256), 0,
                       stream, static_cast<const uint8_t *>(con), rows, d, clip, cc);
    return hipGetLastError();
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

size_t select_workspace_bytes(int B, int N, int d, int J) {
    return align256((size_t)B * N * (J + 1) * 4) + align256((size_t)B * J * N * 8) +
           align256((size_t)B * J * d);
}

SelectWorkspace select_workspace_carve(void *ws, int B, int N, int d, int J) {
    uint8_t *p = static_cast<uint8_t *>(ws);
    SelectWorkspace w;
    w.stats = reinterpret_cast<int32_t *>(p);
    p += align256((size_t)B * N * (J + 1) * 4);
    w.keys = reinterpret_cast<int64_t *>(p);
    p += align256((size_t)B * J * N * 8);
    w.ccodes = reinterpret_cast<int8_t *>(p);
    return w;
}

hipError_t launch_select(p4q_dtype dt, int B, int N, int d, const void *vis, const void *concepts,
                         int J, const void *text, int T, int K, float clip, int32_t *idx_out,
                         void *tokens_out, const SelectWorkspace &ws, hipStream_t stream) {
    const bool bf16 = (dt == P4Q_BF16);
    const bool clip1 = (clip == 1.0f);
    // 2^LS >= (64 d)^2: LS = 2 * ceil(log2(64 d))
    int lg = 0;
    while ((1ll << lg) < 64ll * d) ++lg;
    const int LS = 2 * lg;
    hipError_t e;
    if (bf16) e = clip1 ? launch_concepts<true, true>(B * J, d, clip, concepts, ws.ccodes, stream)
                        : launch_concepts<true, false>(B * J, d, clip, concepts, ws.ccodes, stream);
    else e = clip1 ? launch_concepts<false, true>(B * J, d, clip, concepts, ws.ccodes, stream)
                   : launch_concepts<false, false>(B * J, d, clip, concepts, ws.ccodes, stream);
    if (e != hipSuccess) return e;
    if (bf16) e = clip1 ? launch_score_typed<true, true>(B, N, d, J, clip, LS, vis, ws, stream)
                        : launch_score_typed<true, false>(B, N, d, J, clip, LS, vis, ws, stream);
    else e = clip1 ? launch_score_typed<false, true>(B, N, d, J, clip, LS, vis, ws, stream)
                   : launch_score_typed<false, false>(B, N, d, J, clip, LS, vis, ws, stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_select_topk, dim3(B), dim3(kTkThreads), 0, stream, ws.keys, N, J, K,
                       idx_out);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t rows = (int64_t)B * (K + T);
    hipLaunchKernelGGL(k_select_gather, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream,
                       static_cast<const uint4 *>(vis), static_cast<const uint4 *>(text), idx_out,
                       B, N, K, T, d / 8, static_cast<uint4 *>(tokens_out));
    return hipGetLastError();
}

}  // namespace p4q
