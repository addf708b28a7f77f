// Visual Diversity completion of the three-stage selector (P4Q Sec. 3.2,
// the diversity term of Eq. p4q_progressive_selection): greedy max-min
// selection on the cosine similarities of the fake-quantized copies.
//
// Every candidate i (a token not yet kept) carries m_i = the maximum over the
// kept set S of cos(i, t); each step keeps the candidate with the smallest
// m_i (equal values: lower index), then raises every m_i to cos(i, new) where
// that is larger.  Cosines come from the code Gram matrix G = C C^T (exact
// int32; Nv_i = G[i][i]):
//     cos(i, t) = G[i][t] / sqrt(Nv_i Nv_t)   (0 when G[i][t] == 0),
// compared through the exact rational sgn(cos) cos^2.  With an empty kept set
// the first pick is the most salient token (largest CLS weight).
//
// State of a candidate: the pair (p, q) with m_i^2-value p / (Nv_i q), where
// a cosine to t gives (sgn(D) D^2, Nv_t) and a zero cosine (0, 1).  For one
// candidate, (p', q') > (p, q) <=> p' q > p q': with d <= 8192, |p| <= 2^38 and
// q <= 2^19, so both products are exact in int64.
//
// Across candidates the step compares fp32 approximations of the values
// (each within a few ulps of the exact rational); when the two smallest lie
// within a small ulp window, every candidate in that window is compared
// exactly with 128-bit cross products, so the pick is always the exact
// minimum (equal values: lower index).
#include "p4q_internal.h"

#include "wave_ops.h"

#include <algorithm>

namespace p4q {
namespace {

constexpr int64_t kNoneP = -(1LL << 40);      // below every cosine: "S empty"
constexpr uint64_t kIdxMask = 0x1FFFull;      // 13 index bits (N <= 8192)
constexpr uint64_t kNoKey = ~0ull;
constexpr uint32_t kNone32 = 0xFFFFFFFFu;

// the pair of cos(i, t) from D = G[i][t] and Nv_t
__device__ __forceinline__ void cos_pair(int32_t D, int32_t nvt, int64_t &p, int32_t &q) {
    const int64_t d2 = (int64_t)D * (int64_t)D;
    p = D > 0 ? d2 : -d2;
    q = D != 0 ? nvt : 1;
}

// (p1, q1) above (p0, q0) for one candidate
__device__ __forceinline__ bool pair_gt(int64_t p1, int32_t q1, int64_t p0, int32_t q0) {
    return p1 * (int64_t)q0 > p0 * (int64_t)q1;
}

// exact p_a / den_a < p_b / den_b (den > 0), by 128-bit cross products
__device__ __forceinline__ bool val_lt(int64_t pa, uint64_t da, int64_t pb, uint64_t db) {
    const int sa = (pa > 0) - (pa < 0), sb = (pb > 0) - (pb < 0);
    if (sa != sb) return sa < sb;
    if (sa == 0) return false;
    const uint64_t ma = (uint64_t)(sa > 0 ? pa : -pa), mb = (uint64_t)(sb > 0 ? pb : -pb);
    const uint64_t lh = __umul64hi(ma, db), ll = ma * db;
    const uint64_t rh = __umul64hi(mb, da), rl = mb * da;
    const bool lt = lh < rh || (lh == rh && ll < rl);
    const bool gt = lh > rh || (lh == rh && ll > rl);
    return sa > 0 ? lt : gt;
}

// merge two (smallest, second smallest) pairs
__device__ __forceinline__ void merge2(uint64_t &k1, uint64_t &k2, uint64_t o1, uint64_t o2) {
    const uint64_t lo = k1 < o1 ? k1 : o1;
    const uint64_t hi = k1 < o1 ? o1 : k1;
    const uint64_t m2 = k2 < o2 ? k2 : o2;
    k1 = lo;
    k2 = hi < m2 ? hi : m2;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    return (uint64_t)__shfl_xor((unsigned long long)v, m);
}

// ---------------------------------------------------------------------------
// Initial state: for every token i, the maximum over the n0 tokens already
// kept of the pair of cos(i, t).  Grid (ceil(N / 256), B, C): block z takes
// the kept tokens [z n0 / C, (z + 1) n0 / C) and writes its partial maximum
// to plane z of mp / mq ([C][B][N]); the greedy kernel merges the planes.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_div_init(const int32_t *__restrict__ G, int N,
                                                  const int32_t *__restrict__ stages, int K, int n0,
                                                  int64_t *__restrict__ mp, int32_t *__restrict__ mq) {
    extern __shared__ int32_t s_list[];            // [cnt] tokens, then [cnt] Nv
    const int b = blockIdx.y, z = blockIdx.z, C = gridDim.z;
    const int q0 = (int)((int64_t)z * n0 / C), cnt = (int)((int64_t)(z + 1) * n0 / C) - q0;
    int32_t *s_nv = s_list + cnt;
    const int32_t *Gb = G + (int64_t)b * N * N;
    for (int q = threadIdx.x; q < cnt; q += 256) {
        int tk = stages[(int64_t)b * K + q0 + q];
        if ((unsigned)tk >= (unsigned)N) tk = 0;   // never taken: the stages hold valid tokens
        s_list[q] = tk;
        s_nv[q] = Gb[(int64_t)tk * N + tk];
    }
    __syncthreads();
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= N) return;
    int64_t p = kNoneP;
    int32_t q = 1;
    constexpr int U = 16;                          // loads in flight per thread
    for (int u0 = 0; u0 < cnt; u0 += U) {
        int32_t D[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            D[u] = (u0 + u < cnt) ? Gb[(int64_t)s_list[u0 + u] * N + i] : 0;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (u0 + u < cnt) {
                int64_t pp;
                int32_t qq;
                cos_pair(D[u], s_nv[u0 + u], pp, qq);
                if (pair_gt(pp, qq, p, q)) { p = pp; q = qq; }
            }
        }
    }
    const int64_t o = ((int64_t)z * gridDim.y + b) * N + i;
    mp[o] = p;
    mq[o] = q;
}

// ---------------------------------------------------------------------------
// Cross-lane pieces of the greedy step: DPP moves inside rows of 16 lanes,
// readlane across the 4 rows.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
    const int lo = __builtin_amdgcn_mov_dpp((int)(uint32_t)v, CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_mov_dpp((int)(uint32_t)(v >> 32), CTRL, 0xF, 0xF, false);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
    const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}

template <int CTRL>
__device__ __forceinline__ void merge_dpp(uint64_t &k1, uint64_t &k2) {
    const uint64_t o1 = dpp64<CTRL>(k1), o2 = dpp64<CTRL>(k2);
    merge2(k1, k2, o1, o2);
}

// (smallest, second smallest) of each row of 16 lanes, in every lane of it
__device__ __forceinline__ void row_min2(uint64_t &k1, uint64_t &k2) {
    merge_dpp<0xB1>(k1, k2);     // quad_perm [1,0,3,2]: lane ^ 1
    merge_dpp<0x4E>(k1, k2);     // quad_perm [2,3,0,1]: lane ^ 2
    merge_dpp<0x141>(k1, k2);    // row_half_mirror: the other quad of the 8
    merge_dpp<0x140>(k1, k2);    // row_mirror: the other 8 of the row
}

// ... of the whole wavefront, wave-uniform
__device__ __forceinline__ void wave_min2(uint64_t &k1, uint64_t &k2) {
    row_min2(k1, k2);
    uint64_t a1 = readlane64(k1, 0), a2 = readlane64(k2, 0);
#pragma unroll
    for (int r = 1; r < 4; ++r) merge2(a1, a2, readlane64(k1, 16 * r), readlane64(k2, 16 * r));
    k1 = a1;
    k2 = a2;
}

template <int CTRL>
__device__ __forceinline__ uint64_t min_dpp(uint64_t a) {
    const uint64_t b = dpp64<CTRL>(a);
    return b < a ? b : a;
}

// smallest key of the wavefront, wave-uniform
__device__ __forceinline__ uint64_t wave_min1(uint64_t a) {
    a = min_dpp<0xB1>(a);
    a = min_dpp<0x4E>(a);
    a = min_dpp<0x141>(a);
    a = min_dpp<0x140>(a);
    uint64_t r = readlane64(a, 0);
#pragma unroll
    for (int w = 1; w < 4; ++w) {
        const uint64_t x = readlane64(a, 16 * w);
        r = x < r ? x : r;
    }
    return r;
}

template <int CTRL>
__device__ __forceinline__ uint32_t min_dpp32(uint32_t a) {
    return min(a, (uint32_t)__builtin_amdgcn_mov_dpp((int)a, CTRL, 0xF, 0xF, false));
}

// smallest value of the wavefront, wave-uniform
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t a) {
    a = min_dpp32<0xB1>(a);
    a = min_dpp32<0x4E>(a);
    a = min_dpp32<0x141>(a);
    a = min_dpp32<0x140>(a);
    const uint32_t r0 = __builtin_amdgcn_readlane((int)a, 0), r1 = __builtin_amdgcn_readlane((int)a, 16);
    const uint32_t r2 = __builtin_amdgcn_readlane((int)a, 32), r3 = __builtin_amdgcn_readlane((int)a, 48);
    return min(min(r0, r1), min(r2, r3));
}

// order-preserving bits of an fp32 value (-0 below +0)
__device__ __forceinline__ uint32_t ord32(float v) {
    const uint32_t u = __float_as_uint(v);
    return (u >> 31) ? ~u : (u | 0x80000000u);
}

// Candidates whose approximate values lie within this many fp32 ulps of each
// other are compared exactly (the approximations err by at most ~10 ulps).
constexpr uint32_t kUlpTol = 32;

// ---------------------------------------------------------------------------
// The greedy scan: one NT-thread work-group per sample; thread t owns
// candidates i = e * NT + t (e < E), so a row of G is read with coalesced
// loads.  Per candidate the exact pair (p, q) is kept with vf ~ p / (Nv_i q)
// in fp32 (relative error <= 5 * 2^-24: three roundings and two correctly
// rounded reciprocals).  A step:
//   1. key = (ord32(vf) << 32) | i; the block's smallest two keys (DPP
//      inside wavefronts, one LDS exchange, one barrier);
//   2. if the two smallest values are more than kUlpTol ulps apart, the
//      smallest key's token is the exact minimum; otherwise every candidate
//      within kUlpTol ulps of the smallest is compared exactly (128-bit
//      cross products; equal values: lower index);
//   3. the new token's row D = G[best][.] updates each candidate from
//      c = D |D| / (Nv_i Nv_best) in fp32: clearly below vf -> unchanged,
//      clearly above -> replaced, within kUlpTol ulps -> exact comparison of
//      the pairs.
// ---------------------------------------------------------------------------
template <int E, int NT>
__global__ __launch_bounds__(NT) void k_div_greedy(const int32_t *__restrict__ G, int N,
                                                   const int64_t *__restrict__ mp,
                                                   const int32_t *__restrict__ mq,
                                                   const float *__restrict__ cls, int K, int n0,
                                                   int kd, int nplanes, int32_t *__restrict__ stages,
                                                   int32_t *__restrict__ idx_out) {
    constexpr int NW = NT / 64;
    static_assert(NT >= 256 && NT <= 1024 && NT % 64 == 0, "one bitmap word per thread");
    // greedy picks verified per block-wide selection (fewer at 1024 threads,
    // where a thread has 128 registers)
    constexpr int kBatch = NT <= 512 ? (E <= 6 ? 16 : 8) : (E <= 5 ? 4 : 2);
    __shared__ uint32_t bm[256];                                   // kept bitmap (N <= 8192)
    __shared__ unsigned long long r1[2][NW], r2[2][NW];
    __shared__ long long xp[NW];
    __shared__ unsigned long long xd[NW];
    __shared__ int xi[NW];
    __shared__ __attribute__((aligned(16))) uint32_t wtot[16];
    __shared__ int32_t nvs[8192];                                  // Nv of the candidates
    __shared__ uint32_t wlv[NW][kBatch + 1], wli[NW][kBatch + 1];  // per-wavefront smallest values, tokens
    __shared__ uint32_t vflag[2];                                  // verified list positions

    const int b = blockIdx.x, t = threadIdx.x, lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int32_t *Gb = G + (int64_t)b * N * N;
    int32_t *st = stages + (int64_t)b * K;
    for (int q = t; q < 256; q += NT) bm[q] = 0;
    __syncthreads();
    for (int q = t; q < n0; q += NT) {
        const int tk = st[q];
        if ((unsigned)tk < (unsigned)N) atomicOr(&bm[tk >> 5], 1u << (tk & 31));
    }
    __syncthreads();

    int64_t p[E];
    int32_t q[E], nv[E];
    float vf[E], inv[E];
    uint32_t live = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int i = e * NT + t;
        p[e] = kNoneP;
        q[e] = 1;
        nv[e] = 0;
        inv[e] = 0.0f;
        vf[e] = -__builtin_huge_valf();
        if (kd > 0 && i < N && !((bm[i >> 5] >> (i & 31)) & 1u)) {
            live |= 1u << e;
            nv[e] = Gb[(int64_t)i * N + i];
            nvs[i] = nv[e];
            inv[e] = nv[e] > 0 ? 1.0f / (float)nv[e] : 0.0f;
            if (n0 > 0) {
                for (int z = 0; z < nplanes; ++z) {
                    const int64_t o = ((int64_t)z * gridDim.x + b) * N + i;
                    const int64_t pz = mp[o];
                    const int32_t qz = mq[o];
                    if (pair_gt(pz, qz, p[e], q[e])) { p[e] = pz; q[e] = qz; }
                }
                vf[e] = p[e] == 0 ? 0.0f : ((float)p[e] * inv[e]) * (1.0f / (float)q[e]);
            }
        }
    }

    // block-wide smallest two of the per-thread pairs; `par` alternates the
    // LDS slots between consecutive steps (one barrier per step)
    auto block_min2 = [&](uint64_t k1, uint64_t k2, int par, uint64_t &o1, uint64_t &o2) {
        wave_min2(k1, k2);
        if (lane == 0) { r1[par][wave] = k1; r2[par][wave] = k2; }
        __syncthreads();
        uint64_t a1 = lane < NW ? r1[par][lane] : kNoKey;
        uint64_t a2 = lane < NW ? r2[par][lane] : kNoKey;
        row_min2(a1, a2);
        o1 = readlane64(a1, 0);
        o2 = readlane64(a2, 0);
    };

    // exact minimum among the candidates whose ord32 value is <= vmax
    auto exact_min = [&](uint32_t vmax) -> int {
        int64_t bp = 0;
        uint64_t bd = 1;
        int bi = 0x7FFFFFFF;
        auto take = [&](int64_t op, uint64_t od, int oi) {
            if (oi == 0x7FFFFFFF) return;
            if (bi == 0x7FFFFFFF || val_lt(op, od, bp, bd) || (!val_lt(bp, bd, op, od) && oi < bi)) {
                bp = op; bd = od; bi = oi;
            }
        };
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if (((live >> e) & 1u) && ord32(vf[e]) <= vmax)
                take(p[e], p[e] == 0 ? 1ull : (uint64_t)nv[e] * (uint64_t)q[e], e * NT + t);
        }
#pragma unroll
        for (int m = 1; m < 64; m <<= 1) {
            const int64_t op = (int64_t)__shfl_xor((long long)bp, m);
            const uint64_t od = (uint64_t)__shfl_xor((unsigned long long)bd, m);
            const int oi = __shfl_xor(bi, m);
            take(op, od, oi);
        }
        if (lane == 0) { xp[wave] = bp; xd[wave] = bd; xi[wave] = bi; }
        __syncthreads();
        if (lane < NW) { bp = xp[lane]; bd = xd[lane]; bi = xi[lane]; }
        else { bp = 0; bd = 1; bi = 0x7FFFFFFF; }
#pragma unroll
        for (int m = 1; m < NW; m <<= 1) {
            const int64_t op = (int64_t)__shfl_xor((long long)bp, m);
            const uint64_t od = (uint64_t)__shfl_xor((unsigned long long)bd, m);
            const int oi = __shfl_xor(bi, m);
            take(op, od, oi);
        }
        return __shfl(bi, 0);
    };

    // keep token `best`; update the candidates from its row of G unless it
    // was the last pick.  The row of `next` (the runner-up, almost always the
    // next pick: a new token rarely raises the runner-up's maximum) is loaded
    // ahead into Dn, so the next step usually finds its row in registers.
    const __amdgpu_buffer_rsrc_t gres =
        __builtin_amdgcn_make_buffer_rsrc((void *)Gb, 0, (int)(N * N * 4), 0x00020000);
    uint32_t coff[E];                     // byte offsets of this thread's columns
#pragma unroll
    for (int e = 0; e < E; ++e) coff[e] = (e * NT + t < N) ? (uint32_t)(e * NT + t) * 4u : 0x80000000u;
    auto load_row = [&](int r, int32_t *dst) {
        const uint32_t rb = (uint32_t)r * (uint32_t)N * 4u;
#pragma unroll
        for (int e = 0; e < E; ++e)
            dst[e] = __builtin_amdgcn_raw_buffer_load_b32(gres, coff[e] == 0x80000000u ? coff[e] : rb + coff[e], 0, 0);
    };
    int picks = 0;
    int pre = -1;
    int32_t Dn[E];
#pragma unroll
    for (int e = 0; e < E; ++e) Dn[e] = 0;
    __syncthreads();                                               // nvs complete
    auto keep = [&](int best, int next) {
        if (t == 0) {
            st[n0 + picks] = best;
            bm[best >> 5] |= 1u << (best & 31);
        }
        if ((best % NT) == t) live &= ~(1u << (best / NT));
        ++picks;
        if (picks == kd) return;
        // Row loads are unconditional buffer loads (offsets past the row read
        // as 0), so the compiler's wait before the update only covers the
        // older loads and leaves the prefetch in flight.
        int32_t D[E];
        if (best == pre) {
#pragma unroll
            for (int e = 0; e < E; ++e) D[e] = Dn[e];
        } else {
            load_row(best, D);
        }
        pre = next;
        load_row(next >= 0 ? next : best, Dn);
        const int32_t nvb = nvs[best];
        const float invb = nvb > 0 ? 1.0f / (float)nvb : 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if ((live >> e) & 1u) {
                const float df = (float)D[e];
                const float cf = ((df * __builtin_fabsf(df)) * inv[e]) * invb;
                const int64_t oc = ord32(cf), ov = ord32(vf[e]);
                if (oc + (int64_t)kUlpTol < ov) continue;          // clearly not above
                int64_t pp;
                int32_t qq;
                cos_pair(D[e], nvb, pp, qq);
                if (oc > ov + (int64_t)kUlpTol || pair_gt(pp, qq, p[e], q[e])) {
                    p[e] = pp;
                    q[e] = qq;
                    vf[e] = cf;
                }
            }
        }
    };

    if (t == 0) { vflag[0] = 0; vflag[1] = 0; }
    __syncthreads();
    int par = 0;
    if (n0 == 0 && kd > 0) {
        // seed: the most salient token (largest CLS weight, lower index first)
        uint64_t k1 = kNoKey, k2 = kNoKey;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if ((live >> e) & 1u) {
                const int i = e * NT + t;
                uint32_t u = __float_as_uint(cls[(int64_t)b * N + i]);
                if (u == 0x80000000u) u = 0;                                 // -0 ranks as +0
                const uint32_t o = (u >> 31) ? ~u : (u | 0x80000000u);       // larger weight -> larger o
                merge2(k1, k2, ((uint64_t)(~o) << 32) | (uint64_t)i, kNoKey);
            }
        }
        uint64_t o1, o2;
        block_min2(k1, k2, par, o1, o2);
        par ^= 1;
        if (o1 != kNoKey) keep((int)(o1 & kIdxMask), -1);
    }
    // Batched steps.  The kBatch + 1 smallest approximate values c_0 <= c_1
    // <= ... are taken in one block-wide selection and their rows loaded
    // together.  c_0 is the exact minimum when it is more than kUlpTol ulps
    // below c_1 (otherwise the exact comparison picks one token and the batch
    // ends there).  c_j (j >= 1) is the exact minimum after c_0 .. c_{j-1} are
    // kept when its value raised by their rows is still more than kUlpTol ulps
    // below the value of c_{j+1}: every other candidate's value can only have
    // grown from at least that.  The verified prefix is kept and every
    // candidate is updated from its rows.
    int nbatch = 0;
    while (picks < kd) {
        // (1) selection on the order-preserving bits of vf (ties between
        //     equal values are left to the verification, which never accepts
        //     them): per wavefront the kBatch + 1 smallest, then the same
        //     extraction over the wavefronts' lists
        uint32_t lv[kBatch + 1], li[kBatch + 1];
        {
            uint32_t ov[E];
#pragma unroll
            for (int e = 0; e < E; ++e) ov[e] = ((live >> e) & 1u) ? ord32(vf[e]) : kNone32;
            uint32_t ext = 0;
            auto local_min = [&]() {
                uint32_t m = kNone32;
#pragma unroll
                for (int e = 0; e < E; ++e) m = ((ext >> e) & 1u) ? m : min(m, ov[e]);
                return m;
            };
            uint32_t lm = local_min();
#pragma unroll
            for (int r = 0; r <= kBatch; ++r) {
                const uint32_t v = wave_min_u32(lm);
                uint32_t tok = kNone32;
                if (v != kNone32) {
                    const int src = (int)__builtin_ctzll(__ballot(lm == v));      // lowest lane holding v
                    int slot = 0;
                    if (lane == src) {
#pragma unroll
                        for (int e = E - 1; e >= 0; --e)
                            if (!((ext >> e) & 1u) && ov[e] == v) slot = e;
                        ext |= 1u << slot;
                        lm = local_min();
                    }
                    tok = (uint32_t)__shfl(slot * NT + t, src);
                }
                if (lane == 0) { wlv[wave][r] = v; wli[wave][r] = tok; }
            }
            __syncthreads();
            constexpr int NE = NW * (kBatch + 1);
            constexpr int PER = (NE + 63) / 64;
            uint32_t av[PER], ai[PER];
#pragma unroll
            for (int u = 0; u < PER; ++u) {
                const int q = lane + 64 * u;
                av[u] = q < NE ? wlv[q / (kBatch + 1)][q % (kBatch + 1)] : kNone32;
                ai[u] = q < NE ? wli[q / (kBatch + 1)][q % (kBatch + 1)] : kNone32;
            }
#pragma unroll
            for (int r = 0; r <= kBatch; ++r) {
                uint32_t m = kNone32;
#pragma unroll
                for (int u = 0; u < PER; ++u) m = min(m, av[u]);
                const uint32_t v = wave_min_u32(m);
                uint32_t tok = kNone32;
                if (v != kNone32) {
                    const int src = (int)__builtin_ctzll(__ballot(m == v));
                    uint32_t mine = kNone32;
                    if (lane == src) {
                        bool done = false;
#pragma unroll
                        for (int u = 0; u < PER; ++u)
                            if (!done && av[u] == v) { mine = ai[u]; av[u] = kNone32; done = true; }
                    }
                    tok = (uint32_t)__shfl((int)mine, src);
                }
                lv[r] = v;
                li[r] = tok;
            }
        }
        if (lv[0] == kNone32) break;          // no candidate left (not reached for kd <= N - n0)
        // (2) the head: exact unless it is clear of the runner-up
        const bool head_clear = lv[1] == kNone32 || lv[1] - lv[0] > kUlpTol;
        int nb = head_clear ? min(kBatch, kd - picks) : 1;
        int c[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) c[j] = (int)li[j];
        if (!head_clear) c[0] = exact_min(lv[0] + kUlpTol);
        for (int j = 1; j < kBatch; ++j)      // the list may run out
            if (j < nb && lv[j] == kNone32) nb = j;
        // (3) rows of the batch, all in flight together
        int32_t Drow[kBatch][E];
        float invb[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            if (j < nb) {
                load_row(c[j], Drow[j]);
                const int32_t nvb = nvs[c[j]];
                invb[j] = nvb > 0 ? 1.0f / (float)nvb : 0.0f;
            }
        }
        // (4) verify c_1 .. c_{nb-1}: the owner of c_j raises its value by the
        // rows of c_0 .. c_{j-1} and compares with the value of c_{j+1}
        const int fb = nbatch & 1;            // alternating flag word: one barrier per batch
        ++nbatch;
        if (nb > 1) {
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const int i = e * NT + t;
#pragma unroll
                for (int j = 1; j < kBatch; ++j) {
                    if (j < nb && i == c[j] && ((live >> e) & 1u)) {
                        float v = vf[e];
#pragma unroll
                        for (int k2 = 0; k2 < kBatch; ++k2) {
                            if (k2 < j) {
                                const float df = (float)Drow[k2][e];
                                v = __builtin_fmaxf(v, ((df * __builtin_fabsf(df)) * inv[e]) * invb[k2]);
                            }
                        }
                        if (lv[j + 1] == kNone32 || (int64_t)ord32(v) + (int64_t)kUlpTol < (int64_t)lv[j + 1])
                            atomicOr(&vflag[fb], 1u << j);
                    }
                }
            }
        }
        __syncthreads();
        const uint32_t fl = vflag[fb];
        int a = 1;
        while (a < nb && ((fl >> a) & 1u)) ++a;
        // (5) keep c_0 .. c_{a-1}
        if (t == 0) {
            for (int j = 0; j < a; ++j) {
                st[n0 + picks + j] = c[j];
                bm[c[j] >> 5] |= 1u << (c[j] & 31);
            }
            vflag[fb ^ 1] = 0;                // the next batch's word
        }
#pragma unroll
        for (int j = 0; j < kBatch; ++j)
            if (j < a && (c[j] % NT) == t) live &= ~(1u << (c[j] / NT));
        picks += a;
        if (picks >= kd) break;
        // (6) update every candidate from the kept rows: the largest fp32
        // cosine of the batch against vf first (the usual case ends there)
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if (!((live >> e) & 1u)) continue;
            float cmax = -__builtin_huge_valf();
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                if (j < a) {
                    const float df = (float)Drow[j][e];
                    cmax = __builtin_fmaxf(cmax, ((df * __builtin_fabsf(df)) * inv[e]) * invb[j]);
                }
            }
            if ((int64_t)ord32(cmax) + (int64_t)kUlpTol < (int64_t)ord32(vf[e])) continue;   // clearly not above
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {                    // rare: row by row
                if (j < a) {
                    const float df = (float)Drow[j][e];
                    const float cf = ((df * __builtin_fabsf(df)) * inv[e]) * invb[j];
                    const int64_t oc = ord32(cf), ov = ord32(vf[e]);
                    if (oc + (int64_t)kUlpTol < ov) continue;
                    int64_t pp;
                    int32_t qq;
                    cos_pair(Drow[j][e], nvs[c[j]], pp, qq);
                    if (oc > ov + (int64_t)kUlpTol || pair_gt(pp, qq, p[e], q[e])) {
                        p[e] = pp;
                        q[e] = qq;
                        vf[e] = cf;
                    }
                }
            }
        }
    }

    // idx_out[b] = the kept set in ascending order (one bitmap word per
    // thread: N <= 8192 = 32 * 256 <= 32 * NT)
    __syncthreads();
    const int nwords = (N + 31) / 32;
    uint32_t w = 0;
    if (t < nwords) {
        w = bm[t];
        if (32 * t + 32 > N) w &= (1u << (N - 32 * t)) - 1u;
    }
    const uint32_t cnt = __builtin_popcount(w);
    const uint32_t inc = wave_inclusive_scan(cnt);
    if (lane == 63) wtot[wave] = inc;
    __syncthreads();
    uint32_t pos = inc - cnt + waves_before(wtot, wave);
    int32_t *out = idx_out + (int64_t)b * K;
    while (w) {
        const int bit = __builtin_ctz(w);
        w &= w - 1;
        if (pos < (uint32_t)K) out[pos] = 32 * t + bit;
        ++pos;
    }
}

}  // namespace

hipError_t launch_diversity(int B, int N, int K, int n0, int kd, const int32_t *gram,
                            const float *cls_attn, int64_t *mp, int32_t *mq, int32_t *stages,
                            int32_t *idx_out, hipStream_t stream) {
    // planes of the initial maxima: about 40 kept tokens per block
    const int planes = n0 > 0 ? std::min(kDivInitPlanes, (n0 + 39) / 40) : 0;
    if (kd > 0 && n0 > 0) {
        const int per = (n0 + planes - 1) / planes;
        hipLaunchKernelGGL(k_div_init, dim3((N + 255) / 256, B, planes), dim3(256), (size_t)per * 8, stream,
                           gram, N, stages, K, n0, mp, mq);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    // 512 threads while every thread holds at most 8 candidates, else 1024
#define P4Q_DV(E, NT)                                                                              \
    hipLaunchKernelGGL((k_div_greedy<E, NT>), dim3(B), dim3(NT), 0, stream, gram, N, mp, mq, cls_attn, K, \
                       n0, kd, planes, stages, idx_out)
    switch ((N + 511) / 512) {
        case 1: P4Q_DV(1, 512); break;
        case 2: P4Q_DV(2, 512); break;
        case 3: P4Q_DV(3, 512); break;
        case 4: P4Q_DV(4, 512); break;
        case 5: P4Q_DV(5, 512); break;
        case 6: P4Q_DV(6, 512); break;
        case 7: P4Q_DV(7, 512); break;
        case 8: P4Q_DV(8, 512); break;
        case 9: case 10: P4Q_DV(5, 1024); break;
        case 11: case 12: P4Q_DV(6, 1024); break;
        case 13: case 14: P4Q_DV(7, 1024); break;
        case 15: case 16: P4Q_DV(8, 1024); break;
        default: return hipErrorInvalidValue;
    }
#undef P4Q_DV
    return hipGetLastError();
}

}  // namespace p4q
