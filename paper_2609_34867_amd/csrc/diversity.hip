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
// Across candidates the step compares a 64-bit key: the fp64 quotient
// p / (Nv_i q) (exact operands, correctly rounded, hence monotone in the exact
// value), mapped to order-preserving bits, its low 13 bits replaced by the
// token index.  When the two smallest keys differ above the index bits, the
// smallest key's token is the exact minimum; otherwise (ties and near-ties,
// rare) the candidates sharing that truncated value are compared exactly with
// 128-bit cross products.
#include "p4q_internal.h"

#include "wave_ops.h"

namespace p4q {
namespace {

constexpr int64_t kNoneP = -(1LL << 40);      // below every cosine: "S empty"
constexpr int kDvThreads = 1024;
constexpr int kDvWaves = kDvThreads / 64;
constexpr uint64_t kIdxMask = 0x1FFFull;      // 13 index bits (N <= 8192)
constexpr uint64_t kNoKey = ~0ull;

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

__device__ __forceinline__ uint64_t cand_key(int64_t p, int32_t q, int32_t nvi, int i) {
    const double v = (p == 0) ? 0.0 : (double)p / ((double)nvi * (double)q);
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint64_t o = (u >> 63) ? ~u : (u | 0x8000000000000000ull);
    return (o & ~kIdxMask) | (uint64_t)i;
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
// kept of the pair of cos(i, t).  Grid (ceil(N / 256), B).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_div_init(const int32_t *__restrict__ G, int N,
                                                  const int32_t *__restrict__ stages, int K, int n0,
                                                  int64_t *__restrict__ mp, int32_t *__restrict__ mq) {
    extern __shared__ int32_t s_list[];            // [n0] tokens, then [n0] Nv
    int32_t *s_nv = s_list + n0;
    const int b = blockIdx.y;
    const int32_t *Gb = G + (int64_t)b * N * N;
    for (int q = threadIdx.x; q < n0; q += 256) {
        int tk = stages[(int64_t)b * K + q];
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
    for (int u0 = 0; u0 < n0; u0 += U) {
        int32_t D[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            D[u] = (u0 + u < n0) ? Gb[(int64_t)s_list[u0 + u] * N + i] : 0;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (u0 + u < n0) {
                int64_t pp;
                int32_t qq;
                cos_pair(D[u], s_nv[u0 + u], pp, qq);
                if (pair_gt(pp, qq, p, q)) { p = pp; q = qq; }
            }
        }
    }
    mp[(int64_t)b * N + i] = p;
    mq[(int64_t)b * N + i] = q;
}

// ---------------------------------------------------------------------------
// The greedy scan: one 1024-thread work-group per sample.  Thread t owns
// candidates i = e * 1024 + t (e < E), so each row of G is read with
// coalesced loads.  Per step: local (smallest, second smallest) key, a
// wavefront reduction, one LDS exchange between the 16 wavefronts (each
// wavefront then reduces the 16 partials itself, so one barrier per step),
// the exact tie-break when needed, and the update from the new token's row.
// ---------------------------------------------------------------------------
template <int E>
__global__ __launch_bounds__(kDvThreads) void k_div_greedy(const int32_t *__restrict__ G, int N,
                                                           const int64_t *__restrict__ mp,
                                                           const int32_t *__restrict__ mq,
                                                           const float *__restrict__ cls, int K, int n0,
                                                           int kd, int32_t *__restrict__ stages,
                                                           int32_t *__restrict__ idx_out) {
    __shared__ uint32_t bm[256];                                   // kept bitmap (N <= 8192)
    __shared__ unsigned long long r1[2][kDvWaves], r2[2][kDvWaves];
    __shared__ long long xp[kDvWaves];
    __shared__ unsigned long long xd[kDvWaves];
    __shared__ int xi[kDvWaves];
    __shared__ __attribute__((aligned(16))) uint32_t wtot[kDvWaves];

    const int b = blockIdx.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int32_t *Gb = G + (int64_t)b * N * N;
    int32_t *st = stages + (int64_t)b * K;
    for (int q = t; q < 256; q += kDvThreads) bm[q] = 0;
    __syncthreads();
    for (int q = t; q < n0; q += kDvThreads) {
        const int tk = st[q];
        if ((unsigned)tk < (unsigned)N) atomicOr(&bm[tk >> 5], 1u << (tk & 31));
    }
    __syncthreads();

    int64_t p[E];
    int32_t q[E], nv[E];
    uint64_t key[E];
    uint32_t live = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int i = e * kDvThreads + t;
        p[e] = kNoneP;
        q[e] = 1;
        nv[e] = 0;
        key[e] = kNoKey;
        if (kd > 0 && i < N && !((bm[i >> 5] >> (i & 31)) & 1u)) {
            live |= 1u << e;
            nv[e] = Gb[(int64_t)i * N + i];
            if (n0 > 0) {
                p[e] = mp[(int64_t)b * N + i];
                q[e] = mq[(int64_t)b * N + i];
                key[e] = cand_key(p[e], q[e], nv[e], i);
            }
        }
    }

    // block-wide (smallest, second smallest) of per-thread pairs; `par`
    // alternates the LDS slots between consecutive steps
    auto block_min2 = [&](uint64_t k1, uint64_t k2, int par, uint64_t &o1, uint64_t &o2) {
#pragma unroll
        for (int m = 1; m < 64; m <<= 1) merge2(k1, k2, shfl_xor_u64(k1, m), shfl_xor_u64(k2, m));
        if (lane == 0) { r1[par][wave] = k1; r2[par][wave] = k2; }
        __syncthreads();
        uint64_t a1 = lane < kDvWaves ? r1[par][lane] : kNoKey;
        uint64_t a2 = lane < kDvWaves ? r2[par][lane] : kNoKey;
#pragma unroll
        for (int m = 1; m < kDvWaves; m <<= 1) merge2(a1, a2, shfl_xor_u64(a1, m), shfl_xor_u64(a2, m));
        o1 = (uint64_t)__shfl((unsigned long long)a1, 0);
        o2 = (uint64_t)__shfl((unsigned long long)a2, 0);
    };

    // exact minimum among the candidates whose key shares the value bits `tv`
    auto exact_min = [&](uint64_t tv) -> int {
        int64_t bp = 0;
        uint64_t bd = 1;
        int bi = 0x7FFFFFFF;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if (((live >> e) & 1u) && (key[e] & ~kIdxMask) == tv) {
                const int i = e * kDvThreads + t;
                const uint64_t den = p[e] == 0 ? 1ull : (uint64_t)nv[e] * (uint64_t)q[e];
                if (bi == 0x7FFFFFFF || val_lt(p[e], den, bp, bd)) { bp = p[e]; bd = den; bi = i; }
            }
        }
        auto take = [&](int64_t op, uint64_t od, int oi) {
            if (oi == 0x7FFFFFFF) return;
            if (bi == 0x7FFFFFFF || val_lt(op, od, bp, bd) || (!val_lt(bp, bd, op, od) && oi < bi)) {
                bp = op; bd = od; bi = oi;
            }
        };
#pragma unroll
        for (int m = 1; m < 64; m <<= 1) {
            const int64_t op = (int64_t)__shfl_xor((long long)bp, m);
            const uint64_t od = (uint64_t)__shfl_xor((unsigned long long)bd, m);
            const int oi = __shfl_xor(bi, m);
            take(op, od, oi);
        }
        if (lane == 0) { xp[wave] = bp; xd[wave] = bd; xi[wave] = bi; }
        __syncthreads();
        if (lane < kDvWaves) { bp = xp[lane]; bd = xd[lane]; bi = xi[lane]; }
        else { bp = 0; bd = 1; bi = 0x7FFFFFFF; }
#pragma unroll
        for (int m = 1; m < kDvWaves; m <<= 1) {
            const int64_t op = (int64_t)__shfl_xor((long long)bp, m);
            const uint64_t od = (uint64_t)__shfl_xor((unsigned long long)bd, m);
            const int oi = __shfl_xor(bi, m);
            take(op, od, oi);
        }
        return __shfl(bi, 0);
    };

    // keep token `best`; update the candidates from its row of G unless it
    // was the last pick
    int picks = 0;
    auto keep = [&](int best) {
        if (t == 0) {
            st[n0 + picks] = best;
            bm[best >> 5] |= 1u << (best & 31);
        }
        if ((best & (kDvThreads - 1)) == t) live &= ~(1u << (best / kDvThreads));
        ++picks;
        if (picks == kd) return;
        const int32_t *row = Gb + (int64_t)best * N;
        int32_t D[E];
#pragma unroll
        for (int e = 0; e < E; ++e) D[e] = ((live >> e) & 1u) ? row[e * kDvThreads + t] : 0;
        const int32_t nvb = row[best];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if ((live >> e) & 1u) {
                int64_t pp;
                int32_t qq;
                cos_pair(D[e], nvb, pp, qq);
                if (pair_gt(pp, qq, p[e], q[e]) || key[e] == kNoKey) {
                    p[e] = pp;
                    q[e] = qq;
                    key[e] = cand_key(pp, qq, nv[e], e * kDvThreads + t);
                }
            }
        }
    };

    int par = 0;
    if (n0 == 0 && kd > 0) {
        // seed: the most salient token (largest CLS weight, lower index first)
        uint64_t k1 = kNoKey, k2 = kNoKey;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if ((live >> e) & 1u) {
                const int i = e * kDvThreads + t;
                uint32_t u = __float_as_uint(cls[(int64_t)b * N + i]);
                if (u == 0x80000000u) u = 0;                                 // -0 ranks as +0
                const uint32_t o = (u >> 31) ? ~u : (u | 0x80000000u);   // larger weight -> larger o
                const uint64_t k = ((uint64_t)(~o) << 13) | (uint64_t)i;
                merge2(k1, k2, k, kNoKey);
            }
        }
        uint64_t o1, o2;
        block_min2(k1, k2, par, o1, o2);
        par ^= 1;
        if (o1 != kNoKey) keep((int)(o1 & kIdxMask));
    }
    while (picks < kd) {
        uint64_t k1 = kNoKey, k2 = kNoKey;
#pragma unroll
        for (int e = 0; e < E; ++e)
            if ((live >> e) & 1u) merge2(k1, k2, key[e], kNoKey);
        uint64_t o1, o2;
        block_min2(k1, k2, par, o1, o2);
        par ^= 1;
        if (o1 == kNoKey) break;             // no candidate left (not reached for kd <= N - n0)
        int best = (int)(o1 & kIdxMask);
        if (o2 != kNoKey && (o1 & ~kIdxMask) == (o2 & ~kIdxMask)) best = exact_min(o1 & ~kIdxMask);
        keep(best);
    }

    // idx_out[b] = the kept set in ascending order
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
    if (kd > 0 && n0 > 0) {
        hipLaunchKernelGGL(k_div_init, dim3((N + 255) / 256, B), dim3(256), (size_t)n0 * 8, stream,
                           gram, N, stages, K, n0, mp, mq);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    switch ((N + kDvThreads - 1) / kDvThreads) {      // candidates per thread, N <= 8192
#define P4Q_DV(E)                                                                                 \
    case E:                                                                                      \
        hipLaunchKernelGGL(k_div_greedy<E>, dim3(B), dim3(kDvThreads), 0, stream, gram, N, mp, mq, \
                           cls_attn, K, n0, kd, stages, idx_out);                                \
        break;
        P4Q_DV(1) P4Q_DV(2) P4Q_DV(3) P4Q_DV(4) P4Q_DV(5) P4Q_DV(6) P4Q_DV(7) P4Q_DV(8)
#undef P4Q_DV
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace p4q
