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

#include <algorithm>

namespace p4q {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf2 __attribute__((ext_vector_type(2)));

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

// bits of one output value (same roundings as store_out)
template <bool BF16OUT>
__device__ __forceinline__ uint32_t out_bits(float v) {
    if constexpr (BF16OUT) {
        const uint32_t u = __float_as_uint(v);
        return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
    } else {
        asm volatile("" : "+v"(v));                          // see store_out
        return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v);
    }
}

// 128 x 128 tile, 4 wavefronts of 64 x 64, register-staged double
// buffering.  Serves the code Gram matrices of images with fewer than 1024
// tokens (y == nullptr: int32 accumulators only, no scales read).
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
        // y == nullptr: accumulators only (Gram matrices), no scales read
        const float swn = (y && n < N) ? sw[n] : 0.0f;
#pragma unroll
        for (int f = 0; f < 4; ++f) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int m = m0 + wm * 64 + f * 16 + 4 * (lane >> 4) + e;
                if (m < M && n < N) {
                    const int v = acc[f][g][e] >> 8;
                    if (y) {
                        const float t1 = __fmul_rn((float)v, sa[m]);
                        store_out<BF16OUT>(y, (int64_t)m * ldy + n, __fmul_rn(t1, swn));
                    }
                    if (acc_out) acc_out[(int64_t)m * N + n] = v;
                }
            }
        }
    }
}


// ---------------------------------------------------------------------------
// Small-M kernel (M < 1024: one image's pruned sequence): the same 128 x 128
// tile as k_w4a4_gemm, computed by 8 wavefronts in two K-slices.  At these M
// there are only 1-2 tiles per CU; two slices put two wavefronts of the tile
// on every SIMD, so one's LDS reads, unpacking and barrier waits overlap the
// other's MFMAs, with no partial sums leaving the chip: slice 1 hands its
// accumulators to slice 0 through LDS at the end.
//  * Stage = 256 k (two 64-byte halves of a 128-byte LDS row per operand
//    row; slice s reads half s).  16-byte chunk c of row r sits at chunk
//    c ^ ((r >> 1) & 7): the 16 rows of one fragment read hit distinct banks.
//  * Global -> registers -> LDS double buffering, as k_w4a4_gemm.
// ---------------------------------------------------------------------------
constexpr int KS_THREADS = 512;
constexpr int KS_ROW = 128;                 // LDS row bytes (256 k)
constexpr int KS_STAGE = 2 * BM * KS_ROW;   // A and W: 32 KB

__device__ __forceinline__ int ks_off(int row, int c) {
    return row * KS_ROW + ((c ^ ((row >> 1) & 7)) << 4);
}

// SPLIT: blockIdx.z covers k-tiles [z kps, (z + 1) kps) and the block
// writes its exact partial sums to part[z][M][N] (int32) instead of y; a
// second kernel adds the partials and applies the epilogue.
template <bool BF16OUT, bool SPLIT>
__global__ __launch_bounds__(KS_THREADS, 2) void k_w4a4_gemm_ks(
    const uint8_t *__restrict__ A, const float *__restrict__ sa, const uint8_t *__restrict__ W,
    const float *__restrict__ sw, int M, int N, int Kb, void *__restrict__ y, int64_t ldy,
    int32_t *__restrict__ acc_out, int kps, int32_t *__restrict__ part) {
    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * KS_STAGE];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int slice = wave >> 2, wm = (wave >> 1) & 1, wn = wave & 1;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int kt_all = (Kb + KS_ROW - 1) / KS_ROW;
    const int kt0 = SPLIT ? (int)blockIdx.z * kps : 0;
    const int ktiles = SPLIT ? min(kps, kt_all - kt0) : kt_all;

    // staging: per operand 128 rows x 8 chunks = 1024 chunks, 2 per thread
    int lrow[2], lc[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int q = t + KS_THREADS * i;
        lrow[i] = q >> 3;
        lc[i] = q & 7;
    }
    uint4 ra[2], rb[2];
    auto gload = [&](int kt) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int kbyte = (kt0 + kt) * KS_ROW + lc[i] * 16;
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
        uint8_t *sA = smem + st * KS_STAGE, *sB = sA + BM * KS_ROW;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            *reinterpret_cast<uint4 *>(sA + ks_off(lrow[i], lc[i])) = ra[i];
            *reinterpret_cast<uint4 *>(sB + ks_off(lrow[i], lc[i])) = rb[i];
        }
    };

    v4i acc[4][4];
#pragma unroll
    for (int f = 0; f < 4; ++f)
#pragma unroll
        for (int g = 0; g < 4; ++g) acc[f][g] = v4i{0, 0, 0, 0};

    if (ktiles > 0) gload(0);
    sstore(0);
    __syncthreads();
    const int c = 4 * slice + (lane >> 4);       // this lane's chunk of a row
    for (int kt = 0; kt < ktiles; ++kt) {
        const int st = kt & 1;
        if (kt + 1 < ktiles) gload(kt + 1);
        const uint8_t *sA = smem + st * KS_STAGE, *sB = sA + BM * KS_ROW;
        v4i a0[4], a1[4], b0[4], b1[4];
#pragma unroll
        for (int f = 0; f < 4; ++f) {
            const int ar = wm * 64 + f * 16 + (lane & 15);
            const uint4 pa = *reinterpret_cast<const uint4 *>(sA + ks_off(ar, c));
            a0[f] = v4i{(int)nib_lo(pa.x), (int)nib_hi(pa.x), (int)nib_lo(pa.y), (int)nib_hi(pa.y)};
            a1[f] = v4i{(int)nib_lo(pa.z), (int)nib_hi(pa.z), (int)nib_lo(pa.w), (int)nib_hi(pa.w)};
            const int br = wn * 64 + f * 16 + (lane & 15);
            const uint4 pb = *reinterpret_cast<const uint4 *>(sB + ks_off(br, c));
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

    // slice 1 -> LDS ([wave][register][lane], 16 KB per wavefront), slice 0 adds
    int32_t *red = reinterpret_cast<int32_t *>(smem) + (wave & 3) * (64 * 64);
    if (slice == 1) {
#pragma unroll
        for (int f = 0; f < 4; ++f)
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int e = 0; e < 4; ++e) red[((f * 4 + g) * 4 + e) * 64 + lane] = acc[f][g][e];
    }
    __syncthreads();
    if (slice == 1) return;
#pragma unroll
    for (int f = 0; f < 4; ++f)
#pragma unroll
        for (int g = 0; g < 4; ++g)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[f][g][e] += red[((f * 4 + g) * 4 + e) * 64 + lane];

    // epilogue: lane holds rows 4*(lane>>4)+e, column lane&15 of each 16x16 tile
    if constexpr (SPLIT) {
        int32_t *pz = part + (int64_t)blockIdx.z * M * N;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int n = n0 + wn * 64 + g * 16 + (lane & 15);
#pragma unroll
            for (int f = 0; f < 4; ++f)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int m = m0 + wm * 64 + f * 16 + 4 * (lane >> 4) + e;
                    if (m < M && n < N) pz[(int64_t)m * N + n] = acc[f][g][e] >> 8;
                }
        }
        return;
    }
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

// sum of the S partial accumulators (exact integers), then the epilogue of
// the unsplit kernels; 4 consecutive outputs per thread (N % 4 == 0)
template <bool BF16OUT>
__global__ __launch_bounds__(256) void k_splitk_epilogue(const int32_t *__restrict__ part, int S,
                                                         int M, int N, const float *__restrict__ sa,
                                                         const float *__restrict__ sw,
                                                         void *__restrict__ y, int64_t ldy,
                                                         int32_t *__restrict__ acc_out) {
    const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t total = (int64_t)M * N / 4;
    if (q >= total) return;
    const int64_t o = 4 * q;
    const int m = (int)(o / N), n = (int)(o % N);
    int4 v = *reinterpret_cast<const int4 *>(part + o);
    for (int z = 1; z < S; ++z) {
        const int4 p = *reinterpret_cast<const int4 *>(part + (int64_t)z * M * N + o);
        v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
    }
    const int vv[4] = {v.x, v.y, v.z, v.w};
    const float sam = sa[m];
#pragma unroll
    for (int e = 0; e < 4; ++e)
        store_out<BF16OUT>(y, (int64_t)m * ldy + n + e, __fmul_rn(__fmul_rn((float)vv[e], sam), sw[n + e]));
    if (acc_out) {
#pragma unroll
        for (int e = 0; e < 4; ++e) acc_out[o + e] = vv[e];
    }
}

// ---------------------------------------------------------------------------
// Two-blocks-per-CU kernel: BMT (m) x 128 (n) block tile, BMT = 256 for the
// large shapes and 128 for one image's pruned sequence; 4 wavefronts of
// BMT/2 x 64 (4 x BMT/32 tiles of v_mfma_i32_16x16x64_i8: 128 or 64
// accumulator registers), and at most 256 registers per lane, so TWO blocks
// are resident per CU: one wavefront of each block on every SIMD.  While one block waits on its
// operand DMA, its LDS reads or its epilogue, the other block's wavefront
// keeps the SIMD's matrix unit busy.
//  * Packed int4 tiles go straight from HBM to LDS (buffer_load ... lds): no
//    staging registers and no LDS store instructions.  Out-of-range rows and
//    k-chunks are zero-filled by the buffer's range check.  A ring of 3 LDS
//    stages (24 or 16 KB each) keeps 2 k-tiles in flight; waits are
//    explicit (vmcnt + a bare s_barrier).
//  * After the LDS read each wave unpacks its fragments to int8 in registers.
//  * The weight fragment is the MFMA's first operand: lane l then owns four
//    consecutive output columns n of one row m.
//  * Epilogue: the dequantized tile is assembled in LDS and leaves as full
//    256-byte row segments, one 16-byte store per lane, with no waits between
//    stores.  The block's scales were fetched into LDS with the first stage.
//  * Work-group ids are remapped so that each XCD (ids are dealt round-robin
//    over 8 XCDs) walks a contiguous, M-grouped range of tiles, sharing A and
//    W panels in its own L2.
//  * SPLIT: work-group (tile, z) covers only k-tiles [z kps, (z + 1) kps) of
//    its tile and stores its exact int32 partial sums to part[z][M][N];
//    k_splitk_epilogue adds the slices and applies the epilogue.  For the
//    narrow batch-1 launches, whose tiles alone would leave most CUs idle.
// ---------------------------------------------------------------------------
constexpr int L_BM = 256, L_BN = 128;
// Ring depth: 3 stages (24 KB for 256-row tiles, 16 KB for 128-row tiles,
// so that three 128-row blocks fit on a CU).  Measured at the batch-1
// shapes: a fourth stage (two blocks per CU) or a fifth (one) made the
// launches 10-50% slower; the kernel is written for any depth up to 5.
constexpr int kMidStages = 3;
template <int BMT> constexpr int l_stages() { return BMT == 256 ? 3 : kMidStages; }
template <int BMT> constexpr int l_stage() { return (BMT + L_BN) * BKB; }   // packed codes
template <int BMT> constexpr int l_scale_off() { return l_stages<BMT>() * l_stage<BMT>(); }
constexpr int kXcds = 8;
constexpr int kGroupM = 8;

typedef __attribute__((address_space(3))) void *lds_ptr_t;

// Buffer descriptor of a raw byte range (stride 0, range-checked: loads past
// `bytes` return zeros).
__device__ __forceinline__ v4i buffer_desc(const void *base, uint32_t bytes) {
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    return v4i{(int)(uint32_t)b, (int)((b >> 32) & 0xFFFFu), (int)bytes, 0x00020000};
}

// 16 (or 4) bytes per lane from a buffer straight into LDS at lds + 16 *
// lane (4 * lane).  Issued as inline asm so the compiler does not add its
// conservative vmcnt(0) before every LDS read (it cannot tell the ring slots
// apart); the kernel waits with explicit vmcnt counts instead.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(v4i desc, uint32_t voffset, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                 :
                 : "v"(voffset), "s"(desc), "s"(lds_addr)
                 : "memory", "m0");
}
__device__ __forceinline__ void dma4(v4i desc, uint32_t voffset, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dword %0, %1, 0 offen lds"
                 :
                 : "v"(voffset), "s"(desc), "s"(lds_addr)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ uint32_t lds_addr(const void *p) {
    return (uint32_t)(size_t)(lds_ptr_t)p;
}

// Work-group id -> logical index such that the ids of one XCD (dealt
// round-robin) form a contiguous range of [0, total).
__device__ __forceinline__ int xcd_logical(int wg, int total) {
    const int q = total / kXcds, r = total % kXcds;
    const int x = wg % kXcds, i = wg / kXcds;
    return (x < r) ? x * (q + 1) + i : r * (q + 1) + (x - r) * q + i;
}

// logical index -> tile, walking groups of kGroupM tile rows column by column
__device__ __forceinline__ void grouped_tile(int logical, int tiles_m, int tiles_n, int &tm,
                                             int &tn) {
    const int per_group = kGroupM * tiles_n;
    const int g = logical / per_group;
    const int first_m = g * kGroupM;
    const int gsize = min(tiles_m - first_m, kGroupM);
    const int in_g = logical - g * per_group;
    tm = first_m + in_g % gsize;
    tn = in_g / gsize;
}

// Gram mode (M == N, A == W): only tiles holding an entry on or above the
// diagonal, i.e. tn >= 2 tm for 256 x 128 tiles; row tm of tiles holds
// tiles_n - 2 tm of them.  Same XCD-contiguous dealing as xcd_logical.
__device__ __forceinline__ void gram_tile_coords(int wg, int total, int tiles_n, int &tm, int &tn) {
    const int q = total / kXcds, r = total % kXcds;
    const int x = wg % kXcds, i = wg / kXcds;
    int logical = (x < r) ? x * (q + 1) + i : r * (q + 1) + (x - r) * q + i;
    tm = 0;
    while (true) {
        const int c = max(0, tiles_n - 2 * tm);
        if (logical < c) break;
        logical -= c;
        ++tm;
    }
    tn = 2 * tm + logical;
}

// Two adjacent packed words: the low nibbles of both move up by one 64-bit
// shift (bits crossing from w0 into w1 land in w1's low nibbles, which the
// mask clears), so the pair takes 5 VALU instructions instead of 6.
__device__ __forceinline__ v4i unpack2(uint32_t w0, uint32_t w1) {
    const uint64_t q0 = ((uint64_t)w1 << 32) | w0;
    uint64_t q;
    asm("v_lshlrev_b64 %0, 4, %1" : "=v"(q) : "v"(q0));
    return v4i{(int)((uint32_t)q & 0xF0F0F0F0u), (int)nib_hi(w0),
               (int)((uint32_t)(q >> 32) & 0xF0F0F0F0u), (int)nib_hi(w1)};
}

// YOUT = false is the Gram mode (A == W, M == N): only the int32
// accumulators are stored (acc_out, row stride N), no scales are read and no
// y is written; only tiles reaching the diagonal or above run (tiles_m then
// holds their count), each entry m < n is stored at [m][n] and at [n][m];
// blockIdx.y selects one problem of a batch (A, W, acc_out advanced by their
// strides).
template <int BMT, bool BF16OUT, bool ACC, bool YOUT, bool SPLIT>
__global__ __launch_bounds__(256, BMT == 64 ? 4 : 2) void k_w4a4_gemm_2cu(const uint8_t *__restrict__ A,
                                                          const float *__restrict__ sa,
                                                          const uint8_t *__restrict__ W,
                                                          const float *__restrict__ sw, int M,
                                                          int N, int Kb, void *__restrict__ y,
                                                          int64_t ldy,
                                                          int32_t *__restrict__ acc_out,
                                                          int tiles_m, int tiles_n,
                                                          int64_t a_bstride, int64_t w_bstride,
                                                          int64_t acc_bstride, int kps,
                                                          int32_t *__restrict__ part, int tdp,
                                                          int nsplit,
                                                          uint32_t *__restrict__ arrivals) {
    static_assert(BMT == 256 || ((BMT == 128 || BMT == 64) && YOUT), "tile height");
    static_assert(!SPLIT || YOUT, "split-K is a mode of the y-output kernel");
    constexpr int L_STAGE = l_stage<BMT>();
    constexpr int AI = BMT / 64;          // A DMA instructions per wavefront and stage
    constexpr int AF = BMT / 32;          // A fragments (16 rows) per wavefront
    __shared__ __attribute__((aligned(1024))) uint8_t smem[l_scale_off<BMT>() + (BMT + L_BN) * 4];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    if constexpr (!SPLIT) {               // Gram mode: blockIdx.y selects the problem
        A += blockIdx.y * a_bstride;
        W += blockIdx.y * w_bstride;
        if constexpr (ACC) acc_out += blockIdx.y * acc_bstride;
    }
    const int wm = wave >> 1, wn = wave & 1;
    int tm, tn, split = 0, rslot = 0;
    bool slice = false;                   // SPLIT: this block covers one k-range of a tile
    if constexpr (YOUT) {
        const int T = tiles_m * tiles_n;
        int logical;
        if constexpr (SPLIT) {
            const int b = (int)blockIdx.x;
            if (b < tdp) {
                logical = xcd_logical(b, tdp);
            } else {
                slice = true;
                rslot = (b - tdp) / nsplit;
                split = b - tdp - rslot * nsplit;
                logical = tdp + rslot;
            }
        } else {
            logical = xcd_logical((int)blockIdx.x, T);
        }
        grouped_tile(logical, tiles_m, tiles_n, tm, tn);
    } else {
        gram_tile_coords(blockIdx.x, tiles_m, tiles_n, tm, tn);
    }
    const int m0 = tm * BMT, n0 = tn * L_BN;
    // this block's k-tiles [kbeg, kbeg + ktiles); the launch makes every split non-empty
    const int ktiles_all = (Kb + BKB - 1) / BKB;
    const int kbeg = slice ? split * kps : 0;
    const int ktiles = slice ? min(ktiles_all - kbeg, kps) : ktiles_all;

    const v4i dA = buffer_desc(A + (int64_t)m0 * Kb, (uint32_t)(min(M - m0, BMT) * Kb));
    const v4i dW = buffer_desc(W + (int64_t)n0 * Kb, (uint32_t)(min(N - n0, L_BN) * Kb));

    // DMA: one 1 KB instruction fills 16 rows of 64 bytes; lane L -> row
    // +L/4, slot L%4, which holds k-chunk (L%4) ^ ((row >> 1) & 3).  Wave w
    // copies A rows [w BMT/4, (w + 1) BMT/4) (AI instructions) and W rows
    // [32w, 32w+32) (2 instructions).
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    uint32_t voffA[AI], voffW[2];
    int kcA[AI], kcW[2];
#pragma unroll
    for (int i = 0; i < AI; ++i) {
        const int row = (BMT / 4) * wave + 16 * i + (lane >> 2);
        kcA[i] = ((lane & 3) ^ ((row >> 1) & 3)) * 16;
        voffA[i] = (uint32_t)(row * Kb + kcA[i]);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int row = 32 * wave + 16 * i + (lane >> 2);
        kcW[i] = ((lane & 3) ^ ((row >> 1) & 3)) * 16;
        voffW[i] = (uint32_t)(row * Kb + kcW[i]);
    }
    const uint32_t ldsA = lds_addr(smem) + wave_u * (BMT / 4) * BKB;
    const uint32_t ldsW = lds_addr(smem) + BMT * BKB + wave_u * 2048;
    auto issue = [&](int slot, int kt) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < AI; ++i) {
            const uint32_t o = (kt * BKB + kcA[i] < Kb) ? voffA[i] + (uint32_t)(kt * BKB) : 0x80000000u;
            dma16(dA, o, ldsA + slot * L_STAGE + i * 1024);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const uint32_t o = (kt * BKB + kcW[i] < Kb) ? voffW[i] + (uint32_t)(kt * BKB) : 0x80000000u;
            dma16(dW, o, ldsW + slot * L_STAGE + i * 1024);
        }
    };

    if constexpr (YOUT) {             // the block's scales -> LDS (zeros past M / N), ahead of the stages
        const v4i dSa = buffer_desc(sa + m0, (uint32_t)(min(M - m0, BMT) * 4));
        const v4i dSw = buffer_desc(sw + n0, (uint32_t)(min(N - n0, L_BN) * 4));
        const uint32_t sbase = lds_addr(smem) + l_scale_off<BMT>();
        if constexpr (BMT == 256) {
            dma4(dSa, (uint32_t)(64 * wave + lane) * 4u, sbase + wave_u * 256);
            if (wave_u < 2) dma4(dSw, (uint32_t)(64 * wave + lane) * 4u, sbase + 1024 + wave_u * 256);
        } else if constexpr (BMT == 128) {   // 128 + 128 scales: waves 0, 1 and 2, 3
            if (wave_u < 2) dma4(dSa, (uint32_t)(64 * wave + lane) * 4u, sbase + wave_u * 256);
            else dma4(dSw, (uint32_t)(64 * (wave - 2) + lane) * 4u, sbase + 512 + (wave_u - 2) * 256);
        } else {                             // 64 + 128 scales: wave 0 and waves 1, 2
            if (wave_u == 0) dma4(dSa, (uint32_t)lane * 4u, sbase);
            else if (wave_u < 3) dma4(dSw, (uint32_t)(64 * (wave - 1) + lane) * 4u, sbase + 256 + (wave_u - 1) * 256);
        }
    }
    constexpr int NST = l_stages<BMT>();
#pragma unroll
    for (int q = 0; q < NST - 1; ++q)
        if (q < ktiles) issue(q, kbeg + q);

    v4i acc[4][AF];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < AF; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    // Fragments: W f = 0..3 (rows wn*64 + 16f), A f = 4..3+AF (rows
    // wm*BMT/2 + 16(f-4)).  Lane l reads row l%16, chunk l/16 (32 k values;
    // words x,y feed k-step 0 and z,w k-step 1 -- the same placement for A
    // and W, so every k meets its partner exactly once).
    const int r16 = lane & 15, cq = lane >> 4;
    const uint32_t cofs = (uint32_t)((cq ^ ((r16 >> 1) & 3)) << 4);
    const uint32_t fW = BMT * BKB + (wn * 64 + r16) * BKB + cofs;
    const uint32_t fA = (wm * (BMT / 2) + r16) * BKB + cofs;
    constexpr int NF = 4 + AF;
    uint4 P[NF];
    auto read_tile = [&](int slot) __attribute__((always_inline)) {
        const uint8_t *b = smem + slot * L_STAGE;
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const uint32_t o = (f < 4) ? fW + f * 1024 : fA + (f - 4) * 1024;
            P[f] = *reinterpret_cast<const uint4 *>(b + o);
        }
    };
    auto operands = [&](int s, v4i *u) __attribute__((always_inline)) {
#pragma unroll
        for (int f = 0; f < NF; ++f) u[f] = s ? unpack2(P[f].z, P[f].w) : unpack2(P[f].x, P[f].y);
    };
    auto mfma_step = [&](const v4i *u) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < AF; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(u[i], u[4 + j], acc[i][j], 0, 0, 0);
    };

    v4i u0[NF], u1[NF];
    for (int kt = 0; kt < ktiles; ++kt) {
        // tile kt has landed (from every wave) and every wave is done with
        // tile kt-1, whose slot the DMA of tile kt+NST-1 now overwrites.  Each
        // wave issues AI + 2 DMA instructions per tile; the tiles after kt
        // already issued may stay in flight.
        const int ahead = min(NST - 2, ktiles - 1 - kt);
        if constexpr (BMT == 256) {
            if (ahead >= 1) asm volatile("s_waitcnt vmcnt(6)\n\ts_barrier" ::: "memory");
            else asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
        } else if constexpr (BMT == 128) {
            static_assert(l_stages<BMT>() <= 5, "wait counts below cover at most 3 tiles ahead");
            if (ahead >= 3) asm volatile("s_waitcnt vmcnt(12)\n\ts_barrier" ::: "memory");
            else if (ahead == 2) asm volatile("s_waitcnt vmcnt(8)\n\ts_barrier" ::: "memory");
            else if (ahead == 1) asm volatile("s_waitcnt vmcnt(4)\n\ts_barrier" ::: "memory");
            else asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
        } else {                                  // BMT = 64: 3 instructions per tile
            static_assert(l_stages<BMT>() <= 5, "wait counts below cover at most 3 tiles ahead");
            if (ahead >= 3) asm volatile("s_waitcnt vmcnt(9)\n\ts_barrier" ::: "memory");
            else if (ahead == 2) asm volatile("s_waitcnt vmcnt(6)\n\ts_barrier" ::: "memory");
            else if (ahead == 1) asm volatile("s_waitcnt vmcnt(3)\n\ts_barrier" ::: "memory");
            else asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
        }
        if (kt + NST - 1 < ktiles) issue((kt + NST - 1) % NST, kbeg + kt + NST - 1);
        read_tile(kt % NST);
        operands(0, u0);
        __builtin_amdgcn_sched_barrier(0);
        // raised issue priority while this wave streams MFMAs, so the SIMD's
        // arbiter keeps the matrix unit fed and the other block's wave fills
        // the gaps with its DMA, LDS and unpack work
        __builtin_amdgcn_s_setprio(1);
        operands(1, u1);
        mfma_step(u0);
#pragma unroll
        for (int i = 0; i < 2 * NF; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // 1 MFMA
            __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);   // 3 VALU
        }
        __builtin_amdgcn_sched_barrier(0);
        mfma_step(u1);
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(0);
    }

    if constexpr (SPLIT) {
        // A slice block stores its raw accumulators (256 x the exact partial
        // sums; each store instruction covers 256 consecutive bytes) to its
        // own slot of the workspace and
        // counts itself in on the tile's arrival counter; the block that
        // arrives last adds the other slices' sums to its own and goes on to
        // the epilogue, and puts the counter back to zero, so the counters
        // are zero again after every call.  The partial sums move as
        // agent-scope (device-coherent) atomic stores and loads, and every
        // store has completed (vmcnt(0)) before the block counts itself in,
        // so no L2 write-back or invalidation of the whole cache is needed
        // (agent-scope fences cost this launch more than twice its time).
        if (slice) {
            __shared__ int s_last;
            constexpr int SLICE_V4 = 32 * BMT;              // v4i per slice (BMT x 128 int32)
            int32_t *const rp = part + (int64_t)rslot * nsplit * SLICE_V4 * 4;
            int32_t *const mine = rp + (int64_t)split * SLICE_V4 * 4;
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < AF; ++j)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        __hip_atomic_store(mine + ((((wave * 4 + i) * AF + j) * 4 + e) << 6) + lane,
                                           acc[i][j][e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
            if (t == 0) {
                const uint32_t before = __hip_atomic_fetch_add(arrivals + rslot, 1u, __ATOMIC_RELAXED,
                                                               __HIP_MEMORY_SCOPE_AGENT);
                s_last = (before == (uint32_t)(nsplit - 1));
                if (s_last) __hip_atomic_store(arrivals + rslot, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            __syncthreads();
            if (!s_last) return;
            for (int z = 0; z < nsplit; ++z) {
                if (z == split) continue;
                const int32_t *src = rp + (int64_t)z * SLICE_V4 * 4;
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < AF; ++j)
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            acc[i][j][e] += __hip_atomic_load(
                                src + ((((wave * 4 + i) * AF + j) * 4 + e) << 6) + lane, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    }

    if constexpr (!YOUT) {      // Gram mode: int32 accumulators only
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int nb = n0 + wn * 64 + 16 * i + 4 * cq;
#pragma unroll
            for (int j = 0; j < AF; ++j) {
                const int m = m0 + wm * (BMT / 2) + 16 * j + r16;
                if (m < M) {
                    int v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = acc[i][j][e] >> 8;
                    int32_t *dst = acc_out + (int64_t)m * N + nb;
                    if (nb + 3 < N && (N & 3) == 0) {
                        *reinterpret_cast<int4 *>(dst) = make_int4(v[0], v[1], v[2], v[3]);
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (nb + e < N) dst[e] = v[e];
                    }
                    // mirror of the strictly upper entries: 16 lanes write 64
                    // contiguous bytes of row nb + e
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (m < nb + e && nb + e < N) acc_out[(int64_t)(nb + e) * N + m] = v[e];
                }
            }
        }
        return;
    }

    // Epilogue.  acc[i][j] lane l, register e holds
    //   n = n0 + wn*64 + 16 i + 4 (l/16) + e,  m = m0 + wm*BMT/2 + 16 j + l%16.
    // The BMT x 128 tile is assembled in LDS: row m of 256 bytes, 8-byte unit
    // u (4 columns) stored at unit u ^ 2 (m & 15), which keeps both the
    // 8-byte writes and the 16-byte row reads free of bank conflicts.
    __syncthreads();
    // int32 rows 16-byte aligned: N % 4 == 0 and an aligned base
    const bool acc_vec = ACC && (N & 3) == 0 && ((reinterpret_cast<uintptr_t>(acc_out) & 15) == 0);
    const float *s_sa = reinterpret_cast<const float *>(smem + l_scale_off<BMT>());
    const float *s_sw = s_sa + BMT;
    float sam[AF];
#pragma unroll
    for (int j = 0; j < AF; ++j) sam[j] = s_sa[wm * (BMT / 2) + 16 * j + r16];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int nl = wn * 64 + 16 * i + 4 * cq;
        const float4 swv = *reinterpret_cast<const float4 *>(s_sw + nl);
        const float swe[4] = {swv.x, swv.y, swv.z, swv.w};
#pragma unroll
        for (int j = 0; j < AF; ++j) {
            int v[4];
            float o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[e] = acc[i][j][e] >> 8;
                o[e] = __fmul_rn(__fmul_rn((float)v[e], sam[j]), swe[e]);
            }
            uint2 packed;
            if constexpr (BF16OUT) {
                // v_cvt_pk_bf16_f32: two fp32 -> bf16, round to nearest even
                packed.x = __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{o[0], o[1]}, bf2));
                packed.y = __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{o[2], o[3]}, bf2));
            } else {
                uint32_t h[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float ov = o[e];
                    asm volatile("" : "+v"(ov));
                    h[e] = __builtin_bit_cast(uint16_t, (_Float16)ov);
                }
                packed = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
            }
            const int r = wm * (BMT / 2) + 16 * j + r16;
            const int u = (nl >> 2) ^ (r16 << 1);
            *reinterpret_cast<uint2 *>(smem + r * 256 + u * 8) = packed;
            if constexpr (ACC) {
                const int m = m0 + r, nb = n0 + nl;
                if (m < M) {
                    int32_t *dst = acc_out + (int64_t)m * N + nb;
                    if (acc_vec && nb + 3 < N) {      // the lane's 4 columns as one 16-byte store
                        *reinterpret_cast<v4i *>(dst) = v4i{v[0], v[1], v[2], v[3]};
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (nb + e < N) dst[e] = v[e];
                    }
                }
            }
        }
    }
    __syncthreads();
    const int rows_left = M - m0, cols_left = N - n0;
    const bool vec16 = ((ldy & 7) == 0) && ((reinterpret_cast<uintptr_t>(y) & 15) == 0);
    const bool full = vec16 && rows_left >= BMT && cols_left >= L_BN;
    const int cch = lane & 15;
    uint16_t *yb = static_cast<uint16_t *>(y) + (int64_t)m0 * ldy + n0 + 8 * cch;
#pragma unroll 4
    for (int i = 0; i < BMT / 16; ++i) {
        const int r = (BMT / 4) * wave + 4 * i + (lane >> 4);
        const uint4 val = *reinterpret_cast<const uint4 *>(smem + r * 256 + ((cch ^ (r & 15)) << 4));
        uint16_t *dst = yb + (int64_t)r * ldy;
        if (full) {
            *reinterpret_cast<uint4 *>(dst) = val;
        } else if (r < rows_left) {
            if (vec16 && 8 * cch + 8 <= cols_left) {
                *reinterpret_cast<uint4 *>(dst) = val;
            } else {
                const uint32_t w4[4] = {val.x, val.y, val.z, val.w};
#pragma unroll
                for (int jj = 0; jj < 8; ++jj)
                    if (8 * cch + jj < cols_left) dst[jj] = (uint16_t)(w4[jj >> 1] >> (16 * (jj & 1)));
            }
        }
    }
}


// ---------------------------------------------------------------------------
// Persistent-tile form of the kernel above (y output, no split): a grid of at
// most two blocks per CU, each walking a list of tiles, with one DMA ring
// running on across its tile boundaries.
//  * Tile list: the work-groups of XCD x (ids x, x + 8, ...) share that XCD's
//    contiguous range of M-grouped tiles (as in xcd_logical); the i-th of them
//    takes tiles i, i + nb, i + 2 nb, ... of the range (nb = its work-groups),
//    so at any time an XCD works on a window of consecutive tiles.
//  * The ring is indexed by the block's global k-tile count g (tile g / KT,
//    k-tile g % KT): the DMA of the next tile's first stages (and its scales,
//    into one of three scale buffers) is issued during the current tile's
//    last k-tiles, so a new tile starts with its operands in LDS instead of
//    a full memory round trip, and no block is relaunched per tile.
//  * Epilogue: one barrier, then each wavefront stages its own 128 x 64
//    sub-tile through 4 KB of the ring slot just consumed, 32 rows at a
//    time, and stores full 128-byte row segments.  No other barrier: every
//    wavefront only reads back what it wrote itself, and the slot is not
//    refilled before the barrier at the top of the next k-tile.  The stores
//    are non-temporal: outputs of these shapes (92-500 MB) do not stay in
//    the caches anyway, and dirty output lines held there cost the operand
//    reads of this and the next launch (measured: 1.5% on the layer).
//  * Waits: loads (the DMA) complete in order among themselves, so waiting
//    until at most 6 instructions (one stage of this wave) are outstanding
//    guarantees every older stage has landed; epilogue stores in between
//    can only make such a wait longer, never shorter.
// ---------------------------------------------------------------------------
constexpr int kScaleBufs = 3;

template <bool BF16OUT, bool ACC>
__global__ __launch_bounds__(256, 2) void k_w4a4_gemm_pt(const uint8_t *__restrict__ A,
                                                         const float *__restrict__ sa,
                                                         const uint8_t *__restrict__ W,
                                                         const float *__restrict__ sw, int M,
                                                         int N, int Kb, void *__restrict__ y,
                                                         int64_t ldy,
                                                         int32_t *__restrict__ acc_out,
                                                         int tiles_m, int tiles_n) {
    constexpr int BMT = L_BM, NST = 3, AI = BMT / 64, AF = BMT / 32;
    constexpr int L_STAGE = l_stage<BMT>();
    constexpr int SCALE_OFF = NST * L_STAGE;
    constexpr int SCALE_BUF = (BMT + L_BN) * 4;
    __shared__ __attribute__((aligned(1024))) uint8_t smem[SCALE_OFF + kScaleBufs * SCALE_BUF];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);

    // this block's tiles: start + i0 + k nb, k < nt
    const int T = tiles_m * tiles_n;
    const int xcd = blockIdx.x % kXcds, i0 = blockIdx.x / kXcds;
    const int nb = ((int)gridDim.x - xcd + kXcds - 1) / kXcds;
    const int q = T / kXcds, rr = T % kXcds;
    const int start = (xcd < rr) ? xcd * (q + 1) : rr * (q + 1) + (xcd - rr) * q;
    const int len = q + (xcd < rr ? 1 : 0);
    const int nt = (i0 < len) ? (len - i0 + nb - 1) / nb : 0;
    const int KT = (Kb + BKB - 1) / BKB;
    const int g_end = nt * KT;
    auto tile_origin = [&](int k, int &m0, int &n0) __attribute__((always_inline)) {
        int tm, tn;
        grouped_tile(start + i0 + k * nb, tiles_m, tiles_n, tm, tn);
        m0 = tm * BMT;
        n0 = tn * L_BN;
    };

    // DMA placement: as in k_w4a4_gemm_2cu (16 rows of 64 bytes per 1 KB
    // instruction, k-chunk index XORed with (row >> 1) & 3)
    uint32_t voffA[AI], voffW[2];
    int kcA[AI], kcW[2];
#pragma unroll
    for (int i = 0; i < AI; ++i) {
        const int row = (BMT / 4) * wave + 16 * i + (lane >> 2);
        kcA[i] = ((lane & 3) ^ ((row >> 1) & 3)) * 16;
        voffA[i] = (uint32_t)(row * Kb + kcA[i]);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int row = 32 * wave + 16 * i + (lane >> 2);
        kcW[i] = ((lane & 3) ^ ((row >> 1) & 3)) * 16;
        voffW[i] = (uint32_t)(row * Kb + kcW[i]);
    }
    const uint32_t ldsA = lds_addr(smem) + wave_u * (BMT / 4) * BKB;
    const uint32_t ldsW = lds_addr(smem) + BMT * BKB + wave_u * 2048;
    const uint32_t sbase = lds_addr(smem) + SCALE_OFF;

    // issue side: the tile whose stages are being issued, its descriptors
    int iss_k = -1, iss_kt = 0;
    v4i dA, dW;
    auto issue = [&](int g) __attribute__((always_inline)) {
        if (iss_kt == 0) {                      // first stage of a new tile
            ++iss_k;
            int m0, n0;
            tile_origin(iss_k, m0, n0);
            dA = buffer_desc(A + (int64_t)m0 * Kb, (uint32_t)(min(M - m0, BMT) * Kb));
            dW = buffer_desc(W + (int64_t)n0 * Kb, (uint32_t)(min(N - n0, L_BN) * Kb));
            // the tile's scales (zeros past M / N) into scale buffer iss_k % 3
            const v4i dSa = buffer_desc(sa + m0, (uint32_t)(min(M - m0, BMT) * 4));
            const v4i dSw = buffer_desc(sw + n0, (uint32_t)(min(N - n0, L_BN) * 4));
            const uint32_t sb = sbase + (uint32_t)((iss_k % kScaleBufs) * SCALE_BUF);
            dma4(dSa, (uint32_t)(64 * wave + lane) * 4u, sb + wave_u * 256);
            if (wave_u < 2) dma4(dSw, (uint32_t)(64 * wave + lane) * 4u, sb + BMT * 4 + wave_u * 256);
        }
        const int slot = g % NST, kt = iss_kt;
#pragma unroll
        for (int i = 0; i < AI; ++i) {
            const uint32_t o = (kt * BKB + kcA[i] < Kb) ? voffA[i] + (uint32_t)(kt * BKB) : 0x80000000u;
            dma16(dA, o, ldsA + slot * L_STAGE + i * 1024);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const uint32_t o = (kt * BKB + kcW[i] < Kb) ? voffW[i] + (uint32_t)(kt * BKB) : 0x80000000u;
            dma16(dW, o, ldsW + slot * L_STAGE + i * 1024);
        }
        if (++iss_kt == KT) iss_kt = 0;
    };
#pragma unroll
    for (int g = 0; g < NST - 1; ++g)
        if (g < g_end) issue(g);

    v4i acc[4][AF];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < AF; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    const int r16 = lane & 15, cq = lane >> 4;
    const uint32_t cofs = (uint32_t)((cq ^ ((r16 >> 1) & 3)) << 4);
    const uint32_t fW = BMT * BKB + (wn * 64 + r16) * BKB + cofs;
    const uint32_t fA = (wm * (BMT / 2) + r16) * BKB + cofs;
    constexpr int NF = 4 + AF;
    uint4 P[NF];
    auto read_tile = [&](int slot) __attribute__((always_inline)) {
        const uint8_t *b = smem + slot * L_STAGE;
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const uint32_t o = (f < 4) ? fW + f * 1024 : fA + (f - 4) * 1024;
            P[f] = *reinterpret_cast<const uint4 *>(b + o);
        }
    };
    auto operands = [&](int s, v4i *u) __attribute__((always_inline)) {
#pragma unroll
        for (int f = 0; f < NF; ++f) u[f] = s ? unpack2(P[f].z, P[f].w) : unpack2(P[f].x, P[f].y);
    };
    auto mfma_step = [&](const v4i *u) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < AF; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(u[i], u[4 + j], acc[i][j], 0, 0, 0);
    };
    const bool vec16 = ((ldy & 7) == 0) && ((reinterpret_cast<uintptr_t>(y) & 15) == 0);
    const bool acc_vec = ACC && (N & 3) == 0 && ((reinterpret_cast<uintptr_t>(acc_out) & 15) == 0);

    v4i u0[NF], u1[NF];
    int ck = 0, ckt = 0;                        // compute side: tile, k-tile
    for (int g = 0; g < g_end; ++g) {
        // stage g has landed (every wave) and every wave is done with stage
        // g-1, whose slot the DMA of stage g+NST-1 now overwrites
        if (g + 1 < g_end) asm volatile("s_waitcnt vmcnt(6)\n\ts_barrier" ::: "memory");
        else asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
        if (g + NST - 1 < g_end) issue(g + NST - 1);
        read_tile(g % NST);
        operands(0, u0);
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(1);
        operands(1, u1);
        mfma_step(u0);
#pragma unroll
        for (int i = 0; i < 2 * NF; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // 1 MFMA
            __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);   // 3 VALU
        }
        __builtin_amdgcn_sched_barrier(0);
        mfma_step(u1);
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(0);

        if (++ckt < KT) continue;
        // tile ck complete: epilogue from registers, then the next tile
        ckt = 0;
        int m0, n0;
        tile_origin(ck, m0, n0);
        const float *s_sa = reinterpret_cast<const float *>(smem + SCALE_OFF + (ck % kScaleBufs) * SCALE_BUF);
        const float *s_sw = s_sa + BMT;
        // Staging: the ring slot this last k-tile was read from (the next
        // tile's two stages sit in the other slots), after one barrier that
        // lets every wave finish its reads of it.  Each wave then works on
        // its own 4 KB of the slot, no further barrier: four passes over its
        // fragment pairs j = 2p, 2p + 1 (32 rows x 64 columns of its 128 x 64
        // sub-tile) -- 8-byte units written in MFMA layout (unit index XORed
        // with 2 ((row >> 1) & 7): conflict-free), read back as 16-byte
        // chunks, stored as full 128-byte row segments.
        __syncthreads();
        // lane-derived values made opaque here, so that the epilogue's
        // address arithmetic stays in the epilogue instead of being hoisted
        // out of the k-loop into registers the loop needs
        int r16e = r16, cqe = cq, lanee = lane;
        asm volatile("" : "+v"(r16e), "+v"(cqe), "+v"(lanee));
        uint8_t *stg = smem + (g % NST) * L_STAGE + wave * 4096;
        const int rows_left = M - m0, cols_left = N - n0;
        const bool full = vec16 && rows_left >= BMT && cols_left >= L_BN;
        const int rc = lanee & 7;                           // 16-byte chunk of a row read back
#pragma unroll
        for (int pass = 0; pass < AF / 2; ++pass) {
#pragma unroll
            for (int jj = 0; jj < 2; ++jj) {
                const int j = 2 * pass + jj;
                const int rl = wm * (BMT / 2) + 16 * j + r16e;
                const float sam = s_sa[rl];
                const int rs = 16 * jj + r16e;                    // staging row (0..31)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int nl = wn * 64 + 16 * i + 4 * cqe;
                    const float4 swv = *reinterpret_cast<const float4 *>(s_sw + nl);
                    const float swe[4] = {swv.x, swv.y, swv.z, swv.w};
                    int v[4];
                    float o[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        v[e] = acc[i][j][e] >> 8;
                        o[e] = __fmul_rn(__fmul_rn((float)v[e], sam), swe[e]);
                    }
                    uint2 packed;
                    if constexpr (BF16OUT) {
                        packed.x = __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{o[0], o[1]}, bf2));
                        packed.y = __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{o[2], o[3]}, bf2));
                    } else {
                        uint32_t h[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            float ov = o[e];
                            asm volatile("" : "+v"(ov));
                            h[e] = __builtin_bit_cast(uint16_t, (_Float16)ov);
                        }
                        packed = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
                    }
                    const int u = (4 * i + cqe) ^ (2 * ((rs >> 1) & 7));
                    *reinterpret_cast<uint2 *>(stg + rs * 128 + u * 8) = packed;
                    if constexpr (ACC) {
                        const int m = m0 + rl, nb0 = n0 + nl;
                        if (m < M) {
                            int32_t *dst = acc_out + (int64_t)m * N + nb0;
                            if (acc_vec && nb0 + 3 < N) {
                                *reinterpret_cast<v4i *>(dst) = v4i{v[0], v[1], v[2], v[3]};
                            } else {
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    if (nb0 + e < N) dst[e] = v[e];
                            }
                        }
                    }
                    acc[i][j] = v4i{0, 0, 0, 0};
                }
            }
            // the wave's own 32 x 64 block back as 16-byte chunks: lane l,
            // step s reads row 8 s + l / 8, chunk l % 8 (LDS operations of one
            // wave take effect in issue order)
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                const int rs = 8 * s4 + (lanee >> 3);
                const int cu = (2 * rc) ^ (2 * ((rs >> 1) & 7));     // even: the pair stays in order
                const uint4 val = *reinterpret_cast<const uint4 *>(stg + rs * 128 + cu * 8);
                const int rt = wm * (BMT / 2) + 32 * pass + rs;        // tile row
                const int ct = wn * 64 + 8 * rc;                       // tile column
                uint16_t *dst = static_cast<uint16_t *>(y) + (int64_t)(m0 + rt) * ldy + n0 + ct;
                if (full) {
                    __builtin_nontemporal_store(__builtin_bit_cast(v4i, val), reinterpret_cast<v4i *>(dst));
                } else if (rt < rows_left) {
                    if (vec16 && ct + 8 <= cols_left) {
                        __builtin_nontemporal_store(__builtin_bit_cast(v4i, val), reinterpret_cast<v4i *>(dst));
                    } else {
                        const uint32_t w4[4] = {val.x, val.y, val.z, val.w};
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (ct + e < cols_left) dst[e] = (uint16_t)(w4[e >> 1] >> (16 * (e & 1)));
                    }
                }
            }
        }
        ++ck;
    }
}


// ---------------------------------------------------------------------------
// Decode-shaped kernel (M <= 16): the weights are streamed from HBM once, so
// the kernel is bound by HBM bandwidth and by how many bytes are in flight.
// A work-group of NW wavefronts (8, or 16 for long rows) computes 16 output
// rows (one MFMA fragment) at a time.  Work-groups are persistent: each walks row groups blockIdx.x,
// blockIdx.x + gridDim.x, ... and loads the next group's weights before
// computing on the current ones, so HBM latency overlaps with the MFMAs, the
// reduction and the epilogue.
//
// The 16 rows of a group are one contiguous block of 16 * Kb bytes.  Each
// wavefront loads 16 / NW whole rows of it, 1 KB of consecutive bytes per
// instruction, and the block passes through LDS (row stride: an odd number of
// 16-byte chunks, so the 16 rows of a fragment read fall in distinct banks)
// to reach the MFMA layout.  Loading the fragments straight from HBM would
// make every quarter-wavefront touch 16 rows with 16 bytes each.
//
// For the contraction, the NW wavefronts split K into contiguous ranges of at
// most G_BATCH 128-value k-tiles.  Per k-tile, lane (r, c) takes the 16
// bytes at [64 kt + 16 c, +16) of weight row r (from LDS) and of activation
// row r (from HBM, once per wavefront; rows past M read as zeros): both
// operands use the same k placement, so the MFMA sums every k exactly once.
// The NW partial accumulators are summed through LDS (integer sums: exact and
// order-independent) before the epilogue.
// ---------------------------------------------------------------------------
constexpr int G_ROWS = 16;
constexpr int G_MAX_KIN = 14336;            // 7 k-tiles for each of 16 wavefronts

// range-checked 16-byte load: offsets at or past the range read as zeros
__device__ __forceinline__ uint4 gbuf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2));
}

template <int G_BATCH, int NW, bool BF16OUT>
__global__ __launch_bounds__(64 * NW) void k_w4a4_gemv(const uint8_t *__restrict__ A,
                                                            const float *__restrict__ sa,
                                                            const uint8_t *__restrict__ W,
                                                            const float *__restrict__ sw, int M,
                                                            int N, int Kb, void *__restrict__ y,
                                                            int64_t ldy,
                                                            int32_t *__restrict__ acc_out) {
    // Kb <= 64 NW G_BATCH, so a row holds at most 4 NW G_BATCH chunks of 16 bytes
    __shared__ uint4 stage[G_ROWS * (4 * NW * G_BATCH + 1)];
    __shared__ v4i red[NW][64];
    constexpr int RPW = G_ROWS / NW;                        // rows staged per wavefront
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r = lane & 15, c = lane >> 4;
    const int ktiles = (Kb + 63) / 64;
    const int kt0 = (int)((int64_t)ktiles * wave / NW);
    const int nk = (int)((int64_t)ktiles * (wave + 1) / NW) - kt0;   // <= G_BATCH
    const int groups = (N + G_ROWS - 1) / G_ROWS;
    const int kc = Kb >> 4;                                 // 16-byte chunks per row
    const int rs = kc | 1;                                  // LDS row stride in chunks (odd)

    // whole-matrix descriptors: rows past N or M fall outside the ranges and
    // read as zero
    const __amdgpu_buffer_rsrc_t dW =
        __builtin_amdgcn_make_buffer_rsrc((void *)W, 0, (int)min((int64_t)N * Kb, (int64_t)0x7FFFFFFF), 0x00020000);
    const __amdgpu_buffer_rsrc_t dA =
        __builtin_amdgcn_make_buffer_rsrc((void *)A, 0, M * Kb, 0x00020000);
    const uint32_t off = (uint32_t)(r * Kb + 16 * c + 64 * kt0);
    uint32_t kin = 0;                                       // bit u: k-tile kt0+u in range
#pragma unroll
    for (int u = 0; u < G_BATCH; ++u)
        if (u < nk && 64 * (kt0 + u) + 16 * c < Kb) kin |= 1u << u;

    // staging: chunk f = 64 u + lane of this wavefront's rows RPW wave, ...,
    // RPW wave + RPW - 1 (bit u of sin: f < RPW kc); its LDS slot skips the
    // padding
    uint32_t sin = 0;
#pragma unroll
    for (int u = 0; u < G_BATCH; ++u)
        if (64 * u + lane < RPW * kc) sin |= 1u << u;
    const uint32_t soff = (uint32_t)(RPW * wave * Kb + 16 * lane);
    auto load_w = [&](int g, uint4 *w) {
        const uint32_t base = (uint32_t)(g * G_ROWS) * (uint32_t)Kb + soff;
#pragma unroll
        for (int u = 0; u < G_BATCH; ++u)
            w[u] = gbuf_load16(dW, ((sin >> u) & 1) ? base + 1024 * u : 0x80000000u);
    };
    auto unpack = [](uint32_t w0, uint32_t w1) {
        return v4i{(int)nib_lo(w0), (int)nib_hi(w0), (int)nib_lo(w1), (int)nib_hi(w1)};
    };

    // this wavefront's activation fragments (packed), loaded once for all groups
    uint4 a[G_BATCH];
#pragma unroll
    for (int u = 0; u < G_BATCH; ++u)
        a[u] = gbuf_load16(dA, ((kin >> u) & 1) ? off + 64 * u : 0x80000000u);

    // epilogue operands: lane l serves m = l & 15 and n = 16 g + 4 (l >> 4) + e
    const int m = lane & 15;
    const float sam = (m < M) ? sa[m] : 0.0f;
    const __amdgpu_buffer_rsrc_t dS = __builtin_amdgcn_make_buffer_rsrc((void *)sw, 0, N * 4, 0x00020000);
    auto load_sw = [&](int g) {
        return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(
                                              dS, (uint32_t)(g * G_ROWS + 4 * (lane >> 4)) * 4u, 0, 0));
    };

    // 4 consecutive outputs per lane go out as one 8-byte store when aligned
    const bool vec_y = ((reinterpret_cast<uintptr_t>(y) & 7) == 0) && ((ldy & 3) == 0);
    const bool vec_acc = ((reinterpret_cast<uintptr_t>(acc_out) & 15) == 0) && ((N & 3) == 0);

    int g = blockIdx.x;
    uint4 wc[G_BATCH];
    float4 swc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (g < groups) {
        load_w(g, wc);
        swc = load_sw(g);
    }
    for (; g < groups; g += gridDim.x) {
        // the previous group's fragment reads ended at its reduction barrier
#pragma unroll
        for (int u = 0; u < G_BATCH; ++u) {
            if ((sin >> u) & 1) {
                const int f = 64 * u + lane;
                stage[RPW * wave * rs + f + (RPW > 1 && f >= kc ? rs - kc : 0)] = wc[u];
            }
        }
        // with the block in LDS its registers take the next group's loads
        const float4 sws = swc;
        const int gn = g + gridDim.x;
        if (gn < groups) {
            load_w(gn, wc);
            swc = load_sw(gn);
        }
        __syncthreads();
        v4i acc = v4i{0, 0, 0, 0};
#pragma unroll
        for (int u = 0; u < G_BATCH; ++u) {
            const uint4 wf = ((kin >> u) & 1) ? stage[r * rs + 4 * (kt0 + u) + c]
                                              : make_uint4(0u, 0u, 0u, 0u);
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(unpack(wf.x, wf.y),
                                                        unpack(a[u].x, a[u].y), acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(unpack(wf.z, wf.w),
                                                        unpack(a[u].z, a[u].w), acc, 0, 0, 0);
        }
        red[wave][lane] = acc;
        __syncthreads();
        // wave 0 reads red before it reaches the next group's first barrier,
        // and no wavefront writes red again before that barrier
        if (wave == 0) {
            v4i s = red[0][lane];
#pragma unroll
            for (int w = 1; w < NW; ++w) s += red[w][lane];
            const int nb = g * G_ROWS + 4 * (lane >> 4);
            const float swv[4] = {sws.x, sws.y, sws.z, sws.w};
            if (m < M) {
                if (vec_y && nb + 3 < N) {                   // one 8-byte store per lane
                    uint32_t h[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        h[e] = out_bits<BF16OUT>(__fmul_rn(__fmul_rn((float)(s[e] >> 8), sam), swv[e]));
                    *reinterpret_cast<uint2 *>(static_cast<uint16_t *>(y) + (int64_t)m * ldy + nb) =
                        make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
                    if (acc_out) {
                        if (vec_acc)
                            *reinterpret_cast<v4i *>(acc_out + (int64_t)m * N + nb) =
                                v4i{s[0] >> 8, s[1] >> 8, s[2] >> 8, s[3] >> 8};
                        else
                            for (int e = 0; e < 4; ++e) acc_out[(int64_t)m * N + nb + e] = s[e] >> 8;
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int n = nb + e;
                        if (n < N) {
                            const int v = s[e] >> 8;
                            store_out<BF16OUT>(y, (int64_t)m * ldy + n,
                                               __fmul_rn(__fmul_rn((float)v, sam), swv[e]));
                            if (acc_out) acc_out[(int64_t)m * N + n] = v;
                        }
                    }
                }
            }
        }
    }
}

}  // namespace

// Dispatch of the prefill shapes (M > 16):
//  * M >= 1024 and N >= 1024: 256 x 128 tiles, two blocks per CU, persistent
//    over their tiles (k_w4a4_gemm_pt);
//  * M < 1024 and N >= 1024 (one image's pruned sequence): k_w4a4_gemm_2cu
//    with 128 x 128 tiles, or 64 x 128 (mid_bm); given the caller's
//    workspace, the tiles past the last whole round per CU are split along
//    K and reduced in the kernel (mid_plan);
//  * anything narrower: the small-M kernel, whose K slices are summed by a
//    second kernel (small_m_splits).
static bool use_large_tiles(int M, int N) { return M >= 1024 && N >= 1024; }
static bool use_mid_tiles(int M, int N) { return M > 16 && M < 1024 && N >= 1024; }

// Tile height of the mid path: 128 rows, or 64 where 128-row tiles would
// leave most CUs with a single block (fewer than 1.5 tiles per CU) and
// K_in <= 4096.  64-row tiles are less efficient per tile (their fragment
// reads per MFMA double), but there they fill the CUs with 2-3 blocks each:
// measured with the in-kernel split of the last round, q|k|v at M = 384
// (288 tiles of 128 rows) 28.4-29.2 -> 26.1-27.3 us; gate|up (516 tiles) and
// everything at M = 704 were 5-20% slower on 64-row tiles.  Before that
// split: o_proj at M = 704, 21.5 us unsplit on 352 tiles of 64 rows against
// 27.7 us on 192 tiles of 128 split in two.
static int mid_bm(int M, int N, int K) {
    const int64_t tiles128 = (((int64_t)M + 127) / 128) * (((int64_t)N + L_BN - 1) / L_BN);
    return (2 * tiles128 < 3 * (int64_t)device_cus() && K <= 4096) ? 64 : 128;
}

// Split plan of the mid-tile launches (needs the caller's workspace).  The
// tiles are dealt as whole tiles per CU as far as they go; the last T % C
// tiles (C = CUs), or all of them when T < C, are split along K into S slices
// whose blocks meet in the workspace (the last to arrive adds the others'
// exact int32 sums and writes the tile), so every CU gets about the same
// share of k-tiles:
//  * T < C: S = 512 / T, at most 8, each slice at least 16 k-tiles of 128
//    (measured at M = 384 / 704: down_proj, K = 11008, is fastest at 4-5
//    slices; every slice adds 64 KB of partial sums per tile written and
//    read back);
//  * T >= C: S = C / (T % C), at most 8, each slice at least 4 k-tiles.
//    A whole last round of T % C tiles on as many CUs costs a batch-1 layer
//    ~14 us of ~118 (timed with the remainder tiles left out).
// bytes of arrival counters at the head of a split launch's workspace
constexpr size_t kArrivalBytes = 4096;
struct MidPlan {
    int bm, T, tdp, rem, S, kps;   // tiles [tdp, T) split into S slices of kps k-tiles
};
static MidPlan mid_plan(int M, int N, int K) {
    MidPlan p{};
    p.bm = mid_bm(M, N, K);
    const int64_t T64 = (((int64_t)M + p.bm - 1) / p.bm) * (((int64_t)N + L_BN - 1) / L_BN);
    p.T = (int)std::min<int64_t>(T64, 1 << 30);
    p.tdp = p.T;
    p.S = 1;
    const int kt_all = (int)(((int64_t)K / 2 + BKB - 1) / BKB);
    p.kps = kt_all;
    if (!use_mid_tiles(M, N) || T64 >= (1 << 30)) return p;
    const int cus = device_cus();
    int S, rem;
    if (p.T < cus) {
        rem = p.T;
        S = std::min(std::min(512 / p.T, 8), kt_all / 16);
    } else {
        rem = p.T % cus;
        if (rem == 0) return p;
        S = std::min(std::min(cus / rem, 8), kt_all / 4);
    }
    if (S < 2 || rem > (int)(kArrivalBytes / 4)) return p;   // one arrival counter per split tile
    p.kps = (kt_all + S - 1) / S;
    p.S = (kt_all + p.kps - 1) / p.kps;              // every slice non-empty
    p.rem = rem;
    p.tdp = p.T - rem;
    return p;
}
// workspace of a split mid launch: arrival counters (zero between calls),
// then one BM x 128 int32 slot per slice
static size_t mid_split_bytes(const MidPlan &p) {
    return p.S > 1 ? kArrivalBytes + (size_t)p.rem * p.S * p.bm * L_BN * 4 : 0;
}

// Small-M shapes with fewer 128 x 128 tiles than CUs split K across
// work-groups (exact int32 partials, summed by the epilogue kernel):
// S = ceil(256 / tiles), at most 4, each slice at least 4 k-tiles of 256.
// Not for the decode GEMV or the tile kernels above, nor when N % 4 != 0
// (the epilogue writes 4 outputs per thread).
static int small_m_splits(int M, int N, int K) {
    if (M <= 16 || use_large_tiles(M, N) || use_mid_tiles(M, N) || N % 4 != 0) return 1;
    const int64_t tiles = (((int64_t)M + BM - 1) / BM) * (((int64_t)N + BN - 1) / BN);
    const int kt_all = (K / 2 + KS_ROW - 1) / KS_ROW;
    if (tiles >= 256) return 1;
    int S = (int)((256 + tiles - 1) / tiles);
    S = std::min(S, 4);
    S = std::min(S, kt_all / 4);
    return std::max(S, 1);
}

namespace {
__global__ __launch_bounds__(256) void k_clear_words(uint32_t *__restrict__ p, int n) {
    const int i = (int)(blockIdx.x * 256 + threadIdx.x);
    if (i < n) p[i] = 0u;
}
}  // namespace

hipError_t gemm_workspace_clear(void *ws, size_t ws_bytes, hipStream_t stream) {
    if (!ws || ws_bytes < kArrivalBytes) return hipSuccess;
    const int n = (int)(kArrivalBytes / 4);
    hipLaunchKernelGGL(k_clear_words, dim3((n + 255) / 256), dim3(256), 0, stream,
                       static_cast<uint32_t *>(ws), n);
    return hipGetLastError();
}

size_t gemm_workspace_bytes(int M, int N, int K) {
    if (use_mid_tiles(M, N)) return mid_split_bytes(mid_plan(M, N, K));
    const int S = small_m_splits(M, N, K);
    return S > 1 ? (size_t)S * M * N * 4 : 0;
}

hipError_t launch_w4a4_gemm(int M, int N, int K, const uint8_t *a, const float *sa,
                            const uint8_t *w, const float *sw, p4q_dtype out_dt, void *y,
                            int64_t ldy, int32_t *acc_out, void *ws, size_t ws_bytes,
                            hipStream_t stream) {
    const bool bf16 = (out_dt == P4Q_BF16);
    // decode kernel: 32-bit buffer offsets need N * K_in / 2 < 2^31
    if (M <= 16 && K <= G_MAX_KIN && (int64_t)N * (K / 2) < 0x7FFF0000LL) {
        const int cus = device_cus();
        const int groups = (N + G_ROWS - 1) / G_ROWS;
        const int ktiles = (K + 127) / 128;
        auto go = [&](auto kern, int nw, int blocks_per_cu) {
            hipLaunchKernelGGL(kern, dim3(min(groups, blocks_per_cu * cus)), dim3(64 * nw), 0,
                               stream, a, sa, w, sw, M, N, K / 2, y, ldy, acc_out);
            return hipGetLastError();
        };
        // up to 6 k-tiles per wavefront: 8 wavefronts, two work-groups per CU;
        // longer rows: 16 wavefronts (at most 7 k-tiles each), one per CU
#define P4Q_GEMV(NB, NW, BPC)                                                               \
    if (ktiles <= NB * NW)                                                                 \
        return bf16 ? go(k_w4a4_gemv<NB, NW, true>, NW, BPC)                               \
                    : go(k_w4a4_gemv<NB, NW, false>, NW, BPC);
        P4Q_GEMV(2, 8, 2)
        P4Q_GEMV(4, 8, 2)
        P4Q_GEMV(6, 8, 2)
        P4Q_GEMV(5, 16, 1)
        P4Q_GEMV(7, 16, 1)
#undef P4Q_GEMV
    }
    const bool ws_ok = ws && ((uintptr_t)ws & 15) == 0 && ws_bytes >= gemm_workspace_bytes(M, N, K);
    const unsigned eb = (unsigned)(((int64_t)M * N / 4 + 255) / 256);   // split-K epilogue blocks
    if (use_large_tiles(M, N) || use_mid_tiles(M, N)) {
        const bool large = use_large_tiles(M, N);
        const MidPlan plan = large ? MidPlan{} : mid_plan(M, N, K);
        const int bm = large ? L_BM : plan.bm;
        const int tiles_m = (M + bm - 1) / bm, tiles_n = (N + L_BN - 1) / L_BN;
        const int T = tiles_m * tiles_n;
        if (!large && plan.S > 1 && ws_ok) {
            uint32_t *arrivals = static_cast<uint32_t *>(ws);
            int32_t *part = reinterpret_cast<int32_t *>(static_cast<uint8_t *>(ws) + kArrivalBytes);
            const dim3 grid((unsigned)(plan.tdp + plan.rem * plan.S));
            auto gs = [&](auto kern) {
                hipLaunchKernelGGL(kern, grid, dim3(256), 0, stream, a, sa, w, sw, M, N, K / 2, y, ldy,
                                   acc_out, tiles_m, tiles_n, (int64_t)0, (int64_t)0, (int64_t)0,
                                   plan.kps, part, plan.tdp, plan.S, arrivals);
                return hipGetLastError();
            };
#define P4Q_SPLIT(BMT)                                                                        \
    if (bf16) return acc_out ? gs(k_w4a4_gemm_2cu<BMT, true, true, true, true>)                \
                             : gs(k_w4a4_gemm_2cu<BMT, true, false, true, true>);             \
    return acc_out ? gs(k_w4a4_gemm_2cu<BMT, false, true, true, true>)                         \
                   : gs(k_w4a4_gemm_2cu<BMT, false, false, true, true>);
            if (bm == 64) { P4Q_SPLIT(64) }
            P4Q_SPLIT(128)
#undef P4Q_SPLIT
        }
        auto go = [&](auto kern) {
            hipLaunchKernelGGL(kern, dim3(T), dim3(256), 0, stream, a, sa, w, sw, M, N, K / 2, y, ldy,
                               acc_out, tiles_m, tiles_n, (int64_t)0, (int64_t)0, (int64_t)0, 0,
                               (int32_t *)nullptr, 0, 1, (uint32_t *)nullptr);
            return hipGetLastError();
        };
#define P4Q_TILES(BMT)                                                                        \
    if (bf16) return acc_out ? go(k_w4a4_gemm_2cu<BMT, true, true, true, false>)               \
                             : go(k_w4a4_gemm_2cu<BMT, true, false, true, false>);            \
    return acc_out ? go(k_w4a4_gemm_2cu<BMT, false, true, true, false>)                        \
                   : go(k_w4a4_gemm_2cu<BMT, false, false, true, false>);
        if (large) {
            // persistent tiles: at most two resident blocks per CU
            const unsigned grid = (unsigned)std::min<int64_t>(T, 2LL * device_cus());
            auto gp = [&](auto kern) {
                hipLaunchKernelGGL(kern, dim3(grid), dim3(256), 0, stream, a, sa, w, sw, M, N, K / 2,
                                   y, ldy, acc_out, tiles_m, tiles_n);
                return hipGetLastError();
            };
            if (bf16) return acc_out ? gp(k_w4a4_gemm_pt<true, true>) : gp(k_w4a4_gemm_pt<true, false>);
            return acc_out ? gp(k_w4a4_gemm_pt<false, true>) : gp(k_w4a4_gemm_pt<false, false>);
        }
        if (bm == 64) { P4Q_TILES(64) }
        P4Q_TILES(128)
#undef P4Q_TILES
    }
    const dim3 grid((N + BN - 1) / BN, (M + BM - 1) / BM);
    const int S = small_m_splits(M, N, K);
    if (S > 1 && ws_ok) {
        const int kt_all = (K / 2 + KS_ROW - 1) / KS_ROW, kps = (kt_all + S - 1) / S;
        int32_t *part = static_cast<int32_t *>(ws);
        const dim3 gs(grid.x, grid.y, (kt_all + kps - 1) / kps);
        const int Sr = (int)gs.z;
        if (bf16) {
            hipLaunchKernelGGL((k_w4a4_gemm_ks<true, true>), gs, dim3(KS_THREADS), 0, stream, a, sa,
                               w, sw, M, N, K / 2, y, ldy, acc_out, kps, part);
            hipLaunchKernelGGL(k_splitk_epilogue<true>, dim3(eb), dim3(256), 0, stream, part, Sr, M,
                               N, sa, sw, y, ldy, acc_out);
        } else {
            hipLaunchKernelGGL((k_w4a4_gemm_ks<false, true>), gs, dim3(KS_THREADS), 0, stream, a, sa,
                               w, sw, M, N, K / 2, y, ldy, acc_out, kps, part);
            hipLaunchKernelGGL(k_splitk_epilogue<false>, dim3(eb), dim3(256), 0, stream, part, Sr, M,
                               N, sa, sw, y, ldy, acc_out);
        }
        return hipGetLastError();
    }
    if (bf16)
        hipLaunchKernelGGL((k_w4a4_gemm_ks<true, false>), grid, dim3(KS_THREADS), 0, stream, a, sa,
                           w, sw, M, N, K / 2, y, ldy, acc_out, 0, nullptr);
    else
        hipLaunchKernelGGL((k_w4a4_gemm_ks<false, false>), grid, dim3(KS_THREADS), 0, stream, a, sa,
                           w, sw, M, N, K / 2, y, ldy, acc_out, 0, nullptr);
    return hipGetLastError();
}

// Gram matrices of a batch of packed code blocks: G_b = C_b C_b^T (int32,
// [n, n] each, row-major), C_b = codes + b * n * (k/2).  Exact integer sums.
hipError_t launch_code_gram(int B, int n, int k, const uint8_t *codes, int32_t *G,
                            hipStream_t stream) {
    const int kb = k / 2;
    if (n >= 1024) {
        const int tiles_m = (n + L_BM - 1) / L_BM, tiles_n = (n + L_BN - 1) / L_BN;
        int upper = 0;                              // tiles with tn >= 2 tm
        for (int tm = 0; tm < tiles_m; ++tm) upper += std::max(0, tiles_n - 2 * tm);
        hipLaunchKernelGGL((k_w4a4_gemm_2cu<256, true, true, false, false>), dim3(upper, B),
                           dim3(256), 0, stream, codes, nullptr, codes, nullptr, n, n, kb, nullptr,
                           (int64_t)n, G, upper, tiles_n, (int64_t)n * kb, (int64_t)n * kb,
                           (int64_t)n * n, 0, (int32_t *)nullptr, 0, 1, (uint32_t *)nullptr);
        return hipGetLastError();
    }
    const dim3 grid((n + BN - 1) / BN, (n + BM - 1) / BM);
    for (int b = 0; b < B; ++b) {
        const uint8_t *cb = codes + (int64_t)b * n * kb;
        hipLaunchKernelGGL(k_w4a4_gemm<true>, grid, dim3(kThreads), 0, stream, cb, nullptr, cb, nullptr, n,
                           n, kb, nullptr, (int64_t)n, G + (int64_t)b * n * n);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace p4q
