// Device-side pieces of the per-row symmetric 4-bit RTN quantizer
// (P4Q Appendix A / B.3 W4A4 setting) shared by the quantize-and-pack kernel
// and the selector's fake-quant + score kernel.
//
// Q4(x; c):  a = max|x|,  s = fl32(fl32(c*a)/7),
//            code = clamp(rne(fl32(x/s)), -8, 7)   (s == 0 -> code 0)
//
// Exactness of the fast path.  With r = fl32(1/s), the fma x*r + 1.5*2^23
// rounds the exact product x*r to the nearest integer (ties to even) in the
// low mantissa bits, and fma(x, r, -q) gives the exact residual x*r - q up to
// one rounding.  For |x/s| < 8, |x*r - x/s| <= 8*2^-24 and
// |fl32(x/s) - x/s| <= 2^-22, so when x*r is farther than 2^-19 from every
// half-integer, rne(x*r) == rne(fl32(x/s)).  Otherwise the values are
// recomputed with the correctly rounded division (HIP's default fp32 '/').
// Past |x/s| >= 8 only clamped codes are produced, which both paths agree on.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace p4q {

constexpr float kRneMagic = 12582912.0f;        // 1.5 * 2^23
constexpr float kNearHalf = 0.5f - 0x1p-19f;    // residual above this -> exact path
constexpr float kTinyScale = 0x1p-100f;         // below: 1/s may overflow -> exact path

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// streaming 16-byte load (data read once: non-temporal hint)
__device__ __forceinline__ uint4 load_nt(const uint4 *p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// decode the low / high 16-bit half of a word (fp16 or bf16) to fp32, exactly
template <bool BF16>
__device__ __forceinline__ float lo_f32(uint32_t w) {
    if constexpr (BF16) return __uint_as_float(w << 16);
    else return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu));
}
template <bool BF16>
__device__ __forceinline__ float hi_f32(uint32_t w) {
    if constexpr (BF16) return __uint_as_float(w & 0xFFFF0000u);
    else return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
}

// magnitude bits of a 16-bit float (fp16 and bf16 alike) order like |x|
template <bool BF16>
__device__ __forceinline__ float mag_to_f32(uint32_t m16) {
    if constexpr (BF16) return __uint_as_float(m16 << 16);
    else return (float)__builtin_bit_cast(_Float16, (uint16_t)m16);
}

// running per-half maximum of |x| bit patterns over packed 16-bit pairs
__device__ __forceinline__ uint32_t absmax2(uint32_t m, uint32_t w) {
    u16x2 a = __builtin_bit_cast(u16x2, m);
    u16x2 b = __builtin_bit_cast(u16x2, w & 0x7FFF7FFFu);
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(a, b));
}

__device__ __forceinline__ uint32_t absmax_chunk(uint32_t m, uint4 v) {
    m = absmax2(m, v.x);
    m = absmax2(m, v.y);
    m = absmax2(m, v.z);
    return absmax2(m, v.w);
}

// Maximum over the 64 lanes, wave-uniform result.  DPP moves within each
// row of 16 lanes (quad swaps, half-row and row mirrors) leave every lane
// holding its row's maximum; the four rows meet through lane reads.  No LDS
// round trip (a shuffle chain costs six).  Every lane must be active.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));   // quad [1,0,3,2]
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));   // quad [2,3,0,1]
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));  // row_half_mirror
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));  // row_mirror
    const uint32_t a = max((uint32_t)__builtin_amdgcn_readlane((int)v, 0),
                           (uint32_t)__builtin_amdgcn_readlane((int)v, 16));
    const uint32_t b = max((uint32_t)__builtin_amdgcn_readlane((int)v, 32),
                           (uint32_t)__builtin_amdgcn_readlane((int)v, 48));
    return max(a, b);
}

// s = fl32(fl32(c*a)/7); both operations correctly rounded (no fast-math)
template <bool CLIP1>
__device__ __forceinline__ float row_scale(float a, float clip) {
    if constexpr (CLIP1) return a / 7.0f;
    else return __fmul_rn(clip, a) / 7.0f;
}

// Fast path for one value.  Returns a word whose low byte (and low nibble)
// is the two's-complement code; sets `near` when the exact path is needed.
template <bool CLIP1>
__device__ __forceinline__ uint32_t q4_fast(float x, float r, uint32_t &near) {
    float t = __builtin_fmaf(x, r, kRneMagic);
    float q = t - kRneMagic;                     // exact: rne(x*r)
    float f = __builtin_fmaf(x, r, -q);          // x*r - q, one rounding
    near |= (uint32_t)(__builtin_fabsf(f) > kNearHalf);
    if constexpr (!CLIP1) t = __builtin_amdgcn_fmed3f(t, kRneMagic - 8.0f, kRneMagic + 7.0f);
    return __float_as_uint(t);
}

// Exact path: correctly rounded fp32 division, ties-to-even, clamp.
__device__ __forceinline__ uint32_t q4_exact(float x, float s) {
    float q = x / s;
    float c = __builtin_rintf(q);
    c = __builtin_amdgcn_fmed3f(c, -8.0f, 7.0f);
    return (uint32_t)(int)c;
}

// low bytes of four words -> one word of four int8 (byte i from w_i)
__device__ __forceinline__ uint32_t bytes4(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3) {
    uint32_t lo = __builtin_amdgcn_perm(w1, w0, 0x0c0c0400u);   // [w0.b0, w1.b0, 0, 0]
    uint32_t hi = __builtin_amdgcn_perm(w3, w2, 0x04000c0cu);   // [0, 0, w2.b0, w3.b0]
    return lo | hi;
}

// low nibbles of eight words -> packed int4 word (nibble i from w_i), with
// two byte gathers and one bit-field insert
__device__ __forceinline__ uint32_t pack_nibbles(const uint32_t *w) {
    const uint32_t e = bytes4(w[0], w[2], w[4], w[6]);   // even values, one per byte
    const uint32_t o = bytes4(w[1], w[3], w[5], w[7]);   // odd values
    return (e & 0x0F0F0F0Fu) | ((o << 4) & 0xF0F0F0F0u);
}

// Quantize the 8 values of one 16-byte chunk.  out[i] low byte = code of
// value i (value order = memory order).
template <bool BF16, bool CLIP1>
__device__ __forceinline__ void q4_chunk_fast(uint4 v, float r, uint32_t *out, uint32_t &near) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        out[2 * i] = q4_fast<CLIP1>(lo_f32<BF16>(w[i]), r, near);
        out[2 * i + 1] = q4_fast<CLIP1>(hi_f32<BF16>(w[i]), r, near);
    }
}

// Bracketed fast path for the 8 values of one 16-byte chunk.  With
// r = fl32(1/s), rhi = fl32(r (1 + 2^-20)) and rlo = fl32(r (1 - 2^-20)),
// x*rhi and x*rlo (each rounded once, inside the fma) enclose fl32(x/s):
// r and fl32(x/s) each err by at most 2^-24 relative.  rne is monotone, so
// where the two bracket ends round to the same integer so does fl32(x/s);
// where they differ a half-integer lies inside and the exact path decides.
// Two mixed-precision fmas and one three-input bitwise op per value: `dif`
// collects lo ^ hi (nonzero: some bracket of this chunk straddles).  out[i]
// low byte = code of value i (two's complement; clamped unless CLIP1, where
// |x| <= amax keeps |x/s| <= 7).
template <bool BF16, bool CLIP1>
__device__ __forceinline__ void q4_chunk_bracket(uint4 v, float rhi, float rlo, uint32_t *out,
                                                 uint32_t &dif) {
    const uint32_t x4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const float x = h ? hi_f32<BF16>(x4[i]) : lo_f32<BF16>(x4[i]);
            float tq = __builtin_fmaf(x, rhi, kRneMagic);
            const float tl = __builtin_fmaf(x, rlo, kRneMagic);
            // dif |= tq ^ tl (as asm: left to itself the compiler turns the
            // merge into a compare and select per value)
            asm("v_bitop3_b32 %0, %0, %1, %2 bitop3:0xf6"
                : "+v"(dif)
                : "v"(__float_as_uint(tq)), "v"(__float_as_uint(tl)));
            if constexpr (!CLIP1) tq = __builtin_amdgcn_fmed3f(tq, kRneMagic - 8.0f, kRneMagic + 7.0f);
            out[2 * i + h] = __float_as_uint(tq);
        }
    }
}

// Largest |x| bit pattern (sign bit clear) among a lane's CH chunks.
// fp16: a running packed maximum and minimum, each three-input op folding
// two more words, then max(|max|, |min|) per half; bf16: 16-bit maxima of
// the bit patterns with the sign masked.  Finite inputs.
template <int CH, bool BF16>
__device__ __forceinline__ uint32_t lane_absmax_bits(const uint4 *v) {
    if constexpr (BF16) {
        uint32_t m2 = 0;
#pragma unroll
        for (int c = 0; c < CH; ++c) m2 = absmax_chunk(m2, v[c]);
        return max(m2 & 0xFFFFu, m2 >> 16);
    } else {
        uint32_t w[4 * CH];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            w[4 * c] = v[c].x;
            w[4 * c + 1] = v[c].y;
            w[4 * c + 2] = v[c].z;
            w[4 * c + 3] = v[c].w;
        }
        uint32_t hi = w[0], lo = w[0];
#pragma unroll
        for (int k = 1; k < 4 * CH; k += 2) {
            const uint32_t b = (k + 1 < 4 * CH) ? w[k + 1] : w[k];
            asm("v_pk_maximum3_f16 %0, %0, %1, %2" : "+v"(hi) : "v"(w[k]), "v"(b));
            asm("v_pk_minimum3_f16 %0, %0, %1, %2" : "+v"(lo) : "v"(w[k]), "v"(b));
        }
        // every |x| lies below max(|hi|, |lo|), per half
        const uint32_t m2 = absmax2(absmax2(0u, hi), lo);
        return max(m2 & 0xFFFFu, m2 >> 16);
    }
}

template <bool BF16>
__device__ __forceinline__ void q4_chunk_exact(uint4 v, float s, uint32_t *out) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        out[2 * i] = q4_exact(lo_f32<BF16>(w[i]), s);
        out[2 * i + 1] = q4_exact(hi_f32<BF16>(w[i]), s);
    }
}

}  // namespace p4q
