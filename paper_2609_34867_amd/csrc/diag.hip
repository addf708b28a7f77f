// Microbenchmarks of the two ceilings the hot path is measured against: the
// int8 MFMA rate and the HBM read rate of this device.  They are not part of
// the method; the benchmark reports its kernels as fractions of both the
// published peaks and these measured ones.
#include "p4q_internal.h"

namespace p4q {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

// Every wavefront issues `iters` rounds of 16 independent
// v_mfma_i32_16x16x64_i8 (16 accumulators, so no MFMA waits on the previous
// one), cycling through 4 A and 4 B operand registers filled with
// pseudo-random bytes: the operand bits change from one MFMA to the next as
// they do in a GEMM (the sustained clock depends on that switching).
__global__ __launch_bounds__(256) void k_diag_mfma_i8(int iters, int32_t *__restrict__ out) {
    const uint32_t t = blockIdx.x * 256u + threadIdx.x;
    v4i a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t h = t * 0x9E3779B1u + 0x7F4A7C15u * (i + 1);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            h ^= h << 13;
            h ^= h >> 17;
            h ^= h << 5;
            a[i][e] = (int)h;
            h ^= h << 13;
            h ^= h >> 17;
            h ^= h << 5;
            b[i][e] = (int)h;
        }
    }
    v4i acc[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = v4i{0, 0, 0, 0};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < 16; ++j)
            acc[j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[j & 3], b[(j >> 2) & 3], acc[j], 0, 0, 0);
    }
    int s = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) s += acc[j][0] ^ acc[j][1] ^ acc[j][2] ^ acc[j][3];
    out[t] = s;
}

// A plain streaming read: every thread reads 16-byte chunks i, i + stride,
// ... (four loads in flight per round) and stores one word of their xor, so
// the loads cannot be removed.
__global__ __launch_bounds__(256) void k_diag_read(const v4u *__restrict__ p, size_t n16,
                                                   uint32_t *__restrict__ out) {
    const size_t stride = (size_t)gridDim.x * 256;
    size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    uint32_t acc = 0;
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const v4u x0 = __builtin_nontemporal_load(p + i);
        const v4u x1 = __builtin_nontemporal_load(p + i + stride);
        const v4u x2 = __builtin_nontemporal_load(p + i + 2 * stride);
        const v4u x3 = __builtin_nontemporal_load(p + i + 3 * stride);
        acc ^= x0.x ^ x0.y ^ x0.z ^ x0.w ^ x1.x ^ x1.y ^ x1.z ^ x1.w;
        acc ^= x2.x ^ x2.y ^ x2.z ^ x2.w ^ x3.x ^ x3.y ^ x3.z ^ x3.w;
    }
    for (; i < n16; i += stride) {
        const v4u x = p[i];
        acc ^= x.x ^ x.y ^ x.z ^ x.w;
    }
    out[(size_t)blockIdx.x * 256 + threadIdx.x] = acc;
}

}  // namespace

hipError_t launch_diag_mfma_i8(int blocks, int iters, int32_t *out, hipStream_t stream) {
    hipLaunchKernelGGL(k_diag_mfma_i8, dim3(blocks), dim3(256), 0, stream, iters, out);
    return hipGetLastError();
}

hipError_t launch_diag_read(const void *src, size_t bytes, int blocks, uint32_t *out,
                            hipStream_t stream) {
    hipLaunchKernelGGL(k_diag_read, dim3(blocks), dim3(256), 0, stream,
                       static_cast<const v4u *>(src), bytes / 16, out);
    return hipGetLastError();
}

}  // namespace p4q
