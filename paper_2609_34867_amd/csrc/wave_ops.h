// Wavefront-level scans used by the selection kernels (64-lane wavefronts).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace p4q {

// Inclusive prefix sum over the 64 lanes of a wavefront with DPP row shifts
// and row broadcasts (no LDS round trips).
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t v) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, true);  // row_shr:1
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, true);  // row_shr:2
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, true);  // row_shr:4
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, true);  // row_shr:8
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false); // row_bcast:15
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false); // row_bcast:31
    return v;
}

// sum of wtot[0 .. wave) read as four 16-byte words (up to 16 wavefronts)
__device__ __forceinline__ uint32_t waves_before(const uint32_t *wtot, int wave) {
    const uint4 *w4 = reinterpret_cast<const uint4 *>(wtot);
    uint32_t s = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const uint4 v = w4[q];
        s += (4 * q + 0 < wave ? v.x : 0u) + (4 * q + 1 < wave ? v.y : 0u) +
             (4 * q + 2 < wave ? v.z : 0u) + (4 * q + 3 < wave ? v.w : 0u);
    }
    return s;
}

}  // namespace p4q
