// Internal launchers behind the C ABI (include/p4q.h).  Arguments have been
// validated by the caller; each launcher only enqueues kernels on `stream`
// and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/p4q.h"

namespace p4q {

// ---- quantize + pack (Q4 per row) ------------------------------------------
hipError_t launch_quant_act(p4q_dtype dt, int M, int K_in, const void *x, int64_t ldx,
                            float clip, uint8_t *codes, float *scales, hipStream_t stream);

// ---- selector ---------------------------------------------------------------
struct SelectWorkspace {
    int32_t *stats;      // [B][N][J+1]: D_0..D_{J-1}, Nv   (documented)
    int64_t *keys;       // [B][J][N]: exact order keys (internal)
    int8_t *ccodes;      // [B][J][d]: concept codes (internal)
};
size_t select_workspace_bytes(int B, int N, int d, int J);
SelectWorkspace select_workspace_carve(void *ws, int B, int N, int d, int J);

hipError_t launch_select(p4q_dtype dt, int B, int N, int d, const void *vis,
                         const void *concepts, int J, const void *text, int T, int K,
                         float clip, int32_t *idx_out, void *tokens_out,
                         const SelectWorkspace &ws, hipStream_t stream);

// ---- W4A4 GEMM ---------------------------------------------------------------
size_t gemm_workspace_bytes(int M, int N, int K);
hipError_t launch_w4a4_gemm(int M, int N, int K, const uint8_t *a, const float *sa,
                            const uint8_t *w, const float *sw, p4q_dtype out_dt, void *y,
                            int64_t ldy, int32_t *acc_out, void *ws, size_t ws_bytes,
                            hipStream_t stream);

}  // namespace p4q
