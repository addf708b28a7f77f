// Internal launchers behind the C ABI (include/p4q.h).  Arguments have been
// validated by the caller; each launcher only enqueues kernels on `stream`
// and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>

#include "../../include/p4q.h"

namespace p4q {

// ---- per-device constants -----------------------------------------------------
// Launch shapes depend on the device's CU count and on how many blocks of a
// kernel fit on a CU.  Both are fixed for a device, so they are queried once
// per device ordinal and kept in a cache of atomics: concurrent first calls
// from several host threads each store the same value, and no other state
// is shared between calls.
constexpr int kMaxDevices = 64;

inline int current_device() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
    return dev;
}

// cached value of query() for the current device; query() returns > 0
template <class Query>
inline int per_device_cached(std::atomic<int> (&cache)[kMaxDevices], Query query) {
    const int dev = current_device();
    if (dev >= kMaxDevices) return query(dev);
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v <= 0) {
        v = query(dev);
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

// compute units of the current device (256 on MI355X if the query fails)
inline int device_cus() {
    static std::atomic<int> cache[kMaxDevices];
    return per_device_cached(cache, [](int dev) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
        return cus;
    });
}

// ---- quantize + pack (Q4 per row) ------------------------------------------
hipError_t launch_quant_act(p4q_dtype dt, int M, int K_in, const void *x, int64_t ldx,
                            float clip, uint8_t *codes, float *scales, hipStream_t stream);

// ---- fused prologue: per-token Q4 of RMSNorm(x) * gamma ------------------------
hipError_t launch_rmsnorm_quant(p4q_dtype dt, int M, int d, const void *x, int64_t ldx,
                                const void *gamma, float eps, float clip, uint8_t *codes,
                                float *scales, hipStream_t stream);

// ---- attention prefill (FP16 / BF16 Q, K, V; head dimension 128) -------------
hipError_t launch_attention(p4q_dtype dt, int B, int L, int H, const void *q, const void *k,
                            const void *v, int64_t ld, void *o, int64_t ldo, int causal,
                            hipStream_t stream);

// ---- selector ---------------------------------------------------------------
struct SelectWorkspace {
    int32_t *stats;      // [B][N][J+1]: D_0..D_{J-1}, Nv   (documented)
    int64_t *keys;       // [B][J][N]: exact order keys (internal)
    uint32_t *vcodes = nullptr;   // [B][N][d/8] packed visual codes, or none
};

// the three-stage selector's workspace: the above, then
struct SelectFullWorkspace {
    SelectWorkspace sel;    // vcodes set
    int32_t *gram;          // [B][N][N] code Gram matrices (exact int32)
    int64_t *mp;            // [kDivInitPlanes][B][N] partial maxima over the kept
    int32_t *mq;            //        set, as pairs (p, q) (see diversity.hip)
    int32_t *stages;        // [B][K] stage picks when the caller gives none
};
size_t select_full_workspace_bytes(int B, int N, int d, int J, int K);
SelectFullWorkspace select_full_workspace_carve(void *ws, int B, int N, int d, int J, int K);
size_t select_workspace_bytes(int B, int N, int d, int J);
SelectWorkspace select_workspace_carve(void *ws, int B, int N, int d, int J);

hipError_t launch_select(p4q_dtype dt, int B, int N, int d, const void *vis,
                         const void *concepts, int J, const void *text, int T, int K,
                         float clip, int32_t *idx_out, void *tokens_out,
                         const SelectWorkspace &ws, hipStream_t stream);

hipError_t launch_select_full(p4q_dtype dt, int B, int N, int d, const void *vis,
                              const void *concepts, int J, const float *cls_attn,
                              const void *text, int T, int K, int kq, int ks, float clip,
                              int32_t *idx_out, int32_t *stages_out, void *tokens_out,
                              const SelectFullWorkspace &ws, hipStream_t stream);

constexpr int kDivInitPlanes = 8;

// Visual Diversity completion (diversity.hip): n0 = kq + ks tokens already
// in stages[b][0, n0); kd greedy picks appended there in pick order;
// idx_out[b][0, K) = all K kept tokens, ascending.
hipError_t launch_diversity(int B, int N, int K, int n0, int kd, const int32_t *gram,
                            const float *cls_attn, int64_t *mp, int32_t *mq, int32_t *stages,
                            int32_t *idx_out, hipStream_t stream);

// ---- calibration mechanics (calib.hip) ---------------------------------------
hipError_t launch_quant_scaled(p4q_dtype dt, int R, int K, const void *z, int64_t ldz,
                               const float *sigma, int divide, float clip, const float *clip_rows,
                               uint8_t *codes, float *scales, float *absmax, int32_t *kstar,
                               hipStream_t stream);
size_t calib_linear_workspace_bytes(int M, int N, int K);
hipError_t launch_calib_linear(p4q_dtype dt, int M, int N, int K, const void *x, int64_t ldx,
                               const void *w, int64_t ldw, const float *target, int64_t ldt,
                               const float *sigma, float clip_a, const float *clip_w,
                               float *loss, float *grad_sigma, float *grad_clip_a,
                               float *grad_clip_w, void *ws, hipStream_t stream);

size_t calib_block_workspace_bytes(int M, int d, int f, int H);
hipError_t launch_calib_block(int M, int d, int f, int H, const void *x, const float *target,
                              int64_t ldt, const void *w_qkv, const void *w_o, const void *w_gu,
                              const void *w_down, const void *gamma1, const void *gamma2,
                              float eps, float rope_base, const float *sigma, const float *clip_a,
                              const float *clip_w, float *loss, float *grad_sigma,
                              float *grad_clip_a, float *grad_clip_w, void *ws,
                              hipStream_t stream);

// ---- W4A4 GEMM ---------------------------------------------------------------
// G_b = C_b C_b^T for b < B, C_b = codes + b * n * (k/2) packed [n, k/2];
// G int32 [B][n][n].
hipError_t launch_code_gram(int B, int n, int k, const uint8_t *codes, int32_t *G,
                            hipStream_t stream);
size_t gemm_workspace_bytes(int M, int N, int K);
// Zeroes the arrival counters at the head of a GEMM workspace (a fill kernel
// on the stream; the GEMM calls leave them zero, so this is needed once per
// workspace whose contents are not known to be zero).
hipError_t gemm_workspace_clear(void *ws, size_t ws_bytes, hipStream_t stream);
hipError_t launch_w4a4_gemm(int M, int N, int K, const uint8_t *a, const float *sa,
                            const uint8_t *w, const float *sw, p4q_dtype out_dt, void *y,
                            int64_t ldy, int32_t *acc_out, void *ws, size_t ws_bytes,
                            hipStream_t stream);

// ---- diagnostics (diag.hip) ----------------------------------------------------
hipError_t launch_diag_mfma_i8(int blocks, int iters, int32_t *out, hipStream_t stream);
hipError_t launch_diag_read(const void *src, size_t bytes, int blocks, uint32_t *out,
                            hipStream_t stream);

}  // namespace p4q
