// C ABI of libp4q (declared in include/p4q.h): argument validation, workspace
// sizing and dispatch.  Every check runs on the host before any HIP call, so a
// rejected call enqueues nothing; launch failures map to P4Q_ERR_HIP.
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "p4q_internal.h"

namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return status;
}

int ok() {
    g_last_error[0] = '\0';
    return P4Q_OK;
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool valid_dtype(int dt) { return dt == P4Q_FP16 || dt == P4Q_BF16; }

// clip in [2^-16, 1]; NaN fails both comparisons
bool valid_clip(float c) { return c >= 0x1p-16f && c <= 1.0f; }

int hip_status(hipError_t e, const char *what) {
    if (e != hipSuccess)
        return fail(P4Q_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

}  // namespace

extern "C" {

const char *p4q_version(void) { return "p4q 0.1.0 gfx950"; }

const char *p4q_status_string(int status) {
    switch (status) {
        case P4Q_OK: return "P4Q_OK";
        case P4Q_ERR_INVALID_ARG: return "P4Q_ERR_INVALID_ARG";
        case P4Q_ERR_UNSUPPORTED: return "P4Q_ERR_UNSUPPORTED";
        case P4Q_ERR_WORKSPACE: return "P4Q_ERR_WORKSPACE";
        case P4Q_ERR_HIP: return "P4Q_ERR_HIP";
        default: return "P4Q_ERR_UNKNOWN";
    }
}

const char *p4q_last_error(void) { return g_last_error; }

// the selector's size limits (outside them p4q_select rejects the call)
static bool select_shape_ok(int B, int N, int d, int J) {
    return B > 0 && N > 0 && N <= 8192 && d >= 32 && d <= 16384 && d % 32 == 0 && J > 0 &&
           J <= 8 && !(J > 4 && d > 8192);
}

size_t p4q_select_workspace_bytes(int B, int N, int d, int J) {
    if (!select_shape_ok(B, N, d, J)) return 0;
    return p4q::select_workspace_bytes(B, N, d, J);
}

// Checks shared by p4q_select and p4q_select_noalloc: everything but the
// workspace.  Returns P4Q_OK or the failing status (message recorded).
static int check_select_args(const char *who, p4q_dtype dt, int B, int N, int d,
                             const void *vis, const void *concepts, int J, const void *text,
                             int T, int K, float clip, const int32_t *idx_out,
                             const void *tokens_out) {
    if (!valid_dtype(dt)) return fail(P4Q_ERR_UNSUPPORTED, "%s: dtype %d", who, (int)dt);
    if (B <= 0 || N <= 0 || d <= 0 || J <= 0 || K <= 0 || T < 0)
        return fail(P4Q_ERR_INVALID_ARG, "%s: sizes must be positive (B=%d N=%d d=%d J=%d K=%d T=%d)",
                    who, B, N, d, J, K, T);
    if (K > N) return fail(P4Q_ERR_INVALID_ARG, "%s: K=%d > N=%d", who, K, N);
    if (!vis || !concepts || !idx_out || !tokens_out)
        return fail(P4Q_ERR_INVALID_ARG, "%s: null pointer", who);
    if ((T > 0) != (text != nullptr))
        return fail(P4Q_ERR_INVALID_ARG, "%s: text must be given iff T > 0", who);
    if (!valid_clip(clip)) return fail(P4Q_ERR_INVALID_ARG, "%s: clip %g outside [2^-16, 1]", who, clip);
    if (d % 32 != 0) return fail(P4Q_ERR_INVALID_ARG, "%s: d=%d not a multiple of 32", who, d);
    if (!aligned(vis, 16) || !aligned(concepts, 16) || !aligned(tokens_out, 16) ||
        (text && !aligned(text, 16)) || !aligned(idx_out, 4))
        return fail(P4Q_ERR_INVALID_ARG, "%s: misaligned pointer", who);
    if (N > 8192) return fail(P4Q_ERR_UNSUPPORTED, "%s: N=%d > 8192", who, N);
    if (J > 8) return fail(P4Q_ERR_UNSUPPORTED, "%s: J=%d > 8", who, J);
    if (d > 16384) return fail(P4Q_ERR_UNSUPPORTED, "%s: d=%d > 16384", who, d);
    if (J > 4 && d > 8192) return fail(P4Q_ERR_UNSUPPORTED, "%s: J > 4 needs d <= 8192", who);
    return P4Q_OK;
}

int p4q_select(p4q_dtype dt, int B, int N, int d, const void *vis, const void *concepts, int J,
               const void *text, int T, int K, float clip, int32_t *idx_out, void *tokens_out,
               void *ws, size_t ws_bytes, hipStream_t stream) {
    if (const int st = check_select_args("p4q_select", dt, B, N, d, vis, concepts, J, text, T, K,
                                         clip, idx_out, tokens_out))
        return st;
    const size_t need = p4q::select_workspace_bytes(B, N, d, J);
    if (!ws || ws_bytes < need)
        return fail(P4Q_ERR_WORKSPACE, "p4q_select: workspace %zu < %zu bytes", ws_bytes, need);
    if (!aligned(ws, 256)) return fail(P4Q_ERR_INVALID_ARG, "p4q_select: workspace not 256-byte aligned");
    const p4q::SelectWorkspace w = p4q::select_workspace_carve(ws, B, N, d, J);
    return hip_status(p4q::launch_select(dt, B, N, d, vis, concepts, J, text, T, K, clip, idx_out,
                                         tokens_out, w, stream),
                      "p4q_select");
}

}  // extern "C"

// ---- the selector without a caller-supplied workspace ------------------------
// Its workspace lives in `scratch`, one array per device in the library's
// device image.  In host code the name `scratch` is only a stand-in for the
// symbol: its device address is looked up (hipGetSymbolAddress) once per
// device, with that device current, and only that address is ever passed on.
static __device__ __align__(256) uint8_t scratch[P4Q_SELECT_SCRATCH_BYTES];

namespace {

std::atomic<uintptr_t> g_scratch_addr[p4q::kMaxDevices];

// Device address of `scratch` on the device `stream` belongs to (the
// caller's current device for the null stream).  Returns P4Q_OK or an error
// status with the message recorded.
int scratch_address(hipStream_t stream, void **addr, const char *who) {
    int dev = 0, cur = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e == hipSuccess) {
        dev = cur;
        if (stream) e = hipStreamGetDevice(stream, &dev);
    }
    if (e != hipSuccess) return fail(P4Q_ERR_HIP, "%s: device of the stream: %s", who, hipGetErrorString(e));
    if (dev < 0 || dev >= p4q::kMaxDevices)
        return fail(P4Q_ERR_UNSUPPORTED, "%s: device %d beyond the %d supported", who, dev, p4q::kMaxDevices);
    uintptr_t a = g_scratch_addr[dev].load(std::memory_order_acquire);
    if (a == 0) {
        // with that device current: each device holds its own copy of the array
        if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess)
            return fail(P4Q_ERR_HIP, "%s: hipSetDevice(%d): %s", who, dev, hipGetErrorString(e));
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        const hipError_t e2 = (dev != cur) ? hipSetDevice(cur) : hipSuccess;
        if (e != hipSuccess || p == nullptr)
            return fail(P4Q_ERR_HIP, "%s: hipGetSymbolAddress(scratch): %s", who,
                        hipGetErrorString(e != hipSuccess ? e : hipErrorInvalidSymbol));
        if (e2 != hipSuccess)
            return fail(P4Q_ERR_HIP, "%s: hipSetDevice(%d): %s", who, cur, hipGetErrorString(e2));
        a = reinterpret_cast<uintptr_t>(p);
        g_scratch_addr[dev].store(a, std::memory_order_release);   // racing first calls store the same
    }
    *addr = reinterpret_cast<void *>(a);
    return P4Q_OK;
}

}  // namespace

extern "C" {

int p4q_select_noalloc(p4q_dtype dt, int B, int N, int d, const void *vis, const void *concepts,
                       int J, const void *text, int T, int K, float clip, int32_t *idx_out,
                       void *tokens_out, hipStream_t stream) {
    if (const int st = check_select_args("p4q_select_noalloc", dt, B, N, d, vis, concepts, J, text,
                                         T, K, clip, idx_out, tokens_out))
        return st;
    const size_t need = p4q::select_workspace_bytes(B, N, d, J);
    if (need > (size_t)P4Q_SELECT_SCRATCH_BYTES)
        return fail(P4Q_ERR_WORKSPACE,
                    "p4q_select_noalloc: B=%d N=%d d=%d J=%d needs %zu bytes of scratch, more than "
                    "the %zu the library holds per device (use p4q_select with a workspace)",
                    B, N, d, J, need, (size_t)P4Q_SELECT_SCRATCH_BYTES);
    void *ws = nullptr;
    if (const int st = scratch_address(stream, &ws, "p4q_select_noalloc")) return st;
    const p4q::SelectWorkspace w = p4q::select_workspace_carve(ws, B, N, d, J);
    return hip_status(p4q::launch_select(dt, B, N, d, vis, concepts, J, text, T, K, clip, idx_out,
                                         tokens_out, w, stream),
                      "p4q_select_noalloc");
}

size_t p4q_select_full_workspace_bytes(int B, int N, int d, int J, int K) {
    if (!select_shape_ok(B, N, d, J) || d > 8192 || K <= 0 || K > N) return 0;
    return p4q::select_full_workspace_bytes(B, N, d, J, K);
}

int p4q_select_budgets(int K, int *kq, int *ks, int *kd) {
    if (K < 0 || !kq || !ks || !kd) return fail(P4Q_ERR_INVALID_ARG, "p4q_select_budgets: K=%d or null output", K);
    *kq = (int)((int64_t)K * 3 / 10);
    *ks = (int)((int64_t)K * 2 / 10);
    *kd = K - *kq - *ks;
    return ok();
}

int p4q_select_full(p4q_dtype dt, int B, int N, int d, const void *vis, const void *concepts, int J,
                    const float *cls_attn, const void *text, int T, int K, int kq, int ks, float clip,
                    int32_t *idx_out, int32_t *stages_out, void *tokens_out, void *ws, size_t ws_bytes,
                    hipStream_t stream) {
    if (!valid_dtype(dt)) return fail(P4Q_ERR_UNSUPPORTED, "p4q_select_full: dtype %d", (int)dt);
    if (B <= 0 || N <= 0 || d <= 0 || J <= 0 || K <= 0 || T < 0)
        return fail(P4Q_ERR_INVALID_ARG,
                    "p4q_select_full: sizes must be positive (B=%d N=%d d=%d J=%d K=%d T=%d)", B, N, d, J, K, T);
    if (K > N) return fail(P4Q_ERR_INVALID_ARG, "p4q_select_full: K=%d > N=%d", K, N);
    if (kq < 0 || ks < 0 || (int64_t)kq + ks > K)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_select_full: budgets kq=%d ks=%d do not fit K=%d", kq, ks, K);
    if (!vis || !concepts || !cls_attn || !idx_out || !tokens_out)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_select_full: null pointer");
    if ((T > 0) != (text != nullptr))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_select_full: text must be given iff T > 0");
    if (!valid_clip(clip))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_select_full: clip %g outside [2^-16, 1]", clip);
    if (d % 32 != 0) return fail(P4Q_ERR_INVALID_ARG, "p4q_select_full: d=%d not a multiple of 32", d);
    if (!aligned(vis, 16) || !aligned(concepts, 16) || !aligned(tokens_out, 16) ||
        (text && !aligned(text, 16)) || !aligned(idx_out, 4) || !aligned(cls_attn, 4) ||
        (stages_out && !aligned(stages_out, 4)))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_select_full: misaligned pointer");
    if (N > 8192) return fail(P4Q_ERR_UNSUPPORTED, "p4q_select_full: N=%d > 8192", N);
    if (J > 8) return fail(P4Q_ERR_UNSUPPORTED, "p4q_select_full: J=%d > 8", J);
    if (d > 8192) return fail(P4Q_ERR_UNSUPPORTED, "p4q_select_full: d=%d > 8192", d);
    if (B > 65535) return fail(P4Q_ERR_UNSUPPORTED, "p4q_select_full: B=%d > 65535", B);
    const size_t need = p4q::select_full_workspace_bytes(B, N, d, J, K);
    if (!ws || ws_bytes < need)
        return fail(P4Q_ERR_WORKSPACE, "p4q_select_full: workspace %zu < %zu bytes", ws_bytes, need);
    if (!aligned(ws, 256)) return fail(P4Q_ERR_INVALID_ARG, "p4q_select_full: workspace not 256-byte aligned");
    const p4q::SelectFullWorkspace w = p4q::select_full_workspace_carve(ws, B, N, d, J, K);
    return hip_status(p4q::launch_select_full(dt, B, N, d, vis, concepts, J, cls_attn, text, T, K, kq, ks,
                                              clip, idx_out, stages_out, tokens_out, w, stream),
                      "p4q_select_full");
}

int p4q_quant_act(p4q_dtype dt, int M, int K_in, const void *x, int64_t ldx, float clip,
                  uint8_t *codes, float *scales, hipStream_t stream) {
    if (!valid_dtype(dt)) return fail(P4Q_ERR_UNSUPPORTED, "p4q_quant_act: dtype %d", (int)dt);
    if (M <= 0 || K_in <= 0) return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_act: M=%d K_in=%d", M, K_in);
    if (K_in % 32 != 0) return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_act: K_in=%d not a multiple of 32", K_in);
    if (K_in > 65536) return fail(P4Q_ERR_UNSUPPORTED, "p4q_quant_act: K_in=%d > 65536", K_in);
    if (ldx < K_in || ldx % 8 != 0)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_act: ldx=%lld (need >= K_in, multiple of 8)", (long long)ldx);
    if (!x || !codes || !scales) return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_act: null pointer");
    if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scales, 4))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_act: misaligned pointer");
    if (!valid_clip(clip)) return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_act: clip %g outside [2^-16, 1]", clip);
    return hip_status(p4q::launch_quant_act(dt, M, K_in, x, ldx, clip, codes, scales, stream),
                      "p4q_quant_act");
}

int p4q_rmsnorm_quant(p4q_dtype dt, int M, int d, const void *x, int64_t ldx, const void *gamma,
                      float eps, float clip, uint8_t *codes, float *scales, hipStream_t stream) {
    if (!valid_dtype(dt)) return fail(P4Q_ERR_UNSUPPORTED, "p4q_rmsnorm_quant: dtype %d", (int)dt);
    if (M <= 0 || d <= 0) return fail(P4Q_ERR_INVALID_ARG, "p4q_rmsnorm_quant: M=%d d=%d", M, d);
    if (d % 32 != 0) return fail(P4Q_ERR_INVALID_ARG, "p4q_rmsnorm_quant: d=%d not a multiple of 32", d);
    if (d > 16384) return fail(P4Q_ERR_UNSUPPORTED, "p4q_rmsnorm_quant: d=%d > 16384", d);
    if (ldx < d || ldx % 8 != 0)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_rmsnorm_quant: ldx=%lld (need >= d, multiple of 8)", (long long)ldx);
    if (!x || !gamma || !codes || !scales) return fail(P4Q_ERR_INVALID_ARG, "p4q_rmsnorm_quant: null pointer");
    if (!aligned(x, 16) || !aligned(gamma, 16) || !aligned(codes, 16) || !aligned(scales, 4))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_rmsnorm_quant: misaligned pointer");
    if (!(eps >= 0.0f && eps <= 1.0f)) return fail(P4Q_ERR_INVALID_ARG, "p4q_rmsnorm_quant: eps %g outside [0, 1]", eps);
    if (!valid_clip(clip)) return fail(P4Q_ERR_INVALID_ARG, "p4q_rmsnorm_quant: clip %g outside [2^-16, 1]", clip);
    return hip_status(p4q::launch_rmsnorm_quant(dt, M, d, x, ldx, gamma, eps, clip, codes, scales, stream),
                      "p4q_rmsnorm_quant");
}

int p4q_attention_prefill(p4q_dtype dt, int B, int L, int H, int D, const void *q, const void *k,
                          const void *v, int64_t ld, void *out, int64_t ld_out, int causal,
                          hipStream_t stream) {
    if (!valid_dtype(dt)) return fail(P4Q_ERR_UNSUPPORTED, "p4q_attention_prefill: dtype %d", (int)dt);
    if (B <= 0 || L <= 0 || H <= 0 || D <= 0)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_attention_prefill: B=%d L=%d H=%d D=%d", B, L, H, D);
    if (D != 128) return fail(P4Q_ERR_UNSUPPORTED, "p4q_attention_prefill: head dimension %d (128 only)", D);
    if (causal != 0 && causal != 1) return fail(P4Q_ERR_INVALID_ARG, "p4q_attention_prefill: causal=%d", causal);
    if (ld < (int64_t)H * D || ld % 8 != 0 || ld_out < (int64_t)H * D || ld_out % 4 != 0)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_attention_prefill: ld=%lld ld_out=%lld (need >= H*D; multiples of 8 / 4)",
                    (long long)ld, (long long)ld_out);
    if (!q || !k || !v || !out) return fail(P4Q_ERR_INVALID_ARG, "p4q_attention_prefill: null pointer");
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 8))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_attention_prefill: misaligned pointer");
    if (B > 65535 || H > 65535 || (int64_t)L * ld * 2 >= (1LL << 31))
        return fail(P4Q_ERR_UNSUPPORTED, "p4q_attention_prefill: B=%d H=%d L=%d ld=%lld too large (L*ld*2 < 2^31)",
                    B, H, L, (long long)ld);
    return hip_status(p4q::launch_attention(dt, B, L, H, q, k, v, ld, out, ld_out, causal, stream),
                      "p4q_attention_prefill");
}

static int calib_block_shape_error(int M, int d, int f, int H) {
    if (M <= 0 || d <= 0 || f <= 0 || H <= 0) return P4Q_ERR_INVALID_ARG;
    if (d % 128 != 0 || f % 128 != 0 || d % H != 0 || (d / H) % 2 != 0) return P4Q_ERR_INVALID_ARG;
    if (M > 4096 || d > 16384 || f > 16384 || (int64_t)M * 2 * f >= (1LL << 31) ||
        (int64_t)3 * d * d >= (1LL << 31) || (int64_t)2 * f * d >= (1LL << 31))
        return P4Q_ERR_UNSUPPORTED;
    return P4Q_OK;
}

size_t p4q_calib_block_workspace_bytes(int M, int d, int f, int H) {
    if (calib_block_shape_error(M, d, f, H) != P4Q_OK) return 0;
    return p4q::calib_block_workspace_bytes(M, d, f, H);
}

int p4q_calib_block_grad(p4q_dtype dt, int M, int d, int f, int H, const void *x,
                         const float *target, int64_t ldt, const void *w_qkv, const void *w_o,
                         const void *w_gu, const void *w_down, const void *gamma1,
                         const void *gamma2, float eps, float rope_base, const float *sigma,
                         const float *clip_a, const float *clip_w, float *loss,
                         float *grad_sigma, float *grad_clip_a, float *grad_clip_w, void *ws,
                         size_t ws_bytes, hipStream_t stream) {
    if (dt != P4Q_FP16) return fail(P4Q_ERR_UNSUPPORTED, "p4q_calib_block_grad: only fp16 blocks");
    if (const int st = calib_block_shape_error(M, d, f, H))
        return fail(st, "p4q_calib_block_grad: M=%d d=%d f=%d H=%d outside the limits", M, d, f, H);
    if (ldt < d) return fail(P4Q_ERR_INVALID_ARG, "p4q_calib_block_grad: ldt=%lld < d", (long long)ldt);
    if (!(eps >= 0.0f && eps <= 1.0f) || !(rope_base > 1.0f))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_calib_block_grad: eps=%g rope_base=%g", (double)eps,
                    (double)rope_base);
    if (!x || !target || !w_qkv || !w_o || !w_gu || !w_down || !gamma1 || !gamma2 || !sigma ||
        !clip_a || !clip_w || !loss || !grad_sigma || !grad_clip_a || !grad_clip_w)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_calib_block_grad: null pointer");
    for (int g = 0; g < 4; ++g)
        if (!(clip_a[g] > 0.0f && clip_a[g] <= 1.0f))
            return fail(P4Q_ERR_INVALID_ARG, "p4q_calib_block_grad: clip_a[%d]=%g outside (0, 1]", g,
                        (double)clip_a[g]);
    const void *ptrs[] = {x, target, w_qkv, w_o, w_gu, w_down, gamma1, gamma2, sigma, clip_w,
                          loss, grad_sigma, grad_clip_a, grad_clip_w};
    for (const void *q : ptrs)
        if (!aligned(q, 16)) return fail(P4Q_ERR_INVALID_ARG, "p4q_calib_block_grad: misaligned pointer");
    if (ldt % 4 != 0) return fail(P4Q_ERR_INVALID_ARG, "p4q_calib_block_grad: ldt not a multiple of 4");
    const size_t need = p4q::calib_block_workspace_bytes(M, d, f, H);
    if (!ws || ws_bytes < need)
        return fail(P4Q_ERR_WORKSPACE, "p4q_calib_block_grad: workspace %zu < %zu bytes", ws_bytes, need);
    if (!aligned(ws, 256)) return fail(P4Q_ERR_INVALID_ARG, "p4q_calib_block_grad: workspace not 256-byte aligned");
    return hip_status(p4q::launch_calib_block(M, d, f, H, x, target, ldt, w_qkv, w_o, w_gu, w_down,
                                              gamma1, gamma2, eps, rope_base, sigma, clip_a, clip_w,
                                              loss, grad_sigma, grad_clip_a, grad_clip_w, ws, stream),
                      "p4q_calib_block_grad");
}

size_t p4q_w4a4_linear_workspace_bytes(int M, int N_out, int K_in) {
    if (M <= 0 || N_out <= 0 || K_in <= 0 || K_in % 32 != 0 || K_in > 131072 ||
        (int64_t)M > 65535LL * 128)
        return 0;
    return p4q::gemm_workspace_bytes(M, N_out, K_in);
}

int p4q_w4a4_linear(int M, int N_out, int K_in, const uint8_t *a_codes, const float *a_scales,
                    const uint8_t *w_codes, const float *w_scales, p4q_dtype out_dt, void *y,
                    int64_t ldy, int32_t *acc_out, void *ws, size_t ws_bytes, hipStream_t stream) {
    if (!valid_dtype(out_dt)) return fail(P4Q_ERR_UNSUPPORTED, "p4q_w4a4_linear: dtype %d", (int)out_dt);
    if (M <= 0 || N_out <= 0 || K_in <= 0)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_w4a4_linear: M=%d N_out=%d K_in=%d", M, N_out, K_in);
    if (K_in % 32 != 0) return fail(P4Q_ERR_INVALID_ARG, "p4q_w4a4_linear: K_in=%d not a multiple of 32", K_in);
    if (K_in > 131072) return fail(P4Q_ERR_UNSUPPORTED, "p4q_w4a4_linear: K_in=%d > 131072", K_in);
    if (ldy < N_out) return fail(P4Q_ERR_INVALID_ARG, "p4q_w4a4_linear: ldy=%lld < N_out", (long long)ldy);
    if (!a_codes || !a_scales || !w_codes || !w_scales || !y)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_w4a4_linear: null pointer");
    if (!aligned(a_codes, 16) || !aligned(w_codes, 16) || !aligned(y, 4) || !aligned(a_scales, 4) ||
        !aligned(w_scales, 4) || (acc_out && !aligned(acc_out, 4)))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_w4a4_linear: misaligned pointer");
    if ((int64_t)M > 65535LL * 128) return fail(P4Q_ERR_UNSUPPORTED, "p4q_w4a4_linear: M too large");
    return hip_status(p4q::launch_w4a4_gemm(M, N_out, K_in, a_codes, a_scales, w_codes, w_scales,
                                            out_dt, y, ldy, acc_out, ws, ws_bytes, stream),
                      "p4q_w4a4_linear");
}

int p4q_quant_scaled(p4q_dtype dt, int R, int K, const void *z, int64_t ldz, const float *sigma,
                     int divide, float clip, const float *clip_rows, uint8_t *codes,
                     float *scales, float *absmax, int32_t *kstar, hipStream_t stream) {
    if (!valid_dtype(dt)) return fail(P4Q_ERR_UNSUPPORTED, "p4q_quant_scaled: dtype %d", (int)dt);
    if (R <= 0 || K <= 0) return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_scaled: R=%d K=%d", R, K);
    if (K % 32 != 0) return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_scaled: K=%d not a multiple of 32", K);
    if (K > 16384) return fail(P4Q_ERR_UNSUPPORTED, "p4q_quant_scaled: K=%d > 16384", K);
    if (ldz < K || ldz % 8 != 0)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_scaled: ldz=%lld (need >= K, multiple of 8)", (long long)ldz);
    if (divide != 0 && divide != 1) return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_scaled: divide=%d", divide);
    if (!clip_rows && !(clip > 0.0f && clip <= 1.0f))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_scaled: clip=%g outside (0, 1]", (double)clip);
    if (!z || !sigma || !codes || !scales) return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_scaled: null pointer");
    if (!aligned(z, 16) || !aligned(sigma, 16) || !aligned(codes, 16) || !aligned(scales, 4) ||
        (clip_rows && !aligned(clip_rows, 4)) || (absmax && !aligned(absmax, 4)) || (kstar && !aligned(kstar, 4)))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_quant_scaled: misaligned pointer");
    return hip_status(p4q::launch_quant_scaled(dt, R, K, z, ldz, sigma, divide, clip, clip_rows, codes,
                                               scales, absmax, kstar, stream),
                      "p4q_quant_scaled");
}

static int calib_shape_error(int M, int N, int K) {
    if (M <= 0 || N <= 0 || K <= 0) return P4Q_ERR_INVALID_ARG;
    if (N % 64 != 0 || K % 128 != 0) return P4Q_ERR_INVALID_ARG;
    if (K > 16384 || M > (1 << 20) || N > (1 << 20) || (int64_t)M * N >= (1LL << 31) ||
        (int64_t)N * K >= (1LL << 31))
        return P4Q_ERR_UNSUPPORTED;
    return P4Q_OK;
}

size_t p4q_calib_linear_workspace_bytes(int M, int N, int K) {
    if (calib_shape_error(M, N, K) != P4Q_OK) return 0;
    return p4q::calib_linear_workspace_bytes(M, N, K);
}

int p4q_calib_linear_grad(p4q_dtype dt, int M, int N, int K, const void *x, int64_t ldx,
                          const void *w, int64_t ldw, const float *target, int64_t ldt,
                          const float *sigma, float clip_a, const float *clip_w, float *loss,
                          float *grad_sigma, float *grad_clip_a, float *grad_clip_w, void *ws,
                          size_t ws_bytes, hipStream_t stream) {
    if (!valid_dtype(dt)) return fail(P4Q_ERR_UNSUPPORTED, "p4q_calib_linear_grad: dtype %d", (int)dt);
    const int se = calib_shape_error(M, N, K);
    if (se != P4Q_OK)
        return fail(se, "p4q_calib_linear_grad: M=%d N=%d K=%d (need N %% 64 == 0, K %% 128 == 0, "
                    "K <= 16384, M*N and N*K < 2^31)", M, N, K);
    if (ldx < K || ldx % 8 != 0 || ldw < K || ldw % 8 != 0 || ldt < N || ldt % 4 != 0)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_calib_linear_grad: ldx=%lld ldw=%lld ldt=%lld",
                    (long long)ldx, (long long)ldw, (long long)ldt);
    if (!(clip_a > 0.0f && clip_a <= 1.0f))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_calib_linear_grad: clip_a=%g outside (0, 1]", (double)clip_a);
    if (!x || !w || !target || !sigma || !clip_w || !loss || !grad_sigma || !grad_clip_a || !grad_clip_w)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_calib_linear_grad: null pointer");
    if (!aligned(x, 16) || !aligned(w, 16) || !aligned(target, 16) || !aligned(sigma, 16) ||
        !aligned(clip_w, 4) || !aligned(loss, 4) || !aligned(grad_sigma, 4) ||
        !aligned(grad_clip_a, 4) || !aligned(grad_clip_w, 4) || (ws && !aligned(ws, 256)))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_calib_linear_grad: misaligned pointer");
    const size_t need = p4q::calib_linear_workspace_bytes(M, N, K);
    if (!ws || ws_bytes < need)
        return fail(P4Q_ERR_WORKSPACE, "p4q_calib_linear_grad: workspace %zu < %zu bytes", ws_bytes, need);
    return hip_status(p4q::launch_calib_linear(dt, M, N, K, x, ldx, w, ldw, target, ldt, sigma, clip_a,
                                               clip_w, loss, grad_sigma, grad_clip_a, grad_clip_w, ws,
                                               stream),
                      "p4q_calib_linear_grad");
}

int p4q_diag_mfma_i8(int blocks, int iters, int32_t *out, hipStream_t stream) {
    if (blocks < 1 || blocks > (1 << 20) || iters < 1 || iters > (1 << 20))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_diag_mfma_i8: blocks=%d iters=%d", blocks, iters);
    if (!out || !aligned(out, 4)) return fail(P4Q_ERR_INVALID_ARG, "p4q_diag_mfma_i8: out");
    return hip_status(p4q::launch_diag_mfma_i8(blocks, iters, out, stream), "p4q_diag_mfma_i8");
}

int p4q_diag_stream_read(const void *src, size_t bytes, int blocks, uint32_t *out,
                         hipStream_t stream) {
    if (blocks < 1 || blocks > (1 << 20) || bytes % 16 != 0 || bytes == 0)
        return fail(P4Q_ERR_INVALID_ARG, "p4q_diag_stream_read: blocks=%d bytes=%zu", blocks, bytes);
    if (!src || !out || !aligned(src, 16) || !aligned(out, 4))
        return fail(P4Q_ERR_INVALID_ARG, "p4q_diag_stream_read: pointer");
    return hip_status(p4q::launch_diag_read(src, bytes, blocks, out, stream), "p4q_diag_stream_read");
}

}  // extern "C"
