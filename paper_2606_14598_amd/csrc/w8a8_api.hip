// C ABI of libw8a8.so: argument validation, tile selection and launches on the
// caller's stream. Nothing here allocates, frees or synchronizes.
#include "../../include/w8a8.h"
#include "w8a8_internal.hpp"

#include <mutex>

namespace {

using namespace w8a8;

constexpr int64_t kMaxElems = int64_t(1) << 62;
constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool product_ok(int64_t a, int64_t b) { return a == 0 || b <= kMaxElems / a; }

hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

w8a8_status from_hip(hipError_t e) { return e == hipSuccess ? W8A8_OK : W8A8_ERR_HIP; }

bool aligned16(const void *p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }

static_assert(W8A8_ACT_NONE == ACT_NONE && W8A8_ACT_GELU == ACT_GELU, "act codes");

bool act_ok(int act) { return act == W8A8_ACT_NONE || act == W8A8_ACT_GELU; }

w8a8_status check_quant(const void *v, int64_t rows, int64_t K, const void *q,
                        const void *scale) {
    if (rows < 0 || K < 0 || !product_ok(rows, K))
        return W8A8_ERR_SHAPE;
    if (rows > 0 && !scale)
        return W8A8_ERR_NULL;
    if (rows > 0 && K > 0 && (!v || !q))
        return W8A8_ERR_NULL;
    return W8A8_OK;
}

w8a8_status check_gemm(const int8_t *xq, const int8_t *wq, const void *out, int64_t M,
                       int64_t N, int64_t K) {
    if (M < 0 || N < 0 || K < 0 || !product_ok(M, K) || !product_ok(N, K) ||
        !product_ok(M, N))
        return W8A8_ERR_SHAPE;
    if (K > W8A8_MAX_K)
        return W8A8_ERR_K_OVERFLOW;
    if (M == 0 || N == 0)
        return W8A8_OK;
    if (!out)
        return W8A8_ERR_NULL;
    if (K > 0 && (!xq || !wq))
        return W8A8_ERR_NULL;
    // Tile offsets inside one workgroup's panel are 32-bit (TN * K bytes < 2^31).
    return W8A8_OK;
}

w8a8_status run_gemm(const int8_t *xq, const float *sx, const int8_t *wq, const float *sw,
                     const uint16_t *bias, void *out, Epilogue epi, int64_t M, int64_t N,
                     int64_t K, void *ws, size_t ws_bytes, int tile_id, hipStream_t s) {
    if (tile_id < -1 || tile_id >= tile_count())
        return W8A8_ERR_ARG;
    if (M == 0 || N == 0)
        return W8A8_OK;
    const int id = tile_id >= 0 ? tile_id : select_tile(M, N, K);
    const size_t need = tile_workspace_bytes(id, M, N, K);
    if (need > 0 && (ws == nullptr || ws_bytes < need))
        return W8A8_ERR_WORKSPACE;
    GemmArgs a;
    a.xq = xq;
    a.wq = wq;
    a.sx = sx;
    a.sw = sw;
    a.bias = bias;
    a.out = out;
    a.M = M;
    a.N = N;
    a.K = K;
    const bool vec = (K % 16 == 0) && aligned16(xq) && aligned16(wq);
    return from_hip(launch_gemm(id, epi, vec, a, ws, ws_bytes, s));
}

// Scratch of w8a8_linear_noalloc: Xq, sx and the GEMM's split-K partials, laid out as
// in w8a8_linear's workspace. Each device holds its own copy from the time the library's
// code object is loaded onto it until the process ends. In host code `scratch` names a
// host-side shadow, not device memory: kernels get the address hipGetSymbolAddress
// returns for the current device, never the name itself.
static __device__ __align__(256) char scratch[W8A8_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address, looked up once per device (with that device
// current) and kept.
hipError_t scratch_for_current_device(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        if (!p || reinterpret_cast<uintptr_t>(p) % kAlign != 0)
            return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

#pragma GCC visibility push(default)
extern "C" {

w8a8_status w8a8_quantize_weight_ex(const uint16_t *w, int64_t N, int64_t K,
                                    const float *col_mul, int8_t *wq, float *w_scale,
                                    void *stream) {
    const w8a8_status st = check_quant(w, N, K, wq, w_scale);
    if (st != W8A8_OK)
        return st;
    return from_hip(launch_quant_rows(w, N, K, ACT_NONE, col_mul, wq, w_scale,
                                      as_stream(stream)));
}

w8a8_status w8a8_quantize_weight(const uint16_t *w, int64_t N, int64_t K, int8_t *wq,
                                 float *w_scale, void *stream) {
    return w8a8_quantize_weight_ex(w, N, K, nullptr, wq, w_scale, stream);
}

w8a8_status w8a8_quantize_act_ex(const uint16_t *x, int64_t M, int64_t K, int act,
                                 const float *col_mul, int8_t *xq, float *x_scale,
                                 void *stream) {
    if (!act_ok(act))
        return W8A8_ERR_ARG;
    const w8a8_status st = check_quant(x, M, K, xq, x_scale);
    if (st != W8A8_OK)
        return st;
    return from_hip(launch_quant_rows(x, M, K, act, col_mul, xq, x_scale, as_stream(stream)));
}

w8a8_status w8a8_quantize_act(const uint16_t *x, int64_t M, int64_t K, int8_t *xq,
                              float *x_scale, void *stream) {
    return w8a8_quantize_act_ex(x, M, K, W8A8_ACT_NONE, nullptr, xq, x_scale, stream);
}

w8a8_status w8a8_col_absmax(const uint16_t *v, int64_t R, int64_t K, int act, float *amax,
                            int accumulate, void *stream) {
    if (!act_ok(act))
        return W8A8_ERR_ARG;
    if (R < 0 || K < 0 || !product_ok(R, K))
        return W8A8_ERR_SHAPE;
    if (K > 0 && (!amax || (R > 0 && !v)))
        return W8A8_ERR_NULL;
    return from_hip(launch_col_absmax(v, R, K, act, amax, accumulate != 0, as_stream(stream)));
}

w8a8_status w8a8_smooth_factors(const float *x_amax, const float *w_amax, int64_t K,
                                float alpha, float *smooth, float *smooth_inv,
                                void *stream) {
    if (!(alpha >= 0.0f && alpha <= 1.0f))
        return W8A8_ERR_ARG;
    if (K < 0)
        return W8A8_ERR_SHAPE;
    if (K > 0 && (!x_amax || !w_amax || !smooth || !smooth_inv))
        return W8A8_ERR_NULL;
    return from_hip(launch_smooth_factors(x_amax, w_amax, K, alpha, smooth, smooth_inv,
                                          as_stream(stream)));
}

size_t w8a8_gemm_workspace_bytes_ex(int64_t M, int64_t N, int64_t K, int tile_id) {
    if (M <= 0 || N <= 0 || K < 0 || K > W8A8_MAX_K || tile_id < -1 ||
        tile_id >= tile_count() || !product_ok(M, N))
        return 0;
    return tile_workspace_bytes(tile_id >= 0 ? tile_id : select_tile(M, N, K), M, N, K);
}

size_t w8a8_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    return w8a8_gemm_workspace_bytes_ex(M, N, K, -1);
}

w8a8_status w8a8_gemm_ex(const int8_t *xq, const float *x_scale, const int8_t *wq,
                         const float *w_scale, const uint16_t *bias, uint16_t *y,
                         int64_t M, int64_t N, int64_t K, void *workspace,
                         size_t workspace_bytes, int tile_id, void *stream) {
    w8a8_status st = check_gemm(xq, wq, y, M, N, K);
    if (st != W8A8_OK)
        return st;
    if (M > 0 && N > 0 && (!x_scale || !w_scale))
        return W8A8_ERR_NULL;
    return run_gemm(xq, x_scale, wq, w_scale, bias, y, EPI_BF16, M, N, K, workspace,
                    workspace_bytes, tile_id, as_stream(stream));
}

w8a8_status w8a8_gemm(const int8_t *xq, const float *x_scale, const int8_t *wq,
                      const float *w_scale, const uint16_t *bias, uint16_t *y,
                      int64_t M, int64_t N, int64_t K, void *workspace,
                      size_t workspace_bytes, void *stream) {
    return w8a8_gemm_ex(xq, x_scale, wq, w_scale, bias, y, M, N, K, workspace,
                        workspace_bytes, -1, stream);
}

size_t w8a8_linear_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    if (M <= 0 || N < 0 || K < 0 || !product_ok(M, K))
        return 0;
    return align_up((size_t)(M * K)) + align_up((size_t)M * sizeof(float)) +
           w8a8_gemm_workspace_bytes(M, N, K);
}

w8a8_status w8a8_linear_ex(const uint16_t *x, int act, const float *col_mul,
                           const int8_t *wq, const float *w_scale, const uint16_t *bias,
                           uint16_t *y, int64_t M, int64_t N, int64_t K, void *workspace,
                           size_t workspace_bytes, void *stream) {
    if (!act_ok(act))
        return W8A8_ERR_ARG;
    if (M < 0 || N < 0 || K < 0 || !product_ok(M, K) || !product_ok(N, K) ||
        !product_ok(M, N))
        return W8A8_ERR_SHAPE;
    if (K > W8A8_MAX_K)
        return W8A8_ERR_K_OVERFLOW;
    if (M == 0 || N == 0)
        return W8A8_OK;
    if (!y || !w_scale || (K > 0 && (!x || !wq)))
        return W8A8_ERR_NULL;
    const size_t need = w8a8_linear_workspace_bytes(M, N, K);
    if (!workspace || workspace_bytes < need)
        return W8A8_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0)
        return W8A8_ERR_WORKSPACE;
    int8_t *xq = static_cast<int8_t *>(workspace);
    float *sx = reinterpret_cast<float *>(static_cast<char *>(workspace) +
                                          align_up((size_t)(M * K)));
    char *gws = reinterpret_cast<char *>(sx) + align_up((size_t)M * sizeof(float));
    hipStream_t s = as_stream(stream);
    // Few tokens, plain rule: quantizer and GEMM in one launch (the workspace is unused).
    if (act == W8A8_ACT_NONE && !col_mul && linear_small_applies(M, N, K, x, wq))
        return from_hip(launch_linear_small(x, wq, w_scale, bias, y, M, N, K, s));
    hipError_t e = launch_quant_rows(x, M, K, act, col_mul, xq, sx, s);
    if (e != hipSuccess)
        return W8A8_ERR_HIP;
    return run_gemm(xq, sx, wq, w_scale, bias, y, EPI_BF16, M, N, K, gws,
                    workspace_bytes - (size_t)(gws - static_cast<char *>(workspace)), -1, s);
}

w8a8_status w8a8_linear(const uint16_t *x, const int8_t *wq, const float *w_scale,
                        const uint16_t *bias, uint16_t *y, int64_t M, int64_t N,
                        int64_t K, void *workspace, size_t workspace_bytes,
                        void *stream) {
    return w8a8_linear_ex(x, W8A8_ACT_NONE, nullptr, wq, w_scale, bias, y, M, N, K,
                          workspace, workspace_bytes, stream);
}

w8a8_status w8a8_linear_noalloc(const uint16_t *x, int act, const float *col_mul,
                                const int8_t *wq, const float *w_scale,
                                const uint16_t *bias, uint16_t *y, int64_t M, int64_t N,
                                int64_t K, void *stream) {
    // The same checks as w8a8_linear_ex, then the size limit, all before any HIP call.
    if (!act_ok(act))
        return W8A8_ERR_ARG;
    if (M < 0 || N < 0 || K < 0 || !product_ok(M, K) || !product_ok(N, K) ||
        !product_ok(M, N))
        return W8A8_ERR_SHAPE;
    if (K > W8A8_MAX_K)
        return W8A8_ERR_K_OVERFLOW;
    if (M == 0 || N == 0)
        return W8A8_OK;
    if (!y || !w_scale || (K > 0 && (!x || !wq)))
        return W8A8_ERR_NULL;
    const size_t need = w8a8_linear_workspace_bytes(M, N, K);
    if (need > W8A8_NOALLOC_SCRATCH_BYTES)
        return W8A8_ERR_SCRATCH;
    void *ptr = nullptr;
    if (scratch_for_current_device(&ptr) != hipSuccess)
        return W8A8_ERR_HIP;
    return w8a8_linear_ex(x, act, col_mul, wq, w_scale, bias, y, M, N, K, ptr,
                          W8A8_NOALLOC_SCRATCH_BYTES, stream);
}

w8a8_status w8a8_gemm_acc_i32_ex(const int8_t *xq, const int8_t *wq, int32_t *acc,
                                 int64_t M, int64_t N, int64_t K, int tile_id,
                                 void *stream) {
    const w8a8_status st = check_gemm(xq, wq, acc, M, N, K);
    if (st != W8A8_OK)
        return st;
    if (tile_id < -1 || tile_id >= tile_count())
        return W8A8_ERR_ARG;
    if (M == 0 || N == 0)
        return W8A8_OK;
    int id = tile_id >= 0 ? tile_id : select_tile(M, N, K);
    // The debug accumulator has no workspace: a split tile runs unsplit.
    if (tile_info(id)->base >= 0)
        id = tile_info(id)->base;
    if (tile_workspace_bytes(id, M, N, K) > 0)
        return W8A8_ERR_ARG;
    return run_gemm(xq, nullptr, wq, nullptr, nullptr, acc, EPI_I32, M, N, K, nullptr, 0,
                    id, as_stream(stream));
}

w8a8_status w8a8_gemm_acc_i32(const int8_t *xq, const int8_t *wq, int32_t *acc,
                              int64_t M, int64_t N, int64_t K, void *stream) {
    return w8a8_gemm_acc_i32_ex(xq, wq, acc, M, N, K, -1, stream);
}

int w8a8_linear_one_launch(int64_t M, int64_t N, int64_t K) {
    if (M <= 0 || N <= 0 || K < 0 || K > W8A8_MAX_K || !product_ok(M, K) ||
        !product_ok(N, K) || !product_ok(M, N))
        return 0;
    return linear_small_shape(M, N, K) ? 1 : 0;
}

int w8a8_tile_count(void) { return tile_count(); }

const char *w8a8_tile_name(int tile_id) {
    const TileInfo *t = tile_info(tile_id);
    return t ? t->name : nullptr;
}

int w8a8_select_tile(int64_t M, int64_t N, int64_t K) {
    if (M <= 0 || N <= 0 || K < 0)
        return -1;
    return select_tile(M, N, K);
}

int w8a8_default_tile(int64_t M, int64_t N, int64_t K) {
    if (M <= 0 || N <= 0 || K < 0)
        return -1;
    return default_tile(M, N, K);
}

const char *w8a8_status_string(w8a8_status status) {
    switch (status) {
    case W8A8_OK: return "ok";
    case W8A8_ERR_NULL: return "a required pointer is NULL";
    case W8A8_ERR_SHAPE: return "invalid shape (negative size or element count overflow)";
    case W8A8_ERR_K_OVERFLOW: return "K too large: 127*127*K does not fit int32";
    case W8A8_ERR_HIP: return "HIP launch error";
    case W8A8_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case W8A8_ERR_ARG: return "invalid argument";
    case W8A8_ERR_SCRATCH:
        return "problem needs more than the no-allocation entry point's scratch";
    default: return "unknown status";
    }
}

int64_t w8a8_mfma_ceiling_ops(int64_t iters) {
    return iters < 1 || iters > W8A8_CEILING_MAX_ITERS ? -1 : mfma_ceiling_ops(iters);
}

w8a8_status w8a8_mfma_ceiling(const int8_t *xq, const int8_t *wq, int64_t M, int64_t N,
                              int64_t K, int64_t iters, uint32_t *wave_sums, void *stream) {
    if (!xq || !wq || !wave_sums)
        return W8A8_ERR_NULL;
    if (M < 1 || N < 1 || K < 32 || K % 32 != 0 || !product_ok(M, K) || !product_ok(N, K))
        return W8A8_ERR_SHAPE;
    if (K > W8A8_MAX_K)
        return W8A8_ERR_K_OVERFLOW;
    if (iters < 1 || iters > W8A8_CEILING_MAX_ITERS || !aligned16(xq) || !aligned16(wq) ||
        reinterpret_cast<uintptr_t>(wave_sums) % 4 != 0)
        return W8A8_ERR_ARG;
    return from_hip(launch_mfma_ceiling(xq, wq, M, N, K, (int)iters, wave_sums,
                                        as_stream(stream)));
}

w8a8_status w8a8_read_ceiling(const void *p, int64_t bytes, uint32_t *sums, void *stream) {
    if (!p || !sums)
        return W8A8_ERR_NULL;
    if (bytes < 16 * kReadBlocks || bytes % (16 * kReadBlocks) != 0)
        return W8A8_ERR_SHAPE;
    if (!aligned16(p) || reinterpret_cast<uintptr_t>(sums) % 4 != 0)
        return W8A8_ERR_ARG;
    return from_hip(launch_read_ceiling(p, bytes, sums, as_stream(stream)));
}

const char *w8a8_version(void) { return "w8a8-gfx950 0.1.0"; }

}  // extern "C"
#pragma GCC visibility pop
