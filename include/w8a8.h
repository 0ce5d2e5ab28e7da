/*
 * w8a8.h -- C ABI of libw8a8.so, a fused W8A8 quantized linear for AMD Instinct
 * MI355X (gfx950).
 *
 * The operation (Section 3 of "Realizing Native INT8 Compute for Diffusion
 * Transformers on Consumer GPUs", paragraphs "The quantization recipe (reused)" and
 * "The fused kernel"): a bf16 linear layer Y = X W^T + b, with X [M,K] (M tokens),
 * W [N,K] (N output channels) and b [N], is replaced by
 *   1. per-output-channel int8 weights Wq [N,K] with float32 scales sw [N]
 *      (computed once, offline);
 *   2. per-token dynamic int8 activations Xq [M,K] with float32 scales sx [M]
 *      (computed on every call);
 *   3. the exact product acc = Xq Wq^T in int32 on the int8 matrix cores, whose
 *      epilogue dequantizes off the accumulator and adds the bias:
 *      Y[m][n] = bf16(fmaf((float)acc[m][n], sx[m] * sw[n], b[n])).
 *
 * Quantization of a row v[0..K) (both W and X):
 *   a = max_k |v[k]|, s = a / 127, q[k] = clamp(rne(v[k] * (127 / a)), -127, 127);
 *   every division is a correctly rounded float32 division, rne is round half to even;
 *   a row with a == 0, or with 127/a overflowing float32, gets s = 0 and q = 0.
 *
 * Conventions for every entry point:
 *   - bf16 tensors are passed as their raw 16-bit patterns (uint16_t).
 *   - All matrices are row-major and contiguous with K innermost: X [M,K], W [N,K],
 *     Xq [M,K], Wq [N,K]; Y and acc are [M,N] with N innermost.
 *   - Tensor pointers are device pointers (HIP device memory of the current device);
 *     `stream` is a hipStream_t (NULL = the legacy default stream). All work is
 *     enqueued on `stream`; no call synchronizes, allocates or frees memory.
 *   - The caller owns every buffer. The library keeps no state besides its immutable
 *     kernel and tile tables, so concurrent calls on different streams are safe when
 *     their output and workspace buffers do not overlap.
 *   - Arguments are validated before anything is launched; on a non-zero status
 *     nothing was enqueued (W8A8_ERR_HIP excepted: a launch that HIP rejected).
 *   - M == 0 or N == 0 is a valid no-op. K == 0 is valid: every code is 0, every
 *     scale 0, and Y = b.
 *   - Inputs must be finite; for non-finite X, W or b the results are unspecified.
 *   - Any alignment and any K are accepted; 16-byte aligned operands with K a multiple
 *     of 16 take the fast kernels, others a slower generic kernel with the same results.
 */
#ifndef W8A8_H
#define W8A8_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int w8a8_status;

enum {
    W8A8_OK = 0,
    W8A8_ERR_NULL = 1,        /* a pointer that the sizes make necessary is NULL */
    W8A8_ERR_SHAPE = 2,       /* a negative size, or M*K / N*K / M*N beyond 2^62 */
    W8A8_ERR_K_OVERFLOW = 3,  /* K > W8A8_MAX_K: 127*127*K would not fit int32 */
    W8A8_ERR_HIP = 4,         /* HIP reported an error for a launch */
    W8A8_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than the query returns */
    W8A8_ERR_ARG = 6,         /* another invalid argument (e.g. unknown tile id) */
    W8A8_ERR_SCRATCH = 7      /* w8a8_linear_noalloc: the problem exceeds its scratch */
};

/* Largest K for which |acc| <= 127 * 127 * K fits int32. */
#define W8A8_MAX_K 133144

/* Per-output-channel weight quantization (step 1; offline, once per layer).
 * w: [N,K] bf16. Out: wq [N,K] int8, w_scale [N] float32. */
w8a8_status w8a8_quantize_weight(const uint16_t *w, int64_t N, int64_t K, int8_t *wq,
                                 float *w_scale, void *stream);

/* Per-token dynamic activation quantization (step 2; every forward).
 * x: [M,K] bf16. Out: xq [M,K] int8, x_scale [M] float32. Same rule as above. */
w8a8_status w8a8_quantize_act(const uint16_t *x, int64_t M, int64_t K, int8_t *xq,
                              float *x_scale, void *stream);

/* Fused int8 GEMM + dequantization epilogue (step 3): Y = bf16(fmaf((float)(Xq Wq^T),
 * sx[m] * sw[n], b[n])). bias: [N] bf16 or NULL (no bias). y: [M,N] bf16.
 * workspace: device scratch of at least w8a8_gemm_workspace_bytes(M,N,K) bytes (NULL
 * allowed when that is 0); 256-byte aligned. */
w8a8_status w8a8_gemm(const int8_t *xq, const float *x_scale, const int8_t *wq,
                      const float *w_scale, const uint16_t *bias, uint16_t *y,
                      int64_t M, int64_t N, int64_t K, void *workspace,
                      size_t workspace_bytes, void *stream);

size_t w8a8_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);

/* Workspace of w8a8_gemm_ex with a given tile id (-1: the table's choice). Tiles that
 * split K among several workgroups per output tile keep int32 partial products
 * [splits][M][N] there; the others need none (0). */
size_t w8a8_gemm_workspace_bytes_ex(int64_t M, int64_t N, int64_t K, int tile_id);

/* The whole quantized linear: per-token quantization of x into the workspace, then the
 * fused GEMM (steps 2 and 3). wq / w_scale come from w8a8_quantize_weight.
 * workspace: at least w8a8_linear_workspace_bytes(M,N,K) bytes, 256-byte aligned; it
 * holds Xq [M,K] and sx [M] (and whatever the GEMM needs) and may be reused once the
 * call's work on `stream` has finished. With few tokens (the GEMM tile streams the
 * weight, K % 16 == 0, 16-byte aligned x and wq, and a short quantization per
 * workgroup) quantizer and GEMM run as one launch, each workgroup quantizing its own
 * token rows into LDS with the same arithmetic; the workspace is then left untouched
 * and the result is the same. */
w8a8_status w8a8_linear(const uint16_t *x, const int8_t *wq, const float *w_scale,
                        const uint16_t *bias, uint16_t *y, int64_t M, int64_t N,
                        int64_t K, void *workspace, size_t workspace_bytes,
                        void *stream);

size_t w8a8_linear_workspace_bytes(int64_t M, int64_t N, int64_t K);

/* For callers that cannot allocate (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): w8a8_linear_ex without a workspace argument. The
 * workspace lives in a file-scope device array of W8A8_NOALLOC_SCRATCH_BYTES that each
 * device holds from the library's load until the process ends; the call itself allocates
 * nothing (no hipMalloc, no allocating library routine). Its first call on a device
 * looks up that device's array once (hipGetSymbolAddress), so make it outside graph
 * capture. Problems whose w8a8_linear_workspace_bytes(M,N,K) exceeds the array return
 * W8A8_ERR_SCRATCH before anything is launched (128 MiB holds, e.g., Xq of 4608 tokens
 * at K = 16384). Every call on a device shares that device's array and leaves its
 * contents behind (nothing in it needs to start at zero): calls that overlap on one
 * device, on different streams or from different threads, race and give undefined
 * results. Arguments and results are those of w8a8_linear_ex. */
#define W8A8_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
w8a8_status w8a8_linear_noalloc(const uint16_t *x, int act, const float *col_mul,
                                const int8_t *wq, const float *w_scale,
                                const uint16_t *bias, uint16_t *y, int64_t M, int64_t N,
                                int64_t K, void *stream);

/* 1 if w8a8_linear runs quantizer and GEMM as one launch for this shape when x and wq
 * are 16-byte aligned (the few-token path above; its token block, codes and scales,
 * must fit the workgroup's LDS beside the tile's own), else 0. A pure host query: it
 * launches nothing and needs no device. */
int w8a8_linear_one_launch(int64_t M, int64_t N, int64_t K);

/* Debug: the raw int32 accumulator acc [M,N] = Xq Wq^T, with no epilogue. It is the
 * exactness check the paper runs against a library integer matmul (Section 5,
 * "The kernel is exact and the GEMMs are compute-bound"). */
w8a8_status w8a8_gemm_acc_i32(const int8_t *xq, const int8_t *wq, int32_t *acc,
                              int64_t M, int64_t N, int64_t K, void *stream);

/* Tile configurations (the per-shape table chosen offline, Section 3, "Why
 * autotuning is load-bearing"). w8a8_select_tile returns the id the table picks for a
 * shape (M within an entry's token range, N and K equal), else the fallback rule's;
 * w8a8_default_tile returns the fallback rule's choice alone, the untuned arm of the
 * tuning ablation. Both return -1 for M <= 0, N <= 0 or K < 0. The _ex variants run a
 * given id (-1 = the table's choice) for offline sweeps and tests. An id outside
 * [0, w8a8_tile_count()) returns W8A8_ERR_ARG. Tiles whose name ends in _k<s> divide K
 * among s workgroups per output tile and sum the int32 partials in a second kernel (the
 * result is the same: integer sums are exact); w8a8_gemm_acc_i32[_ex] runs them
 * unsplit. */
int w8a8_tile_count(void);
const char *w8a8_tile_name(int tile_id);
int w8a8_select_tile(int64_t M, int64_t N, int64_t K);
int w8a8_default_tile(int64_t M, int64_t N, int64_t K);

w8a8_status w8a8_gemm_ex(const int8_t *xq, const float *x_scale, const int8_t *wq,
                         const float *w_scale, const uint16_t *bias, uint16_t *y,
                         int64_t M, int64_t N, int64_t K, void *workspace,
                         size_t workspace_bytes, int tile_id, void *stream);

w8a8_status w8a8_gemm_acc_i32_ex(const int8_t *xq, const int8_t *wq, int32_t *acc,
                                 int64_t M, int64_t N, int64_t K, int tile_id,
                                 void *stream);

/* ---- Transformed activations and SmoothQuant (Section 3, "The quantization recipe
 * (reused)": per-channel int8 weights, per-token dynamic int8 activations, and
 * SmoothQuant with alpha = 0.5).
 *
 * SmoothQuant moves quantization difficulty from activations to weights per input
 * channel k: X is multiplied by smooth_inv[k] = 1 / s[k] and W by s[k], which leaves
 * X W^T unchanged, with s[k] = max|X[:,k]|^alpha / max|W[:,k]|^(1 - alpha) calibrated
 * offline. The weight side is folded once (w8a8_quantize_weight_ex); the activation
 * side is a multiply inside the per-token quantizer, so it costs no pass over X.
 *
 * act selects a transform T applied to the bf16 input before the multiplier:
 *   W8A8_ACT_NONE  T(x) = x
 *   W8A8_ACT_GELU  T(x) = x * Phi(x), the exact (erf) GELU, evaluated in float32
 *                  through a Chebyshev fit of erfc (Numerical Recipes' erfcc,
 *                  fractional error < 1.2e-7) on the hardware reciprocal and exp2:
 *                  relative error about 3e-7 where |x| < 4, growing in the far left
 *                  tail with the float32 rounding of x^2 / 2 (there GELU(x) is below
 *                  1e-4 |x|). It feeds the MLP down-projection from the
 *                  pre-activation, with no GELU pass of its own.
 * The quantizer then applies the row rule above to v[k] = T(x[k]) * col_mul[k]
 * (float32 multiply; col_mul NULL means no multiplier). Any other act value returns
 * W8A8_ERR_ARG. */
#define W8A8_ACT_NONE 0
#define W8A8_ACT_GELU 1

/* Per-token quantization of T(x) * col_mul. x: [M,K] bf16; col_mul: [K] float32 or
 * NULL. Out: xq [M,K] int8, x_scale [M] float32. */
w8a8_status w8a8_quantize_act_ex(const uint16_t *x, int64_t M, int64_t K, int act,
                                 const float *col_mul, int8_t *xq, float *x_scale,
                                 void *stream);

/* Per-output-channel quantization of w[n][k] * col_mul[k] (the SmoothQuant fold; col_mul
 * = s, or NULL for the plain rule). w: [N,K] bf16. Out: wq [N,K], w_scale [N]. */
w8a8_status w8a8_quantize_weight_ex(const uint16_t *w, int64_t N, int64_t K,
                                    const float *col_mul, int8_t *wq, float *w_scale,
                                    void *stream);

/* w8a8_linear on T(x) * col_mul: for a smoothed layer col_mul = smooth_inv and wq was
 * quantized with col_mul = smooth. Same workspace as w8a8_linear. */
w8a8_status w8a8_linear_ex(const uint16_t *x, int act, const float *col_mul,
                           const int8_t *wq, const float *w_scale, const uint16_t *bias,
                           uint16_t *y, int64_t M, int64_t N, int64_t K, void *workspace,
                           size_t workspace_bytes, void *stream);

/* Calibration: amax[k] = max over the R rows of |T(v[r][k])| (float32). With
 * accumulate != 0 the result is merged (max) into amax's current contents, so several
 * calibration batches can be folded in; otherwise amax is overwritten. v: [R,K] bf16
 * (activations, or W itself for the weight maxima). amax: [K] float32. */
w8a8_status w8a8_col_absmax(const uint16_t *v, int64_t R, int64_t K, int act, float *amax,
                            int accumulate, void *stream);

/* SmoothQuant factors from calibrated maxima: smooth[k] = x_amax^alpha /
 * w_amax^(1 - alpha), smooth_inv[k] = 1.0f / smooth[k]. alpha = 0.5 (the recipe's
 * value) computes sqrtf(x_amax) / sqrtf(w_amax), each step correctly rounded; other
 * alpha use powf. A channel whose maxima are not both positive and finite, or whose
 * factor is 0 or infinite, gets smooth = 1. alpha outside [0, 1] returns
 * W8A8_ERR_ARG. All arrays [K] float32 on the device. */
w8a8_status w8a8_smooth_factors(const float *x_amax, const float *w_amax, int64_t K,
                                float alpha, float *smooth, float *smooth_inv,
                                void *stream);

/* ---- Measurement aid (not part of the linear): the int8 matrix-core ceiling on given
 * operands. The sustained rate of v_mfma_i32_32x32x32_i8 depends on the operand bits
 * (the clock drops under the matrix cores' switching power), so the datasheet peak is
 * not reachable on every input. This call replays the GEMM's per-K-step MFMA sequence
 * of its 160 x 256 tile (per wavefront, 2 weight x 5 token fragments) on fragments of
 * xq [M,K] and wq [N,K] held in registers: 256 workgroups of 4 wavefronts, each loading
 * 8 K-steps of its tile's fragments (rows and channels wrapped modulo M and N), then
 * `iters` sweeps over them with no memory traffic. Its rate, w8a8_mfma_ceiling_ops(iters)
 * / launch time, is the matrix-core ceiling for these codes.
 *   wave_sums: [1024] uint32 on the device; wavefront w of workgroup b writes entry
 *              4b + w, the sum of its accumulator elements modulo 2^32 (a checksum).
 * Needs K % 32 == 0 (else W8A8_ERR_SHAPE), 16-byte aligned xq and wq and 1 <= iters <=
 * W8A8_CEILING_MAX_ITERS (else W8A8_ERR_ARG). w8a8_mfma_ceiling_ops returns the int8
 * ops (2 per multiply-accumulate) of one launch, or -1 for iters out of range. */
#define W8A8_CEILING_MAX_ITERS 1000000
int64_t w8a8_mfma_ceiling_ops(int64_t iters);
w8a8_status w8a8_mfma_ceiling(const int8_t *xq, const int8_t *wq, int64_t M, int64_t N,
                              int64_t K, int64_t iters, uint32_t *wave_sums, void *stream);

/* ---- Measurement aid (not part of the linear): the HBM read ceiling for a byte count.
 * A weight-streaming GEMM with few tokens is bound by reading Wq once; the rate HBM
 * delivers for a read of that size (with its ramp and drain) is below the datasheet's
 * 8 TB/s, and this call measures it: a plain streaming read of `bytes` bytes at p
 * (device memory, 16-byte aligned) by W8A8_READ_BLOCKS workgroups, workgroup b reading
 * the b-th contiguous chunk of bytes / W8A8_READ_BLOCKS bytes and writing the XOR of its
 * 32-bit words to sums[b] (uint32 [W8A8_READ_BLOCKS] on the device; a checksum, so the
 * reads cannot be elided). bytes must be a positive multiple of 16 * W8A8_READ_BLOCKS
 * (else W8A8_ERR_SHAPE); a misaligned p or sums returns W8A8_ERR_ARG. */
#define W8A8_READ_BLOCKS 2048
w8a8_status w8a8_read_ceiling(const void *p, int64_t bytes, uint32_t *sums, void *stream);

/* Static description of a status code. */
const char *w8a8_status_string(w8a8_status status);

/* Library version string. */
const char *w8a8_version(void);

#ifdef __cplusplus
}
#endif

#endif /* W8A8_H */
