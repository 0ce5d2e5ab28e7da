// Internal declarations shared by the HIP translation units of libw8a8.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace w8a8 {

// ---------------------------------------------------------------- quantizer
enum Act : int { ACT_NONE = 0, ACT_GELU = 1 };

// Launches the per-row absmax quantizer over a [rows, K] bf16 matrix on `stream`, on
// the values T(x) * colmul[k] (T = identity or GELU; colmul [K] float32 or nullptr).
// Returns hipSuccess or the launch error.
hipError_t launch_quant_rows(const uint16_t *v, int64_t rows, int64_t K, int act,
                             const float *colmul, int8_t *q, float *scale,
                             hipStream_t stream);
// Per-column max |T(x)| of a [rows, K] bf16 matrix into amax [K] (merged with its
// current contents when `accumulate`, else replacing them).
hipError_t launch_col_absmax(const uint16_t *v, int64_t rows, int64_t K, int act,
                             float *amax, bool accumulate, hipStream_t stream);
// SmoothQuant factors and their reciprocals from per-channel maxima of X and W.
hipError_t launch_smooth_factors(const float *ax, const float *aw, int64_t K, float alpha,
                                 float *smooth, float *smooth_inv, hipStream_t stream);

// ---------------------------------------------------------------- GEMM
enum Epilogue : int { EPI_BF16 = 0, EPI_I32 = 1 };

struct GemmArgs {
    const int8_t *xq;       // [M,K]
    const int8_t *wq;       // [N,K]
    const float *sx;        // [M]   (EPI_BF16)
    const float *sw;        // [N]   (EPI_BF16)
    const uint16_t *bias;   // [N] or nullptr
    void *out;              // [M,N] bf16 or int32
    int64_t M, N, K;
};

struct TileInfo {
    const char *name;
    int tm, tn, bk;      // workgroup tile (tokens x channels x K step)
    int threads;         // workgroup size
    int lds_bytes;       // static LDS per workgroup
    int ksplit;          // K divided among this many workgroups per tile (1: no split)
    int base;            // for a split tile, the id of the same tile unsplit (else -1)
    int streaming;       // 1: the weight-streaming kernel for few tokens
};

int tile_count();
const TileInfo *tile_info(int id);
// Table lookup of the tile id for a shape (offline-chosen, with a fallback rule).
int select_tile(int64_t M, int64_t N, int64_t K);
// The fallback rule alone (what a shape gets without a table entry).
int default_tile(int64_t M, int64_t N, int64_t K);
// Extra device scratch a tile needs for a shape: the int32 partial products of a split
// tile (splits x M x N x 4 bytes), 0 for the others.
size_t tile_workspace_bytes(int id, int64_t M, int64_t N, int64_t K);
// Launch tile `id` with epilogue `epi`; `vec` selects the 16-byte-aligned load path.
hipError_t launch_gemm(int id, Epilogue epi, bool vec, const GemmArgs &a, void *ws,
                       size_t ws_bytes, hipStream_t stream);

// The small fused linear: quantizer and GEMM in one launch, for shapes whose chosen tile
// is a weight-streaming one and whose token blocks are small enough to be quantized by
// every workgroup that uses them (plain rule only: no transform, no multiplier).
bool linear_small_applies(int64_t M, int64_t N, int64_t K, const void *x, const void *wq);
// The shape part of that rule (operands assumed 16-byte aligned).
bool linear_small_shape(int64_t M, int64_t N, int64_t K);
hipError_t launch_linear_small(const uint16_t *x, const int8_t *wq, const float *sw,
                               const uint16_t *bias, uint16_t *y, int64_t M, int64_t N,
                               int64_t K, hipStream_t stream);

// ---------------------------------------------------------------- measurement aid
// Int8 ops (2 per multiply-accumulate) of one launch of the matrix-core ceiling kernel.
int64_t mfma_ceiling_ops(int64_t iters);
// The GEMM's MFMA sequence replayed from registers on fragments of xq / wq (K % 32 == 0,
// 16-byte aligned), iters sweeps; one uint32 checksum per wavefront into wave_sums[1024].
hipError_t launch_mfma_ceiling(const int8_t *xq, const int8_t *wq, int64_t M, int64_t N,
                               int64_t K, int iters, uint32_t *wave_sums, hipStream_t s);

// Plain streaming read of `bytes` bytes (a multiple of 16 * kReadBlocks) at p: workgroup
// b of kReadBlocks XORs the 32-bit words of the b-th contiguous chunk into sums[b].
constexpr int kReadBlocks = 2048;
hipError_t launch_read_ceiling(const void *p, int64_t bytes, uint32_t *sums, hipStream_t s);

}  // namespace w8a8
