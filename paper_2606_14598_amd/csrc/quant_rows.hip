// Per-row symmetric absmax int8 quantizer for gfx950.
//
// One rule serves both operands of the W8A8 linear (Section 3, "The quantization
// recipe (reused)"): per output channel for the weight W [N,K] (offline) and per token
// for the activation X [M,K] (online, every forward; "The fused kernel"). For a row v:
//   a = max_k |v[k]|, s = a / 127, q[k] = clamp(rne(v[k] * (127 / a)), -127, 127),
// and a row with a == 0 or with 127/a overflowing float32 gets s = 0, q = 0.
//
// The kernel is HBM-bound (3 bytes moved per element: 2 read, 1 written). Rows whose
// K fits the register file are read once with 16-byte loads, kept in VGPRs for the
// second (quantizing) pass and written with 8-byte stores, by a persistent grid that
// prefetches the next rows while it finishes the current ones; the row maximum is taken
// on the bf16 bit patterns (|v| ordered as an unsigned integer, exact for finite values)
// with a wavefront butterfly and, for 256-thread rows, one LDS exchange.
#include "w8a8_internal.hpp"

namespace w8a8 {
namespace {

__device__ __forceinline__ float bf16_to_f32(uint32_t h) {
    return __uint_as_float(h << 16);
}

// Largest |v| bit pattern among the 8 bf16 values in a 16-byte vector.
__device__ __forceinline__ uint32_t absmax8(uint4 d) {
    uint32_t w[4] = {d.x, d.y, d.z, d.w};
    uint32_t m = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t lo = w[i] & 0x7FFFu, hi = (w[i] >> 16) & 0x7FFFu;
        m = max(m, max(lo, hi));
    }
    return m;
}

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        v = max(v, (uint32_t)__shfl_xor((int)v, off, 64));
    return v;
}

// Code of one element: clamp(rne(v * inv), -127, 127) as a byte. inv is 0 for a zero
// row, which yields a zero code (never 0 * inf).
__device__ __forceinline__ uint32_t code(uint32_t h, float inv) {
    float p = bf16_to_f32(h) * inv;
    float r = __builtin_rintf(p);
    r = fminf(fmaxf(r, -127.0f), 127.0f);
    return (uint32_t)((int)r) & 0xFFu;
}

// 8 codes of a 16-byte bf16 vector packed into 8 bytes.
__device__ __forceinline__ uint2 code8(uint4 d, float inv) {
    uint32_t w[4] = {d.x, d.y, d.z, d.w};
    uint32_t c[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        c[2 * i] = code(w[i] & 0xFFFFu, inv);
        c[2 * i + 1] = code(w[i] >> 16, inv);
    }
    uint2 o;
    o.x = c[0] | (c[1] << 8) | (c[2] << 16) | (c[3] << 24);
    o.y = c[4] | (c[5] << 8) | (c[6] << 16) | (c[7] << 24);
    return o;
}

struct RowScale {
    float inv;    // 127 / a, or 0 for a zero row
    float scale;  // a / 127, or 0 for a zero row
};

__device__ __forceinline__ RowScale row_scale(uint32_t amax_bits) {
    float a = bf16_to_f32(amax_bits);
    float inv = 127.0f / a;     // correctly rounded (no fast-math)
    float s = a / 127.0f;
    bool zero = !(a > 0.0f) || !__builtin_isfinite(inv);
    RowScale r;
    r.inv = zero ? 0.0f : inv;
    r.scale = zero ? 0.0f : s;
    return r;
}

// Register-resident path, persistent and software-pipelined: TPR threads per row
// (64 = one wavefront, 256 = the block), NV 16-byte vectors per thread (K % 8 == 0,
// v 16-byte and q 8-byte aligned). Row group j of a block holds rows j*RPB .. j*RPB +
// RPB - 1; block b handles row groups b, b + G, b + 2G, ... (G = gridDim.x) and loads
// group j + G while it reduces, quantizes and stores group j, so the HBM reads of the
// next rows overlap the work and the stores of the current ones.
template <int TPR, int NV>
__global__ void __launch_bounds__(256)
quant_rows_reg(const uint16_t *__restrict__ v, int64_t rows, int64_t K,
               int8_t *__restrict__ q, float *__restrict__ scale) {
    constexpr int RPB = 256 / TPR;
    const int t = threadIdx.x % TPR;
    const int sub = threadIdx.x / TPR;
    const int64_t nvec = K >> 3;
    const int64_t groups = (rows + RPB - 1) / RPB;
    __shared__ uint32_t part[RPB][TPR / 64];

    auto load = [&](uint4 (&d)[NV], int64_t grp) {
        const int64_t row = grp * RPB + sub;
        const bool live = grp < groups && row < rows;
        const uint4 *src = reinterpret_cast<const uint4 *>(v + (live ? row : 0) * K);
#pragma unroll
        for (int j = 0; j < NV; ++j) {
            const int64_t vi = (int64_t)j * TPR + t;
            if (live && vi < nvec)
                d[j] = src[vi];
            else
                d[j] = make_uint4(0, 0, 0, 0);
        }
    };
    auto process = [&](const uint4 (&d)[NV], int64_t grp) {
        const int64_t row = grp * RPB + sub;
        uint32_t m = 0;
#pragma unroll
        for (int j = 0; j < NV; ++j)
            m = max(m, absmax8(d[j]));
        m = wave_max(m);
        if constexpr (TPR == 256) {
            if ((threadIdx.x & 63) == 0)
                part[sub][(threadIdx.x >> 6) & 3] = m;
            __syncthreads();
            m = max(max(part[sub][0], part[sub][1]), max(part[sub][2], part[sub][3]));
            __syncthreads();   // part is rewritten by the next row group
        }
        const RowScale rs = row_scale(m);
        if (row >= rows)
            return;
        if (t == 0)
            scale[row] = rs.scale;
        uint2 *dst = reinterpret_cast<uint2 *>(q + row * K);
#pragma unroll
        for (int j = 0; j < NV; ++j) {
            const int64_t vi = (int64_t)j * TPR + t;
            if (vi < nvec)
                dst[vi] = code8(d[j], rs.inv);
        }
    };

    uint4 a[NV], b[NV];
    int64_t grp = blockIdx.x;
    load(a, grp);
    for (; grp < groups; grp += 2 * (int64_t)gridDim.x) {
        load(b, grp + gridDim.x);
        process(a, grp);
        if (grp + gridDim.x >= groups)
            break;
        load(a, grp + 2 * (int64_t)gridDim.x);
        process(b, grp + gridDim.x);
    }
}

// General path: one 256-thread block per row, two passes over the row (the second
// re-reads it, normally from L2). VEC selects 16-byte loads (K % 8 == 0 and aligned
// pointers); otherwise every element is loaded and stored on its own, for any K and
// any alignment.
template <bool VEC>
__global__ void __launch_bounds__(256)
quant_rows_loop(const uint16_t *__restrict__ v, int64_t rows, int64_t K,
                int8_t *__restrict__ q, float *__restrict__ scale) {
    const int64_t row = blockIdx.x;
    const int t = threadIdx.x;
    const uint16_t *src = v + row * K;
    uint32_t m = 0;
    if constexpr (VEC) {
        const uint4 *s4 = reinterpret_cast<const uint4 *>(src);
        for (int64_t vi = t; vi < (K >> 3); vi += 256)
            m = max(m, absmax8(s4[vi]));
    } else {
        for (int64_t k = t; k < K; k += 256)
            m = max(m, (uint32_t)src[k] & 0x7FFFu);
    }
    m = wave_max(m);
    __shared__ uint32_t part[4];
    if ((t & 63) == 0)
        part[t >> 6] = m;
    __syncthreads();
    m = max(max(part[0], part[1]), max(part[2], part[3]));
    const RowScale rs = row_scale(m);
    if (t == 0)
        scale[row] = rs.scale;
    int8_t *dst = q + row * K;
    if constexpr (VEC) {
        const uint4 *s4 = reinterpret_cast<const uint4 *>(src);
        uint2 *d2 = reinterpret_cast<uint2 *>(dst);
        for (int64_t vi = t; vi < (K >> 3); vi += 256)
            d2[vi] = code8(s4[vi], rs.inv);
    } else {
        for (int64_t k = t; k < K; k += 256)
            dst[k] = (int8_t)code((uint32_t)src[k], rs.inv);
    }
}

template <int TPR, int NV>
hipError_t launch_reg(const uint16_t *v, int64_t rows, int64_t K, int8_t *q,
                      float *scale, hipStream_t s) {
    constexpr int RPB = 256 / TPR;
    const int64_t groups = (rows + RPB - 1) / RPB;
    // Persistent grid: a few blocks per CU, each walking row groups with prefetch.
    const int64_t max_blocks = 256 * 8;
    const int64_t blocks = groups < max_blocks ? groups : max_blocks;
    hipLaunchKernelGGL((quant_rows_reg<TPR, NV>), dim3((unsigned)blocks), dim3(256), 0, s,
                       v, rows, K, q, scale);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_quant_rows(const uint16_t *v, int64_t rows, int64_t K, int8_t *q,
                             float *scale, hipStream_t s) {
    if (rows <= 0)
        return hipSuccess;
    const bool vec = (K % 8 == 0) && (reinterpret_cast<uintptr_t>(v) % 16 == 0) &&
                     (reinterpret_cast<uintptr_t>(q) % 8 == 0);
    const int64_t nvec = K / 8;
    if (vec && K > 0) {
        if (nvec <= 64)
            return launch_reg<64, 1>(v, rows, K, q, scale, s);
        if (nvec <= 128)
            return launch_reg<64, 2>(v, rows, K, q, scale, s);
        if (nvec <= 256)
            return launch_reg<64, 4>(v, rows, K, q, scale, s);
        if (nvec <= 512)
            return launch_reg<64, 8>(v, rows, K, q, scale, s);
        if (nvec <= 1024)
            return launch_reg<256, 4>(v, rows, K, q, scale, s);
        if (nvec <= 2048)
            return launch_reg<256, 8>(v, rows, K, q, scale, s);
    }
    if (vec)
        hipLaunchKernelGGL((quant_rows_loop<true>), dim3((unsigned)rows), dim3(256), 0, s,
                           v, rows, K, q, scale);
    else
        hipLaunchKernelGGL((quant_rows_loop<false>), dim3((unsigned)rows), dim3(256), 0, s,
                           v, rows, K, q, scale);
    return hipGetLastError();
}

}  // namespace w8a8
