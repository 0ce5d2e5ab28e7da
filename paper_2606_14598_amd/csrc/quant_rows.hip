// Per-row symmetric absmax int8 quantizer for gfx950.
//
// One rule serves both operands of the W8A8 linear (Section 3, "The quantization
// recipe (reused)"): per output channel for the weight W [N,K] (offline) and per token
// for the activation X [M,K] (online, every forward; "The fused kernel"). For a row v:
//   a = max_k |v[k]|, s = a / 127, q[k] = clamp(rne(v[k] * (127 / a)), -127, 127),
// and a row with a == 0 or with 127/a overflowing float32 gets s = 0, q = 0.
//
// The rule can run on transformed values v[k] = T(x[k]) * c[k] instead of the bf16
// inputs themselves: T is the identity or the exact GELU x * Phi(x) (the activation in
// front of the MLP down-projection, applied here so that it costs no pass of its own),
// and c is a per-input-channel multiplier, the run-time half of SmoothQuant (the recipe
// of Section 3 smooths the activations by 1/s[k] and folds s[k] into the weights).
// Both are evaluated in float32; the row maximum is then taken on float32 values.
//
// The kernel is HBM-bound (3 bytes moved per element: 2 read, 1 written), or ALU-bound
// with GELU. Rows whose K fits the register file (K <= 65536 for the plain rule) are read
// once with 16-byte loads, kept in VGPRs for the second (quantizing) pass and written
// with 16-byte streaming stores where alignment allows (8-byte stores otherwise), by a
// persistent grid that prefetches the next rows while it finishes the current ones; the
// row maximum is taken on the bf16 bit patterns (|v| ordered as an unsigned integer,
// exact for finite values) with a wavefront butterfly and, for rows of several
// wavefronts, one LDS exchange. Longer rows are read twice by a looped kernel.
#include "w8a8_internal.hpp"
#include "quant_math.hpp"

namespace w8a8 {
namespace {

using namespace qmath;

typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

// Swap with the neighbouring lane (lane l <-> l ^ 1) by a DPP quad permutation [1,0,3,2].
__device__ __forceinline__ uint32_t swap_lane_pair(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
}


// erfc(z) for z >= 0 by the Chebyshev fit of Numerical Recipes (Press, Teukolsky,
// Vetterling, Flannery, "erfcc"): t = 1 / (1 + z/2), erfc(z) ~ t exp(-z^2 + P(t)) with a
// degree-9 polynomial P, fractional error below 1.2e-7 for every z >= 0. One hardware
// reciprocal, one hardware exp2 and ten FMAs: the quantizer stays near the HBM bound.
__device__ __forceinline__ float erfc_nonneg(float z) {
    const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(0.5f, z, 1.0f));
    float p = 0.17087277f;
    p = __builtin_fmaf(t, p, -0.82215223f);
    p = __builtin_fmaf(t, p, 1.48851587f);
    p = __builtin_fmaf(t, p, -1.13520398f);
    p = __builtin_fmaf(t, p, 0.27886807f);
    p = __builtin_fmaf(t, p, -0.18628806f);
    p = __builtin_fmaf(t, p, 0.09678418f);
    p = __builtin_fmaf(t, p, 0.37409196f);
    p = __builtin_fmaf(t, p, 1.00002368f);
    const float arg = __builtin_fmaf(t, p, __builtin_fmaf(-z, z, -1.26551223f));
    return t * __builtin_amdgcn_exp2f(arg * 1.44269504088896341f);
}

// GELU(x) = x * Phi(x) with 2 Phi(x) = erfc(-x / sqrt(2)): for x < 0 that is
// erfc(|x| / sqrt(2)) (no cancellation in the left tail), for x >= 0 it is 2 - erfc.
__device__ __forceinline__ float gelu_f32(float x) {
    const float e = erfc_nonneg(__builtin_fabsf(x) * 0.70710678118654752440f);
    return 0.5f * x * (x < 0.0f ? e : 2.0f - e);
}

// The value the row rule sees: T(x), times the channel multiplier c when there is one.
template <int ACT, bool CM>
__device__ __forceinline__ float transform(float x, float c) {
    float t = x;
    if constexpr (ACT == ACT_GELU)
        t = gelu_f32(x);
    if constexpr (CM)
        t = t * c;
    return t;
}

// Code of a float32 value (transformed rows).
__device__ __forceinline__ uint32_t code_f(float v, float inv) {
    const float r = __builtin_amdgcn_fmed3f(__builtin_rintf(v * inv), -127.0f, 127.0f);
    return (uint32_t)((int)r) & 0xFFu;
}

__device__ __forceinline__ uint32_t abs_bits(float v) {
    return __float_as_uint(v) & 0x7FFFFFFFu;
}

// Register-resident path, persistent and software-pipelined: TPR threads per row
// (64 = one wavefront, up to 1024 = the block), NV 16-byte vectors per thread (K % 8 ==
// 0, v 16-byte and q 8-byte aligned). Blocks have max(TPR, 256) threads. Row group j of
// a block holds rows j*RPB .. j*RPB + RPB - 1; block b handles row groups b, b + G, b +
// 2G, ... (G = gridDim.x) and loads
// group j + G while it reduces, quantizes and stores group j, so the HBM reads of the
// next rows overlap the work and the stores of the current ones.
// With a transform (ACT != ACT_NONE or a multiplier), each thread's columns are the
// same for every row, so its multipliers are loaded once into registers; the
// transformed row is held as float32 between the maximum and the coding pass.
template <int TPR>
constexpr int reg_block_threads() { return TPR > 256 ? TPR : 256; }

template <int TPR, int NV, int ACT, bool CM>
__global__ void __launch_bounds__(reg_block_threads<TPR>())
quant_rows_reg(const uint16_t *__restrict__ v, int64_t rows, int64_t K,
               const float *__restrict__ colmul, int8_t *__restrict__ q,
               float *__restrict__ scale) {
    constexpr bool PLAIN = ACT == ACT_NONE && !CM;
    constexpr int RPB = reg_block_threads<TPR>() / TPR;
    const int t = threadIdx.x % TPR;
    const int sub = threadIdx.x / TPR;
    const int64_t nvec = K >> 3;
    const int64_t groups = (rows + RPB - 1) / RPB;
    const bool wide = (K % 16 == 0) && (reinterpret_cast<uintptr_t>(q) % 16 == 0);
    __shared__ uint32_t part[RPB][TPR / 64];

    float cmr[CM ? NV : 1][8];
    if constexpr (CM) {
#pragma unroll
        for (int j = 0; j < NV; ++j) {
            const int64_t vi = (int64_t)j * TPR + t;
            const float4 *c4 = reinterpret_cast<const float4 *>(colmul) + 2 * vi;
            const float4 lo = vi < nvec ? c4[0] : make_float4(0, 0, 0, 0);
            const float4 hi = vi < nvec ? c4[1] : make_float4(0, 0, 0, 0);
            cmr[j][0] = lo.x; cmr[j][1] = lo.y; cmr[j][2] = lo.z; cmr[j][3] = lo.w;
            cmr[j][4] = hi.x; cmr[j][5] = hi.y; cmr[j][6] = hi.z; cmr[j][7] = hi.w;
        }
    }

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
        float f[PLAIN ? 1 : NV][8];
        if constexpr (PLAIN) {
#pragma unroll
            for (int j = 0; j < NV; ++j)
                m = max(m, absmax8(d[j]));
        } else {
            float fm = 0.0f;
#pragma unroll
            for (int j = 0; j < NV; ++j) {
                const uint32_t w[4] = {d[j].x, d[j].y, d[j].z, d[j].w};
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint32_t h = (e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xFFFFu);
                    f[j][e] = transform<ACT, CM>(bf16_to_f32(h), CM ? cmr[j][e] : 1.0f);
                    fm = fmaxf(fm, __builtin_fabsf(f[j][e]));
                }
            }
            m = __float_as_uint(fm);   // |v| >= 0: its bit pattern orders like the value
        }
        m = wave_max(m);
        if constexpr (TPR > 64) {
            constexpr int WPR = TPR / 64;   // wavefronts per row
            if ((threadIdx.x & 63) == 0)
                part[sub][(threadIdx.x >> 6) % WPR] = m;
            __syncthreads();
#pragma unroll
            for (int w = 0; w < WPR; ++w)
                m = max(m, part[sub][w]);
            __syncthreads();   // part is rewritten by the next row group
        }
        const RowScale rs = PLAIN ? row_scale(m) : row_scale_f(__uint_as_float(m));
        if (row >= rows)
            return;
        if (t == 0)
            scale[row] = rs.scale;
        uint2 *dst = reinterpret_cast<uint2 *>(q + row * K);
        // Codes of vector j of this lane (8 bytes).
        auto codes = [&](int j) __attribute__((always_inline)) {
            uint2 o;
            if constexpr (PLAIN) {
                o = code8(d[j], rs.inv);
            } else {
                uint32_t c[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    c[e] = code_f(f[j][e], rs.inv);
                o.x = c[0] | (c[1] << 8) | (c[2] << 16) | (c[3] << 24);
                o.y = c[4] | (c[5] << 8) | (c[6] << 16) | (c[7] << 24);
            }
            return o;
        };
        // The paired path for the plain rule, and for transformed rows with two vectors
        // per thread; with more, transformed rows measured 3-12% slower with it (GELU and
        // multiplier variants at K = 12288 and 16384) and keep 8-byte stores.
        constexpr bool PAIRS = PLAIN || NV == 2;
        if (PAIRS && wide) {
            // 16-byte streaming stores (K % 16 == 0, q 16-byte aligned), one pair of
            // vectors at a time. Vectors j and j+1 of lane t are j*TPR + t and
            // (j+1)*TPR + t; neighbouring lanes swap one code word pair so that the even
            // lane holds vectors j*TPR + t, +1 and the odd lane (j+1)*TPR + t - 1, +1.
            // Streaming 16-byte stores leave no dirty lines in this XCD's L2 for the
            // kernel's end to write back before the consumer starts (plain stores, and
            // 8-byte streaming ones, delayed the next kernel by 1.5-2.5 us).
            const bool odd = t & 1;
#pragma unroll
            for (int j = 0; j + 1 < NV; j += 2) {
                // Selects on scalars (a select between array elements would put the
                // array in memory).
                const uint2 ca = codes(j), cb = codes(j + 1);
                const uint32_t a0 = ca.x, a1 = ca.y, b0 = cb.x, b1 = cb.y;
                const uint32_t r0 = swap_lane_pair(odd ? a0 : b0);
                const uint32_t r1 = swap_lane_pair(odd ? a1 : b1);
                const int64_t v0 = (int64_t)(odd ? j + 1 : j) * TPR + t - (odd ? 1 : 0);
                const u32x4v o = odd ? u32x4v{r0, r1, b0, b1} : u32x4v{a0, a1, r0, r1};
                if (v0 + 1 < nvec)
                    __builtin_nontemporal_store(o, reinterpret_cast<u32x4v *>(dst + v0));
                else if (v0 < nvec)
                    dst[v0] = make_uint2(o.x, o.y);
            }
            if constexpr (NV % 2 == 1) {
                // The last vector of an odd count: the even lane of each pair takes its
                // neighbour's codes (vector j*TPR + t + 1) and stores both.
                const uint2 c = codes(NV - 1);
                const uint32_t n0 = swap_lane_pair(c.x), n1 = swap_lane_pair(c.y);
                const int64_t vi = (int64_t)(NV - 1) * TPR + t;
                if (!odd) {
                    if (vi + 1 < nvec)
                        __builtin_nontemporal_store(u32x4v{c.x, c.y, n0, n1},
                                                    reinterpret_cast<u32x4v *>(dst + vi));
                    else if (vi < nvec)
                        dst[vi] = c;
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < NV; ++j) {
                const int64_t vi = (int64_t)j * TPR + t;
                if (vi < nvec)
                    dst[vi] = codes(j);
            }
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

// General path: a 256-thread block per row (a block takes every G-th row when there are
// more rows than the grid's G blocks), two passes over the row (the second re-reads it,
// normally from L2). VEC selects 16-byte loads and 8-byte stores (K % 8 ==
// 0; v and colmul 16-byte, q 8-byte aligned); a transform is then evaluated on the 8
// values of a vector in both passes. Otherwise every element is loaded and stored on
// its own, for any K and any alignment.
template <bool VEC, int ACT, bool CM>
__global__ void __launch_bounds__(256)
quant_rows_loop(const uint16_t *__restrict__ v, int64_t rows, int64_t K,
                const float *__restrict__ colmul, int8_t *__restrict__ q,
                float *__restrict__ scale) {
    constexpr bool PLAIN = ACT == ACT_NONE && !CM;
    const int t = threadIdx.x;
    const int64_t nvec = K >> 3;
    __shared__ uint32_t part[4];
    // Block b takes rows b, b + G, b + 2G, ... (G = gridDim.x, at most 65536 blocks).
    for (int64_t row = blockIdx.x; row < rows; row += gridDim.x) {
        const uint16_t *src = v + row * K;
        auto value = [&](int64_t k) {
            return transform<ACT, CM>(bf16_to_f32(src[k]), CM ? colmul[k] : 1.0f);
        };
        // The 8 transformed values of vector vi.
        auto values8 = [&](int64_t vi, float (&f)[8]) __attribute__((always_inline)) {
            const uint4 d = reinterpret_cast<const uint4 *>(src)[vi];
            float c[8] = {1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f, 1.0f};
            if constexpr (CM) {
                const float4 *c4 = reinterpret_cast<const float4 *>(colmul) + 2 * vi;
                const float4 lo = c4[0], hi = c4[1];
                c[0] = lo.x; c[1] = lo.y; c[2] = lo.z; c[3] = lo.w;
                c[4] = hi.x; c[5] = hi.y; c[6] = hi.z; c[7] = hi.w;
            }
            const uint32_t w[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint32_t h = (e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xFFFFu);
                f[e] = transform<ACT, CM>(bf16_to_f32(h), c[e]);
            }
        };
        uint32_t m = 0;
        if constexpr (VEC && PLAIN) {
            const uint4 *s4 = reinterpret_cast<const uint4 *>(src);
            for (int64_t vi = t; vi < nvec; vi += 256)
                m = max(m, absmax8(s4[vi]));
        } else if constexpr (VEC) {
            float fm = 0.0f;
            for (int64_t vi = t; vi < nvec; vi += 256) {
                float f[8];
                values8(vi, f);
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    fm = fmaxf(fm, __builtin_fabsf(f[e]));
            }
            m = abs_bits(fm);
        } else if constexpr (PLAIN) {
            for (int64_t k = t; k < K; k += 256)
                m = max(m, (uint32_t)src[k] & 0x7FFFu);
        } else {
            for (int64_t k = t; k < K; k += 256)
                m = max(m, abs_bits(value(k)));
        }
        m = wave_max(m);
        if ((t & 63) == 0)
            part[t >> 6] = m;
        __syncthreads();
        m = max(max(part[0], part[1]), max(part[2], part[3]));
        __syncthreads();   // part is rewritten for the next row
        const RowScale rs = PLAIN ? row_scale(m) : row_scale_f(__uint_as_float(m));
        if (t == 0)
            scale[row] = rs.scale;
        int8_t *dst = q + row * K;
        if constexpr (VEC && PLAIN) {
            const uint4 *s4 = reinterpret_cast<const uint4 *>(src);
            uint2 *d2 = reinterpret_cast<uint2 *>(dst);
            for (int64_t vi = t; vi < nvec; vi += 256)
                d2[vi] = code8(s4[vi], rs.inv);
        } else if constexpr (VEC) {
            uint2 *d2 = reinterpret_cast<uint2 *>(dst);
            for (int64_t vi = t; vi < nvec; vi += 256) {
                float f[8];
                values8(vi, f);
                uint32_t c[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    c[e] = code_f(f[e], rs.inv);
                d2[vi] = make_uint2(c[0] | (c[1] << 8) | (c[2] << 16) | (c[3] << 24),
                                    c[4] | (c[5] << 8) | (c[6] << 16) | (c[7] << 24));
            }
        } else if constexpr (PLAIN) {
            for (int64_t k = t; k < K; k += 256)
                dst[k] = (int8_t)code((uint32_t)src[k], rs.inv);
        } else {
            for (int64_t k = t; k < K; k += 256)
                dst[k] = (int8_t)code_f(value(k), rs.inv);
        }
    }
}

template <int TPR, int NV, int ACT, bool CM>
hipError_t launch_reg(const uint16_t *v, int64_t rows, int64_t K, const float *colmul,
                      int8_t *q, float *scale, hipStream_t s) {
    constexpr int BS = reg_block_threads<TPR>();
    constexpr int RPB = BS / TPR;
    const int64_t groups = (rows + RPB - 1) / RPB;
    // Persistent grid: up to 2048 threads per CU, each block walking row groups with
    // prefetch.
    const int64_t max_blocks = 256 * 2048 / BS;
    const int64_t blocks = groups < max_blocks ? groups : max_blocks;
    hipLaunchKernelGGL((quant_rows_reg<TPR, NV, ACT, CM>), dim3((unsigned)blocks), dim3(BS),
                       0, s, v, rows, K, colmul, q, scale);
    return hipGetLastError();
}

template <int ACT, bool CM>
hipError_t launch_rows(const uint16_t *v, int64_t rows, int64_t K, const float *colmul,
                       int8_t *q, float *scale, hipStream_t s) {
    constexpr bool PLAIN = ACT == ACT_NONE && !CM;
    const bool vec = (K % 8 == 0) && (reinterpret_cast<uintptr_t>(v) % 16 == 0) &&
                     (reinterpret_cast<uintptr_t>(q) % 8 == 0) &&
                     (reinterpret_cast<uintptr_t>(colmul) % 16 == 0);
    const int64_t nvec = K / 8;
    // Threads per row and vectors per thread past 256 vectors per row, from sweeps of
    // both over rows x K (HIP-graph replays of the quantizer on its own, the plain rule
    // and GELU rows). The vector count per thread is the smallest that covers the row,
    // so few lanes idle (at K = 4608 a 256 x 4 row leaves 44% of them idle: 11-24%
    // slower than 128 x 5 for the plain rule, 21-28% for GELU rows, which are ALU-bound);
    // fewer rows spread a row over more threads. Every choice is within 7% of the
    // sweeps' best on the shapes measured. Transformed rows differ at K <= 4096 (256 x 2
    // below 4096 rows; from there one wavefront per row up to K = 3584, 3072 without
    // GELU, and 128 x 4 above), at K <= 8192 from 4096 rows up (256 x 4) and at
    // K <= 16384 (the 256-thread block beats 1024-thread rows).
    if (vec && nvec > 256 && nvec <= 2048) {
        if (nvec <= 512) {
            // One wavefront per row with exactly the vectors the row needs.
            auto wave_row = [&]() {
                if (nvec <= 320)
                    return launch_reg<64, 5, ACT, CM>(v, rows, K, colmul, q, scale, s);
                if (nvec <= 384)
                    return launch_reg<64, 6, ACT, CM>(v, rows, K, colmul, q, scale, s);
                if (nvec <= 448)
                    return launch_reg<64, 7, ACT, CM>(v, rows, K, colmul, q, scale, s);
                return launch_reg<64, 8, ACT, CM>(v, rows, K, colmul, q, scale, s);
            };
            if constexpr (PLAIN) {
                if (rows < 1024)
                    return launch_reg<512, 1, ACT, CM>(v, rows, K, colmul, q, scale, s);
                if (rows >= 4096 || nvec <= 384)
                    return wave_row();
            } else {
                // Two vectors per thread keep the 16-byte store pairs of transformed
                // rows (4 vectors measured 5-8% slower with the multiplier below 4096 rows).
                if (rows < 4096)
                    return launch_reg<256, 2, ACT, CM>(v, rows, K, colmul, q, scale, s);
                // Multiplier-only rows are memory-bound: 7 vectors (8-byte stores) measured
                // 8-9% slower for them than 128 x 4; GELU rows gain up to 8% from it.
                if (nvec <= (ACT == ACT_GELU ? 448 : 384))
                    return wave_row();
            }
            return launch_reg<128, 4, ACT, CM>(v, rows, K, colmul, q, scale, s);
        }
        if (nvec <= 768 && rows < 1024)
            return launch_reg<256, 3, ACT, CM>(v, rows, K, colmul, q, scale, s);
        if (nvec <= 640)
            return launch_reg<128, 5, ACT, CM>(v, rows, K, colmul, q, scale, s);
        if (nvec <= 768)
            return launch_reg<128, 6, ACT, CM>(v, rows, K, colmul, q, scale, s);
        if (nvec <= 1024) {
            if constexpr (PLAIN)
                if (rows >= 4096)
                    return launch_reg<128, 8, ACT, CM>(v, rows, K, colmul, q, scale, s);
            return launch_reg<256, 4, ACT, CM>(v, rows, K, colmul, q, scale, s);
        }
        // Few long rows (K > 8192 below 256 rows): 512 threads per row, 5-9% faster
        // than the 256-thread block.
        if (rows < 256)
            return nvec <= 1536 ? launch_reg<512, 3, ACT, CM>(v, rows, K, colmul, q, scale, s)
                                : launch_reg<512, 4, ACT, CM>(v, rows, K, colmul, q, scale, s);
        if (nvec <= 1536)
            return launch_reg<256, 6, ACT, CM>(v, rows, K, colmul, q, scale, s);
        if constexpr (PLAIN)
            if (rows >= 2048)
                return launch_reg<1024, 2, ACT, CM>(v, rows, K, colmul, q, scale, s);
        return launch_reg<256, 8, ACT, CM>(v, rows, K, colmul, q, scale, s);
    }
    if (vec && K > 0) {
        // K <= 2048: below 1024 rows a row takes 128 or 256 threads with one vector each
        // (8-13% faster than a wavefront per row at K = 1536-2048, 32% with GELU);
        // from 1024 rows up a wavefront per row with exactly the row's vectors.
        if (nvec <= 64)
            return launch_reg<64, 1, ACT, CM>(v, rows, K, colmul, q, scale, s);
        if (nvec <= 128)
            return rows < 1024 ? launch_reg<128, 1, ACT, CM>(v, rows, K, colmul, q, scale, s)
                               : launch_reg<64, 2, ACT, CM>(v, rows, K, colmul, q, scale, s);
        if (nvec <= 256) {
            if (rows < 1024)
                return launch_reg<256, 1, ACT, CM>(v, rows, K, colmul, q, scale, s);
            return nvec <= 192 ? launch_reg<64, 3, ACT, CM>(v, rows, K, colmul, q, scale, s)
                               : launch_reg<64, 4, ACT, CM>(v, rows, K, colmul, q, scale, s);
        }
        // Long rows (K up to 65536 for the plain rule, e.g. a 53248-wide projection
        // input; 32768 for transformed rows, whose float32 copy of 8 vectors per thread
        // would not fit 128 VGPRs): a 1024-thread block per row, still read once. The
        // looped kernel below reads such rows twice, the second time mostly from the
        // MALL, since 32 CUs' rows overflow an XCD's L2.
        if (nvec <= 4096)
            return launch_reg<1024, 4, ACT, CM>(v, rows, K, colmul, q, scale, s);
        if constexpr (PLAIN)
            if (nvec <= 8192)
                return launch_reg<1024, 8, ACT, CM>(v, rows, K, colmul, q, scale, s);
    }
    const unsigned grid = (unsigned)(rows < 65536 ? rows : 65536);
    if (vec)
        hipLaunchKernelGGL((quant_rows_loop<true, ACT, CM>), dim3(grid), dim3(256), 0, s, v,
                           rows, K, colmul, q, scale);
    else
        hipLaunchKernelGGL((quant_rows_loop<false, ACT, CM>), dim3(grid), dim3(256), 0, s, v,
                           rows, K, colmul, q, scale);
    return hipGetLastError();
}

// Calibration: per-column max |T(x)| over a block of rows, merged across blocks with
// an unsigned atomic maximum on the float32 bit patterns (monotone for values >= 0).
template <int ACT>
__global__ void __launch_bounds__(256)
col_absmax_kernel(const uint16_t *__restrict__ v, int64_t rows, int64_t K,
                  int64_t rows_per_block, uint32_t *__restrict__ amax) {
    const int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (k >= K)
        return;
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_block;
    const int64_t r1 = r0 + rows_per_block < rows ? r0 + rows_per_block : rows;
    uint32_t m = 0;
    for (int64_t r = r0; r < r1; ++r)
        m = max(m, abs_bits(transform<ACT, false>(bf16_to_f32(v[r * K + k]), 1.0f)));
    atomicMax(amax + k, m);
}

__global__ void __launch_bounds__(256) fill_zero_u32(uint32_t *p, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n)
        p[i] = 0u;
}

// SmoothQuant factors: s = ax^alpha / aw^(1 - alpha) (alpha = 1/2: sqrtf / sqrtf, each
// correctly rounded); channels without a positive, finite pair, or whose factor is 0
// or infinite, stay unsmoothed (s = 1). s_inv = 1 / s is the activation multiplier.
__global__ void __launch_bounds__(256)
smooth_factors_kernel(const float *__restrict__ ax, const float *__restrict__ aw, int64_t K,
                      float alpha, float *__restrict__ s, float *__restrict__ s_inv) {
    const int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (k >= K)
        return;
    const float a = ax[k], b = aw[k];
    float f = 1.0f;
    if (a > 0.0f && b > 0.0f && __builtin_isfinite(a) && __builtin_isfinite(b)) {
        f = alpha == 0.5f ? sqrtf(a) / sqrtf(b) : powf(a, alpha) / powf(b, 1.0f - alpha);
        if (!(f > 0.0f) || !__builtin_isfinite(f))
            f = 1.0f;
    }
    s[k] = f;
    s_inv[k] = 1.0f / f;
}

}  // namespace

hipError_t launch_quant_rows(const uint16_t *v, int64_t rows, int64_t K, int act,
                             const float *colmul, int8_t *q, float *scale, hipStream_t s) {
    if (rows <= 0)
        return hipSuccess;
    if (act == ACT_GELU)
        return colmul ? launch_rows<ACT_GELU, true>(v, rows, K, colmul, q, scale, s)
                      : launch_rows<ACT_GELU, false>(v, rows, K, colmul, q, scale, s);
    return colmul ? launch_rows<ACT_NONE, true>(v, rows, K, colmul, q, scale, s)
                  : launch_rows<ACT_NONE, false>(v, rows, K, colmul, q, scale, s);
}

hipError_t launch_col_absmax(const uint16_t *v, int64_t rows, int64_t K, int act,
                             float *amax, bool accumulate, hipStream_t s) {
    if (K <= 0)
        return hipSuccess;
    uint32_t *bits = reinterpret_cast<uint32_t *>(amax);
    const unsigned kb = (unsigned)((K + 255) / 256);
    if (!accumulate)
        hipLaunchKernelGGL(fill_zero_u32, dim3(kb), dim3(256), 0, s, bits, K);
    if (rows > 0) {
        int64_t rpb = 32;
        while ((rows + rpb - 1) / rpb > 65535)
            rpb *= 2;
        const dim3 grid(kb, (unsigned)((rows + rpb - 1) / rpb));
        if (act == ACT_GELU)
            hipLaunchKernelGGL(col_absmax_kernel<ACT_GELU>, grid, dim3(256), 0, s, v, rows, K,
                               rpb, bits);
        else
            hipLaunchKernelGGL(col_absmax_kernel<ACT_NONE>, grid, dim3(256), 0, s, v, rows, K,
                               rpb, bits);
    }
    return hipGetLastError();
}

hipError_t launch_smooth_factors(const float *ax, const float *aw, int64_t K, float alpha,
                                 float *smooth, float *smooth_inv, hipStream_t s) {
    if (K <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(smooth_factors_kernel, dim3((unsigned)((K + 255) / 256)), dim3(256), 0,
                       s, ax, aw, K, alpha, smooth, smooth_inv);
    return hipGetLastError();
}

}  // namespace w8a8
