// int8 x int8 -> int32 GEMM on gfx950 matrix cores with the fused dequantization
// epilogue of the W8A8 linear (Section 3, "The fused kernel").
//
// Y[m][n] = bf16(fmaf((float)acc[m][n], sx[m] * sw[n], b[n])),
// acc[m][n] = sum_k Xq[m][k] * Wq[n][k], with Xq [M,K] and Wq [N,K] both K-contiguous.
//
// Design (one workgroup per TM x TN output tile):
//   * v_mfma_i32_32x32x32_i8: the weight tile is the matrix-core A operand (its 32 rows
//     are output channels n) and the activation tile the B operand (its 32 columns are
//     tokens m). The accumulator layout then gives each lane 4 consecutive channels of
//     one token, so the bf16 epilogue writes 8 contiguous bytes per lane-group and the
//     per-channel scale/bias come in as 16/8-byte vectors.
//   * K-panels of BK bytes are staged in LDS, double buffered: the global loads of
//     panel k+1 (buffer loads: rows past M/N and bytes past K read as zero, so ragged
//     tiles need no branches) are in flight while the matrix cores work on panel k.
//   * LDS rows are BK bytes; their 16-byte chunks are XOR-swizzled by row so that both
//     the 16-byte stores of a wavefront and the 16-byte operand reads (32 rows x one
//     chunk per half-wavefront) hit distinct bank groups.
//   * Workgroup ids are remapped so that each XCD (which receives every 8th id) owns a
//     contiguous run of tiles, traversed in groups of GM token-tiles, so the operand
//     panels a run touches stay in that XCD's L2.
//   * The integer accumulation is exact, so every tiling gives identical bits.
#include "w8a8_internal.hpp"

#include <utility>

namespace w8a8 {
namespace {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Buffer-resource word 3 for gfx9 (raw 32-bit data format, no swizzle).
constexpr int kRsrcWord3 = 0x00020000;
// A voffset beyond any num_records: the load returns zero.
constexpr int kOOB = 0x7FFFFFF0;

// XOR swizzle of the 16-byte chunk index inside an LDS row of BK bytes. It depends only
// on row & 31, so every 32-row MFMA fragment of a wavefront sees the same per-lane
// pattern (fragment addresses differ by constants). With it, the 16-byte operand reads
// (32 consecutive rows x one chunk per half-wavefront) and the 16-byte stores of
// consecutive chunks both hit distinct banks in every 8- and 16-lane phase.
template <int BK>
__device__ __forceinline__ int swz(int row) {
    static_assert(BK == 64 || BK == 128, "BK");
    if constexpr (BK == 128)
        return (row & 7) ^ ((row >> 3) & 3);
    else
        return ((row >> 1) ^ (row >> 3)) & 3;
}

// Logical tile of workgroup `bid`: XCD-contiguous runs, grouped raster inside.
__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int gm,
                                        int &tm, int &tn) {
    const int total = tiles_m * tiles_n;
    const int xcd = bid & 7, slot = bid >> 3;
    const int q = total >> 3, r = total & 7;
    const int t = xcd * q + min(xcd, r) + slot;
    const int per_group = gm * tiles_n;
    const int g = t / per_group;
    const int first = g * gm;
    const int gsz = min(tiles_m - first, gm);
    const int in = t - g * per_group;
    tm = first + in % gsz;
    tn = in / gsz;
}

// 16 bytes of row `row` at byte `k` of a [rows_left, K] panel, zero outside. VEC: one
// buffer load (K % 16 == 0, 16-byte aligned base). Otherwise byte loads.
template <bool VEC>
__device__ __forceinline__ i32x4 load16(__amdgpu_buffer_rsrc_t rsrc, const int8_t *base,
                                        int row, int rows_left, int64_t k, int64_t K) {
    if constexpr (VEC) {
        const int off = (row < rows_left && k < K) ? (int)(row * K + k) : kOOB;
        return __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, 0));
    } else {
        uint32_t w[4] = {0, 0, 0, 0};
        if (row < rows_left) {
            const int8_t *p = base + (int64_t)row * K;
#pragma unroll
            for (int b = 0; b < 16; ++b) {
                if (k + b < K)
                    w[b >> 2] |= ((uint32_t)(uint8_t)p[k + b]) << ((b & 3) * 8);
            }
        }
        i32x4 v = {(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
        return v;
    }
}

struct KParams {
    GemmArgs a;
    int tiles_m, tiles_n;
    int gm;          // token-tiles per raster group
    int out_vec;     // output rows 16-byte aligned with N % 4 == 0, scale/bias aligned
};

// Epilogue of one wavefront's (FN*32 channels) x (FM*32 tokens) accumulator tile whose
// first channel is n_base and first token m_base. Lane l of fragment (i, j) holds token
// m = m_base + 32j + l%32 and, in register 4g+e, channel n = n_base + 32i + 8g + 4(l/32) + e.
// EPI_BF16: y = bf16(fmaf(float(acc), sx[m] * sw[n], b[n])); EPI_I32: the raw accumulator.
template <int FN, int FM, int EPI>
__device__ __forceinline__ void store_tile(const i32x16 (&acc)[FN][FM], const KParams &kp,
                                           int64_t m_base, int64_t n_base, int lane) {
    const GemmArgs &a = kp.a;
    const int64_t M = a.M, N = a.N;
#pragma unroll
    for (int j = 0; j < FM; ++j) {
        const int64_t m = m_base + j * 32 + (lane & 31);
        if (m >= M)
            continue;
        float sxm = 0.0f;
        if constexpr (EPI == EPI_BF16)
            sxm = a.sx[m];
#pragma unroll
        for (int i = 0; i < FN; ++i) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int64_t n = n_base + i * 32 + g * 8 + (lane >> 5) * 4;
                if (n >= N)
                    continue;
                const int32_t v0 = acc[i][j][4 * g + 0], v1 = acc[i][j][4 * g + 1];
                const int32_t v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
                if constexpr (EPI == EPI_I32) {
                    int32_t *o = static_cast<int32_t *>(a.out) + m * N + n;
                    if (kp.out_vec && n + 3 < N) {
                        *reinterpret_cast<i32x4 *>(o) = i32x4{v0, v1, v2, v3};
                    } else {
                        const int32_t vv[4] = {v0, v1, v2, v3};
                        for (int e = 0; e < 4 && n + e < N; ++e)
                            o[e] = vv[e];
                    }
                } else {
                    uint16_t *o = static_cast<uint16_t *>(a.out) + m * N + n;
                    const int32_t vv[4] = {v0, v1, v2, v3};
                    if (kp.out_vec && n + 3 < N) {
                        const f32x4 s4 = *reinterpret_cast<const f32x4 *>(a.sw + n);
                        float b4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                        if (a.bias) {
                            const uint2 bb = *reinterpret_cast<const uint2 *>(a.bias + n);
                            b4[0] = __uint_as_float(bb.x << 16);
                            b4[1] = __uint_as_float(bb.x & 0xFFFF0000u);
                            b4[2] = __uint_as_float(bb.y << 16);
                            b4[3] = __uint_as_float(bb.y & 0xFFFF0000u);
                        }
                        uint16_t h[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float s = sxm * s4[e];
                            const float y = __builtin_fmaf((float)vv[e], s, b4[e]);
                            h[e] = __builtin_bit_cast(uint16_t, (__bf16)y);
                        }
                        uint2 pk;
                        pk.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
                        pk.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
                        *reinterpret_cast<uint2 *>(o) = pk;
                    } else {
                        for (int e = 0; e < 4 && n + e < N; ++e) {
                            const float b = a.bias ? __uint_as_float((uint32_t)a.bias[n + e] << 16) : 0.0f;
                            const float s = sxm * a.sw[n + e];
                            const float y = __builtin_fmaf((float)vv[e], s, b);
                            o[e] = __builtin_bit_cast(uint16_t, (__bf16)y);
                        }
                    }
                }
            }
        }
    }
}

template <int TM, int TN, int BK, int WM, int WN, bool VEC, int EPI>
__global__ void __launch_bounds__(WM *WN * 64)
gemm_i8_kernel(KParams kp) {
    constexpr int NT = WM * WN * 64;
    constexpr int WTM = TM / WM, WTN = TN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int CPR = BK / 16;               // 16-byte chunks per LDS row
    constexpr int LW = TN * CPR / NT;          // weight chunks per thread per panel
    constexpr int LX = TM * CPR / NT;          // activation chunks per thread per panel
    constexpr int STAGE = (TN + TM) * BK;
    static_assert(FM >= 1 && FN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile");
    static_assert((TN * CPR) % NT == 0 && (TM * CPR) % NT == 0, "load split");
    __shared__ __attribute__((aligned(16))) int8_t smem[2 * STAGE];

    const GemmArgs &a = kp.a;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    int tm, tn;
    tile_of(blockIdx.x, kp.tiles_m, kp.tiles_n, kp.gm, tm, tn);
    const int64_t m0 = (int64_t)tm * TM, n0 = (int64_t)tn * TN;
    const int64_t M = a.M, N = a.N, K = a.K;
    const int rows_w = (int)((N - n0) < TN ? (N - n0) : TN);
    const int rows_x = (int)((M - m0) < TM ? (M - m0) : TM);
    const int8_t *wbase = a.wq + n0 * K;
    const int8_t *xbase = a.xq + m0 * K;
    const __amdgpu_buffer_rsrc_t rw_rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void *)wbase, (short)0, (int)(rows_w * K), kRsrcWord3);
    const __amdgpu_buffer_rsrc_t rx_rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void *)xbase, (short)0, (int)(rows_x * K), kRsrcWord3);

    i32x16 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j)
            acc[i][j] = i32x16{};

    i32x4 rw[LW], rx[LX];
    auto gload = [&](int kt) {
        const int64_t k0 = (int64_t)kt * BK;
#pragma unroll
        for (int i = 0; i < LW; ++i) {
            const int c = i * NT + tid;
            rw[i] = load16<VEC>(rw_rsrc, wbase, c / CPR, rows_w, k0 + (c % CPR) * 16, K);
        }
#pragma unroll
        for (int i = 0; i < LX; ++i) {
            const int c = i * NT + tid;
            rx[i] = load16<VEC>(rx_rsrc, xbase, c / CPR, rows_x, k0 + (c % CPR) * 16, K);
        }
    };
    auto sstore = [&](int st) {
        int8_t *sw_ = smem + st * STAGE;
        int8_t *sx_ = sw_ + TN * BK;
#pragma unroll
        for (int i = 0; i < LW; ++i) {
            const int c = i * NT + tid;
            const int row = c / CPR, kc = c % CPR;
            *reinterpret_cast<i32x4 *>(sw_ + row * BK + ((kc ^ swz<BK>(row)) << 4)) = rw[i];
        }
#pragma unroll
        for (int i = 0; i < LX; ++i) {
            const int c = i * NT + tid;
            const int row = c / CPR, kc = c % CPR;
            *reinterpret_cast<i32x4 *>(sx_ + row * BK + ((kc ^ swz<BK>(row)) << 4)) = rx[i];
        }
    };
    auto compute = [&](int st) {
        const int8_t *sw_ = smem + st * STAGE;
        const int8_t *sx_ = sw_ + TN * BK;
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            const int ch = ks * 2 + (lane >> 5);
            i32x4 fa[FN], fb[FM];
#pragma unroll
            for (int i = 0; i < FN; ++i) {
                const int row = wn * WTN + i * 32 + (lane & 31);
                fa[i] = *reinterpret_cast<const i32x4 *>(sw_ + row * BK + ((ch ^ swz<BK>(row)) << 4));
            }
#pragma unroll
            for (int j = 0; j < FM; ++j) {
                const int row = wm * WTM + j * 32 + (lane & 31);
                fb[j] = *reinterpret_cast<const i32x4 *>(sx_ + row * BK + ((ch ^ swz<BK>(row)) << 4));
            }
#pragma unroll
            for (int i = 0; i < FN; ++i)
#pragma unroll
                for (int j = 0; j < FM; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[i], fb[j], acc[i][j], 0, 0, 0);
        }
    };

    const int nk = (int)((K + BK - 1) / BK);
    if (nk > 0) {
        gload(0);
        sstore(0);
        __syncthreads();
        for (int kt = 0; kt < nk; ++kt) {
            const int st = kt & 1;
            if (kt + 1 < nk)
                gload(kt + 1);
            compute(st);
            if (kt + 1 < nk)
                sstore(st ^ 1);
            __syncthreads();
        }
    }

    store_tile<FN, FM, EPI>(acc, kp, m0 + wm * WTM, n0 + wn * WTN, lane);
}


// s_waitcnt immediate for gfx9 that waits until at most n vector-memory operations are
// outstanding (expcnt and lgkmcnt left unconstrained).
__host__ __device__ constexpr int waitcnt_vm(int n) {
    return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8);
}

// Workgroup barrier without the memory fence __syncthreads() carries (the fence would
// make the compiler wait for every outstanding load, draining the LDS ring). Callers
// wait for the loads they need with an explicit vmcnt first; LDS-DMA data are in LDS
// once vmcnt has counted them.
__device__ __forceinline__ void barrier_nofence() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// Pipelined variant for 16-byte aligned operands with K % 16 == 0.
//   * Panels go straight from global memory to LDS (buffer_load_dwordx4 ... lds): lane l
//     of the i-th load of wavefront w fills LDS chunk c = i*NT + 64w + l, i.e. row
//     c / CPR, physical chunk c % CPR, and therefore fetches logical chunk
//     (c % CPR) ^ swz(row) of that row. No staging registers, no ds_write.
//   * S LDS stages in a ring: panel k+S-1 is requested while panel k is multiplied, so a
//     load has S-1 panels of MFMA work to arrive; one wait + barrier per panel makes
//     panel k+1 visible to every wavefront.
//   * MFMA operand fragments are double-buffered across the BK/32 K-steps of a panel:
//     each K-step is two fenced groups, (1) the ds_reads of the next K-step's fragments
//     and a slice of the loads of panel k+S-1, (2) this K-step's MFMAs back to back.
template <int TM, int TN, int BK, int WM, int WN, int S, int EPI>
__global__ void __launch_bounds__(WM *WN * 64)
gemm_i8_lds_kernel(KParams kp) {
    constexpr int NT = WM * WN * 64;
    constexpr int WTM = TM / WM, WTN = TN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int CPR = BK / 16;
    constexpr int RPL = NT / CPR;              // rows covered by one load instruction
    constexpr int LW = TN / RPL, LX = TM / RPL;
    constexpr int NV = LW + LX;                // loads per thread per panel
    constexpr int STAGE = (TN + TM) * BK;
    constexpr int KS = BK / 32;
    static_assert(FM >= 1 && FN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile");
    static_assert(RPL % 32 == 0 && TN % RPL == 0 && TM % RPL == 0, "load split");
    static_assert(S >= 2 && (S - 2) * NV <= 63, "stages");
    __shared__ __attribute__((aligned(1024))) int8_t smem[S * STAGE];

    const GemmArgs &a = kp.a;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave % WM, wn = wave / WM;
    int tm, tn;
    tile_of(blockIdx.x, kp.tiles_m, kp.tiles_n, kp.gm, tm, tn);
    const int64_t m0 = (int64_t)tm * TM, n0 = (int64_t)tn * TN;
    const int64_t M = a.M, N = a.N;
    const int K = (int)a.K;
    const int rows_w = (int)((N - n0) < TN ? (N - n0) : TN);
    const int rows_x = (int)((M - m0) < TM ? (M - m0) : TM);
    const __amdgpu_buffer_rsrc_t rw_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.wq + n0 * K), (short)0, rows_w * K, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t rx_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.xq + m0 * K), (short)0, rows_x * K, kRsrcWord3);

    // This lane's source in every load: row r0 + i*RPL, logical chunk kc0.
    const int c0 = wave * 64 + lane;
    const int r0 = c0 / CPR;
    const int kc0 = (c0 % CPR) ^ swz<BK>(r0);
    const int voff0 = r0 * K + kc0 * 16;

    // This lane's fragment offset inside a stage for K-step ks (the same for every
    // 32-row fragment, whose base differs by a constant).
    int fofs[KS];
    {
        const int sw = swz<BK>(lane & 31), h = lane >> 5;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            fofs[ks] = (lane & 31) * BK + (((2 * ks + h) ^ sw) << 4);
    }

    i32x16 acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j)
            acc[i][j] = i32x16{};

    const int nk = (K + BK - 1) / BK;

    // Per-lane source offset of panel kt's first load and the stride between loads.
    // Only the last panel can reach past K; there, lanes whose chunk starts at or past K
    // read from an offset beyond the buffer and get zeros. Panels kt >= nk read zeros
    // everywhere: the loop requests them to stay branch-free, into stages nobody reads.
    auto panel_src = [&](int kt, int &base, int &step) {
        const int k0 = kt * BK;
        const bool live = (kt < nk) & ((k0 + BK <= K) | (k0 + kc0 * 16 < K));
        base = live ? voff0 + k0 : kOOB;
        step = live ? RPL * K : 0;
    };
    // Loads [I0, I1) of the NV loads of one panel into the stage at byte offset so.
    auto issue = [&](auto i0c, auto i1c, int base, int step, int so) {
        constexpr int I0 = decltype(i0c)::value, I1 = decltype(i1c)::value;
        int8_t *dst = smem + so + wave * 64 * 16;
#pragma unroll
        for (int i = I0; i < I1; ++i) {
            if (i < LW)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rw_rsrc, (__attribute__((address_space(3))) void *)(dst + i * NT * 16), 16,
                    base + i * step, 0, 0, 0);
            else
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rx_rsrc,
                    (__attribute__((address_space(3))) void *)(dst + TN * BK + (i - LW) * NT * 16),
                    16, base + (i - LW) * step, 0, 0, 0);
        }
    };

    i32x4 fa[2][FN], fb[2][FM];
    auto read_frags = [&](int so, int ks, int buf) {
        const int8_t *sw_ = smem + so + wn * WTN * BK + fofs[ks];
        const int8_t *sx_ = smem + so + TN * BK + wm * WTM * BK + fofs[ks];
#pragma unroll
        for (int i = 0; i < FN; ++i)
            fa[buf][i] = *reinterpret_cast<const i32x4 *>(sw_ + i * 32 * BK);
#pragma unroll
        for (int j = 0; j < FM; ++j)
            fb[buf][j] = *reinterpret_cast<const i32x4 *>(sx_ + j * 32 * BK);
    };

    // Each K-step runs as G fenced groups: a slice of the next K-step's fragment reads and
    // of the loads of panel k+S-1, then a slice of this K-step's MFMAs. The matrix core
    // thus always has MFMAs queued while the memory instructions issue, and the reads
    // have the rest of the K-step to land.
    constexpr int NM = FN * FM, NR = FN + FM;
    constexpr int VPS = (NV + KS - 1) / KS;   // loads per K-step
    constexpr int G = NM >= 4 ? 4 : NM;       // groups per K-step
    auto kstep = [&](auto ksc, int so, int base, int step, int so_load) {
        constexpr int ks = decltype(ksc)::value;
        [&]<int... g>(std::integer_sequence<int, g...>) {
            ([&] {
                if constexpr (ks + 1 < KS) {
                    const int8_t *sw_ = smem + so + wn * WTN * BK + fofs[ks + 1];
                    const int8_t *sx_ = smem + so + TN * BK + wm * WTM * BK + fofs[ks + 1];
                    constexpr int r0_ = g * NR / G, r1_ = (g + 1) * NR / G;
#pragma unroll
                    for (int r = r0_; r < r1_; ++r) {
                        if (r < FN)
                            fa[(ks + 1) & 1][r] = *reinterpret_cast<const i32x4 *>(sw_ + r * 32 * BK);
                        else
                            fb[(ks + 1) & 1][r - FN] =
                                *reinterpret_cast<const i32x4 *>(sx_ + (r - FN) * 32 * BK);
                    }
                }
                constexpr int va = ks * VPS + g * VPS / G, vb = ks * VPS + (g + 1) * VPS / G;
                constexpr int v0 = va < NV ? va : NV, v1 = vb < NV ? vb : NV;
                issue(std::integral_constant<int, v0>{}, std::integral_constant<int, v1>{}, base,
                      step, so_load);
                __builtin_amdgcn_sched_barrier(0);
                constexpr int q0 = g * NM / G, q1 = (g + 1) * NM / G;
#pragma unroll
                for (int q = q0; q < q1; ++q)
                    acc[q / FM][q % FM] = __builtin_amdgcn_mfma_i32_32x32x32_i8(
                        fa[ks & 1][q / FM], fb[ks & 1][q % FM], acc[q / FM][q % FM], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
            }(), ...);
        }(std::make_integer_sequence<int, G>{});
    };

    if (nk > 0) {
        // Prologue: panels 0 .. S-2 into stages 0 .. S-2; wait for panel 0.
#pragma unroll
        for (int p = 0; p < S - 1; ++p) {
            int base, step;
            panel_src(p, base, step);
            issue(std::integral_constant<int, 0>{}, std::integral_constant<int, NV>{}, base, step,
                  p * STAGE);
        }
        __builtin_amdgcn_s_waitcnt(waitcnt_vm((S - 2) * NV));
        barrier_nofence();
        int st = 0;            // stage of panel kt
        int ld = S - 1;        // stage of panel kt + S - 1
        for (int kt = 0; kt < nk; ++kt) {
            int base, step;
            panel_src(kt + S - 1, base, step);
            read_frags(st * STAGE, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            [&]<int... ks>(std::integer_sequence<int, ks...>) {
                (kstep(std::integral_constant<int, ks>{}, st * STAGE, base, step, ld * STAGE), ...);
            }(std::make_integer_sequence<int, KS>{});
            // Panel kt+1 has landed once at most the S-2 younger panels are in flight.
            __builtin_amdgcn_s_waitcnt(waitcnt_vm((S - 2) * NV));
            barrier_nofence();
            st = (st + 1 == S) ? 0 : st + 1;
            ld = (ld + 1 == S) ? 0 : ld + 1;
        }
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));   // the zero-filling tail loads
    }
    store_tile<FN, FM, EPI>(acc, kp, m0 + wm * WTM, n0 + wn * WTN, lane);
}

// ---------------------------------------------------------------- tile registry

template <int TM, int TN, int BK, int WM, int WN, int S>
struct Tile {
    // S >= 2: pipelined direct-to-LDS kernel with S stages; S == 0: the simple
    // register-staged kernel only.
    static constexpr bool PIPE = S >= 2;
    static constexpr int threads = WM * WN * 64;
    static constexpr int lds = (PIPE ? S : 2) * (TM + TN) * BK;

    static hipError_t launch(Epilogue epi, bool vec, const KParams &kp, hipStream_t s) {
        const dim3 grid((unsigned)(kp.tiles_m * kp.tiles_n)), block(threads);
        if constexpr (PIPE) {
            if (vec) {
                if (epi == EPI_BF16)
                    hipLaunchKernelGGL((gemm_i8_lds_kernel<TM, TN, BK, WM, WN, S, EPI_BF16>), grid, block, 0, s, kp);
                else
                    hipLaunchKernelGGL((gemm_i8_lds_kernel<TM, TN, BK, WM, WN, S, EPI_I32>), grid, block, 0, s, kp);
                return hipGetLastError();
            }
        }
        if (vec) {
            if (epi == EPI_BF16)
                hipLaunchKernelGGL((gemm_i8_kernel<TM, TN, BK, WM, WN, true, EPI_BF16>), grid, block, 0, s, kp);
            else
                hipLaunchKernelGGL((gemm_i8_kernel<TM, TN, BK, WM, WN, true, EPI_I32>), grid, block, 0, s, kp);
        } else {
            if (epi == EPI_BF16)
                hipLaunchKernelGGL((gemm_i8_kernel<TM, TN, BK, WM, WN, false, EPI_BF16>), grid, block, 0, s, kp);
            else
                hipLaunchKernelGGL((gemm_i8_kernel<TM, TN, BK, WM, WN, false, EPI_I32>), grid, block, 0, s, kp);
        }
        return hipGetLastError();
    }
};

struct TileEntry {
    TileInfo info;
    int gm;
    hipError_t (*launch)(Epilogue, bool, const KParams &, hipStream_t);
};

#define W8A8_TILE(NAME, TM, TN, BK, WM, WN, GM, S)                                          \
    TileEntry {                                                                              \
        {NAME, TM, TN, BK, Tile<TM, TN, BK, WM, WN, S>::threads,                            \
         Tile<TM, TN, BK, WM, WN, S>::lds},                                                  \
            GM, &Tile<TM, TN, BK, WM, WN, S>::launch                                         \
    }

// Names: m<TM>n<TN>k<BK>w<WM>x<WN>[s<S>]; "s<S>" = direct-to-LDS pipelined kernel with S
// stages (used when the operands are 16-byte aligned and K % 16 == 0; otherwise the
// register-staged kernel of the same tile runs).
const TileEntry kTiles[] = {
    W8A8_TILE("m256n256k64w2x2s4", 256, 256, 64, 2, 2, 8, 4),
    W8A8_TILE("m256n256k128w2x2s2", 256, 256, 128, 2, 2, 8, 2),
    W8A8_TILE("m256n128k128w2x2s3", 256, 128, 128, 2, 2, 8, 3),
    W8A8_TILE("m128n256k128w2x2s3", 128, 256, 128, 2, 2, 8, 3),
    W8A8_TILE("m128n128k64w2x2s4", 128, 128, 64, 2, 2, 8, 4),
    W8A8_TILE("m256n256k64w2x4s4", 256, 256, 64, 2, 4, 8, 4),
    W8A8_TILE("m128n128k128w2x2s3", 128, 128, 128, 2, 2, 8, 3),
    W8A8_TILE("m128n128k128w2x2", 128, 128, 128, 2, 2, 8, 0),
    W8A8_TILE("m64n128k128w1x4", 64, 128, 128, 1, 4, 8, 0),
    W8A8_TILE("m32n128k128w1x4", 32, 128, 128, 1, 4, 8, 0),
    W8A8_TILE("m32n64k128w1x2", 32, 64, 128, 1, 2, 8, 0),
};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);

// Offline-chosen tile per shape. Entries are (M lower bound, M upper bound, N, K, tile);
// generated by the tile sweep and copied here.
struct TableEntry {
    int64_t m_lo, m_hi, n, k;
    int tile;
};
#include "tile_table.inc"

int fallback_tile(int64_t M, int64_t N, int64_t K) {
    (void)K;
    // Prefer the largest tile that still gives at least one workgroup per CU.
    const int64_t cus = 256;
    for (int id : {0, 2, 3, 4, 8}) {
        const TileInfo &t = kTiles[id].info;
        const int64_t tiles = ((M + t.tm - 1) / t.tm) * ((N + t.tn - 1) / t.tn);
        if (tiles >= cus)
            return id;
    }
    if (M <= 32)
        return 10;
    if (M <= 64)
        return 9;
    return 8;
}

}  // namespace

int tile_count() { return kNumTiles; }

const TileInfo *tile_info(int id) {
    return (id >= 0 && id < kNumTiles) ? &kTiles[id].info : nullptr;
}

int select_tile(int64_t M, int64_t N, int64_t K) {
    for (const TableEntry &e : kTileTable) {
        if (e.n == N && e.k == K && M >= e.m_lo && M <= e.m_hi && e.tile >= 0 &&
            e.tile < kNumTiles)
            return e.tile;
    }
    return fallback_tile(M, N, K);
}

size_t tile_workspace_bytes(int id, int64_t M, int64_t N, int64_t K) {
    (void)id; (void)M; (void)N; (void)K;
    return 0;
}

hipError_t launch_gemm(int id, Epilogue epi, bool vec, const GemmArgs &a, void *ws,
                       size_t ws_bytes, hipStream_t stream) {
    (void)ws; (void)ws_bytes;
    const TileEntry &t = kTiles[id];
    KParams kp;
    kp.a = a;
    kp.tiles_m = (int)((a.M + t.info.tm - 1) / t.info.tm);
    kp.tiles_n = (int)((a.N + t.info.tn - 1) / t.info.tn);
    kp.gm = t.gm;
    const size_t osz = (epi == EPI_BF16) ? 2 : 4;
    const uintptr_t align_need = (epi == EPI_BF16) ? 8 : 16;
    bool ov = (a.N % 4 == 0) && (reinterpret_cast<uintptr_t>(a.out) % align_need == 0);
    if (epi == EPI_BF16) {
        ov = ov && (reinterpret_cast<uintptr_t>(a.sw) % 16 == 0) &&
             (a.bias == nullptr || reinterpret_cast<uintptr_t>(a.bias) % 8 == 0);
    }
    (void)osz;
    kp.out_vec = ov ? 1 : 0;
    return t.launch(epi, vec, kp, stream);
}

}  // namespace w8a8
