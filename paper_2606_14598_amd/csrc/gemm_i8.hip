// int8 x int8 -> int32 GEMM on gfx950 matrix cores with the fused dequantization
// epilogue of the W8A8 linear (Section 3, "The fused kernel").
//
// Y[m][n] = bf16(fmaf((float)acc[m][n], sx[m] * sw[n], b[n])),
// acc[m][n] = sum_k Xq[m][k] * Wq[n][k], with Xq [M,K] and Wq [N,K] both K-contiguous.
//
// Kernels (one workgroup per TM x TN output tile unless noted):
//   * gemm_i8_lds_kernel, the main one. v_mfma_i32_32x32x32_i8 with the weight tile as
//     operand A (rows = output channels) and the activation tile as operand B (columns
//     = tokens), so each lane's accumulator holds 4 consecutive channels of one token.
//     K-panels of BK bytes move global -> LDS by direct-to-LDS buffer loads into an
//     S-stage ring (panel k+S-1 requested while panel k is multiplied); rows past M/N
//     and bytes past K read as zero through the buffer descriptors, so ragged tiles
//     need no branches. LDS rows are XOR-swizzled by row, conflict-free for the DMA
//     writes and the fragment reads. The bf16 epilogue stages 32-token chunks in LDS and
//     writes whole 16-byte row segments with streaming stores.
//   * Split-K variants of it: K divided among several workgroups per tile, int32
//     partials in a workspace, summed (exactly) by splitk_reduce_kernel, which also runs
//     the epilogue.
//   * gemm_i8_kernel: register-staged copies, for small tiles and for operands that are
//     not 16-byte aligned or whose K is not a multiple of 16 (byte loads).
//   * gemm_i8_skinny_kernel: few tokens (M <= 128). A workgroup streams 16*FNB weight
//     rows once for all tokens with v_mfma_i32_16x16x64_i8, its wavefronts splitting K,
//     partial sums reduced in LDS.
//   * gemm_i8_wsx_kernel: few tokens, in blocks of 16 or 32. The same product with the
//     token block staged once per workgroup in LDS and the weight streamed through a
//     register ring; it also quantizes the bf16 token rows itself for the one-launch
//     linear.
// Workgroup ids are remapped so that each XCD (which receives every 8th id) owns a
// contiguous run of tiles, traversed in groups of GM token-tiles: the operand panels a
// run touches stay in that XCD's L2. The integer accumulation is exact, so every tile,
// split and order gives identical bits.
#include "w8a8_internal.hpp"
#include "quant_math.hpp"

#include <atomic>
#include <utility>

namespace w8a8 {
namespace {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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
    int out_vec;     // 0: scalar stores; 1: rows 8-byte (bf16) / 16-byte (int32) aligned
                     // with N % 4 == 0; 2 (bf16): rows 16-byte aligned with N % 8 == 0
    int k_split;     // workgroups per output tile along K (1: the whole K, direct epilogue)
    int k_chunk;     // K bytes per split (a multiple of BK; K when unsplit)
    int part_vec;    // partial rows 16-byte aligned (N % 4 == 0)
    int32_t *part;   // k_split > 1: int32 partials [k_split][M][N]
    const uint16_t *x;   // the small fused linear: bf16 X [M,K] (a.xq, a.sx unused)
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

// bf16 epilogue through LDS, for outputs whose rows are 16-byte aligned with N % 8 == 0
// (kp.out_vec == 2). The wavefront converts one 32-token chunk of its tile at a time into
// a private LDS region of 32 rows x (2*WTN + 16) bytes (the pad spreads the 32 rows over
// the banks), then writes the chunk back to global memory row by row with 16-byte
// stores, so every store instruction covers whole contiguous row segments. The token
// scales, channel scales and bias (as fp32) of the tile come from LDS (t_sx, t_sw, t_b,
// indexed from the wavefront's first token / channel; out-of-range entries are 0).
// Needs a barrier before it (the region overlaps the panel stages) and
// 32 * (2*WTN + 16) bytes of LDS per wavefront.
//
// With one wavefront per SIMD (NW <= 4) nothing else hides the LDS latencies, so the
// chunks are software-pipelined: the row reads of chunk j are issued, then chunk j+1 is
// converted into the same region while they are in flight, then chunk j is stored. One
// region suffices because a wavefront's LDS instructions execute in order: the reads of
// chunk j see its data before the writes of chunk j+1 replace it. The channel scales and
// bias of narrow wavefront tiles (FN <= 2) are then held in registers. With more
// wavefronts per SIMD registers are short and the other wavefronts hide the latencies:
// each chunk is converted, read back and stored in turn, with the vectors read from LDS.
// A tile that lies wholly inside the output stores without bounds tests.
template <int FN, int FM, int NW>
__device__ __forceinline__ void store_tile_bf16_lds(const i32x16 (&acc)[FN][FM],
                                                    const KParams &kp, int64_t m_base,
                                                    int64_t n_base, int lane,
                                                    int8_t *region, const float *t_sx,
                                                    const float *t_sw, const float *t_b) {
    constexpr int WTN = FN * 32;
    constexpr int RS = 2 * WTN + 16;          // region row stride in bytes
    constexpr int CPRO = WTN / 8;             // 16-byte chunks per output row
    constexpr int RPQ = 64 / CPRO;            // whole rows covered by one 64-lane read
    constexpr int NQ = (32 + RPQ - 1) / RPQ;  // reads (and stores) per lane per chunk
    // With 12 chunks per row (96-channel wavefront tiles) a read covers 5 rows with 60
    // lanes and the 7th read only rows 30 and 31: lanes and rows past those carry nothing.
    constexpr bool EXACT = RPQ * CPRO == 64 && NQ * RPQ == 32;
    static_assert(RPQ >= 1, "row split");
    const GemmArgs &a = kp.a;
    const int64_t M = a.M, N = a.N;
    const int h = lane >> 5, r = lane & 31;
    uint16_t *out = static_cast<uint16_t *>(a.out);

    constexpr bool PIPE = NW <= 4;
    constexpr bool HOIST = PIPE && FN <= 2;
    constexpr int HF = HOIST ? FN : 1;
    f32x4 sw4[HF][4], b4[HF][4];
    if constexpr (HOIST) {
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int c = i * 32 + g * 8 + h * 4;
                sw4[i][g] = *reinterpret_cast<const f32x4 *>(t_sw + c);
                b4[i][g] = *reinterpret_cast<const f32x4 *>(t_b + c);
            }
    }
    float sxv[FM];
#pragma unroll
    for (int j = 0; j < FM; ++j)
        sxv[j] = t_sx[j * 32 + r];
    // Chunk j into the region: this lane's token r, channels c .. c+3 per (i, g).
    auto convert = [&](auto jc) {
        constexpr int j = decltype(jc)::value;
        const float sxm = sxv[j];
#pragma unroll
        for (int i = 0; i < FN; ++i) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int c = i * 32 + g * 8 + h * 4;
                f32x4 s4, c4;
                if constexpr (HOIST) {
                    s4 = sw4[i][g];
                    c4 = b4[i][g];
                } else {
                    s4 = *reinterpret_cast<const f32x4 *>(t_sw + c);
                    c4 = *reinterpret_cast<const f32x4 *>(t_b + c);
                }
                uint16_t hv[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float sc = sxm * s4[e];
                    const float y = __builtin_fmaf((float)acc[i][j][4 * g + e], sc, c4[e]);
                    hv[e] = __builtin_bit_cast(uint16_t, (__bf16)y);
                }
                uint2 pk;
                pk.x = (uint32_t)hv[0] | ((uint32_t)hv[1] << 16);
                pk.y = (uint32_t)hv[2] | ((uint32_t)hv[3] << 16);
                *reinterpret_cast<uint2 *>(region + r * RS + c * 2) = pk;
            }
        }
    };
    // Lane's share of a chunk: rows row0 + RPQ*s, 8 channels at chunk ch.
    const int row0 = lane / CPRO, ch = lane % CPRO;
    auto live = [&](int s) { return EXACT || (lane < RPQ * CPRO && row0 + RPQ * s < 32); };
    const bool full = (m_base + FM * 32 <= M) && (n_base + WTN <= N);   // wave-uniform
    if constexpr (PIPE)
        convert(std::integral_constant<int, 0>{});
    [&]<int... j>(std::integer_sequence<int, j...>) {
        ([&] {
            if constexpr (!PIPE)
                convert(std::integral_constant<int, j>{});
            u32x4 v[NQ];
#pragma unroll
            for (int s = 0; s < NQ; ++s)
                v[s] = live(s) ? *reinterpret_cast<const u32x4 *>(region + (row0 + RPQ * s) * RS +
                                                                  ch * 16)
                               : u32x4{};
            if constexpr (PIPE && j + 1 < FM)
                convert(std::integral_constant<int, j + 1>{});
            const int64_t mm = m_base + j * 32 + row0;
            const int64_t nn = n_base + ch * 8;
            // Streaming (nontemporal) stores: the output is not read again by this
            // kernel, and lines that bypass the L2's write-back set leave less to flush
            // when the kernel ends.
            u32x4 *dst = reinterpret_cast<u32x4 *>(out + mm * N + nn);
            if (full) {
#pragma unroll
                for (int s = 0; s < NQ; ++s)
                    if (live(s))
                        __builtin_nontemporal_store(v[s], dst + (int64_t)s * RPQ * N / 8);
            } else {
#pragma unroll
                for (int s = 0; s < NQ; ++s)
                    if (live(s) && mm + RPQ * s < M && nn < N)
                        __builtin_nontemporal_store(v[s], dst + (int64_t)s * RPQ * N / 8);
            }
        }(), ...);
    }(std::make_integer_sequence<int, FM>{});
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
//   * Panels go straight from global memory to LDS (buffer_load_dwordx4 ... lds). Load
//     g of a panel (wavefront g % NW issues it) fills 64 chunks of 16 bytes of the
//     weight part (g < IW) or of the activation part: lane l writes chunk 64g' + l, i.e.
//     row RPI*g' + l/CPR, physical chunk l % CPR, and therefore fetches logical chunk
//     (l % CPR) ^ swz(row) of that row. No staging registers, no ds_write.
//   * S LDS stages in a ring: panel k+S-1 is requested while panel k is multiplied, so a
//     load has S-1 panels of MFMA work to arrive; one wait + barrier per panel makes
//     panel k+1 visible to every wavefront (with S >= 3 one K-step before panel k ends,
//     so the next panel's first fragments are read behind the last K-step's MFMAs).
//   * MFMA operand fragments are double-buffered across the BK/32 K-steps of a panel:
//     each K-step issues the ds_reads of the next K-step's fragments and its share of
//     the loads of panel k+S-1, one memory instruction between consecutive MFMAs.
//   * Split-K (kp.k_split > 1): the workgroup covers one K-range of its tile and stores
//     the int32 partial instead of running the epilogue.
template <int TM, int TN, int BK, int WM, int WN, int S, int EPI>
__global__ void __launch_bounds__(WM *WN * 64)
gemm_i8_lds_kernel(KParams kp) {
    constexpr int NW = WM * WN;                // wavefronts
    constexpr int WTM = TM / WM, WTN = TN / WN;
    constexpr int FM = WTM / 32, FN = WTN / 32;
    constexpr int CPR = BK / 16;
    constexpr int RPI = 64 / CPR;              // rows filled by one load instruction
    constexpr int IW = TN / RPI, IX = TM / RPI;   // load instructions per panel (whole WG)
    constexpr int NI = IW + IX;
    constexpr int NV = (NI + NW - 1) / NW;     // load instructions per wavefront per panel
    constexpr int STAGE = (TN + TM) * BK;
    constexpr int KS = BK / 32;
    static_assert(FM >= 1 && FN >= 1 && WTM % 32 == 0 && WTN % 32 == 0, "wave tile");
    static_assert(TN % RPI == 0 && TM % RPI == 0, "load split");
    static_assert(S >= 2 && (S - 2) * NV <= 63, "stages");
    // One LDS object holds the panel stages and, behind them, the epilogue vectors of the
    // tile (token scales, channel scales, bias as fp32). A single object keeps the
    // compiler's LDS-DMA tracking exact: with a second LDS variable it makes every
    // ds_read wait for all in-flight panel loads.
    constexpr int NSC = EPI == EPI_BF16 ? 1 : 0;
    __shared__ __attribute__((aligned(1024))) int8_t smem[S * STAGE + NSC * (TM + 2 * TN) * 4];
    float *const t_sx = reinterpret_cast<float *>(smem + S * STAGE);
    float *const t_sw = t_sx + NSC * TM;
    float *const t_b = t_sw + NSC * TN;

    const GemmArgs &a = kp.a;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave % WM, wn = wave / WM;
    // Split-K: workgroup b works on K-range `split` of tile b mod (tiles_m * tiles_n).
    int blk = blockIdx.x, split = 0;
    if (kp.k_split > 1) {
        const int ntiles = kp.tiles_m * kp.tiles_n;
        split = blk / ntiles;
        blk -= split * ntiles;
    }
    int tm, tn;
    tile_of(blk, kp.tiles_m, kp.tiles_n, kp.gm, tm, tn);
    const int64_t m0 = (int64_t)tm * TM, n0 = (int64_t)tn * TN;
    const int64_t M = a.M, N = a.N;
    const int K = (int)a.K;                              // row stride of Xq and Wq
    const int kbeg = split * kp.k_chunk;                 // this workgroup's first K byte
    const int KL = (K - kbeg) < kp.k_chunk ? (K - kbeg) : kp.k_chunk;   // its K length
    const int rows_w = (int)((N - n0) < TN ? (N - n0) : TN);
    const int rows_x = (int)((M - m0) < TM ? (M - m0) : TM);
    const __amdgpu_buffer_rsrc_t rw_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.wq + n0 * K + kbeg), (short)0, rows_w * K - kbeg, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t rx_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.xq + m0 * K + kbeg), (short)0, rows_x * K - kbeg, kRsrcWord3);

    // Load instruction g (0 <= g < NI; the first IW fill the weight part of a stage, the
    // rest the activation part) is issued by wavefront g % NW; its lane l fills LDS chunk
    // 64*g' + l of that part (g' = g or g - IW), i.e. row RPI*g' + l/CPR, physical chunk
    // l % CPR, and so fetches logical chunk (l % CPR) ^ swz(row) of that row.
    const int lrow = lane / CPR, lchunk = lane % CPR;

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

    const int nk = (KL + BK - 1) / BK;

    // Loads [I0, I1) of this wavefront's NV load instructions of panel kt into the stage
    // at byte offset so. Only the last panel can reach past K; there, lanes whose chunk
    // starts at or past K read from an offset beyond the buffer and get zeros. Panels
    // kt >= nk read zeros everywhere: the loop requests them to stay branch-free, into
    // stages nobody reads.
    auto issue = [&](auto i0c, auto i1c, int kt, int so) {
        constexpr int I0 = decltype(i0c)::value, I1 = decltype(i1c)::value;
        const int k0 = kt * BK;
        const bool full = (kt < nk) & (k0 + BK <= KL);
        const bool inrange = kt < nk;
#pragma unroll
        for (int i = I0; i < I1; ++i) {
            const int g = i * NW + wave;
            if (i * NW + NW > NI && g >= NI)
                break;                                       // wave-uniform
            const bool isw = g < IW;
            const int gg = isw ? g : g - IW;
            const int row = gg * RPI + lrow;
            const int kc = lchunk ^ swz<BK>(row);
            const bool ok = full | (inrange & (k0 + kc * 16 < KL));
            const int off = ok ? row * K + k0 + kc * 16 : kOOB;
            int8_t *dst = smem + so + (isw ? 0 : TN * BK) + gg * 1024;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                isw ? rw_rsrc : rx_rsrc, (__attribute__((address_space(3))) void *)dst, 16,
                off, 0, 0, 0);
        }
    };

    // Wait until at most `younger` panels' loads of this wavefront are in flight. When NI
    // is not a multiple of NW the last NW - NI % NW wavefronts issue one load fewer per
    // panel, so their count differs (a wave-uniform branch).
    auto wait_loads = [&](auto youngerc) {
        constexpr int Y = decltype(youngerc)::value;
        if constexpr (NI % NW == 0) {
            __builtin_amdgcn_s_waitcnt(waitcnt_vm(Y * NV));
        } else {
            if (wave < NI % NW)
                __builtin_amdgcn_s_waitcnt(waitcnt_vm(Y * NV));
            else
                __builtin_amdgcn_s_waitcnt(waitcnt_vm(Y * (NV - 1)));
        }
    };
    // Before the last K-step of panel kt (S >= 3): panel kt+1 has landed once at most the
    // full panels kt+2 .. kt+S-2 and the slices of panel kt+S-1 issued so far (K-steps
    // 0 .. KS-2) are in flight. A wavefront with one load fewer skips the last slot.
    auto wait_loads_mid = [&]() {
        constexpr int VPS_ = (NV + KS - 1) / KS;
        constexpr int ISS = (KS - 1) * VPS_ < NV ? (KS - 1) * VPS_ : NV;
        constexpr int ISS1 = (KS - 1) * VPS_ < NV - 1 ? (KS - 1) * VPS_ : NV - 1;
        static_assert(S < 3 || (S - 3) * NV + ISS <= 63, "vmcnt range");
        if constexpr (NI % NW == 0) {
            __builtin_amdgcn_s_waitcnt(waitcnt_vm((S - 3) * NV + ISS));
        } else {
            if (wave < NI % NW)
                __builtin_amdgcn_s_waitcnt(waitcnt_vm((S - 3) * NV + ISS));
            else
                __builtin_amdgcn_s_waitcnt(waitcnt_vm((S - 3) * (NV - 1) + ISS1));
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

    // Each K-step interleaves its memory instructions one by one with its MFMAs: the
    // ds_reads of the next K-step's fragments first (they must land within this step),
    // then its share of the loads of panel k+S-1, each followed by one MFMA, with a
    // scheduling fence around every pair. The matrix core then always has an MFMA
    // queued while a memory instruction issues.
    //
    // With three or more stages (EARLY) the per-panel wait and barrier come one K-step
    // before the panel ends, and the last K-step reads the first fragments of the next
    // panel (from stage so_rd), so their LDS latency hides behind its MFMAs instead of
    // stalling the first MFMA of every panel. With two stages the barrier stays at the
    // panel's end: one K-step earlier it would cut the time the next panel's loads have to
    // land, and measured no faster on the 288 x 256 tile.
    constexpr int NM = FN * FM, NR = FN + FM;
    // Loads per K-step. With three or more stages a panel's loads are spread over all its
    // K-steps (they have S-2 more panels to land). With two stages they all go out in the
    // first K-step: the stage they fill was released by the previous panel's barrier, and
    // the whole panel is then left for them to land before its closing wait (spreading
    // them left the last ones a single K-step; measured 1.5-2% slower on 288 x 256).
    constexpr int LKS = S == 2 ? 1 : KS;
    constexpr int VPS = (NV + LKS - 1) / LKS;
    constexpr bool EARLY = S >= 3;
    static_assert(KS % 2 == 0, "fragment double buffer: K-step 0 of a panel uses buffer 0");
    auto kstep = [&](auto ksc, int so, int kt_load, int so_load, int so_rd) {
        constexpr int ks = decltype(ksc)::value;
        constexpr bool next_panel = EARLY && ks + 1 == KS;
        constexpr int nr = (ks + 1 < KS || next_panel) ? NR : 0;
        constexpr int fk = ks + 1 < KS ? ks + 1 : 0;
        constexpr int va = ks * VPS < NV ? ks * VPS : NV;
        constexpr int vb = (ks + 1) * VPS < NV ? (ks + 1) * VPS : NV;
        constexpr int nops = nr + (vb - va);
        constexpr int steps = NM > nops ? NM : nops;
        const int8_t *sw_ = smem + so_rd + wn * WTN * BK + fofs[fk];
        const int8_t *sx_ = smem + so_rd + TN * BK + wm * WTM * BK + fofs[fk];
        [&]<int... q>(std::integer_sequence<int, q...>) {
            ([&] {
                if constexpr (q < nr) {
                    if constexpr (q < FN)
                        fa[(ks + 1) & 1][q] = *reinterpret_cast<const i32x4 *>(sw_ + q * 32 * BK);
                    else
                        fb[(ks + 1) & 1][q - FN] =
                            *reinterpret_cast<const i32x4 *>(sx_ + (q - FN) * 32 * BK);
                } else if constexpr (q < nops) {
                    issue(std::integral_constant<int, va + q - nr>{},
                          std::integral_constant<int, va + q - nr + 1>{}, kt_load, so_load);
                }
                if constexpr (q < NM) {
                    __builtin_amdgcn_sched_barrier(0);
                    acc[q / FM][q % FM] = __builtin_amdgcn_mfma_i32_32x32x32_i8(
                        fa[ks & 1][q / FM], fb[ks & 1][q % FM], acc[q / FM][q % FM], 0, 0, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
            }(), ...);
        }(std::make_integer_sequence<int, steps>{});
    };

    // Tile vectors for the epilogue: fetched now, parked in LDS after the prologue (their
    // latency hides behind the first panel's).
    constexpr int NT = NW * 64;
    constexpr int VSX = (TM + NT - 1) / NT, VSW = (TN + NT - 1) / NT;
    float r_sx[VSX], r_sw[VSW], r_b[VSW];
    if constexpr (EPI == EPI_BF16) {
#pragma unroll
        for (int v = 0; v < VSX; ++v) {
            const int idx = v * NT + (int)threadIdx.x;
            r_sx[v] = (idx < TM && m0 + idx < M) ? a.sx[m0 + idx] : 0.0f;
        }
#pragma unroll
        for (int v = 0; v < VSW; ++v) {
            const int idx = v * NT + (int)threadIdx.x;
            const bool in = idx < TN && n0 + idx < N;
            r_sw[v] = in ? a.sw[n0 + idx] : 0.0f;
            r_b[v] = (in && a.bias) ? __uint_as_float((uint32_t)a.bias[n0 + idx] << 16) : 0.0f;
        }
    }
    auto park_vectors = [&]() {
        if constexpr (EPI == EPI_BF16) {
#pragma unroll
            for (int v = 0; v < VSX; ++v) {
                const int idx = v * NT + (int)threadIdx.x;
                if (idx < TM)
                    t_sx[idx] = r_sx[v];
            }
#pragma unroll
            for (int v = 0; v < VSW; ++v) {
                const int idx = v * NT + (int)threadIdx.x;
                if (idx < TN) {
                    t_sw[idx] = r_sw[v];
                    t_b[idx] = r_b[v];
                }
            }
            // The next (fence-free) barrier publishes these stores: complete them first.
            __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
        }
    };

    if (nk > 0) {
        // Prologue: panels 0 .. S-2 into stages 0 .. S-2; wait for panel 0.
#pragma unroll
        for (int p = 0; p < S - 1; ++p)
            issue(std::integral_constant<int, 0>{}, std::integral_constant<int, NV>{}, p,
                  p * STAGE);
        wait_loads(std::integral_constant<int, S - 2>{});
        park_vectors();
        barrier_nofence();
        int st = 0;            // stage of panel kt
        int ld = S - 1;        // stage of panel kt + S - 1
        if constexpr (EARLY) {
            read_frags(0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
        for (int kt = 0; kt < nk; ++kt) {
            const int nx = (st + 1 == S) ? 0 : st + 1;
            if constexpr (EARLY) {
                [&]<int... ks>(std::integer_sequence<int, ks...>) {
                    (kstep(std::integral_constant<int, ks>{}, st * STAGE, kt + S - 1, ld * STAGE,
                           st * STAGE), ...);
                }(std::make_integer_sequence<int, KS - 1>{});
                // Panel kt+1 is in LDS for every wavefront after this barrier. The
                // lgkmcnt(0) first: this wavefront's reads of panel kt's stage are done
                // before anyone can pass the barrier and, one panel later, refill it.
                wait_loads_mid();
                __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
                barrier_nofence();
                kstep(std::integral_constant<int, KS - 1>{}, st * STAGE, kt + S - 1,
                      ld * STAGE, nx * STAGE);
            } else {
                read_frags(st * STAGE, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
                [&]<int... ks>(std::integer_sequence<int, ks...>) {
                    (kstep(std::integral_constant<int, ks>{}, st * STAGE, kt + S - 1,
                           ld * STAGE, st * STAGE), ...);
                }(std::make_integer_sequence<int, KS>{});
                // Panel kt+1 has landed once at most the S-2 younger panels are in flight.
                wait_loads(std::integral_constant<int, S - 2>{});
                barrier_nofence();
            }
            st = nx;
            ld = (ld + 1 == S) ? 0 : ld + 1;
        }
        // The zero-filling tail loads, and (S >= 3) the last K-step's reads of the stage
        // after the final panel, whose data nobody uses.
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
        __builtin_amdgcn_s_waitcnt(0xC07F);
    } else {
        park_vectors();
    }
    if (kp.k_split > 1) {
        // Split-K: store this K-range's int32 partial; the reduce kernel sums the splits
        // and runs the epilogue.
        KParams kq = kp;
        kq.a.out = kp.part + (int64_t)split * M * N;
        kq.out_vec = kp.part_vec;
        store_tile<FN, FM, EPI_I32>(acc, kq, m0 + wm * WTM, n0 + wn * WTN, lane);
        return;
    }
    if constexpr (EPI == EPI_BF16) {
        static_assert(NW * 32 * (2 * WTN + 16) <= S * STAGE, "epilogue staging");
        if (kp.out_vec == 2) {
            barrier_nofence();   // every wavefront is done reading the panel stages
            store_tile_bf16_lds<FN, FM, NW>(acc, kp, m0 + wm * WTM, n0 + wn * WTN, lane,
                                        smem + wave * 32 * (2 * WTN + 16), t_sx + wm * WTM,
                                        t_sw + wn * WTN, t_b + wn * WTN);
            return;
        }
    }
    store_tile<FN, FM, EPI>(acc, kp, m0 + wm * WTM, n0 + wn * WTN, lane);
}

// Weight-streaming kernel for few tokens (M <= 16 * FMB): the product is bound by reading
// W once, so there is no LDS staging of operands. A workgroup owns 16 * FNB output
// channels and every token; its NW wavefronts take K in super-steps of 256 bytes
// (super-step j by wavefront j % NW). v_mfma_i32_16x16x64_i8: lane l holds row l % 16 of
// an operand fragment and K-group l / 16. A dot product is unchanged by any permutation
// of K applied to both operands alike, so in super-step j lane (r, g) takes bytes
// [256j + 64s + 16g, +16) of its row for K-step s = 0..3: every load instruction reads
// whole 64-byte row segments, with the same map for W (rows = channels) and X (rows =
// tokens). Partial accumulators are summed across wavefronts in LDS (integer, exact),
// then the epilogue runs as in the tiled kernels: lane l of a 16x16 accumulator holds
// token l % 16 and channels 4(l / 16) + e.
//
// QX (the small fused linear): the workgroup first quantizes its own token rows of the
// bf16 X with the row quantizer's arithmetic (two passes over each row: the absmax,
// then the codes) into LDS, rows of K + 16 bytes, and their scales; the product then
// reads the token fragments and the epilogue the scales from there. The linear is then
// one launch. Each token block is quantized by every channel block that uses it, which
// the host allows only while those repeated reads of X stay small.
template <int FMB, int FNB, int NW, int EPI, bool QX = false>
__global__ void __launch_bounds__(NW * 64)
gemm_i8_skinny_kernel(KParams kp) {
    const GemmArgs &a = kp.a;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r = lane & 15, g = lane >> 4;
    extern __shared__ __attribute__((aligned(16))) int8_t qx_lds[];
    // Workgroup b: channel block b % tiles_n, token block b / tiles_n (more than one
    // token block only when more than 16 * FMB tokens are forced onto this kernel).
    const int64_t n0 = (int64_t)(blockIdx.x % kp.tiles_n) * (16 * FNB);
    const int64_t mb = (int64_t)(blockIdx.x / kp.tiles_n) * (16 * FMB);
    const int64_t N = a.N;
    const int K = (int)a.K;
    const int rows_w = (int)((N - n0) < 16 * FNB ? (N - n0) : 16 * FNB);
    const int rows_x = (int)((a.M - mb) < 16 * FMB ? (a.M - mb) : 16 * FMB);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.wq + n0 * K), (short)0, rows_w * K, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.xq + mb * K), (short)0, rows_x * K, kRsrcWord3);
    // QX: codes of token row i at qx_lds + i * QS, its scale at qx_scale[i].
    const int QS = K + 16;
    float *const qx_scale = reinterpret_cast<float *>(qx_lds + rows_x * QS);
    if constexpr (QX) {
        // One wavefront per row: the absmax pass, then the codes (the row is read again,
        // from cache).
        const int nvec = K >> 3;
        for (int i = wave; i < rows_x; i += NW) {
            const uint4 *src = reinterpret_cast<const uint4 *>(kp.x + (mb + i) * (int64_t)K);
            uint32_t mx = 0;
            for (int vi = lane; vi < nvec; vi += 64)
                mx = max(mx, qmath::absmax8(src[vi]));
            mx = qmath::wave_max(mx);
            const qmath::RowScale rs = qmath::row_scale(mx);
            for (int vi = lane; vi < nvec; vi += 64)
                *reinterpret_cast<uint2 *>(qx_lds + i * QS + vi * 8) = qmath::code8(src[vi], rs.inv);
            if (lane == 0)
                qx_scale[i] = rs.scale;
        }
        __syncthreads();
    }

    i32x4 acc[FNB][FMB];
#pragma unroll
    for (int c = 0; c < FNB; ++c)
#pragma unroll
        for (int b = 0; b < FMB; ++b)
            acc[c][b] = i32x4{0, 0, 0, 0};

    const int nss = (K + 255) / 256;
    for (int j = wave; j < nss; j += NW) {
        const int kb = j * 256 + g * 16;
        i32x4 wv[FNB][4];
#pragma unroll
        for (int c = 0; c < FNB; ++c)
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int k = kb + s * 64, row = c * 16 + r;
                const int off = (k < K && row < rows_w) ? row * K + k : kOOB;
                wv[c][s] = __builtin_bit_cast(
                    i32x4, __builtin_amdgcn_raw_buffer_load_b128(rw, off, 0, 0));
            }
#pragma unroll
        for (int b = 0; b < FMB; ++b) {
            const int m = b * 16 + r;
            i32x4 xv[4];
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int k = kb + s * 64;
                if constexpr (QX) {
                    xv[s] = (k < K && m < rows_x)
                                ? *reinterpret_cast<const i32x4 *>(qx_lds + m * QS + k)
                                : i32x4{0, 0, 0, 0};
                } else {
                    const int off = (k < K && m < rows_x) ? m * K + k : kOOB;
                    xv[s] = __builtin_bit_cast(
                        i32x4, __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, 0));
                }
            }
#pragma unroll
            for (int c = 0; c < FNB; ++c)
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    acc[c][b] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wv[c][s], xv[s], acc[c][b],
                                                                     0, 0, 0);
        }
    }

    // Cross-wavefront reduction: red[wave][c][b] holds each lane's 4 partial sums.
    __shared__ i32x4 red[NW][FNB * FMB][64];
#pragma unroll
    for (int c = 0; c < FNB; ++c)
#pragma unroll
        for (int b = 0; b < FMB; ++b)
            red[wave][c * FMB + b][lane] = acc[c][b];
    __syncthreads();
    for (int cb = wave; cb < FNB * FMB; cb += NW) {
        const int c = cb / FMB, b = cb % FMB;
        i32x4 t = red[0][cb][lane];
#pragma unroll
        for (int w = 1; w < NW; ++w)
            t += red[w][cb][lane];
        const int64_t n = n0 + c * 16 + g * 4;
        if (b * 16 + r >= rows_x || n >= N)
            continue;
        const int64_t m = mb + b * 16 + r;
        if constexpr (EPI == EPI_I32) {
            int32_t *o = static_cast<int32_t *>(a.out) + m * N + n;
            if (kp.out_vec && n + 3 < N) {
                *reinterpret_cast<i32x4 *>(o) = t;
            } else {
                for (int e = 0; e < 4 && n + e < N; ++e)
                    o[e] = t[e];
            }
        } else {
            uint16_t *o = static_cast<uint16_t *>(a.out) + m * N + n;
            const float sxm = QX ? qx_scale[b * 16 + r] : a.sx[m];
            uint16_t hv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (n + e < N) {
                    const float bb = a.bias ? __uint_as_float((uint32_t)a.bias[n + e] << 16) : 0.0f;
                    const float y = __builtin_fmaf((float)t[e], sxm * a.sw[n + e], bb);
                    hv[e] = __builtin_bit_cast(uint16_t, (__bf16)y);
                }
            }
            if (kp.out_vec && n + 3 < N) {
                uint2 pk;
                pk.x = (uint32_t)hv[0] | ((uint32_t)hv[1] << 16);
                pk.y = (uint32_t)hv[2] | ((uint32_t)hv[3] << 16);
                *reinterpret_cast<uint2 *>(o) = pk;
            } else {
                for (int e = 0; e < 4 && n + e < N; ++e)
                    o[e] = hv[e];
            }
        }
    }
}

// LDS layout of the few-token kernel with the token block in LDS (gemm_i8_wsx_kernel):
// a head of 16 * fmb row scales and nw cross-wavefront maxima (256-byte aligned), then
// the token code rows of wsx_row_stride(K) bytes (= 16 mod 256: the 16 rows of a
// fragment read fall in distinct banks) and, with QX, the bf16 rows of
// wsx_stage_stride(K) bytes. After the main loop the reduction array (nw x fnb x fmb x
// 1 KB) takes the place of the rows, so the object holds the larger of the two.
__host__ __device__ constexpr int wsx_row_stride(int K) { return (K + 1023) / 1024 * 1024 + 16; }
__host__ __device__ constexpr int wsx_stage_stride(int K) { return (2 * K + 1023) / 1024 * 1024; }
__host__ __device__ constexpr int wsx_head_bytes(int fmb, int nw) {
    return (64 * fmb + 4 * nw + 255) / 256 * 256;
}
__host__ __device__ constexpr int64_t wsx_lds_bytes(int64_t rows, int64_t K, bool qx, int fmb,
                                                    int fnb, int nw) {
    const int64_t body = rows * ((K + 1023) / 1024 * 1024 + 16) +
                         (qx ? rows * ((2 * K + 1023) / 1024 * 1024) : 0);
    const int64_t red = (int64_t)nw * fnb * fmb * 1024;
    return wsx_head_bytes(fmb, nw) + (body > red ? body : red);
}

// Weight-streaming kernel with a register ring and the token block staged in LDS, for a
// few tokens (M <= 16 * FMB per block). The product is bound by reading W once. A
// workgroup owns 16 * FNB channels; its NW wavefronts split K in super-steps of 128
// bytes (super-step j to wavefront j % NW) and keep D super-steps of their weight
// fragments in flight in registers, loaded straight from global memory. Every
// wavefront needs the whole token block, so the block goes to LDS once per workgroup:
// its loads are issued first, by direct-to-LDS buffer loads, then the weight ring, and
// the workgroup waits only for the token loads before it starts (the weight loads stay
// in flight). With QX (the one-launch linear) the bf16 rows are staged instead and
// quantized in LDS with the row quantizer's arithmetic while the weight loads are in
// flight.
//
// v_mfma_i32_16x16x64_i8: lane (r, g) holds row r = lane % 16 of a fragment and 16
// K-bytes; in super-step j it takes bytes [128 j + 64 s + 16 g, +16) for K-step s = 0, 1
// (the same permutation of K for both operands leaves the dot product unchanged), so a
// weight load reads 64 contiguous bytes of 16 rows. Weight rows past N and bytes past K
// read as zero through the buffer descriptor. LDS rows of the token block are QS bytes
// apart, QS = 16 (mod 256), so the 16 rows of a fragment read hit distinct banks. Partial
// sums meet in LDS (integer, exact), then the epilogue runs.
template <int FMB, int FNB, int NW, int D, int EPI, bool QX>
__global__ void __launch_bounds__(NW * 64)
gemm_i8_wsx_kernel(KParams kp) {
    const GemmArgs &a = kp.a;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int r = lane & 15, g = lane >> 4;
    const int64_t n0 = (int64_t)(blockIdx.x % kp.tiles_n) * (16 * FNB);
    const int64_t mb = (int64_t)(blockIdx.x / kp.tiles_n) * (16 * FMB);
    const int64_t M = a.M, N = a.N;
    const int K = (int)a.K;
    const int rows_w = (int)((N - n0) < 16 * FNB ? (N - n0) : 16 * FNB);
    const int rows_x = (int)((M - mb) < 16 * FMB ? (M - mb) : 16 * FMB);
    const int QS = wsx_row_stride(K);

    // One dynamic LDS object (the compiler's tracking of direct-to-LDS loads stays
    // exact), laid out as wsx_lds_bytes describes: QX scales and cross-wavefront maxima,
    // then the token rows and QX staging rows, whose place the reduction array takes
    // after the main loop.
    extern __shared__ __attribute__((aligned(1024))) int8_t wsx_lds[];
    const int SB = wsx_stage_stride(K);
    float *const qscale = reinterpret_cast<float *>(wsx_lds);
    uint32_t *const pmax = reinterpret_cast<uint32_t *>(qscale + 16 * FMB);
    int8_t *const xs = wsx_lds + wsx_head_bytes(FMB, NW);         // rows_x x QS codes
    int8_t *const stage = xs + rows_x * QS;                       // QX: bf16 rows
    i32x4 *const red = reinterpret_cast<i32x4 *>(xs);

    // Token block loads first: segment t (1 KB) of row t / SEG lands at its LDS row.
    {
        const int SEG = QX ? SB / 1024 : QS / 1024;           // 1 KB segments per row
        const int rowbytes = QX ? 2 * K : K;
        const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
            QX ? (void *)(kp.x + mb * K) : (void *)(a.xq + mb * K), (short)0,
            rows_x * rowbytes, kRsrcWord3);
        for (int t = wave; t < rows_x * SEG; t += NW) {
            const int row = t / SEG, seg = t - row * SEG;
            const int col = seg * 1024 + lane * 16;
            const int off = col < rowbytes ? row * rowbytes + col : kOOB;
            int8_t *dst = (QX ? stage + row * SB : xs + row * QS) + seg * 1024;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rx, (__attribute__((address_space(3))) void *)dst, 16, off, 0, 0, 0);
        }
    }
    __builtin_amdgcn_sched_barrier(0);

    // The weight ring: super-step ss of this wavefront into slot `slot`.
    constexpr uint32_t kFar = 1u << 30;
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.wq + n0 * K), (short)0, rows_w * K, kRsrcWord3);
    uint32_t wrow[FNB];
#pragma unroll
    for (int c = 0; c < FNB; ++c)
        wrow[c] = (c * 16 + r < rows_w) ? (uint32_t)((c * 16 + r) * K) : kFar;
    const int nss = (K + 127) / 128;
    const int mine = wave < nss ? (nss - wave + NW - 1) / NW : 0;
    i32x4 wv[D][FNB][2];
    auto load = [&](auto slotc, int ss) {
        constexpr int slot = decltype(slotc)::value;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int k = ss * 128 + s * 64 + g * 16;
            const uint32_t kk = (uint32_t)k + ((uint32_t)((K - 1 - k) >> 31) & kFar);
#pragma unroll
            for (int c = 0; c < FNB; ++c)
                wv[slot][c][s] = __builtin_bit_cast(
                    i32x4, __builtin_amdgcn_raw_buffer_load_b128(rw, (int)(wrow[c] + kk), 0, 0));
        }
    };
    [&]<int... d>(std::integer_sequence<int, d...>) {
        ((load(std::integral_constant<int, d>{}, wave + d * NW),
          __builtin_amdgcn_sched_barrier(0)), ...);
    }(std::make_integer_sequence<int, D>{});

    // The token loads are older than the D * FNB * 2 weight loads of this wavefront.
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(D * FNB * 2));
    barrier_nofence();

    if constexpr (QX) {
        // Row i is quantized by WPR wavefronts (all NW share the rows evenly), each
        // taking every WPR-th 16-byte vector of the row: absmax, cross-wavefront max,
        // then the codes.
        const int nvec = K >> 3;
        int wpr = 1;                                 // a power of two, wpr * rows_x <= NW
        while (2 * wpr * rows_x <= NW)
            wpr *= 2;
        const int part = wave % wpr, groups = NW / wpr;
        const int rows_lim = (rows_x + groups - 1) / groups * groups;   // same trip count
        for (int i0 = wave / wpr; i0 < rows_lim; i0 += groups) {
            const bool live = i0 < rows_x;                     // wave-uniform
            const uint4 *src = reinterpret_cast<const uint4 *>(stage + (live ? i0 : 0) * SB);
            uint32_t mx = 0;
            if (live)
                for (int v = part * 64 + lane; v < nvec; v += wpr * 64)
                    mx = max(mx, qmath::absmax8(src[v]));
            mx = qmath::wave_max(mx);
            if (lane == 0)
                pmax[wave] = mx;
            __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
            barrier_nofence();
            if (live) {
                uint32_t am = 0;
                for (int w = 0; w < wpr; ++w)
                    am = max(am, pmax[(wave / wpr) * wpr + w]);
                const qmath::RowScale rs = qmath::row_scale(am);
                for (int v = part * 64 + lane; v < nvec; v += wpr * 64)
                    *reinterpret_cast<uint2 *>(xs + i0 * QS + v * 8) = qmath::code8(src[v], rs.inv);
                if (part == 0 && lane == 0)
                    qscale[i0] = rs.scale;
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);
            barrier_nofence();
        }
    }

    i32x4 acc[FNB][FMB];
#pragma unroll
    for (int c = 0; c < FNB; ++c)
#pragma unroll
        for (int b = 0; b < FMB; ++b)
            acc[c][b] = i32x4{0, 0, 0, 0};
    // Token fragment rows past the block read row 0 and are zeroed.
    int xrow[FMB];
    bool xlive[FMB];
#pragma unroll
    for (int b = 0; b < FMB; ++b) {
        xlive[b] = b * 16 + r < rows_x;
        xrow[b] = (xlive[b] ? b * 16 + r : 0) * QS;
    }
    for (int it = 0; it < mine; it += D) {
        [&]<int... d>(std::integer_sequence<int, d...>) {
            ([&] {
                const int ss = wave + (it + d) * NW;
                __builtin_amdgcn_sched_barrier(0);
                i32x4 xv[FMB][2];
#pragma unroll
                for (int s = 0; s < 2; ++s)
#pragma unroll
                    for (int b = 0; b < FMB; ++b) {
                        const i32x4 t = *reinterpret_cast<const i32x4 *>(
                            xs + xrow[b] + ss * 128 + s * 64 + g * 16);
                        xv[b][s] = xlive[b] ? t : i32x4{0, 0, 0, 0};
                    }
#pragma unroll
                for (int s = 0; s < 2; ++s)
#pragma unroll
                    for (int c = 0; c < FNB; ++c)
#pragma unroll
                        for (int b = 0; b < FMB; ++b)
                            acc[c][b] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                                wv[d][c][s], xv[b][s], acc[c][b], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
                load(std::integral_constant<int, d>{}, ss + D * NW);
            }(), ...);
        }(std::make_integer_sequence<int, D>{});
    }
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    // The reduction array overwrites the token rows: every wavefront's reads of them
    // have to be done first.
    __syncthreads();

    // Cross-wavefront reduction: entry (wave, c * FMB + b) holds each lane's 4 sums.
    constexpr int NCB = FNB * FMB;
#pragma unroll
    for (int c = 0; c < FNB; ++c)
#pragma unroll
        for (int b = 0; b < FMB; ++b)
            red[(wave * NCB + c * FMB + b) * 64 + lane] = acc[c][b];
    __syncthreads();
    for (int cb = wave; cb < NCB; cb += NW) {
        const int c = cb / FMB, b = cb % FMB;
        i32x4 t = red[cb * 64 + lane];
#pragma unroll
        for (int w = 1; w < NW; ++w)
            t += red[(w * NCB + cb) * 64 + lane];
        const int64_t n = n0 + c * 16 + g * 4;
        if (b * 16 + r >= rows_x || n >= N)
            continue;
        const int64_t m = mb + b * 16 + r;
        if constexpr (EPI == EPI_I32) {
            int32_t *o = static_cast<int32_t *>(a.out) + m * N + n;
            if (kp.out_vec && n + 3 < N) {
                *reinterpret_cast<i32x4 *>(o) = t;
            } else {
                for (int e = 0; e < 4 && n + e < N; ++e)
                    o[e] = t[e];
            }
        } else {
            uint16_t *o = static_cast<uint16_t *>(a.out) + m * N + n;
            const float sxm = QX ? qscale[b * 16 + r] : a.sx[m];
            uint16_t hv[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if (n + e < N) {
                    const float bb = a.bias ? __uint_as_float((uint32_t)a.bias[n + e] << 16) : 0.0f;
                    const float y = __builtin_fmaf((float)t[e], sxm * a.sw[n + e], bb);
                    hv[e] = __builtin_bit_cast(uint16_t, (__bf16)y);
                }
            }
            if (kp.out_vec && n + 3 < N) {
                uint2 pk;
                pk.x = (uint32_t)hv[0] | ((uint32_t)hv[1] << 16);
                pk.y = (uint32_t)hv[2] | ((uint32_t)hv[3] << 16);
                *reinterpret_cast<uint2 *>(o) = pk;
            } else {
                for (int e = 0; e < 4 && n + e < N; ++e)
                    o[e] = hv[e];
            }
        }
    }
}

// ---------------------------------------------------------------- tile registry

// Split-K reduction and epilogue: acc = sum of the k_split int32 partials (exact in any
// order), then the same epilogue as the tiled kernels, y = bf16(fmaf(float(acc),
// sx[m] * sw[n], b[n])), or the int32 sum itself. Four channels per thread when the
// partial rows are 16-byte aligned, one otherwise.
template <int EPI>
__global__ void __launch_bounds__(256) splitk_reduce_kernel(KParams kp) {
    const GemmArgs &a = kp.a;
    const int64_t M = a.M, N = a.N, MN = M * N;
    const int S = kp.k_split;
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (kp.part_vec) {
        const int64_t nq = N / 4;
        if (t >= M * nq)
            return;
        const int64_t m = t / nq, n = (t - m * nq) * 4;
        const int32_t *p = kp.part + m * N + n;
        i32x4 acc = *reinterpret_cast<const i32x4 *>(p);
        for (int sp = 1; sp < S; ++sp)
            acc += *reinterpret_cast<const i32x4 *>(p + sp * MN);
        if constexpr (EPI == EPI_I32) {
            *reinterpret_cast<i32x4 *>(static_cast<int32_t *>(a.out) + m * N + n) = acc;
        } else {
            const float sxm = a.sx[m];
            uint16_t h[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float b = a.bias ? __uint_as_float((uint32_t)a.bias[n + e] << 16) : 0.0f;
                const float y = __builtin_fmaf((float)acc[e], sxm * a.sw[n + e], b);
                h[e] = __builtin_bit_cast(uint16_t, (__bf16)y);
            }
            uint16_t *o = static_cast<uint16_t *>(a.out) + m * N + n;
            if (kp.out_vec) {
                uint2 pk;
                pk.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
                pk.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
                *reinterpret_cast<uint2 *>(o) = pk;
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    o[e] = h[e];
            }
        }
    } else {
        if (t >= MN)
            return;
        const int64_t m = t / N, n = t - m * N;
        int32_t acc = kp.part[t];
        for (int sp = 1; sp < S; ++sp)
            acc += kp.part[t + sp * MN];
        if constexpr (EPI == EPI_I32) {
            static_cast<int32_t *>(a.out)[t] = acc;
        } else {
            const float b = a.bias ? __uint_as_float((uint32_t)a.bias[n] << 16) : 0.0f;
            const float y = __builtin_fmaf((float)acc, a.sx[m] * a.sw[n], b);
            static_cast<uint16_t *>(a.out)[t] = __builtin_bit_cast(uint16_t, (__bf16)y);
        }
    }
}

template <int TM, int TN, int BK, int WM, int WN, int S>
struct Tile {
    // S >= 2: pipelined direct-to-LDS kernel with S stages; S == 0: the simple
    // register-staged kernel only.
    static constexpr bool PIPE = S >= 2;
    static constexpr int threads = WM * WN * 64;
    static constexpr int lds = (PIPE ? S : 2) * (TM + TN) * BK;

    // Aligned operands only (16-byte pointers, K % 16 == 0); launch_gemm sends the rest
    // to the generic tile.
    static hipError_t launch(Epilogue epi, const KParams &kp, hipStream_t s) {
        const dim3 grid((unsigned)(kp.tiles_m * kp.tiles_n * kp.k_split)), block(threads);
        if constexpr (PIPE) {
            if (epi == EPI_BF16)
                hipLaunchKernelGGL((gemm_i8_lds_kernel<TM, TN, BK, WM, WN, S, EPI_BF16>), grid, block, 0, s, kp);
            else
                hipLaunchKernelGGL((gemm_i8_lds_kernel<TM, TN, BK, WM, WN, S, EPI_I32>), grid, block, 0, s, kp);
        } else {
            if (epi == EPI_BF16)
                hipLaunchKernelGGL((gemm_i8_kernel<TM, TN, BK, WM, WN, true, EPI_BF16>), grid, block, 0, s, kp);
            else
                hipLaunchKernelGGL((gemm_i8_kernel<TM, TN, BK, WM, WN, true, EPI_I32>), grid, block, 0, s, kp);
        }
        return hipGetLastError();
    }
};

// Few tokens: the weight-streaming kernel (one workgroup per 16 channels).
template <int FMB, int FNB, int NW>
struct SkinnyTile {
    static constexpr int threads = NW * 64;
    static constexpr int lds = NW * FNB * FMB * 64 * 16;
    static hipError_t launch(Epilogue epi, const KParams &kp, hipStream_t s) {
        const dim3 grid((unsigned)(kp.tiles_m * kp.tiles_n)), block(threads);
        if (kp.x) {
            // The small fused linear: LDS for the token block's codes and scales.
            const int rows = (int)(kp.a.M < 16 * FMB ? kp.a.M : 16 * FMB);
            const size_t dyn = (size_t)rows * (kp.a.K + 16) + (size_t)rows * 4;
            hipLaunchKernelGGL((gemm_i8_skinny_kernel<FMB, FNB, NW, EPI_BF16, true>), grid, block,
                               dyn, s, kp);
        } else if (epi == EPI_BF16) {
            hipLaunchKernelGGL((gemm_i8_skinny_kernel<FMB, FNB, NW, EPI_BF16>), grid, block, 0, s, kp);
        } else {
            hipLaunchKernelGGL((gemm_i8_skinny_kernel<FMB, FNB, NW, EPI_I32>), grid, block, 0, s, kp);
        }
        return hipGetLastError();
    }
};

// Few tokens with the token block in LDS (the weight streamed through a register ring).
// A token block too large for LDS runs the register-staged streaming kernel of the same
// tile instead; the one-launch linear (kp.x set) is only chosen where it fits.
template <int FMB, int FNB, int NW, int D>
struct WsxTile {
    static constexpr int threads = NW * 64;
    template <int EPI, bool QX>
    static hipError_t go(const KParams &kp, size_t dyn, hipStream_t s) {
        // Dynamic LDS beyond the default limit: a property of the kernel on each device,
        // set on a device's first launch (one bit per device; setting it twice from
        // racing threads is harmless).
        static std::atomic<uint64_t> attr_set{0};
        int dev = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess)
            return e;
        const uint64_t bit = dev < 64 ? (uint64_t)1 << dev : 0;
        if (bit == 0 || (attr_set.load(std::memory_order_relaxed) & bit) == 0) {
            e = hipFuncSetAttribute(
                reinterpret_cast<const void *>(&gemm_i8_wsx_kernel<FMB, FNB, NW, D, EPI, QX>),
                hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            if (e != hipSuccess)
                return e;
            attr_set.fetch_or(bit, std::memory_order_relaxed);
        }
        hipLaunchKernelGGL((gemm_i8_wsx_kernel<FMB, FNB, NW, D, EPI, QX>),
                           dim3((unsigned)(kp.tiles_m * kp.tiles_n)), dim3(threads), dyn, s, kp);
        return hipGetLastError();
    }
    static hipError_t launch(Epilogue epi, const KParams &kp, hipStream_t s) {
        const int64_t rows = kp.a.M < 16 * FMB ? kp.a.M : 16 * FMB;
        const bool qx = kp.x != nullptr;
        const int64_t dyn = wsx_lds_bytes(rows, kp.a.K, qx, FMB, FNB, NW);
        if (dyn > 160 * 1024) {
            if (qx)
                return hipErrorInvalidValue;
            return SkinnyTile<FMB, FNB, 16>::launch(epi, kp, s);
        }
        if (qx)
            return go<EPI_BF16, true>(kp, (size_t)dyn, s);
        return epi == EPI_BF16 ? go<EPI_BF16, false>(kp, (size_t)dyn, s)
                               : go<EPI_I32, false>(kp, (size_t)dyn, s);
    }
};

// Unaligned operands or K % 16 != 0: the register-staged kernel with byte loads.
struct GenericTile {
    static constexpr int tm = 128, tn = 128;
    static hipError_t launch(Epilogue epi, const KParams &kp, hipStream_t s) {
        const dim3 grid((unsigned)(kp.tiles_m * kp.tiles_n)), block(256);
        if (epi == EPI_BF16)
            hipLaunchKernelGGL((gemm_i8_kernel<128, 128, 128, 2, 2, false, EPI_BF16>), grid, block, 0, s, kp);
        else
            hipLaunchKernelGGL((gemm_i8_kernel<128, 128, 128, 2, 2, false, EPI_I32>), grid, block, 0, s, kp);
        return hipGetLastError();
    }
};

struct TileEntry {
    TileInfo info;
    int gm;
    hipError_t (*launch)(Epilogue, const KParams &, hipStream_t);
};

#define W8A8_TILE(NAME, TM, TN, BK, WM, WN, GM, S)                                          \
    TileEntry {                                                                              \
        {NAME, TM, TN, BK, Tile<TM, TN, BK, WM, WN, S>::threads,                            \
         Tile<TM, TN, BK, WM, WN, S>::lds, 1, -1, 0},                                        \
            GM, &Tile<TM, TN, BK, WM, WN, S>::launch                                         \
    }

// The same pipelined tile with K divided among KSPLIT workgroups (BASE: its unsplit id).
#define W8A8_TILE_SPLIT(NAME, TM, TN, BK, WM, WN, GM, S, KSPLIT, BASE)                    \
    TileEntry {                                                                              \
        {NAME, TM, TN, BK, Tile<TM, TN, BK, WM, WN, S>::threads,                            \
         Tile<TM, TN, BK, WM, WN, S>::lds, KSPLIT, BASE, 0},                                 \
            GM, &Tile<TM, TN, BK, WM, WN, S>::launch                                         \
    }

#define W8A8_SKINNY(NAME, FMB, FNB, NW)                                                  \
    TileEntry {                                                                              \
        {NAME, 16 * FMB, 16 * FNB, 256, SkinnyTile<FMB, FNB, NW>::threads,                  \
         SkinnyTile<FMB, FNB, NW>::lds, 1, -1, 1},                                           \
            1, &SkinnyTile<FMB, FNB, NW>::launch                                             \
    }

#define W8A8_WSX(NAME, FMB, FNB, NW, D)                                                     \
    TileEntry {                                                                              \
        {NAME, 16 * FMB, 16 * FNB, 128, WsxTile<FMB, FNB, NW, D>::threads, 0, 1, -1, 2},     \
            1, &WsxTile<FMB, FNB, NW, D>::launch                                             \
    }

// Names: m<TM>n<TN>k<BK>w<WM>x<WN>[s<S>]; skinny_m<Mmax>n<C>w<NW> = weight-streaming
// kernel for at most Mmax tokens, C channels per workgroup. "s<S>" = direct-to-LDS pipelined kernel with S
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
    W8A8_TILE("m160n256k128w1x4s3", 160, 256, 128, 1, 4, 8, 3),
    W8A8_TILE("m160n256k64w1x4s4", 160, 256, 64, 1, 4, 8, 4),
    W8A8_TILE("m288n256k128w3x4s2", 288, 256, 128, 3, 4, 8, 2),
    W8A8_TILE("m288n256k64w3x4s3", 288, 256, 64, 3, 4, 8, 3),
    W8A8_TILE("m128n128k128w2x2", 128, 128, 128, 2, 2, 8, 0),
    W8A8_TILE("m64n128k128w1x4", 64, 128, 128, 1, 4, 8, 0),
    W8A8_TILE("m32n128k128w1x4", 32, 128, 128, 1, 4, 8, 0),
    W8A8_TILE("m32n64k128w1x2", 32, 64, 128, 1, 2, 8, 0),
    W8A8_SKINNY("skinny_m16n16w16", 1, 1, 16),
    W8A8_SKINNY("skinny_m32n16w16", 2, 1, 16),
    W8A8_SKINNY("skinny_m16n64w16", 1, 4, 16),
    W8A8_SKINNY("skinny_m64n32w16", 4, 2, 16),
    W8A8_SKINNY("skinny_m128n32w8", 8, 2, 8),
    // Few tokens (a few hundred): small tiles with deep rings keep enough bytes in flight
    // per CU for the panel loads, which their little MFMA work per panel cannot hide.
    W8A8_TILE("m128n128k128w2x2s4", 128, 128, 128, 2, 2, 8, 4),
    W8A8_TILE("m64n128k128w1x4s6", 64, 128, 128, 1, 4, 8, 6),
    W8A8_TILE("m32n128k128w1x4s6", 32, 128, 128, 1, 4, 8, 6),
    W8A8_TILE("m64n64k128w2x2s8", 64, 64, 128, 2, 2, 8, 8),
    W8A8_TILE("m64n64k128w1x2s8", 64, 64, 128, 1, 2, 8, 8),
    // Split-K: few output tiles and a long K; the int32 partials are summed by a second
    // kernel that also runs the epilogue.
    W8A8_TILE_SPLIT("m128n128k128w2x2s4_k2", 128, 128, 128, 2, 2, 8, 4, 2, 20),
    W8A8_TILE_SPLIT("m128n128k128w2x2s4_k4", 128, 128, 128, 2, 2, 8, 4, 4, 20),
    W8A8_TILE_SPLIT("m64n128k128w1x4s6_k2", 64, 128, 128, 1, 4, 8, 6, 2, 21),
    W8A8_TILE_SPLIT("m64n128k128w1x4s6_k4", 64, 128, 128, 1, 4, 8, 6, 4, 21),
    W8A8_TILE_SPLIT("m32n128k128w1x4s6_k4", 32, 128, 128, 1, 4, 8, 6, 4, 22),
    W8A8_TILE_SPLIT("m128n256k128w2x2s3_k2", 128, 256, 128, 2, 2, 8, 3, 2, 3),
    W8A8_TILE_SPLIT("m256n128k128w2x2s3_k2", 256, 128, 128, 2, 2, 8, 3, 2, 2),
    W8A8_TILE_SPLIT("m160n256k128w1x4s3_k2", 160, 256, 128, 1, 4, 8, 3, 2, 7),
    // 96-channel tiles (wavefront tiles of 32 or 64 tokens x 96 channels): 192
    // workgroups, three quarters of a round, where 128-wide tiles give 144 (N = 4608 at
    // 512 or 1024 tokens; 7-8% faster there).
    W8A8_TILE("m128n96k128w4x1s4", 128, 96, 128, 4, 1, 8, 4),
    W8A8_TILE("m256n96k128w4x1s3", 256, 96, 128, 4, 1, 8, 3),
    // 96 x 256: exactly 256 workgroups at 333 (..384) tokens and N = 16384 (7% faster
    // there than 128 x 256 on 192).
    W8A8_TILE("m96n256k128w1x4s3", 96, 256, 128, 1, 4, 8, 3),
    // Few tokens, token block in LDS, weight through a register ring:
    // wsx_m<Mmax>n<C>w<NW>d<D>.
    W8A8_WSX("wsx_m16n16w8d4", 1, 1, 8, 4),
    W8A8_WSX("wsx_m16n32w8d4", 1, 2, 8, 4),
    W8A8_WSX("wsx_m16n64w8d4", 1, 4, 8, 4),
    W8A8_WSX("wsx_m32n32w8d2", 2, 2, 8, 2),
};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);

// Offline-chosen tile per shape. Entries are (M lower bound, M upper bound, N, K, tile);
// generated by the tile sweep and copied here.
struct TableEntry {
    int64_t m_lo, m_hi, n, k;
    int tile;
};
struct TileCost {
    double c;   // ms per round, fixed part
    double d;   // ms per round per 1e9 (K * TM * TN)
};
#include "tile_table.inc"

static_assert(sizeof(kTileCost) / sizeof(kTileCost[0]) == kNumTiles, "one cost per tile");

// Shapes without a table entry. Above 128 tokens a wave-quantization cost model picks
// the tile: a launch of T workgroups on 256 CUs takes ceil(T / 256) rounds, and a round
// of tile t costs c_t + d_t * K * TM * TN / 1e9 (kTileCost, fitted offline to the
// sweep). With few tokens, rules from a sweep of the weight-streaming and deep-ring
// tiles pick it.
int fallback_tile(int64_t M, int64_t N, int64_t K) {
    const int64_t cus = 256;
    if (M > 128) {
        int best = -1;
        double best_cost = 0.0;
        for (int id = 0; id < kNumTiles; ++id) {
            if (!(kTileCost[id].d > 0.0))
                continue;
            const TileInfo &t = kTiles[id].info;
            const int64_t tiles = ((M + t.tm - 1) / t.tm) * ((N + t.tn - 1) / t.tn);
            const int64_t rounds = (tiles + cus - 1) / cus;
            const double cost =
                (double)rounds * (kTileCost[id].c + kTileCost[id].d * (double)K * t.tm * t.tn * 1e-9);
            if (best < 0 || cost < best_cost) {
                best = id;
                best_cost = cost;
            }
        }
        if (best >= 0)
            return best;
    }
    // Few tokens (a sweep of the streaming and deep-ring tiles over M = 2..128,
    // N = 1024..16384, K = 1024..16384). Up to 16 tokens: the token block in LDS, except
    // for 2-16 tokens on a wide weight, where the deep-ring 64 x 64 tile streams it faster.
    if (M <= 16)
        return (M > 1 && N >= 16384) ? 23 : 36;
    // Few channels: the token block in LDS on 16 (32) channels per workgroup.
    if (N <= 2048)
        return M <= 64 ? 36 : 37;
    // A long K on a few thousand channels: the deep-ring tiles with K split in four.
    if (K >= 8192 && N < 8192)
        return M <= 64 ? 29 : 28;
    // Many channels: the deep-ring tiles fill the CUs.
    if (N >= 8192)
        return M <= 64 ? 22 : 21;
    if (M <= 32)
        return 16;
    return M <= 64 ? 39 : 23;
}

}  // namespace

int tile_count() { return kNumTiles; }

const TileInfo *tile_info(int id) {
    return (id >= 0 && id < kNumTiles) ? &kTiles[id].info : nullptr;
}

int default_tile(int64_t M, int64_t N, int64_t K) { return fallback_tile(M, N, K); }

int select_tile(int64_t M, int64_t N, int64_t K) {
    for (const TableEntry &e : kTileTable) {
        if (e.n == N && e.k == K && M >= e.m_lo && M <= e.m_hi && e.tile >= 0 &&
            e.tile < kNumTiles)
            return e.tile;
    }
    return fallback_tile(M, N, K);
}

// Splits of a split tile for K: panels of BK bytes dealt out in equal runs; a short K
// gets fewer splits (one: no split at all).
static int split_count(const TileInfo &t, int64_t K, int *chunk) {
    const int64_t panels = (K + t.bk - 1) / t.bk;
    const int64_t per = (panels + t.ksplit - 1) / t.ksplit;
    if (chunk)
        *chunk = (int)(per * t.bk);
    return per > 0 ? (int)((panels + per - 1) / per) : 1;
}

size_t tile_workspace_bytes(int id, int64_t M, int64_t N, int64_t K) {
    if (id < 0 || id >= kNumTiles || kTiles[id].info.ksplit <= 1)
        return 0;
    const int splits = split_count(kTiles[id].info, K, nullptr);
    return splits > 1 ? (size_t)splits * (size_t)M * (size_t)N * sizeof(int32_t) : 0;
}

// LDS of one workgroup on gfx950.
constexpr int64_t kLdsPerWorkgroup = 160 * 1024;

// The small fused linear (see gemm_i8_skinny_kernel, QX): the chosen tile streams the
// weight, K % 16 == 0 with 16-byte aligned operands, a token block's codes and scales fit
// in 48 KB of LDS and, with the tile's static LDS (its cross-wavefront reduction array),
// in the workgroup's 160 KB, and the repeated reads of X (once per channel block) total
// at most 16 MB.
bool linear_small_applies(int64_t M, int64_t N, int64_t K, const void *x, const void *wq) {
    if (reinterpret_cast<uintptr_t>(x) % 16 != 0 || reinterpret_cast<uintptr_t>(wq) % 16 != 0)
        return false;
    return linear_small_shape(M, N, K);
}

bool linear_small_shape(int64_t M, int64_t N, int64_t K) {
    if (M <= 0 || N <= 0 || K <= 0 || K % 16 != 0)
        return false;
    const TileInfo &t = kTiles[select_tile(M, N, K)].info;
    if (!t.streaming)
        return false;
    const int64_t rows = M < t.tm ? M : t.tm;
    const int64_t channel_blocks = (N + t.tn - 1) / t.tn;
    if (t.streaming == 2) {
        // Token block in LDS: its bf16 rows, codes and the reduction array must fit; the
        // quantization overlaps the first weight loads, so its length is no concern.
        // Every workgroup reads the block's bf16 rows: at most as many bytes as its
        // weight rows (2 * rows <= channels), else the separate quantizer is cheaper
        // (measured: 16 tokens on 16 channels at K = 2048 run 1.6x slower fused).
        if (wsx_lds_bytes(rows, K, true, t.tm / 16, t.tn / 16, t.threads / 64) > kLdsPerWorkgroup)
            return false;
        if (2 * rows > t.tn)
            return false;
        return channel_blocks * M * K * 2 <= ((int64_t)16 << 20);
    }
    const int64_t dyn = rows * (K + 16) + rows * 4;
    if (dyn > 48 * 1024 || dyn + t.lds_bytes > kLdsPerWorkgroup)
        return false;
    // The quantization is a serial chain per wavefront (one row per wavefront, its
    // 16-byte vectors strided over the lanes, two passes): past 7 vectors per lane it
    // costs more than the separate quantizer launch it saves (measured: M = 1 at K =
    // 3136 fused is faster, at K = 4096 slower).
    const int64_t nw = t.threads / 64;
    if ((K / 8 + 63) / 64 * ((rows + nw - 1) / nw) > 7)
        return false;
    return channel_blocks * M * K * 2 <= ((int64_t)16 << 20);
}

hipError_t launch_linear_small(const uint16_t *x, const int8_t *wq, const float *sw,
                               const uint16_t *bias, uint16_t *y, int64_t M, int64_t N,
                               int64_t K, hipStream_t stream) {
    const TileEntry &t = kTiles[select_tile(M, N, K)];
    KParams kp;
    kp.a.xq = nullptr;
    kp.a.wq = wq;
    kp.a.sx = nullptr;
    kp.a.sw = sw;
    kp.a.bias = bias;
    kp.a.out = y;
    kp.a.M = M;
    kp.a.N = N;
    kp.a.K = K;
    kp.tiles_m = (int)((M + t.info.tm - 1) / t.info.tm);
    kp.tiles_n = (int)((N + t.info.tn - 1) / t.info.tn);
    kp.gm = t.gm;
    const bool ov = (N % 4 == 0) && (reinterpret_cast<uintptr_t>(y) % 8 == 0) &&
                    (reinterpret_cast<uintptr_t>(sw) % 16 == 0) &&
                    (bias == nullptr || reinterpret_cast<uintptr_t>(bias) % 8 == 0);
    kp.out_vec = ov ? 1 : 0;
    kp.k_split = 1;
    kp.k_chunk = (int)K;
    kp.part = nullptr;
    kp.part_vec = 0;
    kp.x = x;
    return t.launch(EPI_BF16, kp, stream);
}

hipError_t launch_gemm(int id, Epilogue epi, bool vec, const GemmArgs &a, void *ws,
                       size_t ws_bytes, hipStream_t stream) {
    const TileEntry &t = kTiles[id];
    const int tm = vec ? t.info.tm : GenericTile::tm;
    const int tn = vec ? t.info.tn : GenericTile::tn;
    KParams kp;
    kp.a = a;
    kp.tiles_m = (int)((a.M + tm - 1) / tm);
    kp.tiles_n = (int)((a.N + tn - 1) / tn);
    kp.gm = t.gm;
    const uintptr_t align_need = (epi == EPI_BF16) ? 8 : 16;
    bool ov = (a.N % 4 == 0) && (reinterpret_cast<uintptr_t>(a.out) % align_need == 0);
    if (epi == EPI_BF16) {
        ov = ov && (reinterpret_cast<uintptr_t>(a.sw) % 16 == 0) &&
             (a.bias == nullptr || reinterpret_cast<uintptr_t>(a.bias) % 8 == 0);
    }
    kp.out_vec = ov ? 1 : 0;
    if (ov && epi == EPI_BF16 && a.N % 8 == 0 && reinterpret_cast<uintptr_t>(a.out) % 16 == 0)
        kp.out_vec = 2;
    kp.k_split = 1;
    kp.k_chunk = (int)a.K;
    kp.part = nullptr;
    kp.part_vec = 0;
    kp.x = nullptr;
    if (!vec)
        return GenericTile::launch(epi, kp, stream);
    if (t.info.ksplit > 1) {
        int chunk = 0;
        const int splits = split_count(t.info, a.K, &chunk);
        if (splits > 1) {
            if (ws == nullptr || ws_bytes < tile_workspace_bytes(id, a.M, a.N, a.K))
                return hipErrorInvalidValue;
            kp.k_split = splits;
            kp.k_chunk = chunk;
            kp.part = static_cast<int32_t *>(ws);
            kp.part_vec = (a.N % 4 == 0 && reinterpret_cast<uintptr_t>(ws) % 16 == 0) ? 1 : 0;
            // The tile kernel stores partials only, so its epilogue flavour is irrelevant.
            const hipError_t e = t.launch(EPI_I32, kp, stream);
            if (e != hipSuccess)
                return e;
            const int64_t items = kp.part_vec ? a.M * (a.N / 4) : a.M * a.N;
            const unsigned blocks = (unsigned)((items + 255) / 256);
            if (epi == EPI_BF16)
                hipLaunchKernelGGL(splitk_reduce_kernel<EPI_BF16>, dim3(blocks), dim3(256), 0,
                                   stream, kp);
            else
                hipLaunchKernelGGL(splitk_reduce_kernel<EPI_I32>, dim3(blocks), dim3(256), 0,
                                   stream, kp);
            return hipGetLastError();
        }
    }
    return t.launch(epi, kp, stream);
}

}  // namespace w8a8
