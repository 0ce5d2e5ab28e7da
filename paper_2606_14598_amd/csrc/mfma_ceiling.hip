// Measurement aids, not part of the linear. The read ceiling (at the end of the file)
// is a plain streaming read of a buffer: the rate HBM actually delivers for that many
// bytes, the floor of a weight-streaming GEMM that reads them once.
//
// Matrix-core ceiling on given int8 operands: the int8 MFMA's sustained rate depends on the operand bits, because the chip
// lowers its clock under the matrix cores' switching power. This kernel replays the
// GEMM's per-K-step MFMA sequence of the 160x256 tile (each wavefront: 2 weight
// fragments x 5 token fragments of v_mfma_i32_32x32x32_i8 per K-step) on fragments of
// the caller's Xq and Wq held in registers, so the loop has no memory traffic, no LDS
// and no barriers: its rate is what the matrix cores sustain on these codes.
//
// Workgroup b (256 of them, 4 wavefronts) takes tile (b / 16, b % 16) of a 16 x 16 grid
// of 160 x 256 tiles (rows and channels wrapped modulo M and N), loads 8 K-steps of its
// fragments (K-step s of workgroup b at byte 32 * ((8b + s) mod K/32)), then runs
// `iters` sweeps over them. Each wavefront writes the sum of its accumulators (uint32,
// wrapping) so that the work cannot be elided and a test can check it:
//   sum = iters * sum_s sum_{k<32} (sum of its 64 weight rows at k_s + k)
//                                 * (sum of its 160 token rows at k_s + k)   (mod 2^32).
#include "w8a8_internal.hpp"

namespace w8a8 {
namespace {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x16 __attribute__((ext_vector_type(16)));

constexpr int kSteps = 8, kFN = 2, kFM = 5;

__global__ void __launch_bounds__(256)
mfma_ceiling_kernel(const int8_t *__restrict__ xq, const int8_t *__restrict__ wq, int64_t M,
                    int64_t N, int64_t K, int iters, uint32_t *__restrict__ wave_sums) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 31, h = lane >> 5;
    const int64_t tm = blockIdx.x / 16, tn = blockIdx.x % 16;
    const int64_t ksteps = K / 32;
    i32x4 A[kSteps][kFN], B[kSteps][kFM];
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
        const int64_t k = (((int64_t)blockIdx.x * kSteps + s) % ksteps) * 32 + h * 16;
#pragma unroll
        for (int i = 0; i < kFN; ++i) {
            const int64_t n = (tn * 256 + wave * 64 + i * 32 + r) % N;
            A[s][i] = *reinterpret_cast<const i32x4 *>(wq + n * K + k);
        }
#pragma unroll
        for (int j = 0; j < kFM; ++j) {
            const int64_t m = (tm * 160 + j * 32 + r) % M;
            B[s][j] = *reinterpret_cast<const i32x4 *>(xq + m * K + k);
        }
    }
    i32x16 acc[kFN][kFM];
#pragma unroll
    for (int i = 0; i < kFN; ++i)
#pragma unroll
        for (int j = 0; j < kFM; ++j)
            acc[i][j] = i32x16{};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int s = 0; s < kSteps; ++s)
#pragma unroll
            for (int i = 0; i < kFN; ++i)
#pragma unroll
                for (int j = 0; j < kFM; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(A[s][i], B[s][j],
                                                                       acc[i][j], 0, 0, 0);
    }
    uint32_t t = 0;
#pragma unroll
    for (int i = 0; i < kFN; ++i)
#pragma unroll
        for (int j = 0; j < kFM; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                t += (uint32_t)acc[i][j][e];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        t += (uint32_t)__shfl_xor((int)t, off, 64);
    if (lane == 0)
        wave_sums[blockIdx.x * 4 + wave] = t;
}

// A plain streaming read: workgroup b XORs the 32-bit words of chunk b (bytes / 2048
// contiguous bytes) into sums[b]; each thread keeps 8 16-byte loads in flight.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256)
read_ceiling_kernel(const u32x4 *__restrict__ p, int64_t per, uint32_t *__restrict__ sums) {
    const u32x4 *q = p + (int64_t)blockIdx.x * per;
    u32x4 a = {0, 0, 0, 0};
    for (int64_t i = threadIdx.x; i < per; i += 256 * 8) {
        u32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            v[u] = (i + u * 256 < per) ? __builtin_nontemporal_load(q + i + u * 256)
                                       : u32x4{0, 0, 0, 0};
#pragma unroll
        for (int u = 0; u < 8; ++u)
            a ^= v[u];
    }
    uint32_t t = a.x ^ a.y ^ a.z ^ a.w;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        t ^= (uint32_t)__shfl_xor((int)t, off, 64);
    __shared__ uint32_t part[4];
    if ((threadIdx.x & 63) == 0)
        part[threadIdx.x >> 6] = t;
    __syncthreads();
    if (threadIdx.x == 0)
        sums[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

}  // namespace

hipError_t launch_read_ceiling(const void *p, int64_t bytes, uint32_t *sums, hipStream_t s) {
    hipLaunchKernelGGL(read_ceiling_kernel, dim3(kReadBlocks), dim3(256), 0, s,
                       static_cast<const u32x4 *>(p), bytes / 16 / kReadBlocks, sums);
    return hipGetLastError();
}

int64_t mfma_ceiling_ops(int64_t iters) {
    return (int64_t)256 * 4 * iters * kSteps * kFN * kFM * (2 * 32 * 32 * 32);
}

hipError_t launch_mfma_ceiling(const int8_t *xq, const int8_t *wq, int64_t M, int64_t N,
                               int64_t K, int iters, uint32_t *wave_sums, hipStream_t s) {
    hipLaunchKernelGGL(mfma_ceiling_kernel, dim3(256), dim3(256), 0, s, xq, wq, M, N, K,
                       iters, wave_sums);
    return hipGetLastError();
}

}  // namespace w8a8
