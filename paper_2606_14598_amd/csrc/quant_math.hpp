// Per-row absmax int8 quantization arithmetic on bf16 inputs, shared by the row
// quantizer and by the small fused linear (which quantizes its own token rows): both
// must give the same codes and scales bit for bit.
//   a = max_k |v[k]|, s = a / 127, q[k] = clamp(rne(v[k] * (127 / a)), -127, 127);
// a row with a == 0, or with 127/a overflowing float32, gets s = 0 and q = 0.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace w8a8 {
namespace qmath {

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

__device__ __forceinline__ RowScale row_scale_f(float a) {
    float inv = 127.0f / a;     // correctly rounded (no fast-math)
    float s = a / 127.0f;
    bool zero = !(a > 0.0f) || !__builtin_isfinite(inv);
    RowScale r;
    r.inv = zero ? 0.0f : inv;
    r.scale = zero ? 0.0f : s;
    return r;
}

__device__ __forceinline__ RowScale row_scale(uint32_t amax_bits) {
    return row_scale_f(bf16_to_f32(amax_bits));
}

}  // namespace qmath
}  // namespace w8a8
