// Shared device helpers of libreadme (gfx950 / CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "readme.h"

namespace readme {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// bf16 bit pattern -> fp32 (exact).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bit pattern, round to nearest even, NaN kept a (quiet) NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float silu_f32(float z) { return z / (1.0f + __expf(-z)); }

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int u = __shfl_up(v, off, 64);
        if (lane >= off) v += u;
    }
    return v;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
    const int lane = threadIdx.x & 63;
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

inline int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

inline size_t dtype_size(readme_dtype dt) { return dt == README_F32 ? 4 : 2; }

// Packed expert layout (see readme_pack_experts):
//   gate/up block: [E][2 * Ip][d], rows in 32-row groups alternating
//                  gate (even group) and up (odd group) for the same 32
//                  intermediate neurons; neurons i >= I are zero rows.
//   down block:    [E][d][Ip], columns i >= I zero.
constexpr int64_t kPadI = 64;
inline int64_t padded_I(int64_t I) { return round_up(I, kPadI); }
inline size_t packed_gate_up_bytes(readme_dtype dt, int64_t E, int64_t d, int64_t I) {
    return (size_t)E * 2 * padded_I(I) * d * dtype_size(dt);
}
inline size_t packed_bytes(readme_dtype dt, int64_t E, int64_t d, int64_t I) {
    return packed_gate_up_bytes(dt, E, d, I) + (size_t)E * d * padded_I(I) * dtype_size(dt);
}

}  // namespace readme
