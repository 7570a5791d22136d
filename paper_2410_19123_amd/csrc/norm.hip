// Pre-norm of the stacked layers: xn[j] = bf16(x[j] * r_j) with
// r_j = 1 / sqrt(mean_k x[j][k]^2 + eps), fp32 arithmetic, for the routed
// grouped rows j < offsets[E].  One workgroup per row; the sum of squares is
// a per-lane fp32 sum, then a wave and a workgroup fold.
#include "common.hpp"
#include "internal.hpp"

namespace readme {

__global__ __launch_bounds__(256) void k_rms_to_bf16(int64_t d, const float* __restrict__ x,
                                                     const int32_t* __restrict__ offsets, int E,
                                                     float eps, uint16_t* __restrict__ xn) {
    __shared__ float part[4];
    const int64_t j = blockIdx.x;
    if (j >= offsets[E]) return;
    const float4* row = reinterpret_cast<const float4*>(x + j * d);
    const int64_t n4 = d / 4;
    float ss = 0.0f;
    for (int64_t c = threadIdx.x; c < n4; c += 256) {
        const float4 v = row[c];
        ss += v.x * v.x;
        ss += v.y * v.y;
        ss += v.z * v.z;
        ss += v.w * v.w;
    }
    for (int off = 32; off >= 1; off >>= 1) ss += __shfl_down(ss, off, 64);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
    __syncthreads();
    const float tot = (part[0] + part[1]) + (part[2] + part[3]);
    const float r = 1.0f / sqrtf(tot / (float)d + eps);
    uint2* out = reinterpret_cast<uint2*>(xn + j * d);
    for (int64_t c = threadIdx.x; c < n4; c += 256) {
        const float4 v = row[c];
        uint2 o;
        o.x = (uint32_t)f32_to_bf16(v.x * r) | ((uint32_t)f32_to_bf16(v.y * r) << 16);
        o.y = (uint32_t)f32_to_bf16(v.z * r) | ((uint32_t)f32_to_bf16(v.w * r) << 16);
        out[c] = o;
    }
}

hipError_t launch_rms_to_bf16(int64_t T, int64_t d, const float* x, const int32_t* offsets, int E,
                              float eps, uint16_t* xn, hipStream_t s) {
    k_rms_to_bf16<<<dim3((unsigned)T), dim3(256), 0, s>>>(d, x, offsets, E, eps, xn);
    return hipGetLastError();
}

}  // namespace readme
