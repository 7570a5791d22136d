// Pre-norm of the stacked layers: xn[j] = bf16(x[j] * r_j) with
// r_j = 1 / sqrt(mean_k x[j][k]^2 + eps), fp32 arithmetic, for the routed
// grouped rows j < offsets[E].  One workgroup per row; the sum of squares is
// a per-lane fp32 sum (lane elements in ascending order), then a wave and a
// workgroup fold.
#include "common.hpp"
#include "internal.hpp"

namespace readme {

// NV > 0: the row is held in registers (at most NV float4 per thread) and
// read once; NV = 0: read twice (sum of squares, then scale).  Both sum each
// lane's elements in the same order, so the results are identical.
template <int NV>
__global__ __launch_bounds__(256) void k_rms_to_bf16(int64_t d, const float* __restrict__ x,
                                                     const int32_t* __restrict__ offsets, int E,
                                                     float eps, uint16_t* __restrict__ xn) {
    __shared__ float part[4];
    const int64_t j = blockIdx.x;
    const float4* row = reinterpret_cast<const float4*>(x + j * d);
    const int n4 = (int)(d / 4);
    const int tid = threadIdx.x;
    float4 v[NV > 0 ? NV : 1];
    float ss = 0.0f;
    if constexpr (NV > 0) {
        // The row (in bounds: the grid has one workgroup per row of x) is
        // requested before the routed-row count, so the two round trips
        // overlap.
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int c = tid + 256 * i;
            v[i] = c < n4 ? row[c] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        }
        if (j >= offsets[E]) return;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            if (tid + 256 * i < n4) {
                ss += v[i].x * v[i].x;
                ss += v[i].y * v[i].y;
                ss += v[i].z * v[i].z;
                ss += v[i].w * v[i].w;
            }
        }
    } else {
        if (j >= offsets[E]) return;
        for (int c = tid; c < n4; c += 256) {
            const float4 w = row[c];
            ss += w.x * w.x;
            ss += w.y * w.y;
            ss += w.z * w.z;
            ss += w.w * w.w;
        }
    }
    for (int off = 32; off >= 1; off >>= 1) ss += __shfl_down(ss, off, 64);
    if ((tid & 63) == 0) part[tid >> 6] = ss;
    __syncthreads();
    const float tot = (part[0] + part[1]) + (part[2] + part[3]);
    const float r = 1.0f / sqrtf(tot / (float)d + eps);
    uint2* out = reinterpret_cast<uint2*>(xn + j * d);
    auto put = [&](int c, const float4 w) {
        uint2 o;
        o.x = (uint32_t)f32_to_bf16(w.x * r) | ((uint32_t)f32_to_bf16(w.y * r) << 16);
        o.y = (uint32_t)f32_to_bf16(w.z * r) | ((uint32_t)f32_to_bf16(w.w * r) << 16);
        out[c] = o;
    };
    if constexpr (NV > 0) {
#pragma unroll
        for (int i = 0; i < NV; ++i)
            if (tid + 256 * i < n4) put(tid + 256 * i, v[i]);
    } else {
        for (int c = tid; c < n4; c += 256) put(c, row[c]);
    }
}

hipError_t launch_rms_to_bf16(int64_t T, int64_t d, const float* x, const int32_t* offsets, int E,
                              float eps, uint16_t* xn, hipStream_t s) {
    const dim3 grid((unsigned)T), block(256);
    const int64_t per = ceil_div(d / 4, 256);  // float4 per thread
    if (per <= 4)
        k_rms_to_bf16<4><<<grid, block, 0, s>>>(d, x, offsets, E, eps, xn);
    else if (per <= 8)
        k_rms_to_bf16<8><<<grid, block, 0, s>>>(d, x, offsets, E, eps, xn);
    else
        k_rms_to_bf16<0><<<grid, block, 0, s>>>(d, x, offsets, E, eps, xn);
    return hipGetLastError();
}

}  // namespace readme
