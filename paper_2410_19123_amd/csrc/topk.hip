// Top-K routing (Eq. 2 with K > 1): each token's K highest-logit experts
// and their gate weights, and the gate-weighted sum of the K expert outputs.
//
// Selection reads the router's fp32 logits (summed in the canonical order,
// route.hip) and only compares, so it is exact: slot k takes, among the
// experts not yet taken, the first in ascending index order unless a later
// one has a strictly larger logit.  Top-1 is the router's own argmax; ties
// go to the lower index and a later NaN never wins.  The weights are the
// softmax of the K selected logits, renormalised over the slots, so K = 1
// gives weight 1 (the unweighted top-1 layer).
#include "common.hpp"
#include "internal.hpp"

namespace readme {

// One thread per token; the taken set is a bit mask over at most
// README_MAX_EXPERTS experts.
__global__ __launch_bounds__(256) void k_topk(int64_t T, int E, int K,
                                              const float* __restrict__ logits,
                                              int32_t* __restrict__ ids,
                                              float* __restrict__ weights) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= T) return;
    const float* l = logits + t * E;
    uint64_t taken[README_MAX_EXPERTS / 64] = {};
    float top = 0.0f, sum = 0.0f;
    for (int k = 0; k < K; ++k) {
        int best_id = -1;
        float best = 0.0f;
        for (int e = 0; e < E; ++e) {
            if ((taken[e >> 6] >> (e & 63)) & 1u) continue;
            const float v = l[e];
            if (best_id < 0 || v > best) {
                best_id = e;
                best = v;
            }
        }
        taken[best_id >> 6] |= 1ull << (best_id & 63);
        ids[t * K + k] = best_id;
        if (k == 0) top = best;
        const float z = expf(best - top);  // <= 1 for finite logits
        weights[t * K + k] = z;
        sum += z;
    }
    const float inv = 1.0f / sum;
    for (int k = 0; k < K; ++k) weights[t * K + k] *= inv;
}

hipError_t launch_topk(int64_t T, int E, int K, const float* logits, int32_t* ids, float* weights,
                       hipStream_t s) {
    const unsigned blocks = (unsigned)ceil_div(T, 256);
    k_topk<<<dim3(blocks), dim3(256), 0, s>>>(T, E, K, logits, ids, weights);
    return hipGetLastError();
}

// Gate weight of a top-1 token, the softmax of its logits at its expert:
// p_t = exp(l[t,e_t] - m_t) / sum_e exp(l[t,e] - m_t), m_t = max_e l[t,e],
// fp32 with the experts in ascending order; written in grouped order,
// row_scale[inv_perm[t]], for routed tokens only.  One thread per token.
__global__ __launch_bounds__(256) void k_gate_weights(int64_t T, int E,
                                                      const float* __restrict__ logits,
                                                      const int32_t* __restrict__ ids,
                                                      const int32_t* __restrict__ inv_perm,
                                                      float* __restrict__ row_scale) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= T) return;
    const int e_t = ids[t];
    const int32_t j = inv_perm[t];
    if (e_t < 0 || e_t >= E || j < 0) return;
    const float* l = logits + t * E;
    float m = l[0];
    for (int e = 1; e < E; ++e) m = fmaxf(m, l[e]);
    float sum = 0.0f;
    for (int e = 0; e < E; ++e) sum += expf(l[e] - m);
    row_scale[j] = expf(l[e_t] - m) / sum;
}

hipError_t launch_gate_weights(int64_t T, int E, const float* logits, const int32_t* ids,
                               const int32_t* inv_perm, float* row_scale, hipStream_t s) {
    const unsigned blocks = (unsigned)ceil_div(T, 256);
    k_gate_weights<<<dim3(blocks), dim3(256), 0, s>>>(T, E, logits, ids, inv_perm, row_scale);
    return hipGetLastError();
}

// y[t] = sum over slots k = 0 .. K-1 of w[t,k] * y_pairs[t*K + k], in fp32
// in slot order, rounded once.  Each thread owns one 16-byte piece of a
// token's row; the K pair rows of a token are adjacent in memory.
template <bool F32>
__global__ __launch_bounds__(256) void k_combine(int64_t T, int64_t pieces, int K,
                                                 const uint4* __restrict__ y_pairs,
                                                 const float* __restrict__ w,
                                                 uint4* __restrict__ y) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= T * pieces) return;
    const int64_t t = i / pieces, c = i - t * pieces;
    constexpr int N = F32 ? 4 : 8;
    float acc[N];
#pragma unroll
    for (int q = 0; q < N; ++q) acc[q] = 0.0f;
    for (int k = 0; k < K; ++k) {
        const float wk = w[t * K + k];
        const uint4 v = y_pairs[(t * K + k) * pieces + c];
        const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if constexpr (F32) {
                acc[q] = __builtin_fmaf(wk, __uint_as_float(u[q]), acc[q]);
            } else {
                acc[2 * q] = __builtin_fmaf(wk, bf16_lo(u[q]), acc[2 * q]);
                acc[2 * q + 1] = __builtin_fmaf(wk, bf16_hi(u[q]), acc[2 * q + 1]);
            }
        }
    }
    uint4 o;
    if constexpr (F32) {
        o = make_uint4(__float_as_uint(acc[0]), __float_as_uint(acc[1]), __float_as_uint(acc[2]),
                       __float_as_uint(acc[3]));
    } else {
        uint32_t p[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
            p[q] = (uint32_t)f32_to_bf16(acc[2 * q]) | ((uint32_t)f32_to_bf16(acc[2 * q + 1]) << 16);
        o = make_uint4(p[0], p[1], p[2], p[3]);
    }
    y[t * pieces + c] = o;
}

hipError_t launch_combine(bool f32, int64_t T, int64_t d, int K, const void* y_pairs,
                          const float* weights, void* y, hipStream_t s) {
    const int64_t pieces = d * (f32 ? 4 : 2) / 16;
    const int64_t n = T * pieces;
    if (n == 0) return hipSuccess;
    const unsigned blocks = (unsigned)ceil_div(n, 256);
    const uint4* src = reinterpret_cast<const uint4*>(y_pairs);
    uint4* dst = reinterpret_cast<uint4*>(y);
    if (f32)
        k_combine<true><<<dim3(blocks), dim3(256), 0, s>>>(T, pieces, K, src, weights, dst);
    else
        k_combine<false><<<dim3(blocks), dim3(256), 0, s>>>(T, pieces, K, src, weights, dst);
    return hipGetLastError();
}

}  // namespace readme
