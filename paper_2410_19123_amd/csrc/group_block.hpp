// The grouping step (histogram, exclusive scan, stable counting-sort ranks)
// as one workgroup's routine (k_group runs it; any kernel that ends with the
// grouping of its ids can too).  NT threads; smem: SMEM_INTS ints of LDS.
//   1. histogram of ids in LDS (order-free, so LDS atomics are exact);
//   2. exclusive scan -> counts, offsets;
//   3. stable ranks, NT tokens per round: each wave finds, by ballots over
//      the id bits, the lanes that share its id (a match mask); rank within
//      the wave = popcount of the lower matching lanes; per-wave per-expert
//      counts are scanned across the waves in wave order, so the rank of
//      token t is #{t' < t with the same id}: a stable counting sort, with no
//      atomics in the ordering.
#pragma once

#include "common.hpp"

namespace readme {

template <int NT>
struct GroupBlock {
    static constexpr int NW = NT / 64;
    static constexpr int SMEM_INTS = (2 + 2 * NW) * README_MAX_EXPERTS;

    __device__ static void run(int T, int E, int nbits, const int32_t* ids, int32_t* counts,
                               int32_t* offsets, int32_t* perm, int32_t* inv_perm, int* smem) {
        int* hist = smem;
        int* cursor = smem + README_MAX_EXPERTS;
        int* wcnt = smem + 2 * README_MAX_EXPERTS;           // [NW][MAX_EXPERTS]
        int* wbase = wcnt + NW * README_MAX_EXPERTS;          // [NW][MAX_EXPERTS]
        const int tid = threadIdx.x;
        const int wave = tid >> 6;

        for (int i = tid; i < README_MAX_EXPERTS; i += NT) hist[i] = 0;
        for (int i = tid; i < NW * README_MAX_EXPERTS; i += NT) wcnt[i] = 0;
        __syncthreads();
        for (int t = tid; t < T; t += NT) {
            const int e = ids[t];
            if (e >= 0 && e < E) atomicAdd(&hist[e], 1);
        }
        __syncthreads();
        if (tid == 0) {
            int s = 0;
            offsets[0] = 0;
            for (int e = 0; e < E; ++e) {
                cursor[e] = s;
                counts[e] = hist[e];
                s += hist[e];
                offsets[e + 1] = s;
            }
            hist[0] = s;  // routed tokens
        }
        __syncthreads();
        const int routed = hist[0];

        for (int base = 0; base < T; base += NT) {
            const int t = base + tid;
            const int e = t < T ? ids[t] : -1;
            const bool valid = e >= 0 && e < E;
            uint64_t match = __ballot(valid);
            for (int b = 0; b < nbits; ++b) {
                const bool bit = valid && ((e >> b) & 1);
                const uint64_t ones = __ballot(bit);
                match &= bit ? ones : ~ones;
            }
            const int rank = __popcll(match & lanemask_lt());
            if (valid && rank == 0) wcnt[wave * README_MAX_EXPERTS + e] = __popcll(match);
            __syncthreads();
            for (int x = tid; x < E; x += NT) {
                int s = cursor[x];
                for (int w = 0; w < NW; ++w) {
                    wbase[w * README_MAX_EXPERTS + x] = s;
                    s += wcnt[w * README_MAX_EXPERTS + x];
                    wcnt[w * README_MAX_EXPERTS + x] = 0;
                }
                cursor[x] = s;
            }
            __syncthreads();
            if (t < T) {
                if (valid) {
                    const int j = wbase[wave * README_MAX_EXPERTS + e] + rank;
                    perm[j] = t;
                    inv_perm[t] = j;
                } else {
                    inv_perm[t] = -1;
                }
            }
            __syncthreads();
        }
        for (int j = routed + tid; j < T; j += NT) perm[j] = -1;
    }
};

}  // namespace readme
