// Grouping tokens by expert (the per-expert queues of the expert-aware
// batching, Sec. 4.2 Alg. 1) and the row moves around the expert FFN.
//
// k_group: one 1024-thread workgroup running GroupBlock (group_block.hpp):
//   histogram, exclusive scan, stable counting-sort ranks.
// k_move_rows: dst[r] = src[idx[r]] (zero row if idx[r] < 0), 16-byte
//   vector copies, one row per 64-lane wave slice; serves both the gather
//   into grouped order (idx = perm) and the ungroup (idx = inv_perm).
#include "common.hpp"
#include "group_block.hpp"
#include "internal.hpp"

namespace readme {

constexpr int kGroupThreads = 1024;

__global__ __launch_bounds__(kGroupThreads) void k_group(int T, int E, int nbits,
                                                         const int32_t* __restrict__ ids,
                                                         int32_t* __restrict__ counts,
                                                         int32_t* __restrict__ offsets,
                                                         int32_t* __restrict__ perm,
                                                         int32_t* __restrict__ inv_perm) {
    __shared__ int smem[GroupBlock<kGroupThreads>::SMEM_INTS];
    GroupBlock<kGroupThreads>::run(T, E, nbits, ids, counts, offsets, perm, inv_perm, smem);
}

hipError_t launch_group(int64_t T, int E, const int32_t* ids, int32_t* counts, int32_t* offsets,
                        int32_t* perm, int32_t* inv_perm, hipStream_t s) {
    int nbits = 0;
    while ((1 << nbits) < E) ++nbits;
    k_group<<<dim3(1), dim3(kGroupThreads), 0, s>>>((int)T, E, nbits, ids, counts, offsets, perm,
                                                    inv_perm);
    return hipGetLastError();
}

// Each 64-lane slice of a block moves whole rows; ROWS rows per block.
template <int ROWS>
__global__ __launch_bounds__(256) void k_move_rows(int64_t nrows, int64_t row_chunks,
                                                   const uint4* __restrict__ src,
                                                   const int32_t* __restrict__ idx,
                                                   int64_t src_rows, uint4* __restrict__ dst) {
    const int lane = threadIdx.x & 63;
    const int slice = threadIdx.x >> 6;
    for (int k = slice; k < ROWS; k += 4) {
        const int64_t r = (int64_t)blockIdx.x * ROWS + k;
        if (r >= nrows) return;
        const int32_t s = idx[r];
        uint4* out = dst + r * row_chunks;
        if (s < 0 || s >= src_rows) {
            for (int64_t c = lane; c < row_chunks; c += 64) out[c] = make_uint4(0, 0, 0, 0);
        } else {
            const uint4* in = src + (int64_t)s * row_chunks;
            int64_t c = lane;
            for (; c + 192 < row_chunks; c += 256) {
                const uint4 a = in[c], b = in[c + 64], d2 = in[c + 128], e2 = in[c + 192];
                out[c] = a;
                out[c + 64] = b;
                out[c + 128] = d2;
                out[c + 192] = e2;
            }
            for (; c < row_chunks; c += 64) out[c] = in[c];
        }
    }
}

hipError_t launch_move_rows(int64_t nrows, int64_t row_bytes, const void* src, const int32_t* idx,
                            int64_t src_rows, void* dst, hipStream_t s) {
    constexpr int ROWS = 8;
    const int64_t blocks = ceil_div(nrows, ROWS);
    k_move_rows<ROWS><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(
        nrows, row_bytes / 16, reinterpret_cast<const uint4*>(src), idx, src_rows,
        reinterpret_cast<uint4*>(dst));
    return hipGetLastError();
}

}  // namespace readme
