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

// Scaled ungroup: dst[r] = round(src[idx[r]] * scale[idx[r]]), the product
// in fp32 and rounded once to the element type (zero row if idx[r] < 0).
// One thread per 16-byte piece of an output row.
template <bool F32>
__global__ __launch_bounds__(256) void k_scale_rows(int64_t nrows, int64_t pieces,
                                                    const uint4* __restrict__ src,
                                                    const int32_t* __restrict__ idx,
                                                    const float* __restrict__ scale,
                                                    int64_t src_rows, uint4* __restrict__ dst) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= nrows * pieces) return;
    const int64_t r = i / pieces, c = i - r * pieces;
    const int32_t s = idx[r];
    uint4 o = make_uint4(0, 0, 0, 0);
    if (s >= 0 && s < src_rows) {
        const uint4 v = src[(int64_t)s * pieces + c];
        const float f = scale[s];
        if constexpr (F32) {
            o.x = __float_as_uint(__uint_as_float(v.x) * f);
            o.y = __float_as_uint(__uint_as_float(v.y) * f);
            o.z = __float_as_uint(__uint_as_float(v.z) * f);
            o.w = __float_as_uint(__uint_as_float(v.w) * f);
        } else {
            auto two = [&](uint32_t w) {
                const uint32_t lo = f32_to_bf16(bf16_lo(w) * f);
                const uint32_t hi = f32_to_bf16(bf16_hi(w) * f);
                return lo | (hi << 16);
            };
            o.x = two(v.x);
            o.y = two(v.y);
            o.z = two(v.z);
            o.w = two(v.w);
        }
    }
    dst[r * pieces + c] = o;
}

hipError_t launch_scale_rows(bool f32, int64_t nrows, int64_t row_bytes, const void* src,
                             const int32_t* idx, const float* scale, int64_t src_rows, void* dst,
                             hipStream_t s) {
    const int64_t pieces = row_bytes / 16;
    const int64_t blocks = ceil_div(nrows * pieces, 256);
    if (blocks == 0) return hipSuccess;
    if (f32)
        k_scale_rows<true><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(
            nrows, pieces, reinterpret_cast<const uint4*>(src), idx, scale, src_rows,
            reinterpret_cast<uint4*>(dst));
    else
        k_scale_rows<false><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(
            nrows, pieces, reinterpret_cast<const uint4*>(src), idx, scale, src_rows,
            reinterpret_cast<uint4*>(dst));
    return hipGetLastError();
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
