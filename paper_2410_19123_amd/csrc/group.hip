// Grouping tokens by expert (the per-expert queues of the expert-aware
// batching, Sec. 4.2 Alg. 1) and the row moves around the expert FFN.
//
// k_group: one 1024-thread workgroup running GroupBlock (group_block.hpp):
//   histogram, exclusive scan, stable counting-sort ranks.
// For large T the same counting sort runs over many workgroups, one chunk of
//   1024 tokens each, in four launches (k_group_hist, k_group_scan,
//   k_group_rank, k_group_inverse; see launch_group).
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

// ---- the counting sort over many workgroups (chunk b = tokens b*1024 ..) ----
//
// Until k_group_inverse runs, the first B*E entries of inv_perm hold H, the
// per-chunk counts H[b][e] = #{t in chunk b : ids[t] == e}, which k_group_scan
// turns into each chunk's first grouped row per expert,
//   H[b][e] <- offsets[e] + sum over b' < b of H[b'][e],
// so that token t (chunk b, id e, rank r among the chunk's tokens of id e in
// token order) goes to grouped row H[b][e] + r: the stable counting sort.
// The four launches order the phases; no workgroup reads what another one
// writes within a launch.

__global__ __launch_bounds__(kGroupThreads) void k_group_hist(int T, int E,
                                                              const int32_t* __restrict__ ids,
                                                              int32_t* __restrict__ H) {
    __shared__ int hist[README_MAX_EXPERTS];
    const int tid = threadIdx.x;
    for (int i = tid; i < E; i += kGroupThreads) hist[i] = 0;
    __syncthreads();
    const int t = blockIdx.x * kGroupThreads + tid;
    if (t < T) {
        const int e = ids[t];
        if (e >= 0 && e < E) atomicAdd(&hist[e], 1);  // order-free: exact
    }
    __syncthreads();
    for (int i = tid; i < E; i += kGroupThreads) H[(int64_t)blockIdx.x * E + i] = hist[i];
}

// One workgroup of README_MAX_EXPERTS threads; thread e owns expert e's
// column of H.
__global__ __launch_bounds__(README_MAX_EXPERTS) void k_group_scan(int B, int E,
                                                                   int32_t* __restrict__ H,
                                                                   int32_t* __restrict__ counts,
                                                                   int32_t* __restrict__ offsets) {
    __shared__ int first[README_MAX_EXPERTS];
    const int e = threadIdx.x;
    int total = 0;
    if (e < E)
        for (int b = 0; b < B; ++b) total += H[(int64_t)b * E + e];
    first[e] = total;
    __syncthreads();
    if (e == 0) {
        int run = 0;
        offsets[0] = 0;
        for (int x = 0; x < E; ++x) {
            const int c = first[x];
            first[x] = run;
            counts[x] = c;
            run += c;
            offsets[x + 1] = run;
        }
    }
    __syncthreads();
    if (e < E) {
        int run = first[e];
        for (int b = 0; b < B; ++b) {
            const int64_t i = (int64_t)b * E + e;
            const int h = H[i];
            H[i] = run;
            run += h;
        }
    }
}

// One round of GroupBlock's ranking per chunk, starting from the chunk's
// first rows: ballots over the id bits find the lanes of a wave that share
// an id, the rank inside the wave is the popcount of the lower ones, and the
// per-wave counts are summed in wave order.
__global__ __launch_bounds__(kGroupThreads) void k_group_rank(int T, int E, int nbits,
                                                              const int32_t* __restrict__ ids,
                                                              const int32_t* __restrict__ H,
                                                              int32_t* __restrict__ perm) {
    constexpr int NW = kGroupThreads / 64;
    __shared__ int wcnt[NW * README_MAX_EXPERTS];
    __shared__ int wbase[NW * README_MAX_EXPERTS];
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    for (int i = tid; i < NW * README_MAX_EXPERTS; i += kGroupThreads) wcnt[i] = 0;
    __syncthreads();
    const int t = blockIdx.x * kGroupThreads + tid;
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
    for (int x = tid; x < E; x += kGroupThreads) {
        int run = H[(int64_t)blockIdx.x * E + x];
        for (int w = 0; w < NW; ++w) {
            wbase[w * README_MAX_EXPERTS + x] = run;
            run += wcnt[w * README_MAX_EXPERTS + x];
        }
    }
    __syncthreads();
    if (valid) perm[wbase[wave * README_MAX_EXPERTS + e] + rank] = t;
}

// k_group_scan and k_group_rank in one launch, for few chunks: every
// workgroup forms its own first rows from the whole of H (B * E reads per
// workgroup), and workgroup 0 also writes counts and offsets.  The per-
// expert sums run over the chunks in order, and the scan over experts in
// expert order, so the rows equal the two-launch form.
__global__ __launch_bounds__(kGroupThreads) void k_group_scan_rank(
    int T, int E, int nbits, int B, const int32_t* __restrict__ ids,
    const int32_t* __restrict__ H, int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ perm) {
    constexpr int NW = kGroupThreads / 64;
    __shared__ int wcnt[NW * README_MAX_EXPERTS];
    __shared__ int wbase[NW * README_MAX_EXPERTS];
    __shared__ int total[README_MAX_EXPERTS];
    __shared__ int before[README_MAX_EXPERTS];  // this chunk's tokens of e in earlier chunks
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int b0 = blockIdx.x;
    for (int i = tid; i < NW * README_MAX_EXPERTS; i += kGroupThreads) wcnt[i] = 0;
    for (int x = tid; x < README_MAX_EXPERTS; x += kGroupThreads) {
        int pre = 0, all = 0;
        if (x < E) {
            for (int b = 0; b < B; ++b) {
                const int h = H[(int64_t)b * E + x];
                if (b < b0) pre += h;
                all += h;
            }
        }
        before[x] = pre;
        total[x] = all;
    }
    __syncthreads();
    // Exclusive scan of total over the experts by wave 0: lane l sums experts
    // 4l .. 4l+3 in order, then the lanes are scanned in lane order.
    if (wave == 0) {
        int v[4], sum = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            v[k] = total[4 * lane + k];
            sum += v[k];
        }
        int run = wave_incl_scan(sum, lane) - sum;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int x = 4 * lane + k;
            if (x < E) {
                if (b0 == 0) {
                    counts[x] = v[k];
                    offsets[x] = run;
                    if (x == E - 1) offsets[E] = run + v[k];
                }
                before[x] += run;  // first grouped row of this chunk's tokens of x
            }
            run += v[k];
        }
    }
    const int t = b0 * kGroupThreads + tid;
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
    for (int x = tid; x < E; x += kGroupThreads) {
        int run = before[x];
        for (int w = 0; w < NW; ++w) {
            wbase[w * README_MAX_EXPERTS + x] = run;
            run += wcnt[w * README_MAX_EXPERTS + x];
        }
    }
    __syncthreads();
    if (valid) perm[wbase[wave * README_MAX_EXPERTS + e] + rank] = t;
}

// inv_perm from perm (overwriting H), -1 for unrouted tokens and for the
// rows past the routed ones.
__global__ __launch_bounds__(256) void k_group_inverse(int T, int E,
                                                       const int32_t* __restrict__ ids,
                                                       const int32_t* __restrict__ offsets,
                                                       int32_t* __restrict__ perm,
                                                       int32_t* __restrict__ inv_perm) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= T) return;
    const int routed = offsets[E];
    if (i < routed)
        inv_perm[perm[i]] = i;
    else
        perm[i] = -1;
    const int e = ids[i];
    if (!(e >= 0 && e < E)) inv_perm[i] = -1;
}

// Many workgroups from 8192 tokens: one workgroup needs T/1024 rounds of
// ballots and barriers on one CU (27 us at T = 16384), the four launches
// run each phase on T/1024 CUs.  Up to 2^20 tokens (1024 chunks), so that
// k_group_scan's per-expert walk over the chunks stays short; the counts
// H need B*E <= T entries of inv_perm.
constexpr int64_t kGroupMultiMin = 8192;
constexpr int64_t kGroupMultiMax = 1 << 20;
// Each launch costs a few microseconds however little it does, so up to this
// many counts the scan is repeated inside every ranking workgroup instead of
// running as a launch of its own.
constexpr int64_t kGroupScanInline = 16384;

hipError_t launch_group(int64_t T, int E, const int32_t* ids, int32_t* counts, int32_t* offsets,
                        int32_t* perm, int32_t* inv_perm, hipStream_t s) {
    int nbits = 0;
    while ((1 << nbits) < E) ++nbits;
    const int64_t B = ceil_div(T, (int64_t)kGroupThreads);
    if (T >= kGroupMultiMin && T <= kGroupMultiMax && B * E <= T) {
        int32_t* H = inv_perm;
        k_group_hist<<<dim3((unsigned)B), dim3(kGroupThreads), 0, s>>>((int)T, E, ids, H);
        if (B * E <= kGroupScanInline) {
            k_group_scan_rank<<<dim3((unsigned)B), dim3(kGroupThreads), 0, s>>>(
                (int)T, E, nbits, (int)B, ids, H, counts, offsets, perm);
        } else {
            k_group_scan<<<dim3(1), dim3(README_MAX_EXPERTS), 0, s>>>((int)B, E, H, counts,
                                                                      offsets);
            k_group_rank<<<dim3((unsigned)B), dim3(kGroupThreads), 0, s>>>((int)T, E, nbits, ids,
                                                                           H, perm);
        }
        k_group_inverse<<<dim3((unsigned)ceil_div(T, (int64_t)256)), dim3(256), 0, s>>>(
            (int)T, E, ids, offsets, perm, inv_perm);
        return hipGetLastError();
    }
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
