// Pre-gating router G (Sec. 2.3, Table 1): one causal transformer block over
// each request's tokens, then the linear gate of readme_route on the block's
// normed output (Eq. 2 with K = 1).
//
// Block (pre-norm residual, the norm without gain, fp32 residual stream):
//   x  = E[token]                       (rows of a bf16 table, zero if the
//                                        id is outside the vocabulary)
//   a  = bf16(rmsnorm(x));  [q k v] = bf16(a [Wq; Wk; Wv]^T)
//   q, k <- bf16(RoPE(q, k))            rotate-half pairs (i, i + 64) of each
//                                       128-dim head by p * 10000^(-2i/128),
//                                       p = the token's position in its request
//   o  = bf16(softmax(q k^T / sqrt(128)) v), causal inside each request
//   x += o Wo^T
//   x += W2 (silu(W1 m) * W3 m),  m = bf16(rmsnorm(x))
//   f  = bf16(rmsnorm(x));  ids, logits = gate(f)
// The projections and the MLP run on the grouped-GEMM kernels with one
// "expert" (offsets {0, T}).  Here: the embedding gather fused with the
// first norm, the MLP's norm, RoPE, causal attention, and the final norm
// fused with the gate (readme_route's canonical fp32 order).  Nine launches
// per call (embedding + norm, q|k|v, RoPE, attention, Wo, norm, gate/up, down,
// norm + gate; the last is two, norm then gate, for D > 2048).
#include <limits.h>
#include <math.h>

#include "common.hpp"
#include "internal.hpp"

namespace readme {

namespace {

constexpr int kHeadDim = 128;
// log2(e) / sqrt(128): scores go to exp2 in one multiply.
constexpr float kScoreScale = 0.12751743082459868f;
// Mean request length from which attention runs eight waves per workgroup
// (128 queries, two wave groups over alternate key blocks, every block
// shared by four waves); below it one wave per workgroup loops only over its
// own queries' blocks (a request batch of short requests then needs one key
// block per wave and no wave waits at another's barrier).
constexpr int kAttnLongMean = 128;

// First token of t's request, from the in-request position (clamped, so a
// malformed position never leads outside [0, t]).
__device__ __forceinline__ int64_t request_start(int64_t t, const int32_t* __restrict__ pos) {
    int64_t p = pos[t];
    if (p < 0) p = 0;
    if (p > t) p = t;
    return t - p;
}

// Position of token t in its request: t - ro[r] for the last r with
// ro[r] <= t (ro = request offsets [R + 1], ro[0] = 0, ro[R] = T).
__device__ __forceinline__ int32_t position_of(int64_t t, int32_t R,
                                               const int32_t* __restrict__ ro) {
    int lo = 0, hi = R;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (ro[mid] <= t) lo = mid;
        else hi = mid;
    }
    int64_t start = ro[lo];
    if (start < 0) start = 0;
    if (start > t) start = t;
    return (int32_t)(t - start);
}

// Request offsets staged in LDS for the position search when they fit.
constexpr int kRoLds = 4096;

// Sum over the wave to lane 0 in a fixed order, then broadcast, so that every
// lane holds the same fp32 total.
__device__ __forceinline__ float wave_sum_bcast(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_down(v, off, 64);
    return __shfl(v, 0, 64);
}

// Embedding and the pre-attention norm, one wave per token (four per
// workgroup): x[t] = fp32(emb[tokens[t]]) (zeros for an id outside [0, V)),
// a[t] = bf16(x[t] * r), r = 1 / sqrt(mean x^2 + eps) in fp32 (each lane sums
// its elements in ascending order, then the wave folds).  Lane l owns the
// 8-element chunks l, l + 64, ...: NC > 0 of them (D <= 512 NC) held in
// registers, or with NC = 0 any number, the row read once more from the
// (cached) table for the second pass.  The token id is read before the
// workgroup's barrier, so its round trip overlaps the staging of the request
// offsets in LDS (when R + 1 <= 4096) that the position search of lane 0
// reads; thread 0 of block 0 writes the offsets {0, T} of the one-group
// GEMMs.
template <int NC>
__global__ __launch_bounds__(256) void k_embed_norm(int64_t T, int64_t D, int32_t R, int64_t V,
                                                    float eps,
                                                    const int32_t* __restrict__ tokens,
                                                    const int32_t* __restrict__ ro,
                                                    const uint16_t* __restrict__ emb,
                                                    float* __restrict__ x,
                                                    uint16_t* __restrict__ a,
                                                    int32_t* __restrict__ pos,
                                                    int32_t* __restrict__ offs) {
    __shared__ int32_t ro_lds[kRoLds];
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t tok = t < T ? (int64_t)tokens[t] : -1;
    const bool staged = R + 1 <= kRoLds;
    if (staged)
        for (int i = threadIdx.x; i <= R; i += blockDim.x) ro_lds[i] = ro[i];
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        offs[0] = 0;
        offs[1] = (int32_t)T;
    }
    __syncthreads();
    if (t >= T) return;
    const bool ok = tok >= 0 && tok < V;
    const uint16_t* er = emb + (ok ? tok : 0) * D;
    const int64_t nch = D / 8;
    auto load = [&](int64_t c) {
        uint4 w = make_uint4(0u, 0u, 0u, 0u);
        if (ok) w = *reinterpret_cast<const uint4*>(er + c * 8);
        return w;
    };
    auto put_x = [&](int64_t c, const uint4 w, float& ss) {
        const float v[8] = {bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y),
                            bf16_lo(w.z), bf16_hi(w.z), bf16_lo(w.w), bf16_hi(w.w)};
        float4* dst = reinterpret_cast<float4*>(x + t * D + c * 8);
        dst[0] = make_float4(v[0], v[1], v[2], v[3]);
        dst[1] = make_float4(v[4], v[5], v[6], v[7]);
#pragma unroll
        for (int k = 0; k < 8; ++k) ss += v[k] * v[k];
    };
    auto put_a = [&](int64_t c, const uint4 w, float r) {
        uint4 o;
        o.x = (uint32_t)f32_to_bf16(bf16_lo(w.x) * r) | ((uint32_t)f32_to_bf16(bf16_hi(w.x) * r) << 16);
        o.y = (uint32_t)f32_to_bf16(bf16_lo(w.y) * r) | ((uint32_t)f32_to_bf16(bf16_hi(w.y) * r) << 16);
        o.z = (uint32_t)f32_to_bf16(bf16_lo(w.z) * r) | ((uint32_t)f32_to_bf16(bf16_hi(w.z) * r) << 16);
        o.w = (uint32_t)f32_to_bf16(bf16_lo(w.w) * r) | ((uint32_t)f32_to_bf16(bf16_hi(w.w) * r) << 16);
        *reinterpret_cast<uint4*>(a + t * D + c * 8) = o;
    };
    float ss = 0.0f;
    if constexpr (NC > 0) {
        uint4 w[NC];
#pragma unroll
        for (int j = 0; j < NC; ++j)
            if (lane + 64 * j < nch) w[j] = load(lane + 64 * j);
        if (lane == 0) pos[t] = position_of(t, R, staged ? ro_lds : ro);
#pragma unroll
        for (int j = 0; j < NC; ++j)
            if (lane + 64 * j < nch) put_x(lane + 64 * j, w[j], ss);
        const float r = 1.0f / sqrtf(wave_sum_bcast(ss) / (float)D + eps);
#pragma unroll
        for (int j = 0; j < NC; ++j)
            if (lane + 64 * j < nch) put_a(lane + 64 * j, w[j], r);
    } else {
        if (lane == 0) pos[t] = position_of(t, R, staged ? ro_lds : ro);
        for (int64_t c = lane; c < nch; c += 64) put_x(c, load(c), ss);
        const float r = 1.0f / sqrtf(wave_sum_bcast(ss) / (float)D + eps);
        for (int64_t c = lane; c < nch; c += 64) put_a(c, load(c), r);
    }
}

// m[t] = bf16(x[t] * r), r as above; one wave per row, lane l owning the
// 4-element chunks l, l + 64, ... (the row read twice, the second time from
// cache).
__global__ __launch_bounds__(256) void k_rms_rows(int64_t T, int64_t D, float eps,
                                                  const float* __restrict__ x,
                                                  uint16_t* __restrict__ m) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;
    const float4* row = reinterpret_cast<const float4*>(x + t * D);
    const int64_t n4 = D / 4;
    float ss = 0.0f;
    for (int64_t c = lane; c < n4; c += 64) {
        const float4 v = row[c];
        ss += v.x * v.x;
        ss += v.y * v.y;
        ss += v.z * v.z;
        ss += v.w * v.w;
    }
    const float r = 1.0f / sqrtf(wave_sum_bcast(ss) / (float)D + eps);
    uint2* out = reinterpret_cast<uint2*>(m + t * D);
    for (int64_t c = lane; c < n4; c += 64) {
        const float4 v = row[c];
        uint2 o;
        o.x = (uint32_t)f32_to_bf16(v.x * r) | ((uint32_t)f32_to_bf16(v.y * r) << 16);
        o.y = (uint32_t)f32_to_bf16(v.z * r) | ((uint32_t)f32_to_bf16(v.w * r) << 16);
        out[c] = o;
    }
}

// The final norm and the gate in one pass, one wave per token, for D <= 2048
// (at most NC = 4 chunks of 8 per lane, held in registers):
//   f[t] = bf16(x[t] * r)                         (written out)
//   logit[t][e] = canonical fp32 sum of f[t][k] * w_router[e][k] + bias[e]
// The canonical order (the one readme_route follows): 16-byte chunks of f and
// w_router (8 bf16 values), chunk c to partial c mod 64 -- here lane c mod
// 64 -- each partial fusing multiply-adds in ascending k from +0, the 64
// partials folded pairwise (p[l] += p[l + off], off = 32 .. 1), then the
// bias added.  id = first e of largest logit (strict '>' from e = 0).
template <int NC>
__global__ __launch_bounds__(256) void k_norm_gate(int64_t T, int64_t D, int E, float eps,
                                                   const float* __restrict__ x,
                                                   const uint16_t* __restrict__ w,
                                                   const float* __restrict__ bias,
                                                   uint16_t* __restrict__ f,
                                                   int32_t* __restrict__ ids,
                                                   float* __restrict__ logits) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;
    const int nch = (int)(D / 8);
    // The first eight experts' gate rows are requested with x, so that their
    // round trip overlaps the norm.
    uint4 w0[8][NC];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int e = i < E ? i : E - 1;
#pragma unroll
        for (int j = 0; j < NC; ++j) {
            const int c = lane + 64 * j;
            if (c < nch) w0[i][j] = *reinterpret_cast<const uint4*>(w + (int64_t)e * D + (int64_t)c * 8);
        }
    }
    float v[NC][8];
    float ss = 0.0f;
#pragma unroll
    for (int j = 0; j < NC; ++j) {
        const int c = lane + 64 * j;
        if (c < nch) {
            const float4* src = reinterpret_cast<const float4*>(x + t * D + (int64_t)c * 8);
            const float4 p0 = src[0], p1 = src[1];
            v[j][0] = p0.x; v[j][1] = p0.y; v[j][2] = p0.z; v[j][3] = p0.w;
            v[j][4] = p1.x; v[j][5] = p1.y; v[j][6] = p1.z; v[j][7] = p1.w;
#pragma unroll
            for (int k = 0; k < 8; ++k) ss += v[j][k] * v[j][k];
        }
    }
    const float r = 1.0f / sqrtf(wave_sum_bcast(ss) / (float)D + eps);
#pragma unroll
    for (int j = 0; j < NC; ++j) {
        const int c = lane + 64 * j;
        if (c < nch) {
            uint16_t b[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                b[k] = f32_to_bf16(v[j][k] * r);
                v[j][k] = bf16_lo(b[k]);
            }
            uint4 o;
            o.x = (uint32_t)b[0] | ((uint32_t)b[1] << 16);
            o.y = (uint32_t)b[2] | ((uint32_t)b[3] << 16);
            o.z = (uint32_t)b[4] | ((uint32_t)b[5] << 16);
            o.w = (uint32_t)b[6] | ((uint32_t)b[7] << 16);
            *reinterpret_cast<uint4*>(f + t * D + (int64_t)c * 8) = o;
        }
    }
    // Eight experts at a time, so that their partial sums and pairwise folds
    // proceed side by side.
    int best_e = 0;
    float best = 0.0f;
    for (int e0 = 0; e0 < E; e0 += 8) {
        float p[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) p[i] = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = e0 + i < E ? e0 + i : E - 1;   // clamped rows are not used
#pragma unroll
            for (int j = 0; j < NC; ++j) {
                const int c = lane + 64 * j;
                if (c < nch) {
                    const uint4 wv =
                        e0 == 0 ? w0[i][j]
                                : *reinterpret_cast<const uint4*>(w + (int64_t)e * D + (int64_t)c * 8);
                    const float wf[8] = {bf16_lo(wv.x), bf16_hi(wv.x), bf16_lo(wv.y),
                                         bf16_hi(wv.y), bf16_lo(wv.z), bf16_hi(wv.z),
                                         bf16_lo(wv.w), bf16_hi(wv.w)};
#pragma unroll
                    for (int k = 0; k < 8; ++k) p[i] = fmaf(v[j][k], wf[k], p[i]);
                }
            }
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1)
#pragma unroll
            for (int i = 0; i < 8; ++i) p[i] = p[i] + __shfl_down(p[i], off, 64);
        if (lane == 0) {
            for (int i = 0; i < 8 && e0 + i < E; ++i) {
                const int e = e0 + i;
                const float lg = bias ? p[i] + bias[e] : p[i];
                if (logits) logits[t * E + e] = lg;
                if (e == 0 || lg > best) {
                    best = lg;
                    best_e = e;
                }
            }
        }
    }
    if (lane == 0) ids[t] = best_e;
}

__global__ __launch_bounds__(256) void k_positions(int64_t T, int32_t R,
                                                   const int32_t* __restrict__ ro,
                                                   int32_t* __restrict__ pos) {
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < T;
         t += (int64_t)gridDim.x * blockDim.x)
        pos[t] = position_of(t, R, ro);
}

// RoPE in place on NH heads of 128 bf16 values per row (row t at x + t*ld).
// One thread per (token, pair indices i0 and i0 + 1): per i the angle
// pos[t] * 10000^(-2i/128) and its cosine and sine in fp64 (the 64 inverse
// frequencies computed once per workgroup), then for each head the 4-byte
// runs (x_i0, x_i0+1) and (x_i0+64, x_i0+65), each pair rotated in fp64
// without fused multiply-adds and rounded to fp32 and then to bf16 (nearest
// even).  Two pairs per thread keep four waves per SIMD for the fp64 sine
// and cosine.
__global__ __launch_bounds__(256) void k_rope(int64_t T, int NH,
                                              const int32_t* __restrict__ pos,
                                              uint16_t* __restrict__ x, int64_t ld) {
#pragma clang fp contract(off)
    __shared__ double inv_lds[64];
    if (threadIdx.x < 64)
        inv_lds[threadIdx.x] = pow(10000.0, -2.0 * (double)threadIdx.x / (double)kHeadDim);
    __syncthreads();
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= T * 32) return;
    const int64_t t = g >> 5;
    const int i0 = (int)(g & 31) * 2;
    const double p = (double)pos[t];
    double cs[2], sn[2];
    sincos(p * inv_lds[i0], &sn[0], &cs[0]);
    sincos(p * inv_lds[i0 + 1], &sn[1], &cs[1]);
    uint16_t* row = x + t * ld + i0;
    // Heads in batches of 8: every load of a batch is issued before its
    // first store (a store could alias a later head's load otherwise, which
    // would serialise the loads).
    for (int h0 = 0; h0 < NH; h0 += 8) {
        const int nb = NH - h0 < 8 ? NH - h0 : 8;
        uint32_t wa[8], wb[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (j < nb) {
                const uint16_t* lo = row + (int64_t)(h0 + j) * kHeadDim;
                wa[j] = *reinterpret_cast<const uint32_t*>(lo);
                wb[j] = *reinterpret_cast<const uint32_t*>(lo + 64);
            }
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (j >= nb) continue;
            uint32_t oa = 0, ob = 0;
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const double av = (double)(k ? bf16_hi(wa[j]) : bf16_lo(wa[j]));
                const double bv = (double)(k ? bf16_hi(wb[j]) : bf16_lo(wb[j]));
                const double xa = av * cs[k] - bv * sn[k];
                const double xb = bv * cs[k] + av * sn[k];
                oa |= (uint32_t)f32_to_bf16((float)xa) << (16 * k);
                ob |= (uint32_t)f32_to_bf16((float)xb) << (16 * k);
            }
            uint16_t* lo = row + (int64_t)(h0 + j) * kHeadDim;
            *reinterpret_cast<uint32_t*>(lo) = oa;
            *reinterpret_cast<uint32_t*>(lo + 64) = ob;
        }
    }
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Causal attention of one 128-dim head over 32 * QW queries per workgroup
// (QW = NW / KS waves of queries, KS = 1 or 2 wave groups over the keys).
//   Wave w owns queries t = q0 + 32 (w % QW) + (lane % 32); both half-waves
//   hold the same queries (the matrix-core layout splits each 32-key block
//   between them).  Per key block of 32 rows, staged in LDS (K row-major,
//   V transposed):
//     S^T = K Q^T     8 MFMAs 32x32x16, Q in registers, so each lane holds
//                     16 of its query's 32 scores and the softmax needs one
//                     cross-lane step (lane ^ 32);
//     mask            key in [start(t), t] (same request, not after t);
//     online softmax  running max m and sum l per query, fp32, hardware
//                     exp2 (a rescale by exactly 1 is skipped wave-wide);
//     O^T += V^T P^T  P split into bf16 hi + lo parts (p - hi is exact in
//                     fp32) by the packed hardware conversion, 2 x 8 MFMAs,
//                     so the weights carry ~16 bits; the key order of P's
//                     operand is the score layout's, and V^T is read from
//                     LDS in the same order.
//   o = O / l, rounded to bf16.  Key blocks run from the first query's
//   request start to the last query; a wave skips the blocks outside its own
//   queries' range (the workgroup still passes every barrier).
//   NW = 1 (short requests): each wave loads only its own blocks, one LDS
//   buffer.  NW = 8, KS = 2 (long requests): wave group g = w / 4 takes the
//   blocks kb0 + 2i + g, so the longest chain of blocks is halved and each
//   SIMD runs two waves; the eight waves load each pair of blocks together,
//   two LDS buffers, the next pair requested into registers before this one
//   is computed and written to the other buffer after it, one barrier per
//   pair.  At the end group 1 hands (m, l, O) to group 0 through LDS, which
//   merges the two online softmaxes: m = max(m0, m1), O = O0 2^(m0-m) +
//   O1 2^(m1-m), l likewise.  The two forms add the keys in different
//   orders, so their last bits may differ.
template <int NW, int KS>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2)))
void k_attention_causal(int64_t T, const int32_t* __restrict__ pos,
                        const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                        const uint16_t* __restrict__ v, int64_t ldi, uint16_t* __restrict__ o,
                        int64_t ldo) {
    constexpr int QW = NW / KS;       // waves of distinct queries
    constexpr int KP = kHeadDim + 8;  // K rows in LDS, 272 bytes apart
    constexpr int VP = 32 + 8;        // V^T rows (one per dim), 80 bytes apart
    constexpr bool PF = NW > 1;       // next blocks in flight during these
    constexpr int NB = PF ? 2 : 1;    // LDS buffers
    constexpr int NCH = KS * 32 * (kHeadDim / 8) / (64 * NW);  // 16-byte chunks per thread
    static_assert(NCH >= 1 && KS * 32 * (kHeadDim / 8) == NCH * 64 * NW, "chunk split");
    constexpr int BLK = 32 * KP + kHeadDim * VP;  // one key block (K, V^T), uint16
    __shared__ __attribute__((aligned(16))) uint16_t lds[NB * KS * BLK];
    auto k_at = [&](int b, int h) { return lds + (b * KS + h) * BLK; };
    auto vt_at = [&](int b, int h) { return lds + (b * KS + h) * BLK + 32 * KP; };

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int qg = wv % QW, grp = wv / QW;
    const int hf = lane >> 5, col = lane & 31;
    const int64_t hoff = (int64_t)blockIdx.y * kHeadDim;
    const int64_t q0 = (int64_t)blockIdx.x * (32 * QW);
    const int64_t t = q0 + 32 * qg + col;
    const bool tv = t < T;
    const int64_t tq = tv ? t : T - 1;
    const int64_t start = request_start(tq, pos);
    const int64_t wfirst = q0 + 32 * qg;
    const bool wact = wfirst < T;
    const int64_t wlo = request_start(wact ? wfirst : T - 1, pos);
    const int64_t whi = wfirst + 31 < T - 1 ? wfirst + 31 : T - 1;
    const int64_t lo = request_start(q0, pos);
    const int64_t hi = q0 + 32 * QW - 1 < T - 1 ? q0 + 32 * QW - 1 : T - 1;
    const int64_t kb0 = lo >> 5, kb1 = hi >> 5;

    // Chunk i of this thread: block group c / 512, key row (c % 512) / 16 of
    // that block, 8 dims at 8 * (c % 16).
    uint4 kr[NCH], vr[NCH];
    auto fetch = [&](int64_t kbase) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int c = tid + i * 64 * NW;
            const int64_t key = (kbase + (c >> 9)) * 32 + ((c & 511) >> 4);
            kr[i] = make_uint4(0u, 0u, 0u, 0u);
            vr[i] = kr[i];
            if (key <= kb1 * 32 + 31 && key < T) {
                kr[i] = *reinterpret_cast<const uint4*>(k + key * ldi + hoff + (c & 15) * 8);
                vr[i] = *reinterpret_cast<const uint4*>(v + key * ldi + hoff + (c & 15) * 8);
            }
        }
    };
    auto stash = [&](int b) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int c = tid + i * 64 * NW;
            const int h = c >> 9, r = (c & 511) >> 4, ch = c & 15;
            *reinterpret_cast<uint4*>(k_at(b, h) + r * KP + ch * 8) = kr[i];
            uint16_t* vt = vt_at(b, h);
            const uint32_t vw[4] = {vr[i].x, vr[i].y, vr[i].z, vr[i].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                vt[(ch * 8 + 2 * e) * VP + r] = (uint16_t)(vw[e] & 0xffffu);
                vt[(ch * 8 + 2 * e + 1) * VP + r] = (uint16_t)(vw[e] >> 16);
            }
        }
    };

    bf16x8 qf[8];
    {
        const uint16_t* qrow = q + tq * ldi + hoff + hf * 8;
#pragma unroll
        for (int s = 0; s < 8; ++s) qf[s] = *reinterpret_cast<const bf16x8*>(qrow + s * 16);
    }
    f32x16 acc[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mt][r] = 0.0f;
    float m_run = -INFINITY, l_run = 0.0f;

    auto compute = [&](int64_t kb, int b) __attribute__((always_inline)) {
        const int64_t k0 = kb * 32;
        if (!(wact && kb <= kb1 && k0 <= whi && k0 + 31 >= wlo)) return;
        const uint16_t* kl = k_at(b, grp);
        const uint16_t* vl = vt_at(b, grp);
        f32x16 s;
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kl + col * KP + ks * 16 + hf * 8);
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s, 0, 0, 0);
        }
        // lane holds keys k0 + 4*hf + off(r), off(r) = 8*(r/4) + (r%4), of
        // query t; the key is valid for lo_off <= off(r) <= hi_off
        const int lo_off = (int)(start - k0) - 4 * hf;
        const int hi_off = tv ? (int)(t - k0) - 4 * hf : -1;
        float sv[16];
        float mb = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int off = 8 * (r >> 2) + (r & 3);
            sv[r] = ((off >= lo_off) & (off <= hi_off)) ? s[r] * kScoreScale : -INFINITY;
            mb = fmaxf(mb, sv[r]);
        }
        mb = fmaxf(mb, __shfl_xor(mb, 32, 64));
        const float mn = fmaxf(m_run, mb);
        const float base = mn == -INFINITY ? 0.0f : mn;
        const float alpha = __builtin_amdgcn_exp2f(m_run - base);
        m_run = mn;
        l_run *= alpha;
        // The weights' hi and lo bf16 parts, two per instruction (the
        // hardware conversion rounds to nearest even; p is finite)
        uint32_t ph[8], pl[8];
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
            const f32x2 p = {__builtin_amdgcn_exp2f(sv[r] - base),
                             __builtin_amdgcn_exp2f(sv[r + 1] - base)};
            l_run += p[0];
            l_run += p[1];
            const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(p, bf16x2));
            const f32x2 e = {p[0] - bf16_lo(h), p[1] - bf16_hi(h)};
            ph[r >> 1] = h;
            pl[r >> 1] = __builtin_bit_cast(uint32_t, __builtin_convertvector(e, bf16x2));
        }
        if (__any(alpha != 1.0f)) {  // a factor of exactly 1 changes nothing
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mt][r] *= alpha;
        }
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const u32x4 bh = {ph[4 * kk], ph[4 * kk + 1], ph[4 * kk + 2], ph[4 * kk + 3]};
            const u32x4 bl = {pl[4 * kk], pl[4 * kk + 1], pl[4 * kk + 2], pl[4 * kk + 3]};
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const uint16_t* vp = vl + (mt * 32 + col) * VP + 16 * kk + 4 * hf;
                const uint2 a0 = *reinterpret_cast<const uint2*>(vp);
                const uint2 a1 = *reinterpret_cast<const uint2*>(vp + 8);
                const u32x4 av = {a0.x, a0.y, a1.x, a1.y};
                acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, av), __builtin_bit_cast(bf16x8, bh), acc[mt], 0,
                    0, 0);
                acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, av), __builtin_bit_cast(bf16x8, bl), acc[mt], 0,
                    0, 0);
            }
        }
    };

    // Steps of KS blocks: step p holds blocks kb0 + KS p .. + KS - 1.
    const int64_t np = (kb1 - kb0 + KS) / KS;
    if constexpr (PF) {
        fetch(kb0);
        stash(0);
        __syncthreads();
        for (int64_t p = 0; p < np; ++p) {
            const int b = (int)(p & 1);
            if (p + 1 < np) fetch(kb0 + KS * (p + 1));
            compute(kb0 + KS * p + grp, b);
            if (p + 1 < np) stash(b ^ 1);
            __syncthreads();
        }
    } else {
        for (int64_t p = 0; p < np; ++p) {
            fetch(kb0 + p);
            stash(0);
            __syncthreads();
            compute(kb0 + p, 0);
            __syncthreads();
        }
    }

    if constexpr (KS == 2) {
        // Group 1 hands its state to group 0 (the loop's last barrier has
        // passed, so the LDS blocks are free): lane-major, 66 floats a lane.
        float* xs = reinterpret_cast<float*>(lds) + qg * 66 * 64;
        static_assert(QW * 66 * 64 * 4 <= NB * KS * BLK * 2, "merge area");
        if (grp == 1) {
            xs[lane] = m_run;
            xs[64 + lane] = l_run;
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int r = 0; r < 16; ++r) xs[(2 + mt * 16 + r) * 64 + lane] = acc[mt][r];
        }
        __syncthreads();
        if (grp == 1) return;
        const float m1 = xs[lane], l1 = xs[64 + lane];
        const float mn = fmaxf(m_run, m1);
        const float base = mn == -INFINITY ? 0.0f : mn;
        const float a0 = __builtin_amdgcn_exp2f(m_run - base);
        const float a1 = __builtin_amdgcn_exp2f(m1 - base);
        l_run = l_run * a0 + l1 * a1;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[mt][r] = acc[mt][r] * a0 + xs[(2 + mt * 16 + r) * 64 + lane] * a1;
    }

    const float lt = l_run + __shfl_xor(l_run, 32, 64);
    if (!tv) return;
    const float inv = 1.0f / lt;
    uint16_t* orow = o + t * ldo + hoff;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            // regs 4g .. 4g+3 hold dims 32*mt + 8*g + 4*hf + 0..3
            uint2 w;
            w.x = (uint32_t)f32_to_bf16(acc[mt][4 * g] * inv) |
                  ((uint32_t)f32_to_bf16(acc[mt][4 * g + 1] * inv) << 16);
            w.y = (uint32_t)f32_to_bf16(acc[mt][4 * g + 2] * inv) |
                  ((uint32_t)f32_to_bf16(acc[mt][4 * g + 3] * inv) << 16);
            *reinterpret_cast<uint2*>(orow + mt * 32 + 8 * g + 4 * hf) = w;
        }
    }
}

unsigned grid_of(int64_t n, int64_t cap) {
    const int64_t b = ceil_div(n, 256);
    return (unsigned)(b < 1 ? 1 : (b > cap ? cap : b));
}

hipError_t launch_embed_norm(int64_t T, int64_t D, int32_t R, int64_t V, float eps,
                             const int32_t* tokens, const int32_t* ro, const void* emb,
                             float* x, uint16_t* a, int32_t* pos, int32_t* offs,
                             hipStream_t s) {
    const unsigned grid = (unsigned)ceil_div(T, 4);
    const auto* eb = reinterpret_cast<const uint16_t*>(emb);
    if (D <= 512)
        k_embed_norm<1><<<grid, 256, 0, s>>>(T, D, R, V, eps, tokens, ro, eb, x, a, pos, offs);
    else if (D <= 1024)
        k_embed_norm<2><<<grid, 256, 0, s>>>(T, D, R, V, eps, tokens, ro, eb, x, a, pos, offs);
    else if (D <= 2048)
        k_embed_norm<4><<<grid, 256, 0, s>>>(T, D, R, V, eps, tokens, ro, eb, x, a, pos, offs);
    else
        k_embed_norm<0><<<grid, 256, 0, s>>>(T, D, R, V, eps, tokens, ro, eb, x, a, pos, offs);
    return hipGetLastError();
}

hipError_t launch_rms_rows(int64_t T, int64_t D, float eps, const float* x, uint16_t* m,
                           hipStream_t s) {
    k_rms_rows<<<(unsigned)ceil_div(T, 4), 256, 0, s>>>(T, D, eps, x, m);
    return hipGetLastError();
}

// Final norm + gate: fused for D <= 2048, else the norm then readme_route's
// kernel (the same canonical gate).
hipError_t launch_norm_gate(int64_t T, int64_t D, int E, float eps, const float* x,
                            const void* w, const float* bias, uint16_t* f, int32_t* ids,
                            float* logits, hipStream_t s) {
    const unsigned grid = (unsigned)ceil_div(T, 4);
    const uint16_t* wb = reinterpret_cast<const uint16_t*>(w);
    if (D <= 512)
        k_norm_gate<1><<<grid, 256, 0, s>>>(T, D, E, eps, x, wb, bias, f, ids, logits);
    else if (D <= 1024)
        k_norm_gate<2><<<grid, 256, 0, s>>>(T, D, E, eps, x, wb, bias, f, ids, logits);
    else if (D <= 2048)
        k_norm_gate<4><<<grid, 256, 0, s>>>(T, D, E, eps, x, wb, bias, f, ids, logits);
    else {
        hipError_t e = launch_rms_rows(T, D, eps, x, f, s);
        if (e != hipSuccess) return e;
        return launch_route(README_BF16, T, D, E, f, w, bias, ids, logits, s);
    }
    return hipGetLastError();
}

hipError_t launch_positions(int64_t T, int32_t R, const int32_t* ro, int32_t* pos,
                            hipStream_t s) {
    k_positions<<<grid_of(T, 1 << 16), 256, 0, s>>>(T, R, ro, pos);
    return hipGetLastError();
}

hipError_t launch_rope(int64_t T, int NH, const int32_t* pos, void* x, int64_t ld,
                       hipStream_t s) {
    k_rope<<<(unsigned)ceil_div(T * 32, 256), 256, 0, s>>>(T, NH, pos,
                                                          reinterpret_cast<uint16_t*>(x), ld);
    return hipGetLastError();
}

// Requests of 128 tokens or more on average take the four-wave pipelined
// form (the waves share each key block); shorter ones the single-wave form.
hipError_t launch_attention(int64_t T, int H, int32_t R, const int32_t* pos, const void* q,
                            const void* k, const void* v, int64_t ldi, void* o, int64_t ldo,
                            hipStream_t s) {
    const auto* qb = reinterpret_cast<const uint16_t*>(q);
    const auto* kb = reinterpret_cast<const uint16_t*>(k);
    const auto* vb = reinterpret_cast<const uint16_t*>(v);
    auto* ob = reinterpret_cast<uint16_t*>(o);
    if (T >= (int64_t)kAttnLongMean * (R > 0 ? R : 1)) {
        const dim3 grid((unsigned)ceil_div(T, 128), (unsigned)H);
        k_attention_causal<8, 2><<<grid, 512, 0, s>>>(T, pos, qb, kb, vb, ldi, ob, ldo);
    } else {
        const dim3 grid((unsigned)ceil_div(T, 32), (unsigned)H);
        k_attention_causal<1, 1><<<grid, 64, 0, s>>>(T, pos, qb, kb, vb, ldi, ob, ldo);
    }
    return hipGetLastError();
}

// Tile configurations (TILE_* of the grouped GEMM) of the block's GEMMs
// from a sweep of all tiles at 8192 tokens, D = F = 512: q|k|v (N = 3D)
// 27.4 us with the eight-wave 256-row tiles, o and down (N = D) 15.6 -
// 16.3 us with 64 x 256 four-wave tiles against 28 us automatic, gate/up
// (N = 2F) 18.2 us with 128 x 256 LDS tiles against 28.6.
constexpr int kTileQkv = 30;     // TILE_MIX8_256
constexpr int kTileNarrow = 13;  // TILE_BD_64x256
constexpr int kTileGateUp = 4;   // TILE_128x256

// C[T][ldc] (+)= A[T][K] W^T over one group of all T rows, W a blocked bf16
// [N][K] matrix.
GemmArgs plain_args(const void* A, int64_t K, const void* W, int64_t N, const int32_t* offs,
                    int64_t T, void* C, int64_t ldc) {
    GemmArgs g{};
    g.A = A;
    g.lda = K;
    g.B = W;
    g.ldb = K;
    g.b_expert_stride = N * K;
    g.N = N;
    g.K = K;
    g.offsets = offs;
    g.E = 1;
    g.T = T;
    g.C = C;
    g.ldc = ldc;
    g.m_tiles32 = (int)ceil_div(T, 32);
    return g;
}

inline readme_status st_of(hipError_t e) { return e == hipSuccess ? README_OK : README_ERR_HIP; }
inline bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// Supported block shapes: heads of 128 (D a multiple of 128), every packed
// matrix addressable with 32-bit offsets.
readme_status check_block(int64_t D, int64_t F) {
    if (D <= 0 || F < 1) return README_ERR_ARG;
    if (D % kHeadDim != 0 || D > 16384 || padded_I(F) * 2 * D * 2 > INT32_MAX)
        return README_ERR_UNSUPPORTED;
    return README_OK;
}

// Byte offsets of the workspace regions (each 256-byte aligned).
int64_t region_offset(int64_t T, int64_t D, int64_t F, int region) {
    const int64_t Fp = padded_I(F);
    const int64_t sizes[README_RTF_END] = {
        T * D * 4,      // X: fp32 residual
        T * D * 2,      // A: bf16 pre-attention norm
        T * 3 * D * 2,  // QKV
        T * D * 2,      // O
        T * D * 2,      // M: bf16 pre-MLP norm
        T * Fp * 2,     // H: silu(W1 m) * W3 m
        T * D * 2,      // FEAT: bf16 final norm
        T * 4,          // POS
        8,              // OFFS
    };
    int64_t off = 0;
    for (int i = 0; i < region; ++i) off += round_up(sizes[i], 256);
    return off;
}

}  // namespace

}  // namespace readme

using namespace readme;

extern "C" {

size_t readme_router_tf_packed_bytes(int64_t D, int64_t F) {
    if (check_block(D, F) != README_OK) return 0;
    return (size_t)4 * D * D * 2 + packed_bytes(README_BF16, 1, D, F);
}

readme_status readme_router_tf_pack(int64_t D, int64_t F, const void* wq, const void* wk,
                                    const void* wv, const void* wo, const void* w1,
                                    const void* w3, const void* w2, void* packed,
                                    size_t packed_bytes_given, void* stream) {
    const readme_status st = check_block(D, F);
    if (st != README_OK) return st;
    if (!wq || !wk || !wv || !wo || !w1 || !w3 || !w2 || !packed) return README_ERR_ARG;
    if (!al16(packed)) return README_ERR_ARG;
    if (packed_bytes_given < readme_router_tf_packed_bytes(D, F)) return README_ERR_WORKSPACE;
    hipStream_t s = as_stream(stream);
    char* p = reinterpret_cast<char*>(packed);
    hipError_t e = launch_pack_rows_bf16(3 * D, D, 0, D, wq, D, p, s);
    if (e == hipSuccess) e = launch_pack_rows_bf16(3 * D, D, D, D, wk, D, p, s);
    if (e == hipSuccess) e = launch_pack_rows_bf16(3 * D, D, 2 * D, D, wv, D, p, s);
    if (e == hipSuccess) e = launch_pack_rows_bf16(D, D, 0, D, wo, D, p + 3 * D * D * 2, s);
    if (e == hipSuccess) e = launch_pack(README_BF16, 1, D, F, w1, w3, w2, p + 4 * D * D * 2, s);
    return st_of(e);
}

int64_t readme_router_tf_workspace_offset(int64_t T, int64_t D, int64_t F, int32_t region) {
    if (T < 0 || check_block(D, F) != README_OK || region < 0 || region > README_RTF_END)
        return -1;
    return region_offset(T, D, F, region);
}

size_t readme_router_tf_workspace_bytes(int64_t T, int64_t D, int64_t F) {
    const int64_t n = readme_router_tf_workspace_offset(T, D, F, README_RTF_END);
    return n < 0 ? 0 : (size_t)n;
}

readme_status readme_request_positions(int64_t T, int32_t R, const int32_t* req_offsets,
                                       int32_t* pos, void* stream) {
    if (T < 0 || R < 0) return README_ERR_ARG;
    if (T > INT32_MAX) return README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (R < 1 || !req_offsets || !pos) return README_ERR_ARG;
    return st_of(launch_positions(T, R, req_offsets, pos, as_stream(stream)));
}

readme_status readme_rope(int64_t T, int32_t H, const int32_t* pos, void* x, int64_t ld,
                          void* stream) {
    if (T < 0 || H < 0 || ld < (int64_t)H * kHeadDim) return README_ERR_ARG;
    if (T > INT32_MAX) return README_ERR_UNSUPPORTED;
    if (T == 0 || H == 0) return README_OK;
    if (!pos || !x || !al16(x) || ld % 8) return README_ERR_ARG;
    return st_of(launch_rope(T, H, pos, x, ld, as_stream(stream)));
}

readme_status readme_attention_causal(int64_t T, int32_t H, int32_t R, const int32_t* pos,
                                      const void* q, const void* k, const void* v, int64_t ld_in,
                                      void* o, int64_t ld_out, void* stream) {
    if (T < 0 || H < 0 || R < 0) return README_ERR_ARG;
    if (ld_in < (int64_t)H * kHeadDim || ld_out < (int64_t)H * kHeadDim) return README_ERR_ARG;
    if (T > INT32_MAX || H > 65535) return README_ERR_UNSUPPORTED;
    if (T == 0 || H == 0) return README_OK;
    if (!pos || !q || !k || !v || !o) return README_ERR_ARG;
    if (!al16(q) || !al16(k) || !al16(v) || !al16(o) || ld_in % 8 || ld_out % 8)
        return README_ERR_ARG;
    return st_of(launch_attention(T, H, R, pos, q, k, v, ld_in, o, ld_out, as_stream(stream)));
}

readme_status readme_router_tf(int64_t T, int32_t R, int64_t D, int64_t F, int32_t E, int64_t V,
                               const int32_t* tokens, const int32_t* req_offsets,
                               const void* emb, const void* packed, const void* w_router,
                               const float* bias, float rms_eps, int32_t* expert_ids,
                               float* logits, void* workspace, size_t workspace_bytes,
                               void* stream) {
    readme_status st = check_block(D, F);
    if (st != README_OK) return st;
    if (T < 0 || R < 0 || V < 1 || !(rms_eps >= 0.0f)) return README_ERR_ARG;
    if (E < 1 || E > README_MAX_EXPERTS || T > INT32_MAX) return README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (R < 1 || !tokens || !req_offsets || !emb || !packed || !w_router || !expert_ids ||
        !workspace)
        return README_ERR_ARG;
    if (!al16(emb) || !al16(packed) || !al16(w_router) || !al16(workspace)) return README_ERR_ARG;
    if (workspace_bytes < readme_router_tf_workspace_bytes(T, D, F)) return README_ERR_WORKSPACE;

    hipStream_t s = as_stream(stream);
    char* ws = reinterpret_cast<char*>(workspace);
    auto at = [&](int r) { return ws + region_offset(T, D, F, r); };
    float* x = reinterpret_cast<float*>(at(README_RTF_X));
    uint16_t* a = reinterpret_cast<uint16_t*>(at(README_RTF_A));
    uint16_t* qkv = reinterpret_cast<uint16_t*>(at(README_RTF_QKV));
    uint16_t* o = reinterpret_cast<uint16_t*>(at(README_RTF_O));
    uint16_t* m = reinterpret_cast<uint16_t*>(at(README_RTF_M));
    uint16_t* h = reinterpret_cast<uint16_t*>(at(README_RTF_H));
    uint16_t* feat = reinterpret_cast<uint16_t*>(at(README_RTF_FEAT));
    int32_t* pos = reinterpret_cast<int32_t*>(at(README_RTF_POS));
    int32_t* offs = reinterpret_cast<int32_t*>(at(README_RTF_OFFS));
    const char* pk = reinterpret_cast<const char*>(packed);
    const int H = (int)(D / kHeadDim);

    // Tiles of the four GEMMs (K = D): measured on MI355X at Table 1's widths
    // over 8192 tokens, where the automatic choice (tuned for the experts'
    // K of 4096 - 8192) leaves most CUs idle on the N = D products.
    const bool wide = T >= 2048 && D <= 1024;
    hipError_t e = launch_embed_norm(T, D, R, V, rms_eps, tokens, req_offsets, emb, x, a, pos,
                                     offs, s);
    if (e == hipSuccess) {
        GemmArgs g = plain_args(a, D, pk, 3 * D, offs, T, qkv, 3 * D);
        g.tile = wide ? kTileQkv : 0;
        e = launch_grouped_gemm(false, EPI_STORE, g, s);
    }
    if (e == hipSuccess) e = launch_rope(T, 2 * H, pos, qkv, 3 * D, s);
    if (e == hipSuccess)
        e = launch_attention(T, H, R, pos, qkv, qkv + D, qkv + 2 * D, 3 * D, o, D, s);
    if (e == hipSuccess) {
        GemmArgs g = plain_args(o, D, pk + 3 * D * D * 2, D, offs, T, x, D);
        g.tile = wide ? kTileNarrow : 0;
        e = launch_grouped_gemm(false, EPI_RESID_ADD, g, s);
    }
    if (e == hipSuccess) e = launch_rms_rows(T, D, rms_eps, x, m, s);
    const void* mlp = pk + 4 * D * D * 2;
    if (e == hipSuccess) {
        GemmArgs gu = gate_up_args(README_BF16, T, D, 1, F, m, offs, mlp, h);
        gu.m_tiles32 = (int)ceil_div(T, 32);
        gu.tile = wide ? kTileGateUp : 0;
        e = launch_grouped_gemm(false, EPI_GATE_UP_SILU, gu, s);
    }
    if (e == hipSuccess) {
        GemmArgs dn = down_args(README_BF16, T, D, 1, F, h, offs, mlp, x);
        dn.m_tiles32 = (int)ceil_div(T, 32);
        dn.tile = wide ? kTileNarrow : 0;
        e = launch_grouped_gemm(false, EPI_RESID_ADD, dn, s);
    }
    if (e == hipSuccess)
        e = launch_norm_gate(T, D, E, rms_eps, x, w_router, bias, feat, expert_ids, logits, s);
    return st_of(e);
}

}  // extern "C"
