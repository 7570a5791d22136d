// Pre-gating router, top-1 (Eq. 2 with K = 1): one expert id per token,
// computed once ahead of all layers.
//
// The argmax decides an integer, so every logit is summed in one fixed fp32
// order (stated in readme.h): hardware lane l of a wave owns 16-byte chunks
// l, l + 64, l + 128, ... of the token row and of the router row, fuses
// multiply-adds over them in ascending k from +0, and the 64 lane partials
// fold pairwise with offsets 32, 16, 8, 4, 2, 1.  Each wave handles R tokens
// at once so that one router-row load feeds R tokens; each router row chunk
// is a coalesced 1 KB wave load.  The path is VALU-bound (fp32 FMA), not
// MFMA: an MFMA's internal accumulation order is not this order.
#include <type_traits>

#include "common.hpp"
#include "internal.hpp"

namespace readme {

template <int W>
struct Chunk;
template <>
struct Chunk<8> {  // 8 bf16
    __device__ static void unpack(const uint4 q, float* v) {
        v[0] = bf16_lo(q.x); v[1] = bf16_hi(q.x);
        v[2] = bf16_lo(q.y); v[3] = bf16_hi(q.y);
        v[4] = bf16_lo(q.z); v[5] = bf16_hi(q.z);
        v[6] = bf16_lo(q.w); v[7] = bf16_hi(q.w);
    }
    __device__ static void load(const void* base, int64_t idx, float* v) {
        unpack(reinterpret_cast<const uint4*>(base)[idx], v);
    }
};
template <>
struct Chunk<4> {  // 4 fp32
    __device__ static void unpack(const uint4 q, float* v) {
        v[0] = __uint_as_float(q.x); v[1] = __uint_as_float(q.y);
        v[2] = __uint_as_float(q.z); v[3] = __uint_as_float(q.w);
    }
    __device__ static void load(const void* base, int64_t idx, float* v) {
        unpack(reinterpret_cast<const uint4*>(base)[idx], v);
    }
};

template <int R, int EB, int W>
__global__ __launch_bounds__(256) void k_route(int64_t T, int64_t d, int E,
                                               const void* __restrict__ x,
                                               const void* __restrict__ wr,
                                               const float* __restrict__ bias,
                                               int32_t* __restrict__ ids,
                                               float* __restrict__ logits) {
    const int lane = threadIdx.x & 63;
    const int64_t t0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * R;
    if (t0 >= T) return;
    const int64_t nchunks = d / W;  // chunks per row

    int64_t trow[R];
#pragma unroll
    for (int r = 0; r < R; ++r) trow[r] = (t0 + r < T ? t0 + r : T - 1) * nchunks;

    float best[R];
    int bid[R];
#pragma unroll
    for (int r = 0; r < R; ++r) { best[r] = 0.0f; bid[r] = 0; }

    for (int e0 = 0; e0 < E; e0 += EB) {
        float acc[R][EB];
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int b = 0; b < EB; ++b) acc[r][b] = 0.0f;

        for (int64_t c = lane; c < nchunks; c += 64) {
            float xv[R][W];
#pragma unroll
            for (int r = 0; r < R; ++r) Chunk<W>::load(x, trow[r] + c, xv[r]);
#pragma unroll
            for (int b = 0; b < EB; ++b) {
                if (e0 + b < E) {
                    float wv[W];
                    Chunk<W>::load(wr, (int64_t)(e0 + b) * nchunks + c, wv);
#pragma unroll
                    for (int r = 0; r < R; ++r)
#pragma unroll
                        for (int q = 0; q < W; ++q)
                            acc[r][b] = __builtin_fmaf(xv[r][q], wv[q], acc[r][b]);
                }
            }
        }

#pragma unroll
        for (int b = 0; b < EB; ++b) {
            const int e = e0 + b;
            if (e >= E) break;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                float v = acc[r][b];
#pragma unroll
                for (int off = 32; off >= 1; off >>= 1) {
                    const float o = __shfl_down(v, off, 64);
                    v = v + o;
                }
                float logit = __shfl(v, 0, 64);
                if (bias) logit = logit + bias[e];
                if (logits && lane == 0 && t0 + r < T) logits[(t0 + r) * E + e] = logit;
                if (e == 0) {
                    best[r] = logit;
                    bid[r] = 0;
                } else if (logit > best[r]) {
                    best[r] = logit;
                    bid[r] = e;
                }
            }
        }
    }
    if (lane == 0) {
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (t0 + r < T) ids[t0 + r] = bid[r];
    }
}

// Register-resident variant for rows of at most 64*CPL chunks: the lane's
// chunks of its R token rows are loaded once, up front; the router rows are
// then streamed expert by expert with the next expert's chunks in flight
// while the current one is summed.  Same summation order as k_route.
template <int R, int CPL, int W>
__global__ __launch_bounds__(256) void k_route_reg(int64_t T, int64_t d, int E,
                                                   const void* __restrict__ x,
                                                   const void* __restrict__ wr,
                                                   const float* __restrict__ bias,
                                                   int32_t* __restrict__ ids,
                                                   float* __restrict__ logits) {
    const int lane = threadIdx.x & 63;
    const int64_t t0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * R;
    if (t0 >= T) return;
    const int nchunks = (int)(d / W);
    const uint4* xq = reinterpret_cast<const uint4*>(x);
    const uint4* wq = reinterpret_cast<const uint4*>(wr);

    uint4 xr[R][CPL];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t row = (t0 + r < T ? t0 + r : T - 1) * nchunks;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            const int c = lane + 64 * j;
            xr[r][j] = c < nchunks ? xq[row + c] : make_uint4(0, 0, 0, 0);
        }
    }
    auto load_w = [&](uint4* wb, int e) {
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            const int c = lane + 64 * j;
            wb[j] = c < nchunks ? wq[(int64_t)e * nchunks + c] : make_uint4(0, 0, 0, 0);
        }
    };

    float best[R];
    int bid[R];
#pragma unroll
    for (int r = 0; r < R; ++r) { best[r] = 0.0f; bid[r] = 0; }

    // Logit of expert e from router chunks wb, then the running argmax.
    auto expert = [&](const uint4* wb, int e) {
        float acc[R];
#pragma unroll
        for (int r = 0; r < R; ++r) acc[r] = 0.0f;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            if (lane + 64 * j >= nchunks) break;
            float wv[W];
            Chunk<W>::unpack(wb[j], wv);
#pragma unroll
            for (int r = 0; r < R; ++r) {
                float xv[W];
                Chunk<W>::unpack(xr[r][j], xv);
#pragma unroll
                for (int q = 0; q < W; ++q) acc[r] = __builtin_fmaf(xv[q], wv[q], acc[r]);
            }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            float v = acc[r];
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                const float o = __shfl_down(v, off, 64);
                v = v + o;
            }
            float logit = __shfl(v, 0, 64);
            if (bias) logit = logit + bias[e];
            if (logits && lane == 0 && t0 + r < T) logits[(t0 + r) * E + e] = logit;
            if (e == 0) {
                best[r] = logit;
                bid[r] = 0;
            } else if (logit > best[r]) {
                best[r] = logit;
                bid[r] = e;
            }
        }
    };

    // Two named buffers (not an array indexed by e & 1, which would go to
    // scratch): the next expert's row is in flight while this one is summed.
    uint4 wa[CPL], wb[CPL];
    load_w(wa, 0);
    for (int e = 0; e < E; e += 2) {
        if (e + 1 < E) load_w(wb, e + 1);
        expert(wa, e);
        if (e + 1 >= E) break;
        if (e + 2 < E) load_w(wa, e + 2);
        expert(wb, e + 1);
    }
    if (lane == 0) {
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (t0 + r < T) ids[t0 + r] = bid[r];
    }
}

template <int R, int W>
static hipError_t launch_route_r(int64_t T, int64_t d, int E, const void* x, const void* w,
                                 const float* bias, int32_t* ids, float* logits,
                                 hipStream_t s) {
    const int64_t blocks = ceil_div(T, 4 * R);
    if (E <= 4)
        k_route<R, 4, W><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(T, d, E, x, w, bias, ids, logits);
    else if (E <= 8)
        k_route<R, 8, W><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(T, d, E, x, w, bias, ids, logits);
    else
        k_route<R, 16, W><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(T, d, E, x, w, bias, ids, logits);
    return hipGetLastError();
}

// LDS-resident variant: the whole router matrix (E*d elements, at most
// LDS_BYTES) is staged in LDS once per workgroup; each of the 8 waves then
// walks R-token groups of the workgroup's TB tokens with the token rows in
// registers, reading router chunks from LDS (consecutive lanes read
// consecutive 16 bytes: conflict-free).  Same summation order as k_route.
template <int R, int CPL, int W, int LDS_BYTES, int EB>
__global__ __launch_bounds__(512) void k_route_lds(int64_t T, int64_t d, int E, int tb,
                                                   const void* __restrict__ x,
                                                   const void* __restrict__ wr,
                                                   const float* __restrict__ bias,
                                                   int32_t* __restrict__ ids,
                                                   float* __restrict__ logits) {
    __shared__ uint4 wl[LDS_BYTES / 16];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int nchunks = (int)(d / W);
    const uint4* xq = reinterpret_cast<const uint4*>(x);
    const int64_t tb0 = (int64_t)blockIdx.x * tb;
    uint4 xr[R][CPL];
    auto load_x = [&](int64_t t0) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int64_t row = (t0 + r < T ? t0 + r : T - 1) * nchunks;
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                const int c = lane + 64 * j;
                xr[r][j] = c < nchunks ? xq[row + c] : make_uint4(0, 0, 0, 0);
            }
        }
    };
    // The first token group's rows are requested before the router matrix
    // is staged, so the two memory latencies overlap (when the rows fit in
    // registers next to the staging buffer).
    constexpr bool EARLY = R * CPL < 16;
    if (EARLY && wave * R < tb && tb0 + wave * R < T) load_x(tb0 + wave * R);
    {
        // All loads of the staging are issued before the first LDS store.
        constexpr int PER = LDS_BYTES / 16 / 512;
        const uint4* wq = reinterpret_cast<const uint4*>(wr);
        const int n = E * nchunks;
        constexpr int BATCH = PER < 8 ? PER : 8;
#pragma unroll
        for (int k0 = 0; k0 < PER; k0 += BATCH) {
            uint4 tmp[BATCH];
#pragma unroll
            for (int k = 0; k < BATCH; ++k) {
                const int i = (int)threadIdx.x + 512 * (k0 + k);
                tmp[k] = i < n ? wq[i] : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
            for (int k = 0; k < BATCH; ++k) {
                const int i = (int)threadIdx.x + 512 * (k0 + k);
                if (i < n) wl[i] = tmp[k];
            }
        }
    }
    __syncthreads();

    for (int g = wave; g * R < tb; g += 8) {
        const int64_t t0 = tb0 + (int64_t)g * R;
        if (t0 >= T) break;
        if (!EARLY || g != wave) load_x(t0);
        float best[R];
        int bid[R];
#pragma unroll
        for (int r = 0; r < R; ++r) { best[r] = 0.0f; bid[r] = 0; }
        // Experts in blocks of EB: all R x EB partial sums are formed first,
        // then folded together, so the cross-lane shuffles of different
        // (token, expert) pairs overlap instead of running one chain at a
        // time.  Each pair's own order is the canonical one.
        for (int e0 = 0; e0 < E; e0 += EB) {
            float acc[R][EB];
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int b = 0; b < EB; ++b) acc[r][b] = 0.0f;
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                const int c = lane + 64 * j;
                if (c >= nchunks) break;
                float xv[R][W];
#pragma unroll
                for (int r = 0; r < R; ++r) Chunk<W>::unpack(xr[r][j], xv[r]);
#pragma unroll
                for (int b = 0; b < EB; ++b) {
                    if (e0 + b >= E) break;
                    float wv[W];
                    Chunk<W>::unpack(wl[(e0 + b) * nchunks + c], wv);
#pragma unroll
                    for (int r = 0; r < R; ++r)
#pragma unroll
                        for (int q = 0; q < W; ++q)
                            acc[r][b] = __builtin_fmaf(xv[r][q], wv[q], acc[r][b]);
                }
            }
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1)
#pragma unroll
                for (int r = 0; r < R; ++r)
#pragma unroll
                    for (int b = 0; b < EB; ++b) {
                        const float o = __shfl_down(acc[r][b], off, 64);
                        acc[r][b] = acc[r][b] + o;
                    }
#pragma unroll
            for (int b = 0; b < EB; ++b) {
                const int e = e0 + b;
                if (e >= E) break;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    float logit = __shfl(acc[r][b], 0, 64);
                    if (bias) logit = logit + bias[e];
                    if (logits && lane == 0 && t0 + r < T) logits[(t0 + r) * E + e] = logit;
                    if (e == 0) {
                        best[r] = logit;
                        bid[r] = 0;
                    } else if (logit > best[r]) {
                        best[r] = logit;
                        bid[r] = e;
                    }
                }
            }
        }
        if (lane == 0) {
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (t0 + r < T) ids[t0 + r] = bid[r];
        }
    }
}

// bf16 variant for one token per wave: the router matrix is staged in LDS
// as fp32, in two planes (elements 0-3 and 4-7 of each 8-element chunk, so
// consecutive lanes still read consecutive 16 bytes), converted once per
// workgroup instead of once per token.  Same summation order as k_route.
template <int CPL, int LDS_BYTES, int EB>
__global__ __launch_bounds__(512) void k_route_lds_f32w(int64_t T, int64_t d, int E, int tb,
                                                        const void* __restrict__ x,
                                                        const void* __restrict__ wr,
                                                        const float* __restrict__ bias,
                                                        int32_t* __restrict__ ids,
                                                        float* __restrict__ logits) {
    constexpr int PLANE = LDS_BYTES / 32;  // float4 per plane
    __shared__ float4 wl[2][PLANE];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int nchunks = (int)(d / 8);
    const uint4* xq = reinterpret_cast<const uint4*>(x);
    const int64_t tb0 = (int64_t)blockIdx.x * tb;
    uint4 xr[CPL];
    auto load_x = [&](int64_t t) {
        const int64_t row = (t < T ? t : T - 1) * nchunks;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            const int c = lane + 64 * j;
            xr[j] = c < nchunks ? xq[row + c] : make_uint4(0, 0, 0, 0);
        }
    };
    // The first token row is requested before the router matrix is staged.
    if (wave < tb && tb0 + wave < T) load_x(tb0 + wave);
    {
        const uint4* wq = reinterpret_cast<const uint4*>(wr);
        const int n = E * nchunks;
        constexpr int PER = PLANE / 512;
        constexpr int BATCH = PER < 8 ? PER : 8;
#pragma unroll
        for (int k0 = 0; k0 < PER; k0 += BATCH) {
            uint4 tmp[BATCH];
#pragma unroll
            for (int k = 0; k < BATCH; ++k) {
                const int i = (int)threadIdx.x + 512 * (k0 + k);
                tmp[k] = i < n ? wq[i] : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
            for (int k = 0; k < BATCH; ++k) {
                const int i = (int)threadIdx.x + 512 * (k0 + k);
                if (i < n) {
                    float v[8];
                    Chunk<8>::unpack(tmp[k], v);
                    wl[0][i] = make_float4(v[0], v[1], v[2], v[3]);
                    wl[1][i] = make_float4(v[4], v[5], v[6], v[7]);
                }
            }
        }
    }
    __syncthreads();

    for (int g = wave; g < tb; g += 8) {
        const int64_t t = tb0 + g;
        if (t >= T) break;
        if (g != wave) load_x(t);
        float best = 0.0f;
        int bid = 0;
        for (int e0 = 0; e0 < E; e0 += EB) {
            float acc[EB];
#pragma unroll
            for (int b = 0; b < EB; ++b) acc[b] = 0.0f;
#pragma unroll
            for (int j = 0; j < CPL; ++j) {
                const int c = lane + 64 * j;
                if (c >= nchunks) break;
                float xv[8];
                Chunk<8>::unpack(xr[j], xv);
#pragma unroll
                for (int b = 0; b < EB; ++b) {
                    if (e0 + b >= E) break;
                    const float4 w0 = wl[0][(e0 + b) * nchunks + c];
                    const float4 w1 = wl[1][(e0 + b) * nchunks + c];
                    acc[b] = __builtin_fmaf(xv[0], w0.x, acc[b]);
                    acc[b] = __builtin_fmaf(xv[1], w0.y, acc[b]);
                    acc[b] = __builtin_fmaf(xv[2], w0.z, acc[b]);
                    acc[b] = __builtin_fmaf(xv[3], w0.w, acc[b]);
                    acc[b] = __builtin_fmaf(xv[4], w1.x, acc[b]);
                    acc[b] = __builtin_fmaf(xv[5], w1.y, acc[b]);
                    acc[b] = __builtin_fmaf(xv[6], w1.z, acc[b]);
                    acc[b] = __builtin_fmaf(xv[7], w1.w, acc[b]);
                }
            }
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1)
#pragma unroll
                for (int b = 0; b < EB; ++b) {
                    const float o = __shfl_down(acc[b], off, 64);
                    acc[b] = acc[b] + o;
                }
#pragma unroll
            for (int b = 0; b < EB; ++b) {
                const int e = e0 + b;
                if (e >= E) break;
                float logit = __shfl(acc[b], 0, 64);
                if (bias) logit = logit + bias[e];
                if (logits && lane == 0) logits[t * E + e] = logit;
                if (e == 0) {
                    best = logit;
                    bid = 0;
                } else if (logit > best) {
                    best = logit;
                    bid = e;
                }
            }
        }
        if (lane == 0) ids[t] = bid;
    }
}

// Many tokens, 9..16 experts (bf16): four tokens per wave, all experts'
// partial sums in registers, and the 64 lane partials of the 64 (token,
// expert) pairs folded together.  The canonical fold adds lane l + off into
// lane l for off = 32, 16, ..., 1; here, at the step of `off`, each lane keeps
// the half of its pairs whose pair index agrees with the lane index in that
// bit and adds the partner lane's (l ^ off) values for them, so after six
// steps lane l holds pair l's sum, formed by the same additions (fp32
// addition is commutative, so a + b and b + a are the same bits) -- one
// exchange per pair instead of six.  The router matrix is staged in LDS;
// token chunks are streamed one chunk ahead.  Same summation order as k_route.
template <int CPL>
__global__ __launch_bounds__(512) void k_route_fold16(int64_t T, int64_t d, int E, int tb,
                                                      const void* __restrict__ x,
                                                      const void* __restrict__ wr,
                                                      const float* __restrict__ bias,
                                                      int32_t* __restrict__ ids,
                                                      float* __restrict__ logits) {
    constexpr int R = 4, EP = 16;
    __shared__ uint4 wl[131072 / 16];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int nchunks = (int)(d / 8);
    const uint4* xq = reinterpret_cast<const uint4*>(x);
    const int64_t tb0 = (int64_t)blockIdx.x * tb;
    {
        // Rows of experts E .. 15 are staged as zeros, so every expert slot
        // is summed without a branch (their logits are never used).
        const uint4* wq = reinterpret_cast<const uint4*>(wr);
        const int n = E * nchunks, n16 = EP * nchunks;
        constexpr int PER = 131072 / 16 / 512;
#pragma unroll
        for (int k0 = 0; k0 < PER; k0 += 8) {
            uint4 tmp[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int i = (int)threadIdx.x + 512 * (k0 + k);
                tmp[k] = i < n ? wq[i] : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int i = (int)threadIdx.x + 512 * (k0 + k);
                if (i < n16) wl[i] = tmp[k];
            }
        }
    }
    __syncthreads();

    for (int g = wave; g * R < tb; g += 8) {
        const int64_t t0 = tb0 + (int64_t)g * R;
        if (t0 >= T) break;
        int64_t row[R];
#pragma unroll
        for (int r = 0; r < R; ++r) row[r] = (t0 + r < T ? t0 + r : T - 1) * nchunks;
        auto load = [&](uint4 (&q)[R], int j) {
            const int c = lane + 64 * j;
#pragma unroll
            for (int r = 0; r < R; ++r) q[r] = c < nchunks ? xq[row[r] + c] : make_uint4(0, 0, 0, 0);
        };
        float acc[R * EP];
#pragma unroll
        for (int p = 0; p < R * EP; ++p) acc[p] = 0.0f;
        uint4 xa[R], xb[R];
        load(xa, 0);
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            // chunk j in xa (even j) or xb (odd j); the next one is requested first
            uint4 (&cur)[R] = (j & 1) ? xb : xa;
            uint4 (&nxt)[R] = (j & 1) ? xa : xb;
            if (j + 1 < CPL) load(nxt, j + 1);
            const int c = lane + 64 * j;
            if (c < nchunks) {
                float xv[R][8];
#pragma unroll
                for (int r = 0; r < R; ++r) Chunk<8>::unpack(cur[r], xv[r]);
#pragma unroll
                for (int e = 0; e < EP; ++e) {
                    float wv[8];
                    Chunk<8>::unpack(wl[e * nchunks + c], wv);
#pragma unroll
                    for (int r = 0; r < R; ++r)
#pragma unroll
                        for (int q = 0; q < 8; ++q)
                            acc[r * EP + e] = __builtin_fmaf(xv[r][q], wv[q], acc[r * EP + e]);
                }
            }
        }
        // Fold: pair p = r * EP + e; after the step of `off` a lane keeps the
        // pairs whose bit log2(off) equals its own.
        auto fold_step = [&](auto half_c) {
            constexpr int H = decltype(half_c)::value;  // pairs kept = H
            const bool up = (lane & H) != 0;
#pragma unroll
            for (int i = 0; i < H; ++i) {
                const float mine = up ? acc[H + i] : acc[i];
                const float give = up ? acc[i] : acc[H + i];
                const float got = __shfl_xor(give, H, 64);
                acc[i] = mine + got;
            }
        };
        fold_step(std::integral_constant<int, 32>{});
        fold_step(std::integral_constant<int, 16>{});
        fold_step(std::integral_constant<int, 8>{});
        fold_step(std::integral_constant<int, 4>{});
        fold_step(std::integral_constant<int, 2>{});
        fold_step(std::integral_constant<int, 1>{});
        // Lane l now holds pair l: token r = l / EP, expert e = l % EP.
        const int r = lane / EP, e = lane % EP;
        float logit = acc[0];
        if (bias && e < E) logit = logit + bias[e];
        if (logits && e < E && t0 + r < T) logits[(t0 + r) * E + e] = logit;
        // First maximum in index order (strict >: ties to the lowest index,
        // a NaN never wins), each lane scanning its token's E logits.
        float best = __shfl(logit, r * EP, 64);
        int bid = 0;
        for (int k = 1; k < E; ++k) {
            const float v = __shfl(logit, r * EP + k, 64);
            if (v > best) {
                best = v;
                bid = k;
            }
        }
        if (e == 0 && t0 + r < T) ids[t0 + r] = bid;
    }
}

template <int CPL>
static hipError_t launch_route_fold16(int64_t T, int64_t d, int E, const void* x, const void* w,
                                      const float* bias, int32_t* ids, float* logits,
                                      hipStream_t s) {
    int64_t tb = ceil_div(T, 256);
    tb = tb < 8 ? 8 : (tb > 128 ? 128 : tb);
    tb = round_up(tb, 4);
    k_route_fold16<CPL><<<dim3((unsigned)ceil_div(T, tb)), dim3(512), 0, s>>>(
        T, d, E, (int)tb, x, w, bias, ids, logits);
    return hipGetLastError();
}

template <int R, int CPL, int W, int LDS_BYTES>
static hipError_t launch_route_lds_r(int64_t T, int64_t d, int E, const void* x, const void* w,
                                     const float* bias, int32_t* ids, float* logits,
                                     hipStream_t s) {
    // Tokens per workgroup: enough workgroups to fill the chip, and enough
    // tokens per workgroup to amortise staging the router matrix.
    int64_t tb = ceil_div(T, 256);
    tb = tb < 8 ? 8 : (tb > 128 ? 128 : tb);
    tb = round_up(tb, R);
    const dim3 grid((unsigned)ceil_div(T, tb)), block(512);
    // Expert block: up to 16 partial sums per token, fewer when the token
    // rows already take many registers (two waves per SIMD, no spills).
    constexpr int EBMAX = R * CPL >= 16 ? 8 : 16;
    if (E <= 4)
        k_route_lds<R, CPL, W, LDS_BYTES, 4><<<grid, block, 0, s>>>(T, d, E, (int)tb, x, w, bias, ids, logits);
    else if (E <= 8)
        k_route_lds<R, CPL, W, LDS_BYTES, 8><<<grid, block, 0, s>>>(T, d, E, (int)tb, x, w, bias, ids, logits);
    else
        k_route_lds<R, CPL, W, LDS_BYTES, EBMAX><<<grid, block, 0, s>>>(T, d, E, (int)tb, x, w, bias, ids, logits);
    return hipGetLastError();
}

// R tokens per wave group: as many as the token rows' registers allow with
// two waves per SIMD (no spills).
// One token per wave with the router as fp32 planes (bf16, E * d * 4 <= 128 KB).
template <int CPL>
static hipError_t launch_route_f32w(int64_t T, int64_t d, int E, const void* x, const void* w,
                                    const float* bias, int32_t* ids, float* logits,
                                    hipStream_t s) {
    int64_t tb = ceil_div(T, 256);
    tb = tb < 8 ? 8 : (tb > 128 ? 128 : tb);
    const dim3 grid((unsigned)ceil_div(T, tb)), block(512);
    if ((int64_t)E * d * 4 <= 65536)
        k_route_lds_f32w<CPL, 65536, 4><<<grid, block, 0, s>>>(T, d, E, (int)tb, x, w, bias, ids, logits);
    else
        k_route_lds_f32w<CPL, 131072, 4><<<grid, block, 0, s>>>(T, d, E, (int)tb, x, w, bias, ids, logits);
    return hipGetLastError();
}

template <int W, int LDS_BYTES>
static hipError_t launch_route_lds(int cpl, int64_t T, int64_t d, int E, const void* x,
                                   const void* w, const float* bias, int32_t* ids, float* logits,
                                   hipStream_t s) {
    // Few tokens per CU: one token per wave keeps all eight waves busy.
    if (T <= 4096 && cpl <= 16) {
        switch (cpl) {
            case 1: return launch_route_lds_r<1, 1, W, LDS_BYTES>(T, d, E, x, w, bias, ids, logits, s);
            case 2: return launch_route_lds_r<1, 2, W, LDS_BYTES>(T, d, E, x, w, bias, ids, logits, s);
            case 4: return launch_route_lds_r<1, 4, W, LDS_BYTES>(T, d, E, x, w, bias, ids, logits, s);
            case 8: return launch_route_lds_r<1, 8, W, LDS_BYTES>(T, d, E, x, w, bias, ids, logits, s);
            default: break;
        }
    }
    switch (cpl) {
        case 1: return launch_route_lds_r<4, 1, W, LDS_BYTES>(T, d, E, x, w, bias, ids, logits, s);
        case 2: return launch_route_lds_r<4, 2, W, LDS_BYTES>(T, d, E, x, w, bias, ids, logits, s);
        case 4: return launch_route_lds_r<4, 4, W, LDS_BYTES>(T, d, E, x, w, bias, ids, logits, s);
        case 8: return launch_route_lds_r<2, 8, W, LDS_BYTES>(T, d, E, x, w, bias, ids, logits, s);
        default: return launch_route_lds_r<1, 16, W, LDS_BYTES>(T, d, E, x, w, bias, ids, logits, s);
    }
}

template <int R, int W>
static hipError_t launch_route_reg(int cpl, int64_t T, int64_t d, int E, const void* x,
                                   const void* w, const float* bias, int32_t* ids, float* logits,
                                   hipStream_t s) {
    const dim3 grid((unsigned)ceil_div(T, 4 * R)), block(256);
    switch (cpl) {
        case 1: k_route_reg<R, 1, W><<<grid, block, 0, s>>>(T, d, E, x, w, bias, ids, logits); break;
        case 2: k_route_reg<R, 2, W><<<grid, block, 0, s>>>(T, d, E, x, w, bias, ids, logits); break;
        case 4: k_route_reg<R, 4, W><<<grid, block, 0, s>>>(T, d, E, x, w, bias, ids, logits); break;
        case 8: k_route_reg<R, 8, W><<<grid, block, 0, s>>>(T, d, E, x, w, bias, ids, logits); break;
        default: k_route_reg<R, 16, W><<<grid, block, 0, s>>>(T, d, E, x, w, bias, ids, logits); break;
    }
    return hipGetLastError();
}

hipError_t launch_route(readme_dtype dt, int64_t T, int64_t d, int E, const void* x,
                        const void* w, const float* bias, int32_t* ids, float* logits,
                        hipStream_t s) {
    // Rows of up to 1024 chunks (8192 bf16 / 4096 fp32) stay in registers.
    const int64_t nchunks = d / (dt == README_BF16 ? 8 : 4);
    if (nchunks <= 64 * 16) {
        int cpl = 1;
        while (64 * cpl < nchunks) cpl *= 2;
        // Router matrix in LDS when it fits (64 KB, or 128 KB for many tokens).
        const int64_t wbytes = (int64_t)E * d * (dt == README_BF16 ? 2 : 4);
        // bf16 with one token per wave: router unpacked to fp32 once per
        // workgroup when it fits (measured at T = 2048, d = 4096, E = 8:
        // 10.9 vs 11.9 us).
        if (dt == README_BF16 && 2 * wbytes <= 131072 && T <= 4096) {
            switch (cpl) {
                case 1: return launch_route_f32w<1>(T, d, E, x, w, bias, ids, logits, s);
                case 2: return launch_route_f32w<2>(T, d, E, x, w, bias, ids, logits, s);
                case 4: return launch_route_f32w<4>(T, d, E, x, w, bias, ids, logits, s);
                case 8: return launch_route_f32w<8>(T, d, E, x, w, bias, ids, logits, s);
                default: break;
            }
        }
        if (wbytes <= 65536) {
            if (dt == README_BF16)
                return launch_route_lds<8, 65536>(cpl, T, d, E, x, w, bias, ids, logits, s);
            return launch_route_lds<4, 65536>(cpl, T, d, E, x, w, bias, ids, logits, s);
        }
        // Many tokens, 9..16 experts: the folded kernel (16 router rows,
        // zero-padded past E, in LDS).
        if (dt == README_BF16 && E > 8 && E <= 16 && 16 * d * 2 <= 131072 && T >= 8192) {
            switch (cpl) {
                case 1: return launch_route_fold16<1>(T, d, E, x, w, bias, ids, logits, s);
                case 2: return launch_route_fold16<2>(T, d, E, x, w, bias, ids, logits, s);
                case 4: return launch_route_fold16<4>(T, d, E, x, w, bias, ids, logits, s);
                case 8: return launch_route_fold16<8>(T, d, E, x, w, bias, ids, logits, s);
                default: break;
            }
        }
        if (wbytes <= 131072 && T >= 8192) {
            if (dt == README_BF16)
                return launch_route_lds<8, 131072>(cpl, T, d, E, x, w, bias, ids, logits, s);
            return launch_route_lds<4, 131072>(cpl, T, d, E, x, w, bias, ids, logits, s);
        }
        if (dt == README_BF16)
            return T >= 8192 ? launch_route_reg<2, 8>(cpl, T, d, E, x, w, bias, ids, logits, s)
                             : launch_route_reg<1, 8>(cpl, T, d, E, x, w, bias, ids, logits, s);
        return T >= 8192 ? launch_route_reg<2, 4>(cpl, T, d, E, x, w, bias, ids, logits, s)
                         : launch_route_reg<1, 4>(cpl, T, d, E, x, w, bias, ids, logits, s);
    }
    // Few tokens: one token per wave spreads the work over the chip; many
    // tokens: four per wave so that one router-row load serves four tokens.
    const bool many = T >= 8192;
    if (dt == README_BF16)
        return many ? launch_route_r<4, 8>(T, d, E, x, w, bias, ids, logits, s)
                    : launch_route_r<1, 8>(T, d, E, x, w, bias, ids, logits, s);
    return many ? launch_route_r<4, 4>(T, d, E, x, w, bias, ids, logits, s)
                : launch_route_r<1, 4>(T, d, E, x, w, bias, ids, logits, s);
}

}  // namespace readme
