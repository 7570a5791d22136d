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
// "expert" (offsets {0, T}); the norms and the gate reuse the FFN stack's
// kernels.  New here: the embedding gather, RoPE and causal attention.
#include <limits.h>
#include <math.h>

#include "common.hpp"
#include "internal.hpp"

namespace readme {

namespace {

constexpr int kHeadDim = 128;
// log2(e) / sqrt(128): scores go to exp2 in one multiply.
constexpr float kScoreScale = 0.12751743082459868f;

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

// x[t] = fp32(emb[tokens[t]]) (zeros outside [0, V)), 8 elements per thread;
// the first chunk's thread also writes pos[t], thread 0 the offsets {0, T}
// of the one-group GEMM launches.
__global__ __launch_bounds__(256) void k_embed(int64_t T, int64_t D, int32_t R, int64_t V,
                                               const int32_t* __restrict__ tokens,
                                               const int32_t* __restrict__ ro,
                                               const uint16_t* __restrict__ emb,
                                               float* __restrict__ x, int32_t* __restrict__ pos,
                                               int32_t* __restrict__ offs) {
    const int64_t n8 = D / 8, total = T * n8;
    const int64_t first = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (first == 0) {
        offs[0] = 0;
        offs[1] = (int32_t)T;
    }
    for (int64_t i = first; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t t = i / n8, c = i - t * n8;
        const int64_t tok = tokens[t];
        uint4 w = make_uint4(0u, 0u, 0u, 0u);
        if (tok >= 0 && tok < V) w = *reinterpret_cast<const uint4*>(emb + tok * D + c * 8);
        float4* dst = reinterpret_cast<float4*>(x + t * D + c * 8);
        dst[0] = make_float4(bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y));
        dst[1] = make_float4(bf16_lo(w.z), bf16_hi(w.z), bf16_lo(w.w), bf16_hi(w.w));
        if (c == 0) pos[t] = position_of(t, R, ro);
    }
}

__global__ __launch_bounds__(256) void k_positions(int64_t T, int32_t R,
                                                   const int32_t* __restrict__ ro,
                                                   int32_t* __restrict__ pos) {
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < T;
         t += (int64_t)gridDim.x * blockDim.x)
        pos[t] = position_of(t, R, ro);
}

// RoPE in place on NH heads of 128 bf16 values per row (row t at x + t*ld).
// One thread per (token, pair index i): the angle and its cosine and sine
// in fp64, the rotation of each head's pair (i, i + 64) in fp64 without
// fused multiply-adds, then the round to fp32 and to bf16 (nearest even).
__global__ __launch_bounds__(256) void k_rope(int64_t T, int NH,
                                              const int32_t* __restrict__ pos,
                                              uint16_t* __restrict__ x, int64_t ld) {
#pragma clang fp contract(off)
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= T * 64) return;
    const int64_t t = g >> 6;
    const int i = (int)(g & 63);
    const double inv = pow(10000.0, -2.0 * (double)i / (double)kHeadDim);
    const double ang = (double)pos[t] * inv;
    double sn, cs;
    sincos(ang, &sn, &cs);
    uint16_t* row = x + t * ld;
    for (int hh = 0; hh < NH; ++hh) {
        uint16_t* p = row + (int64_t)hh * kHeadDim;
        const double a = (double)bf16_lo(p[i]);
        const double b = (double)bf16_lo(p[i + 64]);
        const double ra = a * cs - b * sn;
        const double rb = b * cs + a * sn;
        p[i] = f32_to_bf16((float)ra);
        p[i + 64] = f32_to_bf16((float)rb);
    }
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Causal attention of one 128-dim head over 128 queries per workgroup.
//   Wave w owns queries t = q0 + 32w + (lane % 32); both half-waves hold the
//   same queries (the matrix-core layout splits each key block between
//   them).  Per key block of 32 rows, staged in LDS (K row-major, V
//   transposed):
//     S^T = K Q^T     8 MFMAs 32x32x16, Q in registers, so each lane holds
//                     16 of its query's 32 scores and the softmax needs one
//                     cross-lane step (lane ^ 32);
//     mask            key in [start(t), t] (same request, not after t);
//     online softmax  running max m and sum l per query, fp32, exp2;
//     O^T += V^T P^T  P split into bf16 hi + lo parts (p - hi is exact in
//                     fp32), 2 x 8 MFMAs, so the weights carry ~16 bits;
//                     the key order of P's operand is the score layout's,
//                     and V^T is read from LDS in the same order.
//   o = O / l, rounded to bf16.  Key blocks run from the first query's
//   request start to the last query; a wave skips the blocks outside its own
//   queries' range (the workgroup still passes every barrier).
__global__ __launch_bounds__(256) void k_attention_causal(
    int64_t T, const int32_t* __restrict__ pos, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, int64_t ldi,
    uint16_t* __restrict__ o, int64_t ldo) {
    constexpr int KP = kHeadDim + 8;  // K rows in LDS, 272 bytes apart
    constexpr int VP = 32 + 8;        // V^T rows (one per dim), 80 bytes apart
    __shared__ __attribute__((aligned(16))) uint16_t k_lds[32 * KP];
    __shared__ __attribute__((aligned(16))) uint16_t vt_lds[kHeadDim * VP];

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int hf = lane >> 5, col = lane & 31;
    const int64_t hoff = (int64_t)blockIdx.y * kHeadDim;
    const int64_t q0 = (int64_t)blockIdx.x * 128;
    const int64_t t = q0 + 32 * wv + col;
    const bool tv = t < T;
    const int64_t tq = tv ? t : T - 1;
    const int64_t start = request_start(tq, pos);
    const int64_t wfirst = q0 + 32 * wv;
    const bool wact = wfirst < T;
    const int64_t wlo = request_start(wact ? wfirst : T - 1, pos);
    const int64_t whi = wfirst + 31 < T - 1 ? wfirst + 31 : T - 1;
    const int64_t lo = request_start(q0, pos);
    const int64_t hi = q0 + 127 < T - 1 ? q0 + 127 : T - 1;

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

    for (int64_t kb = lo >> 5; kb <= (hi >> 5); ++kb) {
        const int64_t k0 = kb * 32;
        for (int c = tid; c < 32 * (kHeadDim / 8); c += 256) {
            const int r = c >> 4, ch = c & 15;
            const int64_t key = k0 + r;
            uint4 kv = make_uint4(0u, 0u, 0u, 0u), vv = kv;
            if (key < T) {
                kv = *reinterpret_cast<const uint4*>(k + key * ldi + hoff + ch * 8);
                vv = *reinterpret_cast<const uint4*>(v + key * ldi + hoff + ch * 8);
            }
            *reinterpret_cast<uint4*>(k_lds + r * KP + ch * 8) = kv;
            const uint32_t vw[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                vt_lds[(ch * 8 + 2 * e) * VP + r] = (uint16_t)(vw[e] & 0xffffu);
                vt_lds[(ch * 8 + 2 * e + 1) * VP + r] = (uint16_t)(vw[e] >> 16);
            }
        }
        __syncthreads();
        if (wact && k0 <= whi && k0 + 31 >= wlo) {
            f32x16 s;
#pragma unroll
            for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
                const bf16x8 kf =
                    *reinterpret_cast<const bf16x8*>(k_lds + col * KP + ks * 16 + hf * 8);
                s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s, 0, 0, 0);
            }
            // lane holds keys k0 + 8*(r/4) + 4*hf + (r%4) of query t
            float sv[16];
            float mb = -INFINITY;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t key = k0 + 8 * (r >> 2) + 4 * hf + (r & 3);
                const bool ok = tv && key >= start && key <= t;
                sv[r] = ok ? s[r] * kScoreScale : -INFINITY;
                mb = fmaxf(mb, sv[r]);
            }
            mb = fmaxf(mb, __shfl_xor(mb, 32, 64));
            const float mn = fmaxf(m_run, mb);
            const float base = mn == -INFINITY ? 0.0f : mn;
            const float alpha = exp2f(m_run - base);
            m_run = mn;
            l_run *= alpha;
            uint32_t ph[8], pl[8];
#pragma unroll
            for (int r = 0; r < 16; r += 2) {
                const float p0 = exp2f(sv[r] - base), p1 = exp2f(sv[r + 1] - base);
                l_run += p0;
                l_run += p1;
                const uint16_t h0 = f32_to_bf16(p0), h1 = f32_to_bf16(p1);
                const uint16_t e0 = f32_to_bf16(p0 - bf16_lo(h0));
                const uint16_t e1 = f32_to_bf16(p1 - bf16_lo(h1));
                ph[r >> 1] = (uint32_t)h0 | ((uint32_t)h1 << 16);
                pl[r >> 1] = (uint32_t)e0 | ((uint32_t)e1 << 16);
            }
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mt][r] *= alpha;
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                const u32x4 bh = {ph[4 * kk], ph[4 * kk + 1], ph[4 * kk + 2], ph[4 * kk + 3]};
                const u32x4 bl = {pl[4 * kk], pl[4 * kk + 1], pl[4 * kk + 2], pl[4 * kk + 3]};
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    const uint16_t* vr = vt_lds + (mt * 32 + col) * VP + 16 * kk + 4 * hf;
                    const uint2 a0 = *reinterpret_cast<const uint2*>(vr);
                    const uint2 a1 = *reinterpret_cast<const uint2*>(vr + 8);
                    const u32x4 av = {a0.x, a0.y, a1.x, a1.y};
                    acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, av), __builtin_bit_cast(bf16x8, bh), acc[mt],
                        0, 0, 0);
                    acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, av), __builtin_bit_cast(bf16x8, bl), acc[mt],
                        0, 0, 0);
                }
            }
        }
        __syncthreads();
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

hipError_t launch_embed(int64_t T, int64_t D, int32_t R, int64_t V, const int32_t* tokens,
                        const int32_t* ro, const void* emb, float* x, int32_t* pos,
                        int32_t* offs, hipStream_t s) {
    k_embed<<<grid_of(T * (D / 8), 1 << 16), 256, 0, s>>>(
        T, D, R, V, tokens, ro, reinterpret_cast<const uint16_t*>(emb), x, pos, offs);
    return hipGetLastError();
}

hipError_t launch_positions(int64_t T, int32_t R, const int32_t* ro, int32_t* pos,
                            hipStream_t s) {
    k_positions<<<grid_of(T, 1 << 16), 256, 0, s>>>(T, R, ro, pos);
    return hipGetLastError();
}

hipError_t launch_rope(int64_t T, int NH, const int32_t* pos, void* x, int64_t ld,
                       hipStream_t s) {
    k_rope<<<(unsigned)ceil_div(T * 64, 256), 256, 0, s>>>(T, NH, pos,
                                                          reinterpret_cast<uint16_t*>(x), ld);
    return hipGetLastError();
}

hipError_t launch_attention(int64_t T, int H, const int32_t* pos, const void* q, const void* k,
                            const void* v, int64_t ldi, void* o, int64_t ldo, hipStream_t s) {
    const dim3 grid((unsigned)ceil_div(T, 128), (unsigned)H);
    k_attention_causal<<<grid, 256, 0, s>>>(
        T, pos, reinterpret_cast<const uint16_t*>(q), reinterpret_cast<const uint16_t*>(k),
        reinterpret_cast<const uint16_t*>(v), ldi, reinterpret_cast<uint16_t*>(o), ldo);
    return hipGetLastError();
}

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
    if (!pos || !x) return README_ERR_ARG;
    return st_of(launch_rope(T, H, pos, x, ld, as_stream(stream)));
}

readme_status readme_attention_causal(int64_t T, int32_t H, const int32_t* pos, const void* q,
                                      const void* k, const void* v, int64_t ld_in, void* o,
                                      int64_t ld_out, void* stream) {
    if (T < 0 || H < 0) return README_ERR_ARG;
    if (ld_in < (int64_t)H * kHeadDim || ld_out < (int64_t)H * kHeadDim) return README_ERR_ARG;
    if (T > INT32_MAX || H > 65535) return README_ERR_UNSUPPORTED;
    if (T == 0 || H == 0) return README_OK;
    if (!pos || !q || !k || !v || !o) return README_ERR_ARG;
    if (!al16(q) || !al16(k) || !al16(v) || !al16(o) || ld_in % 8 || ld_out % 8)
        return README_ERR_ARG;
    return st_of(launch_attention(T, H, pos, q, k, v, ld_in, o, ld_out, as_stream(stream)));
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

    hipError_t e = launch_embed(T, D, R, V, tokens, req_offsets, emb, x, pos, offs, s);
    if (e == hipSuccess) e = launch_rms_to_bf16(T, D, x, offs, 1, rms_eps, a, s);
    if (e == hipSuccess)
        e = launch_grouped_gemm(false, EPI_STORE, plain_args(a, D, pk, 3 * D, offs, T, qkv, 3 * D),
                                s);
    if (e == hipSuccess) e = launch_rope(T, 2 * H, pos, qkv, 3 * D, s);
    if (e == hipSuccess)
        e = launch_attention(T, H, pos, qkv, qkv + D, qkv + 2 * D, 3 * D, o, D, s);
    if (e == hipSuccess)
        e = launch_grouped_gemm(false, EPI_RESID_ADD,
                                plain_args(o, D, pk + 3 * D * D * 2, D, offs, T, x, D), s);
    if (e == hipSuccess) e = launch_rms_to_bf16(T, D, x, offs, 1, rms_eps, m, s);
    const void* mlp = pk + 4 * D * D * 2;
    if (e == hipSuccess) {
        GemmArgs gu = gate_up_args(README_BF16, T, D, 1, F, m, offs, mlp, h);
        gu.m_tiles32 = (int)ceil_div(T, 32);
        e = launch_grouped_gemm(false, EPI_GATE_UP_SILU, gu, s);
    }
    if (e == hipSuccess) {
        GemmArgs dn = down_args(README_BF16, T, D, 1, F, h, offs, mlp, x);
        dn.m_tiles32 = (int)ceil_div(T, 32);
        e = launch_grouped_gemm(false, EPI_RESID_ADD, dn, s);
    }
    if (e == hipSuccess) e = launch_rms_to_bf16(T, D, x, offs, 1, rms_eps, feat, s);
    if (e == hipSuccess)
        e = launch_route(README_BF16, T, D, E, feat, w_router, bias, expert_ids, logits, s);
    return st_of(e);
}

}  // extern "C"
