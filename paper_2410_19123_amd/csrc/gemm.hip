// Ragged grouped GEMM of the expert FFN on CDNA4 matrix cores.
//
// For every expert e, the block of grouped rows [offsets[e], offsets[e+1])
// is multiplied by that expert's weight, C = A * B_e^T, where both operands
// are K-contiguous (A: token rows of length K; B_e: weight rows of length K).
// One kernel serves the three products of the layer (Eq. 2 with the SwiGLU
// expert of Table 1):
//   EPI_GATE_UP_SILU  B_e = packed [W_gate; W_up] rows (32-row groups
//                     alternate), output h = silu(g) * u in registers;
//   EPI_STORE         B_e = W_down, output y;
//   EPI_RESID_ADD     B_e = W_down, fp32 residual += y (stacked layers).
//
// Tiling.  A workgroup owns a BM x BN output tile of one expert; each of its
// WGM x WGN waves owns a (BM/WGM) x (BN/WGN) sub-tile made of 32x32 MFMA
// tiles (v_mfma_f32_32x32x16_bf16, or 4 x v_mfma_f32_32x32x2_f32 for fp32,
// both consuming one 16-byte fragment per lane and operand).  A K-step moves
// 128 bytes of every A and B row through LDS (64 bf16 / 32 fp32), double
// buffered; 16-byte chunks are XOR-swizzled by row (chunk c of row r sits in
// slot c ^ (r & 7)) so that the 32 rows a fragment load touches spread over
// all LDS banks.
//
// Scheduling.  The number of M tiles per expert is only known on the device,
// so the grid is launched for an upper bound, sum_e ceil(T_e/BM) <=
// (T + E*(BM-1)) / BM, and each workgroup finds its expert by scanning the
// device offsets; workgroups past the last tile exit at once.  Workgroups are
// dealt to the 8 XCDs round-robin by the dispatcher; the linear tile index is
// remapped so that each XCD receives a contiguous run of tiles, M fastest:
// the M tiles that share one expert's weight tile run on the same XCD and
// share its L2.
#include "common.hpp"
#include "internal.hpp"

namespace readme {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int BM, int BN, int WGM, int WGN, bool F32, int EPI>
__global__ __launch_bounds__(WGM* WGN * 64) void k_grouped_gemm(GemmArgs g) {
    constexpr int NT = WGM * WGN * 64;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int CPR = 8;                 // 16-byte chunks per row per K-step
    constexpr int EPC = F32 ? 4 : 8;       // elements per chunk
    constexpr int BK = CPR * EPC;          // K elements per step
    constexpr int ESZ = F32 ? 4 : 2;
    constexpr int A_LD = BM * CPR / NT;    // chunk loads per thread
    constexpr int B_LD = BN * CPR / NT;
    static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile");
    static_assert(A_LD * NT == BM * CPR && B_LD * NT == BN * CPR, "load split");
    static_assert(EPI != EPI_GATE_UP_SILU || WN % 64 == 0, "gate/up pairs");

    __shared__ u32x4 lds[2][(BM + BN) * CPR];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;

    // Linear tile index, remapped so that each XCD gets a contiguous run.
    const int nb = gridDim.x;
    const int bid = blockIdx.x;
    const int L = (bid & 7) * (nb >> 3) + (bid >> 3);
    const int n_tile = L / g.m_tiles_max;
    const int mt = L - n_tile * g.m_tiles_max;
    if (n_tile >= g.n_tiles) return;

    int e = -1;
    int64_t m0 = 0;
    int rows = 0;
    {
        int acc = 0;
        int64_t prev = 0;
        for (int ee = 0; ee < g.E; ++ee) {
            int64_t s = g.offsets[ee], en = g.offsets[ee + 1];
            s = s < prev ? prev : (s > g.T ? g.T : s);
            en = en < s ? s : (en > g.T ? g.T : en);
            prev = en;
            const int nt = (int)((en - s + BM - 1) / BM);
            if (mt < acc + nt) {
                e = ee;
                m0 = s + (int64_t)(mt - acc) * BM;
                rows = (int)((en - m0) < BM ? (en - m0) : BM);
                break;
            }
            acc += nt;
        }
    }
    if (e < 0) return;
    const int64_t n0 = (int64_t)n_tile * BN;

    // Global chunk pointers of this thread's loads (row clamped in bounds;
    // rows past the expert's block are loaded and never stored).
    const char* Ab = reinterpret_cast<const char*>(g.A);
    const char* Bb = reinterpret_cast<const char*>(g.B) + (int64_t)e * g.b_expert_stride * ESZ;
    const u32x4* a_src[A_LD];
    const u32x4* b_src[B_LD];
    int a_dst[A_LD], b_dst[B_LD];
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
        const int q = tid + i * NT, r = q / CPR, c = q % CPR;
        int64_t row = m0 + r;
        row = row < g.T ? row : g.T - 1;
        a_src[i] = reinterpret_cast<const u32x4*>(Ab + (row * g.lda) * ESZ) + c;
        a_dst[i] = r * CPR + (c ^ (r & 7));
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
        const int q = tid + i * NT, r = q / CPR, c = q % CPR;
        int64_t row = n0 + r;
        row = row < g.N ? row : g.N - 1;
        b_src[i] = reinterpret_cast<const u32x4*>(Bb + (row * g.ldb) * ESZ) + c;
        b_dst[i] = BM * CPR + r * CPR + (c ^ (r & 7));
    }

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    const int nk = (int)(g.K / BK);
    u32x4 ra[A_LD], rb[B_LD];
#pragma unroll
    for (int i = 0; i < A_LD; ++i) ra[i] = a_src[i][0];
#pragma unroll
    for (int i = 0; i < B_LD; ++i) rb[i] = b_src[i][0];
#pragma unroll
    for (int i = 0; i < A_LD; ++i) lds[0][a_dst[i]] = ra[i];
#pragma unroll
    for (int i = 0; i < B_LD; ++i) lds[0][b_dst[i]] = rb[i];
    __syncthreads();

    const int frow = lane & 31;   // fragment row within a 32-row tile
    const int fhalf = lane >> 5;  // which chunk of the pair
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        const bool more = kt + 1 < nk;
        if (more) {
            const int64_t step = (int64_t)(kt + 1) * CPR;  // in chunks
#pragma unroll
            for (int i = 0; i < A_LD; ++i) ra[i] = a_src[i][step];
#pragma unroll
            for (int i = 0; i < B_LD; ++i) rb[i] = b_src[i][step];
        }
        const u32x4* As = &lds[cur][0];
        const u32x4* Bs = &lds[cur][BM * CPR];
#pragma unroll
        for (int kk = 0; kk < CPR / 2; ++kk) {
            const int ch = (2 * kk + fhalf) ^ (frow & 7);
            u32x4 af[TM], bfr[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) af[i] = As[(wm * WM + i * 32 + frow) * CPR + ch];
#pragma unroll
            for (int j = 0; j < TN; ++j) bfr[j] = Bs[(wn * WN + j * 32 + frow) * CPR + ch];
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    if constexpr (F32) {
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                                __uint_as_float(af[i][q]), __uint_as_float(bfr[j][q]), acc[i][j],
                                0, 0, 0);
                    } else {
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            __builtin_bit_cast(bf16x8, af[i]), __builtin_bit_cast(bf16x8, bfr[j]),
                            acc[i][j], 0, 0, 0);
                    }
                }
        }
        if (more) {
#pragma unroll
            for (int i = 0; i < A_LD; ++i) lds[cur ^ 1][a_dst[i]] = ra[i];
#pragma unroll
            for (int i = 0; i < B_LD; ++i) lds[cur ^ 1][b_dst[i]] = rb[i];
        }
        __syncthreads();
    }

    // Epilogue.  32x32 accumulator layout: register r of lane l holds row
    // 8*(r/4) + 4*(l/32) + r%4, column l%32.
    const int col = lane & 31;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int rt = wm * WM + i * 32 + 8 * (r >> 2) + 4 * fhalf + (r & 3);
            if (rt >= rows) continue;
            const int64_t grow = m0 + rt;
            if constexpr (EPI == EPI_GATE_UP_SILU) {
#pragma unroll
                for (int j = 0; j < TN; j += 2) {
                    const int64_t nb0 = n0 + wn * WN + j * 32;  // gate group start
                    if (nb0 >= g.N) continue;
                    const float gv = acc[i][j][r], uv = acc[i][j + 1][r];
                    const float h = silu_f32(gv) * uv;
                    const int64_t hc = nb0 / 2 + col;
                    if constexpr (F32)
                        reinterpret_cast<float*>(g.C)[grow * g.ldc + hc] = h;
                    else
                        reinterpret_cast<uint16_t*>(g.C)[grow * g.ldc + hc] = f32_to_bf16(h);
                }
            } else {
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const int64_t c = n0 + wn * WN + j * 32 + col;
                    if (n0 + wn * WN + j * 32 >= g.N) continue;
                    const float v = acc[i][j][r];
                    if constexpr (EPI == EPI_RESID_ADD) {
                        float* y = reinterpret_cast<float*>(g.C) + grow * g.ldc + c;
                        *y = *y + v;
                    } else if constexpr (F32) {
                        reinterpret_cast<float*>(g.C)[grow * g.ldc + c] = v;
                    } else {
                        reinterpret_cast<uint16_t*>(g.C)[grow * g.ldc + c] = f32_to_bf16(v);
                    }
                }
            }
        }
    }
}

template <int BM, int BN, int WGM, int WGN, bool F32, int EPI>
static hipError_t launch_cfg(GemmArgs g, hipStream_t s) {
    g.n_tiles = (int)ceil_div(g.N, BN);
    int64_t mt = (g.T + (int64_t)g.E * (BM - 1)) / BM;
    if (mt > g.T) mt = g.T;
    g.m_tiles_max = (int)mt;
    const int64_t blocks = round_up((int64_t)g.n_tiles * g.m_tiles_max, 8);
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    k_grouped_gemm<BM, BN, WGM, WGN, F32, EPI>
        <<<dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, s>>>(g);
    return hipGetLastError();
}

// Tile shape by tokens per expert: many rows per expert favour large tiles
// (fewer LDS and L2 bytes per flop); few rows favour short tiles (no MFMA
// work on padding rows).
template <bool F32, int EPI>
static hipError_t launch_by_shape(GemmArgs g, hipStream_t s) {
    const int64_t per_expert = g.T / (g.E > 0 ? g.E : 1);
    if (!F32 && per_expert >= 768) return launch_cfg<256, 256, 2, 2, F32, EPI>(g, s);
    if (per_expert >= 96) return launch_cfg<128, 128, 2, 2, F32, EPI>(g, s);
    return launch_cfg<32, 128, 1, 2, F32, EPI>(g, s);
}

hipError_t launch_grouped_gemm(bool f32, int epi, GemmArgs g, hipStream_t s) {
    if (f32) {
        if (epi == EPI_GATE_UP_SILU) return launch_by_shape<true, EPI_GATE_UP_SILU>(g, s);
        return launch_by_shape<true, EPI_STORE>(g, s);
    }
    if (epi == EPI_GATE_UP_SILU) return launch_by_shape<false, EPI_GATE_UP_SILU>(g, s);
    if (epi == EPI_RESID_ADD) return launch_by_shape<false, EPI_RESID_ADD>(g, s);
    return launch_by_shape<false, EPI_STORE>(g, s);
}

}  // namespace readme
