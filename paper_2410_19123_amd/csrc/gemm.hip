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
// Optional row maps gather A rows (a_rows) and scatter output rows (c_rows),
// which lets the row moves around the FFN ride inside the two GEMMs.
//
// Tiling.  A workgroup owns a BM x BN output tile of one expert; each of its
// WGM x WGN waves owns a (BM/WGM) x (BN/WGN) sub-tile made of 32x32 MFMA
// tiles (v_mfma_f32_32x32x16_bf16, or 4 x v_mfma_f32_32x32x2_f32 for fp32;
// both consume one 16-byte fragment per lane and operand, and the two
// operands use the same k order inside a fragment, so the product is exact
// whatever order the unit sums in).
//
// Data movement.  A K-step moves 128 bytes of every A and B row (64 bf16 /
// 32 fp32) from global memory straight into LDS with global_load_lds_dwordx4
// (no VGPR staging); one wave instruction fills 1 KB = 8 rows.  In LDS,
// 16-byte chunk c of tile row r sits in slot r*8 + (c ^ ((r >> 1) & 7)): a
// fragment read serves 16 lanes = 16 consecutive rows per LDS cycle over 64
// four-byte banks, a 128-byte row covers half of them and rows alternate
// halves, so each parity class needs 8 distinct slots -- the XOR gives that
// and the reads are bank-conflict free.
//   A (activations, row-major): each lane fetches the chunk its slot holds,
//     i.e. the swizzle is applied on the global side.
//   B (packed weights): stored already in blocks of 32 rows x 128 bytes in
//     the LDS slot order (see pack.hip), so each DMA instruction copies one
//     contiguous KB and a workgroup streams each weight row group as one
//     sequential run (4 KB per K-step), which keeps DRAM pages open.
// NSTAGE K-steps are in flight: at step kt the workgroup waits for stage kt
// (s_waitcnt vmcnt counts this wave's later stages), meets at one barrier,
// refills the buffer freed by step kt-1 with step kt+NSTAGE-1, then runs
// step kt's MFMAs with fragments double-buffered in registers.  The barrier
// is a bare s_barrier: the DMA completion is covered by the explicit vmcnt
// wait, so the compiler's conservative full wait is not needed.
//
// Scheduling.  The number of M tiles per expert is only known on the device,
// so the grid is launched for an upper bound, sum_e ceil(T_e/BM) <=
// (T + E*(BM-1)) / BM, times the N tiles, and each workgroup finds its tile
// by scanning the device offsets; workgroups past the last tile exit at
// once.  Workgroups are dealt to the 8 XCDs round-robin by the dispatcher;
// the linear tile index is remapped so that each XCD receives a contiguous
// run of tiles.  Within one expert the run walks groups of up to GROUP_M
// M tiles: for each N tile, the group's M tiles, so that the workgroups an
// XCD runs together share both their activation rows (across N tiles) and
// their weight rows (across the group) in that XCD's L2.
#include "common.hpp"
#include "internal.hpp"

namespace readme {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// One 16-byte global -> LDS transfer per lane; the LDS address is the
// wave-uniform `lds` plus 16 * lane.  (Kept out of lambdas: the host pass of
// a kernel drops its launch stub if a lambda in it names this builtin.)
__device__ __forceinline__ void dma16(const char* gsrc, u32x4* lds) {
    __builtin_amdgcn_global_load_lds(gsrc, (LDS_AS void*)lds, 16, 0, 0);
}

__device__ __forceinline__ void block_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// LDS slot of logical 16-byte chunk c of tile row r (an XOR: its own inverse).
__device__ __forceinline__ int swz(int c, int r) { return c ^ ((r >> 1) & 7); }

constexpr int GROUP_M = 4;
constexpr int CPR = 8;  // 16-byte chunks per row per K-step (128 bytes)

template <int BM, int BN, int WGM, int WGN, int NSTAGE, bool F32, int EPI>
__global__ __launch_bounds__(WGM* WGN * 64) void k_grouped_gemm(GemmArgs g) {
    constexpr int NW = WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int EPC = F32 ? 4 : 8;       // elements per chunk
    constexpr int BK = CPR * EPC;          // K elements per step
    constexpr int ESZ = F32 ? 4 : 2;
    constexpr int A_INS = BM / 8 / NW;     // DMA instructions per wave per stage
    constexpr int B_INS = BN / 8 / NW;
    constexpr int LPS = A_INS + B_INS;
    constexpr int STAGE = (BM + BN) * CPR; // u32x4 slots per stage
    static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile");
    static_assert(A_INS * 8 * NW == BM && B_INS * 8 * NW == BN, "DMA split");
    static_assert(EPI != EPI_GATE_UP_SILU || WN % 64 == 0, "gate/up pairs");
    static_assert(NSTAGE >= 2 && LPS * (NSTAGE - 2) < 64, "stages");

    __shared__ u32x4 lds[NSTAGE * STAGE];
    __shared__ int32_t crow[BM];  // output row of each tile row (row map)

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // The wave index is uniform across a wave; readfirstlane tells the
    // compiler so, which keeps every wave-level quantity (tile offsets, LDS
    // bases of the DMA, loop conditions) in scalar registers.
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WGN, wn = wave % WGN;

    // Linear tile index, remapped so that each XCD gets a contiguous run.
    const int nb = gridDim.x;
    const int bid = blockIdx.x;
    const int L = (bid & 7) * (nb >> 3) + (bid >> 3);

    // Find (expert, M tile, N tile) of L: experts in order, each expert's
    // tiles in groups of GROUP_M M tiles, N tiles outer, M tiles inner.
    int e = -1, n_tile = 0;
    int64_t m0 = 0, m_end = 0;
    int rows = 0;
    {
        int64_t acc = 0, prev = 0;
        const int nt_n = g.n_tiles;
        for (int ee = 0; ee < g.E; ++ee) {
            int64_t s = g.offsets[ee], en = g.offsets[ee + 1];
            s = s < prev ? prev : (s > g.T ? g.T : s);
            en = en < s ? s : (en > g.T ? g.T : en);
            prev = en;
            const int mt_e = (int)((en - s + BM - 1) / BM);
            const int64_t tiles = (int64_t)mt_e * nt_n;
            if (L < acc + tiles) {
                const int local = (int)(L - acc);
                const int grp = local / (GROUP_M * nt_n);
                const int gm = min(GROUP_M, mt_e - grp * GROUP_M);
                const int within = local - grp * GROUP_M * nt_n;
                n_tile = within / gm;
                const int mt = grp * GROUP_M + (within - n_tile * gm);
                e = ee;
                m0 = s + (int64_t)mt * BM;
                m_end = en;
                rows = (int)((en - m0) < BM ? (en - m0) : BM);
                break;
            }
            acc += tiles;
        }
    }
    if (e < 0) return;
    const int64_t n0 = (int64_t)n_tile * BN;

    // A sources.  Instruction i of this wave fills tile rows 8*(wave+NW*i)
    // .. +7: lane -> row +lane/8, slot lane%8, which holds logical chunk
    // swz(lane%8, r).  Rows past the expert's block are clamped to its last
    // row (fetched, never stored); with a row map the A row comes from
    // a_rows[row], a valid token row for every row inside the block.
    const int rsub = lane >> 3;
    const char* Ab = reinterpret_cast<const char*>(g.A);
    const char* a_src[A_INS];
#pragma unroll
    for (int i = 0; i < A_INS; ++i) {
        const int r = 8 * (wave + NW * i) + rsub;
        int64_t row = m0 + r;
        row = row < m_end ? row : m_end - 1;
        if (g.a_rows) {
            row = g.a_rows[row];
            row = (row >= 0 && row < g.T) ? row : 0;  // a corrupt map stays in bounds
        }
        a_src[i] = Ab + row * g.lda * ESZ + swz(lane & 7, r) * 16;
    }
    // B sources: blocked weights, (32-row group, K step) blocks of 4 KB.
    // Instruction i copies tile rows 8*(wave+NW*i) .. +7 = one contiguous KB
    // of their group's block; N tiles past the last group reuse it (their
    // columns are never stored).
    const int64_t ksteps = g.K / BK;
    const char* Bb = reinterpret_cast<const char*>(g.B) + (int64_t)e * g.b_expert_stride * ESZ;
    const char* b_src[B_INS];
#pragma unroll
    for (int i = 0; i < B_INS; ++i) {
        const int r = 8 * (wave + NW * i);
        int64_t grp = (n0 + r) >> 5;
        const int64_t last = (g.N >> 5) - 1;
        grp = grp < last ? grp : last;
        b_src[i] = Bb + (grp * ksteps * 32 + (r & 31)) * 128 + lane * 16;
    }

    auto issue = [&](int stage, int kt) {
        u32x4* base = lds + stage * STAGE;
        const int64_t aoff = (int64_t)kt * 128;
        const int64_t boff = (int64_t)kt * 4096;
#pragma unroll
        for (int i = 0; i < A_INS; ++i) dma16(a_src[i] + aoff, base + 8 * (wave + NW * i) * CPR);
#pragma unroll
        for (int i = 0; i < B_INS; ++i)
            dma16(b_src[i] + boff, base + (BM + 8 * (wave + NW * i)) * CPR);
    };

    // Output rows of this tile, staged once: the epilogue then needs no
    // dependent global load (the first K-step's barrier orders this store
    // before every read).
    if (g.c_rows) {
        for (int r = tid; r < BM; r += NW * 64) {
            int64_t row = m0 + r;
            row = row < m_end ? row : m_end - 1;
            crow[r] = g.c_rows[row];
        }
    }

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    // Residual epilogue: the residual values this wave will update are read
    // now, ahead of the K loop, so the epilogue does not wait on them (each
    // element belongs to exactly one workgroup, so nothing else writes it).
    if constexpr (EPI == EPI_RESID_ADD) {
        const float* res = reinterpret_cast<const float*>(g.C);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rt = wm * WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                const int64_t grow = m0 + (rt < rows ? rt : 0);
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    int64_t c = n0 + wn * WN + j * 32 + (lane & 31);
                    c = c < g.N ? c : g.N - 1;
                    acc[i][j][r] = res[grow * g.ldc + c];
                }
            }
    }

    const int nk = (int)ksteps;
#pragma unroll
    for (int s = 0; s < NSTAGE - 1; ++s)
        if (s < nk) issue(s, s);

    const int frow = lane & 31;   // fragment row within a 32-row tile
    const int fhalf = lane >> 5;  // which chunk of the k-pair
    const int a_row0 = (wm * WM + frow) * CPR;
    const int b_row0 = (BM + wn * WN + frow) * CPR;

    for (int kt = 0; kt < nk; ++kt) {
        if (kt + NSTAGE - 2 < nk)
            wait_vmcnt<LPS * (NSTAGE - 2)>();
        else
            wait_vmcnt<0>();
        block_barrier();
        if (kt + NSTAGE - 1 < nk) issue((kt + NSTAGE - 1) % NSTAGE, kt + NSTAGE - 1);

        const u32x4* S = lds + (kt % NSTAGE) * STAGE;
        u32x4 af[2][TM], bfr[2][TN];
        auto frag = [&](int buf, int kk) {
            const int ch = swz(2 * kk + fhalf, frow);
#pragma unroll
            for (int i = 0; i < TM; ++i) af[buf][i] = S[a_row0 + i * 32 * CPR + ch];
#pragma unroll
            for (int j = 0; j < TN; ++j) bfr[buf][j] = S[b_row0 + j * 32 * CPR + ch];
        };
        frag(0, 0);
#pragma unroll
        for (int kk = 0; kk < CPR / 2; ++kk) {
            if (kk + 1 < CPR / 2) frag((kk + 1) & 1, kk + 1);
            const int cb = kk & 1;
#pragma unroll
            for (int i = 0; i < TM; ++i) {
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    if constexpr (F32) {
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                                __uint_as_float(af[cb][i][q]), __uint_as_float(bfr[cb][j][q]),
                                acc[i][j], 0, 0, 0);
                    } else {
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            __builtin_bit_cast(bf16x8, af[cb][i]),
                            __builtin_bit_cast(bf16x8, bfr[cb][j]), acc[i][j], 0, 0, 0);
                    }
                }
            }
        }
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
            const int64_t grow = g.c_rows ? (int64_t)crow[rt] : m0 + rt;
            if (grow < 0 || grow >= g.T) continue;  // a corrupt map writes nothing
            if constexpr (EPI == EPI_GATE_UP_SILU) {
#pragma unroll
                for (int j = 0; j < TN; j += 2) {
                    const int64_t nb0 = n0 + wn * WN + j * 32;  // gate group start
                    if (nb0 >= g.N) continue;
                    const float h = silu_f32(acc[i][j][r]) * acc[i][j + 1][r];
                    const int64_t hc = nb0 / 2 + col;
                    if constexpr (F32)
                        reinterpret_cast<float*>(g.C)[grow * g.ldc + hc] = h;
                    else
                        reinterpret_cast<uint16_t*>(g.C)[grow * g.ldc + hc] = f32_to_bf16(h);
                }
            } else {
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    if (n0 + wn * WN + j * 32 >= g.N) continue;
                    const int64_t c = n0 + wn * WN + j * 32 + col;
                    const float v = acc[i][j][r];
                    if constexpr (EPI == EPI_RESID_ADD) {
                        // acc started from the residual value: store the sum.
                        reinterpret_cast<float*>(g.C)[grow * g.ldc + c] = v;
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

template <int BM, int BN, int WGM, int WGN, int NSTAGE, bool F32, int EPI>
static hipError_t launch_cfg(GemmArgs g, hipStream_t s) {
    g.n_tiles = (int)ceil_div(g.N, BN);
    int64_t mt = (g.T + (int64_t)g.E * (BM - 1)) / BM;
    if (mt > g.T) mt = g.T;
    g.m_tiles_max = (int)mt;
    const int64_t blocks = round_up((int64_t)g.n_tiles * g.m_tiles_max, 8);
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    k_grouped_gemm<BM, BN, WGM, WGN, NSTAGE, F32, EPI>
        <<<dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, s>>>(g);
    return hipGetLastError();
}

// Tile configurations: workgroup tile, wave grid (wave tile), K-steps in
// flight, LDS.  readme_set_gemm_tile() forces one process-wide.
enum TileCfg {
    TILE_AUTO = 0,
    TILE_256x256 = 1,  // 2x4 waves of 128x64, 2 stages, 128 KB
    TILE_256x128 = 2,  // 4x2 waves of  64x64, 3 stages, 144 KB
    TILE_128x128 = 3,  // 2x2 waves of  64x64, 4 stages, 128 KB
    TILE_128x256 = 4,  // 2x4 waves of  64x64, 3 stages, 144 KB
    TILE_64x128 = 5,   // 2x2 waves of  32x64, 4 stages,  96 KB
    TILE_32x128 = 6,   // 1x2 waves of  32x64, 4 stages,  80 KB (few rows per expert)
    TILE_32x64 = 7,    // 1 wave of 32x64, 6 stages, 72 KB (2 per CU; decode)
    TILE_32x128_S6 = 8,  // 1x2 waves of 32x64, 6 stages, 120 KB (decode)
    TILE_LAST = TILE_32x128_S6,
};

static int g_forced_tile = TILE_AUTO;
static int forced_tile() { return __atomic_load_n(&g_forced_tile, __ATOMIC_RELAXED); }

bool set_gemm_tile(int tile) {
    if (tile < TILE_AUTO || tile > TILE_LAST) return false;
    __atomic_store_n(&g_forced_tile, tile, __ATOMIC_RELAXED);
    return true;
}

template <bool F32, int EPI>
static hipError_t launch_tile(int tile, GemmArgs g, hipStream_t s) {
    switch (tile) {
        case TILE_256x256: return launch_cfg<256, 256, 2, 4, 2, F32, EPI>(g, s);
        case TILE_256x128: return launch_cfg<256, 128, 4, 2, 3, F32, EPI>(g, s);
        case TILE_128x128: return launch_cfg<128, 128, 2, 2, 4, F32, EPI>(g, s);
        case TILE_128x256: return launch_cfg<128, 256, 2, 4, 3, F32, EPI>(g, s);
        case TILE_64x128: return launch_cfg<64, 128, 2, 2, 4, F32, EPI>(g, s);
        case TILE_32x64: return launch_cfg<32, 64, 1, 1, 6, F32, EPI>(g, s);
        case TILE_32x128_S6: return launch_cfg<32, 128, 1, 2, 6, F32, EPI>(g, s);
        default: return launch_cfg<32, 128, 1, 2, 4, F32, EPI>(g, s);
    }
}

// Tile shape by tokens per expert (the host knows T and E, not the split):
// many rows per expert favour large tiles (fewer LDS and L2 bytes per
// flop); few rows favour short tiles (no MFMA work on padding rows, more
// workgroups to spread a weight stream over).  The down projection (N = d)
// has more N tiles than gate/up at these shapes, so it switches to the
// large tile earlier.  Thresholds come from tile sweeps on MI355X.
template <bool F32, int EPI>
static hipError_t launch_by_shape(GemmArgs g, hipStream_t s) {
    const int f = forced_tile();
    if (f > 0) return launch_tile<F32, EPI>(f, g, s);
    const int64_t per_expert = g.T / (g.E > 0 ? g.E : 1);
    const int64_t big = EPI == EPI_GATE_UP_SILU ? 768 : 192;
    if (per_expert >= big) return launch_tile<F32, EPI>(TILE_256x256, g, s);
    if (per_expert >= 96) return launch_tile<F32, EPI>(TILE_128x256, g, s);
    return launch_tile<F32, EPI>(TILE_32x128, g, s);
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
