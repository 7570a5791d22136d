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
// which lets the row moves around the FFN ride inside the two GEMMs; in a
// top-K layer the gather map holds (token, slot) pairs and the A row is the
// pair's token.
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
//   B (packed weights): stored in blocks of 32 rows x 128 bytes, each block
//     as its four operand fragments of 1 KB (pack.hip), so each DMA
//     instruction copies one contiguous KB, the fragment reads are
//     conflict-free (lane l reads slot l), and a workgroup streams each
//     weight row group as one sequential run, 4 KB per K-step.
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
#pragma once

#include <type_traits>

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

// Instruction schedule of one K-step's fragment reads and MFMAs.  Left to
// itself the scheduler reuses one set of fragment registers and waits on
// every LDS read right before the MFMAs that need it; these group barriers
// instead spread the reads of fragment k+1 across the MFMAs of fragment k,
// so LDS latency hides behind matrix work.  NM MFMAs and NR LDS reads per
// fragment, KK fragments per K-step.
template <int NM, int NR, int M>
__device__ __forceinline__ void sched_spread() {
    if constexpr (M < NM) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        constexpr int r = (M + 1) * NR / NM - M * NR / NM;
        if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);  // LDS reads
        sched_spread<NM, NR, M + 1>();
    }
}

template <int NM, int NR, int KK>
__device__ __forceinline__ void sched_kstep() {
    __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);  // fragment 0
#pragma unroll
    for (int kk = 0; kk + 1 < KK; ++kk) sched_spread<NM, NR, 0>();
    __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);  // last fragment
}

// Calls f(integral_constant<I>) for I = B .. E-1 (compile-time unrolling).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// Schedule of a register-streamed K-step: like sched_kstep, plus NV global
// loads (the refill of the registers the fragment's MFMAs just read) after
// each fragment's MFMAs.
template <int NM, int NR, int NV, int KK>
__device__ __forceinline__ void sched_bd_step() {
    __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);  // fragment 0
#pragma unroll
    for (int kk = 0; kk + 1 < KK; ++kk) {
        sched_spread<NM, NR, 0>();
        __builtin_amdgcn_sched_group_barrier(0x020, NV, 0);  // VMEM reads
    }
    __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);  // last fragment
    __builtin_amdgcn_sched_group_barrier(0x020, NV, 0);
}

constexpr int GROUP_M = 8;
constexpr int CPR = 8;  // 16-byte chunks per row per K-step (128 bytes)

// Position of this workgroup's output tile.
struct TileLoc {
    int e, n_tile, rows;
    int64_t m0, m_end;
    int64_t m_start;  // first grouped row of expert e
    int mt_base;      // M tiles of size BMG (locate_tile) of experts before e
};

// Rows [s, en) of row group ee, offsets clamped to [0, T] (a corrupt offsets
// array cannot make a tile leave the rows); returns its M tiles of size BM.
// Groups 0 .. E-1 are the experts; a permanent-expert group (ee >= E) covers
// every routed row.
template <int BM>
__device__ __forceinline__ int expert_rows(const GemmArgs& g, int ee, int& s, int& en) {
    const int i0 = ee < g.E ? ee : g.E - 1;  // one adjacent pair of offsets
    int64_t a = g.offsets[i0], b = g.offsets[i0 + 1];
    if (ee >= g.E) a = 0;
    a = a < 0 ? 0 : (a > g.T ? g.T : a);
    b = b < a ? a : (b > g.T ? g.T : b);
    s = (int)a;
    en = (int)b;
    return (int)((b - a + BM - 1) / BM);
}

// Row groups: the E experts, then the permanent expert's groups.
__device__ __forceinline__ int row_groups(const GemmArgs& g) { return g.E + g.shared_groups; }

// Number of BM-row tiles over all row groups (times g.n_tiles N tiles), read
// from the device offsets 64 groups at a time; wave-uniform.
template <int BM>
__device__ __forceinline__ int count_tiles(const GemmArgs& g) {
    const int lane = threadIdx.x & 63;
    const int G = row_groups(g);
    int total = 0;
    for (int c0 = 0; c0 < G; c0 += 64) {
        int s = 0, en = 0, tiles = 0;
        if (c0 + lane < G) tiles = expert_rows<BM>(g, c0 + lane, s, en) * g.n_tiles;
        total += __shfl(wave_incl_scan(tiles, lane), 63, 64);
    }
    return __builtin_amdgcn_readfirstlane(total);
}

// Tile number L -> (expert, M tile, N tile).  Tiles are numbered by expert,
// then in groups of GROUP_M M tiles with the N tile outer and the M tile
// inner (so neighbouring tiles share activation rows or weight rows).  Also
// returns in t.mt_base the number of BMG-row tiles of the experts before e.
template <int BM, int BMG>
__device__ __forceinline__ bool locate_tile(const GemmArgs& g, int L, TileLoc& t) {
    const int lane = threadIdx.x & 63;
    const int nt_n = g.n_tiles;
    const int G = row_groups(g);
    int base = 0, gbase = 0;
    for (int c0 = 0; c0 < G; c0 += 64) {
        int s = 0, en = 0, mt_e = 0, mg_e = 0;
        if (c0 + lane < G) {
            mt_e = expert_rows<BM>(g, c0 + lane, s, en);
            mg_e = (en - s + BMG - 1) / BMG;
        }
        const int incl = wave_incl_scan(mt_e * nt_n, lane) + base;
        const int gincl = wave_incl_scan(mg_e, lane) + gbase;
        const uint64_t hit = __ballot(c0 + lane < G && L < incl);
        if (hit) {
            const int src = __builtin_ctzll(hit);
            const int e_s = __builtin_amdgcn_readfirstlane(__shfl(s, src, 64));
            const int e_en = __builtin_amdgcn_readfirstlane(__shfl(en, src, 64));
            const int e_mt = __builtin_amdgcn_readfirstlane(__shfl(mt_e, src, 64));
            const int e_incl = __builtin_amdgcn_readfirstlane(__shfl(incl, src, 64));
            const int e_gincl = __builtin_amdgcn_readfirstlane(__shfl(gincl, src, 64));
            const int e_mg = __builtin_amdgcn_readfirstlane(__shfl(mg_e, src, 64));
            const int local = L - (e_incl - e_mt * nt_n);
            const int grp = local / (GROUP_M * nt_n);
            const int gm = min(GROUP_M, e_mt - grp * GROUP_M);
            const int within = local - grp * GROUP_M * nt_n;
            t.n_tile = within / gm;
            const int mt = grp * GROUP_M + (within - t.n_tile * gm);
            t.e = c0 + src;
            t.m_start = e_s;
            t.m0 = e_s + (int64_t)mt * BM;
            t.m_end = e_en;
            t.rows = (int)((e_en - t.m0) < BM ? (e_en - t.m0) : BM);
            t.mt_base = e_gincl - e_mg;
            return true;
        }
        base = __shfl(incl, 63, 64);
        gbase = __shfl(gincl, 63, 64);
    }
    return false;
}

// Maps blockIdx.x to its tile; false if past the last tile.  The grid is
// launched for an upper bound of the tile count.  The dispatcher deals
// workgroups to the 8 XCDs round-robin (XCD = blockIdx % 8); tile numbers are
// given out so that each XCD receives one contiguous run of ceil(total/8)
// tiles, which keeps neighbouring tiles in the same L2 and spreads the work
// evenly over all XCDs whatever the bound's slack.
template <int BM>
__device__ __forceinline__ bool find_tile(const GemmArgs& g, TileLoc& t) {
    const int total = count_tiles<BM>(g);
    const int bid = blockIdx.x;
    const int per_xcd = (total + 7) >> 3;
    const int j = bid >> 3;
    if (j >= per_xcd) return false;
    const int L = (bid & 7) * per_xcd + j;
    if (L >= total) return false;
    return locate_tile<BM, BM>(g, L, t);
}

// The arguments one tile works with: a permanent-expert row group writes
// its own block of output columns.
template <typename OT>
__device__ __forceinline__ GemmArgs tile_args(const GemmArgs& g, int e) {
    GemmArgs a = g;
    if (e >= g.E)
        a.C = reinterpret_cast<OT*>(g.C) + (int64_t)(e - g.E + 1) * g.shared_col_stride;
    return a;
}

// Weights of the K-steps of one tile.  The per-lane part of an address (row
// group, fragment, lane) is the same in every K segment; the segment's base
// and the step within it are wave-uniform.  Segment 0 is the tile's own
// weights (index e), segment s >= 1 the permanent slice of index E+s-1.
//
// The packed layout (pack.hip) stores each index's matrix as 4 KB blocks of
// 32 rows x 128 bytes of K, ordered (K block, row group): K block kt of row
// group grp is at at(kt) + grp * 4096, with at(kt) = base + kt * step_bytes
// and step_bytes = (N / 32) * 4096.
struct WeightSteps {
    const char* own;     // index e
    const char* B0;      // index 0
    int64_t estride;     // bytes per weight index
    int64_t step_bytes;  // bytes per 128-byte K block (all row groups of it)
    uint32_t nks;        // K blocks per segment
    uint32_t mult;       // ceil(2^32 / nks) with several segments, else 0
    int E;

    // Segment of K block kt = floor(kt * mult / 2^32), exact for kt and nks
    // below 2^16 (the launcher checks K); 0 throughout with one segment.
    __device__ __forceinline__ const char* at(int kt) const {
        const uint32_t sg = __umulhi((uint32_t)kt, mult);
        const char* base = sg == 0 ? own : B0 + (int64_t)(E + (int)sg - 1) * estride;
        return base + (int64_t)(kt - (int)(sg * nks)) * step_bytes;
    }
};

// SEG: the kernel may run K segments (the down projection of a layer with a
// permanent expert); otherwise the segment is 0 at compile time.
template <bool SEG>
__device__ __forceinline__ WeightSteps weight_steps(const GemmArgs& g, int e, int esz) {
    WeightSteps w;
    const int segs = SEG && g.k_segs > 1 ? g.k_segs : 1;
    w.B0 = reinterpret_cast<const char*>(g.B);
    w.estride = g.b_expert_stride * esz;
    const int we = g.b_index && e < g.E ? g.b_index[e] : e;  // slot of expert e, if cached
    w.own = w.B0 + (int64_t)we * w.estride;
    w.step_bytes = (g.N >> 5) * 4096;
    w.nks = (uint32_t)(g.K * esz / segs / 128);
    w.mult = segs > 1 ? (uint32_t)(((1ull << 32) + w.nks - 1) / w.nks) : 0u;
    w.E = g.E;
    return w;
}

// Residual epilogue (stacked layers, no row maps): the fp32 residual values
// a wave will update are loaded into its accumulators before the K loop, so
// the epilogue does not wait on them and stores the sum.  Each element
// belongs to exactly one workgroup, so nothing else writes it meanwhile.
template <int TM, int TN>
__device__ __forceinline__ void load_residual(const GemmArgs& g, f32x16 (&acc)[TM][TN], int row0,
                                              int64_t col0, int rows, int64_t m0, int lane) {
    const float* res = reinterpret_cast<const float*>(g.C);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int rt = row0 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            const int64_t grow = m0 + (rt < rows ? rt : 0);
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                int64_t c = col0 + j * 32 + (lane & 31);
                c = c < g.N ? c : g.N - 1;
                acc[i][j][r] = res[grow * g.ldc + c];
            }
        }
}

// Epilogue through LDS.  The accumulator layout gives each lane one column
// of 16 rows per 32x32 tile, so storing straight from registers means 2- or
// 4-byte stores scattered over many rows.  Instead the tile goes out in as
// few chunks as the LDS budget allows, CH 32-row sub-tiles per wave row
// (WGM*32*CH rows x all columns): every wave puts its values (converted,
// SiLU*mul applied) into a row-major LDS chunk, then all threads store the
// chunk row by row with 16-byte stores, each output row a contiguous run.
// Row maps, row bounds and column bounds are applied per 16-byte piece (8
// bf16 or 4 fp32 columns; N is a multiple of 64, so a piece is either wholly
// inside or wholly outside).
template <int TM, int TN, int WGM, int WGN, bool F32, int EPI, int BUDGET>
struct Epilogue {
    using OT = std::conditional_t<(F32 || EPI == EPI_RESID_ADD), float, uint16_t>;
    static constexpr int BN = WGN * TN * 32;
    static constexpr int OC = EPI == EPI_GATE_UP_SILU ? BN / 2 : BN;  // output columns
    static constexpr int PAD = 16 / (int)sizeof(OT);                 // 16 B row skew
    static constexpr int LDC = OC + PAD;                             // LDS row pitch
    static constexpr int SUB = WGM * 32 * LDC * (int)sizeof(OT);     // bytes per sub-tile row
    static constexpr int CH = (TM % 4 == 0 && 4 * SUB <= BUDGET) ? 4
                              : (TM % 2 == 0 && 2 * SUB <= BUDGET) ? 2 : 1;
    static constexpr int ROWS = WGM * 32 * CH;                       // rows per chunk
    static constexpr int LDS_BYTES = CH * SUB;
    static constexpr int PER_ROW = OC * (int)sizeof(OT) / 16;        // 16 B pieces per row

    __device__ __forceinline__ static OT cvt(float v) {
        if constexpr (sizeof(OT) == 4)
            return v;
        else
            return f32_to_bf16(v);
    }

    __device__ static void run(const GemmArgs& g, const f32x16 (&acc)[TM][TN], int wm, int wn,
                               int64_t n0, int rows, int64_t m0, const int32_t* crow,
                               void* lds_raw, int tid, int nthreads) {
        OT* L = reinterpret_cast<OT*>(lds_raw);
        const int lane = tid & 63;
        const int64_t oc0 = EPI == EPI_GATE_UP_SILU ? n0 / 2 : n0;  // first output column
        const int64_t n_out = EPI == EPI_GATE_UP_SILU ? g.N / 2 : g.N;
#pragma unroll
        for (int c = 0; c < TM / CH; ++c) {
            __syncthreads();  // LDS free (K loop or previous chunk done)
#pragma unroll
            for (int ii = 0; ii < CH; ++ii) {
                const int i = c * CH + ii;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int lr = wm * 32 * CH + ii * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                    if constexpr (EPI == EPI_GATE_UP_SILU) {
#pragma unroll
                        for (int j = 0; j < TN; j += 2) {
                            const int lc = (wn * TN * 32 + j * 32) / 2 + (lane & 31);
                            L[lr * LDC + lc] = cvt(silu_f32(acc[i][j][r]) * acc[i][j + 1][r]);
                        }
                    } else {
#pragma unroll
                        for (int j = 0; j < TN; ++j) {
                            const int lc = wn * TN * 32 + j * 32 + (lane & 31);
                            L[lr * LDC + lc] = cvt(acc[i][j][r]);
                        }
                    }
                }
            }
            __syncthreads();
            for (int u = tid; u < ROWS * PER_ROW; u += nthreads) {
                const int lr = u / PER_ROW, pc = u - lr * PER_ROW;
                const int w_row = lr / (32 * CH), sub = lr % (32 * CH);
                const int rt = w_row * (TM * 32) + c * CH * 32 + sub;  // tile row
                if (rt >= rows) continue;
                const int64_t grow = g.c_rows ? (int64_t)crow[rt] : m0 + rt;
                if (grow < 0 || grow >= g.T) continue;  // a corrupt map writes nothing
                const int64_t col = oc0 + (int64_t)pc * PAD;
                if (col >= n_out) continue;
                const u32x4 v = *reinterpret_cast<const u32x4*>(L + lr * LDC + pc * PAD);
                *reinterpret_cast<u32x4*>(reinterpret_cast<OT*>(g.C) + grow * g.ldc + col) = v;
            }
        }
    }
};

// Gate/up epilogue when every wave holds a single 32-column group (one
// wave per 32-row weight group): the gate columns of neuron group n are in
// wave 2n, the up columns in wave 2n+1, so the pair meets in LDS.  The
// waves put their fp32 sums into a row-major LDS tile, then all threads form
// h = silu(g) * u for 8 neurons at a time and store whole output rows with
// 16-byte stores (same fp32 arithmetic as Epilogue, so the same bits).  A
// tall tile of many waves goes through LDS CH 32-row blocks at a time.
template <int TM, int NW>
struct EpiloguePairWaves {
    using OT = uint16_t;
    static constexpr int LDF = NW * 32 + 4;                  // fp32 row pitch
    // 32-row blocks staged at once: the most (dividing TM) that fit 72 KB.
    static constexpr int chunk() {
        int c = TM;
        while (c > 1 && (TM % c != 0 || c * 32 * LDF * 4 > 73728)) --c;
        return c;
    }
    static constexpr int CH = chunk();
    static constexpr int LDS_BYTES = CH * 32 * LDF * 4;
    static constexpr int PER_ROW = NW * 2;                   // 8-neuron pieces per row
    static_assert(NW % 2 == 0, "gate and up waves come in pairs");

    __device__ static void run(const GemmArgs& g, const f32x16 (&acc)[TM][1], int wm, int wn,
                               int64_t n0, int rows, int64_t m0, const int32_t* crow,
                               void* lds_raw, int tid, int nthreads) {
        (void)wm;
        float* L = reinterpret_cast<float*>(lds_raw);
        const int lane = tid & 63;
        const int64_t oc0 = n0 / 2, n_out = g.N / 2;
#pragma unroll
        for (int c0 = 0; c0 < TM; c0 += CH) {
            __syncthreads();  // LDS free (K loop or the previous block done)
#pragma unroll
            for (int i = 0; i < CH; ++i)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int lr = i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                    L[lr * LDF + wn * 32 + (lane & 31)] = acc[c0 + i][0][r];
                }
            __syncthreads();
            for (int u = tid; u < CH * 32 * PER_ROW; u += nthreads) {
                const int rl = u / PER_ROW, pc = u - rl * PER_ROW;  // row in the block
                const int rt = c0 * 32 + rl;                        // row in the tile
                if (rt >= rows) continue;
                const int64_t col = oc0 + (int64_t)pc * 8;
                if (col >= n_out) continue;
                const int64_t grow = g.c_rows ? (int64_t)crow[rt] : m0 + rt;
                if (grow < 0 || grow >= g.T) continue;
                const int ng = pc / 4, w0 = (pc % 4) * 8;  // neuron group, first neuron in it
                const float* gt = L + rl * LDF + (2 * ng) * 32 + w0;
                const float* up = L + rl * LDF + (2 * ng + 1) * 32 + w0;
                uint32_t packed[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t lo = f32_to_bf16(silu_f32(gt[2 * k]) * up[2 * k]);
                    const uint32_t hi = f32_to_bf16(silu_f32(gt[2 * k + 1]) * up[2 * k + 1]);
                    packed[k] = lo | (hi << 16);
                }
                const u32x4 v = {packed[0], packed[1], packed[2], packed[3]};
                *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(g.C) + grow * g.ldc + col) =
                    v;
            }
        }
    }
};

template <int BM, int BN, int WGM, int WGN, int NSTAGE, bool F32, int EPI, int KC = CPR>
__global__ __launch_bounds__(WGM* WGN * 64) void k_grouped_gemm(GemmArgs args) {
    constexpr int NW = WGM * WGN;
    constexpr int WM = BM / WGM, WN = BN / WGN;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int EPC = F32 ? 4 : 8;       // elements per chunk
    // KC 16-byte chunks of K per row per step: 8 (128 bytes) or 4 (64 bytes,
    // half-size steps so that twice as many fit in LDS: more bytes in flight
    // for the same ring).  One DMA instruction moves 1 KB = RPI rows.
    static_assert(KC == 8 || KC == 4, "chunks per step");
    constexpr int RPI = 64 / KC;
    constexpr int BK = KC * EPC;           // K elements per step
    constexpr int ESZ = F32 ? 4 : 2;
    constexpr int A_INS = BM / RPI / NW;   // DMA instructions per wave per stage
    constexpr int B_INS = BN / RPI / NW;
    constexpr int LPS = A_INS + B_INS;
    constexpr int STAGE = (BM + BN) * KC;  // u32x4 slots per stage
    static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile");
    static_assert(A_INS * RPI * NW == BM && B_INS * RPI * NW == BN, "DMA split");
    static_assert(EPI != EPI_GATE_UP_SILU || WN % 64 == 0, "gate/up pairs");
    static_assert(NSTAGE >= 2 && LPS * (NSTAGE - 2) < 64, "stages");

    using Epi = Epilogue<TM, TN, WGM, WGN, F32, EPI, (NSTAGE * STAGE * 16 > 73728 ? NSTAGE * STAGE * 16 : 73728)>;
    constexpr int LDS_SLOTS = NSTAGE * STAGE > Epi::LDS_BYTES / 16 ? NSTAGE * STAGE : Epi::LDS_BYTES / 16;
    __shared__ u32x4 lds[LDS_SLOTS];
    __shared__ int32_t crow[BM];  // output row of each tile row (row map)

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // The wave index is uniform across a wave; readfirstlane tells the
    // compiler so, which keeps every wave-level quantity (tile offsets, LDS
    // bases of the DMA, loop conditions) in scalar registers.
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WGN, wn = wave % WGN;

    TileLoc t;
    if (!find_tile<BM>(args, t)) return;
    const GemmArgs g = tile_args<typename Epi::OT>(args, t.e);
    const int e = t.e;
    const int64_t m0 = t.m0, m_end = t.m_end;
    const int rows = t.rows;
    const int n_tile = t.n_tile;
    const int64_t n0 = (int64_t)n_tile * BN;

    // A sources.  Instruction i of this wave fills tile rows RPI*(wave+NW*i)
    // .. +RPI-1: lane -> row +lane/KC, slot lane%KC, which holds logical chunk
    // swzk(lane%KC, r).  Rows past the expert's block are clamped to its last
    // row (fetched, never stored); with a row map the A row comes from
    // a_rows[row], a valid token row for every row inside the block.
    auto swzk = [](int c, int r) { return KC == 8 ? swz(c, r) : c ^ ((r >> 2) & 3); };
    const int rsub = lane / KC;
    const char* Ab = reinterpret_cast<const char*>(g.A);
    const char* a_src[A_INS];
#pragma unroll
    for (int i = 0; i < A_INS; ++i) {
        const int r = RPI * (wave + NW * i) + rsub;
        int64_t row = m0 + r;
        row = row < m_end ? row : m_end - 1;
        if (g.a_rows) {
            row = g.a_rows[row];
            row = (row >= 0 && row < g.T) ? row : 0;  // a corrupt map stays in bounds
            if (g.a_rows_div > 1) row /= g.a_rows_div;  // pair -> token
        }
        a_src[i] = Ab + row * g.lda * ESZ + swzk(lane % KC, r) * 16;
    }
    // B sources.  A 32-row group's packed weights are 4 KB per 128-byte K
    // block, so a step of the tile copies KC/2 KB of each group's block:
    // KB q of the stage's B region is KB q % (KC/2) of group q / (KC/2)
    // (with half-size steps, of the block's first or second half).  N tiles
    // past the last group reuse it (their columns are never stored).
    const WeightSteps wst = weight_steps<EPI == EPI_STORE>(g, e, ESZ);
    uint32_t b_off[B_INS];
#pragma unroll
    for (int i = 0; i < B_INS; ++i) {
        const int q = wave + NW * i;
        int64_t grp = (n0 >> 5) + q / (KC / 2);
        const int64_t last = (g.N >> 5) - 1;
        grp = grp < last ? grp : last;
        b_off[i] = (uint32_t)(grp * 4096 + (q % (KC / 2)) * 1024 + lane * 16);
    }

    auto issue = [&](int stage, int kt) {
        u32x4* base = lds + stage * STAGE;
        const int64_t aoff = (int64_t)kt * KC * 16;
        const char* bs = KC == 8 ? wst.at(kt) : wst.at(kt >> 1) + (kt & 1) * 2048;
#pragma unroll
        for (int i = 0; i < A_INS; ++i) dma16(a_src[i] + aoff, base + (wave + NW * i) * 64);
#pragma unroll
        for (int i = 0; i < B_INS; ++i) dma16(bs + b_off[i], base + BM * KC + (wave + NW * i) * 64);
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

    if constexpr (EPI == EPI_RESID_ADD)
        load_residual<TM, TN>(g, acc, wm * WM, n0 + wn * WN, rows, m0, lane);

    const int nk = (int)(g.K / BK);
#pragma unroll
    for (int s = 0; s < NSTAGE - 1; ++s)
        if (s < nk) issue(s, s);

    const int frow = lane & 31;   // fragment row within a 32-row tile
    const int fhalf = lane >> 5;  // which chunk of the k-pair
    const int a_row0 = (wm * WM + frow) * KC;
    // B fragments sit in LDS as packed: 32-row group G of the tile at slot
    // BM*KC + 32*KC*G, fragment kk of the step at +64*kk, one slot per lane.
    const int b_frag0 = BM * KC + wn * TN * 32 * KC + lane;

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
            const int ch = swzk(2 * kk + fhalf, frow);
#pragma unroll
            for (int i = 0; i < TM; ++i) af[buf][i] = S[a_row0 + i * 32 * KC + ch];
#pragma unroll
            for (int j = 0; j < TN; ++j) bfr[buf][j] = S[b_frag0 + j * 32 * KC + kk * 64];
        };
        frag(0, 0);
#pragma unroll
        for (int kk = 0; kk < KC / 2; ++kk) {
            if (kk + 1 < KC / 2) frag((kk + 1) & 1, kk + 1);
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
        sched_kstep<TM * TN * (F32 ? 4 : 1), TM + TN, KC / 2>();
    }

    Epi::run(g, acc, wm, wn, n0, rows, m0, crow, lds, tid, NW * 64);
}

// Variant with the weight operand streamed straight into registers.
//
// The NW waves of a workgroup split the tile along N only: each wave owns
// all BM rows and TN 32-column tiles.  Its weight fragments are exactly the
// packed 1 KB fragments of its own row groups, so it loads them with plain
// coalesced 16-byte-per-lane loads into registers, S K-steps ahead, and no
// LDS space, LDS bandwidth or barrier is spent on the weights.  Compared with
// staging both operands in LDS this removes the LDS write of the weights and
// their fragment reads, which for wave tiles of 64x64 and below made LDS,
// not the matrix cores, the busiest unit of the CU.
//
// The activation rows are shared by all waves: each wave loads its share of
// the next K-steps into registers (also S K-steps ahead), writes K-step kt+1
// into one of two LDS buffers while K-step kt is read from the other, and
// one barrier per K-step separates the two.  All loads are ordinary
// register loads, so the compiler's own wait counting stays exact (it
// cannot follow direct-to-LDS loads as precisely and then drains the
// whole queue).
//
// Step kt (register slot s = kt % S, a compile-time index after unrolling):
//   1. fragments of K-step kt from LDS buffer kt%2, MFMAs with weights bq[s];
//   2. loads of K-step kt+S into slot s (activations and weights);
//   3. K-step kt+1's activation registers -> LDS buffer (kt+1)%2;
//   4. barrier.
// Loads past the last K-step re-read K-step nk-1 (never used): every step
// issues the same loads and the loop needs no conditional loads.
template <int BM, int NW, int TN, int S, bool F32, int EPI>
struct BdTile {
    static constexpr int TM = BM / 32;
    static constexpr int STAGE = BM * CPR;  // u32x4 slots per LDS buffer
    // One 32-column group per wave: gate and up meet across waves.
    using Epi = std::conditional_t<(EPI == EPI_GATE_UP_SILU && TN == 1 && !F32),
                                   EpiloguePairWaves<TM, NW>,
                                   Epilogue<TM, TN, 1, NW, F32, EPI, 73728>>;
    static constexpr int LDS_SLOTS =
        2 * STAGE > Epi::LDS_BYTES / 16 ? 2 * STAGE : Epi::LDS_BYTES / 16;

    // One output tile; lds holds LDS_SLOTS slots, crow BM entries.  Starts
    // and ends with a barrier, so consecutive tiles may reuse both.
    __device__ __forceinline__ static void run(const GemmArgs& g, const TileLoc& t, u32x4* lds,
                                               int32_t* crow) {
    constexpr int WN = TN * 32, BN = NW * WN;
    constexpr int EPC = F32 ? 4 : 8;
    constexpr int BK = CPR * EPC;
    constexpr int ESZ = F32 ? 4 : 2;
    constexpr int A_INS = BM / 8 / NW;    // activation loads per wave per K-step
    static_assert(BM % 32 == 0 && A_INS * 8 * NW == BM, "activation split");
    static_assert(EPI != EPI_GATE_UP_SILU || TN % 2 == 0 || (TN == 1 && NW % 2 == 0 && !F32),
                  "gate/up pairs");
    static_assert(S >= 2, "stages");

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    __syncthreads();  // the previous tile's LDS reads are done

    const int64_t m0 = t.m0, m_end = t.m_end;
    const int rows = t.rows;
    const int64_t n0 = (int64_t)t.n_tile * BN;
    const int64_t col0 = n0 + wave * WN;

    // Weight fragments of this wave: row group (col0/32 + j), clamped to the
    // last group for columns past N (loaded, never stored).
    const int nk = (int)(g.K / BK);
    const WeightSteps wst = weight_steps<EPI == EPI_STORE>(g, t.e, ESZ);
    uint32_t b_off[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
        int64_t grp = (col0 >> 5) + j;
        const int64_t last = (g.N >> 5) - 1;
        grp = grp < last ? grp : last;
        b_off[j] = (uint32_t)(grp * 4096 + lane * 16);
    }

    u32x4 bq[S][TN][CPR / 2];
    auto load_b = [&](auto sc, int kt) {
        constexpr int sl = decltype(sc)::value;
        kt = kt < nk ? kt : nk - 1;
        const char* bs = wst.at(kt);
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < CPR / 2; ++q)
                bq[sl][j][q] = *reinterpret_cast<const u32x4*>(bs + b_off[j] + q * 1024);
    };
    // The weight stream does not depend on the row map: its first K-steps
    // are requested before the row map is read.
    static_for<0, S>([&](auto sc) { load_b(sc, decltype(sc)::value); });

    // Activation sources: load i of this wave covers tile rows 8*(wave+NW*i)
    // .. +7; lane -> row +lane/8 and LDS slot lane%8, which holds logical
    // chunk swz(lane%8, row).  Rows past the expert's block are clamped to its
    // last row (loaded, never stored); with a row map the row comes from
    // a_rows[row], a valid token row for every row inside the block.
    const int rsub = lane >> 3;
    const char* Ab = reinterpret_cast<const char*>(g.A);
    const char* a_src[A_INS];
    int a_dst[A_INS];
#pragma unroll
    for (int i = 0; i < A_INS; ++i) {
        const int r = 8 * (wave + NW * i) + rsub;
        int64_t row = m0 + r;
        row = row < m_end ? row : m_end - 1;
        if (g.a_rows) {
            row = g.a_rows[row];
            row = (row >= 0 && row < g.T) ? row : 0;  // a corrupt map stays in bounds
            if (g.a_rows_div > 1) row /= g.a_rows_div;  // pair -> token
        }
        a_src[i] = Ab + row * g.lda * ESZ + swz(lane & 7, r) * 16;
        a_dst[i] = r * CPR + (lane & 7);
    }
    u32x4 aq[S][A_INS];
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
    if constexpr (EPI == EPI_RESID_ADD) load_residual<TM, TN>(g, acc, 0, col0, rows, m0, lane);

    auto load_a = [&](auto sc, int kt) {
        constexpr int sl = decltype(sc)::value;
        kt = kt < nk ? kt : nk - 1;
#pragma unroll
        for (int i = 0; i < A_INS; ++i)
            aq[sl][i] = *reinterpret_cast<const u32x4*>(a_src[i] + (int64_t)kt * 128);
    };
    auto store_a = [&](auto sc, int buf) {
        constexpr int sl = decltype(sc)::value;
#pragma unroll
        for (int i = 0; i < A_INS; ++i) lds[buf * STAGE + a_dst[i]] = aq[sl][i];
    };

    // Prologue: K-steps 0 .. S-1 in flight, K-step 0 in LDS buffer 0.
    static_for<0, S>([&](auto sc) { load_a(sc, decltype(sc)::value); });
    store_a(std::integral_constant<int, 0>{}, 0);
    __syncthreads();

    const int frow = lane & 31;
    const int fhalf = lane >> 5;
    // Loads of K-step kt+S issued right after the MFMAs that free their
    // registers, spread over the step, so the address unit streams while the
    // matrix cores work instead of taking every load at the end of the step.
    constexpr int KK = CPR / 2;
    // kt is already clamped and bs = wst.at(kt), both once per K-step.
    auto refill = [&](auto sc, const char* bs, int kt, int kk) {
        constexpr int sl = decltype(sc)::value;
#pragma unroll
        for (int j = 0; j < TN; ++j)
            bq[sl][j][kk] = *reinterpret_cast<const u32x4*>(bs + b_off[j] + kk * 1024);
#pragma unroll
        for (int i = kk * A_INS / KK; i < (kk + 1) * A_INS / KK; ++i)
            aq[sl][i] = *reinterpret_cast<const u32x4*>(a_src[i] + (int64_t)kt * 128);
    };
    auto step = [&](auto sc, int kt) {
        constexpr int s = decltype(sc)::value;
        const u32x4* L = lds + (kt & 1) * STAGE;
        const int ktn = kt + S < nk ? kt + S : nk - 1;  // K-step the refills fetch
        const char* bsn = wst.at(ktn);
        u32x4 af[2][TM];
        auto frag = [&](int buf, int kk) {
            const int ch = swz(2 * kk + fhalf, frow);
#pragma unroll
            for (int i = 0; i < TM; ++i) af[buf][i] = L[(i * 32 + frow) * CPR + ch];
        };
        frag(0, 0);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            if (kk + 1 < KK) frag((kk + 1) & 1, kk + 1);
            const int cb = kk & 1;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    if constexpr (F32) {
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                                __uint_as_float(af[cb][i][q]), __uint_as_float(bq[s][j][kk][q]),
                                acc[i][j], 0, 0, 0);
                    } else {
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            __builtin_bit_cast(bf16x8, af[cb][i]),
                            __builtin_bit_cast(bf16x8, bq[s][j][kk]), acc[i][j], 0, 0, 0);
                    }
                }
            refill(sc, bsn, ktn, kk);
        }
        sched_bd_step<TM * TN * (F32 ? 4 : 1), TM, TN + A_INS / KK, KK>();
        store_a(std::integral_constant<int, (s + 1) % S>{}, (kt + 1) & 1);
        __syncthreads();
    };
    int kt0 = 0;
    for (; kt0 + S <= nk; kt0 += S)
        static_for<0, S>([&](auto sc) { step(sc, kt0 + decltype(sc)::value); });
    static_for<0, S - 1>([&](auto sc) {
        if (kt0 + decltype(sc)::value < nk) step(sc, kt0 + decltype(sc)::value);
    });

    Epi::run(g, acc, 0, wave, n0, rows, m0, crow, lds, tid, NW * 64);
    __syncthreads();
    }
};

template <int BM, int NW, int TN, int S, bool F32, int EPI>
__global__ __launch_bounds__(NW * 64) void k_grouped_gemm_bd(GemmArgs g) {
    using Tile = BdTile<BM, NW, TN, S, F32, EPI>;
    __shared__ u32x4 lds[Tile::LDS_SLOTS];
    __shared__ int32_t crow[BM];
    TileLoc t;
    if (!find_tile<BM>(g, t)) return;
    Tile::run(tile_args<typename Tile::Epi::OT>(g, t.e), t, lds, crow);
}

// Upper bound of the M tiles over all row groups: sum_e ceil(T_e / BM) <=
// (T + E*(BM-1)) / BM (and <= T) for the experts, ceil(T / BM) per
// permanent-expert group.
inline int64_t m_tiles_bound(const GemmArgs& g, int BM) {
    int64_t mt = (g.T + (int64_t)g.E * (BM - 1)) / BM;
    if (mt > g.T) mt = g.T;
    return mt + (int64_t)g.shared_groups * ceil_div(g.T, (int64_t)BM);
}

template <int BM, int NW, int TN, int SA, bool F32, int EPI>
inline hipError_t launch_bd(GemmArgs g, hipStream_t s) {
    constexpr int BN = NW * TN * 32;
    g.n_tiles = (int)ceil_div(g.N, BN);
    g.m_tiles_max = (int)m_tiles_bound(g, BM);
    const int64_t blocks = round_up((int64_t)g.n_tiles * g.m_tiles_max, 8);
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    k_grouped_gemm_bd<BM, NW, TN, SA, F32, EPI><<<dim3((unsigned)blocks), dim3(NW * 64), 0, s>>>(g);
    return hipGetLastError();
}

template <int BM, int BN, int WGM, int WGN, int NSTAGE, bool F32, int EPI, int KC = CPR>
inline hipError_t launch_cfg(GemmArgs g, hipStream_t s) {
    g.n_tiles = (int)ceil_div(g.N, BN);
    g.m_tiles_max = (int)m_tiles_bound(g, BM);
    const int64_t blocks = round_up((int64_t)g.n_tiles * g.m_tiles_max, 8);
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    k_grouped_gemm<BM, BN, WGM, WGN, NSTAGE, F32, EPI, KC>
        <<<dim3((unsigned)blocks), dim3(WGM * WGN * 64), 0, s>>>(g);
    return hipGetLastError();
}

// Tile configurations: workgroup tile, wave grid (wave tile), K-steps in
// flight, LDS.  readme_set_gemm_tile() forces one process-wide.
enum TileCfg {
    TILE_AUTO = 0,
    TILE_256x256 = 1,      // 2x4 waves of 128x64, 2 stages, 128 KB
    TILE_256x128 = 2,      // 4x2 waves of  64x64, 3 stages, 144 KB
    TILE_128x128 = 3,      // 2x2 waves of  64x64, 4 stages, 128 KB
    TILE_128x256 = 4,      // 2x4 waves of  64x64, 3 stages, 144 KB
    TILE_64x128 = 5,       // 2x2 waves of  32x64, 4 stages,  96 KB
    TILE_32x128 = 6,       // 1x2 waves of  32x64, 4 stages,  80 KB
    TILE_32x64 = 7,        // 1 wave of 32x64, 6 stages, 72 KB (2 per CU)
    TILE_32x128_S6 = 8,    // 1x2 waves of 32x64, 6 stages, 120 KB
    TILE_256x256_W4 = 9,   // 2x2 waves of 128x128, 2 stages, 128 KB
    TILE_256x128_W4 = 10,  // 2x2 waves of 128x64, 3 stages, 144 KB
    TILE_128x256_W4 = 11,  // 1x4 waves of 128x64, 3 stages, 144 KB
    // Weights streamed into registers (k_grouped_gemm_bd; bf16 only, fp32
    // falls back to TILE_32x128): BM x BN, waves along N, K-steps in flight.
    TILE_BD_128x256 = 12,  // 4 waves of 128x64, 4 K-steps
    TILE_BD_64x256 = 13,   // 4 waves of 64x64, 4 K-steps
    TILE_BD_32x256 = 14,   // 4 waves of 32x64, 4 K-steps
    TILE_BD_32x128 = 15,   // 2 waves of 32x64, 6 K-steps
    TILE_BD_256x256 = 16,  // 4 waves of 256x64, 2 K-steps
    // Both operands in LDS, 64-byte K steps (twice as many steps in flight):
    TILE_256x256_K32 = 17,  // 2x4 waves of 128x64, 4 half steps, 128 KB
    TILE_128x256_K32 = 18,  // 2x4 waves of 64x64, 6 half steps, 144 KB
    TILE_BD_128x256_S5 = 19,  // as 12, 5 K-steps in flight
    TILE_BD_128x256_S6 = 20,  // as 12, 6 K-steps in flight
    TILE_BD_192x256 = 21,     // 4 waves of 192x64, 3 K-steps
    TILE_BD_192x256_S2 = 22,  // 4 waves of 192x64, 2 K-steps
    TILE_BD_32x64 = 23,       // 1 wave of 32x64, 6 K-steps
    // Register-streamed tiles of several heights in one launch (bf16; see
    // gemm_mix.hpp): each expert in full tiles of the first height, its
    // remainder in the smallest class that holds it.
    TILE_MIX_256 = 24,  // 256 (2 K-steps), 128, 64, 32 rows (4 K-steps)
    TILE_MIX_192 = 25,  // 192 (2 K-steps), 128, 64, 32 rows
    TILE_MIX_128 = 26,  // 128, 64, 32 rows (4 K-steps)
    // Register-streamed 32 x 128 with four waves of one 32-column weight
    // group each (gate and up paired across waves in the epilogue):
    TILE_BD_32x128_W4 = 27,     // 6 K-steps in flight
    TILE_BD_32x128_W4_S8 = 28,  // 8 K-steps in flight
    TILE_BD_32x128_W4_S4 = 29,  // 4 K-steps in flight
    // Tiles of several heights in one launch, eight waves (two per SIMD) of
    // one 32-column weight group each (256 columns; gate/up paired across
    // waves):
    TILE_MIX8_256 = 30,  // 256 (2 K-steps), 128, 64 rows (4 K-steps)
    TILE_MIX8_192 = 31,  // 192 (3 K-steps), 128, 64 rows (4 K-steps)
    TILE_LAST = TILE_MIX8_192,
};

// Launches one tile configuration (instantiated per element type and
// epilogue in the gemm_*.hip files, so the heavy kernels compile in parallel).
template <bool F32, int EPI>
hipError_t launch_tile(int tile, GemmArgs g, hipStream_t s) {
    switch (tile) {
        case TILE_256x256: return launch_cfg<256, 256, 2, 4, 2, F32, EPI>(g, s);
        case TILE_256x128: return launch_cfg<256, 128, 4, 2, 3, F32, EPI>(g, s);
        case TILE_128x128: return launch_cfg<128, 128, 2, 2, 4, F32, EPI>(g, s);
        case TILE_128x256: return launch_cfg<128, 256, 2, 4, 3, F32, EPI>(g, s);
        case TILE_64x128: return launch_cfg<64, 128, 2, 2, 4, F32, EPI>(g, s);
        case TILE_32x64: return launch_cfg<32, 64, 1, 1, 6, F32, EPI>(g, s);
        case TILE_32x128_S6: return launch_cfg<32, 128, 1, 2, 6, F32, EPI>(g, s);
        case TILE_256x256_W4: return launch_cfg<256, 256, 2, 2, 2, F32, EPI>(g, s);
        case TILE_256x128_W4: return launch_cfg<256, 128, 2, 2, 3, F32, EPI>(g, s);
        case TILE_128x256_W4: return launch_cfg<128, 256, 1, 4, 3, F32, EPI>(g, s);
        case TILE_256x256_K32: return launch_cfg<256, 256, 2, 4, 4, F32, EPI, 4>(g, s);
        case TILE_128x256_K32: return launch_cfg<128, 256, 2, 4, 6, F32, EPI, 4>(g, s);
        default: break;
    }
    if constexpr (!F32) {
        switch (tile) {
            case TILE_BD_128x256: return launch_bd<128, 4, 2, 4, F32, EPI>(g, s);
            case TILE_BD_64x256: return launch_bd<64, 4, 2, 4, F32, EPI>(g, s);
            case TILE_BD_32x256: return launch_bd<32, 4, 2, 4, F32, EPI>(g, s);
            case TILE_BD_32x128: return launch_bd<32, 2, 2, 6, F32, EPI>(g, s);
            case TILE_BD_256x256: return launch_bd<256, 4, 2, 2, F32, EPI>(g, s);
            case TILE_BD_128x256_S5: return launch_bd<128, 4, 2, 5, F32, EPI>(g, s);
            case TILE_BD_128x256_S6: return launch_bd<128, 4, 2, 6, F32, EPI>(g, s);
            case TILE_BD_192x256: return launch_bd<192, 4, 2, 3, F32, EPI>(g, s);
            case TILE_BD_192x256_S2: return launch_bd<192, 4, 2, 2, F32, EPI>(g, s);
            case TILE_BD_32x64: return launch_bd<32, 1, 2, 6, F32, EPI>(g, s);
            case TILE_BD_32x128_W4: return launch_bd<32, 4, 1, 6, F32, EPI>(g, s);
            case TILE_BD_32x128_W4_S8: return launch_bd<32, 4, 1, 8, F32, EPI>(g, s);
            case TILE_BD_32x128_W4_S4: return launch_bd<32, 4, 1, 4, F32, EPI>(g, s);
            default: break;
        }
    }
    return launch_cfg<32, 128, 1, 2, 4, F32, EPI>(g, s);
}

// Entry points of the per-type/epilogue translation units.
hipError_t launch_tile_f32_gate_up(int tile, GemmArgs g, hipStream_t s);
hipError_t launch_tile_f32_store(int tile, GemmArgs g, hipStream_t s);
hipError_t launch_tile_bf16_gate_up(int tile, GemmArgs g, hipStream_t s);
hipError_t launch_tile_bf16_store(int tile, GemmArgs g, hipStream_t s);
hipError_t launch_tile_bf16_resid(int tile, GemmArgs g, hipStream_t s);

}  // namespace readme
