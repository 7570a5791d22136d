// Grouped GEMM with tiles of several row heights in one launch.
//
// With one tile height per launch, every expert's block is cut into tiles of
// that height: an expert whose rows are not a multiple of it runs a last
// tile that is mostly padding, and a small expert costs a whole tile.  Here
// each row group (expert) is cut into full tiles of the largest height B0,
// and its remainder r goes to the class of the smallest height that holds
// it (B1 >= r > B2 -> class 1, and so on); a remainder above B1 takes one
// more B0 tile.  All classes are register-streamed tiles (BdTile) of 256
// output columns with the same waves -- four waves of two 32-column groups,
// or eight waves (two per SIMD) of one group each -- so the launch runs one
// kernel whose workgroups pick their class's tile routine.
//
// Order.  The blocks of class 0 come first, then class 1, and so on, so the
// dispatcher starts the longest tiles first and fills the tail of the launch
// with short ones (largest-first list scheduling).  Inside a class the tiles
// are numbered as in find_tile (experts in order; class 0 in groups of up to
// GROUP_M M tiles with the N tile outer) and each XCD receives a contiguous
// run of them.  The host sizes each class's block range from an upper bound
// of its tile count; blocks past the count found on the device exit at once.
//
// Every class accumulates K in the same order as the single-height kernels
// (a tile's result does not depend on its height), so results are
// bit-identical to any single-height register-streamed launch.
#pragma once

#include "gemm_kernels.hpp"

namespace readme {

template <int B0, int B1, int B2, int B3>
struct MixRows {
    static constexpr int NC = B3 > 0 ? 4 : B2 > 0 ? 3 : B1 > 0 ? 2 : 1;
    static_assert(B0 > B1 && (B1 > B2 || B1 == 0) && (B2 > B3 || B2 == 0) && B3 >= 0,
                  "decreasing heights");

    // Class of a remainder of 0 < r < B0 rows.
    __device__ static __forceinline__ int cls(int r) {
        if (B3 > 0 && r <= B3) return 3;
        if (B2 > 0 && r <= B2) return 2;
        if (B1 > 0 && r <= B1) return 1;
        return 0;
    }

    // M tiles of class c over rows [s, en) of one row group, and the first
    // row they cover.
    __device__ static __forceinline__ int mtiles(int c, int s, int en, int& row0) {
        const int R = en - s;
        const int n0 = R / B0;
        const int r = R - n0 * B0;
        const int rc = r > 0 ? cls(r) : -1;
        if (c == 0) {
            row0 = s;
            return n0 + (rc == 0 ? 1 : 0);
        }
        row0 = s + n0 * B0;
        return rc == c ? 1 : 0;
    }

    __host__ __device__ static constexpr int height(int c) {
        return c == 0 ? B0 : c == 1 ? B1 : c == 2 ? B2 : B3;
    }
};

// Tiles of class c over all row groups (times the N tiles); wave-uniform.
template <class Mix>
__device__ __forceinline__ int mix_count(const GemmArgs& g, int c) {
    const int lane = threadIdx.x & 63;
    const int G = row_groups(g);
    int total = 0;
    for (int c0 = 0; c0 < G; c0 += 64) {
        int tiles = 0;
        if (c0 + lane < G) {
            int s = 0, en = 0, row0 = 0;
            expert_rows<1>(g, c0 + lane, s, en);
            tiles = Mix::mtiles(c, s, en, row0) * g.n_tiles;
        }
        total += __shfl(wave_incl_scan(tiles, lane), 63, 64);
    }
    return __builtin_amdgcn_readfirstlane(total);
}

// Tile number L of class c -> (row group, M tile, N tile).
template <class Mix>
__device__ __forceinline__ bool mix_locate(const GemmArgs& g, int c, int L, TileLoc& t) {
    const int lane = threadIdx.x & 63;
    const int nt_n = g.n_tiles;
    const int G = row_groups(g);
    const int BM = Mix::height(c);
    int base = 0;
    for (int c0 = 0; c0 < G; c0 += 64) {
        int s = 0, en = 0, row0 = 0, mt_e = 0;
        if (c0 + lane < G) {
            expert_rows<1>(g, c0 + lane, s, en);
            mt_e = Mix::mtiles(c, s, en, row0);
        }
        const int incl = wave_incl_scan(mt_e * nt_n, lane) + base;
        const uint64_t hit = __ballot(c0 + lane < G && L < incl);
        if (hit) {
            const int src = __builtin_ctzll(hit);
            const int e_r0 = __builtin_amdgcn_readfirstlane(__shfl(row0, src, 64));
            const int e_en = __builtin_amdgcn_readfirstlane(__shfl(en, src, 64));
            const int e_mt = __builtin_amdgcn_readfirstlane(__shfl(mt_e, src, 64));
            const int e_incl = __builtin_amdgcn_readfirstlane(__shfl(incl, src, 64));
            const int local = L - (e_incl - e_mt * nt_n);
            const int grp = local / (GROUP_M * nt_n);
            const int gm = min(GROUP_M, e_mt - grp * GROUP_M);
            const int within = local - grp * GROUP_M * nt_n;
            t.n_tile = within / gm;
            const int mt = grp * GROUP_M + (within - t.n_tile * gm);
            t.e = c0 + src;
            t.m_start = e_r0;
            t.m0 = e_r0 + (int64_t)mt * BM;
            t.m_end = e_en;
            t.rows = (int)((e_en - t.m0) < BM ? (e_en - t.m0) : BM);
            t.mt_base = 0;
            return true;
        }
        base = __shfl(incl, 63, 64);
    }
    return false;
}

// NW waves of TN 32-column groups each (NW * TN = 8: 256 columns).
template <int B0, int B1, int B2, int B3, int S0, int S1, int S2, int S3, int EPI, int NW,
          int TN>
struct MixKernel {
    static_assert(NW * TN == 8, "256 output columns per tile");
    using Mix = MixRows<B0, B1, B2, B3>;
    // Classes that are absent reuse class 0's routine type (never run).
    using T0 = BdTile<B0, NW, TN, S0, false, EPI>;
    using T1 = BdTile<(B1 > 0 ? B1 : B0), NW, TN, (B1 > 0 ? S1 : S0), false, EPI>;
    using T2 = BdTile<(B2 > 0 ? B2 : B0), NW, TN, (B2 > 0 ? S2 : S0), false, EPI>;
    using T3 = BdTile<(B3 > 0 ? B3 : B0), NW, TN, (B3 > 0 ? S3 : S0), false, EPI>;
    static constexpr int cmax(int a, int b) { return a > b ? a : b; }
    static constexpr int SLOTS =
        cmax(cmax(T0::LDS_SLOTS, T1::LDS_SLOTS), cmax(T2::LDS_SLOTS, T3::LDS_SLOTS));
};

// Eight-wave tiles are compiled for two waves per SIMD (at most 256
// registers per lane, accumulators included).
template <int B0, int B1, int B2, int B3, int S0, int S1, int S2, int S3, int EPI, int NW,
          int TN>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(NW > 4 ? 2 : 1)))
void k_grouped_gemm_mix(GemmArgs g) {
    using K = MixKernel<B0, B1, B2, B3, S0, S1, S2, S3, EPI, NW, TN>;
    using Mix = typename K::Mix;
    __shared__ u32x4 lds[K::SLOTS];
    __shared__ int32_t crow[B0];
    const int bid = blockIdx.x;
    int c = 0;
    while (c + 1 < Mix::NC && bid >= g.mix_start[c + 1]) ++c;
    const int local = bid - g.mix_start[c];
    const int total = mix_count<Mix>(g, c);
    const int per_xcd = (total + 7) >> 3;
    const int j = local >> 3;
    if (j >= per_xcd) return;
    const int L = (local & 7) * per_xcd + j;
    if (L >= total) return;
    TileLoc t;
    if (!mix_locate<Mix>(g, c, L, t)) return;
    using OT = typename K::T0::Epi::OT;
    const GemmArgs a = tile_args<OT>(g, t.e);
    switch (c) {
        case 0: K::T0::run(a, t, lds, crow); break;
        case 1: if constexpr (B1 > 0) K::T1::run(a, t, lds, crow); break;
        case 2: if constexpr (B2 > 0) K::T2::run(a, t, lds, crow); break;
        default: if constexpr (B3 > 0) K::T3::run(a, t, lds, crow); break;
    }
}

// Host: block ranges per class from upper bounds of their tile counts.
template <int B0, int B1, int B2, int B3, int S0, int S1, int S2, int S3, int EPI, int NW,
          int TN>
inline hipError_t launch_mix(GemmArgs g, hipStream_t s) {
    using Mix = MixRows<B0, B1, B2, B3>;
    g.n_tiles = (int)ceil_div(g.N, NW * TN * 32);
    const int64_t groups = (int64_t)g.E + g.shared_groups;
    int64_t start = 0;
    for (int c = 0; c < 4; ++c) {
        g.mix_start[c] = (int)start;
        if (c >= Mix::NC) continue;
        // Class 0: at most ceil(rows / B0) per group; a smaller class: at
        // most one remainder tile per group, and each holds more than the
        // next smaller height's rows.
        int64_t mt = m_tiles_bound(g, B0);
        if (c > 0) {
            const int lower = c + 1 < Mix::NC ? Mix::height(c + 1) : 0;
            const int64_t rows = g.T * (1 + (int64_t)g.shared_groups);
            mt = groups < rows / (lower + 1) ? groups : rows / (lower + 1);
        }
        start += round_up(mt * g.n_tiles, 8);
    }
    g.mix_start[4] = (int)start;
    if (start == 0) return hipSuccess;
    if (start > 0x7fffffffLL) return hipErrorInvalidValue;
    k_grouped_gemm_mix<B0, B1, B2, B3, S0, S1, S2, S3, EPI, NW, TN>
        <<<dim3((unsigned)start), dim3(NW * 64), 0, s>>>(g);
    return hipGetLastError();
}

template <int EPI>
hipError_t launch_mix_tile(int tile, GemmArgs g, hipStream_t s) {
    switch (tile) {
        case TILE_MIX_256: return launch_mix<256, 128, 64, 32, 2, 4, 4, 4, EPI, 4, 2>(g, s);
        case TILE_MIX_192: return launch_mix<192, 128, 64, 32, 2, 4, 4, 4, EPI, 4, 2>(g, s);
        case TILE_MIX_128: return launch_mix<128, 64, 32, 0, 4, 4, 4, 4, EPI, 4, 2>(g, s);
        // Eight waves: a 32-row class would give a wave less than one
        // 8-row activation load, so remainders of up to 64 rows take 64.
        case TILE_MIX8_256: return launch_mix<256, 128, 64, 0, 2, 4, 4, 4, EPI, 8, 1>(g, s);
        case TILE_MIX8_192: return launch_mix<192, 128, 64, 0, 3, 4, 4, 4, EPI, 8, 1>(g, s);
        default: return hipErrorInvalidValue;
    }
}

inline bool is_mix_tile(int tile) {
    return (tile >= TILE_MIX_256 && tile <= TILE_MIX_128) || tile == TILE_MIX8_256 ||
           tile == TILE_MIX8_192;
}

hipError_t launch_mix_bf16_gate_up(int tile, GemmArgs g, hipStream_t s);
hipError_t launch_mix_bf16_store(int tile, GemmArgs g, hipStream_t s);
hipError_t launch_mix_bf16_resid(int tile, GemmArgs g, hipStream_t s);

}  // namespace readme
