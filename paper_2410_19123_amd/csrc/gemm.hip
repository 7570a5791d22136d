// Host side of the grouped GEMM: tile choice and dispatch.  The kernels are
// in gemm_kernels.hpp, instantiated in gemm_f32.hip and gemm_bf16_*.hip.
#include <limits.h>

#include "gemm_mix.hpp"

namespace readme {

// Tile override of the calling host thread (0 = automatic): a tuning and
// test knob that affects only launches made from the thread that set it.
static thread_local int t_forced_tile = TILE_AUTO;
static int forced_tile() { return t_forced_tile; }

bool set_gemm_tile(int tile) {
    if (tile < TILE_AUTO || tile > TILE_LAST) return false;
    t_forced_tile = tile;
    return true;
}

int get_gemm_tile() { return t_forced_tile; }

// Tile shape by tokens per expert (the host knows T and E, not the split):
// many rows per expert favour tall tiles (fewer load bytes per flop); few
// rows favour short tiles (no MFMA work on padding rows, more workgroups to
// spread a weight stream over).  From the prefill shapes up, one launch
// mixes tile heights (gemm_mix.hpp): each expert in full tiles of the
// tallest height, its remainder in the shortest tile that holds it, the
// tall tiles dispatched first -- this removes most padding rows and fills
// the last round of the launch with short tiles.  Thresholds come from tile
// sweeps on MI355X over the Llama-7B-shaped layer (top-1, top-2, with a
// permanent expert), the 16-expert prefill and the d = 8192 request batch.
static int tile_by_shape(bool f32, bool gate_up, const GemmArgs& g) {
    const int f = forced_tile();
    if (f > 0) return f;
    if (g.tile > TILE_AUTO && g.tile <= TILE_LAST) return g.tile;
    const int64_t per_expert = g.T / (g.E > 0 ? g.E : 1);
    if (f32) {  // both operands through LDS (the register-streamed kernels are bf16 only)
        if (per_expert >= (gate_up ? 768 : 192)) return TILE_256x256;
        return per_expert >= 96 && !gate_up ? TILE_128x256 : TILE_32x128;
    }
    if (per_expert < 96) {
        // Decode: 32-row tiles, four waves each streaming one 32-row weight
        // group (more independent weight streams per CU than two waves of
        // two groups: decode stack 1.834 -> 1.809 ms).  When the caller's
        // counts show few tiles (tokens concentrated on few experts), 32x64
        // tiles so that twice as many workgroups stream the weights.
        if (g.m_tiles32 > 0 && (int64_t)g.m_tiles32 * ceil_div(g.N, 128) < 128)
            return TILE_BD_32x64;
        return TILE_BD_32x128_W4;
    }
    if (gate_up) {
        // From 768 rows per expert: eight-wave tiles, two waves per SIMD, so
        // one wave's LDS waits and barrier are covered by the other's MFMAs
        // (skewed prefill 237 -> 223 us at 256 rows; request batch at d =
        // 8192 945 -> 905 us at 192 rows, where 256 rows gave 938).
        if (per_expert >= 768) return g.K >= 8192 ? TILE_MIX8_192 : TILE_MIX8_256;
        // 128-row tiles of four waves while their estimated count (half a
        // tile of padding per row group) fits one round on the chip's 256
        // CUs, so that every CU streams (eight waves: 74-76 vs 71 us at the
        // Llama-7B-shaped layer); past that the eight-wave mixed 256-row
        // launch (permanent-expert groups, 401 estimated tiles: 129 -> 120
        // us against the four-wave mixed launch; top-2 pairs: 127 -> 117 us).
        const int64_t groups = g.E + g.shared_groups;
        const int64_t rows = g.T * (1 + g.shared_groups);
        const int64_t est = (rows / 128 + groups / 2) * ceil_div(g.N, 256);
        return est > 256 ? TILE_MIX8_256 : TILE_BD_128x256;
    }
    // Down: eight-wave mixed launches, 256-row tiles from 768 rows per
    // expert (skewed prefill, K = 704: 173 -> 146 us against four-wave
    // 192-row tiles; request batch 493 -> 486 us), 192-row tiles below
    // (default layer 45.4 -> 41.3 us against the four-wave mixed launch).
    return per_expert >= 768 ? TILE_MIX8_256 : TILE_MIX8_192;
}

hipError_t launch_grouped_gemm(bool f32, int epi, GemmArgs g, hipStream_t s) {
    // The kernels address one weight index with 32-bit per-lane offsets and
    // find a K-step's segment by a multiply-high that is exact below 2^16
    // K-steps (K-steps are at least 32 elements).
    if (g.b_expert_stride * (f32 ? 4 : 2) > INT32_MAX) return hipErrorInvalidValue;
    if (g.K >= (int64_t)32 << 16) return hipErrorInvalidValue;
    if (g.k_segs > 1 && epi != EPI_STORE) return hipErrorInvalidValue;  // segments: down only
    const int tile = tile_by_shape(f32, epi == EPI_GATE_UP_SILU, g);
    if (!f32 && is_mix_tile(tile)) {
        if (epi == EPI_GATE_UP_SILU) return launch_mix_bf16_gate_up(tile, g, s);
        if (epi == EPI_RESID_ADD) return launch_mix_bf16_resid(tile, g, s);
        return launch_mix_bf16_store(tile, g, s);
    }
    if (f32) {
        if (epi == EPI_GATE_UP_SILU) return launch_tile_f32_gate_up(tile, g, s);
        return launch_tile_f32_store(tile, g, s);
    }
    if (epi == EPI_GATE_UP_SILU) return launch_tile_bf16_gate_up(tile, g, s);
    if (epi == EPI_RESID_ADD) return launch_tile_bf16_resid(tile, g, s);
    return launch_tile_bf16_store(tile, g, s);
}

}  // namespace readme
