// Host side of the grouped GEMM: tile choice and dispatch.  The kernels are
// in gemm_kernels.hpp, instantiated in gemm_f32.hip and gemm_bf16_*.hip.
#include <limits.h>

#include "gemm_kernels.hpp"

namespace readme {

static int g_forced_tile = TILE_AUTO;
static int forced_tile() { return __atomic_load_n(&g_forced_tile, __ATOMIC_RELAXED); }

bool set_gemm_tile(int tile) {
    if (tile < TILE_AUTO || tile > TILE_LAST) return false;
    __atomic_store_n(&g_forced_tile, tile, __ATOMIC_RELAXED);
    return true;
}

// Tile shape by tokens per expert (the host knows T and E, not the split):
// many rows per expert favour large tiles (fewer LDS and L2 bytes per
// flop); few rows favour short tiles (no MFMA work on padding rows, more
// workgroups to spread a weight stream over).  The down projection (N = d)
// has more N tiles than gate/up at these shapes, so it switches to the
// large tile earlier.  Thresholds come from tile sweeps on MI355X.
static int tile_by_shape(bool gate_up, const GemmArgs& g) {
    const int f = forced_tile();
    if (f > 0) return f;
    const int64_t per_expert = g.T / (g.E > 0 ? g.E : 1);
    const int64_t big = gate_up ? 768 : 192;
    if (per_expert >= big) return TILE_256x256;
    if (per_expert >= 96) return gate_up ? TILE_BD_128x256 : TILE_128x256;
    return TILE_BD_32x128;  // fp32 runs TILE_32x128 instead
}

hipError_t launch_grouped_gemm(bool f32, int epi, GemmArgs g, hipStream_t s) {
    // The kernels address one weight index with 32-bit per-lane offsets and
    // find a K-step's segment by a multiply-high that is exact below 2^16
    // K-steps (K-steps are at least 32 elements).
    if (g.b_expert_stride * (f32 ? 4 : 2) > INT32_MAX) return hipErrorInvalidValue;
    if (g.K >= (int64_t)32 << 16) return hipErrorInvalidValue;
    if (g.k_segs > 1 && epi != EPI_STORE) return hipErrorInvalidValue;  // segments: down only
    const int tile = tile_by_shape(epi == EPI_GATE_UP_SILU, g);
    if (f32) {
        if (epi == EPI_GATE_UP_SILU) return launch_tile_f32_gate_up(tile, g, s);
        return launch_tile_f32_store(tile, g, s);
    }
    if (epi == EPI_GATE_UP_SILU) return launch_tile_bf16_gate_up(tile, g, s);
    if (epi == EPI_RESID_ADD) return launch_tile_bf16_resid(tile, g, s);
    return launch_tile_bf16_store(tile, g, s);
}

}  // namespace readme
