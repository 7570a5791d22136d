// Internal launchers of libreadme (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "readme.h"

namespace readme {

enum GemmEpilogue { EPI_GATE_UP_SILU = 0, EPI_STORE = 1, EPI_RESID_ADD = 2 };

// C = A * B_e^T on the row block of every expert e (see gemm.hip).
struct GemmArgs {
    const void* A;            // [T][K] grouped rows
    int64_t lda;              // elements
    const void* B;            // expert 0's [N][K]; expert e at + e * b_expert_stride
    int64_t ldb;              // elements
    int64_t b_expert_stride;  // elements
    int64_t N, K;
    const int32_t* offsets;   // [E+1], device
    int E;
    int64_t T;
    void* C;                  // [T][ldc] output
    int64_t ldc;              // elements
    // Optional row maps (fused row moves): A row j is read from A row
    // a_rows[j]; output row j is written to C row c_rows[j].  NULL = identity.
    const int32_t* a_rows;
    const int32_t* c_rows;
    // a_rows_div > 1: a_rows holds (token, slot) pair indices t*div + k of a
    // top-K layer, and the A row is the token, a_rows[j] / div.
    int a_rows_div;
    // Permanent expert (neurons every routed token passes through), stored
    // as slices of one expert's shape at weight indices E, E+1, ...:
    //   shared_groups S > 0 (gate/up): S more row groups after the E experts,
    //     group E+i covering every routed row [0, offsets[E]) with the
    //     weights of index E+i and its output columns shifted right by
    //     (i+1) * shared_col_stride;
    //   k_segs > 1 (down): K is k_segs equal segments; segment 0 multiplies
    //     the expert's own weights, segment s >= 1 those of index E+s-1.
    int shared_groups;
    int64_t shared_col_stride;  // elements
    int k_segs;
    // b_index (device, [E], nullable): expert e's weights are weight index
    // b_index[e] instead of e (a cache of expert slots).
    const int32_t* b_index;
    // m_tiles32 > 0: sum over experts of ceil(rows_e / 32), from token counts
    // the caller knows on the host (the tile choice then sees the split).
    int m_tiles32;
    // tile > 0: this launch's tile configuration (a caller that measured its
    // own shapes); the calling thread's override still takes precedence.
    int tile;
    int n_tiles, m_tiles_max; // filled by the launcher
    // Tiles of several heights in one launch: the block range of class c is
    // [mix_start[c], mix_start[c+1]) (filled by the launcher).
    int mix_start[5];
};

hipError_t launch_route(readme_dtype dt, int64_t T, int64_t d, int E, const void* x,
                        const void* w, const float* bias, int32_t* ids, float* logits,
                        hipStream_t s);
hipError_t launch_group(int64_t T, int E, const int32_t* ids, int32_t* counts, int32_t* offsets,
                        int32_t* perm, int32_t* inv_perm, hipStream_t s);
hipError_t launch_move_rows(int64_t nrows, int64_t row_bytes, const void* src, const int32_t* idx,
                            int64_t src_rows, void* dst, hipStream_t s);
hipError_t launch_pack(readme_dtype dt, int64_t E, int64_t d, int64_t I, const void* wg,
                       const void* wu, const void* wd, void* packed, hipStream_t s);
// Packs n experts into slots e0 .. e0+n-1 of a packed buffer of E_all slots.
// Expert j's gate/up rows at wg/wu + j * I * d (row stride d); its down
// element (c, i) at wd[j * wd_expert_stride + c * wd_row_stride + i].
hipError_t launch_pack_slots(readme_dtype dt, int64_t E_all, int64_t e0, int64_t n, int64_t d,
                             int64_t I, const void* wg, const void* wu, const void* wd,
                             int64_t wd_expert_stride, int64_t wd_row_stride, void* packed,
                             hipStream_t s);
// Rows row0 .. row0+n-1 of a blocked bf16 [N][K] matrix (the packed layout of
// one expert's down block, N a multiple of 32, K of 64) from row-major src.
hipError_t launch_pack_rows_bf16(int64_t N, int64_t K, int64_t row0, int64_t n,
                                 const void* src, int64_t ld, void* packed, hipStream_t s);
hipError_t launch_grouped_gemm(bool f32, int epi, GemmArgs g, hipStream_t s);
// Arguments of the two FFN GEMMs over a packed expert buffer (abi.hip).
GemmArgs gate_up_args(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I,
                      const void* xg, const int32_t* offsets, const void* packed, void* h);
GemmArgs down_args(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I, const void* h,
                   const int32_t* offsets, const void* packed, void* y);
bool set_gemm_tile(int tile);
int get_gemm_tile();
hipError_t launch_topk(int64_t T, int E, int K, const float* logits, int32_t* ids, float* weights,
                       hipStream_t s);
hipError_t launch_gate_weights(int64_t T, int E, const float* logits, const int32_t* ids,
                               const int32_t* inv_perm, float* row_scale, hipStream_t s);
hipError_t launch_scale_rows(bool f32, int64_t nrows, int64_t row_bytes, const void* src,
                             const int32_t* idx, const float* scale, int64_t src_rows, void* dst,
                             hipStream_t s);
hipError_t launch_combine(bool f32, int64_t T, int64_t d, int K, const void* y_pairs,
                          const float* weights, void* y, hipStream_t s);
hipError_t launch_rms_to_bf16(int64_t T, int64_t d, const float* x, const int32_t* offsets, int E,
                              float eps, uint16_t* xn, hipStream_t s);

}  // namespace readme
