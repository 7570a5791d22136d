// C ABI of libreadme: argument checks on the host, then asynchronous
// launches on the caller's stream.  Nothing here reads device memory,
// synchronises, allocates or frees.
#include <limits.h>

#include "common.hpp"
#include "internal.hpp"

using namespace readme;

namespace {

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }
inline bool dtype_ok(readme_dtype dt) { return dt == README_F32 || dt == README_BF16; }
inline bool experts_ok(int32_t E) { return E >= 1 && E <= README_MAX_EXPERTS; }
inline readme_status hip_status(hipError_t e) { return e == hipSuccess ? README_OK : README_ERR_HIP; }
// The kernels move 16-byte vectors: every array they stream must be 16-byte
// aligned (row lengths are checked separately).
inline bool a16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

readme_status check_ffn_shape(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I) {
    if (!dtype_ok(dt) || T < 0 || d <= 0 || I < 1) return README_ERR_ARG;
    if (!experts_ok(E) || d % 64 != 0 || T > INT32_MAX) return README_ERR_UNSUPPORTED;
    return README_OK;
}

}  // namespace

namespace readme {

GemmArgs gate_up_args(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I,
                      const void* xg, const int32_t* offsets, const void* packed, void* h) {
    const int64_t Ip = padded_I(I);
    GemmArgs g{};
    g.A = xg;
    g.lda = d;
    g.B = packed;
    g.ldb = d;
    g.b_expert_stride = 2 * Ip * d;
    g.N = 2 * Ip;
    g.K = d;
    g.offsets = offsets;
    g.E = E;
    g.T = T;
    g.C = h;
    g.ldc = Ip;
    (void)dt;
    return g;
}

GemmArgs down_args(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I, const void* h,
                   const int32_t* offsets, const void* packed, void* y) {
    const int64_t Ip = padded_I(I);
    GemmArgs g{};
    g.A = h;
    g.lda = Ip;
    g.B = reinterpret_cast<const char*>(packed) + packed_gate_up_bytes(dt, E, d, I);
    g.ldb = Ip;
    g.b_expert_stride = d * Ip;
    g.N = d;
    g.K = Ip;
    g.offsets = offsets;
    g.E = E;
    g.T = T;
    g.C = y;
    g.ldc = d;
    return g;
}

// Permanent expert of P neurons, held as P / I slices of one expert's shape.
inline bool permanent_ok(int64_t P, int64_t I) {
    return P >= 0 && I >= 1 && P % I == 0 && P / I <= README_MAX_PERMANENT_SLICES;
}

// The two GEMMs of a layer with a permanent expert of S slices.  h holds
// [T][(1+S)*Ip]: the routed expert's neurons, then each slice's.  Row maps
// as in the fused entry points (NULL = grouped rows in and out).
hipError_t gate_up_permanent(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I,
                             int64_t S, const void* a, const int32_t* a_rows,
                             const int32_t* offsets, const void* packed, void* h, hipStream_t s) {
    GemmArgs gu = gate_up_args(dt, T, d, E, I, a, offsets, packed, h);
    gu.ldc = (1 + S) * padded_I(I);
    gu.shared_groups = (int)S;
    gu.shared_col_stride = padded_I(I);
    gu.a_rows = a_rows;
    return launch_grouped_gemm(dt == README_F32, EPI_GATE_UP_SILU, gu, s);
}

hipError_t down_permanent(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I,
                          int64_t S, const void* h, const int32_t* offsets, const void* packed,
                          void* y, const int32_t* c_rows, hipStream_t s) {
    GemmArgs dn = down_args(dt, T, d, E, I, h, offsets, packed, y);
    dn.B = reinterpret_cast<const char*>(packed) + packed_gate_up_bytes(dt, E + S, d, I);
    dn.lda = (1 + S) * padded_I(I);
    dn.K = (1 + S) * padded_I(I);
    dn.k_segs = (int)(1 + S);
    dn.c_rows = c_rows;
    return launch_grouped_gemm(dt == README_F32, EPI_STORE, dn, s);
}

readme_status ffn_permanent(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I,
                            int64_t S, const void* a, const int32_t* a_rows,
                            const int32_t* offsets, const void* packed, void* y,
                            const int32_t* c_rows, void* h, hipStream_t s) {
    hipError_t err = gate_up_permanent(dt, T, d, E, I, S, a, a_rows, offsets, packed, h, s);
    if (err == hipSuccess) err = down_permanent(dt, T, d, E, I, S, h, offsets, packed, y, c_rows, s);
    return hip_status(err);
}

}  // namespace readme


extern "C" {

const char* readme_status_string(readme_status s) {
    switch (s) {
        case README_OK: return "ok";
        case README_ERR_ARG: return "invalid argument";
        case README_ERR_UNSUPPORTED: return "unsupported size or type";
        case README_ERR_WORKSPACE: return "buffer smaller than required";
        case README_ERR_HIP: return "HIP launch failed";
        default: return "unknown status";
    }
}

int32_t readme_abi_version(void) { return 1; }

int64_t readme_padded_intermediate(int64_t I) { return I < 1 ? 0 : padded_I(I); }

readme_status readme_set_gemm_tile(int32_t tile) {
    return set_gemm_tile(tile) ? README_OK : README_ERR_ARG;
}

int32_t readme_get_gemm_tile(void) { return get_gemm_tile(); }

readme_status readme_route(readme_dtype dt, int64_t T, int64_t d, int32_t E, const void* x,
                           const void* w_router, const float* bias, int32_t* expert_ids,
                           float* logits, void* stream) {
    if (!dtype_ok(dt) || T < 0 || d <= 0) return README_ERR_ARG;
    if (!experts_ok(E) || T > INT32_MAX) return README_ERR_UNSUPPORTED;
    if (d % (dt == README_BF16 ? 8 : 4) != 0) return README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (!x || !w_router || !expert_ids) return README_ERR_ARG;
    if (!a16(x) || !a16(w_router)) return README_ERR_ARG;
    return hip_status(launch_route(dt, T, d, E, x, w_router, bias, expert_ids, logits,
                                   as_stream(stream)));
}

readme_status readme_group_by_expert(int64_t T, int32_t E, const int32_t* expert_ids,
                                     int32_t* counts, int32_t* offsets, int32_t* perm,
                                     int32_t* inv_perm, readme_dtype dt, int64_t d,
                                     const void* x, void* x_grouped, void* stream) {
    if (T < 0) return README_ERR_ARG;
    if (!experts_ok(E) || T > INT32_MAX) return README_ERR_UNSUPPORTED;
    if (!counts || !offsets) return README_ERR_ARG;
    if (T > 0 && (!expert_ids || !perm || !inv_perm)) return README_ERR_ARG;
    const bool gather = x || x_grouped;
    if (gather) {
        if (!x || !x_grouped || !dtype_ok(dt) || d <= 0) return README_ERR_ARG;
        if ((d * (int64_t)dtype_size(dt)) % 16 != 0) return README_ERR_UNSUPPORTED;
        if (!a16(x) || !a16(x_grouped)) return README_ERR_ARG;
    }
    hipStream_t s = as_stream(stream);
    hipError_t err = launch_group(T, E, expert_ids, counts, offsets, perm, inv_perm, s);
    if (err == hipSuccess && gather && T > 0)
        err = launch_move_rows(T, d * (int64_t)dtype_size(dt), x, perm, T, x_grouped, s);
    return hip_status(err);
}

size_t readme_packed_experts_bytes(readme_dtype dt, int32_t E, int64_t d, int64_t I) {
    if (!dtype_ok(dt) || !experts_ok(E) || d <= 0 || I < 1) return 0;
    return packed_bytes(dt, E, d, I);
}

readme_status readme_pack_experts(readme_dtype dt, int32_t E, int64_t d, int64_t I,
                                  const void* w_gate, const void* w_up, const void* w_down,
                                  void* packed, size_t packed_bytes_given, void* stream) {
    readme_status st = check_ffn_shape(dt, 0, d, E, I);
    if (st != README_OK) return st;
    if (!w_gate || !w_up || !w_down || !packed) return README_ERR_ARG;
    if (!a16(packed)) return README_ERR_ARG;
    if (packed_bytes_given < packed_bytes(dt, E, d, I)) return README_ERR_WORKSPACE;
    return hip_status(launch_pack(dt, E, d, I, w_gate, w_up, w_down, packed, as_stream(stream)));
}

size_t readme_moe_ffn_workspace_bytes(readme_dtype dt, int64_t T, int64_t I) {
    if (!dtype_ok(dt) || T < 0 || I < 1) return 0;
    return (size_t)T * padded_I(I) * dtype_size(dt);
}

readme_status readme_moe_gate_up(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I,
                                 const void* x_grouped, const int32_t* offsets,
                                 const void* packed, void* h, void* stream) {
    readme_status st = check_ffn_shape(dt, T, d, E, I);
    if (st != README_OK) return st;
    if (T == 0) return README_OK;
    if (!x_grouped || !offsets || !packed || !h) return README_ERR_ARG;
    if (!a16(x_grouped) || !a16(packed) || !a16(h)) return README_ERR_ARG;
    GemmArgs g = gate_up_args(dt, T, d, E, I, x_grouped, offsets, packed, h);
    return hip_status(
        launch_grouped_gemm(dt == README_F32, EPI_GATE_UP_SILU, g, as_stream(stream)));
}

readme_status readme_moe_down(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I,
                              const void* h, const int32_t* offsets, const void* packed,
                              void* y_grouped, void* stream) {
    readme_status st = check_ffn_shape(dt, T, d, E, I);
    if (st != README_OK) return st;
    if (T == 0) return README_OK;
    if (!h || !offsets || !packed || !y_grouped) return README_ERR_ARG;
    if (!a16(h) || !a16(packed) || !a16(y_grouped)) return README_ERR_ARG;
    GemmArgs g = down_args(dt, T, d, E, I, h, offsets, packed, y_grouped);
    return hip_status(launch_grouped_gemm(dt == README_F32, EPI_STORE, g, as_stream(stream)));
}

readme_status readme_moe_ffn(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I,
                             const void* x_grouped, const int32_t* offsets, const void* packed,
                             void* y_grouped, void* workspace, size_t workspace_bytes,
                             void* stream) {
    readme_status st = check_ffn_shape(dt, T, d, E, I);
    if (st != README_OK) return st;
    if (T == 0) return README_OK;
    if (!x_grouped || !offsets || !packed || !y_grouped || !workspace) return README_ERR_ARG;
    // Every streamed buffer is checked before the first launch, so an error
    // return means nothing was enqueued.
    if (!a16(x_grouped) || !a16(packed) || !a16(y_grouped) || !a16(workspace))
        return README_ERR_ARG;
    if (workspace_bytes < readme_moe_ffn_workspace_bytes(dt, T, I)) return README_ERR_WORKSPACE;
    st = readme_moe_gate_up(dt, T, d, E, I, x_grouped, offsets, packed, workspace, stream);
    if (st != README_OK) return st;
    return readme_moe_down(dt, T, d, E, I, workspace, offsets, packed, y_grouped, stream);
}

readme_status readme_moe_gate_up_gather(readme_dtype dt, int64_t T, int64_t d, int32_t E,
                                        int64_t I, const void* x, const int32_t* perm,
                                        const int32_t* offsets, const void* packed, void* h,
                                        void* stream) {
    readme_status st = check_ffn_shape(dt, T, d, E, I);
    if (st != README_OK) return st;
    if (T == 0) return README_OK;
    if (!x || !perm || !offsets || !packed || !h) return README_ERR_ARG;
    if (!a16(x) || !a16(packed) || !a16(h)) return README_ERR_ARG;
    GemmArgs g = gate_up_args(dt, T, d, E, I, x, offsets, packed, h);
    g.a_rows = perm;  // grouped row j reads token row perm[j]
    return hip_status(
        launch_grouped_gemm(dt == README_F32, EPI_GATE_UP_SILU, g, as_stream(stream)));
}

readme_status readme_moe_down_scatter(readme_dtype dt, int64_t T, int64_t d, int32_t E,
                                      int64_t I, const void* h, const int32_t* perm,
                                      const int32_t* offsets, const void* packed, void* y,
                                      void* stream) {
    readme_status st = check_ffn_shape(dt, T, d, E, I);
    if (st != README_OK) return st;
    if (T == 0) return README_OK;
    if (!h || !perm || !offsets || !packed || !y) return README_ERR_ARG;
    if (!a16(h) || !a16(packed) || !a16(y)) return README_ERR_ARG;
    GemmArgs g = down_args(dt, T, d, E, I, h, offsets, packed, y);
    g.c_rows = perm;  // grouped row j lands in token row perm[j]
    return hip_status(launch_grouped_gemm(dt == README_F32, EPI_STORE, g, as_stream(stream)));
}

readme_status readme_moe_ffn_fused(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I,
                                   const void* x, const int32_t* perm, const int32_t* offsets,
                                   const void* packed, void* y, void* workspace,
                                   size_t workspace_bytes, void* stream) {
    readme_status st = check_ffn_shape(dt, T, d, E, I);
    if (st != README_OK) return st;
    if (T == 0) return README_OK;
    if (!x || !perm || !offsets || !packed || !y || !workspace) return README_ERR_ARG;
    if (!a16(x) || !a16(packed) || !a16(y) || !a16(workspace)) return README_ERR_ARG;
    if (workspace_bytes < readme_moe_ffn_workspace_bytes(dt, T, I)) return README_ERR_WORKSPACE;
    st = readme_moe_gate_up_gather(dt, T, d, E, I, x, perm, offsets, packed, workspace, stream);
    if (st != README_OK) return st;
    return readme_moe_down_scatter(dt, T, d, E, I, workspace, perm, offsets, packed, y, stream);
}

size_t readme_packed_experts_permanent_bytes(readme_dtype dt, int32_t E, int64_t d, int64_t I,
                                             int64_t P) {
    if (!dtype_ok(dt) || !experts_ok(E) || d <= 0 || !permanent_ok(P, I)) return 0;
    return packed_bytes(dt, E + P / I, d, I);
}

readme_status readme_pack_experts_permanent(readme_dtype dt, int32_t E, int64_t d, int64_t I,
                                            int64_t P, const void* w_gate, const void* w_up,
                                            const void* w_down, const void* p_gate,
                                            const void* p_up, const void* p_down, void* packed,
                                            size_t packed_bytes_given, void* stream) {
    readme_status st = check_ffn_shape(dt, 0, d, E, I);
    if (st != README_OK) return st;
    if (!permanent_ok(P, I)) return P < 0 ? README_ERR_ARG : README_ERR_UNSUPPORTED;
    const int64_t S = P / I;
    if (!w_gate || !w_up || !w_down || !packed) return README_ERR_ARG;
    if (S > 0 && (!p_gate || !p_up || !p_down)) return README_ERR_ARG;
    if (!a16(packed)) return README_ERR_ARG;
    if (packed_bytes_given < packed_bytes(dt, E + S, d, I)) return README_ERR_WORKSPACE;
    hipStream_t s = as_stream(stream);
    hipError_t err = launch_pack_slots(dt, E + S, 0, E, d, I, w_gate, w_up, w_down, d * I, I,
                                       packed, s);
    // Slice j of the permanent expert: rows j*I .. of p_gate/p_up, columns
    // j*I .. of p_down (row stride P).
    if (err == hipSuccess && S > 0)
        err = launch_pack_slots(dt, E + S, E, S, d, I, p_gate, p_up, p_down, I, P, packed, s);
    return hip_status(err);
}

size_t readme_moe_ffn_permanent_workspace_bytes(readme_dtype dt, int64_t T, int64_t I,
                                                int64_t P) {
    if (!dtype_ok(dt) || T < 0 || !permanent_ok(P, I)) return 0;
    return (size_t)T * (1 + P / I) * padded_I(I) * dtype_size(dt);
}

readme_status readme_moe_ffn_permanent(readme_dtype dt, int64_t T, int64_t d, int32_t E,
                                       int64_t I, int64_t P, const void* x_grouped,
                                       const int32_t* offsets, const void* packed,
                                       void* y_grouped, void* workspace, size_t workspace_bytes,
                                       void* stream) {
    readme_status st = check_ffn_shape(dt, T, d, E, I);
    if (st != README_OK) return st;
    if (!permanent_ok(P, I)) return P < 0 ? README_ERR_ARG : README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (!x_grouped || !offsets || !packed || !y_grouped || !workspace) return README_ERR_ARG;
    if (!a16(x_grouped) || !a16(packed) || !a16(y_grouped) || !a16(workspace))
        return README_ERR_ARG;
    if (workspace_bytes < readme_moe_ffn_permanent_workspace_bytes(dt, T, I, P))
        return README_ERR_WORKSPACE;
    return ffn_permanent(dt, T, d, E, I, P / I, x_grouped, nullptr, offsets, packed, y_grouped,
                         nullptr, workspace, as_stream(stream));
}

readme_status readme_moe_ffn_permanent_fused(readme_dtype dt, int64_t T, int64_t d, int32_t E,
                                             int64_t I, int64_t P, const void* x,
                                             const int32_t* perm, const int32_t* offsets,
                                             const void* packed, void* y, void* workspace,
                                             size_t workspace_bytes, void* stream) {
    readme_status st = check_ffn_shape(dt, T, d, E, I);
    if (st != README_OK) return st;
    if (!permanent_ok(P, I)) return P < 0 ? README_ERR_ARG : README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (!x || !perm || !offsets || !packed || !y || !workspace) return README_ERR_ARG;
    if (!a16(x) || !a16(packed) || !a16(y) || !a16(workspace)) return README_ERR_ARG;
    if (workspace_bytes < readme_moe_ffn_permanent_workspace_bytes(dt, T, I, P))
        return README_ERR_WORKSPACE;
    return ffn_permanent(dt, T, d, E, I, P / I, x, perm, offsets, packed, y, perm, workspace,
                         as_stream(stream));
}

readme_status readme_moe_gate_up_permanent_gather(readme_dtype dt, int64_t T, int64_t d,
                                                  int32_t E, int64_t I, int64_t P, const void* x,
                                                  const int32_t* perm, const int32_t* offsets,
                                                  const void* packed, void* h, void* stream) {
    readme_status st = check_ffn_shape(dt, T, d, E, I);
    if (st != README_OK) return st;
    if (!permanent_ok(P, I)) return P < 0 ? README_ERR_ARG : README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (!x || !perm || !offsets || !packed || !h) return README_ERR_ARG;
    if (!a16(x) || !a16(packed) || !a16(h)) return README_ERR_ARG;
    return hip_status(gate_up_permanent(dt, T, d, E, I, P / I, x, perm, offsets, packed, h,
                                        as_stream(stream)));
}

readme_status readme_moe_down_permanent_scatter(readme_dtype dt, int64_t T, int64_t d, int32_t E,
                                                int64_t I, int64_t P, const void* h,
                                                const int32_t* perm, const int32_t* offsets,
                                                const void* packed, void* y, void* stream) {
    readme_status st = check_ffn_shape(dt, T, d, E, I);
    if (st != README_OK) return st;
    if (!permanent_ok(P, I)) return P < 0 ? README_ERR_ARG : README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (!h || !perm || !offsets || !packed || !y) return README_ERR_ARG;
    if (!a16(h) || !a16(packed) || !a16(y)) return README_ERR_ARG;
    return hip_status(down_permanent(dt, T, d, E, I, P / I, h, offsets, packed, y, perm,
                                     as_stream(stream)));
}

readme_status readme_topk(int64_t T, int32_t E, int32_t K, const float* logits, int32_t* ids,
                          float* weights, void* stream) {
    if (T < 0 || K < 1 || K > E) return README_ERR_ARG;
    if (!experts_ok(E) || T * K > INT32_MAX) return README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (!logits || !ids || !weights) return README_ERR_ARG;
    return hip_status(launch_topk(T, E, K, logits, ids, weights, as_stream(stream)));
}

readme_status readme_moe_gate_up_gather_topk(readme_dtype dt, int64_t T, int64_t d, int32_t E,
                                             int64_t I, int32_t K, const void* x,
                                             const int32_t* perm, const int32_t* offsets,
                                             const void* packed, void* h, void* stream) {
    if (K < 1 || K > E) return README_ERR_ARG;
    if (T > INT32_MAX / K) return README_ERR_UNSUPPORTED;
    readme_status st = check_ffn_shape(dt, T * K, d, E, I);
    if (st != README_OK) return st;
    if (T == 0) return README_OK;
    if (!x || !perm || !offsets || !packed || !h) return README_ERR_ARG;
    if (!a16(x) || !a16(packed) || !a16(h)) return README_ERR_ARG;
    GemmArgs g = gate_up_args(dt, T * K, d, E, I, x, offsets, packed, h);
    g.a_rows = perm;  // grouped row j is pair perm[j] = t*K + k, activation row t
    g.a_rows_div = K;
    return hip_status(
        launch_grouped_gemm(dt == README_F32, EPI_GATE_UP_SILU, g, as_stream(stream)));
}

readme_status readme_moe_ffn_topk(readme_dtype dt, int64_t T, int64_t d, int32_t E, int64_t I,
                                  int32_t K, const void* x, const int32_t* perm,
                                  const int32_t* offsets, const void* packed, void* y_pairs,
                                  void* workspace, size_t workspace_bytes, void* stream) {
    if (K < 1 || K > E) return README_ERR_ARG;
    if (T > INT32_MAX / K) return README_ERR_UNSUPPORTED;
    readme_status st = check_ffn_shape(dt, T * K, d, E, I);
    if (st != README_OK) return st;
    if (T == 0) return README_OK;
    if (!x || !perm || !offsets || !packed || !y_pairs || !workspace) return README_ERR_ARG;
    if (!a16(x) || !a16(packed) || !a16(y_pairs) || !a16(workspace)) return README_ERR_ARG;
    if (workspace_bytes < readme_moe_ffn_workspace_bytes(dt, T * K, I)) return README_ERR_WORKSPACE;
    st = readme_moe_gate_up_gather_topk(dt, T, d, E, I, K, x, perm, offsets, packed, workspace,
                                        stream);
    if (st != README_OK) return st;
    // Each grouped row's output lands in its pair's row of y_pairs.
    return readme_moe_down_scatter(dt, T * K, d, E, I, workspace, perm, offsets, packed, y_pairs,
                                   stream);
}

readme_status readme_combine_topk(readme_dtype dt, int64_t T, int64_t d, int32_t K,
                                  const void* y_pairs, const float* weights, void* y,
                                  void* stream) {
    if (!dtype_ok(dt) || T < 0 || d <= 0 || K < 1) return README_ERR_ARG;
    if ((d * (int64_t)dtype_size(dt)) % 16 != 0 || K > README_MAX_EXPERTS) return README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (!y_pairs || !weights || !y) return README_ERR_ARG;
    if (!a16(y_pairs) || !a16(y)) return README_ERR_ARG;
    return hip_status(launch_combine(dt == README_F32, T, d, K, y_pairs, weights, y,
                                     as_stream(stream)));
}

readme_status readme_ungroup(readme_dtype dt, int64_t T, int64_t d, const void* y_grouped,
                             const int32_t* inv_perm, void* y, void* stream) {
    if (!dtype_ok(dt) || T < 0 || d <= 0) return README_ERR_ARG;
    if (T > INT32_MAX || (d * (int64_t)dtype_size(dt)) % 16 != 0) return README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (!y_grouped || !inv_perm || !y) return README_ERR_ARG;
    if (!a16(y_grouped) || !a16(y)) return README_ERR_ARG;
    return hip_status(launch_move_rows(T, d * (int64_t)dtype_size(dt), y_grouped, inv_perm, T, y,
                                       as_stream(stream)));
}

readme_status readme_gate_weights(int64_t T, int32_t E, const float* logits,
                                  const int32_t* expert_ids, const int32_t* inv_perm,
                                  float* row_scale, void* stream) {
    if (T < 0) return README_ERR_ARG;
    if (!experts_ok(E) || T > INT32_MAX) return README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (!logits || !expert_ids || !inv_perm || !row_scale) return README_ERR_ARG;
    return hip_status(
        launch_gate_weights(T, E, logits, expert_ids, inv_perm, row_scale, as_stream(stream)));
}

readme_status readme_ungroup_scaled(readme_dtype dt, int64_t T, int64_t d, const void* y_grouped,
                                    const int32_t* inv_perm, const float* row_scale, void* y,
                                    void* stream) {
    if (!dtype_ok(dt) || T < 0 || d <= 0) return README_ERR_ARG;
    if (T > INT32_MAX || (d * (int64_t)dtype_size(dt)) % 16 != 0) return README_ERR_UNSUPPORTED;
    if (T == 0) return README_OK;
    if (!y_grouped || !inv_perm || !row_scale || !y) return README_ERR_ARG;
    if (!a16(y_grouped) || !a16(y)) return README_ERR_ARG;
    return hip_status(launch_scale_rows(dt == README_F32, T, d * (int64_t)dtype_size(dt),
                                        y_grouped, inv_perm, row_scale, T, y, as_stream(stream)));
}

size_t readme_moe_ffn_stack_workspace_bytes(int64_t T, int64_t d, int64_t I) {
    if (T < 0 || d <= 0 || I < 1) return 0;
    return (size_t)T * d * 2 + (size_t)T * padded_I(I) * 2;
}

namespace {

readme_status stack_impl(int64_t T, int64_t d, int32_t E, int64_t I, int32_t L,
                         const void* const* packed_per_layer, const int32_t* offsets,
                         const int32_t* counts, float* x_resid_grouped, float rms_eps,
                         void* workspace, size_t workspace_bytes, void* stream) {
    readme_status st = check_ffn_shape(README_BF16, T, d, E, I);
    if (st != README_OK) return st;
    if (L < 0 || !(rms_eps >= 0.0f)) return README_ERR_ARG;
    if (T == 0 || L == 0) return README_OK;
    if (!packed_per_layer || !offsets || !x_resid_grouped || !workspace) return README_ERR_ARG;
    if (!a16(x_resid_grouped) || !a16(workspace)) return README_ERR_ARG;
    for (int32_t l = 0; l < L; ++l)
        if (!packed_per_layer[l] || !a16(packed_per_layer[l])) return README_ERR_ARG;
    if (workspace_bytes < readme_moe_ffn_stack_workspace_bytes(T, d, I))
        return README_ERR_WORKSPACE;
    int m32 = 0;
    if (counts) {
        for (int32_t e = 0; e < E; ++e) {
            if (counts[e] < 0) return README_ERR_ARG;
            m32 += (counts[e] + 31) / 32;
        }
    }
    hipStream_t s = as_stream(stream);
    uint16_t* xn = reinterpret_cast<uint16_t*>(workspace);
    uint16_t* h = xn + T * d;
    for (int32_t l = 0; l < L; ++l) {
        hipError_t err = launch_rms_to_bf16(T, d, x_resid_grouped, offsets, E, rms_eps, xn, s);
        if (err != hipSuccess) return README_ERR_HIP;
        GemmArgs gu = gate_up_args(README_BF16, T, d, E, I, xn, offsets, packed_per_layer[l], h);
        gu.m_tiles32 = m32;
        err = launch_grouped_gemm(false, EPI_GATE_UP_SILU, gu, s);
        if (err != hipSuccess) return README_ERR_HIP;
        GemmArgs dn = down_args(README_BF16, T, d, E, I, h, offsets, packed_per_layer[l],
                                x_resid_grouped);
        dn.m_tiles32 = m32;
        err = launch_grouped_gemm(false, EPI_RESID_ADD, dn, s);
        if (err != hipSuccess) return README_ERR_HIP;
    }
    return README_OK;
}

}  // namespace

readme_status readme_moe_ffn_stack(int64_t T, int64_t d, int32_t E, int64_t I, int32_t L,
                                   const void* const* packed_per_layer, const int32_t* offsets,
                                   float* x_resid_grouped, float rms_eps, void* workspace,
                                   size_t workspace_bytes, void* stream) {
    return stack_impl(T, d, E, I, L, packed_per_layer, offsets, nullptr, x_resid_grouped,
                      rms_eps, workspace, workspace_bytes, stream);
}

readme_status readme_moe_ffn_stack_counts(int64_t T, int64_t d, int32_t E, int64_t I, int32_t L,
                                          const void* const* packed_per_layer,
                                          const int32_t* offsets, const int32_t* counts,
                                          float* x_resid_grouped, float rms_eps, void* workspace,
                                          size_t workspace_bytes, void* stream) {
    if (!counts) return README_ERR_ARG;
    return stack_impl(T, d, E, I, L, packed_per_layer, offsets, counts, x_resid_grouped,
                      rms_eps, workspace, workspace_bytes, stream);
}

}  // extern "C"
