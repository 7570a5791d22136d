/*
 * readme.h -- C ABI of libreadme, the MI355X (gfx950) hot path of a
 * pre-gated mixture-of-experts layer (Read-ME, arXiv 2410.19123).
 *
 * The paper replaces per-layer routers with one router evaluated once per
 * token ahead of all layers (Sec. 2.3, Eq. 2): a token's expert index is
 * known before layer 1 and is the same at every layer.  With top-1 routing a
 * layer's output for token t is the FFN of its one expert,
 *     y_t = F_{e_t}(x_t),
 * and tokens can be batched by expert across requests (Sec. 4.2, Alg. 1).
 * Each expert is a slice of a dense FFN's intermediate neurons (Sec. 3), here
 * the SwiGLU FFN of the Llama family (Table 1):
 *     F_e(x) = W_down^e ( silu(W_gate^e x) * (W_up^e x) ).
 *
 * The calls, in path order:
 *     readme_router_tf        the router G: one causal transformer block over
 *                             each request's tokens, then the gate below
 *     readme_route            one top-1 expert id per token (G's final gate)
 *     readme_group_by_expert  histogram, exclusive scan, stable permutation,
 *                             row gather into expert-contiguous order
 *     readme_moe_ffn          every expert's SwiGLU FFN on its token block
 *                             (= readme_moe_gate_up then readme_moe_down)
 *     readme_moe_ffn_fused    gather + FFN + ungroup, row moves fused into
 *                             the two GEMMs
 *     readme_ungroup          rows back to token order
 *     readme_moe_ffn_stack    L stacked pre-norm residual layers in grouped
 *                             order (routing and grouping done once)
 *
 * Conventions for every call:
 *   - Arrays are DEVICE pointers owned by the caller, row-major, contiguous.
 *     The library owns no memory between calls and keeps no state, apart
 *     from the executor objects a caller creates (readme_offload_*) and the
 *     calling thread's tile override (readme_set_gemm_tile).
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Calls only enqueue work on it: they never synchronise, allocate or
 *     free, and they read no device data on the host, so a caller may
 *     capture them in a graph.
 *   - Element type `dt` is README_F32 (fp32 throughout) or README_BF16 (bf16
 *     inputs, weights and outputs, fp32 accumulation).
 *   - The return value is README_OK, or an error found on the host before
 *     anything is enqueued (README_ERR_ARG / _UNSUPPORTED / _WORKSPACE), or
 *     README_ERR_HIP if a launch failed.  On an error nothing was enqueued
 *     unless the code is README_ERR_HIP.
 *   - Outputs must not alias inputs.  Arrays the kernels stream (token rows,
 *     weights, packed experts, workspaces) must be 16-byte aligned; a
 *     misaligned pointer is README_ERR_ARG.
 *   - T = 0 is allowed and enqueues nothing (readme_group_by_expert still
 *     writes zero counts and offsets).
 */
#ifndef README_H
#define README_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t readme_status;
#define README_OK 0
#define README_ERR_ARG 1          /* NULL pointer, negative size, bad value */
#define README_ERR_UNSUPPORTED 2  /* a size or type outside the supported set */
#define README_ERR_WORKSPACE 3    /* a buffer smaller than its stated size */
#define README_ERR_HIP 4          /* the HIP runtime refused a launch */

typedef int32_t readme_dtype;
#define README_F32 0
#define README_BF16 1

#define README_MAX_EXPERTS 256
#define README_MAX_PERMANENT_SLICES 16
/* Size of the fixed device array readme_moe_ffn_fused_noalloc keeps h in. */
#define README_NOALLOC_SCRATCH_BYTES (64ll << 20)

/* Human-readable name of a status code (static storage). */
const char *readme_status_string(readme_status s);

/* Version of this ABI (bumped on any signature or layout change). */
int32_t readme_abi_version(void);

/*
 * readme_route -- the pre-gating router's top-1 choice (Eq. 2 with K = 1).
 *
 *   logit[t][e] = sum_k x[t][k] * w_router[e][k] + bias[e]
 *   expert_ids[t] = the e of largest logit; ties go to the lowest index and
 *                   a NaN logit never wins (strict '>' scan from e = 0).
 *
 * The paper's router is a one-block transformer over the token prefix; this
 * call is its final gate, a linear map d -> E applied to given features.
 * The argmax decides an integer, so the logits are summed in one fixed fp32
 * order, identical on every run and on any GPU: 16-byte chunks of x and
 * w_router (8 bf16 or 4 fp32 values) are dealt round-robin to 64 partial
 * sums (chunk c to partial c mod 64), each partial fuses multiply-adds in
 * ascending k starting from +0, the 64 partials are folded pairwise
 * (p[l] += p[l + off] for off = 32, 16, 8, 4, 2, 1), then the bias is added.
 *
 *   x          [T][d]  dt          token features
 *   w_router   [E][d]  dt          router weight
 *   bias       [E]     fp32        or NULL (no bias)
 *   expert_ids [T]     int32 out
 *   logits     [T][E]  fp32 out    or NULL
 * Requires 1 <= E <= README_MAX_EXPERTS, d > 0, d a multiple of 8 (bf16) or
 * 4 (fp32).
 */
readme_status readme_route(readme_dtype dt, int64_t T, int64_t d, int32_t E,
                           const void *x, const void *w_router,
                           const float *bias, int32_t *expert_ids,
                           float *logits, void *stream);

/*
 * readme_group_by_expert -- batch tokens by expert (the per-expert queues of
 * Alg. 1; the same grouping serves every layer because a token's expert does
 * not change between layers).
 *
 *   counts[e]    number of tokens with id e
 *   offsets[e]   exclusive scan of counts; offsets[E] = routed tokens
 *   perm[j]      token at grouped row j: expert blocks in order, tokens of
 *                one expert in ascending token order (a stable sort)
 *   inv_perm[t]  grouped row of token t
 *   x_grouped[j] = x[perm[j]]   (if x and x_grouped are both non-NULL)
 * An id outside [0, E) routes the token nowhere: it is left out of counts,
 * inv_perm[t] = -1, and rows j >= offsets[E] have perm[j] = -1 and a zero
 * x_grouped row.  Callers detect such ids by offsets[E] < T.
 *
 *   expert_ids [T] int32, counts [E] int32 out, offsets [E+1] int32 out,
 *   perm [T] int32 out, inv_perm [T] int32 out,
 *   x [T][d] dt, x_grouped [T][d] dt out (both NULL: no gather).
 * Requires 1 <= E <= README_MAX_EXPERTS, T < 2^31; with a gather, d > 0 and
 * d * element size a multiple of 16 bytes.
 */
readme_status readme_group_by_expert(int64_t T, int32_t E,
                                     const int32_t *expert_ids,
                                     int32_t *counts, int32_t *offsets,
                                     int32_t *perm, int32_t *inv_perm,
                                     readme_dtype dt, int64_t d,
                                     const void *x, void *x_grouped,
                                     void *stream);

/*
 * Expert weights are taken in their natural layout and repacked once into
 * the layout the FFN kernels stream (gate and up rows interleaved so that
 * one tile produces matching g and u columns, the intermediate width padded
 * with zero neurons to a multiple of 64; zero neurons add exact zeros since
 * silu(0) * 0 = 0).  The packed buffer is opaque; its size is
 * readme_packed_experts_bytes().
 *
 *   w_gate [E][I][d], w_up [E][I][d], w_down [E][d][I]   dt
 *   packed  >= readme_packed_experts_bytes(dt, E, d, I) bytes, out
 * Requires 1 <= E <= README_MAX_EXPERTS, I >= 1, d > 0 a multiple of 64.
 */
size_t readme_packed_experts_bytes(readme_dtype dt, int32_t E, int64_t d,
                                   int64_t I);
readme_status readme_pack_experts(readme_dtype dt, int32_t E, int64_t d,
                                  int64_t I, const void *w_gate,
                                  const void *w_up, const void *w_down,
                                  void *packed, size_t packed_bytes,
                                  void *stream);

/* Padded intermediate width of the packed layout: I rounded up to 64. */
int64_t readme_padded_intermediate(int64_t I);

/*
 * readme_set_gemm_tile -- force one workgroup tile for the grouped GEMMs that
 * the CALLING HOST THREAD launches (thread-local: other threads keep their
 * own setting, 0 at start), for tuning and for testing every configuration.
 *   0 = automatic (by tokens per expert, the default)
 *   both operands staged in LDS:
 *     1 = 256x256, 2 = 256x128, 3 = 128x128, 4 = 128x256, 5 = 64x128,
 *     6 = 32x128, 7 = 32x64 (deep pipeline), 8 = 32x128 (deep pipeline),
 *     9 = 256x256, 10 = 256x128, 11 = 128x256 (four waves, larger wave tiles)
 *     17 = 256x256, 18 = 128x256 (half-size K steps, deeper pipeline)
 *   weights streamed straight into registers (bf16; fp32 runs tile 6):
 *     12 = 128x256, 13 = 64x256, 14 = 32x256, 15 = 32x128 (deep pipeline),
 *     16 = 256x256, 19 = 128x256 (5 stages), 20 = 128x256 (6 stages),
 *     21 = 192x256 (3 stages), 22 = 192x256 (2 stages), 23 = 32x64,
 *     27, 28, 29 = 32x128 of four single-group waves (6, 8, 4 stages)
 *   several tile heights in one launch (bf16; fp32 runs tile 6), each
 *   expert in full tiles of the first height, its remainder in the
 *   shortest that holds it, 256 columns:
 *     24 = 256/128/64/32, 25 = 192/128/64/32, 26 = 128/64/32 (four waves),
 *     30 = 256/128/64, 31 = 192/128/64 (eight waves, two per SIMD)
 *   (rows of tokens x columns of outputs)
 * Results do not depend on the tile beyond fp32 summation order.  Returns
 * README_ERR_ARG for any other value.  readme_get_gemm_tile returns the
 * calling thread's current setting.
 */
readme_status readme_set_gemm_tile(int32_t tile);
int32_t readme_get_gemm_tile(void);

/*
 * readme_moe_ffn -- each expert's SwiGLU FFN on its token block (Eq. 2 with
 * a fixed top-1 expert; the output is the expert's, unweighted).
 *
 *   for every e, every j in [offsets[e], offsets[e+1]):
 *     h[j]         = silu(W_gate^e x_grouped[j]) * (W_up^e x_grouped[j])
 *     y_grouped[j] = W_down^e h[j]
 * Rows j >= offsets[E] of y_grouped are not written.
 *
 *   x_grouped [T][d] dt, offsets [E+1] int32 (device; non-decreasing, within
 *   [0, T]), packed (from readme_pack_experts with the same dt, E, d, I),
 *   y_grouped [T][d] dt out,
 *   workspace >= readme_moe_ffn_workspace_bytes(dt, T, I) bytes (holds h).
 * Requires d > 0 a multiple of 64, 1 <= E <= README_MAX_EXPERTS, I >= 1.
 * Offsets are read on the device only, so the host cannot validate them:
 * they must be readme_group_by_expert's (non-decreasing, within [0, T];
 * offsets[E] < T when some ids were outside [0, E)).  The kernels clamp
 * every block to [0, T], so a corrupt array cannot move an access outside
 * the buffers, but the outputs are then unspecified; no flag reports it.
 * Every streamed buffer (x_grouped, packed, y_grouped, workspace) must be
 * 16-byte aligned, and all are checked before the first launch.
 */
size_t readme_moe_ffn_workspace_bytes(readme_dtype dt, int64_t T, int64_t I);
readme_status readme_moe_ffn(readme_dtype dt, int64_t T, int64_t d,
                             int32_t E, int64_t I, const void *x_grouped,
                             const int32_t *offsets, const void *packed,
                             void *y_grouped, void *workspace,
                             size_t workspace_bytes, void *stream);

/*
 * The two halves of readme_moe_ffn, for callers that time or overlap them:
 *   readme_moe_gate_up: h[j][i] = silu(g) * u for i < I, and 0 for the pad
 *     columns I <= i < readme_padded_intermediate(I);
 *     h [T][readme_padded_intermediate(I)] dt out.
 *   readme_moe_down:    y_grouped[j] = W_down^e h[j].
 */
readme_status readme_moe_gate_up(readme_dtype dt, int64_t T, int64_t d,
                                 int32_t E, int64_t I, const void *x_grouped,
                                 const int32_t *offsets, const void *packed,
                                 void *h, void *stream);
readme_status readme_moe_down(readme_dtype dt, int64_t T, int64_t d,
                              int32_t E, int64_t I, const void *h,
                              const int32_t *offsets, const void *packed,
                              void *y_grouped, void *stream);

/*
 * readme_moe_ffn_fused -- readme_group_by_expert's row gather, readme_moe_ffn
 * and readme_ungroup in two launches: the gate/up GEMM reads its activation
 * rows straight from token order through perm, and the down GEMM writes
 * each output row straight to its token's row through perm.
 *   x [T][d] dt (token order), perm [T] and offsets [E+1] int32 from
 *   readme_group_by_expert (called without a gather), packed as for
 *   readme_moe_ffn, y [T][d] dt out (token order), workspace as for
 *   readme_moe_ffn.
 * Results equal readme_moe_ffn followed by readme_ungroup bit for bit
 * (same tiles, same summation order), except that rows of unrouted tokens
 * (ids outside [0, E)) are not written here.  Map entries outside [0, T)
 * are clamped on reads and skipped on writes.
 */
readme_status readme_moe_ffn_fused(readme_dtype dt, int64_t T, int64_t d,
                                   int32_t E, int64_t I, const void *x,
                                   const int32_t *perm, const int32_t *offsets,
                                   const void *packed, void *y,
                                   void *workspace, size_t workspace_bytes,
                                   void *stream);

/*
 * readme_moe_ffn_fused_noalloc -- readme_moe_ffn_fused for callers that
 * cannot allocate device memory (work under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): no workspace argument.
 * h lives in a file-scope device array of README_NOALLOC_SCRATCH_BYTES
 * (64 MiB) that each GPU the library runs on holds until the process ends;
 * its device address is looked up on the first call on the current device
 * (the stream must belong to the current device).  The call allocates and
 * frees nothing.  Same kernels, tiles and summation order as
 * readme_moe_ffn_fused, so the same bits.
 *   Arguments as readme_moe_ffn_fused without workspace.
 * README_ERR_UNSUPPORTED if T * readme_padded_intermediate(I) * element
 * size exceeds README_NOALLOC_SCRATCH_BYTES (checked before anything is
 * enqueued).  All calls on one GPU share its array: calls that overlap on
 * one GPU (other streams or host threads) race on h and give wrong
 * results; the array keeps the last call's contents, which no call reads.
 */
readme_status readme_moe_ffn_fused_noalloc(readme_dtype dt, int64_t T, int64_t d,
                                           int32_t E, int64_t I, const void *x,
                                           const int32_t *perm,
                                           const int32_t *offsets,
                                           const void *packed, void *y, void *stream);

/*
 * The two halves of readme_moe_ffn_fused:
 *   readme_moe_gate_up_gather: h as readme_moe_gate_up, activation row of
 *     grouped row j taken from x[perm[j]] (x in token order);
 *   readme_moe_down_scatter:   readme_moe_down with output row j written
 *     to y[perm[j]] (y in token order).
 */
readme_status readme_moe_gate_up_gather(readme_dtype dt, int64_t T, int64_t d,
                                        int32_t E, int64_t I, const void *x,
                                        const int32_t *perm,
                                        const int32_t *offsets,
                                        const void *packed, void *h,
                                        void *stream);
readme_status readme_moe_down_scatter(readme_dtype dt, int64_t T, int64_t d,
                                      int32_t E, int64_t I, const void *h,
                                      const int32_t *perm,
                                      const int32_t *offsets,
                                      const void *packed, void *y,
                                      void *stream);

/*
 * Permanent expert (Sec. 3): neurons that every token activates, beside its
 * routed expert.  A layer then computes, for every routed token,
 *   y = F_{e_t}(x) + F_perm(x),
 * F_perm the SwiGLU FFN of the permanent neurons, unweighted like the routed
 * term (Eq. 2 with K = 1).  The permanent width P is a whole number of expert
 * widths, P = S * I with 0 <= S <= README_MAX_PERMANENT_SLICES (S = 0 is the
 * plain layer), and is held as S slices of one expert's shape.
 *
 * readme_pack_experts_permanent -- one-time repack as readme_pack_experts,
 *   plus the permanent expert: p_gate [P][d], p_up [P][d], p_down [d][P]
 *   (dtype dt, device), slice j = neurons j*I .. j*I+I-1.  packed must hold
 *   readme_packed_experts_permanent_bytes(dt, E, d, I, P) bytes (0 for
 *   invalid arguments).  Not timed on the hot path.
 * readme_moe_ffn_permanent -- readme_moe_ffn with the permanent expert:
 *   y_grouped[j] = F_e(x_grouped[j]) + F_perm(x_grouped[j]) for
 *   j < offsets[E]; rows past offsets[E] are not written.
 * readme_moe_ffn_permanent_fused -- the same with the row moves folded in,
 *   as readme_moe_ffn_fused: activations read from x[perm[j]] (token order),
 *   output row j written to y[perm[j]]; rows of unrouted tokens are not
 *   written.
 *   workspace >= readme_moe_ffn_permanent_workspace_bytes(dt, T, I, P)
 *   bytes: h [T][(1+S)*Ip], the routed expert's neurons then each slice's.
 * Two launches: the gate/up GEMM treats the slices as S more row groups
 * over all routed rows; the down GEMM runs one K loop over the routed and
 * the permanent neurons of each row, so the sum is formed in fp32 and
 * rounded once.  Requirements and errors as readme_moe_ffn; P not a multiple
 * of I, or more than README_MAX_PERMANENT_SLICES slices, is
 * README_ERR_UNSUPPORTED, P < 0 README_ERR_ARG.
 */
/*
 * The two halves of readme_moe_ffn_permanent_fused, for callers that time or
 * overlap them (h [T][(1+S)*Ip] dt, S = P / I, as in the workspace above):
 *   readme_moe_gate_up_permanent_gather: h[j] = the routed expert's and each
 *     permanent slice's silu(g) * u of x[perm[j]] (pad columns 0);
 *   readme_moe_down_permanent_scatter: y[perm[j]] = W_down^e h[j][routed] +
 *     W_down^perm h[j][permanent], one fp32 sum rounded once.
 */
readme_status readme_moe_gate_up_permanent_gather(readme_dtype dt, int64_t T,
                                                  int64_t d, int32_t E, int64_t I,
                                                  int64_t P, const void *x,
                                                  const int32_t *perm,
                                                  const int32_t *offsets,
                                                  const void *packed, void *h,
                                                  void *stream);
readme_status readme_moe_down_permanent_scatter(readme_dtype dt, int64_t T,
                                                int64_t d, int32_t E, int64_t I,
                                                int64_t P, const void *h,
                                                const int32_t *perm,
                                                const int32_t *offsets,
                                                const void *packed, void *y,
                                                void *stream);
size_t readme_packed_experts_permanent_bytes(readme_dtype dt, int32_t E, int64_t d,
                                             int64_t I, int64_t P);
readme_status readme_pack_experts_permanent(readme_dtype dt, int32_t E, int64_t d,
                                            int64_t I, int64_t P,
                                            const void *w_gate, const void *w_up,
                                            const void *w_down, const void *p_gate,
                                            const void *p_up, const void *p_down,
                                            void *packed, size_t packed_bytes,
                                            void *stream);
size_t readme_moe_ffn_permanent_workspace_bytes(readme_dtype dt, int64_t T,
                                                int64_t I, int64_t P);
readme_status readme_moe_ffn_permanent(readme_dtype dt, int64_t T, int64_t d,
                                       int32_t E, int64_t I, int64_t P,
                                       const void *x_grouped,
                                       const int32_t *offsets,
                                       const void *packed, void *y_grouped,
                                       void *workspace, size_t workspace_bytes,
                                       void *stream);
readme_status readme_moe_ffn_permanent_fused(readme_dtype dt, int64_t T,
                                             int64_t d, int32_t E, int64_t I,
                                             int64_t P, const void *x,
                                             const int32_t *perm,
                                             const int32_t *offsets,
                                             const void *packed, void *y,
                                             void *workspace,
                                             size_t workspace_bytes,
                                             void *stream);

/*
 * Top-K routing (Eq. 2 with K > 1): each token on its K highest-logit
 * experts, the outputs summed with gate weights.  A step is
 *   readme_route (with logits) -> readme_topk -> readme_group_by_expert over
 *   the T*K (token, slot) pairs -> readme_moe_ffn_topk -> readme_combine_topk.
 * Pair p = t*K + k carries token t's k-th expert; grouping the pairs gives
 * perm (pair index per grouped row) and offsets over T*K rows.
 *
 * readme_topk -- ids[t*K + k] = the k-th expert of token t, weights[t*K + k]
 *   its gate weight.  Slot k takes, among the experts not yet taken, the
 *   first in ascending index unless a later one has a strictly larger logit
 *   (top-1 = readme_route's argmax; ties to the lower index; a later NaN
 *   never wins).  Weights: softmax of the K selected logits, renormalised
 *   over the slots (fp32 expf), so K = 1 gives weight 1.
 *   logits [T][E] fp32 (from readme_route), ids [T*K] int32, weights [T*K]
 *   fp32 (device).  Requires 1 <= K <= E <= README_MAX_EXPERTS, T*K < 2^31.
 * readme_moe_gate_up_gather_topk -- readme_moe_gate_up over the T*K grouped
 *   pair rows, the activation row of grouped row j being x[perm[j] / K];
 *   h [T*K][readme_padded_intermediate(I)] dt out.
 * readme_moe_ffn_topk -- gate/up as above, then the down projection with
 *   each grouped row's output written to its pair's row: y_pairs[perm[j]]
 *   (y_pairs [T*K][d] dt, pair order: token t's K rows are adjacent).
 *   workspace >= readme_moe_ffn_workspace_bytes(dt, T*K, I) bytes.
 * readme_combine_topk -- y[t] = sum over k = 0 .. K-1 (in that order, fp32)
 *   of weights[t*K + k] * y_pairs[t*K + k], rounded once to dt; K = 1
 *   reproduces y_pairs bit for bit.  y [T][d] dt; d * element size a
 *   multiple of 16 bytes.
 * Errors as the single-expert entry points; K outside [1, E] is
 * README_ERR_ARG.
 */
readme_status readme_topk(int64_t T, int32_t E, int32_t K, const float *logits,
                          int32_t *ids, float *weights, void *stream);
readme_status readme_moe_gate_up_gather_topk(readme_dtype dt, int64_t T,
                                             int64_t d, int32_t E, int64_t I,
                                             int32_t K, const void *x,
                                             const int32_t *perm,
                                             const int32_t *offsets,
                                             const void *packed, void *h,
                                             void *stream);
readme_status readme_moe_ffn_topk(readme_dtype dt, int64_t T, int64_t d,
                                  int32_t E, int64_t I, int32_t K, const void *x,
                                  const int32_t *perm, const int32_t *offsets,
                                  const void *packed, void *y_pairs,
                                  void *workspace, size_t workspace_bytes,
                                  void *stream);
readme_status readme_combine_topk(readme_dtype dt, int64_t T, int64_t d, int32_t K,
                                  const void *y_pairs, const float *weights,
                                  void *y, void *stream);

/*
 * Serving-side scheduling (Sec. 4), host code: no GPU, no streams; every
 * pointer below is host memory, owned by the caller.
 *
 * readme_expert_batch -- expert-aware batching (Alg. 1): fills one batch of
 *   at most max_tokens tokens from per-expert FIFO queues, repeatedly taking
 *   the longest queue (lowest expert index on ties) whole while it fits in
 *   the room left, else its first `room` tokens, then stopping; it also
 *   stops when every queue is empty.  Queues: tokens of expert e are
 *   queue_items[queue_offsets[e] .. queue_offsets[e+1]) (int32 ids, front
 *   first).  Out: batch [max_tokens] (token ids in batch order),
 *   *batch_len, taken [E] (tokens taken from the front of each queue; the
 *   caller pops them), visited [E] (experts whose tokens entered the batch,
 *   in order) and *n_visited.  Inputs are not modified.
 *   README_ERR_ARG for E < 1, max_tokens < 0, decreasing offsets or a
 *   missing array.
 *
 * readme_cache_simulate -- a demand cache of `capacity` entries over the
 *   reference sequence refs [n] (int32 keys >= 0, e.g. layer * E + expert).
 *   A reference hits if its key is cached; a miss inserts it, first
 *   evicting, when the cache is full, by policy:
 *     README_CACHE_BELADY  the cached key whose next reference is farthest
 *                          ahead (never again = farthest), lowest key on
 *                          ties: the rule of Sec. 4.1, exact because
 *                          pre-gating makes the future references known;
 *     README_CACHE_LRU     the least recently referenced key;
 *     README_CACHE_FIFO    the earliest inserted key;
 *     README_CACHE_RANDOM  the cached keys in ascending order, index
 *                          r mod size, r the next SplitMix64 output from
 *                          `seed` (Steele, Lea and Flood 2014).
 *   Out: hits [n] (1 = hit), evicted [n] (the evicted key, -1 if none),
 *   *n_hits.  O(n log capacity).  README_ERR_ARG for capacity < 1, n < 0, a
 *   negative key, an unknown policy or a missing array.
 */
#define README_CACHE_BELADY 0
#define README_CACHE_LRU 1
#define README_CACHE_FIFO 2
#define README_CACHE_RANDOM 3
readme_status readme_expert_batch(int32_t E, const int32_t *queue_offsets,
                                  const int32_t *queue_items, int64_t max_tokens,
                                  int32_t *batch, int64_t *batch_len,
                                  int32_t *taken, int32_t *visited,
                                  int32_t *n_visited);
readme_status readme_cache_simulate(int32_t policy, int64_t capacity, int64_t n,
                                    const int32_t *refs, uint64_t seed,
                                    uint8_t *hits, int32_t *evicted,
                                    int64_t *n_hits);

/*
 * Expert offload for the layer stack (Sec. 4.1: pre-gating lets the exact
 * experts of every layer be fetched ahead, and the cache replace by the
 * Belady rule).  The packed experts of every layer live in pinned host
 * memory; a device cache of `slots` (layer, expert) slots holds the weights
 * the GEMMs read; a second stream of the library's own (default priority)
 * copies the experts of layer l+1 while the caller's stream computes layer l.
 *
 * readme_offload_create -- copies the L packed layers (device buffers from
 *   readme_pack_experts, bf16, E experts of width I at d; the caller may
 *   free them afterwards) into pinned host memory and allocates the slots
 *   (slots * 3 * readme_padded_intermediate(I) * d * 2 bytes).  policy:
 *   README_CACHE_BELADY or README_CACHE_LRU.  Set-up call: it allocates and
 *   waits for its copies on `stream`.
 * readme_offload_stack -- readme_moe_ffn_stack over the L layers with the
 *   weights fetched through the cache: same kernels, same results bit for
 *   bit.  counts [E] (host) are the token counts of `offsets` (the caller's
 *   scheduler knows them: no device read), next_counts [E] (host, or NULL)
 *   those of the next step, which the Belady rule looks ahead to.  Needs
 *   slots >= 2 * (experts with tokens); else README_ERR_UNSUPPORTED.  The
 *   step's placement is planned as readme_offload_plan states; a plan that
 *   fails leaves the cache unchanged and nothing enqueued.  Host side: plans
 *   the whole step, then enqueues; it waits on the host only for the copy
 *   of its slot table from two steps earlier.  If an enqueue fails
 *   (README_ERR_HIP) the executor forgets every cached key.  Calls on one
 *   executor must not overlap.
 * readme_offload_stats -- cumulative hits, misses and bytes copied.
 * readme_offload_last_plan -- the references of the last successful
 *   readme_offload_stack step, in reference order (layer by layer, experts
 *   ascending): hits [n] (1 = hit), slot [n] (the slot that layer reads the
 *   expert from), evicted [n] (the key a miss evicted, layer*E+expert, -1
 *   none); *n_refs = n.  README_ERR_WORKSPACE if n > max_refs (*n_refs is
 *   still set).  Host only.
 *
 * readme_offload_plan -- the executor's placement planner alone (host only,
 *   no GPU): a cache of `slots` (layer, expert) entries, key layer*E+expert,
 *   over n_steps steps whose tokens per expert are counts [n_steps][E]
 *   (host).  A step references, for l = 0 .. L-1, the key of every expert
 *   with tokens, ascending.  A reference hits if its key is cached; a miss
 *   takes the lowest empty slot, else evicts, among the slots this step has
 *   NOT used at layer l or at layer l-1 (their kernels are enqueued after
 *   the copy), by policy:
 *     README_CACHE_BELADY  the key whose next reference is farthest ahead
 *                          (never = farthest), lowest key on ties, looking
 *                          at the rest of the step and, if lookahead != 0,
 *                          at the next step's references (Sec. 4.1);
 *     README_CACHE_LRU     the least recently referenced key.
 *   Out, per reference in order: hits, slot, evicted as for
 *   readme_offload_last_plan; *n_refs = references written.
 *   README_ERR_UNSUPPORTED if a step has more than slots / 2 experts with
 *   tokens, README_ERR_WORKSPACE if more than max_refs references,
 *   README_ERR_ARG for a bad size, policy or count.
 * readme_offload_destroy -- waits for the executor's copies and for the last
 *   recorded layer of the compute stream, then frees everything.
 */
typedef struct readme_offload readme_offload;
readme_status readme_offload_create(int32_t E, int64_t d, int64_t I, int32_t L,
                                    int32_t slots, int32_t policy,
                                    const void *const *packed_layers,
                                    readme_offload **out, void *stream);
readme_status readme_offload_stack(readme_offload *ex, int64_t T,
                                   const int32_t *offsets, const int32_t *counts,
                                   const int32_t *next_counts,
                                   float *x_resid_grouped, float rms_eps,
                                   void *workspace, size_t workspace_bytes,
                                   void *stream);
readme_status readme_offload_stats(const readme_offload *ex, int64_t *hits,
                                   int64_t *misses, int64_t *bytes_copied);
readme_status readme_offload_last_plan(const readme_offload *ex, int64_t max_refs,
                                       uint8_t *hits, int32_t *slot,
                                       int32_t *evicted, int64_t *n_refs);
readme_status readme_offload_plan(int32_t E, int32_t L, int32_t slots,
                                  int32_t policy, int32_t n_steps,
                                  const int32_t *counts, int32_t lookahead,
                                  int64_t max_refs, uint8_t *hits,
                                  int32_t *slot, int32_t *evicted,
                                  int64_t *n_refs);
void readme_offload_destroy(readme_offload *ex);

/*
 * readme_ungroup -- rows back to token order: y[t] = y_grouped[inv_perm[t]],
 * and a zero row where inv_perm[t] < 0 (an unrouted token).
 *   y_grouped [T][d] dt, inv_perm [T] int32, y [T][d] dt out.
 * Requires d * element size a multiple of 16 bytes.
 */
readme_status readme_ungroup(readme_dtype dt, int64_t T, int64_t d,
                             const void *y_grouped, const int32_t *inv_perm,
                             void *y, void *stream);

/*
 * The softmax-weighted top-1 variant of Eq. 2.  Eq. 2 multiplies each
 * selected expert's output by its gate value G(x)_i, and Eq. 4 applies a
 * softmax to G; the main path takes the top-1 output unweighted (so E = 1
 * is the dense FFN).  These two calls give the weighted form instead:
 *
 * readme_gate_weights -- for every token t with 0 <= expert_ids[t] < E and
 *   inv_perm[t] >= 0:  row_scale[inv_perm[t]] = p_t, the softmax of the
 *   token's logits at its expert,
 *     p_t = exp(l[t][e_t] - m_t) / sum_e exp(l[t][e] - m_t),  m_t = max_e l[t][e],
 *   in fp32 with the sum in ascending e (grouped order, ready for
 *   readme_ungroup_scaled).  Other entries of row_scale are not written.
 *   logits [T][E] fp32 (readme_route's), expert_ids [T], inv_perm [T] int32
 *   (readme_group_by_expert's), row_scale [T] fp32 out.  Finite logits are
 *   assumed (a NaN or +inf logit makes p_t NaN).
 *
 * readme_ungroup_scaled -- readme_ungroup with a weight per grouped row:
 *   y[t] = y_grouped[j] * row_scale[j], j = inv_perm[t], the product taken
 *   in fp32 and rounded once to dt; a zero row where j < 0.
 *   y_grouped [T][d] dt, inv_perm [T] int32, row_scale [T] fp32 (grouped
 *   order), y [T][d] dt out.  Requires d * element size a multiple of 16.
 */
readme_status readme_gate_weights(int64_t T, int32_t E, const float *logits,
                                  const int32_t *expert_ids, const int32_t *inv_perm,
                                  float *row_scale, void *stream);
readme_status readme_ungroup_scaled(readme_dtype dt, int64_t T, int64_t d,
                                    const void *y_grouped, const int32_t *inv_perm,
                                    const float *row_scale, void *y, void *stream);

/*
 * readme_moe_ffn_stack -- L stacked MoE layers of one decode or prefill step,
 * run in grouped order.  The router runs once and a token's expert is the
 * same at every layer (Sec. 2.3 and Sec. 4.2), so grouping is done once and
 * the residual stream stays grouped across layers:
 *   for l = 0 .. L-1:
 *     r_j   = 1 / sqrt(mean_k x[j][k]^2 + rms_eps)        (fp32)
 *     xn_j  = bf16(x[j] * r_j)
 *     x[j] += F^l_{e(j)}(xn_j)                            (fp32 residual)
 * (pre-norm residual layers without a norm gain, which would fold into
 * W_gate and W_up).  bf16 weights only.
 *
 *   packed_per_layer  HOST array of L device pointers, each packed with
 *                     readme_pack_experts(README_BF16, E, d, I, ...)
 *   offsets [E+1] int32 (device), x_resid_grouped [T][d] fp32 in/out,
 *   workspace >= readme_moe_ffn_stack_workspace_bytes(T, d, I) bytes.
 * Requires d > 0 a multiple of 64, 1 <= E <= README_MAX_EXPERTS, I >= 1,
 * L >= 0, rms_eps >= 0.  Rows j >= offsets[E] are left unchanged.
 */
size_t readme_moe_ffn_stack_workspace_bytes(int64_t T, int64_t d, int64_t I);
readme_status readme_moe_ffn_stack(int64_t T, int64_t d, int32_t E,
                                   int64_t I, int32_t L,
                                   const void *const *packed_per_layer,
                                   const int32_t *offsets,
                                   float *x_resid_grouped, float rms_eps,
                                   void *workspace, size_t workspace_bytes,
                                   void *stream);

/*
 * readme_moe_ffn_stack_counts -- readme_moe_ffn_stack for a caller that knows
 * the batch's token counts per expert on the host (a scheduler that formed
 * the batch, e.g. by readme_expert_batch): counts [E] (host) must be the
 * counts of `offsets`.  The tiles are then chosen for the actual split (a
 * batch on few experts gets narrower tiles, so more workgroups stream the
 * weights); results are bit-identical to readme_moe_ffn_stack.
 * README_ERR_ARG for a NULL or negative count.
 */
readme_status readme_moe_ffn_stack_counts(int64_t T, int64_t d, int32_t E, int64_t I,
                                          int32_t L, const void *const *packed_per_layer,
                                          const int32_t *offsets, const int32_t *counts,
                                          float *x_resid_grouped, float rms_eps,
                                          void *workspace, size_t workspace_bytes,
                                          void *stream);

/*
 * The pre-gating router G itself (Sec. 2.3, Table 1): one causal transformer
 * block over each request's tokens, whose normed output feeds the gate of
 * readme_route.  G reads a token and the tokens before it in the same
 * request, and nothing of the expert layers, so it runs once per token
 * before any layer (Sec. 2.3).  The paper fixes the block's type and sizes
 * (one layer, four heads, width 512, SwiGLU MLP, RoPE, RMSNorm); its wiring
 * here is the pre-norm residual block of the Llama family:
 *   x  = emb[token]                     fp32 residual (bf16 table rows; an id
 *                                       outside [0, V) embeds as zeros)
 *   a  = bf16(rmsnorm(x)),  q|k|v = bf16(a [Wq; Wk; Wv]^T)
 *   q, k <- bf16(RoPE(q, k)) (readme_rope)
 *   o  = bf16(causal attention(q, k, v)) (readme_attention_causal)
 *   x += o Wo^T
 *   x += W2 (silu(W1 m) * W3 m),  m = bf16(rmsnorm(x))
 *   f  = bf16(rmsnorm(x)),  expert_ids, logits = readme_route(f, w_router, bias)
 * rmsnorm has no gain: r = 1 / sqrt(mean x^2 + rms_eps), fp32.  Heads are
 * D / 128 slices of 128 dims; bf16 weights only.
 *
 * readme_router_tf_pack -- one-time repack of the block's weights into
 *   `packed` (readme_router_tf_packed_bytes(D, F) bytes, device, 16-byte
 *   aligned):  wq, wk, wv, wo [D][D]; w1, w3 [F][D]; w2 [D][F]  (bf16,
 *   [out][in] row-major, device).  README_ERR_WORKSPACE if packed_bytes is
 *   smaller than required.
 *
 * readme_router_tf -- the router over T tokens of R requests:
 *   tokens       [T]      int32   token ids
 *   req_offsets  [R+1]    int32   request r is tokens [req_offsets[r],
 *                                 req_offsets[r+1]); req_offsets[0] = 0,
 *                                 req_offsets[R] = T, non-decreasing (empty
 *                                 requests allowed).  Other values give
 *                                 unspecified results but no access outside
 *                                 the arrays.
 *   emb          [V][D]   bf16    embedding table
 *   packed                        from readme_router_tf_pack(D, F, ...)
 *   w_router     [E][D]   bf16,   bias [E] fp32 or NULL: the gate
 *   expert_ids   [T]      int32 out;  logits [T][E] fp32 out or NULL
 *   workspace    >= readme_router_tf_workspace_bytes(T, D, F) bytes
 * On return the workspace holds every intermediate, each region at
 * readme_router_tf_workspace_offset(T, D, F, region):
 *   README_RTF_X     [T][D]   fp32   the block's output x (before the final norm)
 *   README_RTF_A     [T][D]   bf16   a
 *   README_RTF_QKV   [T][3D]  bf16   q | k | v (q and k rotated)
 *   README_RTF_O     [T][D]   bf16   attention output
 *   README_RTF_M     [T][D]   bf16   the MLP's normed input m
 *   README_RTF_H     [T][Fp]  bf16   silu(W1 m) * W3 m, Fp = readme_padded_intermediate(F)
 *   README_RTF_FEAT  [T][D]   bf16   f, the gate's input
 *   README_RTF_POS   [T]      int32  each token's position in its request
 *   README_RTF_OFFS  [2]      int32  {0, T}
 * Requires D > 0 a multiple of 128 and at most 16384, F >= 1 (with
 * 4 * Fp * D < 2^31), 1 <= E <= README_MAX_EXPERTS, V >= 1, rms_eps >= 0,
 * R >= 1 when T > 0.  The size queries return 0 (offset: -1) for arguments
 * outside that set.
 */
#define README_RTF_X 0
#define README_RTF_A 1
#define README_RTF_QKV 2
#define README_RTF_O 3
#define README_RTF_M 4
#define README_RTF_H 5
#define README_RTF_FEAT 6
#define README_RTF_POS 7
#define README_RTF_OFFS 8
#define README_RTF_END 9 /* offset of the end = the workspace size */

size_t readme_router_tf_packed_bytes(int64_t D, int64_t F);
readme_status readme_router_tf_pack(int64_t D, int64_t F, const void *wq, const void *wk,
                                    const void *wv, const void *wo, const void *w1,
                                    const void *w3, const void *w2, void *packed,
                                    size_t packed_bytes, void *stream);
size_t readme_router_tf_workspace_bytes(int64_t T, int64_t D, int64_t F);
int64_t readme_router_tf_workspace_offset(int64_t T, int64_t D, int64_t F, int32_t region);
readme_status readme_router_tf(int64_t T, int32_t R, int64_t D, int64_t F, int32_t E,
                               int64_t V, const int32_t *tokens, const int32_t *req_offsets,
                               const void *emb, const void *packed, const void *w_router,
                               const float *bias, float rms_eps, int32_t *expert_ids,
                               float *logits, void *workspace, size_t workspace_bytes,
                               void *stream);

/*
 * readme_request_positions -- pos[t] = t - req_offsets[r] for the request r
 * holding token t (requests as in readme_router_tf): the position that
 * RoPE rotates by and that bounds the causal attention.  pos [T] int32 out.
 */
readme_status readme_request_positions(int64_t T, int32_t R, const int32_t *req_offsets,
                                       int32_t *pos, void *stream);

/*
 * readme_rope -- rotary position embedding (RoPE, the positional encoding of
 * Table 1's block) in place on H heads of 128 bf16 values per row: row t at
 * x + t * ld, head h at columns 128h .. 128h+127.  For i < 64 the pair
 * (x_i, x_{i+64}) of each head turns by the angle pos[t] * 10000^(-2i/128):
 *   x_i     <- x_i cos - x_{i+64} sin
 *   x_{i+64} <- x_{i+64} cos + x_i sin
 * (the rotate-half form), angle, sine, cosine and products in fp64 without
 * fused multiply-adds, each result rounded to fp32 and then to bf16 (nearest
 * even).  pos [T] int32 (readme_request_positions).  Requires ld >= 128 H,
 * ld a multiple of 8 and x 16-byte aligned.
 */
readme_status readme_rope(int64_t T, int32_t H, const int32_t *pos, void *x, int64_t ld,
                          void *stream);

/*
 * readme_attention_causal -- multi-head attention of each token over its
 * request's prefix (Sec. 2.3: G sees the current and earlier tokens):
 *   o[t]_h = sum_j w_tj v[j]_h / sum_j w_tj,   w_tj = exp(q[t]_h . k[j]_h / sqrt(128) - m_t)
 * over j = t - pos[t] .. t, per head h of 128 dims.  Scores and the running
 * softmax in fp32; the weights enter the value product as a bf16 pair
 * (hi + lo, about 16 significant bits), so o is the exact result up to
 * about 2^-16 of the largest |v| plus the final bf16 rounding.
 *   q, k, v  [T][ld_in] bf16 (head h at columns 128h ..), o [T][ld_out] bf16
 *   out, pos [T] int32.  R, the number of requests the tokens form, only
 *   picks the launch shape (from a mean of 128 tokens per request, eight
 *   waves per 128 queries in two groups over alternate key blocks; below,
 *   one wave per 32 queries over its own blocks); both meet the bound above,
 *   their last bits may differ.  Requires
 *   ld_in, ld_out >= 128 H and multiples of 8, 16-byte aligned q, k, v, o,
 *   H <= 65535.  o must not overlap q, k or v.
 */
readme_status readme_attention_causal(int64_t T, int32_t H, int32_t R, const int32_t *pos,
                                      const void *q, const void *k, const void *v,
                                      int64_t ld_in, void *o, int64_t ld_out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* README_H */
