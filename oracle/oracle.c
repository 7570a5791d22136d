/*
 * oracle.c -- plain, slow CPU oracle of the pre-gated expert-FFN layer
 * (Read-ME, arXiv 2410.19123).
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the CPU
 * baseline of the benchmark load this library.  It shares no code, header or
 * table with the HIP library and never calls it.
 *
 * What it computes (one MoE layer, top-1 routing, Sec. 2.3 Eq. 2 with K = 1):
 *   route    logit[t,e] = <x_t, W_r[e]> + b[e]; id[t] = first argmax.
 *   group    stable counting sort of tokens by id (the per-expert request
 *            queues of the expert-aware batching, Sec. 4.2 Alg. 1).
 *   gather   x_g[j] = x[perm[j]].
 *   ffn      y_g[j] = W_down^e (silu(W_gate^e x_g[j]) * (W_up^e x_g[j])),
 *            e the expert owning grouped row j (the expert form of Sec. 3,
 *            instantiated as the Llama SwiGLU FFN of Table 1).
 *   ungroup  y[t] = y_g[inv_perm[t]].
 *   layer    one pre-norm residual layer of a stack that keeps the grouped
 *            order across layers (a token's expert is the same at every
 *            layer, Sec. 4.2): x + F(bf16(x * rsqrt(mean(x^2) + eps))).
 *
 * Precision.  The paper fixes none.  The FFN is evaluated in fp64 on the
 * exact values of its (bf16 or fp32) inputs.  Two steps turn floating point
 * into a discrete result and are taken in the kernel's precision, fp32:
 *   - the router argmax, over fp32 logits summed in the canonical order
 *     described at oracle_route;
 *   - the bf16 rounding of the normalised layer input in oracle_layer_rows.
 * Build with -O2 -ffp-contract=off -fno-fast-math so that no sum is
 * reassociated or contracted.
 *
 * Element types: dtype 0 = fp32, 1 = bf16 given as raw 16-bit patterns.
 * Return value: 0 on success, nonzero on a bad argument.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_F32 0
#define OR_BF16 1

static float bf16_bits_to_float(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* fp32 -> bf16 bit pattern, round to nearest, ties to even; NaN stays NaN. */
static uint16_t float_to_bf16_bits(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7fffu + lsb;
    return (uint16_t)(u >> 16);
}

static float load_f(int dtype, const void *p, int64_t i)
{
    if (dtype == OR_F32)
        return ((const float *)p)[i];
    return bf16_bits_to_float(((const uint16_t *)p)[i]);
}

static size_t elem_size(int dtype) { return dtype == OR_F32 ? 4 : 2; }

/* ------------------------------------------------------------------ route */
/*
 * Router logits and top-1 id (Eq. 2 with K = 1: the expert of largest gate
 * value; ties go to the lowest index).
 *
 * The argmax decides an integer, so the logits are formed in fp32 in one
 * fixed, stated order that the GPU kernel follows as well:
 *   - x_t and W_r[e] are cut into 16-byte chunks (8 bf16 or 4 fp32 values);
 *     chunk c covers elements [c*w, c*w + w), w = 16 / element size;
 *   - 64 partial sums p[0..63] start at +0; p[l] takes chunks l, l+64,
 *     l+128, ... in that order, and inside a chunk the elements in ascending
 *     k, each as p[l] = fmaf(x[k], w[k], p[l]);
 *   - the partials are folded pairwise, for off = 32, 16, 8, 4, 2, 1:
 *     p[l] = p[l] + p[l + off] for l < off; the sum is p[0];
 *   - logit = sum + b[e] (one fp32 add; no bias means no add).
 *   - id = 0, best = logit[0]; for e = 1..E-1, if logit[e] > best then
 *     best = logit[e], id = e.  Strict '>' gives ties to the lowest index
 *     and never lets a NaN win.
 * d must be a multiple of w.
 */
int oracle_route(int dtype, int64_t T, int64_t d, int32_t E, const void *x,
                 const void *w_router, const float *bias, int32_t *ids,
                 float *logits)
{
    if (T < 0 || d <= 0 || E < 1 || !x || !w_router || !ids)
        return 1;
    const int64_t w = 16 / (int64_t)elem_size(dtype);
    if (d % w)
        return 1;
    const int64_t nchunks = d / w;

#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        int32_t id = 0;
        float best = 0.0f;
        for (int32_t e = 0; e < E; ++e) {
            float p[64];
            for (int l = 0; l < 64; ++l) {
                float acc = 0.0f;
                for (int64_t c = l; c < nchunks; c += 64) {
                    for (int64_t q = 0; q < w; ++q) {
                        int64_t k = c * w + q;
                        acc = fmaf(load_f(dtype, x, t * d + k),
                                   load_f(dtype, w_router, (int64_t)e * d + k),
                                   acc);
                    }
                }
                p[l] = acc;
            }
            for (int off = 32; off >= 1; off /= 2)
                for (int l = 0; l < off; ++l)
                    p[l] = p[l] + p[l + off];
            float logit = p[0];
            if (bias)
                logit = logit + bias[e];
            if (logits)
                logits[t * E + e] = logit;
            if (e == 0) {
                best = logit;
                id = 0;
            } else if (logit > best) {
                best = logit;
                id = e;
            }
        }
        ids[t] = id;
    }
    return 0;
}

/* ------------------------------------------------------------------ group */
/*
 * Stable counting sort of tokens by expert id: the per-expert queues of
 * Alg. 1 (their lengths are its per-expert counts).
 *   counts[e]   = #{t : id[t] = e}
 *   offsets[0]  = 0, offsets[e+1] = offsets[e] + counts[e]
 *   perm[j]     = the token at grouped row j; tokens of one expert keep
 *                 their ascending token order
 *   inv_perm[t] = the grouped row of token t
 * An id outside [0, E) routes nowhere: the token is left out of counts and
 * perm, inv_perm[t] = -1, and offsets[E] is the number of routed tokens;
 * perm[j] = -1 for j >= offsets[E].
 */
int oracle_group(int64_t T, int32_t E, const int32_t *ids, int32_t *counts,
                 int32_t *offsets, int32_t *perm, int32_t *inv_perm)
{
    if (T < 0 || E < 1 || (T > 0 && !ids) || !counts || !offsets)
        return 1;
    for (int32_t e = 0; e < E; ++e)
        counts[e] = 0;
    for (int64_t t = 0; t < T; ++t)
        if (ids[t] >= 0 && ids[t] < E)
            counts[ids[t]] += 1;
    offsets[0] = 0;
    for (int32_t e = 0; e < E; ++e)
        offsets[e + 1] = offsets[e] + counts[e];
    int32_t *cursor = (int32_t *)malloc(sizeof(int32_t) * (size_t)E);
    if (!cursor)
        return 2;
    for (int32_t e = 0; e < E; ++e)
        cursor[e] = offsets[e];
    for (int64_t j = 0; j < T; ++j)
        if (perm)
            perm[j] = -1;
    for (int64_t t = 0; t < T; ++t) {
        int32_t e = ids[t];
        if (e < 0 || e >= E) {
            if (inv_perm)
                inv_perm[t] = -1;
            continue;
        }
        int32_t j = cursor[e]++;
        if (perm)
            perm[j] = (int32_t)t;
        if (inv_perm)
            inv_perm[t] = j;
    }
    free(cursor);
    return 0;
}

/* --------------------------------------------------------- gather/ungroup */
/* x_g[j] = x[perm[j]] for j < T; a row with perm[j] < 0 is all zero bits. */
int oracle_gather(int dtype, int64_t T, int64_t d, const int32_t *perm,
                  const void *x, void *x_g)
{
    if (T < 0 || d <= 0 || (T > 0 && (!perm || !x || !x_g)))
        return 1;
    const size_t row = (size_t)d * elem_size(dtype);
    for (int64_t j = 0; j < T; ++j) {
        char *dst = (char *)x_g + (size_t)j * row;
        if (perm[j] < 0 || perm[j] >= T)
            memset(dst, 0, row);
        else
            memcpy(dst, (const char *)x + (size_t)perm[j] * row, row);
    }
    return 0;
}

/* y[t] = y_g[inv_perm[t]] for t < T; a row with inv_perm[t] < 0 is zero.
 * Works on any element size (the bytes are copied). */
int oracle_ungroup(int64_t T, int64_t row_bytes, const int32_t *inv_perm,
                   const void *y_g, void *y)
{
    if (T < 0 || row_bytes <= 0 || (T > 0 && (!inv_perm || !y_g || !y)))
        return 1;
    for (int64_t t = 0; t < T; ++t) {
        char *dst = (char *)y + (size_t)t * (size_t)row_bytes;
        if (inv_perm[t] < 0 || inv_perm[t] >= T)
            memset(dst, 0, (size_t)row_bytes);
        else
            memcpy(dst, (const char *)y_g + (size_t)inv_perm[t] * (size_t)row_bytes,
                   (size_t)row_bytes);
    }
    return 0;
}

/* -------------------------------------------------------------------- ffn */
static double silu_d(double z) { return z / (1.0 + exp(-z)); }

/* The expert owning grouped row j, or -1 if no expert does. */
static int32_t owner(int32_t E, const int32_t *offsets, int64_t j)
{
    for (int32_t e = 0; e < E; ++e)
        if (j >= offsets[e] && j < offsets[e + 1])
            return e;
    return -1;
}

/* One expert's SwiGLU FFN on one fp64 input row (length d) -> y (length d).
 * h is scratch of length I. */
static void expert_ffn_row(int dtype, int64_t d, int64_t I, int32_t e,
                           const double *xr, const void *wg, const void *wu,
                           const void *wd, double *h, double *y)
{
    const int64_t wbase = (int64_t)e * I * d; /* [E][I][d] and [E][d][I] */
    for (int64_t i = 0; i < I; ++i) {
        double g = 0.0, u = 0.0;
        for (int64_t k = 0; k < d; ++k) {
            g += (double)load_f(dtype, wg, wbase + i * d + k) * xr[k];
            u += (double)load_f(dtype, wu, wbase + i * d + k) * xr[k];
        }
        h[i] = silu_d(g) * u;
    }
    for (int64_t c = 0; c < d; ++c) {
        double acc = 0.0;
        for (int64_t i = 0; i < I; ++i)
            acc += (double)load_f(dtype, wd, wbase + c * I + i) * h[i];
        y[c] = acc;
    }
}

/*
 * Expert FFN on grouped rows: for each requested grouped row j (rows[r]),
 * with e the expert whose block [offsets[e], offsets[e+1]) holds j,
 *   g = W_gate[e] x_g[j],  u = W_up[e] x_g[j]   (W_* [E][I][d])
 *   h = silu(g) * u,       silu(z) = z / (1 + exp(-z))
 *   y[r] = W_down[e] h                          (W_down [E][d][I])
 * all in fp64, sums in ascending index order.  The output is unweighted: a
 * token's result is its one expert's FFN output (top-1).
 * rows == NULL means rows 0..nrows-1.  Returns 3 if a row has no expert.
 */
int oracle_moe_ffn_rows(int dtype, int64_t T, int64_t d, int32_t E, int64_t I,
                        const void *x_g, const int32_t *offsets,
                        const void *w_gate, const void *w_up,
                        const void *w_down, int64_t nrows, const int64_t *rows,
                        double *y)
{
    if (T < 0 || d <= 0 || E < 1 || I < 1 || nrows < 0 || !offsets)
        return 1;
    if (nrows > 0 && (!x_g || !w_gate || !w_up || !w_down || !y))
        return 1;
    int bad = 0;
#pragma omp parallel
    {
        double *xr = (double *)malloc(sizeof(double) * (size_t)d);
        double *h = (double *)malloc(sizeof(double) * (size_t)I);
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < nrows; ++r) {
            int64_t j = rows ? rows[r] : r;
            int32_t e = (j >= 0 && j < T) ? owner(E, offsets, j) : -1;
            if (e < 0 || !xr || !h) {
#pragma omp atomic write
                bad = 3;
                continue;
            }
            for (int64_t k = 0; k < d; ++k)
                xr[k] = (double)load_f(dtype, x_g, j * d + k);
            expert_ffn_row(dtype, d, I, e, xr, w_gate, w_up, w_down, h,
                           y + r * d);
        }
        free(xr);
        free(h);
    }
    return bad;
}

/* ------------------------------------------------------------ stack layer */
/*
 * One layer of the decode stack, on grouped rows of the fp32 residual
 * stream x (the grouped order is kept from layer to layer because a token's
 * expert does not change between layers):
 *   r      = 1 / sqrtf(sum_k x[k]^2 / d + eps)    fp32, k ascending
 *   xn[k]  = bf16(x[k] * r)                        fp32 product, RNE
 *   y[r]   = expert FFN of xn in fp64, as in oracle_moe_ffn_rows
 * The caller forms the next residual x + y.  w_* are bf16.
 * xn_out (optional, [nrows][d] bf16 bits) receives the rounded input.
 */
int oracle_layer_rows(int64_t T, int64_t d, int32_t E, int64_t I,
                      const float *x, const int32_t *offsets,
                      const uint16_t *w_gate, const uint16_t *w_up,
                      const uint16_t *w_down, float eps, int64_t nrows,
                      const int64_t *rows, double *y, uint16_t *xn_out)
{
    if (T < 0 || d <= 0 || E < 1 || I < 1 || nrows < 0 || !offsets)
        return 1;
    if (nrows > 0 && (!x || !w_gate || !w_up || !w_down || !y))
        return 1;
    int bad = 0;
#pragma omp parallel
    {
        double *xr = (double *)malloc(sizeof(double) * (size_t)d);
        double *h = (double *)malloc(sizeof(double) * (size_t)I);
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < nrows; ++r) {
            int64_t j = rows ? rows[r] : r;
            int32_t e = (j >= 0 && j < T) ? owner(E, offsets, j) : -1;
            if (e < 0 || !xr || !h) {
#pragma omp atomic write
                bad = 3;
                continue;
            }
            const float *xj = x + j * d;
            float ss = 0.0f;
            for (int64_t k = 0; k < d; ++k)
                ss = ss + xj[k] * xj[k];
            float rs = 1.0f / sqrtf(ss / (float)d + eps);
            for (int64_t k = 0; k < d; ++k) {
                uint16_t b = float_to_bf16_bits(xj[k] * rs);
                if (xn_out)
                    xn_out[r * d + k] = b;
                xr[k] = (double)bf16_bits_to_float(b);
            }
            expert_ffn_row(OR_BF16, d, I, e, xr, w_gate, w_up, w_down, h,
                           y + r * d);
        }
        free(xr);
        free(h);
    }
    return bad;
}

/* bf16 rounding exposed for the pins of the layer input. */
void oracle_f32_to_bf16(int64_t n, const float *src, uint16_t *dst)
{
    for (int64_t i = 0; i < n; ++i)
        dst[i] = float_to_bf16_bits(src[i]);
}

/* Threads the OpenMP loops above use (reported beside oracle timings). */
#ifdef _OPENMP
#include <omp.h>
int oracle_threads(void) { return omp_get_max_threads(); }
#else
int oracle_threads(void) { return 1; }
#endif
