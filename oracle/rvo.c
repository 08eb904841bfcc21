/*
 * rvo.c -- CPU oracle for the RegVGGT per-frame hot path (TEST INFRASTRUCTURE ONLY).
 *
 * Plain fp64 C, written from the paper's definitions (Sec. 3.1 Eq. 2-3 and Sec. 3.3:
 * Eq. 6, the head-specific retention rule, the LSE equation and the A_ij equation).
 * Nothing here is blocked, fused or reordered beyond those definitions; OpenMP only
 * spreads independent (head, query) rows over host cores.  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg may load this file's library.
 */
#define _GNU_SOURCE /* qsort_r */
#include "rvo.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* A bf16 value is the upper half of an IEEE binary32; widening to double is exact. */
static double bf16_to_double(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

int rvo_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Sec. 3.3, "Head-Specific Token Retention": 2x2 (generally stride x stride)
 * non-overlapping windows over the patch grid, keep each window's top-left query. */
int rvo_qsub_index(int grid_h, int grid_w, int n_special, int stride, int32_t *out, int cap)
{
    if (grid_h < 0 || grid_w < 0 || n_special < 0 || stride < 1 || (cap > 0 && !out))
        return -1;
    int n = 0;
    for (int r = 0; r < grid_h; r += stride)
        for (int c = 0; c < grid_w; c += stride) {
            if (n < cap)
                out[n] = n_special + r * grid_w + c;
            n++;
        }
    return n;
}

/* Sec. 3.1 Eq. 2-3 with the LSE equation of Sec. 3.3: for query i of the current frame
 * and head h, the context is every memory row followed by every current-frame key (no
 * mask inside the frame).  z_c = q_i . k_c / sqrt(d);  LSE_i = log sum_c exp(z_c);
 * A_ic = exp(z_c - LSE_i);  o_i = sum_c A_ic v_c. */
int rvo_attend(const uint16_t *Q, const uint16_t *K, const uint16_t *V, int n_tokens,
               int n_heads, int head_dim,
               const uint16_t *memK, const uint16_t *memV, int64_t mem_len, int64_t head_stride,
               const int32_t *rows, int n_rows, double *out, double *lse)
{
    if (!Q || !K || !V || !out || !lse || n_tokens < 0 || n_heads < 1 || head_dim < 1 ||
        mem_len < 0 || n_rows < 0)
        return -1;
    if (mem_len > 0 && (!memK || !memV || head_stride < mem_len))
        return -1;
    if (!rows && n_rows != n_tokens)
        return -1;
    for (int r = 0; rows && r < n_rows; r++)
        if (rows[r] < 0 || rows[r] >= n_tokens)
            return -1;

    const int d = head_dim, H = n_heads;
    const int64_t ctx = mem_len + n_tokens;
    const double inv_sqrt_d = 1.0 / sqrt((double)d);
    int status = 0;

#pragma omp parallel
    {
        double *z = (double *)malloc(sizeof(double) * (size_t)(ctx > 0 ? ctx : 1));
        double *q = (double *)malloc(sizeof(double) * (size_t)d);
        double *o = (double *)malloc(sizeof(double) * (size_t)d);
        const int ok = z && q && o;
        if (!ok) {
#pragma omp atomic write
            status = -2;
        }
        /* every thread takes part in the worksharing loop; one without buffers skips */
#pragma omp for schedule(dynamic, 1) collapse(2)
        for (int h = 0; h < H; h++)
            for (int r = 0; r < n_rows; r++) {
                if (!ok)
                    continue;
                {
                    const int i = rows ? rows[r] : r;
                    const uint16_t *qi = Q + ((int64_t)i * H + h) * d;
                    for (int e = 0; e < d; e++)
                        q[e] = bf16_to_double(qi[e]);
                    /* logits over memory rows, then current-frame keys */
                    for (int64_t c = 0; c < ctx; c++) {
                        const uint16_t *kc = c < mem_len
                                                 ? memK + ((int64_t)h * head_stride + c) * d
                                                 : K + ((c - mem_len) * H + h) * d;
                        double dot = 0.0;
                        for (int e = 0; e < d; e++)
                            dot += q[e] * bf16_to_double(kc[e]);
                        z[c] = dot * inv_sqrt_d;
                    }
                    /* LSE_i = log sum_c exp(z_c), evaluated as m + log sum exp(z_c - m) */
                    double m = -INFINITY;
                    for (int64_t c = 0; c < ctx; c++)
                        if (z[c] > m)
                            m = z[c];
                    double s = 0.0;
                    for (int64_t c = 0; c < ctx; c++)
                        s += exp(z[c] - m);
                    const double L = ctx > 0 ? m + log(s) : -INFINITY;
                    /* o_i = sum_c exp(z_c - LSE_i) v_c */
                    for (int e = 0; e < d; e++)
                        o[e] = 0.0;
                    for (int64_t c = 0; c < ctx; c++) {
                        const double a = exp(z[c] - L);
                        const uint16_t *vc = c < mem_len
                                                 ? memV + ((int64_t)h * head_stride + c) * d
                                                 : V + ((c - mem_len) * H + h) * d;
                        for (int e = 0; e < d; e++)
                            o[e] += a * bf16_to_double(vc[e]);
                    }
                    for (int e = 0; e < d; e++)
                        out[((int64_t)r * H + h) * d + e] = o[e];
                    lse[(int64_t)h * n_rows + r] = L;
                }
            }
        free(z);
        free(q);
        free(o);
    }
    return status;
}

/* Sec. 3.3: S_j = sum_{i in Q~} A_ij with A_ij = exp(Z_ij - LSE_i), Z_ij = q_i . k_j / sqrt(d).
 * The LSE is the one of the full attended context, so A_ij is the exact attention
 * probability; no score matrix is kept, each column is summed on its own. */
int rvo_column_mass(const uint16_t *Q, int n_tokens, int n_heads, int head_dim,
                    const int32_t *qidx, int n_q, const double *lse_q,
                    const uint16_t *keys, int n_keys, int64_t key_tok_stride,
                    int64_t key_head_stride, double *S)
{
    if (!Q || !S || n_tokens < 0 || n_heads < 1 || head_dim < 1 || n_q < 0 || n_keys < 0)
        return -1;
    if (n_q > 0 && (!qidx || !lse_q))
        return -1;
    if (n_keys > 0 && !keys)
        return -1;
    for (int a = 0; a < n_q; a++)
        if (qidx[a] < 0 || qidx[a] >= n_tokens)
            return -1;

    const int d = head_dim, H = n_heads;
    const double inv_sqrt_d = 1.0 / sqrt((double)d);

#pragma omp parallel for schedule(dynamic, 16) collapse(2)
    for (int h = 0; h < H; h++)
        for (int j = 0; j < n_keys; j++) {
            const uint16_t *kj = keys + (int64_t)j * key_tok_stride + (int64_t)h * key_head_stride;
            double sum = 0.0;
            for (int a = 0; a < n_q; a++) {
                const uint16_t *qi = Q + ((int64_t)qidx[a] * H + h) * d;
                double dot = 0.0;
                for (int e = 0; e < d; e++)
                    dot += bf16_to_double(qi[e]) * bf16_to_double(kj[e]);
                sum += exp(dot * inv_sqrt_d - lse_q[(int64_t)h * n_q + a]);
            }
            S[(int64_t)h * n_keys + j] = sum;
        }
    return 0;
}

/* Ordering for the top-k: higher saliency first, then lower token index. */
static int cmp_by_saliency(const void *pa, const void *pb, void *ctx)
{
    const double *sal = (const double *)ctx;
    const int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    const double sa = sal[a], sb = sal[b];
    if (sa > sb)
        return -1;
    if (sa < sb)
        return 1;
    return (a > b) - (a < b);
}

static int cmp_int32(const void *pa, const void *pb)
{
    const int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    return (a > b) - (a < b);
}

/* Sec. 3.3 Eq. 6: Top-k of the frame's tokens by saliency, per head. */
int rvo_topk(const double *sal, int n_tokens, int n_heads, int budget, int32_t *idx)
{
    if (!sal || n_tokens < 0 || n_heads < 1 || budget < 0 || budget > n_tokens ||
        (budget > 0 && !idx))
        return -1;
    int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n_tokens > 0 ? n_tokens : 1));
    if (!order)
        return -2;
    for (int h = 0; h < n_heads; h++) {
        for (int j = 0; j < n_tokens; j++)
            order[j] = j;
        qsort_r(order, (size_t)n_tokens, sizeof(int32_t), cmp_by_saliency,
                (void *)(sal + (int64_t)h * n_tokens));
        qsort(order, (size_t)budget, sizeof(int32_t), cmp_int32);
        memcpy(idx + (int64_t)h * budget, order, sizeof(int32_t) * (size_t)budget);
    }
    free(order);
    return 0;
}

/* Sec. 3.3 Eq. 6: M_t = M_{t-1} united with the selected rows of (K_t, V_t). */
int rvo_append(uint16_t *memK, uint16_t *memV, int64_t mem_len, int64_t head_stride,
               const uint16_t *K, const uint16_t *V, int n_tokens, int n_heads, int head_dim,
               const int32_t *idx, int budget)
{
    if (!memK || !memV || !K || !V || mem_len < 0 || n_heads < 1 || head_dim < 1 ||
        budget < 0 || head_stride < mem_len + budget || (budget > 0 && !idx))
        return -1;
    for (int h = 0; h < n_heads; h++)
        for (int r = 0; r < budget; r++) {
            const int32_t j = idx[(int64_t)h * budget + r];
            if (j < 0 || j >= n_tokens)
                return -1;
            const int64_t dst = ((int64_t)h * head_stride + mem_len + r) * head_dim;
            const int64_t src = ((int64_t)j * n_heads + h) * head_dim;
            memcpy(memK + dst, K + src, sizeof(uint16_t) * (size_t)head_dim);
            memcpy(memV + dst, V + src, sizeof(uint16_t) * (size_t)head_dim);
        }
    return 0;
}
