/*
 * rvo.h -- CPU oracle for the RegVGGT per-frame hot path (TEST INFRASTRUCTURE ONLY).
 *
 * This is a plain, slow, fp64 implementation of what the paper defines, written to be
 * checked by eye against the paper.  It exists to prove the GPU library right; it is not
 * part of the product.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load it.  It shares no code, header, table or helper with the HIP
 * library: the two are separate source trees that meet only in the seeded input
 * generator, which holds none of the method's arithmetic.
 *
 * Conventions (all arrays row-major, caller-owned host memory):
 *   bf16 inputs are passed as their raw 16-bit patterns (uint16_t) and widened exactly
 *   to double before any arithmetic.
 *   Current-frame tensors Q, K, V:  [n_tokens][n_heads][head_dim].
 *   Memory (KV cache) tensors:      [n_heads][head_stride][head_dim]; rows 0..mem_len-1
 *                                   of each head are the admitted tokens, in arena order.
 *   Per-head per-token outputs (lse, saliency): [n_heads][n_rows].
 *
 * Every function returns 0 on success and a negative value on invalid arguments.
 */
#ifndef RVO_H
#define RVO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Query subset Q~ (Sec. 3.3, "Head-Specific Token Retention"): the frame's patch
 * grid (grid_h x grid_w, row-major, after n_special leading special tokens) is cut into
 * stride x stride non-overlapping windows and the top-left query of each window is kept.
 * Partial windows at the right/bottom edge are kept.  Writes at most cap indices
 * (token positions in the frame) to out; returns the number of sampled queries. */
int rvo_qsub_index(int grid_h, int grid_w, int n_special, int stride, int32_t *out, int cap);

/* Temporal-causal attention of the current frame over memory + current frame, with the
 * log-sum-exp of every query (Sec. 3.1 Eq. 2-3; Sec. 3.3 LSE equation).
 * Only the query rows listed in rows[0..n_rows) are computed (rows == NULL: all
 * n_tokens rows, n_rows must then equal n_tokens).
 *   out: [n_rows][n_heads][head_dim] double, lse: [n_heads][n_rows] double (natural log). */
int rvo_attend(const uint16_t *Q, const uint16_t *K, const uint16_t *V, int n_tokens,
               int n_heads, int head_dim,
               const uint16_t *memK, const uint16_t *memV, int64_t mem_len, int64_t head_stride,
               const int32_t *rows, int n_rows, double *out, double *lse);

/* Attention mass received by key columns (Sec. 3.3, saliency score and the A_ij
 * equation): for every head h and key column j,
 *   S[h][j] = sum over sampled queries i of exp(q_i . k_j / sqrt(head_dim) - LSE_i).
 * Keys are read at keys + j*key_tok_stride + h*key_head_stride (element strides), so the
 * same routine scores the current frame's keys (the saliency of the paper) or the memory
 * rows (a diagnostic used to check that each attention row sums to one).
 * qidx/lse_q: the n_q sampled query positions and their LSE values, lse_q[h][n_q]. */
int rvo_column_mass(const uint16_t *Q, int n_tokens, int n_heads, int head_dim,
                    const int32_t *qidx, int n_q, const double *lse_q,
                    const uint16_t *keys, int n_keys, int64_t key_tok_stride,
                    int64_t key_head_stride, double *S);

/* Per-head top-k (Sec. 3.3 Eq. 6 and "Head-Specific Token Retention"): order the
 * tokens of each head by saliency, highest first, ties broken towards the lower token
 * index; keep the first `budget`; return them in ascending index order.
 *   sal: [n_heads][n_tokens], idx: [n_heads][budget]. */
int rvo_topk(const double *sal, int n_tokens, int n_heads, int budget, int32_t *idx);

/* Memory update (Sec. 3.3 Eq. 6): append rows K_t[idx_h[r]][h], V_t[idx_h[r]][h],
 * r = 0..budget-1, to head h of the memory at rows mem_len..mem_len+budget-1.
 * head_stride must be >= mem_len + budget. */
int rvo_append(uint16_t *memK, uint16_t *memV, int64_t mem_len, int64_t head_stride,
               const uint16_t *K, const uint16_t *V, int n_tokens, int n_heads, int head_dim,
               const int32_t *idx, int budget);

/* Number of OpenMP threads the oracle runs with (for reporting). */
int rvo_num_threads(void);

#ifdef __cplusplus
}
#endif
#endif
