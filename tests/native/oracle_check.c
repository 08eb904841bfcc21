/* oracle_check.c -- drives every function of the CPU oracle (oracle/rvo.c) on small
 * inputs, including its edge cases (empty memory, no sampled query, budget 0 and N,
 * one-token frames).  Built with AddressSanitizer and UndefinedBehaviorSanitizer by
 * tests/test_sanitizers.py: any out-of-bounds access, use of freed memory, signed
 * overflow or similar undefined behaviour aborts the run.  Also checks that each
 * query's attention row sums to one and that argument errors are reported.
 * Prints "oracle OK". */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../oracle/rvo.h"

static int g_fail = 0;
#define CHECK(c, msg)                                                  \
    do {                                                               \
        if (!(c)) {                                                    \
            fprintf(stderr, "FAIL %s:%d: %s\n", __FILE__, __LINE__, msg); \
            ++g_fail;                                                  \
        }                                                              \
    } while (0)

static uint32_t g_state = 12345u;
static uint16_t rand_bf16(void)
{
    /* values of magnitude < 1: sign, exponent 120..126, random mantissa */
    g_state = g_state * 1664525u + 1013904223u;
    const uint32_t r = g_state >> 8;
    const uint16_t sign = (uint16_t)((r & 1u) << 15);
    const uint16_t expo = (uint16_t)((120u + (r >> 1) % 7u) << 7);
    return (uint16_t)(sign | expo | ((r >> 4) & 0x7Fu));
}

static void fill(uint16_t *p, size_t n)
{
    for (size_t i = 0; i < n; i++)
        p[i] = rand_bf16();
}

static void run_case(int grid_h, int grid_w, int n_special, int stride, int H, int M, int budget)
{
    const int d = 64, N = grid_h * grid_w + n_special;
    const int cap = M + budget;
    uint16_t *Q = malloc(sizeof(uint16_t) * (size_t)N * H * d);
    uint16_t *K = malloc(sizeof(uint16_t) * (size_t)N * H * d);
    uint16_t *V = malloc(sizeof(uint16_t) * (size_t)N * H * d);
    uint16_t *mK = malloc(sizeof(uint16_t) * (size_t)(cap > 0 ? cap : 1) * H * d);
    uint16_t *mV = malloc(sizeof(uint16_t) * (size_t)(cap > 0 ? cap : 1) * H * d);
    double *out = malloc(sizeof(double) * (size_t)N * H * d);
    double *lse = malloc(sizeof(double) * (size_t)H * N);
    double *S = malloc(sizeof(double) * (size_t)H * N);
    double *Smem = malloc(sizeof(double) * (size_t)H * (M > 0 ? M : 1));
    int32_t *idx = malloc(sizeof(int32_t) * (size_t)H * (budget > 0 ? budget : 1));
    fill(Q, (size_t)N * H * d);
    fill(K, (size_t)N * H * d);
    fill(V, (size_t)N * H * d);
    fill(mK, (size_t)(cap > 0 ? cap : 1) * H * d);
    fill(mV, (size_t)(cap > 0 ? cap : 1) * H * d);

    const int n_q = rvo_qsub_index(grid_h, grid_w, n_special, stride, NULL, 0);
    CHECK(n_q >= 0, "qsub count");
    int32_t *qidx = malloc(sizeof(int32_t) * (size_t)(n_q > 0 ? n_q : 1));
    CHECK(rvo_qsub_index(grid_h, grid_w, n_special, stride, qidx, n_q) == n_q, "qsub fill");

    CHECK(rvo_attend(Q, K, V, N, H, d, mK, mV, M, cap, NULL, N, out, lse) == 0, "attend");
    /* the rows of a sampled subset, with their LSE */
    double *lse_q = malloc(sizeof(double) * (size_t)H * (n_q > 0 ? n_q : 1));
    for (int h = 0; h < H; h++)
        for (int a = 0; a < n_q; a++)
            lse_q[(int64_t)h * n_q + a] = lse[(int64_t)h * N + qidx[a]];
    CHECK(rvo_column_mass(Q, N, H, d, qidx, n_q, lse_q, K, N, (int64_t)H * d, d, S) == 0, "frame mass");
    if (M > 0)
        CHECK(rvo_column_mass(Q, N, H, d, qidx, n_q, lse_q, mK, M, d, (int64_t)cap * d, Smem) == 0, "memory mass");
    /* total mass over the whole context is the number of sampled queries */
    for (int h = 0; h < H; h++) {
        double tot = 0.0;
        for (int j = 0; j < N; j++)
            tot += S[(int64_t)h * N + j];
        for (int c = 0; c < M; c++)
            tot += Smem[(int64_t)h * M + c];
        CHECK(fabs(tot - n_q) <= 1e-9 * (n_q > 0 ? n_q : 1), "total saliency differs from n_q");
    }
    CHECK(rvo_topk(S, N, H, budget, idx) == 0, "topk");
    for (int h = 0; h < H; h++)
        for (int r = 1; r < budget; r++)
            CHECK(idx[(int64_t)h * budget + r - 1] < idx[(int64_t)h * budget + r], "indices ascend");
    CHECK(rvo_append(mK, mV, M, cap, K, V, N, H, d, idx, budget) == 0, "append");
    /* argument errors are reported, not acted on */
    CHECK(rvo_topk(S, N, H, N + 1, idx) != 0, "budget > N accepted");
    CHECK(rvo_append(mK, mV, M, cap, K, V, N, H, d, idx, budget + 1) != 0 || budget + 1 > N,
          "append past capacity accepted");
    CHECK(rvo_qsub_index(-1, 1, 0, 1, NULL, 0) < 0, "negative grid accepted");
    free(Q); free(K); free(V); free(mK); free(mV); free(out); free(lse); free(S); free(Smem);
    free(idx); free(qidx); free(lse_q);
}

int main(void)
{
    run_case(8, 8, 0, 2, 2, 0, 1);     /* the tiny stream's first frame */
    run_case(8, 8, 0, 2, 2, 7, 1);
    run_case(8, 8, 0, 1, 2, 65, 3);    /* every query sampled */
    run_case(0, 5, 4, 2, 2, 10, 2);    /* no sampled query: every saliency 0 */
    run_case(1, 1, 0, 1, 1, 0, 1);     /* one token, budget = N (anchor frame) */
    run_case(3, 5, 2, 2, 3, 130, 0);   /* budget 0 */
    run_case(4, 5, 1, 3, 2, 64, 21);   /* budget = N */
    if (g_fail) {
        fprintf(stderr, "%d checks failed\n", g_fail);
        return 1;
    }
    printf("oracle OK\n");
    return 0;
}
