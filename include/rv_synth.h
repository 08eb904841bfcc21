/*
 * rv_synth.h -- C ABI of librv_synth: seeded synthetic token streams drawn on the GPU.
 *
 * Not part of the method.  It fills device buffers with the same bits as the CPU
 * generator (paper_2609_23286_amd/synth.py) so that a long benchmark stream -- every
 * frame of every layer distinct -- can be made resident in HBM before timing starts.
 * The recipe (Philox4x32-10 counters, order-8 Irwin-Hall near-Gaussian values rounded
 * to bf16, planted salient keys along the mean query direction) is documented in
 * synth.py; both implementations follow it step by step.
 *
 * Buffers are device memory owned by the caller; work is enqueued on `stream`
 * (a hipStream_t, NULL = default).  Returns 0 on success, 1 on invalid arguments,
 * 4 on a HIP error.
 */
#ifndef RV_SYNTH_H
#define RV_SYNTH_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* One frame of n_layers layers (layers layer0 .. layer0+n_layers-1):
 * out = [n_layers][3][n_tokens][n_heads][head_dim] bf16, the three tensors being Q, K, V
 * of that layer, each N(0, sigma^2)-like; with key_lognormal_sigma > 0 every key row is
 * then scaled by a log-normal factor exp(key_lognormal_sigma * xi) (heavy-tailed key
 * norms; the fp64 exponential may differ from the CPU generator's in its last bit, which
 * can move a rare key element by one bf16 step); then, per (layer, head), n_plant key rows
 * at Philox-drawn positions are replaced by alpha * |k| along the sum of that head's
 * queries.  n_tokens <= 8192, head_dim == 64. */
int rvs_frame_qkv(uint64_t seed, uint32_t frame, int layer0, int n_layers, int n_tokens,
                  int n_heads, int head_dim, float sigma, int n_plant, double alpha,
                  double key_lognormal_sigma, uint16_t *out, void *stream);

/* Unit-rate probe (benchmark support): n_workgroups workgroups of eight waves repeat a loop
 * of four independent 32x32x16 bf16 MFMAs and/or a loop of 16 v_exp_f32 with 32 FMA/add
 * iters times; ns_per_iter[11] receives the time per iteration with (0) one MFMA wave per
 * SIMD, (1) one VALU wave per SIMD, (2) one MFMA and one VALU wave per SIMD, (3) both
 * bodies in one wave per SIMD, (4) two MFMA waves per SIMD, (5) as (4) with all-zero MFMA
 * operands, (6) two VALU waves per SIMD, and for a loop of 32 independent FMAs (7) one,
 * (8) two waves per SIMD, of 32 independent v_exp_f32 (9) one, (10) two waves per SIMD.
 * Synchronous; allocates and frees its own output buffer. */
int rvs_unit_rates(int n_workgroups, int iters, float *ns_per_iter);

/* Near-Gaussian bf16 tensor of n elements for counter stream (frame, layer, tag). */
int rvs_normal_bf16(uint64_t seed, uint32_t frame, int layer, int tag, int64_t n, float sigma,
                    uint16_t *out, void *stream);

#ifdef __cplusplus
}
#endif
#endif
