/*
 * rv.h -- C ABI of librv, the MI355X (gfx950) library for RegVGGT's per-frame hot path.
 *
 * For each transformer layer, one incoming frame of N tokens is
 *   1. attended over that layer's regulated KV memory plus its own tokens
 *      (temporal-causal attention, Sec. 3.1 Eq. 2-3), keeping each query's
 *      log-sum-exp (Sec. 3.3, LSE equation);
 *   2. scored: each key of the frame gets the attention mass it receives from a 2x2
 *      spatially sampled subset of the frame's queries, recovered from the LSE without
 *      forming any score matrix (Sec. 3.3, saliency score and the A_ij equation);
 *   3. regulated: per head, the `budget` most salient tokens are appended to the memory
 *      (Sec. 3.3 Eq. 6; budget = floor(gamma * N), gamma = 0.01 in the paper).
 *
 * General conventions
 *   - Every tensor pointer named in a compute call is a DEVICE pointer on the current
 *     HIP device, owned by the caller, unless stated otherwise.
 *   - bf16 means bfloat16: the upper 16 bits of an IEEE-754 binary32, stored as 2-byte
 *     little-endian words; values the library produces in bf16 are rounded to nearest
 *     (ties to even).
 *   - Frame tensors Q, K, V, out: [n_tokens][n_heads][head_dim] bf16, contiguous (the
 *     layout a fused QKV projection writes).  Per-head vectors (lse, saliency):
 *     [n_heads][n_tokens] fp32.  Memory: [n_heads][head_stride][head_dim] bf16, rows
 *     0..mem_len-1 of each head valid.
 *   - head_dim must be 64 (the ViT-L aggregator's 1024 / 16).
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the default stream) and is
 *     asynchronous; nothing here synchronises the device except where stated.
 *   - Set-up: rv_init (or rv_mem_create, or rv_reserve_workspace, which call it) must
 *     have run on the current device before a compute call.  It records the device's
 *     limits and allocates the scratch workspace, so that the compute calls
 *     (rv_attend_frame, rv_attend_staged, rv_admit*) never allocate scratch memory or
 *     synchronise; only the memory arenas grow, inside rv_admit* and rv_mem_* calls.
 *   - Every argument is checked before anything is enqueued.  On failure the call
 *     returns a non-zero rv_status, enqueues nothing, changes no state, and
 *     rv_last_error() describes the problem.  A fault in an earlier kernel surfaces as
 *     RV_ERR_HIP from the next call that reaches the HIP runtime.
 *   - Calls that share an rv_mem, or that run concurrently on one device, must be
 *     ordered on one stream: the library's scratch workspace is shared per device.
 *   - The library never aborts the process.
 *   - Environment overrides of the attention work plan (tests and tuning only; results
 *     are the same under every plan, to the stated tolerances): RV_ATTN_SPLIT (0:
 *     stream-K chunks, k > 0: every unit cut into k aligned pieces), RV_ATTN_WG_PER_CU
 *     (workgroups per CU the plan fills, default 2), RV_ATTN_MIN_CHUNK (smallest chunk
 *     in 64-key tiles, default 2), RV_ATTN_SPLIT_SLACK (tiles by which the aligned split
 *     may exceed stream-K before stream-K is taken, default 1), RV_ATTN_FIRST_PCT (tiles
 *     of a stream-K chunk served by a workgroup dispatched first on its CU, in per cent
 *     of the others'; by default the share that makes the later chunks end on unit
 *     boundaries when one lies in 115-160, else 140).
 */
#ifndef RV_H
#define RV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rv_status {
    RV_OK = 0,
    RV_ERR_INVALID = 1,  /* bad argument: null pointer, size, unsupported shape */
    RV_ERR_OOM = 2,      /* a device allocation failed; state unchanged */
    RV_ERR_CAPACITY = 3, /* memory growth would exceed the rv_mem's max_tokens */
    RV_ERR_HIP = 4,      /* the HIP runtime reported an error */
    RV_ERR_IO = 5        /* a file could not be read or written, or is not a memory snapshot */
} rv_status;

/* One layer's regulated KV memory ("context memory" M_t of Sec. 3.3 Eq. 4-6): K and V
 * arenas [n_heads][capacity][head_dim] bf16, a provenance record per row
 * [n_heads][capacity][2] int32 = (frame_id, token index in that frame), and the number
 * of valid rows, which is the same for every head because every head admits exactly
 * `budget` rows per frame (Eq. 6).  The library owns all of it. */
typedef struct rv_mem_s *rv_mem;

/* Query subset for the saliency score (Sec. 3.3, head-specific retention): the frame is
 * n_special leading special tokens (camera, register) followed by a grid_h x grid_w
 * patch grid in row-major order.  The grid is cut into stride x stride windows and the
 * top-left patch of each window is a sampled query; windows cut by the right or bottom
 * edge count too.  Special tokens are never sampled (they are still scored and may be
 * admitted).  stride 2 is the paper's setting; stride 1 samples every patch. */
typedef struct rv_qsub {
    int32_t grid_h, grid_w, n_special, stride;
} rv_qsub;

/* Human-readable description of the last failure on the calling thread.  The pointer
 * stays valid until the next rv_* call on that thread. */
const char *rv_last_error(void);

/* Library version string. */
const char *rv_version(void);

/* Initialises librv on the current device (idempotent): reads its CU count and LDS
 * limit, counts its XCDs with a probe launch, and allocates the split-KV workspace that
 * every default attention work plan fits (about 18 MB on an MI355X; see
 * rv_reserve_workspace for plans forced through the RV_ATTN_* overrides).  Synchronises
 * the device.  Compute calls on a device where it has not run return RV_ERR_INVALID. */
rv_status rv_init(void);

/* ---- memory (Sec. 3.3 Eq. 4-6) ---------------------------------------------------- */

/* Creates an empty memory on the current device with room for reserve_tokens rows per
 * head (0 allowed) that may grow to max_tokens rows per head.  head_dim must be 64. */
rv_status rv_mem_create(int n_heads, int head_dim, int64_t reserve_tokens, int64_t max_tokens,
                        rv_mem *out);

/* Frees the memory (synchronises its device first).  NULL is accepted. */
rv_status rv_mem_destroy(rv_mem m);

/* Number of valid rows per head, as enqueued (a host-side mirror; no device sync). */
int64_t rv_mem_len(rv_mem m);

/* Rows per head currently allocated. */
int64_t rv_mem_capacity(rv_mem m);

/* Device pointers of the K and V arenas and the row stride between heads (in tokens),
 * suitable for rv_attend_frame.  Growth (in rv_admit*, rv_mem_reserve) moves the
 * arenas: take a fresh view after any call that may grow the memory. */
rv_status rv_mem_view(rv_mem m, const void **memK, const void **memV,
                      int64_t *head_stride_tokens);

/* Ensures capacity >= tokens (<= max_tokens).  Growth is stream-ordered on `stream` and
 * does not synchronise: new arenas (hipMallocAsync), a copy of the valid rows, and the
 * release of the old arenas (hipFreeAsync) are enqueued in that order, so work on
 * another stream must wait for `stream` before it uses the grown memory.  Arenas at
 * creation are ready for every stream. */
rv_status rv_mem_reserve(rv_mem m, int64_t tokens, void *stream);

/* Sets the length to 0 (arena contents are left as they are). */
rv_status rv_mem_reset(rv_mem m);

/* Drops the newest rows: sets the length to n_rows, 0 <= n_rows <= length (RV_ERR_INVALID
 * otherwise), e.g. to roll a memory back to an earlier frame.  Rows past the new length
 * keep their contents until overwritten.  Host-side only: no device work. */
rv_status rv_mem_truncate(rv_mem m, int64_t n_rows);

/* Overwrites rows 0..n_rows-1 of every head with K, V ([n_heads][n_rows][head_dim]
 * bf16, host or device memory) and sets the length to n_rows; provenance of these rows
 * becomes (frame_id, row).  Used to prefill a memory or to restore a snapshot.
 * Synchronous with respect to the host. */
rv_status rv_mem_write(rv_mem m, const void *K, const void *V, int64_t n_rows, int frame_id,
                       void *stream);

/* Copies rows 0..len-1 of every head into K, V ([n_heads][len][head_dim] bf16) and
 * prov ([n_heads][len][2] int32); each destination may be NULL to skip it, and may be
 * host or device memory.  Synchronous with respect to the host. */
rv_status rv_mem_read(rv_mem m, void *K, void *V, int32_t *prov, void *stream);

/* Snapshot of a memory (checkpoint / resume of a stream): writes the valid rows of every
 * head, with their provenance, to `path` (little-endian: 8-byte magic "RVMEMv1\0",
 * int32 n_heads, int32 head_dim, int64 length, then K [n_heads][length][64] bf16,
 * V likewise, provenance [n_heads][length][2] int32).  Synchronises the memory's
 * device.  RV_ERR_IO if the file cannot be written. */
rv_status rv_mem_save(rv_mem m, const char *path);

/* Restores a snapshot written by rv_mem_save into m: the head count must match, the
 * length must not exceed m's max_tokens; m grows as needed.  The file is read and
 * checked completely before m changes, so on any failure (RV_ERR_IO for an unreadable
 * or malformed file, RV_ERR_INVALID for a mismatch, RV_ERR_CAPACITY, RV_ERR_OOM) m is
 * left unchanged.  Synchronous with respect to the host. */
rv_status rv_mem_load(rv_mem m, const char *path);

/* ---- the per-frame hot path ---------------------------------------------------------- */

/* Temporal-causal attention of one frame over memory + frame (Sec. 3.1 Eq. 3): for
 * head h and query i, the context is memory rows 0..mem_len-1 of head h followed by
 * the frame's own n_tokens keys, with no mask inside the frame;
 *   z_ic = q_i . k_c / sqrt(head_dim),  LSE_i = log sum_c exp(z_ic)   (natural log),
 *   out_i = sum_c exp(z_ic - LSE_i) v_c.
 * Q, K, V, out: [n_tokens][n_heads][64] bf16.  memK, memV: [n_heads][head_stride][64]
 * bf16 (mem_len 0 allows NULL).  lse: [n_heads][n_tokens] fp32, required.
 * saliency: NULL, or [n_heads][n_tokens] fp32 that receives, for every frame key j,
 *   S_j = sum over sampled queries i (per *qs) of exp(z_ij - LSE_i)     (Sec. 3.3),
 * in which case qs must be given and describe n_tokens.
 * (A subset with no window -- grid_h or grid_w 0 -- gives S_j = 0, the empty sum.)
 * Arithmetic: bf16 inputs, fp32 logits and softmax, probabilities rounded to bf16 for
 * the value product, fp32 accumulation, out rounded to bf16 (nearest-even).
 * n_tokens 0 is a no-op.  Allocates nothing and does not synchronise: split-KV partial
 * results go to the workspace rv_init allocated (RV_ERR_INVALID if rv_init has not run
 * on this device; RV_ERR_CAPACITY if an RV_ATTN_* override forces a plan with more
 * partial slots than rv_reserve_workspace provided). */
rv_status rv_attend_frame(const void *Q, const void *K, const void *V, int n_tokens,
                          const void *memK, const void *memV, int64_t mem_len,
                          int64_t head_stride_tokens, int n_heads, int head_dim,
                          const rv_qsub *qs, void *out, float *lse, float *saliency,
                          void *stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): rv_attend_frame with the same
 * arguments, results and errors, except that its split-KV partial results live in a
 * static array the library holds on every GPU it runs on (1,152 slots of 17,408 bytes,
 * 20.1 MB, kept until the process ends) instead of the rv_init workspace.  It calls no
 * allocating routine; rv_init must have run on the device (it records the array's
 * address there).  A work plan that needs more than 1,152 partial slots (only forced
 * RV_ATTN_* plans can) is refused with RV_ERR_CAPACITY before anything is enqueued.
 * Nothing in the array needs clearing between calls (each call writes every slot it
 * reads), but all calls on one GPU share it: calls that overlap on one GPU (on
 * different streams) race and must be ordered by the caller. */
rv_status rv_attend_frame_noalloc(const void *Q, const void *K, const void *V, int n_tokens,
                                  const void *memK, const void *memV, int64_t mem_len,
                                  int64_t head_stride_tokens, int n_heads, int head_dim,
                                  const rv_qsub *qs, void *out, float *lse, float *saliency,
                                  void *stream);

/* ---- saliency in the attention epilogue ------------------------------------------------
 *
 * The saliency needs each sampled query's final LSE, which exists only once the key range
 * of the query's 128-query block has been merged; these two calls form it there, right
 * after the attention, from the frame's keys the attention has just read, and leave the
 * top-k to a later launch that needs no keys.  The saliency of key j is split by query
 * block: S_j = sum over b of S_j^(b), with
 *   S_j^(b) = sum over sampled queries i in [RV_QUERY_BLOCK b, RV_QUERY_BLOCK (b + 1))
 *             of exp(z_ij - LSE_i)                                      (Sec. 3.3). */
#define RV_QUERY_BLOCK 128

/* rv_attend_frame (same arguments, layouts, arithmetic and errors; qs required) that also
 * writes, per head h and query block b < ceil(n_tokens / RV_QUERY_BLOCK), the row
 * sal_tiles[h][b][0 .. n_tokens-1] = S_j^(b) (fp32, summed in a fixed order: the same
 * inputs give the same bits).  sal_tiles: [n_heads][ceil(n_tokens / 128)][n_tokens] fp32,
 * device memory, every entry written. */
rv_status rv_attend_frame_fused(const void *Q, const void *K, const void *V, int n_tokens,
                                const void *memK, const void *memV, int64_t mem_len,
                                int64_t head_stride_tokens, int n_heads, int head_dim,
                                const rv_qsub *qs, void *out, float *lse, float *sal_tiles, void *stream);

/* Admission (Sec. 3.3 Eq. 6) of n_layers layers in one launch from the per-block saliency
 * rv_attend_frame_fused wrote: per layer and head, S_j is the sum of the rows b = 0, 1, ...
 * in that order; then the selection and the append of rv_admit_layers.  sal_tiles: host
 * array of n_layers device pointers ([n_heads][ceil(n_tokens / 128)][n_tokens] fp32).
 * saliency_out, idx_out: NULL, or host arrays of n_layers device pointers (each may be
 * NULL) receiving S ([n_heads][n_tokens] fp32) and the selection ([n_heads][budget]).
 * Otherwise as rv_admit_layers (K, V, mems, frame_id, budget, growth and errors). */
rv_status rv_admit_layers_tiled(int n_layers, const float *const *sal_tiles, int n_tokens, int budget,
                                const void *const *K, const void *const *V, const rv_mem *mems,
                                int frame_id, float *const *saliency_out, int32_t *const *idx_out,
                                void *stream);

/* Admission from a given saliency (Sec. 3.3 Eq. 6): per head, selects the `budget`
 * tokens of largest saliency -- equal saliencies ordered by lower token index -- and
 * appends their K and V rows (exact copies) to m in ascending token order; the length
 * grows by `budget` at once on the host.  saliency: [n_heads][n_tokens] fp32, finite,
 * >= 0.  K, V: the frame's [n_tokens][n_heads][64] bf16.  idx_out: NULL or
 * [n_heads][budget] int32 receiving the selected indices, ascending.
 * 0 <= budget <= n_tokens <= 16384; budget == n_tokens appends every token (the anchor
 * frame of Eq. 4, or full retention).  Grows m if needed (RV_ERR_CAPACITY beyond
 * max_tokens, RV_ERR_OOM on allocation failure; m unchanged in both cases). */
rv_status rv_admit(const float *saliency, int budget, const void *K, const void *V,
                   int n_tokens, rv_mem m, int frame_id, int32_t *idx_out, void *stream);

/* Deferred admission for n_layers layers of one frame in one launch: for layer l,
 * computes the saliency of Q[l], K[l] against lse[l] (as rv_attend_frame would),
 * then selects and appends exactly as rv_admit does into mems[l].  Bit-identical to
 * per-layer rv_attend_frame(..., saliency) + rv_admit.  Layer l's memory must not be
 * read by this frame's attention after this call (Eq. 6 makes admissions visible from
 * the next frame on).  Q, K, V, lse, mems: host arrays of n_layers device pointers /
 * handles.  saliency_out, idx_out: NULL, or host arrays of n_layers device pointers
 * ([n_heads][n_tokens] fp32, [n_heads][budget] int32), each of which may be NULL.
 * All layers share n_heads, n_tokens, qs, budget.  1 <= n_layers <= 4096.  Without a
 * saliency output for every layer the workspace's saliency staging is used: it must hold
 * min(n_layers, 24) layers' values (rv_reserve_workspace), else RV_ERR_CAPACITY. */
rv_status rv_admit_layers(int n_layers, const void *const *Q, const void *const *K,
                          const void *const *V, const float *const *lse, int n_tokens,
                          const rv_qsub *qs, int budget, const rv_mem *mems, int frame_id,
                          float *const *saliency_out, int32_t *const *idx_out, void *stream);

/* Head-averaged admission, the arm without head-specific retention in the ablation of
 * Sec. 4.5 (Table 4): exactly as rv_admit_layers, except that each layer selects once,
 * on the sum over heads of the saliency (summed in head order; it ranks tokens as the
 * mean over heads does, ties to the lower index), and every head appends the same
 * tokens.  idx_out[l], if given, receives that selection in every head's row. */
rv_status rv_admit_layers_shared(int n_layers, const void *const *Q, const void *const *K,
                                 const void *const *V, const float *const *lse, int n_tokens,
                                 const rv_qsub *qs, int budget, const rv_mem *mems, int frame_id,
                                 float *const *saliency_out, int32_t *const *idx_out,
                                 void *stream);

/* ---- staged frame: the frame's keys and values written straight into the arena ---------
 *
 * A producer (the layer's K/V projection) can write the frame's K and V directly into
 * the memory's arena, past its valid rows, instead of into separate [n][H][64] tensors.
 * Attention then reads one contiguous key range per head (memory rows followed by the
 * frame), the saliency reads the frame's keys from there, and admission (Sec. 3.3 Eq. 6)
 * becomes an in-place compaction: the selected rows move down to the end of the memory
 * and the rest of the staged rows are dropped.  Given the same K and V, attention
 * results equal the frame entry points' within the same error bounds, and bit for bit
 * when the memory length is a multiple of 64 (the 64-key tiles then coincide; otherwise
 * the frame's keys start mid-tile and the fp32 sums run in another order); admission
 * given the same LSE is bit-identical. */

/* Stages a frame of n_tokens rows: ensures capacity >= length + n_tokens (growing, and so
 * moving, the arenas if needed: RV_ERR_CAPACITY / RV_ERR_OOM leave m unchanged) and
 * returns the device address of row `length` of head 0 in the K and V arenas and the
 * row stride between heads.  Row j of head h of the frame goes to
 * K_tail + (h * head_stride_tokens + j) * 64 (bf16), likewise for V.  The length is not
 * changed; any call that grows m drops the staged rows.  Outputs may be NULL. */
rv_status rv_mem_stage(rv_mem m, int n_tokens, void **K_tail, void **V_tail,
                       int64_t *head_stride_tokens, void *stream);

/* rv_mem_stage, then copies a frame given as [n_tokens][n_heads][64] bf16 K, V (device
 * memory) into the staged rows, on `stream`. */
rv_status rv_mem_stage_frame(rv_mem m, const void *K, const void *V, int n_tokens, void *stream);

/* rv_mem_stage_frame for n_layers memories (one per layer, equal head counts) and their
 * frames K[l], V[l], with one copy launch for up to 24 layers.  Every memory gets its
 * room before anything is enqueued: a failure (RV_ERR_INVALID for a NULL pointer or
 * differing head counts, RV_ERR_CAPACITY / RV_ERR_OOM from the growth of layer l) copies
 * nothing, though layers before l may have grown (dropping nothing: their length is
 * unchanged). */
rv_status rv_mem_stage_frames(int n_layers, const rv_mem *mems, const void *const *K, const void *const *V,
                              int n_tokens, void *stream);

/* rv_attend_frame (Sec. 3.1 Eq. 3, Sec. 3.3 LSE and saliency) for a frame staged in m:
 * the keys and values of head h are arena rows 0 .. length + n_tokens - 1 of m, i.e. the
 * memory followed by the staged frame.  Q, out: [n_tokens][n_heads][64] bf16; lse,
 * saliency (NULL, or with qs): [n_heads][n_tokens] fp32.  RV_ERR_INVALID if fewer than
 * n_tokens rows are staged (capacity < length + n_tokens). */
rv_status rv_attend_staged(const void *Q, int n_tokens, rv_mem m, const rv_qsub *qs, void *out,
                           float *lse, float *saliency, void *stream);

/* rv_admit_layers (Sec. 3.3 saliency and Eq. 6) for frames staged in mems: layer l's
 * saliency uses the staged keys of mems[l]; its `budget` selected rows (ascending token
 * order) are compacted in place to rows length .. length + budget - 1 with provenance
 * (frame_id, token) and the length grows by `budget`.  No memory grows here; every
 * layer must have n_tokens rows staged (RV_ERR_INVALID otherwise). */
rv_status rv_admit_staged_layers(int n_layers, const void *const *Q, const float *const *lse,
                                 int n_tokens, const rv_qsub *qs, int budget, const rv_mem *mems,
                                 int frame_id, float *const *saliency_out, int32_t *const *idx_out,
                                 void *stream);

/* Synchronises the current device and reports any error the HIP runtime recorded for
 * earlier work (RV_ERR_HIP with the runtime's message).  Test harnesses call it after
 * each step. */
rv_status rv_device_status(void);

/* Work plan the attention launch uses for one frame (introspection for tests and
 * tuning; touches no device and allocates nothing).  n_cus and n_queues (XCDs, 1..16)
 * describe the device; the library's own launches use the counts it reads at start-up,
 * and the RV_ATTN_* overrides apply here as there.  Query tiles of 128 and key tiles of
 * 64 make n_units = n_heads * q_tiles units of T key tiles each; queue q owns units
 * unit_base[q] .. unit_base[q+1]-1, laid out as iterations i = u * U + t (t < U; tiles
 * t >= T are padding).  Chunk lengths E (the first n_first chunks of a queue) and E1
 * (the others) are in 1/256 iterations: chunk c (0 <= c < n_chunks[q]) of queue q covers
 * iterations [cut(c), min(cut(c+1), units_q * U)) with cut(c) = floor(c E / 256) for
 * c < n_first and floor((n_first E + (c - n_first) E1) / 256) after; chunk_base[q]
 * numbers the chunks of all queues consecutively, and grid = n_queues * max(n_chunks)
 * workgroups are launched.
 * RV_ERR_INVALID for out-of-range sizes or a NULL `out`. */
typedef struct rv_attn_plan {
    int n_units, q_tiles, T, U, E, E1, n_first, n_queues, grid, total_chunks;
    int unit_base[17];
    int n_chunks[16];
    int chunk_base[16];
} rv_attn_plan;
rv_status rv_attention_plan(int n_tokens, int n_fkeys, int64_t mem_len, int n_heads, int n_cus,
                            int n_queues, rv_attn_plan *out);

/* Grows the current device's scratch workspace (calling rv_init first if needed): the
 * split-KV partial slots of the work plan for frames of n_tokens tokens and n_heads heads
 * over memories of up to max_mem_len rows -- the default plans fit the workspace rv_init
 * allocates; plans forced through RV_ATTN_SPLIT may need more -- and the saliency
 * staging that rv_admit_layers* use when the caller passes no saliency output, for up to
 * n_layers layers per call.  The workspace never shrinks.  Synchronises the device when
 * it replaces a buffer. */
rv_status rv_reserve_workspace(int n_tokens, int n_heads, int64_t max_mem_len, int n_layers);

#ifdef __cplusplus
}
#endif
#endif
