// rv_plan.h -- librv's kernel argument blocks and the host-side work planning that fills
// them (not installed).  Plain C++ with no HIP dependency, so the planning logic also
// builds with a host compiler alone (the sanitizer build of the tests does that).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/rv.h"

// Functions shared with the kernels are compiled for both sides under the HIP compiler.
#if defined(__HIPCC__)
#define RV_HD __host__ __device__
#else
#define RV_HD
#endif

namespace rv {

constexpr int kHeadDim = 64;     // head dimension supported by every kernel
constexpr int kAttnBQ = 128;     // queries per attention workgroup (4 waves x 32)
constexpr int kAttnBK = 64;      // keys per staged K/V tile
constexpr int kAttnThreads = 256;
constexpr int kAdmitThreads = 256;  // saliency and selection workgroups
constexpr int kMaxTokens = 16384;  // frame size limit (LDS-resident sampled queries and selected indices)
constexpr int kMaxLayersPerLaunch = 24;

constexpr int kMaxQueues = 16;     // work queues (one per XCD) in the attention kernel
constexpr int kAttnWgPerCu = 2;    // attention workgroups resident per CU
constexpr int kCutScale = 256;     // chunk lengths are planned in 1/256 iterations

// Attention forward with per-query LSE over [memory ; frame], XCD-local stream-K.
//
// A unit is (head, 128-query tile); its context is T key tiles of 64 keys.  Units are
// dealt to per-XCD queues (contiguous unit ranges); each queue's (unit, key tile)
// iteration space is cut into chunks of E tiles, chunk c of queue q going to workgroup
// c * n_queues + q, which the hardware places on queue q's XCD.  Chunk lengths are
// fractional (planned in 1/kCutScale tiles), so every workgroup slot gets a chunk.
struct AttnArgs {
  const uint16_t* Q;       // [N][H][64]
  const uint16_t* K;
  const uint16_t* V;
  const uint16_t* memK;    // [H][head_stride][64]
  const uint16_t* memV;
  int64_t mem_len;
  int64_t head_stride;
  uint16_t* out;           // [N][H][64]
  float* lse;              // [H][N]
  float* part;             // partial slots, kAttnSlotFloats each
  int n_tokens;            // queries (and, unless staged, the frame's keys)
  int n_fkeys;             // keys of the frame segment: n_tokens, or 0 when the frame's
                           // keys are staged in the arena and counted in mem_len
  int n_heads;
  int q_tiles;
  int nt_mem;              // key tiles of the memory segment
  int T;                   // key tiles per unit (memory + frame)
  int U;                   // iteration stride per unit: T (stream-K) or k * E >= T (k-way split)
  int n_units;             // n_heads * q_tiles
  int n_queues;
  int E;                   // chunk length in 1/kCutScale iterations (the first n_first
  int E1;                  //   chunks of a queue; E1: the later ones, E1 = E unless n_first > 0)
  int n_first;             // chunks per queue of E tiles; the rest hold E1
  int unit_base[kMaxQueues + 1];
  int n_chunks[kMaxQueues];
  int chunk_base[kMaxQueues];
};
// A partial slot: 128 output rows of 64 bf16, then the reference m[128] and sum l[128].
constexpr int kAttnSlotFloats = kAttnBQ * kHeadDim / 2 + 2 * kAttnBQ;
constexpr size_t kAttnSlotBytes = (size_t)kAttnSlotFloats * 4;
// Partial slots of the allocation-free attention entry point's static array (20.1 MB):
// more than the 1,040 the default plans on an MI355X (256 CUs, 8 XCDs) can take.
constexpr int kStaticScratchSlots = 1152;

// Saliency in the attention epilogue (Sec. 3.3, saliency score): the merge launch, once it
// has each query's final LSE, sums exp(z_ij - LSE_i) over the sampled queries of its
// 128-query block for every frame key j, into row b of tiles[h][b][j] (b = block).
struct SalEpi {
  float* tiles;            // [H][q_tiles][N]
  const uint16_t* K;       // frame keys: row j of head h at K + j * kv_row + h * kv_head
  int64_t kv_row;
  int64_t kv_head;
  int q_base;              // sampled query i of the frame: token q_base + r with r < grid_cells,
  int grid_w;              //   (r / grid_w) % stride == 0 and (r % grid_w) % stride == 0
  int grid_cells;
  int stride;
};

// One layer's share of the saliency / selection / append kernel.
struct AdmitLayer {
  const uint16_t* Q;       // [N][H][64]   (saliency)
  const uint16_t* K;       // frame keys: row j of head h at K + j * kv_row + h * kv_head
  const uint16_t* V;       //   (saliency, append); V likewise (append)
  int64_t kv_row;          // elements between a head's consecutive frame rows
  int64_t kv_head;         // elements between heads' rows of one token
  const float* lse;        // [H][N]       (saliency)
  float* sal;              // [H][N]       written by saliency, read by selection
                           //   ([H][sal_tiles][N] per-block rows when sal_tiles > 0)
  float* sal_out;          // [H][N]       the summed saliency (sal_tiles > 0; optional)
  int32_t* idx;            // [H][budget]  optional output
  uint16_t* memK;          // [H][head_stride][64]
  uint16_t* memV;
  int32_t* prov;           // [H][head_stride][2]
  int64_t mem_len;
  int64_t head_stride;
};

enum AdmitMode : int {
  kModeSaliency = 1,       // saliency only
  kModeSelect = 2,         // selection + append from a given saliency
  kModeBoth = 3,           // saliency, then selection + append (two launches)
};

struct AdmitArgs {
  AdmitLayer layer[kMaxLayersPerLaunch];
  int n_q;                 // sampled queries: token q_base + (i / q_cols) * q_row_stride
  int q_cols;              //   + (i % q_cols) * q_col_stride for i < n_q
  int q_base;
  int q_row_stride;
  int q_col_stride;
  int n_tokens;
  int n_heads;
  int n_layers;
  int budget;
  int frame_id;
  int mode;
  int stage_queries;       // saliency: stage the sampled query rows in LDS
  int q_pass;              // saliency: sampled query rows staged per pass (multiple of 32)
  int sal_groups;          // saliency: workgroups per (layer, head)
  int sal_xcds;            // saliency: XCDs the workgroup ids are dealt over (a head's groups
                           //   are numbered to share one; locality only)
  int shared_select;       // selection: one top-k per layer on the head sum, shared by all heads
  int in_place;            // selection: K, V are the staged rows of the destination arena, so
                           //   the append is an in-place compaction (read before write)
  int sal_tiles;           // selection: rows of per-block saliency per head, summed in block
                           //   order before the selection (0: one row, the saliency itself)
};

// Frames copied to staged arena rows, one layer per grid row (rv_mem_stage_frames).
struct StageLayer {
  uint16_t* dK;            // row j of head h goes to dK / dV + (h * head_stride + j) * 64
  uint16_t* dV;
  const uint16_t* K;       // the frame: [n_tokens][n_heads][64] bf16
  const uint16_t* V;
  int64_t head_stride;
};
struct StageArgs {
  StageLayer layer[kMaxLayersPerLaunch];
  int n_tokens;
  int n_heads;
  int n_layers;
};

constexpr int kSalQStride = kHeadDim + 8;  // staged sampled-query rows: 72 elements (144 bytes)
constexpr int kAdmitStaticLdsMargin = 4096;  // LDS left for the admission kernels' static arrays

// ---- attention work plan ------------------------------------------------------------

// Work plan of one attention launch: units (head, 128-query tile) are dealt in
// contiguous ranges to the per-XCD queues, and each queue's (unit, key tile) iterations
// are cut into chunks, one per workgroup, about kAttnWgPerCu per CU.
struct AttnPlan {
  int q_tiles, nt_mem, T, U, n_units, E, E1, n_first, grid, total_chunks;
  int unit_base[kMaxQueues + 1];
  int n_chunks[kMaxQueues];
  int chunk_base[kMaxQueues];
};

// Chunk arithmetic of a plan or of the kernel arguments built from it (both carry E, E1,
// n_first).  Chunk lengths are E (the first n_first chunks of a queue) and E1 in
// 1/kCutScale iterations, and chunk c starts at the iteration its scaled start rounds
// down to, so that the rounding is spread over all chunks.
// Chunk (of 8) that holds logical 16-byte chunk 0 of row r of an attention K/V tile in
// LDS (logical chunk c lies at c ^ attn_tile_swizzle(r)): 8 distinct values on every 8
// aligned rows, 16 distinct (row parity, value) pairs on every 16 (the kernels and the
// host checks share this).
RV_HD inline int attn_tile_swizzle(int r) { return ((2 * (r & 3)) | ((r >> 2) & 1)) ^ (((r >> 3) & 1) << 1); }

template <class A>
RV_HD inline int64_t chunk_cut(const A& a, int c) {
  const int64_t x = c < a.n_first ? (int64_t)c * a.E : (int64_t)a.n_first * a.E + (int64_t)(c - a.n_first) * a.E1;
  return x / kCutScale;
}
// The chunk holding iteration `it`: the last chunk that starts at or before it.
template <class A>
RV_HD inline int chunk_holding(const A& a, int64_t it) {
  const int64_t x = (it + 1) * kCutScale - 1, first = (int64_t)a.n_first * a.E;
  return x < first ? (int)(x / a.E) : a.n_first + (int)((x - first) / a.E1);
}
// Iterations [first, end) of chunk c of a queue of `iters` iterations.
template <class A>
RV_HD inline void chunk_iters(const A& a, int c, int64_t iters, int64_t* first, int64_t* end) {
  const int64_t e = chunk_cut(a, c + 1);
  *first = chunk_cut(a, c);
  *end = e < iters ? e : iters;
}

// Plan for n_tokens queries over mem_len memory keys then n_fkeys frame keys, on a
// device of n_cus CUs and n_queues XCDs (1..kMaxQueues).  Reads the RV_ATTN_* overrides.
AttnPlan plan_attention(int n_cus, int n_queues, int n_tokens, int n_fkeys, int64_t mem_len, int n_heads);

// Whether some unit's key range is split over several chunks (then a merge launch runs).
bool plan_splits_units(const AttnPlan& p);

// Partial slots a plan writes into: two per chunk (a chunk's segment of the unit it starts
// in, and of the unit it ends in).
inline int64_t plan_partial_slots(const AttnPlan& p) { return 2 * (int64_t)p.total_chunks; }

// Upper bound on plan_partial_slots of every plan on this device unless RV_ATTN_SPLIT forces
// a split (a chunk count set by the workgroup slots, whatever the sizes).
int64_t default_partial_slots(int n_cus, int n_queues);

// ---- query subset and admission launch shape -------------------------------------------

// NULL if qs describes a frame of n_tokens tokens, else a description of the problem.
const char* qsub_problem(const rv_qsub* qs, int n_tokens);

// Sampled queries (Sec. 3.3, head-specific retention): query i of the subset is frame
// token q_base + (i / q_cols) * q_row_stride + (i % q_cols) * q_col_stride, the
// top-left patch of the i-th stride x stride window in row-major window order.
void set_qsub(AdmitArgs* b, const rv_qsub& q);

// Dynamic LDS bytes the saliency and selection launches take, the larger of the two for
// the launches a.mode asks for, and the most they may use on a device whose per-workgroup
// LDS limit is max_lds.
size_t sal_lds_bytes(const AdmitArgs& a);
size_t select_lds_bytes(const AdmitArgs& a);
size_t admit_lds_bytes(const AdmitArgs& a);
int admit_max_dynamic_lds(int max_lds);

// Saliency launch shape for n_lh (layer, head) pairs on a device with n_cus CUs: sets
// a->sal_groups, a->q_pass and a->stage_queries (rows staged when they fit max_lds).
void plan_saliency(AdmitArgs* a, int n_lh, int n_cus, int max_lds);

// 32-key blocks [*b0, *b1) of a head's saliency group g: a.sal_groups equal shares of
// n_blocks, in order (the kernel and the host checks share this arithmetic).
RV_HD inline void sal_group_blocks(const AdmitArgs& a, int g, int n_blocks, int* b0, int* b1) {
  const int per = (n_blocks + a.sal_groups - 1) / a.sal_groups;
  const int s = g * per, e = s + per;
  *b0 = s < n_blocks ? s : n_blocks;
  *b1 = e < n_blocks ? e : n_blocks;
}

}  // namespace rv
