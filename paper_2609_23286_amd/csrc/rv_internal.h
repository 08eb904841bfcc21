// rv_internal.h -- shared between librv's host code and its gfx950 kernels (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

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

// Attention forward with per-query LSE over [memory ; frame], XCD-local stream-K.
//
// A unit is (head, 128-query tile); its context is T key tiles of 64 keys.  Units are
// dealt to per-XCD queues (contiguous unit ranges); each queue's (unit, key tile)
// iteration space is cut into chunks of E tiles, chunk c of queue q going to workgroup
// c * n_queues + q, which the hardware places on queue q's XCD.
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
  int E;                   // key tiles per chunk (the first n_first chunks of a queue)
  int E1;                  // key tiles per later chunk (E1 = E unless n_first > 0)
  int n_first;             // chunks per queue of E tiles; the rest hold E1
  int unit_base[kMaxQueues + 1];
  int n_chunks[kMaxQueues];
  int chunk_base[kMaxQueues];
};
constexpr int kAttnSlotFloats = kAttnBQ * kHeadDim / 2 + 2 * kAttnBQ;  // bf16 rows + m, l

// One layer's share of the saliency / selection / append kernel.
struct AdmitLayer {
  const uint16_t* Q;       // [N][H][64]   (saliency)
  const uint16_t* K;       // frame keys: row j of head h at K + j * kv_row + h * kv_head
  const uint16_t* V;       //   (saliency, append); V likewise (append)
  int64_t kv_row;          // elements between a head's consecutive frame rows
  int64_t kv_head;         // elements between heads' rows of one token
  const float* lse;        // [H][N]       (saliency)
  float* sal;              // [H][N]       written by saliency, read by selection
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
  int shared_select;       // selection: one top-k per layer on the head sum, shared by all heads
  int in_place;            // selection: K, V are the staged rows of the destination arena, so
                           //   the append is an in-place compaction (read before write)
};

hipError_t launch_attention(const AttnArgs& a, int grid, bool merge, hipStream_t s);
// Copies a frame's K, V ([n][H][64] bf16) to staged arena rows: row j of head h goes to
// dK / dV + (h * head_stride + j) * 64.
hipError_t launch_stage(uint16_t* dK, uint16_t* dV, int64_t head_stride, const uint16_t* K, const uint16_t* V,
                        int n, int H, hipStream_t s);
// Records the hardware XCC id of each of n_blocks workgroups into ids (device memory).
hipError_t launch_xcc_probe(int* ids, int n_blocks, hipStream_t s);
// Dynamic LDS bytes the admission kernels need for these arguments (the larger of the
// saliency and selection launches), and the most they may use on a device whose
// per-workgroup LDS limit is max_lds (room is left for the kernels' static LDS).
constexpr int kAdmitStaticLdsMargin = 4096;
size_t admit_lds_bytes(const AdmitArgs& a);
int admit_max_dynamic_lds(int max_lds);
// max_lds: the device's LDS limit per workgroup (bytes), for the kernel attribute.
hipError_t launch_admit(const AdmitArgs& a, int max_lds, hipStream_t s);
// Saliency launch shape for n_lh (layer, head) pairs on a device with n_cus CUs: sets
// a->sal_groups and a->stage_queries (rows staged when they fit max_lds).
void plan_saliency(AdmitArgs* a, int n_lh, int n_cus, int max_lds);

}  // namespace rv
