// rv_internal.h -- shared between librv's host code and its gfx950 kernels (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rv {

constexpr int kHeadDim = 64;     // head dimension supported by every kernel
constexpr int kAttnBQ = 128;     // queries per attention workgroup (4 waves x 32)
constexpr int kAttnBK = 64;      // keys per staged K/V tile
constexpr int kAttnThreads = 256;
constexpr int kMaxSplits = 16;   // split-KV partitions per (head, query tile)
constexpr int kSalBK = 128;      // keys per saliency workgroup (4 waves x 32)
constexpr int kAdmitThreads = 256;
constexpr int kMaxTokens = 16384;  // frame size limit (LDS-resident sampled queries and selected indices)
constexpr int kMaxLayersPerLaunch = 24;

// Attention forward with per-query LSE over [memory ; frame].
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
  float* part_o;           // [H*q_tiles][n_splits][BQ][64] fp32, unnormalised
  float* part_ml;          // [H*q_tiles][n_splits][2][BQ]: running max (log2 units), row sum
  int* counters;           // [H*q_tiles] split completion counters, self-resetting
  int n_tokens;
  int n_heads;
  int q_tiles;
  int n_splits;
  int nt_mem;              // key tiles in the memory segment
  int nt_total;            // nt_mem + key tiles in the frame segment
  int n_work;              // H * q_tiles * n_splits
  int per_xcd;             // workgroups mapped to each XCD (grid = 8 * per_xcd)
};

// One layer's share of the saliency / selection / append kernel.
struct AdmitLayer {
  const uint16_t* Q;       // [N][H][64]   (saliency)
  const uint16_t* K;       // [N][H][64]   (saliency, append)
  const uint16_t* V;       // [N][H][64]   (append)
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
  kModeBoth = 3,           // saliency, then the last workgroup of a head selects + appends
};

struct AdmitArgs {
  AdmitLayer layer[kMaxLayersPerLaunch];
  const int32_t* qidx;     // [n_q] sampled query positions
  int* counters;           // [n_layers*H], self-resetting
  int n_q;
  int n_tokens;
  int n_heads;
  int n_layers;
  int budget;
  int frame_id;
  int key_chunks;          // ceil(N / kSalBK)
  int mode;
};

hipError_t launch_attention(const AttnArgs& a, hipStream_t s);
hipError_t launch_admit(const AdmitArgs& a, hipStream_t s);

}  // namespace rv
