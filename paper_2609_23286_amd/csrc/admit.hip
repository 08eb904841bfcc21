// admit.hip -- LSE-saliency, per-head top-k and memory append, gfx950.
//
// Two launches per call, each spread over the whole chip:
//
// sal_kernel (Sec. 3.3, saliency score and the A_ij equation): for key j of the frame,
//   S_j = sum over sampled queries i of exp(q_i . k_j / 8 - LSE_i),
// with the LSE the attention pass saved, so every term is an exact attention
// probability and no score matrix is stored.  A (layer, head) is split over
// `sal_groups` workgroups of 4 wave64s (about three per CU over the launch), each taking
// a contiguous range of 32-key blocks.  The sampled query rows and their LSE are staged
// in LDS once per workgroup; each wave then takes its blocks two at a time (K rows in
// registers) and sweeps the sampled queries in blocks of 32 with
// v_mfma_f32_32x32x16_bf16 (Z = Q~ K^T, each lane owning one key column), each block's
// accumulator seeded with -8 LSE of its rows so that the MFMAs leave 8 (z - LSE).  The
// exponentials are summed in fp32 in a fixed order -- pairwise in-lane, over query
// blocks, then across the two lane halves -- so S is bit-reproducible with no atomics.
// The vector-ALU work is one multiply, one exp and one add per (query, key).
//
// select_kernel (Sec. 3.3 Eq. 6, head-specific retention): one workgroup per
// (layer, head) takes the `budget` largest S_j, equal values ordered by lower index.
// The order is that of the 64-bit key (bits of S, ~j): fp32 bit patterns order like
// the values for S >= 0.  Budgets up to kWaveTopK: each wave extracts the top `budget`
// of its quarter by repeated wave-wide maxima, and one wave extracts the top `budget` of
// the 4 x budget candidates the same way.  Larger budgets: an MSB-first radix select
// over the bit patterns finds the threshold value and how many of its ties to take, and
// block scans emit the indices.  Either way the indices come out ascending and the
// chosen K/V rows are copied to the memory arena at rows mem_len.. with their
// provenance.
#include <type_traits>

#include "rv_internal.h"

namespace rv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int D = kHeadDim;
constexpr int NT = kAdmitThreads;  // 256
constexpr int NW = NT / 64;
constexpr int kBlocksPerStep = 2;  // 32-key blocks a saliency wave holds at once
static_assert(kBlocksPerStep == 2, "a range's last step holds one block or two");
constexpr int QS_STRIDE = kSalQStride;  // staged sampled-query rows, 144 bytes
constexpr int kPrefetchQBlock = 4;  // query block of a step at which the next step's K rows are requested
constexpr int kStageBatch = 9;     // 16-byte query-row loads in flight per thread (one pass of 288 rows)
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kScaleLog2 = kLog2e * 0.125f;

static_assert(NT == 256, "the radix histogram has one bin per thread");

// ---- saliency -----------------------------------------------------------------------

// The two query-row sources are separate instantiations, so that neither path's
// memory waits are merged into the other's loop.
template <bool kStaged>
__device__ __forceinline__ void sal_body(const AdmitArgs& a, unsigned char* smem) {
  const int H = a.n_heads, N = a.n_tokens, tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, half = lane >> 5;
  const int groups = a.sal_groups;
  // Workgroup b runs on XCD b % X (ids are dealt round-robin over the XCDs): group g of
  // (layer, head) lh = l_x X + x is id (g HX + l_x) X + x (HX = pairs per XCD), all of a
  // head's groups on XCD x, so the head's sampled query rows and LSE that every group
  // stages are read once from memory and then from that XCD's L2.  The first groups of
  // all heads come first, so a head's groups are dispatched in different rounds and the
  // later ones find the head's rows in L2.  Placement only affects speed.
  const int X = a.sal_xcds > 0 ? a.sal_xcds : 1;
  const int HX = (a.n_layers * H + X - 1) / X;
  const int xcd = blockIdx.x % X, rr = blockIdx.x / X;
  const int g = rr / HX, lh = (rr - g * HX) * X + xcd;
  if (g >= groups || lh >= a.n_layers * H) return;  // uniform: ids past the last (layer, head)
  // (uniform: the layer's operand addresses then live in scalar registers)
  const int layer = __builtin_amdgcn_readfirstlane(lh / H), h = __builtin_amdgcn_readfirstlane(lh - layer * H);
  const int n_blocks = (N + 31) / 32;
  int blk0, blk1;
  sal_group_blocks(a, g, n_blocks, &blk0, &blk1);
  if (blk0 >= blk1) return;  // uniform over the workgroup
  // The layer's operands, read once: this head's frame keys, query rows, LSE and
  // saliency row.
  const AdmitLayer& L = a.layer[layer];
  const int64_t kv_row = L.kv_row;
  const uint16_t* Kh = L.K + (int64_t)h * L.kv_head;
  const uint16_t* Qh = L.Q + (int64_t)h * D;
  const float* lse_h = L.lse + (int64_t)h * N;
  float* sal_h = L.sal + (int64_t)h * N;
  const int nq_pad = (a.n_q + 31) & ~31;
  if (nq_pad == 0) {  // no sampled queries: every key's saliency is the empty sum
    for (int j = blk0 * 32 + tid; j < min(N, blk1 * 32); j += NT) sal_h[j] = 0.f;
    return;
  }
  float* s_nlse8 = reinterpret_cast<float*>(smem);
  uint16_t* s_q = reinterpret_cast<uint16_t*>(smem + (size_t)nq_pad * 4);

  // -8 LSE of the sampled queries (the initial value of the score accumulators, so that
  // an accumulator ends as q.k - 8 LSE = 8 (z - LSE); padding rows: -inf -> weight 0)
  // and, when they fit, the sampled query rows (padding rows zero), a pass of q_pass
  // rows at a time.  Every load reads a clamped, valid address and padding is selected
  // afterwards, so no load sits behind a branch with a wait of its own: the LSE loads go
  // out together, then each batch of kStageBatch row loads per thread, and the K rows of
  // the wave's first step are requested after the staged data, so that the staging
  // does not wait for them.
  auto q_token = [&](int i) {
    const int qi = i / a.q_cols;
    return a.q_base + qi * a.q_row_stride + (i - qi * a.q_cols) * a.q_col_stride;
  };
  // K rows (B operands, K^T) of a step's blocks: lane's key, dims ds*16 + half*8 ..;
  // a pass's first step's rows are requested after its staging, each next step's rows
  // while the current step computes.
  auto load_k = [&](int bb, bf16x8 (&kf)[kBlocksPerStep][4]) {
#pragma unroll
    for (int b = 0; b < kBlocksPerStep; ++b) {
      const int j = min((bb + b) * 32 + l32, N - 1);  // past the frame or the range: result unused
      const uint16_t* kp = Kh + (int64_t)j * kv_row + half * 8;
#pragma unroll
      for (int ds = 0; ds < 4; ++ds) kf[b][ds] = *reinterpret_cast<const bf16x8*>(kp + ds * 16);
    }
  };
  auto lse_load = [&](int i0, float (&v)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * NT + tid;
      const float x = lse_h[q_token(min(i, a.n_q - 1))];
      v[u] = i < a.n_q ? x : __builtin_inff();
    }
  };
  auto lse_store = [&](int i0, const float (&v)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * NT + tid;
      if (i < nq_pad) s_nlse8[i] = -8.0f * v[u];
    }
  };
  // 16-byte chunk c (row p0 + c/8) of a pass's query rows
  auto rows_load = [&](int p0, int c0, uint4 (&v)[kStageBatch]) {
#pragma unroll
    for (int u = 0; u < kStageBatch; ++u) {
      const int c = c0 + u * NT + tid, i = p0 + (c >> 3), ch = c & 7;
      const uint4 x = *reinterpret_cast<const uint4*>(Qh + (int64_t)q_token(min(i, a.n_q - 1)) * H * D + ch * 8);
      v[u] = i < a.n_q ? x : uint4{0u, 0u, 0u, 0u};
    }
  };
  auto rows_store = [&](int rows, int c0, const uint4 (&v)[kStageBatch]) {
#pragma unroll
    for (int u = 0; u < kStageBatch; ++u) {
      const int c = c0 + u * NT + tid, ch = c & 7;
      if (c < rows * 8) *reinterpret_cast<uint4*>(&s_q[(c >> 3) * QS_STRIDE + ch * 8]) = v[u];
    }
  };
  bf16x8 kf[kBlocksPerStep][4], kn[kBlocksPerStep][4];
  for (int i0 = 0; i0 < nq_pad; i0 += NT * 4) {
    float lv[4];
    lse_load(i0, lv);
    lse_store(i0, lv);
  }

  // Passes over the sampled queries; each key's sum is carried from pass to pass by the
  // lane that owns it (fixed order).
  const int q_pass = kStaged ? a.q_pass : nq_pad;
  for (int p0 = 0; p0 < nq_pad; p0 += q_pass) {
    const int p1 = min(nq_pad, p0 + q_pass), rows = p1 - p0;
    if (kStaged) {
      for (int c0 = 0; c0 < rows * 8; c0 += NT * kStageBatch) {
        uint4 qv[kStageBatch];
        rows_load(p0, c0, qv);
        rows_store(rows, c0, qv);
      }
    }
    load_k(blk0 + wave * kBlocksPerStep, kf);  // (a wave without blocks loads rows it never uses)
    __syncthreads();

    for (int bb = blk0 + wave * kBlocksPerStep; bb < blk1; bb += NW * kBlocksPerStep) {
      // The next step's K rows are requested a few query blocks into this step, not at
      // its start: every workgroup of the launch stages at once, and the workgroups
      // served first would otherwise queue their next step's rows ahead of the staging
      // loads of those served last.
      const bool prefetch = bb + NW * kBlocksPerStep < blk1;
      const int q_prefetch = p0 + 32 * min(kPrefetchQBlock, (p1 - p0) / 32 - 1);
      // NB blocks held (the range's last step may hold fewer than kBlocksPerStep).
      auto sweep = [&](auto nb_c) {
        constexpr int NB = decltype(nb_c)::value;
        float acc[NB] = {};
        // A operand (query rows qb + l32) of a query block, from LDS or memory.
        auto load_q = [&](int qb, bf16x8 (&qf)[4]) {
          if (kStaged) {
#pragma unroll
            for (int ds = 0; ds < 4; ++ds)
              qf[ds] = *reinterpret_cast<const bf16x8*>(&s_q[(qb - p0 + l32) * QS_STRIDE + ds * 16 + half * 8]);
          } else {
            const uint16_t* qp = Qh + (int64_t)q_token(min(qb + l32, a.n_q - 1)) * H * D + half * 8;
#pragma unroll
            for (int ds = 0; ds < 4; ++ds) qf[ds] = *reinterpret_cast<const bf16x8*>(qp + ds * 16);
          }
        };
        bf16x8 qf[4];
        load_q(p0, qf);
        for (int qb = p0; qb < p1; qb += 32) {
          if (prefetch && qb == q_prefetch) load_k(bb + NW * kBlocksPerStep, kn);
          // Wave priority 0 for the MFMAs, 1 from the next block's row reads through the
          // exponentials: of the waves sharing a SIMD, those in their vector work issue
          // first, so the MFMAs of the others run under it (about -2 % per launch against a
          // uniform priority; priority changes no result).
          __builtin_amdgcn_s_setprio(0);
          // Each block's accumulator starts at -8 LSE of its 16 rows (queries
          // qb + 8*(r/4) + 4*half + r%4), so the MFMAs leave 8 (z - LSE) in it and the
          // two blocks' chains are independent.
          f32x16 z[NB];
#pragma unroll
          for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
              const float4 v = *reinterpret_cast<const float4*>(&s_nlse8[qb + 8 * r4 + 4 * half]);
              z[b][4 * r4] = v.x;
              z[b][4 * r4 + 1] = v.y;
              z[b][4 * r4 + 2] = v.z;
              z[b][4 * r4 + 3] = v.w;
            }
#pragma unroll
          for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int ds = 0; ds < 4; ++ds) z[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[ds], kf[b][ds], z[b], 0, 0, 0);
          __builtin_amdgcn_s_setprio(1);
          if (qb + 32 < p1) load_q(qb + 32, qf);  // the next block's rows, under this block's exponentials
#pragma unroll
          for (int b = 0; b < NB; ++b) {
            // exp(z - LSE) = 2^(8 (z - LSE) log2(e) / 8), all 16 independent, then a fixed
            // pairwise sum.
            float e[16];
#pragma unroll
            for (int r = 0; r < 16; ++r) e[r] = __builtin_amdgcn_exp2f(z[b][r] * kScaleLog2);
#pragma unroll
            for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
              for (int r = 0; r < w; ++r) e[r] = e[r] + e[r + w];
            acc[b] += e[0];
          }
        }
        __builtin_amdgcn_s_setprio(0);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          const float tot = acc[b] + __shfl_xor(acc[b], 32);
          const int j = (bb + b) * 32 + l32;
          if (half == 0 && j < N) {
            if (p0 == 0)  // uniform
              sal_h[j] = tot;
            else
              sal_h[j] += tot;
          }
        }
      };
      if (bb + kBlocksPerStep <= blk1)  // uniform
        sweep(std::integral_constant<int, kBlocksPerStep>{});
      else
        sweep(std::integral_constant<int, 1>{});
#pragma unroll
      for (int b = 0; b < kBlocksPerStep; ++b)
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) kf[b][ds] = kn[b][ds];
    }
    if (p1 < nq_pad) __syncthreads();  // the staged rows are replaced by the next pass
  }
}

__global__ __launch_bounds__(NT, 3) void sal_kernel(AdmitArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  if (a.stage_queries)
    sal_body<true>(a, smem);
  else
    sal_body<false>(a, smem);
}

// ---- selection and append -----------------------------------------------------------

// Exclusive prefix sum over the workgroup's threads (every thread must call it).
__device__ int block_exclusive_scan(int v, int* s_wave) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int u = __shfl_up(x, off);
    if (lane >= off) x += u;
  }
  if (lane == 63) s_wave[wave] = x;
  __syncthreads();
  int base = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) base += w < wave ? s_wave[w] : 0;
  __syncthreads();
  return base + x - v;
}

// Top-`budget` of sal[0..N) (ties -> lower index), ascending, into s_idx[0..budget).
__device__ void select_topk(const float* sal, int N, int budget, int32_t* s_idx) {
  __shared__ unsigned int hist[256];
  __shared__ int s_wave[NW];
  __shared__ int s_bin, s_need;
  const int tid = threadIdx.x, lane = tid & 63;

  if (budget >= N) {
    for (int j = tid; j < N; j += NT) s_idx[j] = j;
    __syncthreads();
    return;
  }
  // Radix select, 8 bits per pass from the top: candidates share the prefix found so
  // far; the bin whose upper-tail count first reaches `need` holds the threshold.
  unsigned int prefix = 0u, mask = 0u;
  int need = budget;
  for (int shift = 24; shift >= 0; shift -= 8) {
    hist[tid] = 0u;  // NT == 256 bins
    __syncthreads();
    for (int j = tid; j < N; j += NT) {
      const unsigned int kj = __float_as_uint(sal[j]);
      if ((kj & mask) == prefix) atomicAdd(&hist[(kj >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane i holds bins 255-4i .. 252-4i (descending); suffix counts by a wave scan
      unsigned int c[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) c[m] = hist[255 - 4 * lane - m];
      const unsigned int tot = c[0] + c[1] + c[2] + c[3];
      unsigned int x = tot;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const unsigned int u = __shfl_up(x, off);
        if (lane >= off) x += u;
      }
      unsigned int ge = x - tot;  // elements in bins above this lane's first bin
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const unsigned int gt = ge;
        ge += c[m];
        if (gt < (unsigned int)need && (unsigned int)need <= ge) {
          s_bin = 255 - 4 * lane - m;
          s_need = need - (int)gt;
        }
      }
    }
    __syncthreads();
    prefix |= (unsigned int)s_bin << shift;
    mask |= 255u << shift;
    need = s_need;
  }
  const unsigned int tau = prefix;  // the budget-th largest value; take `need` of its ties

  // Each thread owns a contiguous run of indices; two scans give the tie ranks and the
  // output positions in index order.
  const int E = (N + NT - 1) / NT;
  const int j0 = min(N, tid * E), j1 = min(N, j0 + E);
  int n_gt = 0, n_eq = 0;
  for (int j = j0; j < j1; ++j) {
    const unsigned int kj = __float_as_uint(sal[j]);
    n_gt += kj > tau;
    n_eq += kj == tau;
  }
  const int eq_before = block_exclusive_scan(n_eq, s_wave);
  const int take_eq = max(0, min(n_eq, need - eq_before));
  const int n_sel = n_gt + take_eq;
  int pos = block_exclusive_scan(n_sel, s_wave);
  int eq_seen = eq_before;
  for (int j = j0; j < j1; ++j) {
    const unsigned int kj = __float_as_uint(sal[j]);
    bool sel = kj > tau;
    if (kj == tau) {
      sel = eq_seen < need;
      ++eq_seen;
    }
    if (sel && pos < budget) s_idx[pos++] = j;
  }
  __syncthreads();
}

// Order key of token j: saliency bits above, ~j below, so larger keys are larger
// saliencies and, among equal ones, lower indices.  0 marks "no candidate".
__device__ __forceinline__ uint64_t rank_key(float v, int j) {
  return ((uint64_t)__float_as_uint(v) << 32) | (uint32_t)~(uint32_t)j;
}

template <int CTRL>
__device__ __forceinline__ uint32_t max_dpp(uint32_t x) {
  return max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false));
}

// The larger value of the pair a v_permlane*_swap leaves: the two lanes' values, in some
// order on every lane.
template <class Pair>
__device__ __forceinline__ uint32_t pair_max(const Pair& p) {
  return max((uint32_t)p[0], (uint32_t)p[1]);
}

// Maximum over the wave's 64 lanes, left on every lane: DPP within each 16-lane row
// (quad swaps, half mirror, mirror: each a max with a DPP operand), then rows paired by
// v_permlane16_swap and halves by v_permlane32_swap.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
  x = max_dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  x = max_dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  x = max_dpp<0x141>(x);  // row_half_mirror
  x = max_dpp<0x140>(x);  // row_mirror
  x = pair_max(__builtin_amdgcn_permlane16_swap(x, x, false, false));
  return pair_max(__builtin_amdgcn_permlane32_swap(x, x, false, false));
}

// The largest 64-bit key of the wave, on every lane, in two 32-bit reductions: the
// largest upper half (the saliency bits), then the largest lower half (~index) among
// the lanes holding that upper half.
__device__ __forceinline__ uint64_t wave_max_key(uint64_t k) {
  const uint32_t hi = wave_max_u32((uint32_t)(k >> 32));
  const uint32_t lo = wave_max_u32((uint32_t)(k >> 32) == hi ? (uint32_t)k : 0u);
  return ((uint64_t)hi << 32) | lo;
}

// Top-`budget` (budget <= kWaveTopK) of sal[0..N), ascending, into s_idx.  Wave w owns
// tokens [w*Q, (w+1)*Q), lane l the tokens w*Q + l + 64 m (m < kLaneSlots), kept as
// keys sorted in registers.  Each round the wave's best remaining key is found by a
// wave-wide maximum and its lane drops it.  Wave 0 then extracts the top `budget` of
// the 4 x budget winners the same way (two per lane) and orders them by index.
constexpr int kWaveTopK = 32;
static_assert(NW * kWaveTopK <= 128, "the final extraction holds two candidates per lane");
constexpr int kLaneSlots = 8;  // tokens per lane: the wave path takes N <= 4 * 64 * 8

__device__ void select_small(const float* sal, int N, int budget, int32_t* s_idx, uint64_t* s_cand) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Q = (N + NW - 1) / NW;
  const int lo = min(N, wave * Q), hi = min(N, lo + Q);
  uint64_t v[kLaneSlots];
#pragma unroll
  for (int m = 0; m < kLaneSlots; ++m) {
    const int j = lo + lane + 64 * m;
    v[m] = j < hi ? rank_key(sal[j], j) : 0;
  }
#pragma unroll
  for (int i = 0; i < kLaneSlots - 1; ++i) {  // descending
#pragma unroll
    for (int m = 0; m < kLaneSlots - 1 - i; ++m) {
      const uint64_t x = v[m], y = v[m + 1];
      v[m] = x > y ? x : y;
      v[m + 1] = x > y ? y : x;
    }
  }
  for (int r = 0; r < budget; ++r) {
    const uint64_t win = wave_max_key(v[0]);
    if (lane == 0) s_cand[wave * budget + r] = win;
    if (win != 0 && win == v[0]) {  // this lane owns the winner (keys are distinct)
#pragma unroll
      for (int m = 0; m < kLaneSlots - 1; ++m) v[m] = v[m + 1];
      v[kLaneSlots - 1] = 0;
    }
  }
  __syncthreads();
  if (wave == 0) {
    // The overall top `budget` lie among the NW * budget winners: two per lane, sorted.
    const int nc = NW * budget;
    uint64_t c0 = lane < nc ? s_cand[lane] : 0, c1 = lane + 64 < nc ? s_cand[lane + 64] : 0;
    if (c1 > c0) {
      const uint64_t t = c0;
      c0 = c1;
      c1 = t;
    }
    uint32_t mine = 0;  // lane r: ~index of the r-th winner
    for (int r = 0; r < budget; ++r) {
      const uint64_t win = wave_max_key(c0);
      if (lane == r) mine = (uint32_t)win;
      if (win == c0) {  // (a real key: fewer than budget + 1 tokens never reach this path)
        c0 = c1;
        c1 = 0;
      }
    }
    // lane r < budget: output slot = number of winners with a lower index
    const uint32_t jr = ~mine;
    int pos = 0;
    for (int u = 0; u < budget; ++u) pos += ~(uint32_t)__builtin_amdgcn_readlane((int)mine, u) < jr;
    if (lane < budget) s_idx[pos] = (int32_t)jr;
  }
  __syncthreads();
}

// Head-specific retention (the paper's rule, Sec. 3.3): one workgroup per (layer, head)
// ranks that head's saliency.  Shared selection (the arm without head-specific
// retention in the ablation of Sec. 4.5, Table 4): every head's workgroup ranks the sum
// over heads of the saliencies (summed in head order, so every workgroup of a layer
// reaches the same selection; it orders tokens as the mean does) and appends those
// tokens to its own head.
__global__ __launch_bounds__(NT) void select_kernel(AdmitArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ uint64_t s_cand[NW * kWaveTopK];
  const int H = a.n_heads, N = a.n_tokens, k = a.budget, tid = threadIdx.x;
  const int layer = blockIdx.x / H, h_own = blockIdx.x - layer * H;
  const AdmitLayer& L = a.layer[layer];
  float* s_sal = reinterpret_cast<float*>(smem);
  int32_t* s_idx = reinterpret_cast<int32_t*>(smem + (((size_t)N * 4 + 15) & ~(size_t)15));

  if (a.shared_select) {
    for (int j = tid; j < N; j += NT) {
      float acc = 0.f;
      for (int h = 0; h < H; ++h) acc += L.sal[(int64_t)h * N + j];
      s_sal[j] = acc;
    }
  } else if (a.sal_tiles > 0) {
    // per-block saliency rows of this head (computed in the attention epilogue), summed
    // in block order; the sum is the saliency, written out when asked for
    // (eight rows' loads in flight per step)
    const int T = a.sal_tiles;
    const float* gs = L.sal + (int64_t)h_own * T * N;
    for (int j = tid; j < N; j += NT) {
      float acc = 0.f;
      for (int t0 = 0; t0 < T; t0 += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = t0 + u < T ? gs[(int64_t)(t0 + u) * N + j] : 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (t0 + u < T) acc = (t0 + u == 0) ? v[u] : acc + v[u];
      }
      s_sal[j] = acc;
      if (L.sal_out) L.sal_out[(int64_t)h_own * N + j] = acc;
    }
  } else {
    const float* gs = L.sal + (int64_t)h_own * N;
    if ((N & 3) == 0) {
      for (int j = tid; j < N / 4; j += NT)
        reinterpret_cast<float4*>(s_sal)[j] = reinterpret_cast<const float4*>(gs)[j];
    } else {
      for (int j = tid; j < N; j += NT) s_sal[j] = gs[j];
    }
  }
  __syncthreads();
  if (k <= kWaveTopK && k < N && N <= NW * 64 * kLaneSlots)
    select_small(s_sal, N, k, s_idx, s_cand);
  else
    select_topk(s_sal, N, k, s_idx);
  {
    const int h = h_own;
    if (L.idx)
      for (int r = tid; r < k; r += NT) L.idx[(int64_t)h * k + r] = s_idx[r];
    // 16-byte chunks: 8 per K row, 8 per V row.
    if (!a.in_place) {
      for (int c = tid; c < k * 16; c += NT) {
        const int r = c >> 4, part = c & 15, chunk = part & 7;
        const int j = s_idx[r];
        if (j < 0 || j >= N) continue;  // unreachable: the selection emits exactly k indices < N
        const int64_t src = (int64_t)j * L.kv_row + (int64_t)h * L.kv_head + chunk * 8;
        const int64_t dst = ((int64_t)h * L.head_stride + L.mem_len + r) * D + chunk * 8;
        if (part < 8)
          *reinterpret_cast<uint4*>(L.memK + dst) = *reinterpret_cast<const uint4*>(L.K + src);
        else
          *reinterpret_cast<uint4*>(L.memV + dst) = *reinterpret_cast<const uint4*>(L.V + src);
      }
    } else {
      // Compaction inside the arena: the staged row idx[r] moves to row mem_len + r.
      // Indices ascend, so idx[r] >= r: passes of NT / 16 rows in ascending order read
      // all of a pass's sources before writing its destinations, and no later pass reads
      // a row an earlier one wrote (its sources lie at or past its own destinations).
      for (int r0 = 0; r0 < k; r0 += NT / 16) {
        const int r = r0 + (tid >> 4), part = tid & 15, chunk = part & 7;
        uint4 v = make_uint4(0, 0, 0, 0);
        int64_t dst = -1;
        if (r < k) {
          const int j = s_idx[r];
          if (j >= 0 && j < N) {  // always: the selection emits exactly k indices < N
            const int64_t src = (int64_t)j * L.kv_row + (int64_t)h * L.kv_head + chunk * 8;
            v = *reinterpret_cast<const uint4*>((part < 8 ? L.K : L.V) + src);
            dst = ((int64_t)h * L.head_stride + L.mem_len + r) * D + chunk * 8;
          }
        }
        __syncthreads();
        if (dst >= 0) *reinterpret_cast<uint4*>((part < 8 ? L.memK : L.memV) + dst) = v;
        __syncthreads();
      }
    }
    for (int r = tid; r < k; r += NT) {
      int32_t* pv = L.prov + ((int64_t)h * L.head_stride + L.mem_len + r) * 2;
      pv[0] = a.frame_id;
      pv[1] = s_idx[r];
    }
  }
}

hipError_t set_lds_limit(const void* kernel, int* cached, int limit) {
  if (*cached == limit) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, limit);
  if (e == hipSuccess) *cached = limit;
  return e;
}

}  // namespace

hipError_t launch_admit(const AdmitArgs& a, int max_lds, hipStream_t s) {
  static int sal_attr = 0, sel_attr = 0;
  const int limit = admit_max_dynamic_lds(max_lds);
  if (a.mode & kModeSaliency) {
    hipError_t e = set_lds_limit((const void*)sal_kernel, &sal_attr, limit);
    if (e != hipSuccess) return e;
    const unsigned X = (unsigned)(a.sal_xcds > 0 ? a.sal_xcds : 1);
    const unsigned n_lh = (unsigned)(a.n_layers * a.n_heads);
    const unsigned grid = (n_lh + X - 1) / X * X * (unsigned)a.sal_groups;
    hipLaunchKernelGGL(sal_kernel, dim3(grid), dim3(NT), sal_lds_bytes(a), s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if ((a.mode & kModeSelect) && a.budget > 0) {
    hipError_t e = set_lds_limit((const void*)select_kernel, &sel_attr, limit);
    if (e != hipSuccess) return e;
    const unsigned grid = (unsigned)(a.n_layers * a.n_heads);
    hipLaunchKernelGGL(select_kernel, dim3(grid), dim3(NT), select_lds_bytes(a), s, a);
    return hipGetLastError();
  }
  return hipSuccess;
}

namespace {

// One thread per 16-byte chunk of the frame (8 per row of 64 bf16), in the frame's order.
__global__ __launch_bounds__(256) void stage_kernel(uint16_t* dK, uint16_t* dV, int64_t head_stride,
                                                    const uint16_t* K, const uint16_t* V, int n, int H) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= (int64_t)n * H * 8) return;
  const int chunk = (int)(c & 7);
  const int64_t row = c >> 3;  // token * H + head
  const int h = (int)(row % H);
  const int64_t j = row / H;
  const int64_t d = ((int64_t)h * head_stride + j) * D + chunk * 8;
  *reinterpret_cast<uint4*>(dK + d) = reinterpret_cast<const uint4*>(K)[c];
  *reinterpret_cast<uint4*>(dV + d) = reinterpret_cast<const uint4*>(V)[c];
}

// Several layers' frames in one launch: blockIdx.y is the layer.
__global__ __launch_bounds__(256) void stage_layers_kernel(StageArgs a) {
  const StageLayer& L = a.layer[blockIdx.y];
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= (int64_t)a.n_tokens * a.n_heads * 8) return;
  const int chunk = (int)(c & 7);
  const int64_t row = c >> 3;  // token * H + head
  const int h = (int)(row % a.n_heads);
  const int64_t j = row / a.n_heads;
  const int64_t d = ((int64_t)h * L.head_stride + j) * D + chunk * 8;
  *reinterpret_cast<uint4*>(L.dK + d) = reinterpret_cast<const uint4*>(L.K)[c];
  *reinterpret_cast<uint4*>(L.dV + d) = reinterpret_cast<const uint4*>(L.V)[c];
}

}  // namespace

hipError_t launch_stage(uint16_t* dK, uint16_t* dV, int64_t head_stride, const uint16_t* K, const uint16_t* V,
                        int n, int H, hipStream_t s) {
  const int64_t chunks = (int64_t)n * H * 8;
  hipLaunchKernelGGL(stage_kernel, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, s, dK, dV, head_stride,
                     K, V, n, H);
  return hipGetLastError();
}

hipError_t launch_stage_layers(const StageArgs& a, hipStream_t s) {
  const int64_t chunks = (int64_t)a.n_tokens * a.n_heads * 8;
  hipLaunchKernelGGL(stage_layers_kernel, dim3((unsigned)((chunks + 255) / 256), (unsigned)a.n_layers), dim3(256), 0,
                     s, a);
  return hipGetLastError();
}

}  // namespace rv
