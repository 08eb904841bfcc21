// attend.hip -- temporal-causal attention forward with per-query log-sum-exp, gfx950.
//
// Computes, for one frame and one layer (Sec. 3.1 Eq. 2-3 and the LSE equation of
// Sec. 3.3), for every head h and query i of the frame:
//   z_ic = q_i . k_c / 8 over the context c = [memory rows of h ; the frame's keys],
//   LSE_i = log sum_c exp(z_ic),  o_i = sum_c exp(z_ic - LSE_i) v_c.
//
// Design (CDNA4):
// * Work unit = (head, 128-query tile); 4 wave64s, 32 queries each.  Key/value tiles of
//   64 rows go straight from global memory into LDS (global_load_lds_dwordx4), row-major
//   with an XOR swizzle, through a 4-stage ring whose stage offsets are compile-time
//   constants: two tiles are computed per barrier while the next two stream in.
// * Scores are formed transposed, S^T = K Q^T (v_mfma_f32_32x32x16_bf16), so each lane
//   owns one query column: softmax max/sum are in-lane plus one exchange between the
//   two 32-lane halves sharing a query.  The output is accumulated transposed too,
//   O^T += V^T P^T: P^T is the score accumulator itself (its 16 rows per lane are the
//   8+8 keys the B operand wants), and V^T comes straight from the row-major V tile
//   through ds_read_b64_tr_b16 transposing reads.
// * Online softmax in base 2 with 1/sqrt(64) folded into one FMA.  Probabilities are
//   taken against a running reference that is only raised when a tile could overflow
//   (tile sums >= 2^64), so neither tile maxima nor accumulator rescales are computed in
//   the common case (exact either way: the LSE uses the reference the sums were taken
//   against).
// * Scheduling: 1041 queries x 16 heads is only 144 units, too few for 256 CUs, so each
//   unit's key range is split.  Units are dealt to one queue per XCD (whole heads where
//   possible); each queue's (unit, key tile) iterations, laid out with a stride of U
//   tiles per unit, are cut into chunks, one per workgroup.  With U = T (the unit's
//   tile count) this is stream-K: chunks may straddle units, and the first n_first
//   chunks of a queue (served by the workgroups dispatched first on their CUs, which
//   run faster) hold E tiles against E1 for the rest.  With
//   U = k E >= T every unit is cut into k aligned pieces, so the workgroups holding the
//   query tiles of one head walk the same key tiles at the same time and share them in
//   L2.  A chunk that covers a whole unit writes its output directly; otherwise it
//   writes a partial result (its output normalised by its own row sum, in bf16, with
//   its reference m and row sum l) to its slot and a second launch merges each split
//   unit's partials in chunk order (deterministic; the kernel boundary is the only
//   synchronisation, so results do not depend on where the hardware places the
//   workgroups; the merge workgroups follow the queues' XCD mapping only so that the
//   partials are likely still in that XCD's L2).
#include <type_traits>

#include "rv_internal.h"

namespace rv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BQ = kAttnBQ;
constexpr int BK = kAttnBK;
constexpr int D = kHeadDim;
constexpr int TILE = BK * D;                    // one K or V tile: 64 rows x 128 bytes
constexpr int STAGE = 2 * TILE;                 // K tile then V tile
constexpr int NSTAGE = 4;                       // LDS ring: two tiles computed, two in flight
constexpr float kLn2 = 0.69314718055994531f;
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kScaleLog2 = 1.44269504088896341f * 0.125f;  // log2(e) / sqrt(64)
constexpr float kOverflowGuard = 18446744073709551616.0f;  // 2^64
constexpr float kNegBig = -1.0e30f;

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

template <int P>
struct StageConst {
  static constexpr int value = P;
};

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint2 to_bf16x4(float a, float b, float c, float d) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
  return __builtin_bit_cast(uint2, v);
}

__device__ __forceinline__ int hw_xcc_id() { return __builtin_amdgcn_s_getreg((3 << 11) | 20) & 15; }

// Partner value of the other 32-lane half (lane l <-> l ^ 32): v_permlane32_swap returns
// the two halves exchanged between its operands, so the pair holds {own, partner} in
// some order on every lane; sums and maxima over the pair need no lane test.
__device__ __forceinline__ float half_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// LDS tile layout: 64 rows of 128 bytes, no padding.  The 16-byte chunk c of row r is
// stored at chunk c ^ sw(r), sw(r) = (2 (r & 3) | (r >> 2) & 1) ^ 2 ((r >> 3) & 1), which
// takes 8 distinct values on every 8 aligned rows and, with the row's parity, 16 distinct
// (parity, chunk) pairs on every 16: the 16-byte K reads (one row per lane, 8 or 16
// lanes a cycle) and the transposing V reads (4 rows x 32 bytes per 16 lanes, the rows'
// 32-byte pieces on disjoint chunk pairs) are free of bank conflicts whether the LDS
// serves 128 or 256 bytes a cycle.
__device__ __forceinline__ int sw(int row) { return attn_tile_swizzle(row); }
__device__ __forceinline__ int swz(int row, int chunk) { return row * D + ((chunk ^ sw(row)) << 3); }

// Key/value rows of one head: the memory segment (row stride 64) followed by the frame
// (row stride H*64).  Tiles go straight from global memory to LDS
// (global_load_lds_dwordx4: lane l of a wave writes 16 bytes at the wave's LDS base +
// 16 l), so each thread fetches the global chunk that belongs at its LDS slot: thread
// tid fills physical chunk tid % 8 of rows tid / 8 and tid / 8 + 32, i.e. the global
// chunk (tid % 8) ^ sw(row) of those rows.  Addresses are a wave-uniform base
// plus a 32-bit per-thread byte offset fixed for the whole segment; the last tile of
// each part re-reads its last row in place of the rows past the end (always in
// bounds; their scores are masked).
struct TileCursor {
  const char* km;          // memory K / V rows of this head
  const char* vm;
  const char* kc;          // the frame's K / V rows of this head
  const char* vc;
  int64_t cur_tile;        // bytes between consecutive frame tiles: 64 * H * 64 * 2
  uint32_t off_m0, off_m1;     // thread byte offsets inside a full memory tile
  uint32_t off_c0, off_c1;     // ... inside a full frame tile
  uint32_t dt_m0, dt_m1;   // added for the last memory tile (rows clamped)
  uint32_t dt_c0, dt_c1;   // added for the last frame tile
  int nt_mem;              // memory tiles
  int t_last;              // index of the unit's last tile
  int mem_tail;            // valid rows of the last memory tile
  int tok_tail;            // valid rows of the last frame tile
};

__device__ __forceinline__ int tile_valid(const TileCursor& tc, int t) {
  int v = BK;
  if (t == tc.t_last) v = tc.tok_tail;
  if (t == tc.nt_mem - 1) v = tc.mem_tail;
  return v;
}

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void lds_load16(const char* g, uint16_t* lds_wave_base) {
  __builtin_amdgcn_global_load_lds((const void*)g, (lds_void*)lds_wave_base, 16, 0, 0);
}

// Issue tile t's K and V loads into ring stage S (completion: vmcnt + barrier).
// `ldsw` is the LDS ring plus this wave's row block (rows 8w .. 8w+7 of a tile; the
// second load of each operand fills rows 32 + 8w ..).
template <int S>
__device__ __forceinline__ void load_tile(const TileCursor& tc, int t, uint16_t* ldsw) {
  const char *kb, *vb;
  uint32_t o0, o1;
  if (t < tc.nt_mem) {  // uniform branches
    kb = tc.km + (int64_t)t * (BK * D * 2);
    vb = tc.vm + (int64_t)t * (BK * D * 2);
    o0 = tc.off_m0;
    o1 = tc.off_m1;
    if (t == tc.nt_mem - 1) {  // (additive, so no select between two fields' addresses)
      o0 += tc.dt_m0;
      o1 += tc.dt_m1;
    }
  } else {
    const int tc_i = t - tc.nt_mem;
    kb = tc.kc + tc_i * tc.cur_tile;
    vb = tc.vc + tc_i * tc.cur_tile;
    o0 = tc.off_c0;
    o1 = tc.off_c1;
    if (t == tc.t_last) {
      o0 += tc.dt_c0;
      o1 += tc.dt_c1;
    }
  }
  uint16_t* st = ldsw + S * STAGE;
  lds_load16(kb + o0, st);
  lds_load16(kb + o1, st + 32 * D);
  lds_load16(vb + o0, st + TILE);
  lds_load16(vb + o1, st + TILE + 32 * D);
}

struct SoftmaxState {
  float m;      // running max of z * log2(e) / 8
  float l;      // this lane's share of the row sum
  f32x16 o0;    // O^T rows d = 0..31 for this lane's query (accumulator layout)
  f32x16 o1;    // d = 32..63
};

// One 64-key tile for this wave's 32 queries.  kFirst: the segment's first tile, whose
// running reference is still unset, so its maximum is taken directly (the exact path of
// a later tile, without the rescale of an empty state).
template <bool kFirst>
__device__ __forceinline__ void tile_compute(const uint16_t* stage, const bf16x8 (&qf)[4], int lane, int valid,
                                             SoftmaxState& sm) {
  const int l32 = lane & 31, half = lane >> 5;
  // Wave priority 1 from the score MFMAs through the softmax, 0 for the value product: of
  // the two waves sharing a SIMD, the one in the first part of its tile issues first, which
  // keeps the pair out of step so that one's MFMAs run under the other's vector work
  // (about +1 % per stream over a uniform priority).  Priority changes no result.
  __builtin_amdgcn_s_setprio(1);
  f32x16 s0 = {}, s1 = {};
#pragma unroll
  for (int ds = 0; ds < 4; ++ds) {
    const bf16x8 ka = *reinterpret_cast<const bf16x8*>(&stage[swz(l32, ds * 2 + half)]);
    const bf16x8 kb = *reinterpret_cast<const bf16x8*>(&stage[swz(32 + l32, ds * 2 + half)]);
    s0 = mfma32(ka, qf[ds], s0);
    s1 = mfma32(kb, qf[ds], s1);
  }
  // accumulator entry r of this lane: key 8*(r/4) + 4*half + r%4 (+32 in s1)
  if (__builtin_expect(valid < BK, 0)) {
    // keys >= valid get -1e30: sat(key + 1 - valid) is 1 exactly for them, 0 otherwise
    // (arithmetic masking keeps the 32 lane masks out of scalar registers)
    const float fv = (float)(valid - 4 * half - 1);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float key = (float)(8 * (r >> 2) + (r & 3));
      s0[r] = fmaf(__saturatef(key - fv), kNegBig, s0[r]);
      s1[r] = fmaf(__saturatef(key + 32.0f - fv), kNegBig, s1[r]);
    }
  }
  // P = 2^(z*log2e/8 - m) against the running reference m.  Softmax does not depend on
  // the reference, so the tile maximum is only needed when some p could overflow: a
  // lane whose tile sum reaches 2^64 (or inf; every p starts as inf while m is unset)
  // makes the wave take the exact path -- raise m to the tile maximum, rescale the
  // accumulators, recompute P.  Terms far below the reference underflow to 0, exactly
  // as they would relative to the true maximum.
  bf16x8 p[4];
  float rsum = -0.f;  // -0 + x == x: the first add folds away
  auto exact = [&]() {
    float mx = fmaxf(s0[0], s1[0]);
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, fmaxf(s0[r], s1[r]));
    const float m_new = fmaxf(sm.m, half_max(mx) * kScaleLog2);
    if (!kFirst) {
      const float alpha = __builtin_amdgcn_exp2f(sm.m - m_new);
      sm.l *= alpha;
      sm.o0 *= alpha;
      sm.o1 *= alpha;
    }
    sm.m = m_new;
    rsum = -0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float e0 = __builtin_amdgcn_exp2f(fmaf(s0[r], kScaleLog2, -sm.m));
      const float e1 = __builtin_amdgcn_exp2f(fmaf(s1[r], kScaleLog2, -sm.m));
      rsum += e0 + e1;
      p[r >> 3][r & 7] = (__bf16)e0;
      p[2 + (r >> 3)][r & 7] = (__bf16)e1;
    }
  };
  if (kFirst) {
    exact();
  } else {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float e0 = __builtin_amdgcn_exp2f(fmaf(s0[r], kScaleLog2, -sm.m));
      const float e1 = __builtin_amdgcn_exp2f(fmaf(s1[r], kScaleLog2, -sm.m));
      rsum += e0 + e1;
      p[r >> 3][r & 7] = (__bf16)e0;
      p[2 + (r >> 3)][r & 7] = (__bf16)e1;
    }
    if (__any(!(rsum < kOverflowGuard))) exact();
  }
  sm.l += rsum;
  __builtin_amdgcn_s_setprio(0);

  // V^T operand through transposing LDS reads.  Within each 16-lane group, lane i
  // receives element i%4 of the 8-byte chunk addressed by lane 4r + i/4 (r = 0..3), so
  // lane 4r + j points at row (key) r, columns d0 + 4j .. +3: lane i then holds
  // V[key r][d0 + i] for the 4 keys.  Keys follow the P^T slot order: for k-step ks and
  // lane half hh, slots 0..3 are keys ks*16 + 4hh + r, slots 4..7 keys ks*16 + 8 + 4hh + r.
  const uint16_t* vt = stage + TILE;
  const int g = lane >> 4, i16 = lane & 15, rr = i16 >> 2, jj = i16 & 3, hh = g >> 1;
  const int col = 16 * (g & 1) + 4 * jj;  // logical column (elements) within a 32-dim block
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int row = ks * 16 + 4 * hh + rr;
#pragma unroll
    for (int db = 0; db < 2; ++db) {
      const int lcol = db * 32 + col;
      const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_i16x4*)(vt + swz(row, lcol >> 3) + (lcol & 7)));
      const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_i16x4*)(vt + swz(row + 8, lcol >> 3) + (lcol & 7)));
      const i16x8 w = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      const bf16x8 va = __builtin_bit_cast(bf16x8, w);
      if (db == 0)
        sm.o0 = mfma32(va, p[ks], sm.o0);
      else
        sm.o1 = mfma32(va, p[ks], sm.o1);
    }
  }
}

// Partial slots: chunk c's segment of a unit writes its output rows normalised by its
// own row sum, in bf16 ([BQ][64]), then its reference m[BQ] and row sum l[BQ] (fp32).
constexpr int kSlotStatsFloat = BQ * D / 2;
constexpr int kMergeRows = 32;   // output rows per merge workgroup (8 threads per row)
constexpr int kMergeMax = 8;     // partials whose loads are in flight together

// First iteration of chunk c of a queue (chunk arithmetic: rv_plan.h).
__device__ __forceinline__ int64_t chunk_start(const AttnArgs& a, int c) { return chunk_cut(a, c); }

// Partial slot of chunk c's segment of unit ui: slot 0 if the chunk starts inside the
// unit, slot 1 if it began in an earlier unit.
__device__ __forceinline__ const float* slot_ptr(const AttnArgs& a, int q, int c, int ui) {
  const int slot = 2 * (a.chunk_base[q] + c) + (chunk_start(a, c) >= (int64_t)ui * a.U ? 0 : 1);
  return a.part + (int64_t)slot * kAttnSlotFloats;
}

// Merge the partials of chunks c_first..c_last (in chunk order) for rows
// rb*32 .. rb*32+31 of `unit` and write the final output rows and LSE.  Partial j is
// weighted by 2^(m_j - M) l_j (M the largest m).  Thread -> (row, 8 dims); up to eight
// partials' statistics and rows are loaded in one round trip (indices clamped, surplus
// weights zero).
__device__ void merge_rows(const AttnArgs& a, int q, int unit, int ui, int rb, int c_first, int c_last) {
  const int tid = threadIdx.x;
  const int h = unit / a.q_tiles, qt = unit % a.q_tiles;
  const int row = rb * kMergeRows + (tid >> 3), d8 = (tid & 7) * 8;
  const int qi = qt * BQ + row;
  if (qi >= a.n_tokens) return;
  float mmax = kNegBig, L = 0.f;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  for (int c0 = c_first; c0 <= c_last; c0 += kMergeMax) {
    const int n = min(kMergeMax, c_last - c0 + 1);
    float mv[kMergeMax], lv[kMergeMax];
    uint4 v[kMergeMax];
#pragma unroll
    for (int j = 0; j < kMergeMax; ++j) {
      const float* ps = slot_ptr(a, q, min(c0 + j, c_last), ui);
      mv[j] = ps[kSlotStatsFloat + row];
      lv[j] = ps[kSlotStatsFloat + BQ + row];
      v[j] = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(ps) + row * D + d8);
    }
    float m_new = mmax;
#pragma unroll
    for (int j = 0; j < kMergeMax; ++j) m_new = fmaxf(m_new, mv[j]);  // clamped copies repeat a real one
    const float scale = __builtin_amdgcn_exp2f(mmax - m_new);
    L *= scale;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] *= scale;
    mmax = m_new;
#pragma unroll
    for (int j = 0; j < kMergeMax; ++j) {
      const float w = j < n ? __builtin_amdgcn_exp2f(mv[j] - mmax) * lv[j] : 0.f;
      L += w;
      const uint32_t wd[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[2 * i] = fmaf(w, __uint_as_float(wd[i] << 16), acc[2 * i]);
        acc[2 * i + 1] = fmaf(w, __uint_as_float(wd[i] & 0xFFFF0000u), acc[2 * i + 1]);
      }
    }
  }
  const float inv = 1.f / L;
  uint16_t* op = a.out + ((int64_t)qi * a.n_heads + h) * D + d8;
  const uint2 lo = to_bf16x4(acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
  const uint2 hi = to_bf16x4(acc[4] * inv, acc[5] * inv, acc[6] * inv, acc[7] * inv);
  *reinterpret_cast<uint4*>(op) = make_uint4(lo.x, lo.y, hi.x, hi.y);
  if (d8 == 0) a.lse[(int64_t)h * a.n_tokens + qi] = (mmax + __log2f(L)) * kLn2;
}

// Key tiles t0..t1-1 of `unit` (queue-local index ui) as part of chunk c of queue q.
__device__ void process_segment(const AttnArgs& a, int q, int c, int unit, int ui, int t0, int t1, uint16_t* lds) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = uniform(tid >> 6);
  const int l32 = lane & 31, half = lane >> 5;
  unit = uniform(unit);
  t0 = uniform(t0);
  t1 = uniform(t1);
  const int h = uniform(unit / a.q_tiles), qt = uniform(unit % a.q_tiles);
  const int q0 = qt * BQ + wave * 32;
  const int qi = q0 + l32;
  const bool wave_active = q0 < a.n_tokens;

  TileCursor tc;
  {
    const int r = tid >> 3, c8 = (tid & 7) * 8, rs = a.n_heads * D;
    tc.km = reinterpret_cast<const char*>(a.memK + (int64_t)h * a.head_stride * D);
    tc.vm = reinterpret_cast<const char*>(a.memV + (int64_t)h * a.head_stride * D);
    tc.kc = reinterpret_cast<const char*>(a.K + (int64_t)h * D);
    tc.vc = reinterpret_cast<const char*>(a.V + (int64_t)h * D);
    tc.cur_tile = (int64_t)BK * rs * 2;
    tc.nt_mem = a.nt_mem;
    tc.t_last = a.T - 1;
    tc.mem_tail = a.nt_mem > 0 ? (int)(a.mem_len - (int64_t)(a.nt_mem - 1) * BK) : BK;
    tc.tok_tail = a.T > a.nt_mem ? a.n_fkeys - (a.T - 1 - a.nt_mem) * BK : BK;
    const int r1 = r + 32;
    const int g0 = c8 ^ (sw(r) << 3), g1 = c8 ^ (sw(r1) << 3);
    tc.off_m0 = 2u * (uint32_t)(r * D + g0);
    tc.off_m1 = 2u * (uint32_t)(r1 * D + g1);
    tc.off_c0 = 2u * (uint32_t)(r * rs + g0);
    tc.off_c1 = 2u * (uint32_t)(r1 * rs + g1);
    tc.dt_m0 = 2u * (uint32_t)(min(r, tc.mem_tail - 1) * D + g0) - tc.off_m0;
    tc.dt_m1 = 2u * (uint32_t)(min(r1, tc.mem_tail - 1) * D + g1) - tc.off_m1;
    tc.dt_c0 = 2u * (uint32_t)(min(r, tc.tok_tail - 1) * rs + g0) - tc.off_c0;
    tc.dt_c1 = 2u * (uint32_t)(min(r1, tc.tok_tail - 1) * rs + g1) - tc.off_c1;
  }
  uint16_t* const ldsw = lds + wave * 8 * D;

  // B operand of S^T = K Q^T: this lane's query, head dims ds*16 + half*8 .. +7.
  bf16x8 qf[4];
  {
    const uint16_t* qp = a.Q + ((int64_t)min(qi, a.n_tokens - 1) * a.n_heads + h) * D + half * 8;
#pragma unroll
    for (int ds = 0; ds < 4; ++ds) qf[ds] = *reinterpret_cast<const bf16x8*>(qp + ds * 16);
  }
  SoftmaxState sm;
  sm.m = kNegBig;
  sm.l = 0.f;
  sm.o0 = f32x16{};
  sm.o1 = f32x16{};

  // Ring of NSTAGE (4) tiles, two computed per barrier: tile t0 + j lives in stage j % 4,
  // so every stage offset is a compile-time constant of the unrolled loop.  The next
  // pair streams into the two stages the previous pair used (freed at the last barrier)
  // while this pair is computed.  The first step is peeled off: its first tile sets the
  // running reference.
  auto step = [&](auto phase, auto first, int t) {
    constexpr int P = decltype(phase)::value;
    if (t + 2 < t1) load_tile<(P + 2) % NSTAGE>(tc, t + 2, ldsw);
    if (t + 3 < t1) load_tile<(P + 3) % NSTAGE>(tc, t + 3, ldsw);
    if (wave_active) {
      tile_compute<decltype(first)::value>(lds + P * STAGE, qf, lane, tile_valid(tc, t), sm);
      if (t + 1 < t1) tile_compute<false>(lds + (P + 1) * STAGE, qf, lane, tile_valid(tc, t + 1), sm);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  };
  load_tile<0>(tc, t0, ldsw);
  if (t0 + 1 < t1) load_tile<1>(tc, t0 + 1, ldsw);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  step(StageConst<0>{}, std::true_type{}, t0);
  for (int t = t0 + 2; t < t1; t = uniform(t + 4)) {
    step(StageConst<2>{}, std::false_type{}, t);
    if (t + 2 >= t1) break;
    step(StageConst<0>{}, std::false_type{}, t + 2);
  }

  const float l_tot = half_sum(sm.l);
  // The output rows (normalised by the row sum, bf16) go out through LDS: each wave stages
  // its 32 rows (row stride kOutStageRow elements, so that the 32 rows' 8-byte pieces spread
  // over the banks), then writes whole 128-byte rows, 8 lanes a row (before: each store
  // wrote 16 bytes into each of 32 rows; 2 % per stream).  The ring is free: the last
  // step ended with a barrier.
  constexpr int kOutStageRow = D + 8;
  uint16_t* const st = lds + wave * 32 * kOutStageRow;
  if (wave_active) {
    const float inv = 1.f / l_tot;
    uint16_t* sp = st + l32 * kOutStageRow + 4 * half;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      *reinterpret_cast<uint2*>(sp + 8 * j) =
          to_bf16x4(sm.o0[4 * j] * inv, sm.o0[4 * j + 1] * inv, sm.o0[4 * j + 2] * inv, sm.o0[4 * j + 3] * inv);
      *reinterpret_cast<uint2*>(sp + 32 + 8 * j) =
          to_bf16x4(sm.o1[4 * j] * inv, sm.o1[4 * j + 1] * inv, sm.o1[4 * j + 2] * inv, sm.o1[4 * j + 3] * inv);
    }
  }
  __syncthreads();
  const int r8 = lane >> 3, c8 = (lane & 7) * 8;
  if (t0 == 0 && t1 == a.T) {
    // the whole unit in this chunk: final output rows and LSE
    if (wave_active) {
      if (half == 0 && qi < a.n_tokens) a.lse[(int64_t)h * a.n_tokens + qi] = (sm.m + __log2f(l_tot)) * kLn2;
#pragma unroll
      for (int pass = 0; pass < 4; ++pass) {
        const int r = pass * 8 + r8, qr = q0 + r;
        if (qr < a.n_tokens)
          *reinterpret_cast<uint4*>(a.out + ((int64_t)qr * a.n_heads + h) * D + c8) =
              *reinterpret_cast<const uint4*>(st + r * kOutStageRow + c8);
      }
    }
  } else {
    // partial result, merged by the second launch: the normalised output rows in bf16
    // (the merge weights them by 2^(m - M) l), then m and l in fp32
    const int seg = chunk_start(a, c) >= (int64_t)ui * a.U ? 0 : 1;
    float* ps = a.part + (int64_t)(2 * (a.chunk_base[q] + c) + seg) * kAttnSlotFloats;
    if (wave_active) {
      if (half == 0) {
        const int row = wave * 32 + l32;
        ps[kSlotStatsFloat + row] = sm.m;
        ps[kSlotStatsFloat + BQ + row] = l_tot;
      }
      uint16_t* po = reinterpret_cast<uint16_t*>(ps) + wave * 32 * D;
#pragma unroll
      for (int pass = 0; pass < 4; ++pass) {
        const int r = pass * 8 + r8;
        *reinterpret_cast<uint4*>(po + r * D + c8) = *reinterpret_cast<const uint4*>(st + r * kOutStageRow + c8);
      }
    }
  }
  __syncthreads();  // (the ring is the next segment's)
}

// Requests a field from every 64-byte line of the argument block at once: the reads that
// follow (some of them through indices that other arguments give) then hit the scalar
// cache, instead of each line's first read costing a round trip of its own.
// (The scalars before the tables lie in the lines of Q, lse and unit_base[0]; each table
// spans at most two lines, holding its first and last entries.)
static_assert(offsetof(AttnArgs, lse) / 64 == 1 && offsetof(AttnArgs, unit_base) / 64 == 2 &&
                  offsetof(AttnArgs, chunk_base) + 4 * kMaxQueues + 8 > sizeof(AttnArgs) && kMaxQueues <= 16,
              "touch_args names a field in every line of the argument block");
__device__ __forceinline__ void touch_args(const AttnArgs& a) {
  asm volatile("" ::"s"(a.Q), "s"(a.lse), "s"(a.unit_base[0]), "s"(a.unit_base[kMaxQueues]), "s"(a.n_chunks[0]),
               "s"(a.n_chunks[kMaxQueues - 1]), "s"(a.chunk_base[0]), "s"(a.chunk_base[kMaxQueues - 1]));
}

__global__ __launch_bounds__(kAttnThreads, kAttnWgPerCu) void attn_fwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[NSTAGE * STAGE];
  // Workgroup b serves queue b % n_queues, chunk b / n_queues.  Queues are per XCD (the
  // hardware deals workgroup ids round-robin over the XCDs), which keeps the query
  // tiles of a head under one L2; placement only affects speed, never results.
  touch_args(a);
  const int q = (int)(blockIdx.x % (unsigned)a.n_queues);
  const int c = (int)(blockIdx.x / (unsigned)a.n_queues);
  if (c >= a.n_chunks[q]) return;
  const int ub = a.unit_base[q];
  int64_t first, end;
  chunk_iters(a, c, (int64_t)(a.unit_base[q + 1] - ub) * a.U, &first, &end);
  int it = (int)first;
  const int it_end = (int)end;
  while (it < it_end) {
    const int ui = it / a.U;
    const int t0 = it - ui * a.U;
    if (t0 >= a.T) {  // padding after the unit's last tile (split mode)
      it = (ui + 1) * a.U;
      continue;
    }
    const int seg_end = min(it_end, ui * a.U + a.T);
    process_segment(a, q, c, ub + ui, ui, t0, t0 + (seg_end - it), lds);
    it = (seg_end == ui * a.U + a.T) ? (ui + 1) * a.U : seg_end;
  }
}

// Second launch: for every unit whose key range was split over several chunks, four
// workgroups (32 rows each) merge the partial results (the kernel boundary makes them
// visible on every XCD).
__global__ __launch_bounds__(kAttnThreads) void attn_merge_kernel(AttnArgs a) {
  // Workgroup b merges for queue b % n_queues, like the forward workgroups that wrote
  // the partials (a locality heuristic: the partials may still be in that XCD's L2).
  touch_args(a);
  const int q = (int)(blockIdx.x % (unsigned)a.n_queues);
  const int j = (int)(blockIdx.x / (unsigned)a.n_queues);
  const int ui = j / (BQ / kMergeRows), rb = j % (BQ / kMergeRows);
  if (ui >= a.unit_base[q + 1] - a.unit_base[q]) return;
  const int unit = a.unit_base[q] + ui;
  const int c_first = chunk_holding(a, (int64_t)ui * a.U);
  const int c_last = chunk_holding(a, (int64_t)ui * a.U + a.T - 1);
  if (c_first == c_last) return;  // written whole by its only chunk
  merge_rows(a, q, unit, ui, rb, c_first, c_last);
}

// Merge launch with the saliency in its epilogue (Sec. 3.3: the saliency reuses the LSE,
// so it can only start once a query's LSE is final).  kEpiGroups workgroups per unit
// (head h, 128-query block qt); workgroup g
// * merges output rows 32 g .. 32 g + 31 of a split unit exactly as the merge launch does
//   (a unit whose key range one chunk covered was written by the forward launch);
// * forms the final LSE (log2 units) of all 128 rows -- from the partials' m and l with
//   merge_rows' arithmetic, or read back for a whole unit -- and lists the block's sampled
//   queries (the window rule of SalEpi) in row order, staging their rows in LDS;
// * sums, for the keys of its quarter of the frame's 32-key blocks, exp2(z log2(e) / 8 -
//   LSE log2(e)) over the sampled queries with v_mfma_f32_32x32x16_bf16 (Z = Q~ K^T, one
//   lane per key), in a fixed order -- in-lane over the accumulator rows, over 32-query
//   blocks, then across the lane halves -- into tiles[h][qt][j].
constexpr int kEpiGroups = 4;
constexpr int kEpiQStride = kHeadDim + 8;   // staged query rows, 144 bytes
constexpr int kEpiKeyBatch = 4;             // 32-key blocks whose K rows a wave loads together

// Final LSE (log2 units) of row `row` of a split unit, with merge_rows' arithmetic.
__device__ float merged_lse2(const AttnArgs& a, int q, int ui, int row, int c_first, int c_last) {
  float mmax = kNegBig, L = 0.f;
  for (int c0 = c_first; c0 <= c_last; c0 += kMergeMax) {
    const int n = min(kMergeMax, c_last - c0 + 1);
    float mv[kMergeMax], lv[kMergeMax];
#pragma unroll
    for (int j = 0; j < kMergeMax; ++j) {
      const float* ps = slot_ptr(a, q, min(c0 + j, c_last), ui);
      mv[j] = ps[kSlotStatsFloat + row];
      lv[j] = ps[kSlotStatsFloat + BQ + row];
    }
    float m_new = mmax;
#pragma unroll
    for (int j = 0; j < kMergeMax; ++j) m_new = fmaxf(m_new, mv[j]);
    L *= __builtin_amdgcn_exp2f(mmax - m_new);
    mmax = m_new;
#pragma unroll
    for (int j = 0; j < kMergeMax; ++j) L += j < n ? __builtin_amdgcn_exp2f(mv[j] - mmax) * lv[j] : 0.f;
  }
  return mmax + __log2f(L);
}

__global__ __launch_bounds__(kAttnThreads) void attn_merge_sal_kernel(AttnArgs a, SalEpi e) {
  __shared__ float s_lse2[BQ];                        // by row
  __shared__ float s_lsec[BQ];                        // by sampled position (padding: +inf)
  __shared__ int s_list[BQ];
  __shared__ int s_count[2];
  __shared__ __attribute__((aligned(16))) uint16_t s_q[BQ * kEpiQStride];
  touch_args(a);
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);
  const int q = (int)(blockIdx.x % (unsigned)a.n_queues);
  const int jg = (int)(blockIdx.x / (unsigned)a.n_queues);
  const int ui = jg / kEpiGroups, g = jg % kEpiGroups;
  if (ui >= a.unit_base[q + 1] - a.unit_base[q]) return;  // uniform
  const int unit = a.unit_base[q] + ui;
  const int h = unit / a.q_tiles, qt = unit % a.q_tiles;
  const int N = a.n_tokens;
  const int c_first = chunk_holding(a, (int64_t)ui * a.U);
  const int c_last = chunk_holding(a, (int64_t)ui * a.U + a.T - 1);

  // ---- this group's output rows, and the LSE of all the block's rows ----
  if (c_first != c_last) merge_rows(a, q, unit, ui, g, c_first, c_last);
  if (tid < BQ) {
    const int qi = qt * BQ + tid;
    float l2 = 0.f;
    if (qi < N) l2 = c_first == c_last ? a.lse[(int64_t)h * N + qi] * kLog2e : merged_lse2(a, q, ui, tid, c_first, c_last);
    s_lse2[tid] = l2;
  }

  // ---- the block's sampled queries, in row order (waves 0 and 1 hold rows 0 .. 127) ----
  const int srow = wave * 64 + lane;
  bool sampled = false;
  int before = 0;
  if (wave < 2) {
    const int r = qt * BQ + srow - e.q_base;
    sampled = r >= 0 && r < e.grid_cells && (r / e.grid_w) % e.stride == 0 && (r % e.grid_w) % e.stride == 0;
    const uint64_t bal = __ballot(sampled);
    before = __builtin_popcountll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) s_count[wave] = __builtin_popcountll(bal);
  }
  __syncthreads();
  if (sampled) s_list[(wave == 1 ? s_count[0] : 0) + before] = srow;
  __syncthreads();
  const int n_s = s_count[0] + s_count[1];
  const int ns_pad = (n_s + 31) & ~31;
  const uint16_t* Kh = e.K + (int64_t)h * e.kv_head;
  float* tile_h = e.tiles + ((int64_t)h * a.q_tiles + qt) * N;
  const int n_blocks = (N + 31) / 32;
  const int per_group = (n_blocks + kEpiGroups - 1) / kEpiGroups;
  const int blk0 = g * per_group, blk1 = min(n_blocks, blk0 + per_group);
  if (n_s == 0) {  // no sampled query in this block: its saliency row is the empty sum
    for (int j = blk0 * 32 + tid; j < min(N, blk1 * 32); j += kAttnThreads) tile_h[j] = 0.f;
    return;
  }
  // sampled query rows and their LSE (padding rows: zero rows, +inf -> weight 0)
  for (int x = tid; x < ns_pad * 8; x += kAttnThreads) {
    const int s = x >> 3, ch = x & 7;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (s < n_s) v = *reinterpret_cast<const uint4*>(a.Q + ((int64_t)(qt * BQ + s_list[s]) * a.n_heads + h) * D + ch * 8);
    *reinterpret_cast<uint4*>(&s_q[s * kEpiQStride + ch * 8]) = v;
  }
  for (int s = tid; s < ns_pad; s += kAttnThreads) s_lsec[s] = s < n_s ? s_lse2[s_list[s]] : __builtin_inff();
  __syncthreads();

  // ---- this group's key blocks, kEpiKeyBatch per wave at a time ----
  const int l32 = lane & 31, half = lane >> 5;
  for (int kb0 = blk0 + wave; kb0 < blk1; kb0 += kEpiKeyBatch * (kAttnThreads / 64)) {
    bf16x8 kf[kEpiKeyBatch][4];
#pragma unroll
    for (int bb = 0; bb < kEpiKeyBatch; ++bb) {
      const int j = min((kb0 + bb * (kAttnThreads / 64)) * 32 + l32, N - 1);  // past the range: result unused
      const uint16_t* kp = Kh + (int64_t)j * e.kv_row + half * 8;
#pragma unroll
      for (int ds = 0; ds < 4; ++ds) kf[bb][ds] = *reinterpret_cast<const bf16x8*>(kp + ds * 16);
    }
#pragma unroll
    for (int bb = 0; bb < kEpiKeyBatch; ++bb) {
      const int kb = kb0 + bb * (kAttnThreads / 64);
      if (kb >= blk1) break;  // uniform
      float acc = 0.f;
      for (int qb = 0; qb < ns_pad; qb += 32) {
        bf16x8 qf[4];
#pragma unroll
        for (int ds = 0; ds < 4; ++ds)
          qf[ds] = *reinterpret_cast<const bf16x8*>(&s_q[(qb + l32) * kEpiQStride + ds * 16 + half * 8]);
        f32x16 z = {};
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) z = mfma32(qf[ds], kf[bb][ds], z);
        // accumulator entry r: sampled query qb + 8 (r / 4) + 4 half + r % 4, key kb * 32 + l32
        float s0 = 0.f, s1 = 0.f;
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const int i0 = qb + 8 * (r >> 2) + 4 * half + (r & 3);
          s0 += __builtin_amdgcn_exp2f(fmaf(z[r], kScaleLog2, -s_lsec[i0]));
          s1 += __builtin_amdgcn_exp2f(fmaf(z[r + 1], kScaleLog2, -s_lsec[i0 + 1]));
        }
        acc += s0 + s1;
      }
      const float tot = acc + __shfl_xor(acc, 32);
      const int j = kb * 32 + l32;
      if (half == 0 && j < N) tile_h[j] = tot;
    }
  }
}

__global__ void xcc_probe_kernel(int* ids) {
  if (threadIdx.x == 0) ids[blockIdx.x] = hw_xcc_id();
}

// Split-KV partial slots of the allocation-free entry point: every GPU the library runs
// on holds one copy, from the library's load until the process ends.
static __device__ __align__(256) float scratch[(size_t)kStaticScratchSlots * kAttnSlotFloats];

}  // namespace

hipError_t static_scratch_address(float** ptr) {
  // host code may not use `scratch` itself as a device address: take the current
  // device's copy of the array through the runtime
  return hipGetSymbolAddress(reinterpret_cast<void**>(ptr), HIP_SYMBOL(scratch));
}

hipError_t launch_attention(const AttnArgs& a, int grid, bool merge, hipStream_t s) {
  hipLaunchKernelGGL(attn_fwd_kernel, dim3(grid), dim3(kAttnThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !merge) return e;
  int max_units = 0;
  for (int q = 0; q < a.n_queues; ++q) max_units = max(max_units, a.unit_base[q + 1] - a.unit_base[q]);
  hipLaunchKernelGGL(attn_merge_kernel, dim3(a.n_queues * max_units * (BQ / kMergeRows)), dim3(kAttnThreads), 0,
                     s, a);
  return hipGetLastError();
}

hipError_t launch_attention_saliency(const AttnArgs& a, const SalEpi& e, int grid, hipStream_t s) {
  hipLaunchKernelGGL(attn_fwd_kernel, dim3(grid), dim3(kAttnThreads), 0, s, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  int max_units = 0;
  for (int q = 0; q < a.n_queues; ++q) max_units = max(max_units, a.unit_base[q + 1] - a.unit_base[q]);
  hipLaunchKernelGGL(attn_merge_sal_kernel, dim3(a.n_queues * max_units * kEpiGroups), dim3(kAttnThreads), 0, s,
                     a, e);
  return hipGetLastError();
}

hipError_t launch_xcc_probe(int* ids, int n_blocks, hipStream_t s) {
  hipLaunchKernelGGL(xcc_probe_kernel, dim3(n_blocks), dim3(64), 0, s, ids);
  return hipGetLastError();
}

}  // namespace rv
