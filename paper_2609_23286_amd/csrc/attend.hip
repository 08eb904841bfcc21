// attend.hip -- temporal-causal attention forward with per-query log-sum-exp, gfx950.
//
// Computes, for one frame and one layer (Sec. 3.1 Eq. 2-3 and the LSE equation of
// Sec. 3.3), for every head h and query i of the frame:
//   z_ic = q_i . k_c / 8 over the context c = [memory rows of h ; the frame's keys],
//   LSE_i = log sum_c exp(z_ic),  o_i = sum_c exp(z_ic - LSE_i) v_c.
//
// Design (CDNA4):
// * A workgroup is 4 wave64s and owns 128 queries of one head (32 per wave).  K/V tiles
//   of 64 keys are staged in LDS: K row-major, V transposed, both with padded rows.
// * Scores are formed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16, so that
//   each lane holds one query's column: the softmax max / sum are in-lane reductions
//   plus one exchange between the two 32-lane halves that share a query.
// * The output is accumulated transposed too, O^T += V^T P^T, with P^T taken straight
//   from the score registers: the 16 accumulator rows a lane holds are exactly the 8+8
//   keys the B operand wants, once V^T's columns are stored in the matching order.
// * Online softmax in base 2 with the 1/sqrt(d) scale folded into one FMA; the running
//   maximum is only raised when a tile's maximum exceeds it by more than 2^8, so the
//   rescale of the accumulators is rare (exact in any case: the LSE uses the maximum the
//   sums were taken against).
// * Split-KV: (head, query tile) pairs alone cannot fill 256 CUs (1041 tokens x 16 heads
//   is 144 workgroups), so the key tiles are cut into n_splits ranges.  Every split
//   writes an unnormalised partial (O, max, sum); the last workgroup of a query tile to
//   finish (atomic counter) merges all partials in split order, so the result does not
//   depend on scheduling.
// * Workgroup ids are remapped so that consecutive work items (same head) run on the
//   same XCD and share that head's K/V in the XCD's L2.
#include "rv_internal.h"

namespace rv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BQ = kAttnBQ;
constexpr int BK = kAttnBK;
constexpr int D = kHeadDim;
constexpr int LDS_STRIDE = D + 8;  // 144-byte rows: 16-byte lane reads hit distinct banks
constexpr float kLn2 = 0.69314718055994531f;
constexpr float kScaleLog2 = 1.44269504088896341f * 0.125f;  // log2(e) / sqrt(64)
constexpr float kRescaleSlack = 8.0f;   // allow p <= 2^8 before raising the running max
constexpr float kNegBig = -1.0e30f;

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack2(uint16_t lo, uint16_t hi) {
  return (uint32_t)lo | ((uint32_t)hi << 16);
}

// Four fp32 -> bf16 (round to nearest even), packed into two dwords.
__device__ __forceinline__ uint2 to_bf16x4(float a, float b, float c, float d) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
  return *reinterpret_cast<uint2*>(&v);
}

__global__ __launch_bounds__(kAttnThreads, 2) void attn_fwd_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sK[BK * LDS_STRIDE];
  __shared__ __attribute__((aligned(16))) uint16_t sVt[D * LDS_STRIDE];
  __shared__ int s_last;

  // XCD-aware remap: hardware deals workgroup ids round-robin over the 8 XCDs.
  const int bid = blockIdx.x;
  const int w = (bid & 7) * a.per_xcd + (bid >> 3);
  if (w >= a.n_work) return;
  const int split = w % a.n_splits;
  const int tile_id = w / a.n_splits;  // h * q_tiles + qt
  const int qt = tile_id % a.q_tiles;
  const int h = tile_id / a.q_tiles;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int N = a.n_tokens, H = a.n_heads;
  const int q0 = qt * BQ + wave * 32;
  const int qi = q0 + l32;
  const bool wave_active = q0 < N;

  // B operand of S^T = K Q^T: this lane's query, head dims ds*16 + half*8 .. +7.
  bf16x8 qf[4];
  if (qi < N) {
    const uint16_t* qp = a.Q + ((int64_t)qi * H + h) * D + half * 8;
#pragma unroll
    for (int ds = 0; ds < 4; ++ds) qf[ds] = *reinterpret_cast<const bf16x8*>(qp + ds * 16);
  } else {
#pragma unroll
    for (int ds = 0; ds < 4; ++ds) qf[ds] = bf16x8{};
  }

  const int t_begin = (int)((int64_t)a.nt_total * split / a.n_splits);
  const int t_end = (int)((int64_t)a.nt_total * (split + 1) / a.n_splits);

  float m_run = kNegBig;  // running max of z * log2(e) / 8
  float l_run = 0.f;      // this lane's share of the row sum (its 32 of each 64 keys)
  f32x16 o0 = {}, o1 = {};  // O^T rows d = 0..31 and 32..63 for this lane's query

  for (int t = t_begin; t < t_end; ++t) {
    const uint16_t *kbase, *vbase;
    int64_t rs;
    int valid;
    if (t < a.nt_mem) {
      const int64_t r0 = (int64_t)t * BK;
      kbase = a.memK + ((int64_t)h * a.head_stride + r0) * D;
      vbase = a.memV + ((int64_t)h * a.head_stride + r0) * D;
      rs = D;
      valid = (int)min((int64_t)BK, a.mem_len - r0);
    } else {
      const int r0 = (t - a.nt_mem) * BK;
      kbase = a.K + ((int64_t)r0 * H + h) * D;
      vbase = a.V + ((int64_t)r0 * H + h) * D;
      rs = (int64_t)H * D;
      valid = min(BK, N - r0);
    }

    __syncthreads();  // previous tile fully consumed
    {
      // K tile, row-major: rows tid/8 and tid/8 + 32, 16-byte chunk tid % 8.
      const int r = tid >> 3, c = tid & 7;
      uint4 k0 = {0u, 0u, 0u, 0u}, k1 = {0u, 0u, 0u, 0u};
      if (r < valid) k0 = *reinterpret_cast<const uint4*>(kbase + r * rs + c * 8);
      if (r + 32 < valid) k1 = *reinterpret_cast<const uint4*>(kbase + (r + 32) * rs + c * 8);
      *reinterpret_cast<uint4*>(&sK[r * LDS_STRIDE + c * 8]) = k0;
      *reinterpret_cast<uint4*>(&sK[(r + 32) * LDS_STRIDE + c * 8]) = k1;
    }
    {
      // V tile transposed: wave g takes keys 16g..16g+15, lane = head dim.  Within each
      // 16-key group, columns 0..7 hold keys {0-3, 8-11} and 8..15 hold {4-7, 12-15}:
      // the keys the two lane halves carry in the score accumulator.
      const int d = lane, g = wave;
      uint16_t v[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = g * 16 + i;
        v[i] = key < valid ? vbase[key * rs + d] : (uint16_t)0;
      }
      uint4 lo, hi;
      lo.x = pack2(v[0], v[1]);
      lo.y = pack2(v[2], v[3]);
      lo.z = pack2(v[8], v[9]);
      lo.w = pack2(v[10], v[11]);
      hi.x = pack2(v[4], v[5]);
      hi.y = pack2(v[6], v[7]);
      hi.z = pack2(v[12], v[13]);
      hi.w = pack2(v[14], v[15]);
      *reinterpret_cast<uint4*>(&sVt[d * LDS_STRIDE + g * 16]) = lo;
      *reinterpret_cast<uint4*>(&sVt[d * LDS_STRIDE + g * 16 + 8]) = hi;
    }
    __syncthreads();
    if (!wave_active) continue;

    // S^T (64 keys x 32 queries): s0 keys 0..31, s1 keys 32..63.  Accumulator entry r of
    // a lane is key 8*(r/4) + 4*half + r%4 (+32 for s1) against query qi.
    f32x16 s0 = {}, s1 = {};
#pragma unroll
    for (int ds = 0; ds < 4; ++ds) {
      const bf16x8 ka = *reinterpret_cast<const bf16x8*>(&sK[l32 * LDS_STRIDE + ds * 16 + half * 8]);
      const bf16x8 kb =
          *reinterpret_cast<const bf16x8*>(&sK[(32 + l32) * LDS_STRIDE + ds * 16 + half * 8]);
      s0 = mfma32(ka, qf[ds], s0);
      s1 = mfma32(kb, qf[ds], s1);
    }
    if (valid < BK) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 8 * (r >> 2) + 4 * half + (r & 3);
        if (key >= valid) s0[r] = kNegBig;
        if (key + 32 >= valid) s1[r] = kNegBig;
      }
    }

    float mx = s0[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s0[r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s1[r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_cand = mx * kScaleLog2;
    if (__any(m_cand > m_run + kRescaleSlack)) {
      const float m_new = fmaxf(m_run, m_cand);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
      o0 *= alpha;
      o1 *= alpha;
      m_run = m_new;
    }

    // P = 2^(z*log2e/8 - m), fp32 for the row sum, bf16 for the value product.
    bf16x8 p[4];
    float rsum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float e0 = __builtin_amdgcn_exp2f(fmaf(s0[r], kScaleLog2, -m_run));
      const float e1 = __builtin_amdgcn_exp2f(fmaf(s1[r], kScaleLog2, -m_run));
      rsum += e0 + e1;
      p[r >> 3][r & 7] = (__bf16)e0;
      p[2 + (r >> 3)][r & 7] = (__bf16)e1;
    }
    l_run += rsum;

    // O^T (64 dims x 32 queries) += V^T P^T over four 16-key steps.
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bf16x8 va = *reinterpret_cast<const bf16x8*>(&sVt[l32 * LDS_STRIDE + ks * 16 + half * 8]);
      const bf16x8 vb =
          *reinterpret_cast<const bf16x8*>(&sVt[(32 + l32) * LDS_STRIDE + ks * 16 + half * 8]);
      o0 = mfma32(va, p[ks], o0);
      o1 = mfma32(vb, p[ks], o1);
    }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);

  if (a.n_splits == 1) {
    if (wave_active && qi < N) {
      const float inv = 1.f / l_tot;
      uint16_t* op = a.out + ((int64_t)qi * H + h) * D + 4 * half;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        *reinterpret_cast<uint2*>(op + 8 * j) =
            to_bf16x4(o0[4 * j] * inv, o0[4 * j + 1] * inv, o0[4 * j + 2] * inv, o0[4 * j + 3] * inv);
        *reinterpret_cast<uint2*>(op + 32 + 8 * j) =
            to_bf16x4(o1[4 * j] * inv, o1[4 * j + 1] * inv, o1[4 * j + 2] * inv, o1[4 * j + 3] * inv);
      }
      if (half == 0) a.lse[(int64_t)h * N + qi] = (m_run + __log2f(l_tot)) * kLn2;
    }
    return;
  }

  // ---- split-KV: publish this split's partial, the last split merges ----
  const int64_t slot = (int64_t)tile_id * a.n_splits + split;
  if (wave_active) {
    const int row = wave * 32 + l32;
    float* po = a.part_o + (slot * BQ + row) * D + 4 * half;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      *reinterpret_cast<float4*>(po + 8 * j) = make_float4(o0[4 * j], o0[4 * j + 1], o0[4 * j + 2], o0[4 * j + 3]);
      *reinterpret_cast<float4*>(po + 32 + 8 * j) =
          make_float4(o1[4 * j], o1[4 * j + 1], o1[4 * j + 2], o1[4 * j + 3]);
    }
    if (half == 0) {
      a.part_ml[slot * 2 * BQ + row] = m_run;
      a.part_ml[slot * 2 * BQ + BQ + row] = l_tot;
    }
  }
  __threadfence();
  __syncthreads();
  if (tid == 0) s_last = atomicAdd(&a.counters[tile_id], 1) == a.n_splits - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();

  // Merge, in split order: thread -> (row = tid/2, 32 head dims).
  const int row = tid >> 1, dh = (tid & 1) * 32;
  const int q = qt * BQ + row;
  if (q < N) {
    const int64_t slot0 = (int64_t)tile_id * a.n_splits;
    float mmax = kNegBig;
    for (int s = 0; s < a.n_splits; ++s) mmax = fmaxf(mmax, a.part_ml[(slot0 + s) * 2 * BQ + row]);
    float acc[32];
#pragma unroll
    for (int e = 0; e < 32; ++e) acc[e] = 0.f;
    float L = 0.f;
    for (int s = 0; s < a.n_splits; ++s) {
      const float ms = a.part_ml[(slot0 + s) * 2 * BQ + row];
      const float ls = a.part_ml[(slot0 + s) * 2 * BQ + BQ + row];
      const float wgt = __builtin_amdgcn_exp2f(ms - mmax);
      L += wgt * ls;
      const float4* po = reinterpret_cast<const float4*>(a.part_o + ((slot0 + s) * BQ + row) * D + dh);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float4 v = po[e];
        acc[4 * e] += wgt * v.x;
        acc[4 * e + 1] += wgt * v.y;
        acc[4 * e + 2] += wgt * v.z;
        acc[4 * e + 3] += wgt * v.w;
      }
    }
    const float inv = 1.f / L;
    uint16_t* op = a.out + ((int64_t)q * H + h) * D + dh;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      *reinterpret_cast<uint2*>(op + 4 * e) =
          to_bf16x4(acc[4 * e] * inv, acc[4 * e + 1] * inv, acc[4 * e + 2] * inv, acc[4 * e + 3] * inv);
    if (dh == 0) a.lse[(int64_t)h * N + q] = (mmax + __log2f(L)) * kLn2;
  }
  if (tid == 0) a.counters[tile_id] = 0;  // ready for the next launch
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(attn_fwd_kernel, dim3(8 * a.per_xcd), dim3(kAttnThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace rv
