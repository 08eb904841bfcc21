// admit.hip -- LSE-saliency, per-head top-k and memory append, gfx950.
//
// One workgroup (8 wave64s) owns one (layer, head): it computes the saliency of all N
// keys of the frame, selects, and appends, with no communication between workgroups.
//
// Saliency (Sec. 3.3, saliency score and the A_ij equation): for key j of the frame,
//   S_j = sum over sampled queries i of exp(q_i . k_j / 8 - LSE_i),
// with the LSE the attention pass saved, so every term is an exact attention
// probability and no score matrix is stored.  The sampled query rows and their LSE are
// staged in LDS once.  A wave takes 128 keys at a time (four 32-key blocks whose K rows
// stay in registers) and sweeps all sampled queries in blocks of 32 with
// v_mfma_f32_32x32x16_bf16 (Z = Q~ K^T, each lane owning one key column); the
// exponentials are summed in fp32 in a fixed order -- in-lane, then across the two lane
// halves -- so S is bit-reproducible with no atomics.
//
// Selection (Sec. 3.3 Eq. 6, head-specific retention): the `budget` largest S_j, equal
// values ordered by lower index: an MSB-first radix select over the fp32 bit patterns
// (order-preserving for S >= 0) finds the exact threshold value and how many of its
// ties to take; block scans then emit the chosen indices in ascending order.  The chosen
// K/V rows are copied to the memory arena at rows mem_len.. with their provenance.
#include "rv_internal.h"

namespace rv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int D = kHeadDim;
constexpr int NT = kAdmitThreads;
constexpr int NW = NT / 64;
constexpr int QS_STRIDE = D + 8;  // staged sampled-query rows, 144 bytes
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kScaleLog2 = kLog2e * 0.125f;

// Inclusive prefix sum over the workgroup's threads.
__device__ int block_inclusive_scan(int v, int* s_wave) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int u = __shfl_up(v, off);
    if (lane >= off) v += u;
  }
  if (lane == 63) s_wave[wave] = v;
  __syncthreads();
  int base = 0;
  for (int w = 0; w < wave; ++w) base += s_wave[w];
  __syncthreads();
  return v + base;
}

// Top-`budget` of sal[0..N) (ties -> lower index), ascending, into s_idx[0..budget).
__device__ void select_topk(const float* sal, int N, int budget, int32_t* s_idx) {
  __shared__ unsigned int hist[256];
  __shared__ int s_wave[NW];
  __shared__ int s_bin, s_need;
  const int tid = threadIdx.x;

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
    if (tid < 256) hist[tid] = 0u;
    __syncthreads();
    for (int j = tid; j < N; j += NT) {
      const unsigned int kj = __float_as_uint(sal[j]);
      if ((kj & mask) == prefix) atomicAdd(&hist[(kj >> shift) & 255u], 1u);
    }
    __syncthreads();
    // thread i < 256 holds bin 255 - i: the inclusive scan counts digits >= bin
    const int b = 255 - tid;
    const int cnt = tid < 256 ? (int)hist[b] : 0;
    const int ge = block_inclusive_scan(cnt, s_wave);
    const int gt = ge - cnt;
    if (tid < 256 && gt < need && need <= ge) {
      s_bin = b;
      s_need = need - gt;
    }
    __syncthreads();
    prefix |= (unsigned int)s_bin << shift;
    mask |= 255u << shift;
    need = s_need;
    __syncthreads();
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
  const int eq_before = block_inclusive_scan(n_eq, s_wave) - n_eq;
  const int take_eq = max(0, min(n_eq, need - eq_before));
  const int n_sel = n_gt + take_eq;
  int pos = block_inclusive_scan(n_sel, s_wave) - n_sel;
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

// Select for (layer, h) from s_sal and append the chosen rows.
__device__ void select_and_append(const AdmitArgs& a, const AdmitLayer& L, int h, const float* s_sal,
                                  int32_t* s_idx) {
  const int N = a.n_tokens, H = a.n_heads, k = a.budget, tid = threadIdx.x;
  if (k == 0) return;
  select_topk(s_sal, N, k, s_idx);
  if (L.idx)
    for (int r = tid; r < k; r += NT) L.idx[(int64_t)h * k + r] = s_idx[r];
  // 16-byte chunks: 8 per K row, 8 per V row.
  for (int c = tid; c < k * 16; c += NT) {
    const int r = c >> 4, part = c & 15, chunk = part & 7;
    const int j = s_idx[r];
    if (j < 0 || j >= N) continue;  // unreachable: the selection emits exactly k indices < N
    const int64_t src = ((int64_t)j * H + h) * D + chunk * 8;
    const int64_t dst = ((int64_t)h * L.head_stride + L.mem_len + r) * D + chunk * 8;
    if (part < 8)
      *reinterpret_cast<uint4*>(L.memK + dst) = *reinterpret_cast<const uint4*>(L.K + src);
    else
      *reinterpret_cast<uint4*>(L.memV + dst) = *reinterpret_cast<const uint4*>(L.V + src);
  }
  for (int r = tid; r < k; r += NT) {
    int32_t* pv = L.prov + ((int64_t)h * L.head_stride + L.mem_len + r) * 2;
    pv[0] = a.frame_id;
    pv[1] = s_idx[r];
  }
}

// Saliency of all N keys of (layer, h) into s_sal (and L.sal).
__device__ void saliency(const AdmitArgs& a, const AdmitLayer& L, int h, float* s_sal, float* s_lse2,
                         uint16_t* s_q) {
  const int N = a.n_tokens, H = a.n_heads, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, l32 = lane & 31, half = lane >> 5;
  const int nq_pad = (a.n_q + 31) & ~31;
  const bool staged = s_q != nullptr;

  // LSE of the sampled queries in log2 units (padding rows: +inf -> weight 0), and the
  // sampled query rows themselves (padding rows zero).
  for (int i = tid; i < nq_pad; i += NT)
    s_lse2[i] = i < a.n_q ? L.lse[(int64_t)h * N + a.qidx[i]] * kLog2e : __builtin_inff();
  if (staged) {
    for (int c = tid; c < nq_pad * 8; c += NT) {
      const int i = c >> 3, ch = c & 7;
      uint4 v = {0u, 0u, 0u, 0u};
      if (i < a.n_q) v = *reinterpret_cast<const uint4*>(L.Q + ((int64_t)a.qidx[i] * H + h) * D + ch * 8);
      *reinterpret_cast<uint4*>(&s_q[i * QS_STRIDE + ch * 8]) = v;
    }
  }
  __syncthreads();

  const int n_blocks = (N + 31) / 32;
  const int n_groups = (n_blocks + 3) / 4;
  for (int g = wave; g < n_groups; g += NW) {
    // B operands (K^T) of up to four 32-key blocks: lane's key, dims ds*16 + half*8 ..
    bf16x8 kf[4][4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int j = (4 * g + b) * 32 + l32;
      if (j < N) {
        const uint16_t* kp = L.K + ((int64_t)j * H + h) * D + half * 8;
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) kf[b][ds] = *reinterpret_cast<const bf16x8*>(kp + ds * 16);
      } else {
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) kf[b][ds] = bf16x8{};
      }
    }
    const int nb = min(4, n_blocks - 4 * g);
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int qb = 0; qb < nq_pad; qb += 32) {
      bf16x8 qf[4];
      const int qa = qb + l32;
      if (staged) {
#pragma unroll
        for (int ds = 0; ds < 4; ++ds)
          qf[ds] = *reinterpret_cast<const bf16x8*>(&s_q[qa * QS_STRIDE + ds * 16 + half * 8]);
      } else if (qa < a.n_q) {
        const uint16_t* qp = L.Q + ((int64_t)a.qidx[qa] * H + h) * D + half * 8;
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) qf[ds] = *reinterpret_cast<const bf16x8*>(qp + ds * 16);
      } else {
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) qf[ds] = bf16x8{};
      }
      // LSE of this lane's 16 accumulator rows: queries qb + 8*(r/4) + 4*half + r%4
      float l2[16];
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const float4 v = *reinterpret_cast<const float4*>(&s_lse2[qb + 8 * r4 + 4 * half]);
        l2[4 * r4] = v.x;
        l2[4 * r4 + 1] = v.y;
        l2[4 * r4 + 2] = v.z;
        l2[4 * r4 + 3] = v.w;
      }
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        if (b < nb) {
          f32x16 z = {};
#pragma unroll
          for (int ds = 0; ds < 4; ++ds) z = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[ds], kf[b][ds], z, 0, 0, 0);
          float s = 0.f;
#pragma unroll
          for (int r = 0; r < 16; ++r) s += __builtin_amdgcn_exp2f(fmaf(z[r], kScaleLog2, -l2[r]));
          acc[b] += s;
        }
      }
    }
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const float tot = acc[b] + __shfl_xor(acc[b], 32);
      const int j = (4 * g + b) * 32 + l32;
      if (half == 0 && j < N) {
        s_sal[j] = tot;
        L.sal[(int64_t)h * N + j] = tot;
      }
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(NT) void admit_kernel(AdmitArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int H = a.n_heads, N = a.n_tokens, tid = threadIdx.x;
  const int layer = blockIdx.x / H, h = blockIdx.x % H;
  const AdmitLayer& L = a.layer[layer];
  float* s_sal = reinterpret_cast<float*>(smem);
  unsigned char* rest = smem + (((size_t)N * 4 + 15) & ~(size_t)15);

  if (a.mode == kModeSelect) {
    for (int j = tid; j < N; j += NT) s_sal[j] = L.sal[(int64_t)h * N + j];
    __syncthreads();
  } else {
    const int nq_pad = (a.n_q + 31) & ~31;
    float* s_lse2 = reinterpret_cast<float*>(rest);
    uint16_t* s_q = a.stage_queries ? reinterpret_cast<uint16_t*>(rest + (size_t)nq_pad * 4) : nullptr;
    saliency(a, L, h, s_sal, s_lse2, s_q);
    if (a.mode == kModeSaliency) return;
  }
  select_and_append(a, L, h, s_sal, reinterpret_cast<int32_t*>(rest));
}

}  // namespace

size_t admit_lds_bytes(const AdmitArgs& a) {
  const size_t sal = ((size_t)a.n_tokens * 4 + 15) & ~(size_t)15;
  const size_t nq_pad = (size_t)((a.n_q + 31) & ~31);
  size_t rest = (size_t)a.budget * 4;
  if (a.mode != kModeSelect) {
    size_t sal_rest = nq_pad * 4 + (a.stage_queries ? nq_pad * QS_STRIDE * 2 : 0);
    rest = rest > sal_rest ? rest : sal_rest;
  }
  return sal + rest;
}

int admit_max_dynamic_lds(int max_lds) { return max_lds - kAdmitStaticLdsMargin; }

hipError_t launch_admit(const AdmitArgs& a, int max_lds, hipStream_t s) {
  static int attr_set = 0;
  const int limit = admit_max_dynamic_lds(max_lds);
  if (attr_set != limit) {
    hipError_t e = hipFuncSetAttribute((const void*)admit_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       limit);
    if (e != hipSuccess) return e;
    attr_set = limit;
  }
  hipLaunchKernelGGL(admit_kernel, dim3((unsigned)(a.n_layers * a.n_heads)), dim3(NT), admit_lds_bytes(a), s, a);
  return hipGetLastError();
}

}  // namespace rv
