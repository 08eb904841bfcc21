// admit.hip -- LSE-saliency, per-head top-k and memory append, gfx950.
//
// Saliency (Sec. 3.3, saliency score and the A_ij equation): for key j of the frame,
//   S_j = sum over sampled queries i of exp(q_i . k_j / 8 - LSE_i),
// with the LSE the attention pass saved, so every term is an exact attention
// probability and no score matrix is stored.  A workgroup owns 128 keys of one head
// (32 per wave) and sweeps all sampled queries in blocks of 32 with
// v_mfma_f32_32x32x16_bf16 (Z = Q~ K^T: each lane owns one key column), applies the
// exponential in fp32 and sums in a fixed order -- in-lane, then across the two lane
// halves -- so S is bit-reproducible and no atomics touch it.
//
// Selection (Sec. 3.3 Eq. 6, head-specific retention): the last workgroup of a
// (layer, head) to finish its saliency chunk (atomic counter) selects the `budget`
// largest S_j, equal values ordered by lower index: an MSB-first radix select on the
// fp32 bit patterns (order-preserving for S >= 0) finds the exact threshold value and
// how many of its ties to take; a block scan then emits the chosen indices in
// ascending order.  The same workgroup copies the chosen K/V rows into the memory
// arena at rows mem_len.. and records their provenance.
#include "rv_internal.h"

namespace rv {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int D = kHeadDim;
constexpr int NT = kAdmitThreads;
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kScaleLog2 = kLog2e * 0.125f;

// Inclusive prefix sum over the 256 threads of a workgroup (4 waves).
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
  __shared__ int s_wave[4];
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
    hist[tid] = 0u;
    __syncthreads();
    for (int j = tid; j < N; j += NT) {
      const unsigned int kj = __float_as_uint(sal[j]);
      if ((kj & mask) == prefix) atomicAdd(&hist[(kj >> shift) & 255u], 1u);
    }
    __syncthreads();
    // thread i holds bin 255 - i, so the inclusive scan is the count of digits >= bin
    const int b = 255 - tid;
    const int cnt = (int)hist[b];
    const int ge = block_inclusive_scan(cnt, s_wave);
    const int gt = ge - cnt;
    if (gt < need && need <= ge) {
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

// Select for (layer, h) from L.sal and append the chosen rows.
__device__ void select_and_append(const AdmitArgs& a, const AdmitLayer& L, int h, int32_t* s_idx) {
  const int N = a.n_tokens, H = a.n_heads, k = a.budget, tid = threadIdx.x;
  if (k == 0) return;
  select_topk(L.sal + (int64_t)h * N, N, k, s_idx);

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

__global__ __launch_bounds__(NT) void admit_kernel(AdmitArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ int s_last;
  const int H = a.n_heads, N = a.n_tokens, tid = threadIdx.x;

  if (a.mode == kModeSelect) {
    const int layer = blockIdx.x / H, h = blockIdx.x % H;
    select_and_append(a, a.layer[layer], h, reinterpret_cast<int32_t*>(smem));
    return;
  }

  int b = blockIdx.x;
  const int chunk = b % a.key_chunks;
  b /= a.key_chunks;
  const int h = b % H, layer = b / H;
  const AdmitLayer& L = a.layer[layer];

  // LSE of the sampled queries in log2 units; padding rows get +inf (weight 0).
  float* s_lse2 = reinterpret_cast<float*>(smem);
  const int nq_pad = (a.n_q + 31) & ~31;
  for (int i = tid; i < nq_pad; i += NT)
    s_lse2[i] = i < a.n_q ? L.lse[(int64_t)h * N + a.qidx[i]] * kLog2e : __builtin_inff();
  __syncthreads();

  const int lane = tid & 63, wave = tid >> 6, l32 = lane & 31, half = lane >> 5;
  const int j0 = chunk * kSalBK + wave * 32;
  const int j = j0 + l32;
  if (j0 < N) {
    // B operand (K^T): this lane's key, head dims ds*16 + half*8 .. +7.
    bf16x8 kf[4];
    if (j < N) {
      const uint16_t* kp = L.K + ((int64_t)j * H + h) * D + half * 8;
#pragma unroll
      for (int ds = 0; ds < 4; ++ds) kf[ds] = *reinterpret_cast<const bf16x8*>(kp + ds * 16);
    } else {
#pragma unroll
      for (int ds = 0; ds < 4; ++ds) kf[ds] = bf16x8{};
    }
    float acc = 0.f;
    for (int qb = 0; qb < nq_pad; qb += 32) {
      const int qa = qb + l32;
      bf16x8 qf[4];
      if (qa < a.n_q) {
        const uint16_t* qp = L.Q + ((int64_t)a.qidx[qa] * H + h) * D + half * 8;
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) qf[ds] = *reinterpret_cast<const bf16x8*>(qp + ds * 16);
      } else {
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) qf[ds] = bf16x8{};
      }
      f32x16 z = {};
#pragma unroll
      for (int ds = 0; ds < 4; ++ds) z = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[ds], kf[ds], z, 0, 0, 0);
      // entry r: sampled query qb + 8*(r/4) + 4*half + r%4 against this lane's key
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float l2 = s_lse2[qb + 8 * (r >> 2) + 4 * half + (r & 3)];
        acc += __builtin_amdgcn_exp2f(fmaf(z[r], kScaleLog2, -l2));
      }
    }
    acc += __shfl_xor(acc, 32);
    if (half == 0 && j < N) L.sal[(int64_t)h * N + j] = acc;
  }
  if (a.mode == kModeSaliency) return;

  __threadfence();
  __syncthreads();
  if (tid == 0) s_last = atomicAdd(&a.counters[layer * H + h], 1) == a.key_chunks - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  select_and_append(a, L, h, reinterpret_cast<int32_t*>(smem));
  if (tid == 0) a.counters[layer * H + h] = 0;  // ready for the next launch
}

}  // namespace

hipError_t launch_admit(const AdmitArgs& a, hipStream_t s) {
  const int nq_pad = (a.n_q + 31) & ~31;
  size_t lds = 0;
  unsigned grid;
  if (a.mode == kModeSelect) {
    lds = (size_t)a.budget * sizeof(int32_t);
    grid = (unsigned)(a.n_layers * a.n_heads);
  } else {
    lds = (size_t)nq_pad * sizeof(float);
    if (a.mode == kModeBoth) lds = lds > (size_t)a.budget * 4 ? lds : (size_t)a.budget * 4;
    grid = (unsigned)(a.n_layers * a.n_heads * a.key_chunks);
  }
  if (lds < 16) lds = 16;
  hipLaunchKernelGGL(admit_kernel, dim3(grid), dim3(NT), lds, s, a);
  return hipGetLastError();
}

}  // namespace rv
