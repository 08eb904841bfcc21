// synth_gpu.hip -- GPU twin of the seeded stream generator (see synth.py for the recipe).
// Not part of the method: it only makes benchmark inputs resident in HBM.
#include "../../include/rv_synth.h"

#include <hip/hip_runtime.h>
#include <math.h>

namespace {

constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;
constexpr uint32_t kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;
constexpr int kIHMean = 262140;
constexpr double kIHSd = 53509.91992145008;  // sqrt(8 * (65536^2 - 1) / 12), as the CPU generator
constexpr int kTagPlant = 3;  // Q, K, V use tags 0, 1, 2 (tensor index within a layer)
constexpr int kTagLogn = 6;   // heavy-tailed key scales
constexpr int kMaxPlantTokens = 8192;

struct U4 {
  uint32_t x, y, z, w;
};

// Philox4x32 with 10 rounds (Salmon et al., SC'11).
__device__ __forceinline__ U4 philox10(U4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += kW0;
      k1 += kW1;
    }
    const uint64_t p0 = (uint64_t)kM0 * c.x;
    const uint64_t p1 = (uint64_t)kM1 * c.z;
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    c = U4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
  }
  return c;
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ __forceinline__ uint16_t normal_elem(uint64_t e, uint32_t frame, uint32_t stream_id,
                                                uint32_t k0, uint32_t k1, float scale) {
  const U4 w = philox10(U4{(uint32_t)e, (uint32_t)(e >> 32), frame, stream_id}, k0, k1);
  const int s = (int)(w.x & 0xFFFFu) + (int)(w.x >> 16) + (int)(w.y & 0xFFFFu) + (int)(w.y >> 16) +
                (int)(w.z & 0xFFFFu) + (int)(w.z >> 16) + (int)(w.w & 0xFFFFu) + (int)(w.w >> 16);
  return f32_to_bf16_rne((float)(s - kIHMean) * scale);
}

// out = [n_layers][3][n][H][d]; grid-stride over all elements.  ln_sigma > 0: every key row
// (token j, head h) is scaled by exp(ln_sigma * xi), xi the near-Gaussian of element j * H + h
// of stream (frame, layer << 8 | 6): fp64 exponential, rounded to fp32, one fp32 multiply,
// rounded to bf16 (the CPU generator's steps).
__global__ void gen_qkv_kernel(uint64_t seed, uint32_t frame, int layer0, int n_layers, int64_t per_tensor,
                               float scale, double ln_sigma, uint16_t* out) {
  const int64_t total = per_tensor * 3 * n_layers;
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < total;
       g += (int64_t)gridDim.x * blockDim.x) {
    const int64_t tensor = g / per_tensor;
    const int64_t e = g - tensor * per_tensor;
    const int layer = layer0 + (int)(tensor / 3);
    const int tag = (int)(tensor % 3);
    uint16_t v = normal_elem((uint64_t)e, frame, ((uint32_t)layer << 8) | (uint32_t)tag, k0, k1, scale);
    if (tag == 1 && ln_sigma > 0.0) {
      const uint64_t row = (uint64_t)e / 64;  // token * H + head
      const U4 w = philox10(U4{(uint32_t)row, (uint32_t)(row >> 32), frame, ((uint32_t)layer << 8) | (uint32_t)kTagLogn},
                            k0, k1);
      const int ih = (int)(w.x & 0xFFFFu) + (int)(w.x >> 16) + (int)(w.y & 0xFFFFu) + (int)(w.y >> 16) +
                     (int)(w.z & 0xFFFFu) + (int)(w.z >> 16) + (int)(w.w & 0xFFFFu) + (int)(w.w >> 16) - kIHMean;
      const float s = (float)exp(ln_sigma * ((double)ih / kIHSd));
      v = f32_to_bf16_rne(bf16_to_f32(v) * s);
    }
    out[g] = v;
  }
}

__global__ void gen_normal_kernel(uint64_t seed, uint32_t frame, uint32_t stream_id, int64_t n, float scale,
                                  uint16_t* out) {
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x)
    out[e] = normal_elem((uint64_t)e, frame, stream_id, k0, k1, scale);
}

// One workgroup per (layer, head): planted rows = alpha * |k_j| * qbar / |qbar|.
__global__ __launch_bounds__(256) void plant_kernel(uint64_t seed, uint32_t frame, int layer0, int n, int H,
                                                    int n_plant, double alpha, uint16_t* out) {
#pragma clang fp contract(off)
  __shared__ double s_part[4][64];
  __shared__ double s_qbar[64];
  __shared__ int s_perm[kMaxPlantTokens];
  __shared__ double s_ratio_den;
  const int li = blockIdx.x / H, h = blockIdx.x % H;
  const int layer = layer0 + li;
  const int64_t per_tensor = (int64_t)n * H * 64;
  const uint16_t* Q = out + (int64_t)li * 3 * per_tensor;
  uint16_t* K = out + ((int64_t)li * 3 + 1) * per_tensor;
  const int tid = threadIdx.x, e = tid & 63, part = tid >> 6;

  // qbar: sum of the head's queries in fp64 (exact for these bf16 magnitudes)
  double acc = 0.0;
  for (int i = part; i < n; i += 4) acc += (double)bf16_to_f32(Q[((int64_t)i * H + h) * 64 + e]);
  s_part[part][e] = acc;
  for (int i = tid; i < n; i += 256) s_perm[i] = i;
  __syncthreads();
  if (tid < 64) s_qbar[tid] = ((s_part[0][tid] + s_part[1][tid]) + s_part[2][tid]) + s_part[3][tid];
  __syncthreads();
  if (tid == 0) {
    double nq2 = 0.0;
    for (int d = 0; d < 64; ++d) nq2 = nq2 + s_qbar[d] * s_qbar[d];
    s_ratio_den = nq2;
    // partial Fisher-Yates with Philox words, counter (h, block, frame, layer<<8|3)
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    U4 w{};
    for (int i = 0; i < n_plant; ++i) {
      if ((i & 3) == 0)
        w = philox10(U4{(uint32_t)h, (uint32_t)(i >> 2), frame, ((uint32_t)layer << 8) | (uint32_t)kTagPlant},
                     k0, k1);
      const uint32_t word = (i & 3) == 0 ? w.x : (i & 3) == 1 ? w.y : (i & 3) == 2 ? w.z : w.w;
      const int j = i + (int)(word % (uint32_t)(n - i));
      const int t = s_perm[i];
      s_perm[i] = s_perm[j];
      s_perm[j] = t;
    }
  }
  __syncthreads();
  const double nq2 = s_ratio_den;
  if (nq2 == 0.0) return;
  const double den = sqrt(nq2);
  // wave `part` rewrites planted rows part, part+4, ...; lane e writes head dim e
  for (int p = part; p < n_plant; p += 4) {
    uint16_t* kr = K + ((int64_t)s_perm[p] * H + h) * 64;
    double nk2 = 0.0;
    for (int d = 0; d < 64; ++d) {
      const double v = (double)bf16_to_f32(kr[d]);
      nk2 = nk2 + v * v;
    }
    const double ratio = (alpha * sqrt(nk2)) / den;
    const uint16_t nv = f32_to_bf16_rne((float)(ratio * s_qbar[e]));
    __builtin_amdgcn_wave_barrier();
    kr[e] = nv;
  }
}

// ---- unit-rate probe (benchmark support, not part of the method) ----------------------
// Waves of 512-thread workgroups (wave w runs on SIMD w % 4) repeat a fixed loop body:
// MFMA body = 4 independent v_mfma_f32_32x32x16_bf16; VALU body = 8 independent chains of
// 2 x (FMA, v_exp_f32, add), i.e. 16 exponentials and 32 other VALU instructions.
// mode 0: waves 0-3 MFMA only; 1: waves 0-3 VALU only; 2: waves 0-3 MFMA and waves 4-7
// VALU (one of each per SIMD); 3: waves 0-3 both bodies in one instruction stream; 4: all
// eight waves MFMA only (two per SIMD); 5: as 4 with all-zero MFMA operands; 6: all eight
// waves VALU only (two per SIMD).  Single-unit bodies (issue_rate_kernel): 7 / 8: 32
// independent FMAs per iteration on one / two waves per SIMD; 9 / 10: 32 independent
// v_exp_f32 per iteration on one / two waves per SIMD.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

template <int MODE>
__global__ __launch_bounds__(512) void unit_rate_kernel(float* out, int iters) {
  const int w = threadIdx.x >> 6;
  const bool do_mfma = (MODE == 1 || MODE == 6) ? false : (MODE == 4 || MODE == 5) ? true : w < 4;
  const bool do_valu = MODE == 6 ? true : (MODE == 0 || MODE >= 4) ? false : MODE == 2 ? w >= 4 : w < 4;
  bf16x8_t a, b;
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(MODE == 5 ? 0.f : 0.001f * (threadIdx.x + i));
    b[i] = (__bf16)(MODE == 5 ? 0.f : 0.002f * i);
  }
  // Opaque to the compiler: otherwise it rebuilds the constant operand inside the loop,
  // and each rewrite waits for the previous MFMAs to finish reading it.
  asm volatile("" : "+v"(a), "+v"(b));
  f32x16_t c0 = {}, c1 = {}, c2 = {}, c3 = {};
  float x[8];
  for (int i = 0; i < 8; ++i) x[i] = 0.01f * (threadIdx.x & 7) + i;
  for (int it = 0; it < iters; ++it) {
    if (do_mfma) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
    }
    if (do_valu) {
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int i = 0; i < 8; ++i) x[i] = __builtin_amdgcn_exp2f(fmaf(x[i], 0.5f, -0.25f)) + 0.1f;
    }
  }
  float s = 0.f;
  for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  for (int i = 0; i < 8; ++i) s += x[i];
  out[(int64_t)blockIdx.x * 512 + threadIdx.x] = s;
}

// MODE 7/8: FMA body, 9/10: exponential body; one wave per SIMD (waves 0-3) in 7 and 9,
// two (all eight) in 8 and 10.  Every FMA and every exponential of an iteration is
// independent of the others, so only the unit's rate and one wave's issue limit it.
template <int MODE>
__global__ __launch_bounds__(512) void issue_rate_kernel(float* out, int iters) {
  const bool active = (MODE == 8 || MODE == 10) || (threadIdx.x >> 6) < 4;
  float x[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) x[i] = 0.001f * (threadIdx.x & 15) + 0.01f * i;
  float a = 0.5f + 0.0001f * threadIdx.x, b = -0.25f;
  asm volatile("" : "+v"(a), "+v"(b));
  if (active) {
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int i = 0; i < 32; ++i) x[i] = (MODE == 7 || MODE == 8) ? fmaf(x[i], a, b) : __builtin_amdgcn_exp2f(-x[i]);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 32; ++i) s += x[i];
  out[(int64_t)blockIdx.x * 512 + threadIdx.x] = s;
}

}  // namespace

extern "C" int rvs_unit_rates(int n_workgroups, int iters, float* ns_per_iter) {
  if (n_workgroups < 1 || n_workgroups > 65536 || iters < 1 || !ns_per_iter) return 1;
  float* out = nullptr;
  if (hipMalloc(&out, (size_t)n_workgroups * 512 * sizeof(float)) != hipSuccess) return 4;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = 0;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) rc = 4;
  for (int m = 0; rc == 0 && m < 11; ++m) {
    for (int rep = 0; rc == 0 && rep < 2; ++rep) {  // the first launch warms up
      if (hipEventRecord(e0, nullptr) != hipSuccess) rc = 4;
      if (m == 0) hipLaunchKernelGGL(unit_rate_kernel<0>, dim3(n_workgroups), dim3(512), 0, nullptr, out, iters);
      if (m == 1) hipLaunchKernelGGL(unit_rate_kernel<1>, dim3(n_workgroups), dim3(512), 0, nullptr, out, iters);
      if (m == 2) hipLaunchKernelGGL(unit_rate_kernel<2>, dim3(n_workgroups), dim3(512), 0, nullptr, out, iters);
      if (m == 3) hipLaunchKernelGGL(unit_rate_kernel<3>, dim3(n_workgroups), dim3(512), 0, nullptr, out, iters);
      if (m == 4) hipLaunchKernelGGL(unit_rate_kernel<4>, dim3(n_workgroups), dim3(512), 0, nullptr, out, iters);
      if (m == 5) hipLaunchKernelGGL(unit_rate_kernel<5>, dim3(n_workgroups), dim3(512), 0, nullptr, out, iters);
      if (m == 6) hipLaunchKernelGGL(unit_rate_kernel<6>, dim3(n_workgroups), dim3(512), 0, nullptr, out, iters);
      if (m == 7) hipLaunchKernelGGL(issue_rate_kernel<7>, dim3(n_workgroups), dim3(512), 0, nullptr, out, iters);
      if (m == 8) hipLaunchKernelGGL(issue_rate_kernel<8>, dim3(n_workgroups), dim3(512), 0, nullptr, out, iters);
      if (m == 9) hipLaunchKernelGGL(issue_rate_kernel<9>, dim3(n_workgroups), dim3(512), 0, nullptr, out, iters);
      if (m == 10) hipLaunchKernelGGL(issue_rate_kernel<10>, dim3(n_workgroups), dim3(512), 0, nullptr, out, iters);
      if (hipGetLastError() != hipSuccess || hipEventRecord(e1, nullptr) != hipSuccess ||
          hipEventSynchronize(e1) != hipSuccess)
        rc = 4;
      float ms = 0.f;
      if (rc == 0 && hipEventElapsedTime(&ms, e0, e1) != hipSuccess) rc = 4;
      if (rc == 0) ns_per_iter[m] = ms * 1e6f / (float)iters;
    }
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  (void)hipFree(out);
  return rc;
}

extern "C" int rvs_normal_bf16(uint64_t seed, uint32_t frame, int layer, int tag, int64_t n, float sigma,
                               uint16_t* out, void* stream) {
  if (n < 0 || (n > 0 && !out) || layer < 0 || tag < 0 || tag > 255) return 1;
  if (n == 0) return 0;
  const float scale = (float)((double)sigma / kIHSd);
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(gen_normal_kernel, dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0,
                     (hipStream_t)stream, seed, frame, ((uint32_t)layer << 8) | (uint32_t)tag, n, scale, out);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}

extern "C" int rvs_frame_qkv(uint64_t seed, uint32_t frame, int layer0, int n_layers, int n_tokens, int n_heads,
                             int head_dim, float sigma, int n_plant, double alpha, double key_lognormal_sigma,
                             uint16_t* out, void* stream) {
  if (!out || layer0 < 0 || n_layers < 1 || n_tokens < 1 || n_tokens > kMaxPlantTokens || n_heads < 1 ||
      head_dim != 64 || n_plant < 0 || n_plant > n_tokens || !(key_lognormal_sigma >= 0.0))
    return 1;
  const float scale = (float)((double)sigma / kIHSd);
  const int64_t per_tensor = (int64_t)n_tokens * n_heads * head_dim;
  const int64_t total = per_tensor * 3 * n_layers;
  const int64_t blocks = (total + 255) / 256;
  hipStream_t s = (hipStream_t)stream;
  hipLaunchKernelGGL(gen_qkv_kernel, dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0, s, seed,
                     frame, layer0, n_layers, per_tensor, scale, key_lognormal_sigma, out);
  if (hipGetLastError() != hipSuccess) return 4;
  if (n_plant > 0) {
    hipLaunchKernelGGL(plant_kernel, dim3((unsigned)(n_layers * n_heads)), dim3(256), 0, s, seed, frame, layer0,
                       n_tokens, n_heads, n_plant, alpha, out);
    if (hipGetLastError() != hipSuccess) return 4;
  }
  return 0;
}
