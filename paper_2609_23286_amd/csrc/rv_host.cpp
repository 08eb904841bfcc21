// rv_host.cpp -- librv host side: argument checks, error state, memory arenas,
// per-device scratch workspace and kernel launches.  See include/rv.h for the contract.
#include "../../include/rv.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "rv_internal.h"

namespace {

thread_local std::string g_err;

rv_status fail(rv_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

rv_status hip_fail(hipError_t e, const char* what) {
  return fail(e == hipErrorOutOfMemory ? RV_ERR_OOM : RV_ERR_HIP, "%s: %s", what,
              hipGetErrorString(e));
}

#define RV_HIP(call, what)                       \
  do {                                           \
    hipError_t e_ = (call);                      \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)


// ---- per-device context: placement calibration, limits, scratch workspace --------
//
// Every compute call plans and launches with what rv_init recorded for the current
// device and writes its split-KV partials into the workspace allocated there, so that
// no compute call allocates device memory or synchronises.  rv_reserve_workspace is the
// other call that may allocate (a larger workspace for forced work plans, the saliency
// staging of rv_admit_layers*).
struct Workspace {
  bool ready = false;
  int n_cus = 0;
  int max_lds = 0;
  int n_queues = 1;          // attention work queues: one per XCD
  float* part = nullptr;     // attention partial slots, kAttnSlotFloats floats each
  int64_t part_slots = 0;
  float* sal = nullptr;      // saliency staging when the caller passes none
  size_t sal_floats = 0;
  float* static_part = nullptr;  // this device's copy of the static partial-slot array
};

std::mutex g_ws_mu;
std::map<int, Workspace> g_ws;

// Replaces *p by a buffer of `need` floats if it holds fewer.  Earlier launches may still
// use the old buffer, so the device is synchronised before it is freed.
rv_status grow_floats(float** p, size_t* have, size_t need, const char* what) {
  if (*have >= need) return RV_OK;
  float* q = nullptr;
  hipError_t e = hipMalloc(&q, need * sizeof(float));
  if (e != hipSuccess) return hip_fail(e, what);
  if (*p) {
    e = hipDeviceSynchronize();
    if (e != hipSuccess) {
      (void)hipFree(q);
      return hip_fail(e, what);
    }
    (void)hipFree(*p);
  }
  *p = q;
  *have = need;
  return RV_OK;
}

rv_status reserve_partials(Workspace* ws, int64_t slots) {
  if (slots <= ws->part_slots) return RV_OK;
  size_t have = (size_t)ws->part_slots * rv::kAttnSlotFloats;
  rv_status st = grow_floats(&ws->part, &have, (size_t)slots * rv::kAttnSlotFloats, "attention workspace");
  if (st == RV_OK) ws->part_slots = slots;
  return st;
}

// Reads the CU count and the LDS limit, counts the XCDs (distinct XCC ids seen by a
// probe launch: the attention kernel keeps one work queue per XCD so that the query
// tiles of a head share an L2; placement only steers locality, results never depend on
// it), and allocates the partial slots of every default work plan.  Synchronous.
rv_status init_device(Workspace* ws, int dev) {
  if (ws->ready) return RV_OK;
  RV_HIP(hipDeviceGetAttribute(&ws->n_cus, hipDeviceAttributeMultiprocessorCount, dev), "CU count");
  RV_HIP(hipDeviceGetAttribute(&ws->max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev), "LDS limit");
  const int n_probe = 4096;
  int* d_ids = nullptr;
  RV_HIP(hipMalloc(&d_ids, n_probe * sizeof(int)), "placement probe");
  std::vector<int> ids(n_probe, -1);
  hipError_t e = rv::launch_xcc_probe(d_ids, n_probe, nullptr);
  if (e == hipSuccess) e = hipMemcpy(ids.data(), d_ids, n_probe * sizeof(int), hipMemcpyDeviceToHost);
  (void)hipFree(d_ids);
  if (e != hipSuccess) return hip_fail(e, "placement probe");
  std::vector<int> distinct;
  for (int id : ids)
    if (std::find(distinct.begin(), distinct.end(), id) == distinct.end()) distinct.push_back(id);
  ws->n_queues = std::max(1, std::min((int)distinct.size(), rv::kMaxQueues));
  RV_HIP(rv::static_scratch_address(&ws->static_part), "static scratch address");
  rv_status st = reserve_partials(ws, rv::default_partial_slots(ws->n_cus, ws->n_queues));
  if (st != RV_OK) return st;
  ws->ready = true;
  return RV_OK;
}

// The current device's context, initialised if need be (set-up calls only).
rv_status setup_ws(Workspace** out) {
  int dev = 0;
  RV_HIP(hipGetDevice(&dev), "hipGetDevice");
  Workspace* ws = &g_ws[dev];
  rv_status st = init_device(ws, dev);
  if (st != RV_OK) return st;
  *out = ws;
  return RV_OK;
}

// The current device's context for a compute call: it must have been initialised.
rv_status ready_ws(Workspace** out) {
  int dev = 0;
  RV_HIP(hipGetDevice(&dev), "hipGetDevice");
  auto it = g_ws.find(dev);
  if (it == g_ws.end() || !it->second.ready)
    return fail(RV_ERR_INVALID, "librv is not initialised on device %d: call rv_init() first", dev);
  *out = &it->second;
  return RV_OK;
}

rv_status check_qsub(const rv_qsub* qs, int n_tokens) {
  const char* why = rv::qsub_problem(qs, n_tokens);
  if (why) return fail(RV_ERR_INVALID, "%s", why);
  return RV_OK;
}

}  // namespace

// ---- memory arena ----------------------------------------------------------------
struct rv_mem_s {
  int device = 0;
  int n_heads = 0;
  int64_t cap = 0, max_tokens = 0, len = 0;
  uint16_t* K = nullptr;
  uint16_t* V = nullptr;
  int32_t* prov = nullptr;
};

namespace {

// Arenas are stream-ordered allocations (hipMallocAsync / hipFreeAsync on the stream of
// the call that creates, grows or frees them), so that growth needs no host
// synchronisation: the new arenas, the copy of the valid rows and the release of the old
// ones all take their place in the stream's order.
void arena_free(uint16_t* K, uint16_t* V, int32_t* prov, hipStream_t s) {
  if (K) (void)hipFreeAsync(K, s);
  if (V) (void)hipFreeAsync(V, s);
  if (prov) (void)hipFreeAsync(prov, s);
}

rv_status arena_alloc(int n_heads, int64_t cap, uint16_t** K, uint16_t** V, int32_t** prov, hipStream_t s) {
  *K = *V = nullptr;
  *prov = nullptr;
  if (cap == 0) return RV_OK;
  const size_t rows = (size_t)n_heads * (size_t)cap;
  hipError_t e = hipMallocAsync(reinterpret_cast<void**>(K), rows * rv::kHeadDim * 2, s);
  if (e == hipSuccess) e = hipMallocAsync(reinterpret_cast<void**>(V), rows * rv::kHeadDim * 2, s);
  if (e == hipSuccess) e = hipMallocAsync(reinterpret_cast<void**>(prov), rows * 2 * sizeof(int32_t), s);
  if (e != hipSuccess) {
    arena_free(*K, *V, *prov, s);
    *K = *V = nullptr;
    *prov = nullptr;
    return hip_fail(e, "memory arena allocation");
  }
  return RV_OK;
}

// Grows m to hold at least `tokens` rows per head; strong guarantee on failure (every
// step that can fail does so when it is enqueued, before m changes).  Stream-ordered on
// s: the old arenas are released on s after the copy that reads them.
rv_status arena_reserve(rv_mem m, int64_t tokens, hipStream_t s) {
  if (tokens <= m->cap) return RV_OK;
  if (tokens > m->max_tokens)
    return fail(RV_ERR_CAPACITY, "memory needs %lld rows per head, max_tokens is %lld",
                (long long)tokens, (long long)m->max_tokens);
  int64_t cap = std::max<int64_t>(tokens, std::min<int64_t>(m->max_tokens, std::max<int64_t>(256, m->cap * 2)));
  uint16_t *K, *V;
  int32_t* prov;
  rv_status st = arena_alloc(m->n_heads, cap, &K, &V, &prov, s);
  if (st != RV_OK) return st;
  hipError_t e = hipSuccess;
  if (m->len > 0) {
    const size_t row = rv::kHeadDim * 2;
    e = hipMemcpy2DAsync(K, cap * row, m->K, m->cap * row, m->len * row, m->n_heads,
                         hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess)
      e = hipMemcpy2DAsync(V, cap * row, m->V, m->cap * row, m->len * row, m->n_heads,
                           hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess)
      e = hipMemcpy2DAsync(prov, cap * 8, m->prov, m->cap * 8, m->len * 8, m->n_heads,
                           hipMemcpyDeviceToDevice, s);
  }
  if (e != hipSuccess) {
    arena_free(K, V, prov, s);
    return hip_fail(e, "memory growth copy");
  }
  arena_free(m->K, m->V, m->prov, s);
  m->K = K;
  m->V = V;
  m->prov = prov;
  m->cap = cap;
  return RV_OK;
}

rv_status check_device(rv_mem m) {
  int dev = 0;
  RV_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (dev != m->device)
    return fail(RV_ERR_INVALID, "memory lives on device %d but device %d is current", m->device, dev);
  return RV_OK;
}

}  // namespace

extern "C" {

const char* rv_last_error(void) { return g_err.c_str(); }

const char* rv_version(void) { return "librv 0.1 (gfx950)"; }

rv_status rv_mem_create(int n_heads, int head_dim, int64_t reserve_tokens, int64_t max_tokens,
                        rv_mem* out) {
  if (!out) return fail(RV_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (n_heads < 1) return fail(RV_ERR_INVALID, "n_heads must be >= 1 (got %d)", n_heads);
  if (head_dim != rv::kHeadDim) return fail(RV_ERR_INVALID, "head_dim must be 64 (got %d)", head_dim);
  if (reserve_tokens < 0 || max_tokens < 0 || reserve_tokens > max_tokens)
    return fail(RV_ERR_INVALID, "need 0 <= reserve_tokens <= max_tokens");
  {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    Workspace* ws;
    rv_status st = setup_ws(&ws);
    if (st != RV_OK) return st;
  }
  rv_mem m = new (std::nothrow) rv_mem_s;
  if (!m) return fail(RV_ERR_OOM, "host allocation failed");
  hipError_t e = hipGetDevice(&m->device);
  if (e != hipSuccess) {
    delete m;
    return hip_fail(e, "hipGetDevice");
  }
  m->n_heads = n_heads;
  m->max_tokens = max_tokens;
  rv_status st = arena_alloc(n_heads, reserve_tokens, &m->K, &m->V, &m->prov, nullptr);
  if (st == RV_OK) {  // ready for every stream
    e = hipStreamSynchronize(nullptr);
    if (e != hipSuccess) {
      arena_free(m->K, m->V, m->prov, nullptr);
      st = hip_fail(e, "memory arena allocation");
    }
  }
  if (st != RV_OK) {
    delete m;
    return st;
  }
  m->cap = reserve_tokens;
  *out = m;
  return RV_OK;
}

rv_status rv_mem_destroy(rv_mem m) {
  if (!m) return RV_OK;
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(m->device);
  (void)hipDeviceSynchronize();
  arena_free(m->K, m->V, m->prov, nullptr);
  (void)hipStreamSynchronize(nullptr);
  (void)hipSetDevice(prev);
  delete m;
  return RV_OK;
}

int64_t rv_mem_len(rv_mem m) { return m ? m->len : -1; }

int64_t rv_mem_capacity(rv_mem m) { return m ? m->cap : -1; }

rv_status rv_mem_view(rv_mem m, const void** memK, const void** memV, int64_t* head_stride_tokens) {
  if (!m || !memK || !memV || !head_stride_tokens) return fail(RV_ERR_INVALID, "NULL argument");
  *memK = m->K;
  *memV = m->V;
  *head_stride_tokens = m->cap;
  return RV_OK;
}

rv_status rv_mem_reserve(rv_mem m, int64_t tokens, void* stream) {
  if (!m) return fail(RV_ERR_INVALID, "memory is NULL");
  if (tokens < 0) return fail(RV_ERR_INVALID, "tokens must be >= 0");
  rv_status st = check_device(m);
  if (st != RV_OK) return st;
  return arena_reserve(m, tokens, (hipStream_t)stream);
}

rv_status rv_mem_reset(rv_mem m) {
  if (!m) return fail(RV_ERR_INVALID, "memory is NULL");
  m->len = 0;
  return RV_OK;
}

rv_status rv_mem_truncate(rv_mem m, int64_t n_rows) {
  if (!m) return fail(RV_ERR_INVALID, "memory is NULL");
  if (n_rows < 0 || n_rows > m->len)
    return fail(RV_ERR_INVALID, "n_rows must be in [0, length %lld] (got %lld)", (long long)m->len,
                (long long)n_rows);
  m->len = n_rows;
  return RV_OK;
}

rv_status rv_mem_write(rv_mem m, const void* K, const void* V, int64_t n_rows, int frame_id,
                       void* stream) {
  if (!m || (n_rows > 0 && (!K || !V))) return fail(RV_ERR_INVALID, "NULL argument");
  if (n_rows < 0) return fail(RV_ERR_INVALID, "n_rows must be >= 0");
  rv_status st = check_device(m);
  if (st != RV_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  const int64_t keep = m->len;
  m->len = 0;  // nothing to preserve: rows are overwritten
  st = arena_reserve(m, n_rows, s);
  if (st != RV_OK) {
    m->len = keep;
    return st;
  }
  if (n_rows > 0) {
    const size_t row = rv::kHeadDim * 2;
    std::vector<int32_t> prov((size_t)n_rows * 2);
    for (int64_t r = 0; r < n_rows; ++r) {
      prov[2 * r] = frame_id;
      prov[2 * r + 1] = (int32_t)r;
    }
    hipError_t e = hipMemcpy2DAsync(m->K, m->cap * row, K, n_rows * row, n_rows * row, m->n_heads,
                                    hipMemcpyDefault, s);
    if (e == hipSuccess)
      e = hipMemcpy2DAsync(m->V, m->cap * row, V, n_rows * row, n_rows * row, m->n_heads,
                           hipMemcpyDefault, s);
    for (int h = 0; e == hipSuccess && h < m->n_heads; ++h)
      e = hipMemcpyAsync(m->prov + (size_t)h * m->cap * 2, prov.data(), prov.size() * 4,
                         hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "rv_mem_write copy");
  }
  m->len = n_rows;
  return RV_OK;
}

rv_status rv_mem_read(rv_mem m, void* K, void* V, int32_t* prov, void* stream) {
  if (!m) return fail(RV_ERR_INVALID, "memory is NULL");
  rv_status st = check_device(m);
  if (st != RV_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if (m->len == 0) return RV_OK;
  const size_t row = rv::kHeadDim * 2;
  hipError_t e = hipSuccess;
  if (K) e = hipMemcpy2DAsync(K, m->len * row, m->K, m->cap * row, m->len * row, m->n_heads, hipMemcpyDefault, s);
  if (e == hipSuccess && V)
    e = hipMemcpy2DAsync(V, m->len * row, m->V, m->cap * row, m->len * row, m->n_heads, hipMemcpyDefault, s);
  if (e == hipSuccess && prov)
    e = hipMemcpy2DAsync(prov, m->len * 8, m->prov, m->cap * 8, m->len * 8, m->n_heads, hipMemcpyDefault, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "rv_mem_read copy");
  return RV_OK;
}

namespace {
constexpr char kSnapMagic[8] = {'R', 'V', 'M', 'E', 'M', 'v', '1', '\0'};

struct FileCloser {
  FILE* f;
  ~FileCloser() {
    if (f) fclose(f);
  }
};
}  // namespace

rv_status rv_mem_save(rv_mem m, const char* path) {
  if (!m || !path) return fail(RV_ERR_INVALID, "NULL argument");
  rv_status st = check_device(m);
  if (st != RV_OK) return st;
  const size_t n = (size_t)m->n_heads * (size_t)m->len;
  std::vector<uint16_t> K(n * rv::kHeadDim), V(n * rv::kHeadDim);
  std::vector<int32_t> prov(n * 2);
  st = rv_mem_read(m, K.data(), V.data(), prov.data(), nullptr);
  if (st != RV_OK) return st;
  FileCloser fc{fopen(path, "wb")};
  if (!fc.f) return fail(RV_ERR_IO, "cannot open %s for writing", path);
  const int32_t hdr[2] = {m->n_heads, rv::kHeadDim};
  const int64_t len = m->len;
  bool ok = fwrite(kSnapMagic, 1, 8, fc.f) == 8 && fwrite(hdr, 4, 2, fc.f) == 2 && fwrite(&len, 8, 1, fc.f) == 1;
  ok = ok && fwrite(K.data(), 2, K.size(), fc.f) == K.size() && fwrite(V.data(), 2, V.size(), fc.f) == V.size() &&
       fwrite(prov.data(), 4, prov.size(), fc.f) == prov.size();
  if (!ok || fflush(fc.f) != 0) return fail(RV_ERR_IO, "cannot write %s", path);
  return RV_OK;
}

rv_status rv_mem_load(rv_mem m, const char* path) {
  if (!m || !path) return fail(RV_ERR_INVALID, "NULL argument");
  rv_status st = check_device(m);
  if (st != RV_OK) return st;
  FileCloser fc{fopen(path, "rb")};
  if (!fc.f) return fail(RV_ERR_IO, "cannot open %s", path);
  char magic[8];
  int32_t hdr[2];
  int64_t len = -1;
  if (fread(magic, 1, 8, fc.f) != 8 || memcmp(magic, kSnapMagic, 8) != 0 || fread(hdr, 4, 2, fc.f) != 2 ||
      fread(&len, 8, 1, fc.f) != 1 || len < 0)
    return fail(RV_ERR_IO, "%s is not a memory snapshot", path);
  if (hdr[0] != m->n_heads || hdr[1] != rv::kHeadDim)
    return fail(RV_ERR_INVALID, "snapshot has %d heads of %d, memory has %d of %d", hdr[0], hdr[1], m->n_heads,
                rv::kHeadDim);
  if (len > m->max_tokens) return fail(RV_ERR_CAPACITY, "snapshot of %lld rows exceeds max_tokens", (long long)len);
  const size_t n = (size_t)m->n_heads * (size_t)len;
  std::vector<uint16_t> K(n * rv::kHeadDim), V(n * rv::kHeadDim);
  std::vector<int32_t> prov(n * 2);
  if (fread(K.data(), 2, K.size(), fc.f) != K.size() || fread(V.data(), 2, V.size(), fc.f) != V.size() ||
      fread(prov.data(), 4, prov.size(), fc.f) != prov.size() || fgetc(fc.f) != EOF)
    return fail(RV_ERR_IO, "%s is truncated or has trailing bytes", path);
  const int64_t keep = m->len;
  m->len = 0;  // every row is overwritten: nothing to carry over on growth
  st = arena_reserve(m, len, nullptr);
  m->len = keep;
  if (st != RV_OK) return st;
  if (len > 0) {
    const size_t row = rv::kHeadDim * 2;
    hipError_t e = hipMemcpy2D(m->K, m->cap * row, K.data(), len * row, len * row, m->n_heads, hipMemcpyHostToDevice);
    if (e == hipSuccess)
      e = hipMemcpy2D(m->V, m->cap * row, V.data(), len * row, len * row, m->n_heads, hipMemcpyHostToDevice);
    if (e == hipSuccess)
      e = hipMemcpy2D(m->prov, m->cap * 8, prov.data(), len * 8, len * 8, m->n_heads, hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "rv_mem_load copy");
  }
  m->len = len;
  return RV_OK;
}

rv_status rv_attention_plan(int n_tokens, int n_fkeys, int64_t mem_len, int n_heads, int n_cus, int n_queues,
                            rv_attn_plan* out) {
  static_assert(rv::kMaxQueues == 16, "rv_attn_plan's tables hold kMaxQueues entries");
  if (!out) return fail(RV_ERR_INVALID, "out is NULL");
  if (n_tokens < 1 || n_tokens > rv::kMaxTokens || n_fkeys < 0 || n_fkeys > n_tokens || mem_len < 0 ||
      n_heads < 1 || n_cus < 1 || n_queues < 1 || n_queues > rv::kMaxQueues)
    return fail(RV_ERR_INVALID, "plan sizes out of range");
  const rv::AttnPlan p = rv::plan_attention(n_cus, n_queues, n_tokens, n_fkeys, mem_len, n_heads);
  *out = rv_attn_plan{};
  out->n_units = p.n_units;
  out->q_tiles = p.q_tiles;
  out->T = p.T;
  out->U = p.U;
  out->E = p.E;
  out->E1 = p.E1;
  out->n_first = p.n_first;
  out->n_queues = n_queues;
  out->grid = p.grid;
  out->total_chunks = p.total_chunks;
  for (int q = 0; q <= n_queues; ++q) out->unit_base[q] = p.unit_base[q];
  for (int q = 0; q < n_queues; ++q) {
    out->n_chunks[q] = p.n_chunks[q];
    out->chunk_base[q] = p.chunk_base[q];
  }
  return RV_OK;
}

rv_status rv_init(void) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  Workspace* ws;
  return setup_ws(&ws);
}

rv_status rv_reserve_workspace(int n_tokens, int n_heads, int64_t max_mem_len, int n_layers) {
  if (n_tokens < 1 || n_tokens > rv::kMaxTokens || n_heads < 1 || n_layers < 1 || max_mem_len < 0)
    return fail(RV_ERR_INVALID, "bad workspace sizes");
  std::lock_guard<std::mutex> lk(g_ws_mu);
  Workspace* ws;
  rv_status st = setup_ws(&ws);
  if (st != RV_OK) return st;
  // the chunk count of a forced plan may grow with the context; a default plan's never does
  const rv::AttnPlan p = rv::plan_attention(ws->n_cus, ws->n_queues, n_tokens, n_tokens, max_mem_len, n_heads);
  st = reserve_partials(ws, rv::plan_partial_slots(p));
  if (st != RV_OK) return st;
  return grow_floats(&ws->sal, &ws->sal_floats,
                     (size_t)std::min(n_layers, rv::kMaxLayersPerLaunch) * n_heads * n_tokens, "saliency workspace");
}

rv_status rv_device_status(void) {
  RV_HIP(hipDeviceSynchronize(), "device synchronisation");
  RV_HIP(hipGetLastError(), "device status");
  return RV_OK;
}

}  // extern "C"

namespace {

// Attention (+ saliency) launch shared by the frame and staged entry points.  Keys: the
// mem_len rows of memK/memV, then n_fkeys frame rows of K/V ([n][H][64]).  The saliency's
// keys are the frame's rows j at sK + j * s_row + h * s_head.  Arguments are checked.
// use_static: the partial slots are the static array's (the allocation-free entry point).
// sal_tiles: the saliency is formed in the attention epilogue, per 128-query block, into
// sal_tiles ([H][q_tiles][N]) instead of by a separate launch into `saliency`.
rv_status attend_impl(const void* Q, const void* K, const void* V, int n_tokens, int n_fkeys, const void* memK,
                      const void* memV, int64_t mem_len, int64_t head_stride_tokens, int n_heads,
                      const rv_qsub* qs, void* out, float* lse, float* saliency, const void* sK, int64_t s_row,
                      int64_t s_head, hipStream_t s, bool use_static = false, float* sal_tiles = nullptr) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  Workspace* ws;
  rv_status st = ready_ws(&ws);
  if (st != RV_OK) return st;

  const rv::AttnPlan p = rv::plan_attention(ws->n_cus, ws->n_queues, n_tokens, n_fkeys, mem_len, n_heads);
  if (use_static) {
    if (rv::plan_partial_slots(p) > rv::kStaticScratchSlots)
      return fail(RV_ERR_CAPACITY,
                  "the work plan needs %lld attention partial slots, the static scratch array holds %d "
                  "(%zu bytes)", (long long)rv::plan_partial_slots(p), rv::kStaticScratchSlots,
                  (size_t)rv::kStaticScratchSlots * rv::kAttnSlotBytes);
  } else if (rv::plan_partial_slots(p) > ws->part_slots) {
    return fail(RV_ERR_CAPACITY,
                "the work plan needs %lld attention partial slots, the workspace holds %lld "
                "(a forced plan: call rv_reserve_workspace with this frame's sizes)",
                (long long)rv::plan_partial_slots(p), (long long)ws->part_slots);
  }

  rv::AttnArgs a{};
  a.Q = (const uint16_t*)Q;
  a.K = (const uint16_t*)K;
  a.V = (const uint16_t*)V;
  a.memK = (const uint16_t*)memK;
  a.memV = (const uint16_t*)memV;
  a.mem_len = mem_len;
  a.head_stride = head_stride_tokens;
  a.out = (uint16_t*)out;
  a.lse = lse;
  a.part = use_static ? ws->static_part : ws->part;
  a.n_tokens = n_tokens;
  a.n_fkeys = n_fkeys;
  a.n_heads = n_heads;
  a.q_tiles = p.q_tiles;
  a.nt_mem = p.nt_mem;
  a.T = p.T;
  a.U = p.U;
  a.n_units = p.n_units;
  a.n_queues = ws->n_queues;
  a.E = p.E;
  a.E1 = p.E1;
  a.n_first = p.n_first;
  for (int q = 0; q <= ws->n_queues; ++q) a.unit_base[q] = p.unit_base[q];
  for (int q = 0; q < ws->n_queues; ++q) {
    a.n_chunks[q] = p.n_chunks[q];
    a.chunk_base[q] = p.chunk_base[q];
  }
  if (sal_tiles) {
    rv::SalEpi e{};
    e.tiles = sal_tiles;
    e.K = (const uint16_t*)sK;
    e.kv_row = s_row;
    e.kv_head = s_head;
    e.q_base = qs->n_special;
    e.grid_w = qs->grid_w > 0 ? qs->grid_w : 1;
    e.grid_cells = qs->grid_h * qs->grid_w;
    e.stride = qs->stride;
    RV_HIP(rv::launch_attention_saliency(a, e, p.grid, s), "attention launch");
    return RV_OK;
  }
  // every unit whole in one chunk (no split) needs no merge launch
  RV_HIP(rv::launch_attention(a, p.grid, rv::plan_splits_units(p), s), "attention launch");

  if (saliency) {
    rv::AdmitArgs b{};
    b.layer[0].Q = (const uint16_t*)Q;
    b.layer[0].K = (const uint16_t*)sK;
    b.layer[0].kv_row = s_row;
    b.layer[0].kv_head = s_head;
    b.layer[0].lse = lse;
    b.layer[0].sal = saliency;
    rv::set_qsub(&b, *qs);
    b.n_tokens = n_tokens;
    b.n_heads = n_heads;
    b.n_layers = 1;
    b.mode = rv::kModeSaliency;
    b.sal_xcds = ws->n_queues;
    rv::plan_saliency(&b, n_heads, ws->n_cus, ws->max_lds);
    RV_HIP(rv::launch_admit(b, ws->max_lds, s), "saliency launch");
  }
  return RV_OK;
}

}  // namespace

extern "C" {

rv_status rv_attend_frame(const void* Q, const void* K, const void* V, int n_tokens, const void* memK,
                          const void* memV, int64_t mem_len, int64_t head_stride_tokens, int n_heads,
                          int head_dim, const rv_qsub* qs, void* out, float* lse, float* saliency,
                          void* stream) {
  if (n_tokens < 0 || n_tokens > rv::kMaxTokens)
    return fail(RV_ERR_INVALID, "n_tokens must be in [0, %d] (got %d)", rv::kMaxTokens, n_tokens);
  if (n_heads < 1) return fail(RV_ERR_INVALID, "n_heads must be >= 1");
  if (head_dim != rv::kHeadDim) return fail(RV_ERR_INVALID, "head_dim must be 64 (got %d)", head_dim);
  if (mem_len < 0) return fail(RV_ERR_INVALID, "mem_len must be >= 0");
  if (mem_len > 0 && (!memK || !memV)) return fail(RV_ERR_INVALID, "memK/memV NULL with mem_len > 0");
  if (mem_len > 0 && head_stride_tokens < mem_len)
    return fail(RV_ERR_INVALID, "head_stride_tokens (%lld) < mem_len (%lld)", (long long)head_stride_tokens,
                (long long)mem_len);
  if (n_tokens == 0) return RV_OK;
  if (!Q || !K || !V || !out || !lse) return fail(RV_ERR_INVALID, "Q, K, V, out and lse are required");
  if (saliency) {
    rv_status st = check_qsub(qs, n_tokens);
    if (st != RV_OK) return st;
  }
  return attend_impl(Q, K, V, n_tokens, n_tokens, memK, memV, mem_len, head_stride_tokens, n_heads, qs, out, lse,
                     saliency, K, (int64_t)n_heads * rv::kHeadDim, rv::kHeadDim, (hipStream_t)stream);
}

rv_status rv_attend_frame_fused(const void* Q, const void* K, const void* V, int n_tokens, const void* memK,
                                const void* memV, int64_t mem_len, int64_t head_stride_tokens, int n_heads,
                                int head_dim, const rv_qsub* qs, void* out, float* lse, float* sal_tiles,
                                void* stream) {
  if (n_tokens < 0 || n_tokens > rv::kMaxTokens)
    return fail(RV_ERR_INVALID, "n_tokens must be in [0, %d] (got %d)", rv::kMaxTokens, n_tokens);
  if (n_heads < 1) return fail(RV_ERR_INVALID, "n_heads must be >= 1");
  if (head_dim != rv::kHeadDim) return fail(RV_ERR_INVALID, "head_dim must be 64 (got %d)", head_dim);
  if (mem_len < 0) return fail(RV_ERR_INVALID, "mem_len must be >= 0");
  if (mem_len > 0 && (!memK || !memV)) return fail(RV_ERR_INVALID, "memK/memV NULL with mem_len > 0");
  if (mem_len > 0 && head_stride_tokens < mem_len)
    return fail(RV_ERR_INVALID, "head_stride_tokens (%lld) < mem_len (%lld)", (long long)head_stride_tokens,
                (long long)mem_len);
  if (n_tokens == 0) return RV_OK;
  if (!Q || !K || !V || !out || !lse || !sal_tiles)
    return fail(RV_ERR_INVALID, "Q, K, V, out, lse and sal_tiles are required");
  rv_status st = check_qsub(qs, n_tokens);
  if (st != RV_OK) return st;
  return attend_impl(Q, K, V, n_tokens, n_tokens, memK, memV, mem_len, head_stride_tokens, n_heads, qs, out, lse,
                     nullptr, K, (int64_t)n_heads * rv::kHeadDim, rv::kHeadDim, (hipStream_t)stream, false,
                     sal_tiles);
}

rv_status rv_attend_frame_noalloc(const void* Q, const void* K, const void* V, int n_tokens, const void* memK,
                                  const void* memV, int64_t mem_len, int64_t head_stride_tokens, int n_heads,
                                  int head_dim, const rv_qsub* qs, void* out, float* lse, float* saliency,
                                  void* stream) {
  if (n_tokens < 0 || n_tokens > rv::kMaxTokens)
    return fail(RV_ERR_INVALID, "n_tokens must be in [0, %d] (got %d)", rv::kMaxTokens, n_tokens);
  if (n_heads < 1) return fail(RV_ERR_INVALID, "n_heads must be >= 1");
  if (head_dim != rv::kHeadDim) return fail(RV_ERR_INVALID, "head_dim must be 64 (got %d)", head_dim);
  if (mem_len < 0) return fail(RV_ERR_INVALID, "mem_len must be >= 0");
  if (mem_len > 0 && (!memK || !memV)) return fail(RV_ERR_INVALID, "memK/memV NULL with mem_len > 0");
  if (mem_len > 0 && head_stride_tokens < mem_len)
    return fail(RV_ERR_INVALID, "head_stride_tokens (%lld) < mem_len (%lld)", (long long)head_stride_tokens,
                (long long)mem_len);
  if (n_tokens == 0) return RV_OK;
  if (!Q || !K || !V || !out || !lse) return fail(RV_ERR_INVALID, "Q, K, V, out and lse are required");
  if (saliency) {
    rv_status st = check_qsub(qs, n_tokens);
    if (st != RV_OK) return st;
  }
  return attend_impl(Q, K, V, n_tokens, n_tokens, memK, memV, mem_len, head_stride_tokens, n_heads, qs, out, lse,
                     saliency, K, (int64_t)n_heads * rv::kHeadDim, rv::kHeadDim, (hipStream_t)stream, true);
}

rv_status rv_mem_stage(rv_mem m, int n_tokens, void** K_tail, void** V_tail, int64_t* head_stride_tokens,
                       void* stream) {
  if (!m) return fail(RV_ERR_INVALID, "memory is NULL");
  if (n_tokens < 1 || n_tokens > rv::kMaxTokens)
    return fail(RV_ERR_INVALID, "n_tokens must be in [1, %d] (got %d)", rv::kMaxTokens, n_tokens);
  rv_status st = check_device(m);
  if (st != RV_OK) return st;
  {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    st = arena_reserve(m, m->len + n_tokens, (hipStream_t)stream);
    if (st != RV_OK) return st;
  }
  if (K_tail) *K_tail = m->K + m->len * rv::kHeadDim;
  if (V_tail) *V_tail = m->V + m->len * rv::kHeadDim;
  if (head_stride_tokens) *head_stride_tokens = m->cap;
  return RV_OK;
}

rv_status rv_mem_stage_frame(rv_mem m, const void* K, const void* V, int n_tokens, void* stream) {
  if (!K || !V) return fail(RV_ERR_INVALID, "K and V are required");
  rv_status st = rv_mem_stage(m, n_tokens, nullptr, nullptr, nullptr, stream);
  if (st != RV_OK) return st;
  RV_HIP(rv::launch_stage(m->K + m->len * rv::kHeadDim, m->V + m->len * rv::kHeadDim, m->cap,
                          (const uint16_t*)K, (const uint16_t*)V, n_tokens, m->n_heads, (hipStream_t)stream),
         "stage launch");
  return RV_OK;
}

rv_status rv_mem_stage_frames(int n_layers, const rv_mem* mems, const void* const* K, const void* const* V,
                              int n_tokens, void* stream) {
  if (n_layers < 1) return fail(RV_ERR_INVALID, "n_layers must be >= 1");
  if (!mems || !K || !V) return fail(RV_ERR_INVALID, "mems, K and V are required");
  for (int l = 0; l < n_layers; ++l) {
    if (!mems[l] || !K[l] || !V[l]) return fail(RV_ERR_INVALID, "layer %d: memory, K and V are required", l);
    if (mems[l]->n_heads != mems[0]->n_heads) return fail(RV_ERR_INVALID, "layer %d: head count differs", l);
  }
  // Room for every layer first, so that a failure enqueues nothing.
  for (int l = 0; l < n_layers; ++l) {
    rv_status st = rv_mem_stage(mems[l], n_tokens, nullptr, nullptr, nullptr, stream);
    if (st != RV_OK) return st;
  }
  for (int l0 = 0; l0 < n_layers; l0 += rv::kMaxLayersPerLaunch) {
    rv::StageArgs a{};
    a.n_tokens = n_tokens;
    a.n_heads = mems[0]->n_heads;
    a.n_layers = std::min(rv::kMaxLayersPerLaunch, n_layers - l0);
    for (int i = 0; i < a.n_layers; ++i) {
      const rv_mem m = mems[l0 + i];
      a.layer[i] = rv::StageLayer{m->K + m->len * rv::kHeadDim, m->V + m->len * rv::kHeadDim,
                                  (const uint16_t*)K[l0 + i], (const uint16_t*)V[l0 + i], m->cap};
    }
    RV_HIP(rv::launch_stage_layers(a, (hipStream_t)stream), "stage launch");
  }
  return RV_OK;
}

rv_status rv_attend_staged(const void* Q, int n_tokens, rv_mem m, const rv_qsub* qs, void* out, float* lse,
                           float* saliency, void* stream) {
  if (!m) return fail(RV_ERR_INVALID, "memory is NULL");
  if (n_tokens < 1 || n_tokens > rv::kMaxTokens)
    return fail(RV_ERR_INVALID, "n_tokens must be in [1, %d] (got %d)", rv::kMaxTokens, n_tokens);
  if (!Q || !out || !lse) return fail(RV_ERR_INVALID, "Q, out and lse are required");
  rv_status st = check_device(m);
  if (st != RV_OK) return st;
  if (m->cap < m->len + n_tokens)
    return fail(RV_ERR_INVALID, "no staged frame: capacity %lld < length %lld + n_tokens %d (call rv_mem_stage)",
                (long long)m->cap, (long long)m->len, n_tokens);
  if (saliency) {
    st = check_qsub(qs, n_tokens);
    if (st != RV_OK) return st;
  }
  const uint16_t* kt = m->K + m->len * rv::kHeadDim;
  const uint16_t* vt = m->V + m->len * rv::kHeadDim;
  return attend_impl(Q, kt, vt, n_tokens, 0, m->K, m->V, m->len + n_tokens, m->cap, m->n_heads, qs, out, lse,
                     saliency, kt, rv::kHeadDim, m->cap * rv::kHeadDim, (hipStream_t)stream);
}

rv_status rv_admit(const float* saliency, int budget, const void* K, const void* V, int n_tokens, rv_mem m,
                   int frame_id, int32_t* idx_out, void* stream) {
  if (!m) return fail(RV_ERR_INVALID, "memory is NULL");
  if (n_tokens < 1 || n_tokens > rv::kMaxTokens)
    return fail(RV_ERR_INVALID, "n_tokens must be in [1, %d] (got %d)", rv::kMaxTokens, n_tokens);
  if (budget < 0 || budget > n_tokens)
    return fail(RV_ERR_INVALID, "budget must be in [0, n_tokens] (got %d)", budget);
  if (budget > 0 && (!saliency || !K || !V)) return fail(RV_ERR_INVALID, "saliency, K and V are required");
  rv_status st = check_device(m);
  if (st != RV_OK) return st;
  if (budget == 0) return RV_OK;
  hipStream_t s = (hipStream_t)stream;
  std::lock_guard<std::mutex> lk(g_ws_mu);
  Workspace* ws;
  st = ready_ws(&ws);
  if (st != RV_OK) return st;
  st = arena_reserve(m, m->len + budget, s);
  if (st != RV_OK) return st;

  rv::AdmitArgs b{};
  b.layer[0].K = (const uint16_t*)K;
  b.layer[0].V = (const uint16_t*)V;
  b.layer[0].kv_row = (int64_t)m->n_heads * rv::kHeadDim;
  b.layer[0].kv_head = rv::kHeadDim;
  b.layer[0].sal = const_cast<float*>(saliency);
  b.layer[0].idx = idx_out;
  b.layer[0].memK = m->K;
  b.layer[0].memV = m->V;
  b.layer[0].prov = m->prov;
  b.layer[0].mem_len = m->len;
  b.layer[0].head_stride = m->cap;
  b.n_tokens = n_tokens;
  b.n_heads = m->n_heads;
  b.n_layers = 1;
  b.budget = budget;
  b.frame_id = frame_id;
  b.mode = rv::kModeSelect;
  if (rv::admit_lds_bytes(b) > (size_t)rv::admit_max_dynamic_lds(ws->max_lds))
    return fail(RV_ERR_INVALID, "frame too large for the selection workgroup's LDS");
  RV_HIP(rv::launch_admit(b, ws->max_lds, s), "admit launch");
  m->len += budget;
  return RV_OK;
}

}  // extern "C"

namespace {

// staged: the frame's K, V are the rows each memory staged past its length (K, V
// unused); the selected rows are compacted in place.
// tiles: per-block saliency rows from rv_attend_frame_fused (then Q, lse and qs are unused).
rv_status admit_layers(int n_layers, const void* const* Q, const void* const* K, const void* const* V,
                       const float* const* lse, int n_tokens, const rv_qsub* qs, int budget, const rv_mem* mems,
                       int frame_id, float* const* saliency_out, int32_t* const* idx_out, void* stream,
                       bool shared, bool staged, const float* const* tiles = nullptr) {
  if (n_layers < 1 || n_layers > 4096) return fail(RV_ERR_INVALID, "n_layers must be in [1, 4096]");
  if ((!tiles && (!Q || !lse)) || (!staged && (!K || !V)) || !mems)
    return fail(RV_ERR_INVALID, "NULL pointer array");
  if (n_tokens < 1 || n_tokens > rv::kMaxTokens)
    return fail(RV_ERR_INVALID, "n_tokens must be in [1, %d] (got %d)", rv::kMaxTokens, n_tokens);
  if (budget < 0 || budget > n_tokens)
    return fail(RV_ERR_INVALID, "budget must be in [0, n_tokens] (got %d)", budget);
  rv_status st = tiles ? RV_OK : check_qsub(qs, n_tokens);
  if (st != RV_OK) return st;
  const int H = mems[0] ? mems[0]->n_heads : 0;
  for (int l = 0; l < n_layers; ++l) {
    if ((tiles ? !tiles[l] : (!Q[l] || !lse[l])) || (!staged && (!K[l] || !V[l])) || !mems[l])
      return fail(RV_ERR_INVALID, "layer %d: NULL tensor or memory", l);
    if (mems[l]->n_heads != H) return fail(RV_ERR_INVALID, "layer %d: head count differs", l);
    st = check_device(mems[l]);
    if (st != RV_OK) return st;
    if (mems[l]->len + budget > mems[l]->max_tokens)
      return fail(RV_ERR_CAPACITY, "layer %d: memory would exceed max_tokens", l);
    if (staged && mems[l]->cap < mems[l]->len + n_tokens)
      return fail(RV_ERR_INVALID, "layer %d: no staged frame (call rv_mem_stage)", l);
  }
  hipStream_t s = (hipStream_t)stream;
  std::lock_guard<std::mutex> lk(g_ws_mu);
  Workspace* ws;
  st = ready_ws(&ws);
  if (st != RV_OK) return st;
  rv::AdmitArgs probe{};
  probe.n_tokens = n_tokens;
  probe.budget = budget;
  probe.n_heads = H;
  probe.shared_select = shared ? 1 : 0;
  if (tiles) {
    probe.mode = rv::kModeSelect;
    probe.sal_tiles = (n_tokens + rv::kAttnBQ - 1) / rv::kAttnBQ;
  } else {
    rv::set_qsub(&probe, *qs);
    probe.mode = rv::kModeBoth;
    probe.sal_xcds = ws->n_queues;
    rv::plan_saliency(&probe, std::min(n_layers, rv::kMaxLayersPerLaunch) * H, ws->n_cus, ws->max_lds);
  }
  const size_t lds_cap = (size_t)rv::admit_max_dynamic_lds(ws->max_lds);
  if (rv::admit_lds_bytes(probe) > lds_cap)
    return fail(RV_ERR_INVALID, "frame too large for the admission workgroup's LDS");
  const int chunk_layers = std::min(n_layers, rv::kMaxLayersPerLaunch);
  bool need_ws_sal = !tiles && !saliency_out;
  for (int l = 0; !tiles && saliency_out && l < n_layers; ++l) need_ws_sal |= !saliency_out[l];
  if (need_ws_sal && ws->sal_floats < (size_t)chunk_layers * H * n_tokens)
    return fail(RV_ERR_CAPACITY,
                "no saliency output given and the saliency workspace holds %zu values, %zu needed "
                "(call rv_reserve_workspace with n_layers >= %d)",
                ws->sal_floats, (size_t)chunk_layers * H * n_tokens, chunk_layers);
  // growth for every layer before anything is enqueued (a staged memory has its room)
  for (int l = 0; !staged && l < n_layers; ++l) {
    st = arena_reserve(mems[l], mems[l]->len + budget, s);
    if (st != RV_OK) return st;
  }

  for (int l0 = 0; l0 < n_layers; l0 += rv::kMaxLayersPerLaunch) {
    const int nl = std::min(rv::kMaxLayersPerLaunch, n_layers - l0);
    rv::AdmitArgs b = probe;
    for (int i = 0; i < nl; ++i) {
      const int l = l0 + i;
      rv::AdmitLayer& L = b.layer[i];
      L.Q = tiles ? nullptr : (const uint16_t*)Q[l];
      if (staged) {
        L.K = mems[l]->K + mems[l]->len * rv::kHeadDim;
        L.V = mems[l]->V + mems[l]->len * rv::kHeadDim;
        L.kv_row = rv::kHeadDim;
        L.kv_head = mems[l]->cap * rv::kHeadDim;
      } else {
        L.K = (const uint16_t*)K[l];
        L.V = (const uint16_t*)V[l];
        L.kv_row = (int64_t)H * rv::kHeadDim;
        L.kv_head = rv::kHeadDim;
      }
      if (tiles) {
        L.sal = const_cast<float*>(tiles[l]);
        L.sal_out = saliency_out ? saliency_out[l] : nullptr;
      } else {
        L.lse = lse[l];
        L.sal = (saliency_out && saliency_out[l]) ? saliency_out[l] : ws->sal + (size_t)i * H * n_tokens;
      }
      L.idx = idx_out ? idx_out[l] : nullptr;
      L.memK = mems[l]->K;
      L.memV = mems[l]->V;
      L.prov = mems[l]->prov;
      L.mem_len = mems[l]->len;
      L.head_stride = mems[l]->cap;
    }
    b.n_heads = H;
    b.n_layers = nl;
    b.frame_id = frame_id;
    b.in_place = staged ? 1 : 0;
    RV_HIP(rv::launch_admit(b, ws->max_lds, s), "admit_layers launch");
  }
  for (int l = 0; l < n_layers; ++l) mems[l]->len += budget;
  return RV_OK;
}

}  // namespace

extern "C" {

rv_status rv_admit_layers(int n_layers, const void* const* Q, const void* const* K, const void* const* V,
                          const float* const* lse, int n_tokens, const rv_qsub* qs, int budget,
                          const rv_mem* mems, int frame_id, float* const* saliency_out,
                          int32_t* const* idx_out, void* stream) {
  return admit_layers(n_layers, Q, K, V, lse, n_tokens, qs, budget, mems, frame_id, saliency_out, idx_out,
                      stream, false, false);
}

rv_status rv_admit_layers_shared(int n_layers, const void* const* Q, const void* const* K, const void* const* V,
                                 const float* const* lse, int n_tokens, const rv_qsub* qs, int budget,
                                 const rv_mem* mems, int frame_id, float* const* saliency_out,
                                 int32_t* const* idx_out, void* stream) {
  return admit_layers(n_layers, Q, K, V, lse, n_tokens, qs, budget, mems, frame_id, saliency_out, idx_out,
                      stream, true, false);
}

rv_status rv_admit_layers_tiled(int n_layers, const float* const* sal_tiles, int n_tokens, int budget,
                                const void* const* K, const void* const* V, const rv_mem* mems, int frame_id,
                                float* const* saliency_out, int32_t* const* idx_out, void* stream) {
  if (!sal_tiles) return fail(RV_ERR_INVALID, "sal_tiles is NULL");
  return admit_layers(n_layers, nullptr, K, V, nullptr, n_tokens, nullptr, budget, mems, frame_id, saliency_out,
                      idx_out, stream, false, false, sal_tiles);
}

rv_status rv_admit_staged_layers(int n_layers, const void* const* Q, const float* const* lse, int n_tokens,
                                 const rv_qsub* qs, int budget, const rv_mem* mems, int frame_id,
                                 float* const* saliency_out, int32_t* const* idx_out, void* stream) {
  return admit_layers(n_layers, Q, nullptr, nullptr, lse, n_tokens, qs, budget, mems, frame_id, saliency_out,
                      idx_out, stream, false, true);
}

}  // extern "C"
