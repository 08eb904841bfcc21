// rv_plan.cpp -- librv's host-side work planning: the attention launch's chunking, the
// admission launch's shape and LDS needs, and the query-subset descriptor.  No device
// calls here, so this file also builds with a host compiler alone.
#include "rv_plan.h"

#include <algorithm>
#include <cstdlib>

namespace rv {
namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int env_int(const char* name, int dflt) {
  const char* v = std::getenv(name);
  if (!v || !*v) return dflt;
  return std::atoi(v);
}

int wg_per_queue(int n_cus, int n_queues) {
  return std::max(1, env_int("RV_ATTN_WG_PER_CU", kAttnWgPerCu) * n_cus / n_queues);
}

}  // namespace

// k-way split: each unit's key range is cut into k aligned pieces (iteration stride
// U = k E per unit), so the workgroups on one head's query tiles stream the same key
// tiles together.  Stream-K: U = T, chunks may straddle units.  RV_ATTN_SPLIT forces one
// (0: stream-K, k > 0: k-way).
AttnPlan plan_attention(int n_cus, int n_queues, int n_tokens, int n_fkeys, int64_t mem_len, int n_heads) {
  AttnPlan p{};
  p.q_tiles = (int)ceil_div(n_tokens, kAttnBQ);
  p.nt_mem = (int)ceil_div(mem_len, kAttnBK);
  p.T = p.nt_mem + (int)ceil_div(n_fkeys, kAttnBK);
  p.n_units = p.q_tiles * n_heads;
  const int nq = n_queues;
  const int wgq = wg_per_queue(n_cus, nq);
  int max_units = 0;
  for (int q = 0; q <= nq; ++q) p.unit_base[q] = (int)((int64_t)q * p.n_units / nq);
  for (int q = 0; q < nq; ++q) max_units = std::max(max_units, p.unit_base[q + 1] - p.unit_base[q]);
  const int e_min = std::max(1, env_int("RV_ATTN_MIN_CHUNK", 2));
  // Stream-K balances the tiles exactly but pays, per chunk that straddles two units, a
  // second pipeline start; the aligned split leaves some workgroup slots idle.  Take the
  // split while its chunks are at most kSplitSlackTiles longer than stream-K's.
  constexpr int kSplitSlackTiles = 1;
  // Tiles of a first-dispatched stream-K chunk, in per cent of a later chunk's.
  constexpr int kFirstChunkPct = 140;
  int k = env_int("RV_ATTN_SPLIT", -1);
  if (k < 0) {
    k = wgq / std::max(1, max_units);
    const int64_t e_sk = ceil_div((int64_t)max_units * p.T, wgq);
    if (k >= 1 && ceil_div(p.T, k) > e_sk + env_int("RV_ATTN_SPLIT_SLACK", kSplitSlackTiles)) k = 0;
  }
  p.n_first = 0;
  if (k >= 1) {
    const int e = (int)std::min<int64_t>((int64_t)1 << 22, std::max<int64_t>(e_min, ceil_div(p.T, k)));
    k = (int)ceil_div(p.T, e);  // pieces that hold tiles
    p.U = k * e;
    p.E = p.E1 = e * kCutScale;
  } else {
    // Stream-K.  Workgroup ids are dealt round-robin over the XCDs and then over the
    // CUs, so a queue's first n_cus / nq chunks go to the workgroups dispatched first
    // on their CUs, which run measurably faster than the second ones: those chunks get
    // kFirstChunkPct per cent of the later chunks' tiles (a speed heuristic only; any
    // placement gives the same results).
    p.U = p.T;
    const int64_t work = (int64_t)max_units * p.T;
    const int pct_env = env_int("RV_ATTN_FIRST_PCT", 0);
    const int pct = std::max(100, pct_env > 0 ? pct_env : kFirstChunkPct);
    // (no second workgroup per CU to favour the first over: uniform chunks)
    const int n_first = n_cus / nq < wgq ? std::max(0, n_cus / nq) : 0;
    const int n_rest = wgq - n_first;
    // (lengths are kept below 2^30 scaled positions: a chunk that long only arises with a
    // handful of workgroup slots, and more, shorter chunks are then used instead)
    const int64_t e_lo = (int64_t)e_min * kCutScale, e_hi = (int64_t)1 << 30;
    // Unit-aligned form: later chunks of exactly T/k tiles (k dividing n_rest) cover the
    // queue's last n_rest/k units k to a unit, and the first chunks share the units before
    // them equally, so that every unit boundary is a chunk boundary and no later chunk
    // starts a second segment.  Taken (unless RV_ATTN_FIRST_PCT sets the share) when the
    // first chunks then hold kAlignMinPct..kAlignMaxPct per cent of a later one's tiles,
    // the share closest to kFirstChunkPct if several k qualify.
    constexpr int kAlignMinPct = 115, kAlignMaxPct = 160;
    bool aligned = false;
    if (pct_env <= 0 && n_first > 0) {
      int64_t best_e = 0, best_e1 = 0, best_dist = -1;
      for (int k = 1; k <= n_rest; ++k) {
        const int64_t rest_units = n_rest / k;
        if (n_rest % k != 0 || rest_units >= max_units || ((int64_t)p.T * kCutScale) % k != 0) continue;
        const int64_t first_work = (int64_t)(max_units - rest_units) * p.T * kCutScale;
        if (first_work % n_first != 0) continue;
        const int64_t e1 = (int64_t)p.T * kCutScale / k, e = first_work / n_first;
        if (e * 100 < e1 * kAlignMinPct || e * 100 > e1 * kAlignMaxPct || e1 < e_lo || e > e_hi) continue;
        const int64_t dist = std::abs(e * 100 - e1 * kFirstChunkPct) * 1000 / e1;  // (in 1/1000 per cent)
        if (best_dist < 0 || dist < best_dist) {
          best_dist = dist;
          best_e = e;
          best_e1 = e1;
        }
      }
      if (best_dist >= 0) {
        p.E = (int)best_e;
        p.E1 = (int)best_e1;
        p.n_first = n_first;
        aligned = true;
      }
    }
    if (!aligned) {
      const int64_t e1 =
          std::max<int64_t>(e_lo, ceil_div(work * kCutScale * 100, (int64_t)n_first * pct + (int64_t)n_rest * 100));
      p.E1 = (int)std::min(e_hi, e1);
      p.E = (int)std::min(e_hi, std::max<int64_t>(e_lo, ceil_div((int64_t)p.E1 * pct, 100)));
      p.n_first = p.E == p.E1 ? 0 : n_first;
      if (p.n_first == 0) p.E = p.E1;  // (no first workgroups to favour)
    }
  }
  p.total_chunks = 0;
  int max_chunks = 0;
  for (int q = 0; q < nq; ++q) {
    const int64_t iters = (int64_t)(p.unit_base[q + 1] - p.unit_base[q]) * p.U * kCutScale;  // scaled
    const int64_t first = (int64_t)p.n_first * p.E;
    p.n_chunks[q] = iters <= first ? (int)ceil_div(iters, p.E) : p.n_first + (int)ceil_div(iters - first, p.E1);
    p.chunk_base[q] = p.total_chunks;
    p.total_chunks += p.n_chunks[q];
    max_chunks = std::max(max_chunks, p.n_chunks[q]);
  }
  if (max_chunks <= p.n_first) {  // every chunk is a first one: say so plainly
    p.n_first = 0;
    p.E1 = p.E;
  }
  p.grid = nq * max_chunks;
  return p;
}

bool plan_splits_units(const AttnPlan& p) {  // unless every chunk is exactly one unit
  return !(p.E1 == p.E && p.U == p.T && (int64_t)p.E == (int64_t)p.U * kCutScale);
}

// Without a forced split, a queue's chunk count is set by its workgroup slots: the
// k-way split cuts its units into at most wg_per_queue pieces in all, and stream-K sizes
// its chunks so that n_first of E tiles and the rest of E1 tiles cover the queue's work
// within wg_per_queue chunks (E >= E1 * pct / 100, E1 >= work / (n_first * pct / 100 +
// n_rest)).  One chunk per queue of slack covers the rounding.
int64_t default_partial_slots(int n_cus, int n_queues) {
  return 2 * (int64_t)n_queues * (wg_per_queue(n_cus, n_queues) + 1);
}

const char* qsub_problem(const rv_qsub* qs, int n_tokens) {
  if (!qs) return "query subset descriptor is NULL";
  if (qs->grid_h < 0 || qs->grid_w < 0 || qs->n_special < 0 || qs->stride < 1)
    return "query subset has negative sizes or stride < 1";
  if ((int64_t)qs->grid_h * qs->grid_w + qs->n_special != n_tokens)
    return "query subset does not describe the frame's tokens (grid_h * grid_w + n_special != n_tokens)";
  return nullptr;
}

void set_qsub(AdmitArgs* b, const rv_qsub& q) {
  const int rows = (q.grid_h + q.stride - 1) / q.stride;
  const int cols = (q.grid_w + q.stride - 1) / q.stride;
  b->n_q = rows * cols;
  b->q_cols = cols > 0 ? cols : 1;
  b->q_base = q.n_special;
  b->q_row_stride = q.stride * q.grid_w;
  b->q_col_stride = q.stride;
}

size_t sal_lds_bytes(const AdmitArgs& a) {
  const size_t nq_pad = (size_t)((a.n_q + 31) & ~31);
  return nq_pad * 4 + (a.stage_queries ? (size_t)a.q_pass * kSalQStride * 2 : 0);
}

size_t select_lds_bytes(const AdmitArgs& a) {
  return (((size_t)a.n_tokens * 4 + 15) & ~(size_t)15) + (size_t)a.budget * 4;
}

size_t admit_lds_bytes(const AdmitArgs& a) {
  size_t need = 0;
  if (a.mode & kModeSaliency) need = sal_lds_bytes(a);
  if ((a.mode & kModeSelect) && select_lds_bytes(a) > need) need = select_lds_bytes(a);
  return need;
}

int admit_max_dynamic_lds(int max_lds) { return max_lds - kAdmitStaticLdsMargin; }

void plan_saliency(AdmitArgs* a, int n_lh, int n_cus, int max_lds) {
  // About three 4-wave workgroups per CU over the launch, and at least one 32-key
  // block per wave.
  constexpr int kWaves = kAdmitThreads / 64;
  const int n_blocks = (a->n_tokens + 31) / 32;
  const int max_groups = n_blocks / kWaves > 1 ? n_blocks / kWaves : 1;
  int g = (3 * n_cus + n_lh - 1) / (n_lh > 0 ? n_lh : 1);
  a->sal_groups = g < 1 ? 1 : (g > max_groups ? max_groups : g);
  // Sampled query rows are staged in passes of q_pass rows, sized so that three
  // workgroups fit a CU's LDS; the pass size depends only on n_q and the device, so
  // every launch of the same frame shape sums in the same order.  An empty subset has
  // nothing to stage (every saliency is the empty sum).
  const int nq_pad = (a->n_q + 31) & ~31;
  const long budget_lds = (long)max_lds / 3 - kAdmitStaticLdsMargin - (long)nq_pad * 4;
  const int fit = budget_lds > 0 ? (int)(budget_lds / (kSalQStride * 2)) & ~31 : 0;
  if (nq_pad > 0 && fit >= 32) {
    const int passes = (nq_pad + fit - 1) / fit;
    a->q_pass = ((nq_pad + passes - 1) / passes + 31) & ~31;
    a->stage_queries = 1;
  } else {
    a->q_pass = nq_pad;
    a->stage_queries = 0;
  }
  if (sal_lds_bytes(*a) > (size_t)admit_max_dynamic_lds(max_lds)) a->stage_queries = 0;
}

}  // namespace rv
