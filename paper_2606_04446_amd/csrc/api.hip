// C ABI of libd2sd: host-side validation, planning and kernel dispatch.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <string>
#include <vector>

#include "launchers.h"

namespace {

thread_local std::string g_last_error;

d2sd_status fail(d2sd_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

d2sd_status ok() {
  g_last_error.clear();
  return D2SD_OK;
}

d2sd_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(D2SD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// ---- kernel timing (HIP events around the context-streaming kernel) ----
std::mutex g_timing_mu;
bool g_timing_on = false;
struct TimedLaunch {
  hipEvent_t e0, e1, e2;  // before the main kernel, after it, after the split merge
  bool merged;            // e2 was recorded (the call launched a split merge)
};
std::vector<TimedLaunch> g_timing_pending;
std::vector<hipEvent_t> g_event_pool;

hipEvent_t take_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Reserve three events when timing is on (all null otherwise).
void timing_begin(hipEvent_t (&ev)[3]) {
  ev[0] = ev[1] = ev[2] = nullptr;
  std::lock_guard<std::mutex> lk(g_timing_mu);
  if (!g_timing_on) return;
  for (auto& e : ev) e = take_event();
  if (!ev[0] || !ev[1] || !ev[2]) {
    for (auto& e : ev) {
      if (e) g_event_pool.push_back(e);
      e = nullptr;
    }
  }
}

// Record a timed call after its launches (merged: ev[2] was recorded), or
// return the events to the pool when the launch failed.
void timing_end(hipEvent_t (&ev)[3], bool launched, bool merged) {
  if (!ev[0]) return;
  std::lock_guard<std::mutex> lk(g_timing_mu);
  if (launched)
    g_timing_pending.push_back({ev[0], ev[1], ev[2], merged});
  else
    for (auto& e : ev) g_event_pool.push_back(e);
}

// Wait for every recorded call and return, in call order, the main kernel's
// duration and the split merge's (ms; 0 when the call had no merge);
// recycle the events and clear the record.
hipError_t collect_timings(std::vector<float>* kernel, std::vector<float>* merge) {
  std::vector<TimedLaunch> pend;
  {
    std::lock_guard<std::mutex> lk(g_timing_mu);
    pend.swap(g_timing_pending);
  }
  hipError_t err = hipSuccess;
  kernel->reserve(pend.size());
  merge->reserve(pend.size());
  for (auto& t : pend) {
    float k_ms = 0.0f, m_ms = 0.0f;
    hipError_t e = hipEventSynchronize(t.merged ? t.e2 : t.e1);
    if (e == hipSuccess) e = hipEventElapsedTime(&k_ms, t.e0, t.e1);
    if (e == hipSuccess && t.merged) e = hipEventElapsedTime(&m_ms, t.e1, t.e2);
    if (e != hipSuccess && err == hipSuccess) err = e;
    kernel->push_back(k_ms);
    merge->push_back(m_ms);
  }
  std::lock_guard<std::mutex> lk(g_timing_mu);
  for (auto& t : pend) {
    g_event_pool.push_back(t.e0);
    g_event_pool.push_back(t.e1);
    g_event_pool.push_back(t.e2);
  }
  return err;
}

// Largest tree any entry point accepts: the canonical tree of B = D2SD_MAX_B
// with every re-anchor position (the accept kernel stages one tree in LDS).
constexpr int kMaxTreeNodes = D2SD_MAX_B + D2SD_MAX_B * (D2SD_MAX_B - 1) / 2;

int mask_words_for(int B) {
  if (B < 2 || B > D2SD_MAX_B) return 0;
  return (B + B * (B - 1) / 2 + 31) / 32;
}

// ---- verify-attention planning ----

constexpr int kNumCUs = 256;
constexpr int kMinSplit = 256;      // bf16: shorter splits cost more in partial states than they gain
constexpr int kMinSplitF32 = 64;    // fp32: a split is compute-bound (fp32 MFMA), parallelism pays
constexpr int kMaxSplit = 32768;   // the bf16 kernel stages a split's page ids in LDS

d2sd_status validate_attn(const d2sd_attn_args* a, bool need_ws_fields) {
  if (!a) return fail(D2SD_ERR_INVALID_ARG, "args is NULL");
  if (a->batch < 1) return fail(D2SD_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", a->batch);
  if (a->num_qo_heads < 1 || a->num_kv_heads < 1)
    return fail(D2SD_ERR_INVALID_ARG, "head counts must be >= 1");
  if (a->num_qo_heads % a->num_kv_heads)
    return fail(D2SD_ERR_INVALID_ARG, "num_qo_heads %d is not a multiple of num_kv_heads %d",
                a->num_qo_heads, a->num_kv_heads);
  if (a->head_dim != D2SD_HEAD_DIM)
    return fail(D2SD_ERR_UNSUPPORTED, "head_dim %d unsupported (only %d)", a->head_dim, D2SD_HEAD_DIM);
  if (a->page_size != D2SD_PAGE_SIZE)
    return fail(D2SD_ERR_UNSUPPORTED, "page_size %d unsupported (only %d)", a->page_size, D2SD_PAGE_SIZE);
  if (a->dtype != D2SD_F32 && a->dtype != D2SD_BF16)
    return fail(D2SD_ERR_INVALID_ARG, "dtype %d is not D2SD_F32 or D2SD_BF16", a->dtype);
  if (a->stage < D2SD_STAGE_CASCADE || a->stage > D2SD_STAGE_TREE)
    return fail(D2SD_ERR_INVALID_ARG, "stage %d unknown", a->stage);
  if (a->total_nodes < 0 || a->max_nodes < 0 || a->max_nodes > a->total_nodes)
    return fail(D2SD_ERR_INVALID_ARG, "need 0 <= max_nodes <= total_nodes (got %d, %d)", a->max_nodes,
                a->total_nodes);
  if (a->total_nodes > 0 && a->max_nodes < 1)
    return fail(D2SD_ERR_INVALID_ARG, "max_nodes must be >= 1 when total_nodes > 0");
  if ((long long)a->total_nodes * a->num_qo_heads > (1ll << 30))
    return fail(D2SD_ERR_UNSUPPORTED, "total_nodes * num_qo_heads exceeds 2^30 rows");
  if (a->max_pages < 1 || a->num_pages < 1)
    return fail(D2SD_ERR_INVALID_ARG, "max_pages and num_pages must be >= 1");
  if ((long long)a->num_pages * a->num_kv_heads > 0x7fffffffll)
    return fail(D2SD_ERR_UNSUPPORTED, "num_pages x num_kv_heads = %lld exceeds 2^31 - 1",
                (long long)a->num_pages * a->num_kv_heads);
  if (a->max_ctx_len < 0 || (long long)a->max_ctx_len > (long long)a->max_pages * a->page_size)
    return fail(D2SD_ERR_INVALID_ARG, "max_ctx_len %d outside [0, max_pages*page_size = %lld]",
                a->max_ctx_len, (long long)a->max_pages * a->page_size);
  if (a->kv_split < 0 || a->kv_split % 64 || a->kv_split > kMaxSplit)
    return fail(D2SD_ERR_INVALID_ARG, "kv_split %d must be 0 or a multiple of 64 in [64, %d]", a->kv_split,
                kMaxSplit);
  if (a->packed < 0 || a->packed > 2) return fail(D2SD_ERR_INVALID_ARG, "packed %d must be 0, 1 or 2", a->packed);
  if (a->row_group != 0 && a->row_group != d2sd::kBf16Waves * d2sd::kRowsPerTile &&
      a->row_group != d2sd::kBf16WideWaves * d2sd::kRowsPerTile)
    return fail(D2SD_ERR_INVALID_ARG, "row_group %d must be 0, %d or %d", a->row_group,
                d2sd::kBf16Waves * d2sd::kRowsPerTile, d2sd::kBf16WideWaves * d2sd::kRowsPerTile);
  if (a->stage != D2SD_STAGE_PREFIX && a->mask_words < (a->max_nodes + 31) / 32)
    return fail(D2SD_ERR_INVALID_ARG, "mask_words %d too small for max_nodes %d", a->mask_words,
                a->max_nodes);
  if (a->node_indptr_host) {
    const int* ip = a->node_indptr_host;
    if (ip[0] != 0 || ip[a->batch] != a->total_nodes)
      return fail(D2SD_ERR_INVALID_ARG, "node_indptr_host must start at 0 and end at total_nodes %d (got %d, %d)",
                  a->total_nodes, ip[0], ip[a->batch]);
    for (int b = 0; b < a->batch; ++b)
      if (ip[b + 1] < ip[b] || ip[b + 1] - ip[b] > a->max_nodes)
        return fail(D2SD_ERR_INVALID_ARG, "node_indptr_host: request %d has %d nodes, outside [0, max_nodes %d]",
                    b, ip[b + 1] - ip[b], a->max_nodes);
  }
  if (!need_ws_fields) return D2SD_OK;
  if (!a->q || !a->k_cache || !a->v_cache || !a->page_table || !a->ctx_len || !a->k_tree ||
      !a->v_tree || !a->node_indptr || !a->out)
    return fail(D2SD_ERR_INVALID_ARG, "a required device pointer is NULL");
  if (a->stage != D2SD_STAGE_PREFIX && !a->anc_mask)
    return fail(D2SD_ERR_INVALID_ARG, "anc_mask is NULL");
  // the kernels move Q, K/V and the output in 16-byte chunks
  const void* const chunked[] = {a->q, a->k_cache, a->v_cache, a->k_tree, a->v_tree, a->out};
  const char* const names[] = {"q", "k_cache", "v_cache", "k_tree", "v_tree", "out"};
  for (int i = 0; i < 6; ++i)
    if (reinterpret_cast<uintptr_t>(chunked[i]) % 16 != 0)
      return fail(D2SD_ERR_INVALID_ARG, "%s is not 16-byte aligned", names[i]);
  return D2SD_OK;
}

// Row groups (work items) of one context split over the batch, for groups of
// rows_per_group query rows: exact when the host copy of the node offsets is
// given, else from the mean tree size.
long long groups_per_split(const d2sd_attn_args* a, int G, int rows_per_group) {
  long long groups = 0;
  if (a->node_indptr_host) {
    for (int b = 0; b < a->batch; ++b) {
      const long long rows = (long long)(a->node_indptr_host[b + 1] - a->node_indptr_host[b]) * G;
      groups += (rows + rows_per_group - 1) / rows_per_group;
    }
  } else {
    const double avg_rows = (double)a->total_nodes / a->batch * G;
    groups = (long long)a->batch * max(1, (int)ceil(avg_rows / rows_per_group));
  }
  return max(1ll, groups * a->num_kv_heads);
}

// Relative kernel time of g row groups per split at s splits with R resident
// workgroups: work items of equal length (1/s of a context) run in
// ceil(g s / R) rounds of resident workgroups.
double rounds_time(long long g, long long R, int s) { return (double)((g * s + R - 1) / R) / s; }

// The split count in [s_lo, s_hi] minimising rounds_time, a larger count only
// for a gain of at least 3% (every split adds a partial state that the merge
// reads back).
int best_splits(long long g, long long R, int s_lo, int s_hi, double* t) {
  int best_s = s_lo;
  double best = rounds_time(g, R, s_lo);
  for (int s = s_lo + 1; s <= min(s_hi, 4 * s_lo); ++s) {
    const double ts = rounds_time(g, R, s);
    if (ts < 0.97 * best) {
      best = ts;
      best_s = s;
    }
  }
  *t = best;
  return best_s;
}

// Measured speed of the twelve-wave bf16 shape against the four-wave one for
// the same filled waves (one context read per 384 rows instead of per 128):
// 8% on the 32-request, 16k-context workload.
constexpr double kWideGain = 1.08;

// Query tiles (32 rows) of one split over the batch and KV heads, for the
// packed shape; false when it does not apply (no host node offsets, a batch
// over kPackedMaxBatch, or a stream with fewer than kPackedMinTiles tiles).
bool packed_tiles(const d2sd_attn_args* a, int G, long long* tiles1) {
  if (a->dtype != D2SD_BF16 || !a->node_indptr_host || a->batch > d2sd::kPackedMaxBatch) return false;
  long long t = 0;
  for (int b = 0; b < a->batch; ++b) {
    const long long rows = (long long)(a->node_indptr_host[b + 1] - a->node_indptr_host[b]) * G;
    const long long tb = (rows + d2sd::kRowsPerTile - 1) / d2sd::kRowsPerTile;
    if (tb < d2sd::kPackedMinTiles) return false;
    t += tb;
  }
  *tiles1 = t * a->num_kv_heads;
  return true;
}

// Relative time of the packed shape at s splits: ceil(tiles s / 12)
// workgroups in rounds of one per CU, each 1/s of a context long.
double packed_time(long long tiles1, int s) {
  const long long wgs = (tiles1 * s + d2sd::kBf16WideWaves - 1) / d2sd::kBf16WideWaves;
  return rounds_time(wgs, kNumCUs, 1) / s;
}

struct Shape {
  int waves;
  bool packed;
  int splits;
};

// Packing streams costs extra reads of the streams it cuts and some control
// work per round; it has to beat the one-stream 12-wave shape by 3%.
constexpr double kPackMargin = 0.97;

// Workgroup shape and context tokens per split. R = resident workgroups:
// three 4-wave or one 12-wave bf16 workgroup per CU, one fp32 workgroup.
//  - Grids that fill the chip with one split (g s_lo >= R for 4-wave groups):
//    each shape takes its best split count (best_splits) and the shape with
//    the shorter time wins, the 12-wave shapes counted kWideGain faster; idle
//    waves of partly filled row groups show up as more row groups per split.
//    The packed 12-wave shape fills every wave (workgroups over the sequence
//    of all streams' tiles) and is counted by its tiles; it is taken only
//    when it beats the one-stream 12-wave shape by kPackMargin.
//  - Smaller grids take 4-wave groups and about two rounds of work items.
// No split is shorter than the dtype's minimum (the partial state of a split
// costs as many bytes as ~M/2 keys of K/V, M = rows sharing it; fp32 splits
// are compute-bound and can be shorter) or longer than the staged page list
// allows. An explicit kv_split, row_group or packed fixes that choice.
void choose_shape(const d2sd_attn_args* a, int G, d2sd::AttnPlan* plan) {
  const bool bf16 = a->dtype == D2SD_BF16;
  const int ctx = a->max_ctx_len;
  const int min_split = bf16 ? kMinSplit : kMinSplitF32;
  const int s_lo = max(1, (ctx + kMaxSplit - 1) / kMaxSplit);
  const int s_hi = max(s_lo, ctx / min_split);
  const int s_lo_p = max(s_lo, (ctx + d2sd::kPackedMaxSplit - 1) / d2sd::kPackedMaxSplit);
  const long long g4 = groups_per_split(a, G, d2sd::kBf16Waves * d2sd::kRowsPerTile);
  const long long R4 = (long long)kNumCUs * (bf16 ? 3 : 1);
  const long long g12 = groups_per_split(a, G, d2sd::kBf16WideWaves * d2sd::kRowsPerTile);
  const long long R12 = kNumCUs;
  const bool wide_ok = bf16 && a->row_group != d2sd::kBf16Waves * d2sd::kRowsPerTile;
  const bool wide_forced = bf16 && a->row_group == d2sd::kBf16WideWaves * d2sd::kRowsPerTile;
  long long tiles1 = 0;
  const bool pk_ok = wide_ok && a->packed != 1 && packed_tiles(a, G, &tiles1) && s_hi >= s_lo_p;
  Shape sh{d2sd::kBf16Waves, false, 1};
  if (a->kv_split > 0) {
    const int s = max(1, (ctx + a->kv_split - 1) / a->kv_split);
    sh.splits = s;
    const double t4 = rounds_time(g4, R4, s);
    const double t12 = rounds_time(g12, R12, s) / kWideGain;
    const bool pk_here = pk_ok && a->kv_split <= d2sd::kPackedMaxSplit;
    const double tp = pk_here ? packed_time(tiles1, s) / kWideGain : 1e30;
    const bool large = g4 * s >= R4;
    if (pk_here && (a->packed == 2 || ((wide_forced || large) && tp < kPackMargin * t12 && (wide_forced || tp < t4)))) {
      sh.waves = d2sd::kBf16WideWaves;
      sh.packed = true;
    } else if (wide_forced || (wide_ok && large && t12 < t4)) {
      sh.waves = d2sd::kBf16WideWaves;
    }
  } else if (g4 * s_lo >= R4 || wide_forced || (pk_ok && a->packed == 2)) {
    double t4 = 0.0, t12 = 0.0, tp = 1e30;
    const int s4 = best_splits(g4, R4, s_lo, s_hi, &t4);
    const int s12 = best_splits(g12, R12, s_lo, s_hi, &t12);
    t12 /= kWideGain;
    int sp = s_lo_p;
    if (pk_ok) {
      tp = packed_time(tiles1, s_lo_p);
      for (int s = s_lo_p + 1; s <= min(s_hi, 4 * s_lo_p); ++s) {
        const double ts = packed_time(tiles1, s);
        if (ts < 0.97 * tp) {
          tp = ts;
          sp = s;
        }
      }
      tp /= kWideGain;
    }
    if (pk_ok && (a->packed == 2 || (tp < kPackMargin * t12 && (wide_forced || tp < t4)))) {
      sh = Shape{d2sd::kBf16WideWaves, true, sp};
    } else if (wide_forced || (wide_ok && t12 < t4)) {
      sh = Shape{d2sd::kBf16WideWaves, false, s12};
    } else {
      sh = Shape{d2sd::kBf16Waves, false, s4};
    }
  } else if (ctx > min_split) {
    const int s = (int)((2 * R4 + g4 - 1) / g4);
    sh.splits = max(s_lo, min(s, s_hi));
  }
  plan->waves = sh.waves;
  plan->packed = sh.packed;
  plan->tiles = 0;   // the packed shape's tile count is set by make_plan from the resolved split count
  if (a->kv_split > 0) {
    plan->split = a->kv_split;
  } else if (ctx <= min_split) {
    plan->split = ((max(ctx, 1) + 63) / 64) * 64;
  } else {
    const int per = (ctx + sh.splits - 1) / sh.splits;
    plan->split = ((per + 63) / 64) * 64;
  }
}

d2sd_status make_plan(const d2sd_attn_args* a, d2sd::AttnPlan* plan) {
  plan->G = a->num_qo_heads / a->num_kv_heads;
  choose_shape(a, plan->G, plan);
  const bool ctx = a->stage != D2SD_STAGE_TREE;
  plan->n_ch_max = ctx ? max(1, (a->max_ctx_len + plan->split - 1) / plan->split) : 1;
  if (plan->packed) {
    long long tiles1 = 0;
    packed_tiles(a, plan->G, &tiles1);
    plan->tiles = tiles1 * plan->n_ch_max;
    if (plan->tiles > (1ll << 30)) return fail(D2SD_ERR_UNSUPPORTED, "too many query tiles (%lld)", plan->tiles);
  }
  const long long max_rows = (long long)a->max_nodes * plan->G;
  const int rows_per_group = plan->waves * d2sd::kRowsPerTile;
  plan->n_rg_max = (int)max(1ll, (max_rows + rows_per_group - 1) / rows_per_group);
  plan->items = (long long)a->batch * a->num_kv_heads * plan->n_ch_max * plan->n_rg_max;
  if (plan->items > (1ll << 30)) return fail(D2SD_ERR_UNSUPPORTED, "too many work items (%lld)", plan->items);
  if (plan->n_ch_max > 1 &&
      (long long)a->batch *
              d2sd::merge_chunks_per_request(a->max_nodes, a->num_qo_heads, d2sd::merge_groups(plan->n_ch_max)) >
          (1ll << 30))
    return fail(D2SD_ERR_UNSUPPORTED, "too many split-merge workgroups (batch %d, max_nodes %d)", a->batch,
                a->max_nodes);
  const size_t rows = (size_t)a->total_nodes * a->num_qo_heads;
  // per split and row: the normalised output in the input dtype, then m and l in fp32
  const size_t o_elem = a->dtype == D2SD_BF16 ? 2 : 4;
  plan->ws_bytes = plan->n_ch_max > 1 ? (size_t)plan->n_ch_max * rows * (a->head_dim * o_elem + 2 * sizeof(float)) : 0;
  plan->scale = a->sm_scale > 0.0f ? a->sm_scale : 1.0f / sqrtf((float)a->head_dim);
  return D2SD_OK;
}

}  // namespace

extern "C" {

const char* d2sd_status_string(d2sd_status s) {
  switch (s) {
    case D2SD_OK: return "ok";
    case D2SD_ERR_INVALID_ARG: return "invalid argument";
    case D2SD_ERR_UNSUPPORTED: return "unsupported";
    case D2SD_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case D2SD_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* d2sd_last_error(void) { return g_last_error.c_str(); }

int d2sd_version(void) { return 100; }

int d2sd_mask_words(int B) { return mask_words_for(B); }

d2sd_status d2sd_tree_plan(int batch, int B, const int* K_host, const int* p_host, int Kmax,
                           int* node_indptr_host, int* mask_words_out) {
  if (batch < 1) return fail(D2SD_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", batch);
  if (B < 2 || B > D2SD_MAX_B) return fail(D2SD_ERR_INVALID_ARG, "B = %d outside [2, %d]", B, D2SD_MAX_B);
  if (Kmax < 0) return fail(D2SD_ERR_INVALID_ARG, "Kmax must be >= 0");
  if (!K_host || !node_indptr_host || (Kmax > 0 && !p_host))
    return fail(D2SD_ERR_INVALID_ARG, "a required host pointer is NULL");
  std::vector<int> indptr(batch + 1, 0);
  for (int b = 0; b < batch; ++b) {
    const int K = K_host[b];
    if (K < 0 || K > Kmax || K > B - 1)
      return fail(D2SD_ERR_INVALID_ARG, "request %d: K = %d outside [0, min(Kmax=%d, B-1=%d)]", b, K, Kmax,
                  B - 1);
    unsigned long long seen = 0ull;
    long long n = B;
    for (int k = 0; k < K; ++k) {
      const int pk = p_host[(size_t)b * Kmax + k];
      if (pk < 1 || pk > B - 1)
        return fail(D2SD_ERR_INVALID_ARG, "request %d: re-anchor position %d outside [1, %d]", b, pk, B - 1);
      if ((seen >> pk) & 1ull)
        return fail(D2SD_ERR_INVALID_ARG, "request %d: re-anchor position %d repeated", b, pk);
      seen |= 1ull << pk;
      n += B - pk;
    }
    if ((long long)indptr[b] + n > (1ll << 30)) return fail(D2SD_ERR_INVALID_ARG, "too many tree nodes");
    indptr[b + 1] = indptr[b] + (int)n;
  }
  for (int b = 0; b <= batch; ++b) node_indptr_host[b] = indptr[b];
  if (mask_words_out) *mask_words_out = mask_words_for(B);
  return ok();
}

d2sd_status d2sd_tree_build(int batch, int B, int Kmax, const int* K, const int* p,
                            const int* node_indptr, int total_nodes, int mask_words, int* parent,
                            int* depth, int* path_id, uint32_t* anc_mask, int* path_leaf,
                            hipStream_t stream) {
  if (batch < 1) return fail(D2SD_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", batch);
  if (B < 2 || B > D2SD_MAX_B) return fail(D2SD_ERR_INVALID_ARG, "B = %d outside [2, %d]", B, D2SD_MAX_B);
  if (Kmax < 0) return fail(D2SD_ERR_INVALID_ARG, "Kmax must be >= 0");
  if (total_nodes < 0) return fail(D2SD_ERR_INVALID_ARG, "total_nodes must be >= 0");
  if (mask_words != mask_words_for(B))
    return fail(D2SD_ERR_INVALID_ARG, "mask_words %d != d2sd_mask_words(%d) = %d", mask_words, B,
                mask_words_for(B));
  if (!K || (Kmax > 0 && !p) || !node_indptr || !parent || !depth || !path_id || !anc_mask || !path_leaf)
    return fail(D2SD_ERR_INVALID_ARG, "a required device pointer is NULL");
  return hip_status(d2sd::launch_tree_build(batch, B, Kmax, K, p, node_indptr, total_nodes, mask_words,
                                            parent, depth, path_id, anc_mask, path_leaf, stream),
                    "tree_build launch");
}

d2sd_status d2sd_tree_from_parents(int batch, const int* node_indptr, int total_nodes, int max_nodes,
                                   int mask_words, const int* parent, int* depth, int* path_id,
                                   uint32_t* anc_mask, hipStream_t stream) {
  if (batch < 1) return fail(D2SD_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", batch);
  if (total_nodes < 0) return fail(D2SD_ERR_INVALID_ARG, "total_nodes must be >= 0");
  if (max_nodes < 1 || max_nodes > kMaxTreeNodes)
    return fail(D2SD_ERR_INVALID_ARG, "max_nodes %d outside [1, %d]", max_nodes, kMaxTreeNodes);
  if ((long long)mask_words * 32 < max_nodes)
    return fail(D2SD_ERR_INVALID_ARG, "mask_words %d too small for max_nodes %d", mask_words, max_nodes);
  if (!node_indptr || !parent || !depth || !path_id || !anc_mask)
    return fail(D2SD_ERR_INVALID_ARG, "a required device pointer is NULL");
  return hip_status(d2sd::launch_tree_from_parents(batch, node_indptr, total_nodes, max_nodes, mask_words, parent,
                                                   depth, path_id, anc_mask, stream),
                    "tree_from_parents launch");
}

d2sd_status d2sd_select_reanchor(int batch, int B, int Kmax, const float* conf, const int* K, int* p_out,
                                 double* r_out, hipStream_t stream) {
  if (batch < 1) return fail(D2SD_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", batch);
  if (B < 2 || B > D2SD_MAX_B) return fail(D2SD_ERR_INVALID_ARG, "B = %d outside [2, %d]", B, D2SD_MAX_B);
  if (Kmax < 1) return fail(D2SD_ERR_INVALID_ARG, "Kmax must be >= 1 (got %d)", Kmax);
  if (!conf || !K || !p_out) return fail(D2SD_ERR_INVALID_ARG, "a required device pointer is NULL");
  return hip_status(d2sd::launch_select_reanchor(batch, B, Kmax, conf, K, p_out, r_out, stream),
                    "select_reanchor launch");
}

d2sd_status d2sd_tree_indptr(int batch, int B, int Kmax, const int* K, const int* p, int* node_indptr,
                             hipStream_t stream) {
  if (batch < 1) return fail(D2SD_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", batch);
  if (B < 2 || B > D2SD_MAX_B) return fail(D2SD_ERR_INVALID_ARG, "B = %d outside [2, %d]", B, D2SD_MAX_B);
  if (Kmax < 0) return fail(D2SD_ERR_INVALID_ARG, "Kmax must be >= 0");
  if (!K || (Kmax > 0 && !p) || !node_indptr) return fail(D2SD_ERR_INVALID_ARG, "a required device pointer is NULL");
  return hip_status(d2sd::launch_tree_indptr(batch, B, Kmax, K, p, node_indptr, stream), "tree_indptr launch");
}

d2sd_status d2sd_commit_accepted_kv(int batch, int B, int num_kv_heads, int head_dim, int page_size, int dtype,
                                    int num_pages, int max_pages, int max_ctx_len, const int* node_indptr,
                                    int total_nodes, const int* path_nodes, const int* accept_len,
                                    const void* k_tree, const void* v_tree, const int* page_table, int* ctx_len,
                                    void* k_cache, void* v_cache, hipStream_t stream) {
  if (batch < 1) return fail(D2SD_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", batch);
  if (B < 2 || B > D2SD_MAX_B) return fail(D2SD_ERR_INVALID_ARG, "B = %d outside [2, %d]", B, D2SD_MAX_B);
  if (num_kv_heads < 1) return fail(D2SD_ERR_INVALID_ARG, "num_kv_heads must be >= 1");
  if (head_dim != D2SD_HEAD_DIM) return fail(D2SD_ERR_UNSUPPORTED, "head_dim %d != %d", head_dim, D2SD_HEAD_DIM);
  if (page_size != D2SD_PAGE_SIZE)
    return fail(D2SD_ERR_UNSUPPORTED, "page_size %d != %d", page_size, D2SD_PAGE_SIZE);
  if (dtype != D2SD_F32 && dtype != D2SD_BF16) return fail(D2SD_ERR_INVALID_ARG, "dtype %d unknown", dtype);
  if (num_pages < 1 || max_pages < 1) return fail(D2SD_ERR_INVALID_ARG, "num_pages and max_pages must be >= 1");
  if (total_nodes < 0 || max_ctx_len < 0) return fail(D2SD_ERR_INVALID_ARG, "negative size");
  if ((long long)max_ctx_len + B > (long long)max_pages * page_size)
    return fail(D2SD_ERR_INVALID_ARG, "max_ctx_len + B = %lld exceeds max_pages * page_size = %lld",
                (long long)max_ctx_len + B, (long long)max_pages * page_size);
  if (!node_indptr || !path_nodes || !accept_len || !k_tree || !v_tree || !page_table || !ctx_len || !k_cache ||
      !v_cache)
    return fail(D2SD_ERR_INVALID_ARG, "a required device pointer is NULL");
  const void* const chunked[] = {k_tree, v_tree, k_cache, v_cache};
  const char* const names[] = {"k_tree", "v_tree", "k_cache", "v_cache"};
  for (int i = 0; i < 4; ++i)  // rows move in 16-byte chunks
    if (reinterpret_cast<uintptr_t>(chunked[i]) % 16 != 0)
      return fail(D2SD_ERR_INVALID_ARG, "%s is not 16-byte aligned", names[i]);
  const int row_bytes = head_dim * (dtype == D2SD_BF16 ? 2 : 4);
  if ((long long)B * num_kv_heads * (row_bytes / 16) > 0x7fffffffll)
    return fail(D2SD_ERR_UNSUPPORTED, "B x num_kv_heads x %d chunks exceeds 2^31 - 1", row_bytes / 16);
  return hip_status(d2sd::launch_commit(batch, B, num_kv_heads, row_bytes, num_pages, max_pages, max_ctx_len,
                                        node_indptr, total_nodes, path_nodes, accept_len, k_tree, v_tree,
                                        page_table, ctx_len, k_cache, v_cache, stream),
                    "commit launch");
}

d2sd_status d2sd_cascade_kv_split(const d2sd_attn_args* args, int* kv_split) {
  d2sd_status s = validate_attn(args, false);
  if (s) return s;
  if (!kv_split) return fail(D2SD_ERR_INVALID_ARG, "kv_split is NULL");
  d2sd::AttnPlan plan;
  if ((s = make_plan(args, &plan))) return s;
  *kv_split = plan.split;
  return ok();
}

d2sd_status d2sd_cascade_row_group(const d2sd_attn_args* args, int* rows, int* packed) {
  d2sd_status s = validate_attn(args, false);
  if (s) return s;
  if (!rows) return fail(D2SD_ERR_INVALID_ARG, "rows is NULL");
  d2sd::AttnPlan plan;
  if ((s = make_plan(args, &plan))) return s;
  *rows = plan.waves * d2sd::kRowsPerTile;
  if (packed) *packed = plan.packed ? 1 : 0;
  return ok();
}

d2sd_status d2sd_cascade_workspace_size(const d2sd_attn_args* args, size_t* bytes) {
  d2sd_status s = validate_attn(args, false);
  if (s) return s;
  if (!bytes) return fail(D2SD_ERR_INVALID_ARG, "bytes is NULL");
  d2sd::AttnPlan plan;
  if ((s = make_plan(args, &plan))) return s;
  *bytes = plan.ws_bytes;
  return ok();
}

d2sd_status d2sd_cascade_verify_attention(const d2sd_attn_args* args, void* ws, size_t ws_bytes,
                                          hipStream_t stream) {
  d2sd_status s = validate_attn(args, true);
  if (s) return s;
  d2sd::AttnPlan plan;
  if ((s = make_plan(args, &plan))) return s;
  if (plan.ws_bytes > 0 && (!ws || ws_bytes < plan.ws_bytes))
    return fail(D2SD_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", ws ? ws_bytes : 0,
                plan.ws_bytes);
  if (args->total_nodes == 0) return ok();
  hipEvent_t ev[3];
  timing_begin(ev);
  const hipError_t e = d2sd::launch_cascade_attention(*args, plan, ws, stream, ev);
  timing_end(ev, e == hipSuccess, plan.n_ch_max > 1);
  return hip_status(e, "cascade attention launch");
}

d2sd_status d2sd_cascade_verify_attention_noalloc(const d2sd_attn_args* args, hipStream_t stream) {
  d2sd_status s = validate_attn(args, true);
  if (s) return s;
  d2sd::AttnPlan plan;
  if ((s = make_plan(args, &plan))) return s;
  if (plan.ws_bytes > d2sd::kScratchBytes) {
    if (args->kv_split > 0)
      return fail(D2SD_ERR_WORKSPACE_TOO_SMALL,
                  "kv_split %d needs %zu bytes of partial states; the static scratch holds %zu "
                  "(use a longer kv_split, or the workspace entry point)",
                  args->kv_split, plan.ws_bytes, d2sd::kScratchBytes);
    // automatic split: fewer, longer splits until the partial states fit
    d2sd_attn_args fit = *args;
    const int ctx = args->max_ctx_len;
    const int s_lo = max(1, (ctx + kMaxSplit - 1) / kMaxSplit);
    bool found = false;
    for (int n = plan.n_ch_max - 1; n >= s_lo && !found; --n) {
      fit.kv_split = min(kMaxSplit, ((ctx + n - 1) / n + 63) / 64 * 64);
      if ((s = make_plan(&fit, &plan))) return s;
      found = plan.ws_bytes <= d2sd::kScratchBytes;
    }
    if (!found)
      return fail(D2SD_ERR_WORKSPACE_TOO_SMALL,
                  "the partial states of %d context splits need %zu bytes; the static scratch holds %zu",
                  plan.n_ch_max, plan.ws_bytes, d2sd::kScratchBytes);
  }
  if (args->total_nodes == 0) return ok();
  void* ws = nullptr;
  if (plan.ws_bytes > 0) {
    const hipError_t e = d2sd::scratch_address(&ws);
    if (e != hipSuccess) return hip_status(e, "static scratch address");
  }
  hipEvent_t ev[3];
  timing_begin(ev);
  const hipError_t e = d2sd::launch_cascade_attention(*args, plan, ws, stream, ev);
  timing_end(ev, e == hipSuccess, plan.n_ch_max > 1);
  return hip_status(e, "cascade attention launch");
}

d2sd_status d2sd_noncascade_verify_attention(const d2sd_attn_args* args, hipStream_t stream) {
  d2sd_status s = validate_attn(args, true);
  if (s) return s;
  if (args->stage != D2SD_STAGE_CASCADE)
    return fail(D2SD_ERR_INVALID_ARG, "the non-cascade baseline computes STAGE_CASCADE only");
  if ((long long)args->batch * args->num_kv_heads * args->max_nodes > (1ll << 30))
    return fail(D2SD_ERR_UNSUPPORTED, "too many work items");
  if (args->num_qo_heads / args->num_kv_heads > 4 * d2sd::kRowsPerTile)
    return fail(D2SD_ERR_UNSUPPORTED, "the baseline supports at most %d query heads per KV head",
                4 * d2sd::kRowsPerTile);
  if (args->dtype == D2SD_BF16 && args->max_ctx_len > kMaxSplit)
    return fail(D2SD_ERR_UNSUPPORTED, "the baseline streams at most %d context tokens per request", kMaxSplit);
  if (args->total_nodes == 0) return ok();
  const float scale = args->sm_scale > 0.0f ? args->sm_scale : 1.0f / sqrtf((float)args->head_dim);
  hipEvent_t ev[3];
  timing_begin(ev);
  const hipError_t e = d2sd::launch_noncascade_attention(*args, scale, stream, ev);
  timing_end(ev, e == hipSuccess, false);
  return hip_status(e, "non-cascade attention launch");
}

d2sd_status d2sd_merge_state(int rows, int head_dim, const float* o_a, const float* lse_a,
                             const float* o_b, const float* lse_b, float* o_out, float* lse_out,
                             hipStream_t stream) {
  if (rows < 0) return fail(D2SD_ERR_INVALID_ARG, "rows must be >= 0");
  if (head_dim < 1 || head_dim > 1024) return fail(D2SD_ERR_INVALID_ARG, "head_dim %d outside [1, 1024]", head_dim);
  if (!o_a || !lse_a || !o_b || !lse_b || !o_out || !lse_out)
    return fail(D2SD_ERR_INVALID_ARG, "a required device pointer is NULL");
  if (rows == 0) return ok();
  return hip_status(d2sd::launch_merge_state(rows, head_dim, o_a, lse_a, o_b, lse_b, o_out, lse_out, stream),
                    "merge_state launch");
}

d2sd_status d2sd_accept_path(int batch, int B, const int* node_indptr, int total_nodes,
                             const int* parent, const int* depth, const int* path_id,
                             const int* draft_tokens, const int* target_argmax, int* accept_len,
                             int* best_path, int* accept_node, int* path_nodes, int* out_tokens,
                             hipStream_t stream) {
  if (batch < 1) return fail(D2SD_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", batch);
  if (B < 2 || B > D2SD_MAX_B) return fail(D2SD_ERR_INVALID_ARG, "B = %d outside [2, %d]", B, D2SD_MAX_B);
  if (total_nodes < 0) return fail(D2SD_ERR_INVALID_ARG, "total_nodes must be >= 0");
  if (!node_indptr || !parent || !depth || !path_id || !draft_tokens || !target_argmax || !accept_len ||
      !best_path || !accept_node || !path_nodes || !out_tokens)
    return fail(D2SD_ERR_INVALID_ARG, "a required device pointer is NULL");
  return hip_status(d2sd::launch_accept_path(batch, B, node_indptr, total_nodes, parent, depth, path_id,
                                             draft_tokens, target_argmax, accept_len, best_path,
                                             accept_node, path_nodes, out_tokens, stream),
                    "accept_path launch");
}

d2sd_status d2sd_sample_targets(int batch, const int* node_indptr, int total_nodes, int max_nodes,
                                const int* parent, const int* draft_tokens, int vocab, int dtype,
                                const void* logits, float temperature, const float* uniform,
                                int* context_rep, int* target_tokens, hipStream_t stream) {
  if (batch < 1) return fail(D2SD_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", batch);
  if (total_nodes < 0) return fail(D2SD_ERR_INVALID_ARG, "total_nodes must be >= 0");
  if (max_nodes < 1 || max_nodes > kMaxTreeNodes)
    return fail(D2SD_ERR_INVALID_ARG, "max_nodes = %d outside [1, %d]", max_nodes, kMaxTreeNodes);
  if ((long long)batch * max_nodes > 0x7fffffffLL)
    return fail(D2SD_ERR_INVALID_ARG, "batch * max_nodes = %lld exceeds 2^31 - 1", (long long)batch * max_nodes);
  if (vocab < 1 || vocab > D2SD_MAX_VOCAB)
    return fail(D2SD_ERR_INVALID_ARG, "vocab = %d outside [1, %d]", vocab, D2SD_MAX_VOCAB);
  if (dtype != D2SD_F32 && dtype != D2SD_BF16) return fail(D2SD_ERR_INVALID_ARG, "dtype %d unknown", dtype);
  if (!(temperature == 0.0f || (temperature >= 1e-6f && temperature <= 1e6f)))
    return fail(D2SD_ERR_INVALID_ARG, "temperature must be 0 or in [1e-6, 1e6]");
  if (!node_indptr || !parent || !draft_tokens || !logits || !target_tokens || (temperature != 0.0f && !uniform))
    return fail(D2SD_ERR_INVALID_ARG, "a required device pointer is NULL");
  if (reinterpret_cast<uintptr_t>(logits) % 16 != 0) return fail(D2SD_ERR_INVALID_ARG, "logits not 16-byte aligned");
  return hip_status(d2sd::launch_sample_targets(batch, node_indptr, total_nodes, max_nodes, parent, draft_tokens,
                                                vocab, dtype, logits, temperature, uniform, context_rep,
                                                target_tokens, stream),
                    "sample_targets launch");
}

d2sd_status d2sd_kernel_timing_enable(int enable) {
  std::lock_guard<std::mutex> lk(g_timing_mu);
  g_timing_on = enable != 0;
  return ok();
}

d2sd_status d2sd_kernel_timing_collect(int* launches, double* total_ms) {
  if (!launches || !total_ms) return fail(D2SD_ERR_INVALID_ARG, "output pointer is NULL");
  std::vector<float> kern, merge;
  const hipError_t err = collect_timings(&kern, &merge);
  double sum = 0.0;
  for (size_t i = 0; i < kern.size(); ++i) sum += (double)kern[i] + merge[i];
  *launches = (int)kern.size();
  *total_ms = sum;
  return hip_status(err, "kernel timing");
}

d2sd_status d2sd_kernel_timing_collect_each(int capacity, float* ms_each, int* launches) {
  if (!launches || capacity < 0 || (capacity > 0 && !ms_each))
    return fail(D2SD_ERR_INVALID_ARG, "launches is NULL, capacity < 0, or ms_each is NULL");
  std::vector<float> kern, merge;
  const hipError_t err = collect_timings(&kern, &merge);
  for (size_t i = 0; i < kern.size() && i < (size_t)capacity; ++i) ms_each[i] = kern[i] + merge[i];
  *launches = (int)kern.size();
  return hip_status(err, "kernel timing");
}

d2sd_status d2sd_kernel_timing_collect_parts(int capacity, float* kernel_ms, float* merge_ms, int* launches) {
  if (!launches || capacity < 0 || (capacity > 0 && (!kernel_ms || !merge_ms)))
    return fail(D2SD_ERR_INVALID_ARG, "launches is NULL, capacity < 0, or an output array is NULL");
  std::vector<float> kern, merge;
  const hipError_t err = collect_timings(&kern, &merge);
  for (size_t i = 0; i < kern.size() && i < (size_t)capacity; ++i) {
    kernel_ms[i] = kern[i];
    merge_ms[i] = merge[i];
  }
  *launches = (int)kern.size();
  return hip_status(err, "kernel timing");
}

}  // extern "C"
