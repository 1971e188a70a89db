// Host runtime of RKSC around the GPU path: the RSBCM block table (Sec. 2.4,
// Alg. RsbcmEvict) and the self-calibrating KV probe (Sec. 2.2, paragraph
// "KV probe").
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <map>
#include <set>
#include <tuple>
#include <unordered_map>
#include <vector>

#include "../../include/rksc.h"
#include "status.h"

#define RKSC_EXPORT extern "C" __attribute__((visibility("default")))

using rksc::fail;
using rksc::ok;

// ------------------------------------------------------------------ RSBCM

// Blocks ordered by (omega, insertion sequence): the first element is the one
// Alg. RsbcmEvict removes next. omega = score / (depth + 1) is evaluated in
// double (exact inputs, one correctly rounded division), so equal inputs give
// equal keys and ties fall to the earliest insertion.
struct rksc_block_table {
  struct Entry {
    double omega;
    uint64_t seq;
    int64_t id;
    bool operator<(const Entry& o) const { return std::tie(omega, seq) < std::tie(o.omega, o.seq); }
  };
  struct Info {
    float score;
    int32_t depth;
    uint64_t seq;
  };
  int32_t capacity = 0;
  uint64_t next_seq = 0;
  int64_t evicted_total = 0;
  std::set<Entry> order;
  std::unordered_map<int64_t, Info> blocks;

  static double omega(float score, int32_t depth) { return (double)score / ((double)depth + 1.0); }
};

RKSC_EXPORT rksc_block_table* rksc_block_table_create(int32_t capacity) {
  if (capacity < 0) {
    fail(RKSC_ERR_INVALID_ARGUMENT, "capacity must be >= 0 (got %d)", capacity);
    return nullptr;
  }
  rksc_block_table* t = new rksc_block_table;
  t->capacity = capacity;
  ok();
  return t;
}

RKSC_EXPORT void rksc_block_table_destroy(rksc_block_table* t) { delete t; }

RKSC_EXPORT rksc_status rksc_block_table_insert(rksc_block_table* t, int64_t block_id, float score, int32_t depth) {
  if (!t) return fail(RKSC_ERR_INVALID_ARGUMENT, "table is NULL");
  if (!std::isfinite(score)) return fail(RKSC_ERR_INVALID_ARGUMENT, "score must be finite");
  if (depth < 0) return fail(RKSC_ERR_INVALID_ARGUMENT, "depth must be >= 0 (got %d)", depth);
  if (t->blocks.count(block_id))
    return fail(RKSC_ERR_INVALID_ARGUMENT, "block %lld is already in the table", (long long)block_id);
  const uint64_t seq = t->next_seq++;
  t->blocks.emplace(block_id, rksc_block_table::Info{score, depth, seq});
  t->order.insert({rksc_block_table::omega(score, depth), seq, block_id});
  return ok();
}

RKSC_EXPORT rksc_status rksc_block_table_set_score(rksc_block_table* t, int64_t block_id, float score) {
  if (!t) return fail(RKSC_ERR_INVALID_ARGUMENT, "table is NULL");
  if (!std::isfinite(score)) return fail(RKSC_ERR_INVALID_ARGUMENT, "score must be finite");
  auto it = t->blocks.find(block_id);
  if (it == t->blocks.end())
    return fail(RKSC_ERR_INVALID_ARGUMENT, "block %lld is not in the table", (long long)block_id);
  rksc_block_table::Info& b = it->second;
  t->order.erase({rksc_block_table::omega(b.score, b.depth), b.seq, block_id});
  b.score = score;
  t->order.insert({rksc_block_table::omega(b.score, b.depth), b.seq, block_id});
  return ok();
}

RKSC_EXPORT rksc_status rksc_block_table_remove(rksc_block_table* t, int64_t block_id) {
  if (!t) return fail(RKSC_ERR_INVALID_ARGUMENT, "table is NULL");
  auto it = t->blocks.find(block_id);
  if (it == t->blocks.end())
    return fail(RKSC_ERR_INVALID_ARGUMENT, "block %lld is not in the table", (long long)block_id);
  const rksc_block_table::Info& b = it->second;
  t->order.erase({rksc_block_table::omega(b.score, b.depth), b.seq, block_id});
  t->blocks.erase(it);
  return ok();
}

RKSC_EXPORT rksc_status rksc_block_table_evict(rksc_block_table* t, int64_t* evicted, int32_t max_evicted,
                                               int32_t* n_evicted) {
  if (!t) return fail(RKSC_ERR_INVALID_ARGUMENT, "table is NULL");
  if (!n_evicted) return fail(RKSC_ERR_INVALID_ARGUMENT, "n_evicted is NULL");
  const int64_t over = (int64_t)t->blocks.size() - t->capacity;
  if (over > 0 && (!evicted || max_evicted < over))
    return fail(RKSC_ERR_INVALID_ARGUMENT, "%lld blocks must be evicted but evicted holds %d", (long long)over,
                evicted ? max_evicted : 0);
  int32_t n = 0;
  while ((int64_t)t->blocks.size() > t->capacity) {
    const auto first = t->order.begin();
    const int64_t id = first->id;
    t->order.erase(first);
    t->blocks.erase(id);
    evicted[n++] = id;
  }
  t->evicted_total += n;
  *n_evicted = n;
  return ok();
}

RKSC_EXPORT int32_t rksc_block_table_size(const rksc_block_table* t) { return t ? (int32_t)t->blocks.size() : -1; }

RKSC_EXPORT int64_t rksc_block_table_evicted_total(const rksc_block_table* t) { return t ? t->evicted_total : -1; }

// ------------------------------------------------------------------ KV probe

struct rksc_kv_probe {
  int32_t reps = 3;
  struct Verdict {
    int32_t share;
    float ms[3];
  };
  std::map<int32_t, Verdict> buckets;   // k = floor(n / 64) -> verdict
};

namespace {

constexpr int kProbeBucket = 64;

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

// Regions of the probe's workspace: one scratch area that the three paths use
// in turn, and the buffers that outlive a path.
struct ProbeLayout {
  size_t scratch, cache_full, prefix_k, prefix_v, h_root, cache_sfx, tokens, outs, total;
  size_t cache_full_bytes, cache_sfx_bytes;
};

bool probe_layout(const rksc_model_config* c, int n, int B, int s, ProbeLayout* lay) {
  const size_t ws_full = rksc_decode_workspace_size(c, B, n + s, 0);
  if (!ws_full) return false;
  const size_t ws_pre = rksc_prefill_workspace_size(c, n);
  if (!ws_pre) return false;
  const size_t ws_sfx = rksc_decode_workspace_size(c, B, s, n);
  if (!ws_sfx) return false;
  const size_t T = c->dtype == RKSC_BF16 ? 2 : 4;
  const size_t L = c->n_layers, Hkv = c->n_kv_heads, hd = c->head_dim;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align256(off + bytes);
    return at;
  };
  lay->scratch = take(std::max(ws_full, std::max(ws_pre, ws_sfx)));
  lay->cache_full_bytes = L * B * Hkv * (size_t)(n + s) * hd * T;
  lay->cache_full = take(2 * lay->cache_full_bytes);
  lay->prefix_k = take(L * Hkv * (size_t)n * hd * T);
  lay->prefix_v = take(L * Hkv * (size_t)n * hd * T);
  lay->h_root = take(L * (size_t)c->d_model * 4);
  lay->cache_sfx_bytes = L * B * Hkv * (size_t)s * hd * T;
  lay->cache_sfx = take(2 * lay->cache_sfx_bytes);
  lay->tokens = take((size_t)B * (n + s) * 4);
  lay->outs = take((size_t)B * 12);
  lay->total = off;
  return true;
}

}  // namespace

RKSC_EXPORT rksc_kv_probe* rksc_kv_probe_create(int32_t reps) {
  if (reps < 1) {
    fail(RKSC_ERR_INVALID_ARGUMENT, "reps must be >= 1 (got %d)", reps);
    return nullptr;
  }
  rksc_kv_probe* p = new rksc_kv_probe;
  p->reps = reps;
  ok();
  return p;
}

RKSC_EXPORT void rksc_kv_probe_destroy(rksc_kv_probe* p) { delete p; }

RKSC_EXPORT size_t rksc_kv_probe_workspace_size(const rksc_model_config* cfg, int32_t n_prefix, int32_t n_branches,
                                                int32_t suffix_len) {
  if (n_prefix < 1) {
    fail(RKSC_ERR_INVALID_ARGUMENT, "n_prefix must be >= 1 (got %d)", n_prefix);
    return 0;
  }
  ProbeLayout lay;
  if (!probe_layout(cfg, n_prefix, n_branches, suffix_len, &lay)) return 0;
  return lay.total;
}

RKSC_EXPORT rksc_status rksc_kv_probe_lookup(const rksc_kv_probe* p, int32_t n_prefix, int32_t* share,
                                             float* times_ms) {
  if (!p) return fail(RKSC_ERR_INVALID_ARGUMENT, "probe is NULL");
  if (!share) return fail(RKSC_ERR_INVALID_ARGUMENT, "share is NULL");
  if (n_prefix < 0) return fail(RKSC_ERR_INVALID_ARGUMENT, "n_prefix must be >= 0 (got %d)", n_prefix);
  auto it = p->buckets.find(n_prefix / kProbeBucket);
  if (it == p->buckets.end()) {
    *share = -1;
    return ok();
  }
  *share = it->second.share;
  if (times_ms) std::copy(it->second.ms, it->second.ms + 3, times_ms);
  return ok();
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess)                                                               \
      return fail(RKSC_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));         \
  } while (0)

// Times one path `reps` times on `stream` with HIP events; *best = the minimum.
template <typename F>
static rksc_status time_min(int reps, hipStream_t stream, F&& path, float* best) {
  hipEvent_t a, b;
  HIP_TRY(hipEventCreate(&a));
  if (hipEventCreate(&b) != hipSuccess) {
    (void)hipEventDestroy(a);
    return fail(RKSC_ERR_HIP, "hipEventCreate failed");
  }
  rksc_status st = RKSC_OK;
  float m = INFINITY;
  for (int r = 0; r < reps && st == RKSC_OK; ++r) {
    hipError_t e = hipEventRecord(a, stream);
    if (e == hipSuccess) {
      st = path();
      if (st != RKSC_OK) break;
      e = hipEventRecord(b, stream);
    }
    if (e == hipSuccess) e = hipEventSynchronize(b);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
    if (e != hipSuccess) st = fail(RKSC_ERR_HIP, "probe timing failed: %s", hipGetErrorString(e));
    m = std::min(m, ms);
  }
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  *best = m;
  return st;
}

// The KV probe of Sec. 2.2: at the first call within a 64-token prefix-length
// bucket k = floor(n / 64) it times, as the minimum of `reps` runs each,
// (i) the batched full recompute (every branch's prefix and suffix as one
// sequence, no sharing), (ii) one root forward over the prefix, and (iii) the
// batched suffix decode over that shared cache, and declares sharing
// beneficial iff (ii) + (iii) < (i). Later calls in the bucket return the
// stored verdict without running anything.
RKSC_EXPORT rksc_status rksc_kv_probe_decide(rksc_kv_probe* p, const rksc_weights* w, const int32_t* prefix_tokens,
                                             int32_t n_prefix, const int32_t* suffix_tokens, int32_t n_branches,
                                             int32_t suffix_len, void* workspace, size_t workspace_bytes,
                                             void* stream, int32_t* share, float* times_ms, int32_t* probed) {
  if (!p) return fail(RKSC_ERR_INVALID_ARGUMENT, "probe is NULL");
  if (!share) return fail(RKSC_ERR_INVALID_ARGUMENT, "share is NULL");
  if (n_prefix < 1) return fail(RKSC_ERR_INVALID_ARGUMENT, "n_prefix must be >= 1 (got %d)", n_prefix);
  const int32_t bucket = n_prefix / kProbeBucket;
  auto it = p->buckets.find(bucket);
  if (it != p->buckets.end()) {
    *share = it->second.share;
    if (times_ms) std::copy(it->second.ms, it->second.ms + 3, times_ms);
    if (probed) *probed = 0;
    return ok();
  }
  if (!w) return fail(RKSC_ERR_INVALID_ARGUMENT, "weights is NULL");
  if (!prefix_tokens || !suffix_tokens) return fail(RKSC_ERR_INVALID_ARGUMENT, "token pointers must not be NULL");
  if (!workspace) return fail(RKSC_ERR_INVALID_ARGUMENT, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(RKSC_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  const rksc_model_config* c = &w->cfg;
  ProbeLayout lay;
  if (!probe_layout(c, n_prefix, n_branches, suffix_len, &lay)) return RKSC_ERR_INVALID_ARGUMENT;
  if (workspace_bytes < lay.total)
    return fail(RKSC_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, needs %zu", workspace_bytes, lay.total);

  const int n = n_prefix, B = n_branches, s = suffix_len;
  hipStream_t strm = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  void* scratch = ws + lay.scratch;
  const size_t scratch_bytes = lay.cache_full - lay.scratch;
  int32_t* tokens = reinterpret_cast<int32_t*>(ws + lay.tokens);
  int32_t* next_tok = reinterpret_cast<int32_t*>(ws + lay.outs);
  float* p_top = reinterpret_cast<float*>(next_tok + B);
  float* conf = p_top + B;
  // Path (i)'s token rows: [prefix ; suffix of branch b].
  for (int b = 0; b < B; ++b)
    HIP_TRY(hipMemcpyAsync(tokens + (size_t)b * (n + s), prefix_tokens, (size_t)n * 4, hipMemcpyDeviceToDevice,
                           strm));
  HIP_TRY(hipMemcpy2DAsync(tokens + n, (size_t)(n + s) * 4, suffix_tokens, (size_t)s * 4, (size_t)s * 4, B,
                           hipMemcpyDeviceToDevice, strm));

  const rksc_prefix_kv none{0, nullptr, nullptr};
  const rksc_prefix_kv shared{n, ws + lay.prefix_k, ws + lay.prefix_v};
  auto full = [&]() -> rksc_status {
    rksc_branch_kv bkv{n + s, 0, ws + lay.cache_full, ws + lay.cache_full + lay.cache_full_bytes};
    return rksc_decode_suffix(w, &none, &bkv, tokens, B, n + s, next_tok, p_top, conf, scratch, scratch_bytes,
                              stream);
  };
  auto root = [&]() -> rksc_status {
    return rksc_prefill(w, prefix_tokens, n, ws + lay.prefix_k, ws + lay.prefix_v,
                        reinterpret_cast<float*>(ws + lay.h_root), scratch, scratch_bytes, stream);
  };
  auto suffix = [&]() -> rksc_status {
    rksc_branch_kv bkv{s, 0, ws + lay.cache_sfx, ws + lay.cache_sfx + lay.cache_sfx_bytes};
    return rksc_decode_suffix(w, &shared, &bkv, suffix_tokens, B, s, next_tok, p_top, conf, scratch,
                              scratch_bytes, stream);
  };
  rksc_kv_probe::Verdict v{};
  rksc_status st = time_min(p->reps, strm, full, &v.ms[0]);
  if (st == RKSC_OK) st = time_min(p->reps, strm, root, &v.ms[1]);
  if (st == RKSC_OK) st = time_min(p->reps, strm, suffix, &v.ms[2]);
  if (st != RKSC_OK) return st;
  v.share = v.ms[1] + v.ms[2] < v.ms[0] ? 1 : 0;
  p->buckets[bucket] = v;
  *share = v.share;
  if (times_ms) std::copy(v.ms, v.ms + 3, times_ms);
  if (probed) *probed = 1;
  return ok();
}
