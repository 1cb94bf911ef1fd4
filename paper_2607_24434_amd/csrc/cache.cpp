// Expert cache of the offloaded decoding step (Section 3.5, Algorithm 1):
// the accelerator expert set C as per-layer HBM slots over a pinned host
// pool, the in-flight set P as copies on two copy streams with per-slot
// events, prefetch of predicted verifier experts and on-demand loads of
// misses.  The bookkeeping is plain host code and deterministic; copies and
// waits are HIP stream operations, so nothing here blocks the host except
// the statistics read-out.
#include "../../include/draftexpert.h"

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <new>
#include <utility>
#include <vector>

struct de_cache {
  de_cache_cfg cfg{};
  int L = 0, N = 0, S = 0;
  // Bookkeeping, [L][N] or [L][S] row-major.
  std::vector<int32_t> where;      // slot of each expert, -1 = not resident
  std::vector<int32_t> held;       // expert in each slot, -1 = free
  std::vector<int64_t> last_use;   // LRU time of each slot
  std::vector<uint8_t> prefetched; // slot filled by a prefetch the block's verify has not used
  std::vector<uint8_t> predicted;  // expert predicted for the current block
  int64_t clock = 0;
  de_cache_counts st{};
  // HIP objects (absent with fake copies).
  hipStream_t prefetch_stream = nullptr;
  hipStream_t demand_stream = nullptr;
  std::vector<hipEvent_t> slot_ev;      // completion of the last copy into each slot
  std::vector<uint8_t> slot_ev_live;    // slot_ev has been recorded
  std::vector<hipEvent_t> layer_ev;     // the last compute work reading each layer's slots
  std::vector<uint8_t> layer_ev_live;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> stalls;  // compute-stream waits to time
  std::vector<std::pair<hipEvent_t, hipEvent_t>> spans[2]; // cached layers (draft, verify)
  hipEvent_t span_open = nullptr;
  std::vector<hipEvent_t> spare;        // timing events for reuse
  int32_t* staging = nullptr;           // pinned [L][kStage][N] slot-table uploads
  std::vector<int> stage_next;
  std::vector<hipEvent_t> stage_ev;     // completion of the upload from each staging row
  std::vector<uint8_t> stage_ev_live;
  int32_t* readback = nullptr;          // pinned scratch of the cached step
};

namespace de {

constexpr int kStage = 8;           // slot-table uploads in flight per layer
constexpr int kReadbackInts = 4096; // pinned readback scratch of the cached step

int32_t* cache_readback(de_cache* c) { return c ? c->readback : nullptr; }
int cache_slots_per_layer(const de_cache* c) { return c ? c->S : 0; }
int cache_experts(const de_cache* c) { return c ? c->N : 0; }
int cache_layers(const de_cache* c) { return c ? c->L : 0; }
bool cache_resident(const de_cache* c, int layer, int e) {
  return c->where[(size_t)layer * c->N + e] >= 0;
}

hipEvent_t timing_event(de_cache* c);

// Brackets one cached layer on the compute stream (begin, then end with its
// purpose); the durations are summed by de_cache_stats.
int cache_span(de_cache* c, bool end, int purpose, hipStream_t s) {
  if (c->cfg.fake_copies) return DE_OK;
  hipEvent_t e = timing_event(c);
  if (e == nullptr || hipEventRecord(e, s) != hipSuccess) return DE_ERR_HIP;
  if (!end) {
    c->span_open = e;
    return DE_OK;
  }
  if (c->span_open == nullptr) return DE_ERR_INVALID;
  c->spans[purpose == DE_NEED_VERIFY ? 1 : 0].emplace_back(c->span_open, e);
  c->span_open = nullptr;
  return DE_OK;
}

}  // namespace de

namespace {

bool fake(const de_cache* c) { return c->cfg.fake_copies != 0; }

const char* host_block(const de_cache* c, int l, int e) {
  return static_cast<const char*>(c->cfg.host_pool) +
         ((size_t)l * c->N + e) * (size_t)c->cfg.expert_bytes;
}

char* slot_block(const de_cache* c, int l, int s) {
  return static_cast<char*>(c->cfg.slot_pool) +
         ((size_t)l * c->S + s) * (size_t)c->cfg.slot_stride_bytes;
}

// Victim for a copy into `layer`: a free slot (lowest index), else the least
// recently used slot (ties: lowest index) whose expert is not in `need`;
// experts predicted for the block are taken only when allow_predicted and no
// other slot qualifies.  -1 when none.
int pick_slot(const de_cache* c, int l, const uint8_t* need, bool allow_predicted) {
  const size_t so = (size_t)l * c->S, eo = (size_t)l * c->N;
  for (int s = 0; s < c->S; ++s)
    if (c->held[so + s] < 0) return s;
  for (int tier = 0; tier < (allow_predicted ? 2 : 1); ++tier) {
    int best = -1;
    for (int s = 0; s < c->S; ++s) {
      const int e = c->held[so + s];
      if (need != nullptr && need[e]) continue;
      if ((c->predicted[eo + e] != 0) != (tier == 1)) continue;
      if (best < 0 || c->last_use[so + s] < c->last_use[so + best]) best = s;
    }
    if (best >= 0) return best;
  }
  return -1;
}

// Puts expert e of layer l into slot s (evicting its holder) and starts the
// copy.  Every copy into a slot waits for the previous copy into it and for
// the compute work that last read the layer's slots.
int load(de_cache* c, int l, int e, int s, bool prefetch) {
  const size_t so = (size_t)l * c->S, eo = (size_t)l * c->N;
  const int old = c->held[so + s];
  if (old >= 0) {
    c->where[eo + old] = -1;
    ++c->st.evictions;
    if (c->prefetched[so + s]) ++c->st.prefetch_wasted;  // evicted before its verify used it
  }
  c->held[so + s] = e;
  c->where[eo + e] = s;
  c->last_use[so + s] = ++c->clock;
  c->prefetched[so + s] = prefetch ? 1 : 0;
  c->st.bytes_copied += c->cfg.expert_bytes;
  if (prefetch)
    ++c->st.prefetch_issued;
  else
    ++c->st.demand_loads;
  if (fake(c)) {
    std::memcpy(slot_block(c, l, s), host_block(c, l, e), (size_t)c->cfg.expert_bytes);
    return DE_OK;
  }
  hipStream_t cs = prefetch ? c->prefetch_stream : c->demand_stream;
  if (c->slot_ev_live[so + s] && hipStreamWaitEvent(cs, c->slot_ev[so + s], 0) != hipSuccess)
    return DE_ERR_HIP;
  if (c->layer_ev_live[l] && hipStreamWaitEvent(cs, c->layer_ev[l], 0) != hipSuccess)
    return DE_ERR_HIP;
  if (hipMemcpyAsync(slot_block(c, l, s), host_block(c, l, e), (size_t)c->cfg.expert_bytes,
                     hipMemcpyHostToDevice, cs) != hipSuccess)
    return DE_ERR_HIP;
  if (hipEventRecord(c->slot_ev[so + s], cs) != hipSuccess) return DE_ERR_HIP;
  c->slot_ev_live[so + s] = 1;
  return DE_OK;
}

}  // namespace

hipEvent_t de::timing_event(de_cache* c) {
  if (!c->spare.empty()) {
    hipEvent_t e = c->spare.back();
    c->spare.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

namespace {

using de::timing_event;

// Waits for the end event of every recorded pair and returns the events to
// the pool; `sum` (may be NULL) receives the total elapsed microseconds.
int drain(de_cache* c, std::vector<std::pair<hipEvent_t, hipEvent_t>>& v, double* sum) {
  for (auto& p : v) {
    float ms = 0.f;
    if (hipEventSynchronize(p.second) != hipSuccess) return DE_ERR_HIP;
    if (sum != nullptr) {
      if (hipEventElapsedTime(&ms, p.first, p.second) != hipSuccess) return DE_ERR_HIP;
      *sum += 1e3 * ms;
    }
    c->spare.push_back(p.first);
    c->spare.push_back(p.second);
  }
  v.clear();
  return DE_OK;
}

void release_hip(de_cache* c) {
  if (fake(c)) return;
  if (c->prefetch_stream) hipStreamSynchronize(c->prefetch_stream);
  if (c->demand_stream) hipStreamSynchronize(c->demand_stream);
  for (auto& p : c->stalls) {
    hipEventSynchronize(p.second);
    hipEventDestroy(p.first);
    hipEventDestroy(p.second);
  }
  c->stalls.clear();
  for (auto& v : c->spans) {
    for (auto& p : v) {
      hipEventSynchronize(p.second);
      hipEventDestroy(p.first);
      hipEventDestroy(p.second);
    }
    v.clear();
  }
  if (c->span_open) hipEventDestroy(c->span_open);
  c->span_open = nullptr;
  for (hipEvent_t e : c->spare) hipEventDestroy(e);
  c->spare.clear();
  for (hipEvent_t e : c->slot_ev)
    if (e) hipEventDestroy(e);
  for (hipEvent_t e : c->layer_ev)
    if (e) hipEventDestroy(e);
  for (hipEvent_t e : c->stage_ev)
    if (e) hipEventDestroy(e);
  if (c->prefetch_stream) hipStreamDestroy(c->prefetch_stream);
  if (c->demand_stream) hipStreamDestroy(c->demand_stream);
  if (c->staging) hipHostFree(c->staging);
  if (c->readback) hipHostFree(c->readback);
}

void clear_state(de_cache* c) {
  std::fill(c->where.begin(), c->where.end(), -1);
  std::fill(c->held.begin(), c->held.end(), -1);
  std::fill(c->last_use.begin(), c->last_use.end(), 0);
  std::fill(c->prefetched.begin(), c->prefetched.end(), 0);
  std::fill(c->predicted.begin(), c->predicted.end(), 0);
  c->clock = 0;
  c->st = de_cache_counts{};
}

int check_layer(const de_cache* c, int layer) {
  return (c != nullptr && layer >= 0 && layer < c->L) ? DE_OK : DE_ERR_INVALID;
}

}  // namespace

extern "C" {

int de_cache_create(const de_cache_cfg* cfg, de_cache** out) {
  if (cfg == nullptr || out == nullptr) return DE_ERR_INVALID;
  *out = nullptr;
  const de_cache_cfg& g = *cfg;
  if (g.n_layers < 1 || g.n_layers > 4096 || g.n_experts < 1 || g.n_experts > 256)
    return DE_ERR_INVALID;
  if (g.n_slots < 1 || g.n_slots > g.n_experts) return DE_ERR_INVALID;
  if (g.expert_bytes < 16 || g.expert_bytes % 16) return DE_ERR_INVALID;
  if (g.slot_stride_bytes < g.expert_bytes || g.slot_stride_bytes % 256) return DE_ERR_INVALID;
  if (g.host_pool == nullptr || g.slot_pool == nullptr || g.slot_map == nullptr)
    return DE_ERR_INVALID;
  if ((reinterpret_cast<uintptr_t>(g.slot_pool) & 15u) != 0) return DE_ERR_INVALID;
  if (g.fake_copies != 0 && g.fake_copies != 1) return DE_ERR_INVALID;
  de_cache* c = new (std::nothrow) de_cache;
  if (c == nullptr) return DE_ERR_INVALID;
  c->cfg = g;
  c->L = g.n_layers;
  c->N = g.n_experts;
  c->S = g.n_slots;
  const size_t ls = (size_t)c->L * c->S, le = (size_t)c->L * c->N;
  c->where.assign(le, -1);
  c->held.assign(ls, -1);
  c->last_use.assign(ls, 0);
  c->prefetched.assign(ls, 0);
  c->predicted.assign(le, 0);
  c->stage_next.assign(c->L, 0);
  if (fake(c)) {
    std::fill(g.slot_map, g.slot_map + le, -1);
    *out = c;
    return DE_OK;
  }
  bool ok = hipStreamCreateWithFlags(&c->prefetch_stream, hipStreamNonBlocking) == hipSuccess &&
            hipStreamCreateWithFlags(&c->demand_stream, hipStreamNonBlocking) == hipSuccess;
  c->slot_ev.assign(ls, nullptr);
  c->slot_ev_live.assign(ls, 0);
  c->layer_ev.assign(c->L, nullptr);
  c->layer_ev_live.assign(c->L, 0);
  for (size_t i = 0; ok && i < ls; ++i)
    ok = hipEventCreateWithFlags(&c->slot_ev[i], hipEventDisableTiming) == hipSuccess;
  for (int l = 0; ok && l < c->L; ++l)
    ok = hipEventCreateWithFlags(&c->layer_ev[l], hipEventDisableTiming) == hipSuccess;
  c->stage_ev.assign((size_t)c->L * de::kStage, nullptr);
  c->stage_ev_live.assign((size_t)c->L * de::kStage, 0);
  for (size_t i = 0; ok && i < c->stage_ev.size(); ++i)
    ok = hipEventCreateWithFlags(&c->stage_ev[i], hipEventDisableTiming) == hipSuccess;
  ok = ok && hipHostMalloc(reinterpret_cast<void**>(&c->staging),
                           (size_t)c->L * de::kStage * c->N * sizeof(int32_t),
                           hipHostMallocDefault) == hipSuccess;
  ok = ok && hipHostMalloc(reinterpret_cast<void**>(&c->readback),
                           de::kReadbackInts * sizeof(int32_t), hipHostMallocDefault) == hipSuccess;
  ok = ok && hipMemset(g.slot_map, 0xFF, le * sizeof(int32_t)) == hipSuccess;
  if (!ok) {
    release_hip(c);
    delete c;
    return DE_ERR_HIP;
  }
  *out = c;
  return DE_OK;
}

int de_cache_destroy(de_cache* c) {
  if (c == nullptr) return DE_ERR_INVALID;
  release_hip(c);
  delete c;
  return DE_OK;
}

int de_cache_reset(de_cache* c) {
  if (c == nullptr) return DE_ERR_INVALID;
  if (!fake(c)) {
    if (hipStreamSynchronize(c->prefetch_stream) != hipSuccess ||
        hipStreamSynchronize(c->demand_stream) != hipSuccess)
      return DE_ERR_HIP;
    if (drain(c, c->stalls, nullptr) != DE_OK || drain(c, c->spans[0], nullptr) != DE_OK ||
        drain(c, c->spans[1], nullptr) != DE_OK)
      return DE_ERR_HIP;
  }
  clear_state(c);
  return DE_OK;
}

int de_cache_begin_block(de_cache* c) {
  if (c == nullptr) return DE_ERR_INVALID;
  for (auto& f : c->prefetched) {
    if (f) ++c->st.prefetch_wasted;
    f = 0;
  }
  std::fill(c->predicted.begin(), c->predicted.end(), 0);
  return DE_OK;
}

int de_cache_prefetch(de_cache* c, int layer, const int32_t* experts_host, int n) {
  if (check_layer(c, layer) != DE_OK || n < 0 || (n > 0 && experts_host == nullptr))
    return DE_ERR_INVALID;
  for (int i = 0; i < n; ++i)
    if (experts_host[i] < 0 || experts_host[i] >= c->N) return DE_ERR_INVALID;
  const size_t eo = (size_t)layer * c->N;
  for (int i = 0; i < n; ++i) c->predicted[eo + experts_host[i]] = 1;
  for (int i = 0; i < n; ++i) {
    const int e = experts_host[i];
    if (c->where[eo + e] >= 0) continue;
    const int s = pick_slot(c, layer, nullptr, false);
    if (s < 0) {
      ++c->st.prefetch_skipped;
      continue;
    }
    const int rc = load(c, layer, e, s, true);
    if (rc != DE_OK) return rc;
  }
  return DE_OK;
}

int de_cache_ensure(de_cache* c, int layer, const int32_t* needed_host, int n, int purpose,
                    hipStream_t compute) {
  if (check_layer(c, layer) != DE_OK || n < 1 || n > c->S || needed_host == nullptr)
    return DE_ERR_INVALID;
  if (purpose != DE_NEED_DRAFT && purpose != DE_NEED_VERIFY) return DE_ERR_INVALID;
  std::vector<uint8_t> need(c->N, 0);
  for (int i = 0; i < n; ++i) {
    const int e = needed_host[i];
    if (e < 0 || e >= c->N || need[e]) return DE_ERR_INVALID;
    need[e] = 1;
  }
  const size_t so = (size_t)layer * c->S, eo = (size_t)layer * c->N;
  int hits = 0;
  for (int i = 0; i < n; ++i) {
    const int e = needed_host[i];
    if (c->where[eo + e] >= 0) {
      ++hits;
      continue;
    }
    const int s = pick_slot(c, layer, need.data(), true);
    if (s < 0) return DE_ERR_NOT_RESIDENT;  // unreachable: n <= n_slots
    const int rc = load(c, layer, e, s, false);
    if (rc != DE_OK) return rc;
  }
  if (purpose == DE_NEED_DRAFT) {
    c->st.draft_needed += n;
    c->st.draft_hits += hits;
  } else {
    c->st.verify_needed += n;
    c->st.verify_hits += hits;
  }
  for (int i = 0; i < n; ++i) {
    const int s = c->where[eo + needed_host[i]];
    c->last_use[so + s] = ++c->clock;
    if (purpose == DE_NEED_VERIFY && c->prefetched[so + s]) {
      ++c->st.prefetch_used;
      c->prefetched[so + s] = 0;
    }
  }
  int32_t* row;
  size_t stage = 0;
  if (fake(c)) {
    row = c->cfg.slot_map + eo;
  } else {
    // A staging row is rewritten only after its previous upload has run.
    stage = (size_t)layer * de::kStage + c->stage_next[layer];
    c->stage_next[layer] = (c->stage_next[layer] + 1) % de::kStage;
    if (c->stage_ev_live[stage] && hipEventSynchronize(c->stage_ev[stage]) != hipSuccess)
      return DE_ERR_HIP;
    row = c->staging + stage * c->N;
  }
  std::fill(row, row + c->N, -1);
  for (int i = 0; i < n; ++i) row[needed_host[i]] = c->where[eo + needed_host[i]];
  if (fake(c)) return DE_OK;
  // The compute stream waits for every needed copy still running; each wait is
  // bracketed by timing events (the stall).
  for (int i = 0; i < n; ++i) {
    const int s = c->where[eo + needed_host[i]];
    if (!c->slot_ev_live[so + s]) continue;
    const hipError_t q = hipEventQuery(c->slot_ev[so + s]);
    if (q == hipSuccess) continue;
    if (q != hipErrorNotReady) return DE_ERR_HIP;
    hipEvent_t a = timing_event(c), b = timing_event(c);
    if (a == nullptr || b == nullptr) return DE_ERR_HIP;
    if (hipEventRecord(a, compute) != hipSuccess ||
        hipStreamWaitEvent(compute, c->slot_ev[so + s], 0) != hipSuccess ||
        hipEventRecord(b, compute) != hipSuccess)
      return DE_ERR_HIP;
    c->stalls.emplace_back(a, b);
  }
  if (hipMemcpyAsync(c->cfg.slot_map + eo, row, (size_t)c->N * sizeof(int32_t),
                     hipMemcpyHostToDevice, compute) != hipSuccess ||
      hipEventRecord(c->stage_ev[stage], compute) != hipSuccess)
    return DE_ERR_HIP;
  c->stage_ev_live[stage] = 1;
  return DE_OK;
}

int de_cache_release(de_cache* c, int layer, hipStream_t compute) {
  if (check_layer(c, layer) != DE_OK) return DE_ERR_INVALID;
  if (fake(c)) return DE_OK;
  if (hipEventRecord(c->layer_ev[layer], compute) != hipSuccess) return DE_ERR_HIP;
  c->layer_ev_live[layer] = 1;
  return DE_OK;
}

int de_cache_table(const de_cache* c, int layer, de_expert_table* table) {
  if (check_layer(c, layer) != DE_OK || table == nullptr) return DE_ERR_INVALID;
  table->base = slot_block(c, layer, 0);
  table->slot_stride_bytes = c->cfg.slot_stride_bytes;
  table->slot_of_expert = c->cfg.slot_map + (size_t)layer * c->N;
  table->n_slots = c->S;
  return DE_OK;
}

int de_cache_stats(de_cache* c, de_cache_counts* stats) {
  if (c == nullptr || stats == nullptr) return DE_ERR_INVALID;
  if (!fake(c)) {
    c->st.draft_layers += (int64_t)c->spans[0].size();
    c->st.verify_layers += (int64_t)c->spans[1].size();
    if (drain(c, c->stalls, &c->st.stall_us) != DE_OK ||
        drain(c, c->spans[0], &c->st.draft_layer_us) != DE_OK ||
        drain(c, c->spans[1], &c->st.verify_layer_us) != DE_OK)
      return DE_ERR_HIP;
  }
  *stats = c->st;
  return DE_OK;
}

int de_cache_slots(const de_cache* c, int layer, int32_t* slot_of_expert_host) {
  if (check_layer(c, layer) != DE_OK || slot_of_expert_host == nullptr) return DE_ERR_INVALID;
  std::copy(c->where.begin() + (size_t)layer * c->N, c->where.begin() + (size_t)(layer + 1) * c->N,
            slot_of_expert_host);
  return DE_OK;
}

}  // extern "C"
