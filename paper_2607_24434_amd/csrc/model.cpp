// The stacked model of the decoding step and Algorithm 1 on top of it: the
// drafter generates K tokens one position at a time (Eq. 5 in every MoE
// layer), the target scores the K+1-position block in one pass (Eq. 4), and
// the greedy rule accepts the target-consistent prefix.  Every stage is one
// of the layer calls, enqueued on the caller's stream; the tokens never leave
// device memory, so a whole step runs without a host synchronisation.
#include "../../include/draftexpert.h"
#include "draft_persistent.h"

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <utility>
#include <vector>

namespace de {
int check_table(const de_moe_desc& d, const de_expert_table* t);
int layer_after_route(const de_moe_desc& d, int T, const float* x, const de_expert_table* routed,
                      const int32_t* idx, const float* gate, int ucols, const void* shared_w,
                      const void* draft_w, float gamma, float* y, const de_epilogue* epi,
                      bool dense_on, bool combine_on, int32_t* n_union, void* ws,
                      size_t ws_bytes, hipStream_t stream);
int32_t* cache_readback(de_cache* c);
int cache_slots_per_layer(const de_cache* c);
int cache_experts(const de_cache* c);
int cache_layers(const de_cache* c);
bool cache_resident(const de_cache* c, int layer, int e);
int cache_span(de_cache* c, bool end, int purpose, hipStream_t s);
int draft_layer_chain(const de_moe_desc* d, int T, const float* x, const float* w_router,
                      const float* bias, const de_expert_table* routed, const void* shared_w,
                      const void* draft_w, float gamma, int r, float* y, int32_t* pred_idx,
                      float* pred_gate, const de_epilogue* epi, void* ws, size_t ws_bytes,
                      hipStream_t stream, bool logits_ready, const float* next_router);
int accept_len_embed(int K, int V, const float* target_logits, const int32_t* draft_tokens,
                     int32_t* target_argmax, int32_t* out, void* ws, size_t ws_bytes,
                     const void* emb, int H, float* h, float* normed, float eps,
                     hipStream_t stream);
int verify_layer_chain(const de_moe_desc* d, int T, const float* x, const float* w_router,
                       const float* bias, const de_expert_table* routed, const void* shared_w,
                       float* y, int32_t* topk_idx, float* topk_gate, int32_t* n_union,
                       int32_t* union_ids, int32_t* offsets, int32_t* tok_list, float* gate_list,
                       int32_t* pair_pos, const de_epilogue* epi, void* ws, size_t ws_bytes,
                       hipStream_t stream, bool logits_ready, const float* next_router);
int dense_swiglu_chain(int T, int H, int I, int wdtype, const float* x, const void* w, float* y,
                       const de_epilogue* epi, void* ws, size_t ws_bytes, hipStream_t stream,
                       const de_moe_desc* next_desc, void* next_ws, const float* next_router);
bool combine_route_fits(int H);
int32_t* layer_status_word(void* ws);
int take_status(int32_t* word, hipStream_t stream);
PDLayer pd_layer(const de_layer_weights& w);
int draft_persistent_run(const de_moe_desc& d, int n, const PDLayer* layers, const float* x_in,
                         const float* h_in, bool z_ready, float* y_out, float* normed_out,
                         int32_t* pred_idx, float* pred_gate, float eps, void* ws,
                         size_t ws_bytes, hipStream_t s);
}

namespace {

constexpr int kMaxLayers = 4096;

size_t up256(size_t v) { return (v + 255) & ~size_t(255); }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Scratch of the model calls for blocks of up to T positions.  The two
// regions holding control words come first, at offsets that do not depend on
// T: the acceptance scratch, sized for the largest block (its counters sit at
// its start for every row count), then the layer scratch (its counters sit at
// its start for every block length).  One zero fill of a fresh allocation
// therefore serves calls with any block length.
constexpr int kMaxBlock = 64;

struct ModelLayout {
  size_t accept_ws, accept_bytes;
  size_t layer_ws, layer_bytes;
  size_t dense_ws, dense_bytes;
  size_t misc;                // int32 [2]: acceptance output of the argmax-only calls
  size_t ridx, rgate;         // top-k lists of the cached step's routing [64, k]
  size_t h, h2, n0, n1, logits;  // residual stream (two buffers), two normed buffers, logits
  size_t uhat, tctl;          // truncation: predicted verifier set [L, words], decision [5]
  size_t zt, zd, logits2;     // distillation: router logits of both passes [L, T, N], draft logits
  size_t total;
};

ModelLayout model_layout(const de_model& m, int T) {
  ModelLayout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t r = o;
    o += up256(bytes);
    return r;
  };
  const size_t H = (size_t)m.moe.hidden;
  L.accept_bytes = de_accept_workspace_bytes(kMaxBlock - 1, m.vocab);
  // At least the control area: its status word also serves the embedding.
  L.layer_bytes = std::max<size_t>(de_workspace_bytes(&m.moe, T), 4096);
  L.dense_bytes = m.dense_inter > 0 ? de_dense_workspace_bytes(T, (int)H, m.dense_inter) : 0;
  L.accept_ws = take(L.accept_bytes);
  L.layer_ws = take(L.layer_bytes);
  L.dense_ws = take(L.dense_bytes);
  L.misc = take(8);
  L.ridx = take((size_t)kMaxBlock * m.moe.top_k * 4);
  L.rgate = take((size_t)kMaxBlock * m.moe.top_k * 4);
  L.h = take((size_t)T * H * 4);
  L.h2 = take((size_t)T * H * 4);
  L.n0 = take((size_t)T * H * 4);
  L.n1 = take((size_t)T * H * 4);
  L.logits = take((size_t)T * m.vocab * 4);
  L.uhat = take((size_t)m.n_layers * ((m.moe.n_experts + 63) / 64) * 8);
  L.tctl = take(5 * 4);
  L.zt = take((size_t)m.n_layers * T * m.moe.n_experts * 4);
  L.zd = take((size_t)m.n_layers * T * m.moe.n_experts * 4);
  L.logits2 = take((size_t)T * m.vocab * 4);
  L.total = o;
  return L;
}

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

int check_block(const de_model& m, int T, const void* ws, size_t ws_bytes) {
  if (T < 1 || T > kMaxBlock) return DE_ERR_INVALID;
  if (ws == nullptr || (reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return DE_ERR_WORKSPACE;
  if (ws_bytes < model_layout(m, T).total) return DE_ERR_WORKSPACE;
  return DE_OK;
}

// Routed experts of every draft layer.
int draft_r(const de_model& m) { return m.draft_topr > 0 ? m.draft_topr : 1; }

// Where the argmax of a forward goes.  amax NULL skips the acceptance launch.
struct ArgmaxOut {
  int32_t* amax;          // [T]
  int32_t* out;           // [2]: (n, bonus) against `drafts`
  const int32_t* drafts;  // [T-1] (NULL when T is 1)
  // The acceptance launch also gathers the bonus token's embedding into the
  // residual and normed buffers a forward starts from, so that the next
  // position's forward (called with `embedded`) skips its own gather.
  bool embed_next = false;
};

// MoE layer l with its routed experts behind the cache.  The routing runs
// first and its lists come back to the host (one synchronisation).  Draft
// (T = 1): the top-1 expert is requested, the top-k prefetched (or, with
// `deferred`, appended there for the caller to prefetch later), then the
// grouped part runs over the top-1 column.  Verify: the union's members are
// requested in chunks of at most n_slots (resident or in flight first, then
// the rest, each in ascending id); every chunk runs gate/up and down over its
// members, the first also over the shared path, the last also the combine.
int cached_layer(const de_model& m, de_cache* c, int l, int T, bool draft, const float* x,
                 const float* h_in, float* h_out, float* normed_out, int32_t* n_union,
                 int32_t* pred_out, void* ws, const ModelLayout& L, hipStream_t s,
                 std::vector<int32_t>* deferred) {
  const de_layer_weights& w = m.layers[l];
  const int k = m.moe.top_k, N = m.moe.n_experts;
  const int purpose = draft ? DE_NEED_DRAFT : DE_NEED_VERIFY;
  void* lws = at<void>(ws, L.layer_ws);
  int32_t* ridx = at<int32_t>(ws, L.ridx);
  float* rgate = at<float>(ws, L.rgate);
  int rc = de::cache_span(c, false, purpose, s);
  if (rc != DE_OK) return rc;
  rc = de_route_topk(&m.moe, T, x, w.w_router, w.bias, ridx, rgate, lws, L.layer_bytes, s);
  if (rc != DE_OK) return rc;
  if (pred_out != nullptr &&
      hipMemcpyAsync(pred_out, ridx, (size_t)T * k * 4, hipMemcpyDeviceToDevice, s) != hipSuccess)
    return DE_ERR_HIP;
  int32_t* hb = de::cache_readback(c);
  if (hipMemcpyAsync(hb, ridx, (size_t)T * k * 4, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return DE_ERR_HIP;
  for (int i = 0; i < T * k; ++i)
    if (hb[i] < 0 || hb[i] >= N) return DE_ERR_INVALID;
  de_expert_table tab;
  if ((rc = de_cache_table(c, l, &tab)) != DE_OK) return rc;
  const de_epilogue epi{h_in, normed_out, m.eps};
  if (draft) {
    // The drafter's own experts: its r leading ones.
    const int r = draft_r(m);
    if ((rc = de_cache_ensure(c, l, hb, r, DE_NEED_DRAFT, s)) != DE_OK) return rc;
    if (deferred != nullptr)
      deferred->insert(deferred->end(), hb, hb + k);
    else if ((rc = de_cache_prefetch(c, l, hb, k)) != DE_OK)
      return rc;
    rc = de::layer_after_route(m.moe, 1, x, &tab, ridx, rgate, r, w.shared_w, w.draft_w, w.gamma,
                               h_out, &epi, true, true, nullptr, lws, L.layer_bytes, s);
    if (rc != DE_OK) return rc;
    if ((rc = de_cache_release(c, l, s)) != DE_OK) return rc;
    return de::cache_span(c, true, purpose, s);
  }
  std::vector<uint8_t> in_union(N, 0);
  for (int i = 0; i < T * k; ++i) in_union[hb[i]] = 1;
  std::vector<int32_t> order;
  for (int pass = 0; pass < 2; ++pass)
    for (int e = 0; e < N; ++e)
      if (in_union[e] && de::cache_resident(c, l, e) == (pass == 0)) order.push_back(e);
  const int S = de::cache_slots_per_layer(c);
  const int n = (int)order.size();
  const int chunks = (n + S - 1) / S;
  for (int ci = 0; ci < chunks; ++ci) {
    const int lo = ci * S, cnt = std::min(S, n - lo);
    if ((rc = de_cache_ensure(c, l, order.data() + lo, cnt, DE_NEED_VERIFY, s)) != DE_OK)
      return rc;
    rc = de::layer_after_route(m.moe, T, x, &tab, ridx, rgate, k, w.shared_w, nullptr, 0.f, h_out,
                               &epi, ci == 0, ci == chunks - 1, n_union ? n_union + l : nullptr,
                               lws, L.layer_bytes, s);
    if (rc != DE_OK) return rc;
    // The next chunk's copies may evict this chunk's members: they wait for
    // the launches just enqueued.
    if ((rc = de_cache_release(c, l, s)) != DE_OK) return rc;
  }
  return de::cache_span(c, true, purpose, s);
}

// Per-layer outputs a forward may copy out after each MoE layer: its router
// logits [L, T, N], and (target mode) its residual target [L, T, H].
struct Capture {
  float* z = nullptr;
  float* m = nullptr;
};

// Logits of T positions through the whole stack; the last MoE layer's fused
// epilogue leaves RMSNorm(h) in the normed buffer, which the LM head reads.
// With a cache the routed experts come through it (cached_layer).
int forward(const de_model& m, int T, const int32_t* tokens, int mode, float* logits,
            const ArgmaxOut& am, int32_t* n_union, int32_t* pred_idx, size_t pred_stride,
            void* ws, const ModelLayout& L, hipStream_t s, de_cache* cache = nullptr,
            std::vector<int32_t>* deferred = nullptr, const Capture& cap = Capture{},
            bool embedded = false) {
  const int H = m.moe.hidden;
  // The residual stream ping-pongs between two buffers: a layer reads h and
  // writes h + F(RMSNorm(h)) to the other one.  In the chained launches every
  // block of a position re-reads the residual row while one of them writes the
  // output row, so the two must never be the same memory.
  float* h = at<float>(ws, L.h);
  float* hnext = at<float>(ws, L.h2);
  float* ncur = at<float>(ws, L.n0);
  float* nnext = at<float>(ws, L.n1);
  void* lws = at<void>(ws, L.layer_ws);
  // A single position whose token the previous acceptance launch chose finds
  // its embedding and its RMSNorm already in h and ncur.
  int rc = DE_OK;
  if (!(embedded && T == 1) &&
      (rc = de_embed_gather(T, H, m.vocab, tokens, m.emb, h, ncur, m.eps,
                            de::layer_status_word(lws), s)) != DE_OK)
    return rc;
  // Resident layers are chained: each layer's combine (and the dense layer's)
  // also computes the next layer's router logits, so no MoE layer launches its
  // own routing.  (Not with per-layer captures, which read each layer's own
  // logits.)
  const bool chain = cache == nullptr && cap.z == nullptr && de::combine_route_fits(H);
  const bool dense_chained = chain && m.dense_inter > 0 && m.n_layers > 0;
  if (m.dense_inter > 0) {
    const de_epilogue epi{h, nnext, m.eps};
    rc = de::dense_swiglu_chain(T, H, m.dense_inter, m.dense_wdtype, ncur, m.dense_w, hnext, &epi,
                                at<void>(ws, L.dense_ws), L.dense_bytes, s, &m.moe, lws,
                                dense_chained ? m.layers[0].w_router : nullptr);
    if (rc != DE_OK) return rc;
    std::swap(ncur, nnext);
    std::swap(h, hnext);
  }
  // A draft position through resident layers: every MoE layer in one
  // persistent launch when the shapes allow it.
  bool done = false;
  if (mode == DE_DRAFT && chain && T == 1 && draft_r(m) == 1 && m.n_layers > 0 &&
      (pred_idx == nullptr || pred_stride == (size_t)m.moe.top_k)) {
    std::vector<de::PDLayer> pl(m.n_layers);
    for (int l = 0; l < m.n_layers; ++l) pl[l] = de::pd_layer(m.layers[l]);
    rc = de::draft_persistent_run(m.moe, m.n_layers, pl.data(), ncur, h, dense_chained, hnext,
                                  nnext, pred_idx, nullptr, m.eps, lws, L.layer_bytes, s);
    if (rc == DE_OK) {
      std::swap(ncur, nnext);
      std::swap(h, hnext);
      done = true;
    } else if (rc != de::kPDNotApplicable) {
      return rc;
    }
  }
  for (int l = 0; l < m.n_layers && !done; ++l) {
    const de_layer_weights& w = m.layers[l];
    const de_epilogue epi{h, nnext, m.eps};
    const bool ready = chain && (l > 0 || dense_chained);
    const float* next = chain && l + 1 < m.n_layers ? m.layers[l + 1].w_router : nullptr;
    if (cache != nullptr) {
      rc = cached_layer(m, cache, l, T, mode == DE_DRAFT, ncur, h, hnext, nnext,
                        mode == DE_TARGET ? n_union : nullptr,
                        pred_idx ? pred_idx + l * pred_stride : nullptr, ws, L, s, deferred);
    } else if (mode == DE_TARGET) {
      rc = de::verify_layer_chain(&m.moe, T, ncur, w.w_router, w.bias, &w.routed, w.shared_w,
                                  hnext, nullptr, nullptr, n_union ? n_union + l : nullptr, nullptr,
                                  nullptr, nullptr, nullptr, nullptr, &epi, lws, L.layer_bytes, s,
                                  ready, next);
    } else {
      rc = de::draft_layer_chain(&m.moe, T, ncur, w.w_router, w.bias, &w.routed, w.shared_w,
                                 w.draft_w, w.gamma, draft_r(m), hnext,
                                 pred_idx ? pred_idx + l * pred_stride : nullptr, nullptr, &epi,
                                 lws, L.layer_bytes, s, ready, next);
    }
    if (rc != DE_OK) return rc;
    if (cap.z != nullptr &&
        (rc = de_layer_router_logits(&m.moe, T, lws, L.layer_bytes,
                                     cap.z + (size_t)l * T * m.moe.n_experts, s)) != DE_OK)
      return rc;
    if (cap.m != nullptr && mode == DE_TARGET &&
        (rc = de_residual_target(&m.moe, T, lws, L.layer_bytes, cap.m + (size_t)l * T * H, s)) !=
            DE_OK)
      return rc;
    std::swap(ncur, nnext);
    std::swap(h, hnext);
  }
  rc = de_lm_head(T, H, m.vocab, ncur, m.lm_head, logits, s);
  if (rc != DE_OK || am.amax == nullptr) return rc;
  const bool emb = am.embed_next;
  return de::accept_len_embed(T - 1, m.vocab, logits, am.drafts, am.amax, am.out,
                              at<void>(ws, L.accept_ws), L.accept_bytes, emb ? m.emb : nullptr, H,
                              emb ? at<float>(ws, L.h) : nullptr,
                              emb ? at<float>(ws, L.n0) : nullptr, m.eps, s);
}

}  // namespace

extern "C" {

int de_check_model(const de_model* m) {
  if (m == nullptr) return DE_ERR_INVALID;
  int rc = de_check_desc(&m->moe);
  if (rc != DE_OK) return rc;
  const de_moe_desc& d = m->moe;
  if (m->n_layers < 0 || m->n_layers > kMaxLayers) return DE_ERR_INVALID;
  if (m->vocab < 1 || m->vocab > (1 << 24)) return DE_ERR_INVALID;
  if (!(m->eps >= 0.f) || !std::isfinite(m->eps)) return DE_ERR_INVALID;
  if (d.hidden % 8) return DE_ERR_INVALID;  // bf16 embedding and LM head rows
  if (m->emb == nullptr || m->lm_head == nullptr || !aligned16(m->lm_head)) return DE_ERR_INVALID;
  if (m->dense_inter < 0) return DE_ERR_INVALID;
  if (m->dense_inter > 0) {
    if (m->dense_wdtype != DE_F32 && m->dense_wdtype != DE_BF16) return DE_ERR_UNSUPPORTED;
    const int al = m->dense_wdtype == DE_BF16 ? 8 : 4;
    if (m->dense_inter % al || m->dense_inter > (1 << 17)) return DE_ERR_INVALID;
    if (m->dense_w == nullptr || !aligned16(m->dense_w)) return DE_ERR_INVALID;
  }
  if (m->n_layers > 0 && m->layers == nullptr) return DE_ERR_INVALID;
  if (m->draft_topr < 0 || m->draft_topr > d.top_k) return DE_ERR_INVALID;
  for (int l = 0; l < m->n_layers; ++l) {
    const de_layer_weights& w = m->layers[l];
    if (w.w_router == nullptr || !aligned16(w.w_router) || d.hidden % 4) return DE_ERR_INVALID;
    if (d.shared_inter > 0 && (w.shared_w == nullptr || !aligned16(w.shared_w)))
      return DE_ERR_INVALID;
    if (w.draft_w != nullptr && !aligned16(w.draft_w)) return DE_ERR_INVALID;
    if (!std::isfinite(w.gamma)) return DE_ERR_INVALID;
    if ((rc = de::check_table(d, &w.routed)) != DE_OK) return rc;
  }
  return DE_OK;
}

size_t de_model_workspace_bytes(const de_model* m, int T) {
  if (de_check_model(m) != DE_OK || T < 1 || T > kMaxBlock) return 0;
  return model_layout(*m, T).total;
}

int de_model_status(const de_model* m, void* ws, size_t ws_bytes, hipStream_t stream) {
  int rc = de_check_model(m);
  if (rc != DE_OK) return rc;
  if ((rc = check_block(*m, 1, ws, ws_bytes)) != DE_OK) return rc;
  // The layer scratch sits at an offset that does not depend on the block
  // length, so its status word is found with the one-position layout.
  return de::take_status(de::layer_status_word(at<void>(ws, model_layout(*m, 1).layer_ws)), stream);
}

int de_model_forward(const de_model* m, int T, const int32_t* tokens, int mode, float* logits,
                     int32_t* argmax, int32_t* n_union, void* ws, size_t ws_bytes,
                     hipStream_t stream) {
  int rc = de_check_model(m);
  if (rc != DE_OK) return rc;
  if (mode != DE_TARGET && mode != DE_DRAFT) return DE_ERR_INVALID;
  if (tokens == nullptr || logits == nullptr) return DE_ERR_INVALID;
  if (n_union != nullptr && mode != DE_TARGET) return DE_ERR_INVALID;
  if ((rc = check_block(*m, T, ws, ws_bytes)) != DE_OK) return rc;
  const ModelLayout L = model_layout(*m, T);
  // The acceptance launch also yields (n, bonus) against tokens[1..T-1]; the
  // pair goes to scratch.
  const ArgmaxOut am{argmax, at<int32_t>(ws, L.misc), T > 1 ? tokens + 1 : nullptr};
  return forward(*m, T, tokens, mode, logits, am, n_union, nullptr, 0, ws, L, stream);
}

int de_spec_step(const de_model* m, int K, int32_t* block, int32_t* target_argmax, int32_t* out,
                 int32_t* n_union, int32_t* pred_idx, void* ws, size_t ws_bytes,
                 hipStream_t stream) {
  int rc = de_check_model(m);
  if (rc != DE_OK) return rc;
  if (K < 0 || K > 63 || block == nullptr || target_argmax == nullptr || out == nullptr)
    return DE_ERR_INVALID;
  if ((rc = check_block(*m, K + 1, ws, ws_bytes)) != DE_OK) return rc;
  const ModelLayout L = model_layout(*m, K + 1);
  float* logits = at<float>(ws, L.logits);
  const size_t k = (size_t)m->moe.top_k;
  // Draft loop: position i's token is block[i]; its drafter argmax is block[i+1].
  for (int i = 0; i < K; ++i) {
    const ArgmaxOut am{block + i + 1, at<int32_t>(ws, L.misc), nullptr, i + 1 < K};
    rc = forward(*m, 1, block + i, DE_DRAFT, logits, am, nullptr,
                 pred_idx ? pred_idx + (size_t)i * m->n_layers * k : nullptr, k, ws, L, stream,
                 nullptr, nullptr, Capture{}, i > 0);
    if (rc != DE_OK) return rc;
  }
  // Verify the block [c, d_1..d_K] and accept.
  const ArgmaxOut am{target_argmax, out, K > 0 ? block + 1 : nullptr};
  return forward(*m, K + 1, block, DE_TARGET, logits, am, n_union, nullptr, 0, ws, L, stream);
}

int de_greedy_decode(const de_model* m, int n_steps, int32_t* tokens, void* ws, size_t ws_bytes,
                     hipStream_t stream) {
  int rc = de_check_model(m);
  if (rc != DE_OK) return rc;
  if (n_steps < 0 || tokens == nullptr) return DE_ERR_INVALID;
  if ((rc = check_block(*m, 1, ws, ws_bytes)) != DE_OK) return rc;
  const ModelLayout L = model_layout(*m, 1);
  float* logits = at<float>(ws, L.logits);
  for (int i = 0; i < n_steps; ++i) {
    const ArgmaxOut am{tokens + i + 1, at<int32_t>(ws, L.misc), nullptr, i + 1 < n_steps};
    rc = forward(*m, 1, tokens + i, DE_TARGET, logits, am, nullptr, nullptr, 0, ws, L, stream,
                 nullptr, nullptr, Capture{}, i > 0);
    if (rc != DE_OK) return rc;
  }
  return DE_OK;
}

int de_spec_step_cached(const de_model* m, de_cache* cache, int K, int32_t* block,
                        int32_t* target_argmax, int32_t* out, int32_t* n_union, int32_t* pred_idx,
                        void* ws, size_t ws_bytes, hipStream_t stream) {
  int rc = de_check_model(m);
  if (rc != DE_OK) return rc;
  if (cache == nullptr || de::cache_layers(cache) != m->n_layers ||
      de::cache_experts(cache) != m->moe.n_experts)
    return DE_ERR_INVALID;
  for (int l = 0; l < m->n_layers; ++l) {
    de_expert_table tab;
    if (de_cache_table(cache, l, &tab) != DE_OK || de::check_table(m->moe, &tab) != DE_OK)
      return DE_ERR_INVALID;
  }
  if (K < 0 || K > 63 || block == nullptr || target_argmax == nullptr || out == nullptr)
    return DE_ERR_INVALID;
  if ((rc = check_block(*m, K + 1, ws, ws_bytes)) != DE_OK) return rc;
  const ModelLayout L = model_layout(*m, K + 1);
  float* logits = at<float>(ws, L.logits);
  const size_t k = (size_t)m->moe.top_k;
  if ((rc = de_cache_begin_block(cache)) != DE_OK) return rc;
  for (int i = 0; i < K; ++i) {
    const ArgmaxOut am{block + i + 1, at<int32_t>(ws, L.misc), nullptr};
    rc = forward(*m, 1, block + i, DE_DRAFT, logits, am, nullptr,
                 pred_idx ? pred_idx + (size_t)i * m->n_layers * k : nullptr, k, ws, L, stream,
                 cache);
    if (rc != DE_OK) return rc;
  }
  const ArgmaxOut am{target_argmax, out, K > 0 ? block + 1 : nullptr};
  return forward(*m, K + 1, block, DE_TARGET, logits, am, n_union, nullptr, 0, ws, L, stream,
                 cache);
}

int de_spec_step_trunc(const de_model* m, de_cache* cache, int k_max, const de_trunc_cfg* cfg,
                       int32_t* block, int32_t* target_argmax, int32_t* out, int32_t* n_drafted,
                       int32_t* n_union, int32_t* pred_idx, float* q, int32_t* trace, void* ws,
                       size_t ws_bytes, hipStream_t stream) {
  int rc = de_check_model(m);
  if (rc != DE_OK) return rc;
  if (cfg == nullptr || cfg->tau != cfg->tau || cfg->budget < DE_BUDGET_CACHE || cfg->slots < 0)
    return DE_ERR_INVALID;
  if (k_max < 0 || k_max > 63 || block == nullptr || target_argmax == nullptr ||
      out == nullptr || n_drafted == nullptr || pred_idx == nullptr || q == nullptr)
    return DE_ERR_INVALID;
  if (m->moe.n_experts > 256) return DE_ERR_UNSUPPORTED;
  int slots = cfg->slots;
  if (cache != nullptr) {
    if (de::cache_layers(cache) != m->n_layers || de::cache_experts(cache) != m->moe.n_experts)
      return DE_ERR_INVALID;
    for (int l = 0; l < m->n_layers; ++l) {
      de_expert_table tab;
      if (de_cache_table(cache, l, &tab) != DE_OK || de::check_table(m->moe, &tab) != DE_OK)
        return DE_ERR_INVALID;
    }
    if (slots == 0) slots = de::cache_slots_per_layer(cache);
  }
  if ((rc = check_block(*m, k_max + 1, ws, ws_bytes)) != DE_OK) return rc;
  const ModelLayout L = model_layout(*m, k_max + 1);
  float* logits = at<float>(ws, L.logits);
  int32_t* tctl = at<int32_t>(ws, L.tctl);
  const int k = m->moe.top_k, NL = m->n_layers;
  if (cache != nullptr && (rc = de_cache_begin_block(cache)) != DE_OK) return rc;
  int kept = 0;
  std::vector<int32_t> deferred;
  for (int i = 0; i < k_max; ++i) {
    int32_t* pred = pred_idx + (size_t)i * NL * k;
    deferred.clear();
    const ArgmaxOut am{block + i + 1, at<int32_t>(ws, L.misc), nullptr};
    rc = forward(*m, 1, block + i, DE_DRAFT, logits, am, nullptr, pred, (size_t)k, ws, L, stream,
                 cache, cache != nullptr ? &deferred : nullptr);
    if (rc != DE_OK) return rc;
    if ((rc = de_confidence(1, m->vocab, logits, q + i, stream)) != DE_OK) return rc;
    // A stack without MoE layers predicts nothing: every token is kept.
    int32_t dec[5] = {0, 0, 0, 0, 0};
    if (NL > 0) {
      rc = de_expansion(NL, k, m->moe.n_experts, pred, at<uint64_t>(ws, L.uhat), i == 0, q + i,
                        cfg->tau, cfg->budget, slots, tctl, stream);
      if (rc != DE_OK) return rc;
      if (trace != nullptr && hipMemcpyAsync(trace + 4 * i, tctl, 16, hipMemcpyDeviceToDevice,
                                             stream) != hipSuccess)
        return DE_ERR_HIP;
      if (hipMemcpyAsync(dec, tctl, sizeof(dec), hipMemcpyDeviceToHost, stream) != hipSuccess ||
          hipStreamSynchronize(stream) != hipSuccess)
        return DE_ERR_HIP;
      if (dec[4] != 0) return DE_ERR_INVALID;
    }
    if (dec[1] != 0) break;
    ++kept;
    if (cache != nullptr && cfg->prefetch != 0) {
      for (int l = 0; l < NL; ++l)
        if ((rc = de_cache_prefetch(cache, l, deferred.data() + (size_t)l * k, k)) != DE_OK)
          return rc;
    }
  }
  *n_drafted = kept;
  const ArgmaxOut am{target_argmax, out, kept > 0 ? block + 1 : nullptr};
  return forward(*m, kept + 1, block, DE_TARGET, logits, am, n_union, nullptr, 0, ws, L, stream,
                 cache);
}

int de_distill_signals(const de_model* m, int T, const int32_t* tokens, float tau,
                       float* m_star, float* router_kl, float* logit_kl, float* token_ce,
                       void* ws, size_t ws_bytes, hipStream_t stream) {
  int rc = de_check_model(m);
  if (rc != DE_OK) return rc;
  if (tokens == nullptr || !(tau > 0.f) || !std::isfinite(tau)) return DE_ERR_INVALID;
  if (m->n_layers > 0 && (m_star == nullptr) != (router_kl == nullptr)) return DE_ERR_INVALID;
  if ((logit_kl == nullptr) != (token_ce == nullptr)) return DE_ERR_INVALID;
  if ((rc = check_block(*m, T, ws, ws_bytes)) != DE_OK) return rc;
  const ModelLayout L = model_layout(*m, T);
  const int N = m->moe.n_experts, NL = m->n_layers;
  float* zt = at<float>(ws, L.zt);
  float* zd = at<float>(ws, L.zd);
  float* lt = at<float>(ws, L.logits);
  float* ld = at<float>(ws, L.logits2);
  const ArgmaxOut none{nullptr, nullptr, nullptr};
  // Teacher-forced passes over the same positions: the target (capturing each
  // layer's router logits and residual target), then the drafter.
  Capture ct;
  ct.z = zt;
  ct.m = m_star;
  rc = forward(*m, T, tokens, DE_TARGET, lt, none, nullptr, nullptr, 0, ws, L, stream, nullptr,
               nullptr, ct);
  if (rc != DE_OK) return rc;
  Capture cd;
  cd.z = zd;
  rc = forward(*m, T, tokens, DE_DRAFT, ld, none, nullptr, nullptr, 0, ws, L, stream, nullptr,
               nullptr, cd);
  if (rc != DE_OK) return rc;
  const bool sig = m->moe.score_func == DE_SIGMOID;
  if (router_kl != nullptr) {
    for (int l = 0; l < NL; ++l) {
      const size_t o = (size_t)l * T * N;
      rc = de_row_kl(T, N, zt + o, N, zd + o, N, sig ? nullptr : m->layers[l].bias, sig ? 1 : 0,
                     1.f, router_kl + (size_t)l * T, nullptr, stream);
      if (rc != DE_OK) return rc;
    }
  }
  if (logit_kl != nullptr) {
    rc = de_row_kl(T, m->vocab, lt, m->vocab, ld, m->vocab, nullptr, 0, tau, logit_kl, token_ce,
                   stream);
    if (rc != DE_OK) return rc;
  }
  return DE_OK;
}

}  // extern "C"
