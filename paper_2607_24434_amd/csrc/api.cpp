// C ABI of the draft/verify hot path: argument checks (host only, before any
// HIP call), scratch layout, and the launch sequence of each layer call.
#include "../../include/draftexpert.h"
#include "de_common.h"
#include "draft_persistent.h"
#include "verify_fused.h"

#include <atomic>
#include <cmath>
#include <cstdlib>
#include <cstring>

namespace de {

const DevInfo& dev_info() {
  static DevInfo info[64];
  static bool ready[64] = {false};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (!ready[dev]) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus < 1)
      cus = 256;
    info[dev].device = dev;
    info[dev].num_cus = cus;
    ready[dev] = true;
  }
  return info[dev];
}

int draft_layer_chain(const de_moe_desc* d, int T, const float* x, const float* w_router,
                      const float* bias, const de_expert_table* routed, const void* shared_w,
                      const void* draft_w, float gamma, int r, float* y, int32_t* pred_idx,
                      float* pred_gate, const de_epilogue* epi, void* ws, size_t ws_bytes,
                      hipStream_t stream, bool logits_ready, const float* next_router);
int verify_layer_chain(const de_moe_desc* d, int T, const float* x, const float* w_router,
                       const float* bias, const de_expert_table* routed, const void* shared_w,
                       float* y, int32_t* topk_idx, float* topk_gate, int32_t* n_union,
                       int32_t* union_ids, int32_t* offsets, int32_t* tok_list, float* gate_list,
                       int32_t* pair_pos, const de_epilogue* epi, void* ws, size_t ws_bytes,
                       hipStream_t stream, bool logits_ready, const float* next_router);
int dense_swiglu_chain(int T, int H, int I, int wdtype, const float* x, const void* w, float* y,
                       const de_epilogue* epi, void* ws, size_t ws_bytes, hipStream_t stream,
                       const de_moe_desc* next_desc, void* next_ws, const float* next_router);

// Bytes of a [rows, cols] weight matrix and of a [G|U|D] expert block.
size_t mat_bytes(int wdtype, int rows, int cols) {
  if (wdtype == DE_Q4_0) return (size_t)rows * cols * 9 / 16;
  return (size_t)rows * cols * (wdtype == DE_BF16 ? 2 : 4);
}

size_t expert_bytes(int wdtype, int inter, int hidden) {
  return 2 * mat_bytes(wdtype, inter, hidden) + mat_bytes(wdtype, hidden, inter);
}

// Host checks of an expert table against a layer shape (also used by the
// model calls before they enqueue anything).
int check_table(const de_moe_desc& d, const de_expert_table* t) {
  if (t == nullptr || t->base == nullptr || (reinterpret_cast<uintptr_t>(t->base) & 15u) != 0)
    return DE_ERR_INVALID;
  const int64_t need = (int64_t)expert_bytes(d.wdtype, d.inter, d.hidden);
  if (t->slot_stride_bytes < need || (t->slot_stride_bytes & 15) != 0) return DE_ERR_INVALID;
  if (t->n_slots < 1) return DE_ERR_INVALID;
  if (t->slot_of_expert == nullptr && t->n_slots < d.n_experts) return DE_ERR_INVALID;
  return DE_OK;
}

thread_local hipError_t t_last_hip = hipSuccess;

hipError_t note_hip(hipError_t e) {
  if (e != hipSuccess) t_last_hip = e;
  return e;
}

}  // namespace de

namespace {

constexpr int kMaxT = 64;
constexpr int kMaxK = 32;
constexpr int kMaxN = 256;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
size_t up256(size_t v) { return (v + 255) & ~size_t(255); }
int elem_bytes(int wdtype) { return wdtype == DE_BF16 ? 2 : 4; }
// Element alignment of every row length (16-byte rows; Q4_0: whole blocks).
int elem_align(int wdtype) { return wdtype == DE_Q4_0 ? 32 : (wdtype == DE_BF16 ? 8 : 4); }

// The shared path's down projection runs as up to this many dense sources
// (intermediate chunks), each with its own [T, H] partial.
constexpr int kMaxSharedChunks = 3;

// Chunks of the shared intermediate for the down pass: the fewest (up to
// max_chunks) whose T input rows fit 64 KB and that are no wider than
// `width` (the routed experts' intermediate, so that every down tile of the
// launch streams rows of about the same length), each a whole number of
// 16-byte weight units; when none qualifies, the valid split with the
// smallest chunk.
int shared_chunks(int inter, int T, int max_chunks, int align, int width) {
  int best = 1;
  for (int c = 1; c <= max_chunks; ++c) {
    if (inter % c != 0 || (inter / c) % align != 0) continue;
    if ((size_t)T * (inter / c) * 4 <= 64 * 1024 && inter / c <= width) return c;
    best = c;
  }
  return best;
}

int verify_chunks(const de_moe_desc& d, int T) {
  return d.shared_inter > 0 ? shared_chunks(d.shared_inter, T, kMaxSharedChunks, elem_align(d.wdtype),
                                            d.inter)
                            : 0;
}

constexpr size_t kCtlBytes = 4096;
constexpr size_t kStatusOff = 256;
// The persistent draft pass's arrival flags: at an offset that does not
// depend on the block length, which no other call writes (a call with
// another block length lays its buffers out differently).
constexpr size_t kPDFlagsOff = 1024;
static_assert(kPDFlagsOff + (de::kPDMaxGrid + 32) * 8 <= kCtlBytes, "control area");


struct Layout {
  size_t ctl, z, idx, gate, nu, uids, offs, tok, glist, ppos;
  size_t a_r, a_s, a_d, p_r, p_s, p_d;
  size_t pd;  // persistent draft pass: gate/up outputs [Is + Id + I], row words [H], logit words [N] (8 bytes)
  // The single-launch verify layer (only for the shapes it serves, else
  // fused = false): (value, epoch) words of A_r, A_s, P_r and the shared
  // down chunks' partials.
  bool fused;
  int chunks;     // shared down chunks of that launch
  size_t lds;     // its LDS bytes per block
  size_t t_ar, t_as, t_pr, t_ps, t_pub;
  size_t total;
};

// True when the verify layer of this shape can run as one launch; chunks and
// lds receive the launch's shared down chunks and LDS bytes per block.
bool fused_shape(const de_moe_desc& d, int T, int* chunks, size_t* lds) {
  if (d.wdtype != DE_BF16 || T < 2 || T > kMaxT) return false;
  const int c = verify_chunks(d, T);
  const size_t b = de::verify_fused_lds(T, d.hidden, d.n_experts, d.top_k, d.inter,
                                        d.shared_inter, c);
  if (b == 0) return false;
  if (chunks) *chunks = c;
  if (lds) *lds = b;
  return true;
}

Layout layout(const de_moe_desc& d, int T) {
  Layout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t r = o;
    o += up256(bytes);
    return r;
  };
  const size_t tk = (size_t)T * d.top_k;
  // Control area: the routing launch's arrival counters [T] (zero after
  // de_workspace_init and after every call), the status word at byte 256
  // (sticky until de_layer_status reads it), the persistent draft pass's
  // flags from byte 1024.
  L.ctl = take(kCtlBytes);
  // The persistent draft pass's buffers (its logit and down-row words are
  // tagged), at the same offset in every layout, so that no call of another
  // block length writes there (a value left there by another buffer could
  // carry a matching tag).
  L.pd = take(((size_t)d.shared_inter + d.draft_inter + d.inter) * 4 +
              ((size_t)d.hidden + d.n_experts) * 8);
  L.z = take((size_t)T * d.n_experts * 4);
  L.idx = take(tk * 4);
  L.gate = take(tk * 4);
  L.nu = take(4);
  L.uids = take((size_t)d.n_experts * 4);
  L.offs = take(((size_t)d.n_experts + 1) * 4);
  L.tok = take(tk * 4);
  L.glist = take(tk * 4);
  L.ppos = take(tk * 4);
  L.a_r = take(tk * d.inter * 4);
  L.a_s = take((size_t)T * d.shared_inter * 4);
  L.a_d = take((size_t)T * d.draft_inter * 4);
  L.p_r = take(tk * d.hidden * 4);
  L.p_s = take((size_t)kMaxSharedChunks * T * d.hidden * 4);
  L.p_d = take((size_t)T * d.hidden * 4);
  L.fused = fused_shape(d, T, &L.chunks, &L.lds);
  if (L.fused) {
    L.t_ar = take(tk * d.inter * 8);
    L.t_as = take((size_t)T * d.shared_inter * 8);
    L.t_pr = take(tk * d.hidden * 8);
    L.t_ps = take((size_t)kMaxSharedChunks * T * d.hidden * 8);
    L.t_pub = take(de::verify_fused_pub_words(T, d.n_experts, d.top_k) * 8);
  }
  L.total = o;
  return L;
}

int check_T(int T) { return (T >= 1 && T <= kMaxT) ? DE_OK : DE_ERR_INVALID; }

int check_ws(const de_moe_desc& d, int T, const void* ws, size_t ws_bytes) {
  if (ws == nullptr || (reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return DE_ERR_WORKSPACE;
  if (ws_bytes < layout(d, T).total) return DE_ERR_WORKSPACE;
  return DE_OK;
}

int check_epi(const de_epilogue* epi) {
  if (epi == nullptr) return DE_OK;
  if (epi->normed != nullptr && !(epi->eps >= 0.f)) return DE_ERR_INVALID;
  return DE_OK;
}

int hip_status(hipError_t e) { return de::note_hip(e) == hipSuccess ? DE_OK : DE_ERR_HIP; }

// Router logits (into the workspace) and the ordered top-k lists of every
// position; the layer calls build the union in their gate/up kernel.
hipError_t route(const de_moe_desc& d, int T, const float* x, const float* w_router,
                 const Layout& L, void* ws, const de::TopkUnionArgs& sel, hipStream_t s,
                 bool select = true) {
  de::RouteArgs r{};
  r.sel = sel;
  r.select = select ? 1 : 0;
  r.x = x;
  r.w = w_router;
  r.H = d.hidden;
  r.z = reinterpret_cast<float*>(static_cast<char*>(ws) + L.z);
  r.sel.z = r.z;
  r.counter = reinterpret_cast<unsigned*>(static_cast<char*>(ws) + L.ctl);
  return de::launch_route(r, s);
}

// One-shot phase timers armed by de_time_next_phase (per host thread).
thread_local hipEvent_t t_start[4] = {nullptr, nullptr, nullptr, nullptr};
thread_local hipEvent_t t_stop[4] = {nullptr, nullptr, nullptr, nullptr};

// Launches one phase with its armed events (if any) around it.
template <typename F>
hipError_t timed_phase(int phase, hipStream_t s, F launch) {
  hipEvent_t a = t_start[phase], b = t_stop[phase];
  t_start[phase] = t_stop[phase] = nullptr;
  if (a != nullptr && hipEventRecord(a, s) != hipSuccess) return hipErrorInvalidValue;
  const hipError_t e = launch();
  if (e != hipSuccess) return e;
  if (b != nullptr && hipEventRecord(b, s) != hipSuccess) return hipErrorInvalidValue;
  return hipSuccess;
}

// The single-launch verify layer: every armed phase timer brackets it (the
// gate/up and down phases both run inside it).
template <typename F>
hipError_t timed_layer(hipStream_t s, F launch) {
  hipEvent_t a[3], b[3];
  for (int i = 0; i < 3; ++i) {
    a[i] = t_start[i];
    b[i] = t_stop[i];
    t_start[i] = t_stop[i] = nullptr;
  }
  for (int i = 0; i < 3; ++i)
    if (a[i] != nullptr && hipEventRecord(a[i], s) != hipSuccess) return hipErrorInvalidValue;
  const hipError_t e = launch();
  if (e != hipSuccess) return e;
  for (int i = 0; i < 3; ++i)
    if (b[i] != nullptr && hipEventRecord(b[i], s) != hipSuccess) return hipErrorInvalidValue;
  return hipSuccess;
}

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

// kk: list entries per position that can enter the union (k, or 1 for the
// drafter's top-1), which bounds the union by T * kk.
de::RoutedSrc routed_src(const de_moe_desc& d, int T, int kk, const de_expert_table* tab,
                         const int32_t* nu, const int32_t* uids, const int32_t* offs,
                         const int32_t* tok, const float* glist, float* a_r, float* p_r,
                         int32_t* status) {
  de::RoutedSrc r{};
  r.status = status;
  r.absent_ok = 0;
  r.base = static_cast<const char*>(tab->base);
  r.stride = tab->slot_stride_bytes;
  r.slot_of_expert = tab->slot_of_expert;
  r.n_slots = tab->n_slots;
  r.n_union = nu;
  r.union_ids = uids;
  r.offsets = offs;
  r.tok_list = tok;
  r.gate_list = glist;
  r.max_union = T * kk < d.n_experts ? T * kk : d.n_experts;
  r.n_experts = d.n_experts;
  r.pairs_max = T * d.top_k;  // capacity of the lists, A_r and P_r
  r.inter = d.inter;
  r.a = a_r;
  r.p = p_r;
  return r;
}

// The verify layer as one launch (verify_fused.hip): the same outputs as the
// gate/up, down and combine launches, bit for bit.
int run_fused(const de_moe_desc& d, int T, const float* x, const de::RoutedSrc& r, int kk,
              const void* shared_w, float* y, const de_epilogue* epi, const Layout& L, void* ws,
              const de::TopkUnionArgs& sel, hipStream_t s) {
  static std::atomic<uint32_t> epoch{1};
  uint32_t ep = epoch.fetch_add(1);
  if (ep == 0) ep = epoch.fetch_add(1);  // 0 never tags a word (a zeroed word is always stale)
  de::FusedArgs f{};
  de::GroupedArgs& g = f.gu;
  g.T = T;
  g.H = d.hidden;
  g.x = x;
  g.has_routed = 1;
  g.r = r;
  g.r.a = nullptr;  // A_r only as tagged words
  g.r.a_tag = at<uint64_t>(ws, L.t_ar);
  g.r.p_tag = at<uint64_t>(ws, L.t_pr);
  g.fuse_route = 1;
  g.fuse_select = 1;
  g.sel = sel;
  g.epoch = ep;
  g.n_dense = 0;
  if (shared_w != nullptr && d.shared_inter > 0) {
    de::DenseSrc& ds = g.dense[g.n_dense++];
    ds.w = shared_w;
    ds.inter = d.shared_inter;
    ds.out = nullptr;
    ds.out_tag = at<uint64_t>(ws, L.t_as);
  }
  de::GroupedArgs& h = f.dn;
  h = g;
  h.fuse_route = 0;
  h.fuse_select = 0;
  h.n_dense = 0;
  h.r.p = r.p;  // the plain P_r too (the residual target reads it)
  // Every down input is read from LDS after it is staged; the plain buffers
  // only keep a stray read in bounds.
  h.r.a = r.a;
  de::CombineArgs& c = f.c;
  c.T = T;
  c.H = d.hidden;
  c.n_dense = 0;
  if (shared_w != nullptr && d.shared_inter > 0) {
    const int chunks = L.chunks;
    const int cl = d.shared_inter / chunks;
    const char* D = static_cast<const char*>(shared_w) +
                    2 * de::mat_bytes(d.wdtype, d.shared_inter, d.hidden);
    for (int i = 0; i < chunks; ++i) {
      de::DenseSrc& ds = h.dense[h.n_dense++];
      ds.w = D + (size_t)i * cl * 2;
      ds.inter = cl;
      ds.ld = d.shared_inter;
      ds.rows = d.hidden;
      ds.gate = 1.0f;
      ds.vin = at<float>(ws, L.a_s) + (size_t)i * cl;
      ds.vin_tag = at<uint64_t>(ws, L.t_as) + (size_t)i * cl;
      ds.vin_stride = d.shared_inter;
      ds.out = nullptr;
      ds.out_tag = at<uint64_t>(ws, L.t_ps) + (size_t)i * T * d.hidden;
      ds.out_stride = d.hidden;
      ++c.n_dense;
    }
  }
  c.kk = kk;
  c.pairs_max = r.pairs_max;
  c.y = y;
  c.residual = epi ? epi->residual : nullptr;
  c.normed = epi ? epi->normed : nullptr;
  c.eps = epi ? epi->eps : 0.f;
  f.region_floats = de::verify_fused_region(T, d.hidden, d.inter, d.shared_inter, L.chunks);
  f.status = r.status;
  f.pub = at<uint64_t>(ws, L.t_pub);
  const hipError_t e = timed_layer(s, [&] { return de::launch_verify_fused(f, L.lds, s); });
  return e == hipSuccess ? DE_OK : DE_ERR_HIP;
}

// gate/up + down + combine over the union (kk entries per position) and the
// dense sources (shared path with gate 1, optionally the draft expert).
// With dense_on false the dense sources are left out of the two grouped
// launches (their partials from an earlier call stay in the workspace); with
// combine_on false the combine is not launched.  Both true for a whole layer.
int run_grouped(const de_moe_desc& d, int T, const float* x, const de::RoutedSrc& r,
                const int32_t* pair_pos, int kk, const void* shared_w, const void* draft_w,
                float gamma, float* y, const de_epilogue* epi, const Layout& L, void* ws,
                const de::TopkUnionArgs* fused_sel, hipStream_t s, bool dense_on = true,
                bool combine_on = true, bool fuse_select = false,
                const float* next_router = nullptr) {
  if (fused_sel != nullptr && fuse_select && dense_on && combine_on && next_router == nullptr &&
      draft_w == nullptr && !r.absent_ok && L.fused && de::verify_fused_enabled()) {
    return run_fused(d, T, x, r, kk, shared_w, y, epi, L, ws, *fused_sel, s);
  }
  const bool q4 = d.wdtype == DE_Q4_0;
  const size_t esz = q4 ? 0 : elem_bytes(d.wdtype);
  de::GroupedArgs g{};
  if (fused_sel != nullptr) {
    g.fuse_route = 1;
    g.fuse_select = fuse_select ? 1 : 0;
    g.sel = *fused_sel;
  }
  g.T = T;
  g.H = d.hidden;
  g.x = x;
  g.has_routed = 1;
  g.r = r;
  g.n_dense = 0;
  de::CombineArgs c{};
  c.T = T;
  c.H = d.hidden;
  c.n_dense = 0;
  if (dense_on && shared_w != nullptr && d.shared_inter > 0) {
    de::DenseSrc& ds = g.dense[g.n_dense++];
    ds.w = shared_w;
    ds.inter = d.shared_inter;
    ds.out = at<float>(ws, L.a_s);
  }
  if (dense_on && draft_w != nullptr && d.draft_inter > 0) {
    de::DenseSrc& ds = g.dense[g.n_dense++];
    ds.w = draft_w;
    ds.inter = d.draft_inter;
    ds.out = at<float>(ws, L.a_d);
  }
  hipError_t e = timed_phase(DE_PHASE_GATEUP, s, [&] { return de::launch_gateup(g, d.wdtype, s); });
  if (e != hipSuccess) return DE_ERR_HIP;
  // The down pass reads the gate/up activations of each dense source.  The
  // shared path's down projection is split along its intermediate dimension
  // into chunks whose block of input rows fits a down block's LDS staging
  // (two chunks for two 1408-wide shared experts at T = 9); each chunk writes
  // its own partial, and the combine sums them.
  int nd = 0;
  if (shared_w != nullptr && d.shared_inter > 0) {
    const int max_chunks = kMaxSharedChunks - ((draft_w != nullptr && d.draft_inter > 0) ? 1 : 0);
    const int chunks =
        shared_chunks(d.shared_inter, T, max_chunks, elem_align(d.wdtype), d.inter);
    const int cl = d.shared_inter / chunks;
    const char* D = static_cast<const char*>(shared_w) +
                    2 * de::mat_bytes(d.wdtype, d.shared_inter, d.hidden);
    c.n_dense = 0;
    for (int i = 0; i < chunks; ++i) {
      de::DenseSrc& ds = g.dense[nd++];
      // Columns [i cl, (i+1) cl) of D; Q4_0: their codes, and their scales
      // after the matrix's codes.
      ds.w = D + (q4 ? (size_t)i * cl / 2 : (size_t)i * cl * esz);
      ds.ws = q4 ? D + (size_t)d.hidden * d.shared_inter / 2 + (size_t)i * cl / 16 : nullptr;
      ds.inter = cl;
      ds.ld = d.shared_inter;
      ds.rows = d.hidden;
      ds.gate = 1.0f;
      ds.vin = at<float>(ws, L.a_s) + (size_t)i * cl;
      ds.vin_stride = d.shared_inter;
      ds.out = at<float>(ws, L.p_s) + (size_t)i * T * d.hidden;
      ds.out_stride = d.hidden;
      c.dense_p[c.n_dense++] = ds.out;
    }
  }
  if (draft_w != nullptr && d.draft_inter > 0) {
    de::DenseSrc& ds = g.dense[nd++];
    ds.w = static_cast<const char*>(draft_w) + 2 * de::mat_bytes(d.wdtype, d.draft_inter, d.hidden);
    ds.ws = q4 ? static_cast<const char*>(ds.w) + (size_t)d.hidden * d.draft_inter / 2 : nullptr;
    ds.inter = d.draft_inter;
    ds.ld = d.draft_inter;
    ds.rows = d.hidden;
    ds.gate = gamma;
    ds.vin = at<float>(ws, L.a_d);
    ds.vin_stride = d.draft_inter;
    ds.out = at<float>(ws, L.p_d);
    ds.out_stride = d.hidden;
    c.dense_p[c.n_dense++] = ds.out;
  }
  g.n_dense = dense_on ? nd : 0;  // the combine reads the dense partials either way
  g.fuse_route = 0;
  c.p_r = r.p;
  c.pair_pos = pair_pos;
  c.kk = kk;
  c.pairs_max = r.pairs_max;
  c.y = y;
  c.residual = epi ? epi->residual : nullptr;
  c.normed = epi ? epi->normed : nullptr;
  c.eps = epi ? epi->eps : 0.f;
  e = timed_phase(DE_PHASE_DOWN, s, [&] { return de::launch_down(g, d.wdtype, s); });
  if (e != hipSuccess) return DE_ERR_HIP;
  if (!combine_on) return DE_OK;
  if (next_router != nullptr) {
    // The next layer's router logits go to this workspace's logit rows, where
    // the next layer call (same shape, T and workspace) reads them.
    de::RouteArgs nr{};
    nr.sel.T = T;
    nr.sel.N = d.n_experts;
    nr.w = next_router;
    nr.H = d.hidden;
    nr.z = at<float>(ws, L.z);
    return hip_status(de::launch_combine_route(c, nr, s));
  }
  return hip_status(de::launch_combine(c, s));
}

}  // namespace

namespace de {

int32_t* layer_status_word(void* ws) { return at<int32_t>(ws, kStatusOff); }

// The LM head of a block of positions runs on the matrix cores unless
// DE_LMHEAD_MFMA is "0" (the vector-ALU row-dot then runs; the two differ only
// in the fp32 summation order).
bool lmhead_mfma_enabled() {
  const char* e = std::getenv("DE_LMHEAD_MFMA");
  return e == nullptr || e[0] != '0';
}

// The verify layer runs as one launch, where its shape allows, only when
// DE_VERIFY_FUSED is "1": the down blocks wait for gate/up outputs that the
// last gate/up waves write, so the launch is slower than the separate
// launches (both give the same bits).
bool verify_fused_enabled() {
  const char* e = std::getenv("DE_VERIFY_FUSED");
  return e != nullptr && e[0] == '1';
}

// The persistent draft pass is used unless DE_DRAFT_PERSISTENT is "0" (the
// separate launches then run every draft layer; both give the same bits).
bool draft_persistent_enabled() {
  const char* e = std::getenv("DE_DRAFT_PERSISTENT");
  return e == nullptr || e[0] != '0';
}

// The single draft layer calls (T = 1, r = 1) through the persistent kernel
// as well; DE_PD_SINGLE=0 keeps them on the separate launches.
bool pd_single_enabled() {
  const char* e = std::getenv("DE_PD_SINGLE");
  return e == nullptr || e[0] != '0';
}

// Runs draft layers layers[0..n) (n >= 1) of one position (T = 1, the top-1
// drafter of Eq. 5) in persistent launches of at most kPDMaxLayers layers.  x_in is the
// first layer's input RMSNorm(h), h_in its residual (NULL: y = layer(x));
// z_ready: the first layer's router logits are already in the workspace's
// logit row.  Returns kPDNotApplicable, before enqueueing anything, when the
// shape or the layers do not fit the kernel.
int draft_persistent_run(const de_moe_desc& d, int n, const PDLayer* layers, const float* x_in,
                         const float* h_in, bool z_ready, float* y_out, float* normed_out,
                         int32_t* pred_idx, float* pred_gate, float eps, void* ws,
                         size_t ws_bytes, hipStream_t s) {
  if (!draft_persistent_enabled() || n < 1 || d.wdtype != DE_BF16) return kPDNotApplicable;
  if (ws == nullptr || ws_bytes < layout(d, 1).total) return kPDNotApplicable;
  if (n > kPDMaxLayers && normed_out == nullptr) return kPDNotApplicable;
  // Every layer with a draft block, or none (then the term is dropped).
  const bool has_draft = d.draft_inter > 0 && layers[0].draft != nullptr;
  for (int l = 0; l < n; ++l)
    if ((d.draft_inter > 0 && (layers[l].draft != nullptr) != has_draft) ||
        (d.shared_inter > 0 && !layers[l].shared))
      return kPDNotApplicable;
  // The shared down projection in the chunks the separate launches use.
  const int max_chunks = kMaxSharedChunks - (has_draft ? 1 : 0);
  const int chunks =
      d.shared_inter > 0 ? shared_chunks(d.shared_inter, 1, max_chunks, elem_align(d.wdtype), d.inter)
                         : 0;
  const PDShape sh{d.hidden, d.n_experts, d.top_k, d.inter, d.shared_inter,
                   has_draft ? d.draft_inter : 0, chunks, chunks > 0 ? d.shared_inter / chunks : 0};
  const int grid = dev_info().num_cus;
  if (!draft_persistent_fits(sh, grid, nullptr, nullptr)) return kPDNotApplicable;
  const Layout L = layout(d, 1);
  PDArgs a{};
  a.H = d.hidden;
  a.N = d.n_experts;
  a.k = d.top_k;
  a.I = d.inter;
  a.Is = d.shared_inter;
  a.Id = sh.Id;
  a.n_chunks = sh.n_chunks;
  a.chunk = sh.chunk;
  a.has_draft = has_draft ? 1 : 0;
  a.score_func = d.score_func;
  a.norm_topk = d.norm_topk;
  a.routed_scale = d.routed_scale;
  a.eps = eps;
  a.grid = grid;
  a.spin_limit = 1u << 20;
  a.lds_bytes = draft_persistent_lds(sh);
  a.a_buf = at<float>(ws, L.pd);
  // 8-byte aligned: Is, Id and I are multiples of 8.
  a.d_tag = reinterpret_cast<uint64_t*>(a.a_buf + (sh.Is + sh.Id + sh.I));
  a.z_tag = a.d_tag + d.hidden;
  a.z_plain = at<float>(ws, L.z);
  a.grid_flags = at<uint64_t>(ws, kPDFlagsOff);
  a.status = at<int32_t>(ws, kStatusOff);
  for (int l0 = 0; l0 < n; l0 += kPDMaxLayers) {
    const int cnt = n - l0 < kPDMaxLayers ? n - l0 : kPDMaxLayers;
    a.L = cnt;
    for (int i = 0; i < cnt; ++i) a.layers[i] = layers[l0 + i];
    // Later launches continue from the previous one's output (read by every
    // block before any block writes the output rows).
    a.x_in = l0 == 0 ? x_in : normed_out;
    a.h_in = l0 == 0 ? h_in : y_out;
    a.z_in = (l0 == 0 && z_ready) ? a.z_plain : nullptr;
    a.y_out = y_out;
    a.normed_out = normed_out;
    a.pred_idx = pred_idx ? pred_idx + (size_t)l0 * d.top_k : nullptr;
    a.pred_gate = pred_gate ? pred_gate + (size_t)l0 * d.top_k : nullptr;
    // Every launch gets its own epoch (see PDArgs); 0 never occurs, so a
    // zeroed flag is always behind.
    static std::atomic<uint32_t> epoch{1};
    a.epoch = epoch.fetch_add(1);
    if (a.epoch == 0) a.epoch = epoch.fetch_add(1);
    const hipError_t e =
        timed_phase(DE_PHASE_DRAFT_PASS, s, [&] { return launch_draft_persistent(a, s); });
    if (e != hipSuccess) {
      // A launch that never started (the device cannot hold the grid, for
      // instance) leaves the work to the separate launches.
      if (l0 == 0 && (e == hipErrorCooperativeLaunchTooLarge || e == hipErrorNotSupported))
        return kPDNotApplicable;
      return DE_ERR_HIP;
    }
  }
  return DE_OK;
}

PDLayer pd_layer(const de_layer_weights& w) {
  PDLayer p{};
  p.w_router = w.w_router;
  p.bias = w.bias;
  p.routed = static_cast<const char*>(w.routed.base);
  p.stride = w.routed.slot_stride_bytes;
  p.slot_of_expert = w.routed.slot_of_expert;
  p.n_slots = w.routed.n_slots;
  p.shared = static_cast<const char*>(w.shared_w);
  p.draft = static_cast<const char*>(w.draft_w);
  p.gamma = w.gamma;
  return p;
}

// Reads the status word after the stream's work so far, clears it, and maps
// its bits to a return code (a missing expert first).
int take_status(int32_t* word, hipStream_t stream) {
  int32_t v = 0;
  if (hipMemcpyAsync(&v, word, sizeof(v), hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return DE_ERR_HIP;
  if (v == 0) return DE_OK;
  if (hipMemsetAsync(word, 0, sizeof(v), stream) != hipSuccess) return DE_ERR_HIP;
  return (v & kStatusNotResident) ? DE_ERR_NOT_RESIDENT : DE_ERR_INVALID;
}

// The grouped part of a layer whose routing already ran: the union of the
// first `ucols` entries of each position's lists idx / gate [T, k] (device),
// built in the gate/up prologue, then gate/up and down over the members the
// table marks resident, with the dense sources when dense_on, and the combine
// when combine_on.  Calls over the same lists with disjoint resident members
// (dense_on in exactly one, combine_on in the last) produce the same bits as
// one call with every member resident: each pair's partial is written once,
// and the combine sums them in list order.
int layer_after_route(const de_moe_desc& d, int T, const float* x, const de_expert_table* routed,
                      const int32_t* idx, const float* gate, int ucols, const void* shared_w,
                      const void* draft_w, float gamma, float* y, const de_epilogue* epi,
                      bool dense_on, bool combine_on, int32_t* n_union, void* ws,
                      size_t ws_bytes, hipStream_t stream) {
  int rc = de_check_desc(&d);
  if (rc != DE_OK) return rc;
  if ((rc = check_T(T)) != DE_OK) return rc;
  if (!x || !idx || !gate || !y || !aligned16(x) || ucols < 1 || ucols > d.top_k)
    return DE_ERR_INVALID;
  if (d.shared_inter > 0 && (shared_w == nullptr || !aligned16(shared_w))) return DE_ERR_INVALID;
  if (draft_w != nullptr && !aligned16(draft_w)) return DE_ERR_INVALID;
  if (!std::isfinite(gamma)) return DE_ERR_INVALID;
  if ((rc = check_table(d, routed)) != DE_OK) return rc;
  if ((rc = check_epi(epi)) != DE_OK) return rc;
  if ((rc = check_ws(d, T, ws, ws_bytes)) != DE_OK) return rc;
  const Layout L = layout(d, T);
  TopkUnionArgs a{};
  a.T = T;
  a.N = d.n_experts;
  a.k = d.top_k;
  a.score_func = d.score_func;
  a.norm_topk = d.norm_topk;
  a.routed_scale = d.routed_scale;
  a.idx_out = const_cast<int32_t*>(idx);  // read only: the prologue copies the lists
  a.gate_out = const_cast<float*>(gate);
  a.ucols = ucols;
  a.n_union = n_union ? n_union : at<int32_t>(ws, L.nu);
  a.union_ids = at<int32_t>(ws, L.uids);
  a.offsets = at<int32_t>(ws, L.offs);
  a.tok_list = at<int32_t>(ws, L.tok);
  a.gate_list = at<float>(ws, L.glist);
  a.pair_pos = at<int32_t>(ws, L.ppos);
  a.z = at<float>(ws, L.z);
  RoutedSrc r = routed_src(d, T, ucols, routed, a.n_union, a.union_ids, a.offsets, a.tok_list,
                           a.gate_list, at<float>(ws, L.a_r), at<float>(ws, L.p_r),
                           at<int32_t>(ws, L.ctl + kStatusOff));
  // The cache marks every member outside the requested chunk absent on
  // purpose: their work is skipped, not reported.
  r.absent_ok = 1;
  return run_grouped(d, T, x, r, a.pair_pos, ucols, shared_w, draft_w, gamma, y, epi, L, ws, &a,
                     stream, dense_on, combine_on);
}

}  // namespace de

extern "C" {

const char* de_hip_error_detail(void) {
  return de::t_last_hip == hipSuccess ? "" : hipGetErrorString(de::t_last_hip);
}

int de_check_desc(const de_moe_desc* d) {
  if (d == nullptr) return DE_ERR_INVALID;
  if (d->wdtype != DE_F32 && d->wdtype != DE_BF16 && d->wdtype != DE_Q4_0)
    return DE_ERR_UNSUPPORTED;
  if (d->score_func != DE_SOFTMAX && d->score_func != DE_SIGMOID) return DE_ERR_UNSUPPORTED;
  if (d->norm_topk != 0 && d->norm_topk != 1) return DE_ERR_INVALID;
  if (d->n_experts < 1 || d->n_experts > kMaxN) return DE_ERR_INVALID;
  if (d->top_k < 1 || d->top_k > kMaxK || d->top_k > d->n_experts) return DE_ERR_INVALID;
  const int al = elem_align(d->wdtype);
  if (d->hidden < al || d->hidden > (1 << 16) || d->hidden % al) return DE_ERR_INVALID;
  if (d->inter < al || d->inter > (1 << 17) || d->inter % al) return DE_ERR_INVALID;
  if (d->shared_inter < 0 || d->shared_inter > (1 << 17) || d->shared_inter % al) return DE_ERR_INVALID;
  if (d->draft_inter < 0 || d->draft_inter > (1 << 17) || d->draft_inter % al) return DE_ERR_INVALID;
  if (!std::isfinite(d->routed_scale)) return DE_ERR_INVALID;
  return DE_OK;
}

size_t de_workspace_bytes(const de_moe_desc* d, int T) {
  if (de_check_desc(d) != DE_OK || check_T(T) != DE_OK) return 0;
  return layout(*d, T).total;
}

int de_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream) {
  if (ws == nullptr || (reinterpret_cast<uintptr_t>(ws) & 255u) != 0 || ws_bytes < 256)
    return DE_ERR_WORKSPACE;
  return hip_status(hipMemsetAsync(ws, 0, ws_bytes, stream));
}

int de_route_topk(const de_moe_desc* d, int T, const float* x, const float* w_router,
                  const float* bias, int32_t* topk_idx, float* topk_gate, void* ws,
                  size_t ws_bytes, hipStream_t stream) {
  int rc = de_check_desc(d);
  if (rc != DE_OK) return rc;
  if ((rc = check_T(T)) != DE_OK) return rc;
  if (x == nullptr || w_router == nullptr || topk_idx == nullptr || topk_gate == nullptr)
    return DE_ERR_INVALID;
  if (!aligned16(x) || !aligned16(w_router) || d->hidden % 4) return DE_ERR_INVALID;
  if ((rc = check_ws(*d, T, ws, ws_bytes)) != DE_OK) return rc;
  const Layout L = layout(*d, T);
  de::TopkUnionArgs a{};
  a.T = T;
  a.N = d->n_experts;
  a.k = d->top_k;
  a.bias = bias;
  a.score_func = d->score_func;
  a.norm_topk = d->norm_topk;
  a.routed_scale = d->routed_scale;
  a.idx_out = topk_idx;
  a.gate_out = topk_gate;
  a.ucols = d->top_k;
  return hip_status(route(*d, T, x, w_router, L, ws, a, stream));
}

int de_expert_union(int T, int k, int N, const int32_t* topk_idx, const float* topk_gate,
                    int32_t* n_union, int32_t* union_ids, int32_t* offsets, int32_t* tok_list,
                    float* gate_list, int32_t* pair_pos, hipStream_t stream) {
  if (check_T(T) != DE_OK || N < 1 || N > kMaxN || k < 1 || k > kMaxK || k > N)
    return DE_ERR_INVALID;
  if (!topk_idx || !topk_gate || !n_union || !union_ids || !offsets || !tok_list || !gate_list ||
      !pair_pos)
    return DE_ERR_INVALID;
  de::TopkUnionArgs a{};
  a.T = T;
  a.N = N;
  a.k = k;
  a.z = nullptr;
  a.idx_in = topk_idx;
  a.gate_in = topk_gate;
  a.ucols = k;
  a.n_union = n_union;
  a.union_ids = union_ids;
  a.offsets = offsets;
  a.tok_list = tok_list;
  a.gate_list = gate_list;
  a.pair_pos = pair_pos;
  return hip_status(de::launch_union(a, stream));
}

int de_grouped_swiglu(const de_moe_desc* d, int T, const float* x, const de_expert_table* routed,
                      const int32_t* n_union, const int32_t* union_ids, const int32_t* offsets,
                      const int32_t* tok_list, const float* gate_list, const int32_t* pair_pos,
                      const void* shared_w, float* y, const de_epilogue* epi, void* ws,
                      size_t ws_bytes, hipStream_t stream) {
  int rc = de_check_desc(d);
  if (rc != DE_OK) return rc;
  if ((rc = check_T(T)) != DE_OK) return rc;
  if (!x || !y || !n_union || !union_ids || !offsets || !tok_list || !gate_list || !pair_pos)
    return DE_ERR_INVALID;
  if (!aligned16(x)) return DE_ERR_INVALID;
  if (d->shared_inter > 0 && (shared_w == nullptr || !aligned16(shared_w))) return DE_ERR_INVALID;
  if ((rc = de::check_table(*d, routed)) != DE_OK) return rc;
  if ((rc = check_epi(epi)) != DE_OK) return rc;
  if ((rc = check_ws(*d, T, ws, ws_bytes)) != DE_OK) return rc;
  const Layout L = layout(*d, T);
  const de::RoutedSrc r = routed_src(*d, T, d->top_k, routed, n_union, union_ids, offsets,
                                     tok_list, gate_list, at<float>(ws, L.a_r),
                                     at<float>(ws, L.p_r), at<int32_t>(ws, L.ctl + kStatusOff));
  return run_grouped(*d, T, x, r, pair_pos, d->top_k, shared_w, nullptr, 0.f, y, epi, L, ws,
                     nullptr, stream);
}

int de_draft_layer_topr(const de_moe_desc* d, int T, const float* x, const float* w_router,
                        const float* bias, const de_expert_table* routed, const void* shared_w,
                        const void* draft_w, float gamma, int r, float* y, int32_t* pred_idx,
                        float* pred_gate, const de_epilogue* epi, void* ws, size_t ws_bytes,
                        hipStream_t stream) {
  return de::draft_layer_chain(d, T, x, w_router, bias, routed, shared_w, draft_w, gamma, r, y,
                               pred_idx, pred_gate, epi, ws, ws_bytes, stream, false, nullptr);
}

int de_draft_layer(const de_moe_desc* d, int T, const float* x, const float* w_router,
                   const float* bias, const de_expert_table* routed, const void* shared_w,
                   const void* draft_w, float gamma, float* y, int32_t* pred_idx,
                   float* pred_gate, const de_epilogue* epi, void* ws, size_t ws_bytes,
                   hipStream_t stream) {
  return de_draft_layer_topr(d, T, x, w_router, bias, routed, shared_w, draft_w, gamma, 1, y,
                             pred_idx, pred_gate, epi, ws, ws_bytes, stream);
}

int de_verify_layer(const de_moe_desc* d, int T, const float* x, const float* w_router,
                    const float* bias, const de_expert_table* routed, const void* shared_w,
                    float* y, int32_t* topk_idx, float* topk_gate, int32_t* n_union,
                    int32_t* union_ids, int32_t* offsets, int32_t* tok_list, float* gate_list,
                    int32_t* pair_pos, const de_epilogue* epi, void* ws, size_t ws_bytes,
                    hipStream_t stream) {
  return de::verify_layer_chain(d, T, x, w_router, bias, routed, shared_w, y, topk_idx,
                                topk_gate, n_union, union_ids, offsets, tok_list, gate_list,
                                pair_pos, epi, ws, ws_bytes, stream, false, nullptr);
}

}  // extern "C"

namespace de {

// The layer calls of a chain of MoE layers (the stacked model): with
// logits_ready the router logits were already written to the workspace by the
// previous layer's combine; with next_router this layer's combine also writes
// the next layer's logits (which needs epi->normed).
int draft_layer_chain(const de_moe_desc* d, int T, const float* x, const float* w_router,
                      const float* bias, const de_expert_table* routed, const void* shared_w,
                      const void* draft_w, float gamma, int r, float* y, int32_t* pred_idx,
                      float* pred_gate, const de_epilogue* epi, void* ws, size_t ws_bytes,
                      hipStream_t stream, bool logits_ready, const float* next_router) {
  int rc = de_check_desc(d);
  if (rc != DE_OK) return rc;
  if ((rc = check_T(T)) != DE_OK) return rc;
  if (r < 1 || r > d->top_k) return DE_ERR_INVALID;
  if (!x || !w_router || !y || !aligned16(x) || !aligned16(w_router) || d->hidden % 4)
    return DE_ERR_INVALID;
  if (d->shared_inter > 0 && (shared_w == nullptr || !aligned16(shared_w))) return DE_ERR_INVALID;
  if (draft_w != nullptr && !aligned16(draft_w)) return DE_ERR_INVALID;
  if (!std::isfinite(gamma)) return DE_ERR_INVALID;
  if ((rc = de::check_table(*d, routed)) != DE_OK) return rc;
  if ((rc = check_epi(epi)) != DE_OK) return rc;
  if ((rc = check_ws(*d, T, ws, ws_bytes)) != DE_OK) return rc;
  const Layout L = layout(*d, T);
  de::TopkUnionArgs a{};
  a.T = T;
  a.N = d->n_experts;
  a.k = d->top_k;
  a.bias = bias;
  a.score_func = d->score_func;
  a.norm_topk = d->norm_topk;
  a.routed_scale = d->routed_scale;
  a.idx_out = pred_idx ? pred_idx : at<int32_t>(ws, L.idx);
  a.gate_out = pred_gate ? pred_gate : at<float>(ws, L.gate);
  a.ucols = r;  // the drafter reads only the r leading experts of each position
  // Without the predicted lists and the top-k renormalisation nothing reads
  // past the r leading entries: the prologue selects only those.
  a.rounds = (pred_idx == nullptr && pred_gate == nullptr && !d->norm_topk) ? r : 0;
  a.n_union = at<int32_t>(ws, L.nu);
  a.union_ids = at<int32_t>(ws, L.uids);
  a.offsets = at<int32_t>(ws, L.offs);
  a.tok_list = at<int32_t>(ws, L.tok);
  a.gate_list = at<float>(ws, L.glist);
  a.pair_pos = at<int32_t>(ws, L.ppos);
  a.z = at<float>(ws, L.z);
  // Logits only; the gate/up prologue selects the top-k in every block.
  if (next_router != nullptr && (epi == nullptr || epi->normed == nullptr)) return DE_ERR_INVALID;
  // One position with its leading expert: the persistent kernel runs the
  // whole layer (routing, gate/up, down, combine) in one launch, with the
  // same bits.
  if (T == 1 && r == 1 && !logits_ready && next_router == nullptr && pd_single_enabled()) {
    PDLayer pl{};
    pl.w_router = w_router;
    pl.bias = bias;
    pl.routed = static_cast<const char*>(routed->base);
    pl.stride = routed->slot_stride_bytes;
    pl.slot_of_expert = routed->slot_of_expert;
    pl.n_slots = routed->n_slots;
    pl.shared = static_cast<const char*>(shared_w);
    pl.draft = static_cast<const char*>(draft_w);
    pl.gamma = gamma;
    rc = draft_persistent_run(*d, 1, &pl, x, epi ? epi->residual : nullptr, false, y,
                              epi ? epi->normed : nullptr, pred_idx, pred_gate,
                              epi ? epi->eps : 0.f, ws, ws_bytes, stream);
    if (rc != kPDNotApplicable) return rc;
  }
  if (!logits_ready && route(*d, T, x, w_router, L, ws, a, stream, false) != hipSuccess)
    return DE_ERR_HIP;
  const de::RoutedSrc rs = routed_src(*d, T, r, routed, a.n_union, a.union_ids, a.offsets,
                                      a.tok_list, a.gate_list, at<float>(ws, L.a_r),
                                      at<float>(ws, L.p_r), at<int32_t>(ws, L.ctl + kStatusOff));
  return run_grouped(*d, T, x, rs, a.pair_pos, r, shared_w, draft_w, gamma, y, epi, L, ws, &a,
                     stream, true, true, true, next_router);
}

int verify_layer_chain(const de_moe_desc* d, int T, const float* x, const float* w_router,
                       const float* bias, const de_expert_table* routed, const void* shared_w,
                       float* y, int32_t* topk_idx, float* topk_gate, int32_t* n_union,
                       int32_t* union_ids, int32_t* offsets, int32_t* tok_list, float* gate_list,
                       int32_t* pair_pos, const de_epilogue* epi, void* ws, size_t ws_bytes,
                       hipStream_t stream, bool logits_ready, const float* next_router) {
  int rc = de_check_desc(d);
  if (rc != DE_OK) return rc;
  if ((rc = check_T(T)) != DE_OK) return rc;
  if (!x || !w_router || !y || !aligned16(x) || !aligned16(w_router) || d->hidden % 4)
    return DE_ERR_INVALID;
  if (d->shared_inter > 0 && (shared_w == nullptr || !aligned16(shared_w))) return DE_ERR_INVALID;
  if ((rc = de::check_table(*d, routed)) != DE_OK) return rc;
  if ((rc = check_epi(epi)) != DE_OK) return rc;
  if ((rc = check_ws(*d, T, ws, ws_bytes)) != DE_OK) return rc;
  const Layout L = layout(*d, T);
  de::TopkUnionArgs a{};
  a.T = T;
  a.N = d->n_experts;
  a.k = d->top_k;
  a.bias = bias;
  a.score_func = d->score_func;
  a.norm_topk = d->norm_topk;
  a.routed_scale = d->routed_scale;
  a.idx_out = topk_idx ? topk_idx : at<int32_t>(ws, L.idx);
  a.gate_out = topk_gate ? topk_gate : at<float>(ws, L.gate);
  a.ucols = d->top_k;
  a.n_union = n_union ? n_union : at<int32_t>(ws, L.nu);
  a.union_ids = union_ids ? union_ids : at<int32_t>(ws, L.uids);
  a.offsets = offsets ? offsets : at<int32_t>(ws, L.offs);
  a.tok_list = tok_list ? tok_list : at<int32_t>(ws, L.tok);
  a.gate_list = gate_list ? gate_list : at<float>(ws, L.glist);
  a.pair_pos = pair_pos ? pair_pos : at<int32_t>(ws, L.ppos);
  a.z = at<float>(ws, L.z);
  // Logits only; the gate/up prologue selects the top-k in every block.
  if (next_router != nullptr && (epi == nullptr || epi->normed == nullptr)) return DE_ERR_INVALID;
  if (!logits_ready && route(*d, T, x, w_router, L, ws, a, stream, false) != hipSuccess)
    return DE_ERR_HIP;
  const de::RoutedSrc r = routed_src(*d, T, d->top_k, routed, a.n_union, a.union_ids,
                                     a.offsets, a.tok_list, a.gate_list, at<float>(ws, L.a_r),
                                     at<float>(ws, L.p_r), at<int32_t>(ws, L.ctl + kStatusOff));
  return run_grouped(*d, T, x, r, a.pair_pos, d->top_k, shared_w, nullptr, 0.f, y, epi, L, ws, &a,
                     stream, true, true, true, next_router);
}

int accept_len_embed(int K, int V, const float* target_logits, const int32_t* draft_tokens,
                     int32_t* target_argmax, int32_t* out, void* ws, size_t ws_bytes,
                     const void* emb, int H, float* h, float* normed, float eps,
                     hipStream_t stream);

}  // namespace de

extern "C" {

size_t de_accept_workspace_bytes(int K, int V) {
  if (K < 0 || K > 1024 || V < 1) return 0;
  const size_t rows = (size_t)K + 1, ch = (size_t)de::accept_chunks(V);
  return 256 + up256(rows * 4) + 2 * up256(rows * ch * 4);
}

int de_accept_len(int K, int V, const float* target_logits, const int32_t* draft_tokens,
                  int32_t* target_argmax, int32_t* out, void* ws, size_t ws_bytes,
                  hipStream_t stream) {
  return de::accept_len_embed(K, V, target_logits, draft_tokens, target_argmax, out, ws, ws_bytes,
                              nullptr, 0, nullptr, nullptr, 0.f, stream);
}

}  // extern "C"

namespace de {

// de_accept_len that also writes the bonus token's embedding row to h [H] and
// its RMSNorm to normed when emb (bf16 [V, H]) is not NULL.
int accept_len_embed(int K, int V, const float* target_logits, const int32_t* draft_tokens,
                     int32_t* target_argmax, int32_t* out, void* ws, size_t ws_bytes,
                     const void* emb, int H, float* h, float* normed, float eps,
                     hipStream_t stream) {
  if (K < 0 || K > 1024 || V < 1 || !target_logits || !target_argmax || !out) return DE_ERR_INVALID;
  if (K > 0 && draft_tokens == nullptr) return DE_ERR_INVALID;
  if (emb != nullptr && (H < 1 || h == nullptr || normed == nullptr)) return DE_ERR_INVALID;
  if (ws == nullptr || (reinterpret_cast<uintptr_t>(ws) & 255u) != 0 ||
      ws_bytes < de_accept_workspace_bytes(K, V))
    return DE_ERR_WORKSPACE;
  const size_t rows = (size_t)K + 1, ch = (size_t)de::accept_chunks(V);
  de::AcceptArgs a{};
  a.emb = static_cast<const uint16_t*>(emb);
  a.H = H;
  a.h = h;
  a.normed = normed;
  a.eps = eps;
  a.K = K;
  a.V = V;
  a.logits = target_logits;
  a.drafts = draft_tokens;
  a.amax = target_argmax;
  a.out = out;
  a.done_cnt = at<unsigned>(ws, 0);
  a.row_cnt = at<unsigned>(ws, 256);
  a.part_v = at<float>(ws, 256 + up256(rows * 4));
  a.part_i = at<int32_t>(ws, 256 + up256(rows * 4) + up256(rows * ch * 4));
  return hip_status(de::launch_argmax_accept(a, stream));
}

}  // namespace de

extern "C" {

int de_lm_head(int T, int H, int V, const float* x, const void* w_lm, float* logits,
               hipStream_t stream) {
  if (check_T(T) != DE_OK || H < 8 || H % 8 || V < 1 || !x || !w_lm || !logits) return DE_ERR_INVALID;
  if (!aligned16(x) || !aligned16(w_lm)) return DE_ERR_INVALID;
  // A block of positions on the matrix cores (the vector-ALU row-dot is
  // arithmetic-bound there); one position streams at the HBM rate already.
  if (de::rowdot_mfma_fits(T, H) && de::lmhead_mfma_enabled())
    return hip_status(de::launch_rowdot_mfma(T, H, V, x, w_lm, logits, stream));
  de::GroupedArgs g{};
  g.T = T;
  g.H = H;
  g.x = x;
  g.has_routed = 0;
  g.n_dense = 1;
  g.dense[0].w = w_lm;
  g.dense[0].inter = H;
  g.dense[0].rows = V;
  g.dense[0].gate = 1.0f;
  g.dense[0].vin = x;
  g.dense[0].vin_stride = H;
  g.dense[0].out = logits;
  g.dense[0].out_stride = V;
  return hip_status(de::launch_down(g, DE_BF16, stream));
}

int de_rmsnorm(int T, int H, const float* x, float eps, float* out, hipStream_t stream) {
  if (T < 1 || T > 65536 || H < 1 || !x || !out || !(eps >= 0.f)) return DE_ERR_INVALID;
  return hip_status(de::launch_rmsnorm(T, H, x, eps, out, stream));
}

int de_embed_gather(int T, int H, int V, const int32_t* tokens, const void* emb, float* h,
                    float* normed, float eps, int32_t* status, hipStream_t stream) {
  if (T < 1 || T > 65536 || H < 1 || V < 1 || !tokens || !emb || !h || !(eps >= 0.f))
    return DE_ERR_INVALID;
  return hip_status(de::launch_embed(T, H, V, tokens, static_cast<const uint16_t*>(emb), h, normed,
                                     eps, status, stream));
}

int de_layer_status(void* ws, size_t ws_bytes, hipStream_t stream) {
  if (ws == nullptr || (reinterpret_cast<uintptr_t>(ws) & 255u) != 0 || ws_bytes < kCtlBytes)
    return DE_ERR_WORKSPACE;
  return de::take_status(de::layer_status_word(ws), stream);
}

size_t de_dense_workspace_bytes(int T, int H, int I) {
  if (check_T(T) != DE_OK || H < 1 || I < 1) return 0;
  return up256((size_t)T * I * 4) + (size_t)kMaxSharedChunks * up256((size_t)T * H * 4);
}

// Intermediate chunks of a dense layer's down pass: as many as there are
// dense sources (each a whole number of 16-byte units), so that its few
// output rows are streamed by three times the waves.
int dense_chunks(int I, int align) {
  for (int c = kMaxSharedChunks; c > 1; --c)
    if (I % c == 0 && (I / c) % align == 0) return c;
  return 1;
}

int de_dense_swiglu(int T, int H, int I, int wdtype, const float* x, const void* w, float* y,
                    const de_epilogue* epi, void* ws, size_t ws_bytes, hipStream_t stream) {
  return de::dense_swiglu_chain(T, H, I, wdtype, x, w, y, epi, ws, ws_bytes, stream, nullptr,
                                nullptr, nullptr);
}

}  // extern "C"

namespace de {

// The dense layer in a chain: with next_router, its combine also writes the
// following MoE layer's router logits (next_desc's shape) to that layer's
// workspace next_ws, where its call with the logits ready reads them.
int dense_swiglu_chain(int T, int H, int I, int wdtype, const float* x, const void* w, float* y,
                       const de_epilogue* epi, void* ws, size_t ws_bytes, hipStream_t stream,
                       const de_moe_desc* next_desc, void* next_ws, const float* next_router) {
  if (wdtype != DE_F32 && wdtype != DE_BF16) return DE_ERR_UNSUPPORTED;
  const int al = elem_align(wdtype);
  if (check_T(T) != DE_OK || H < al || H % al || I < al || I % al || I > (1 << 17))
    return DE_ERR_INVALID;
  if (!x || !w || !y || !aligned16(x) || !aligned16(w)) return DE_ERR_INVALID;
  if (check_epi(epi) != DE_OK) return DE_ERR_INVALID;
  if (next_router != nullptr &&
      (next_desc == nullptr || next_ws == nullptr || epi == nullptr || epi->normed == nullptr ||
       next_desc->hidden != H || !de::combine_route_fits(H) || !aligned16(next_router)))
    return DE_ERR_INVALID;
  if (ws == nullptr || (reinterpret_cast<uintptr_t>(ws) & 255u) != 0 ||
      ws_bytes < de_dense_workspace_bytes(T, H, I))
    return DE_ERR_WORKSPACE;
  float* A = static_cast<float*>(ws);
  float* P = at<float>(ws, up256((size_t)T * I * 4));
  const size_t pstride = up256((size_t)T * H * 4) / 4;
  de::GroupedArgs g{};
  g.T = T;
  g.H = H;
  g.x = x;
  g.has_routed = 0;
  g.n_dense = 1;
  g.dense[0].w = w;
  g.dense[0].inter = I;
  g.dense[0].out = A;
  if (timed_phase(DE_PHASE_GATEUP, stream, [&] { return de::launch_gateup(g, wdtype, stream); }) !=
      hipSuccess)
    return DE_ERR_HIP;
  // Down: D [H, I] in column chunks, each a dense source with its own partial.
  const int nc = dense_chunks(I, al);
  const int cw = I / nc;
  const char* D = static_cast<const char*>(w) + 2 * (size_t)I * H * elem_bytes(wdtype);
  g.n_dense = nc;
  for (int i = 0; i < nc; ++i) {
    g.dense[i] = de::DenseSrc{};
    g.dense[i].w = D + (size_t)i * cw * elem_bytes(wdtype);
    g.dense[i].inter = cw;
    g.dense[i].ld = I;
    g.dense[i].rows = H;
    g.dense[i].gate = 1.0f;
    g.dense[i].vin = A + (size_t)i * cw;
    g.dense[i].vin_stride = I;
    g.dense[i].out = P + (size_t)i * pstride;
    g.dense[i].out_stride = H;
  }
  if (timed_phase(DE_PHASE_DOWN, stream, [&] { return de::launch_down(g, wdtype, stream); }) !=
      hipSuccess)
    return DE_ERR_HIP;
  de::CombineArgs c{};
  c.T = T;
  c.H = H;
  c.n_dense = nc;
  for (int i = 0; i < nc; ++i) c.dense_p[i] = P + (size_t)i * pstride;
  c.y = y;
  c.residual = epi ? epi->residual : nullptr;
  c.normed = epi ? epi->normed : nullptr;
  c.eps = epi ? epi->eps : 0.f;
  if (next_router != nullptr) {
    de::RouteArgs nr{};
    nr.sel.T = T;
    nr.sel.N = next_desc->n_experts;
    nr.w = next_router;
    nr.H = H;
    nr.z = at<float>(next_ws, layout(*next_desc, T).z);
    return hip_status(de::launch_combine_route(c, nr, stream));
  }
  return hip_status(de::launch_combine(c, stream));
}

}  // namespace de

extern "C" {

int de_verify_single_launch(const de_moe_desc* d, int T) {
  if (de_check_desc(d) != DE_OK || check_T(T) != DE_OK || !de::verify_fused_enabled()) return 0;
  return fused_shape(*d, T, nullptr, nullptr) ? 1 : 0;
}

int de_time_next_phase(int phase, hipEvent_t start, hipEvent_t stop) {
  if (phase != DE_PHASE_GATEUP && phase != DE_PHASE_DOWN && phase != DE_PHASE_LAYER &&
      phase != DE_PHASE_DRAFT_PASS)
    return DE_ERR_INVALID;
  t_start[phase] = start;
  t_stop[phase] = stop;
  return DE_OK;
}

int de_confidence(int T, int V, const float* logits, float* q, hipStream_t stream) {
  if (T < 1 || T > 65536 || V < 1 || !logits || !q) return DE_ERR_INVALID;
  return hip_status(de::launch_confidence(T, V, logits, q, stream));
}

int de_expansion(int L, int k, int N, const int32_t* pred_idx, uint64_t* uhat, int first,
                 const float* q, float tau, int budget, int slots, int32_t* out,
                 hipStream_t stream) {
  if (L < 1 || L > 65536 || N < 1 || N > 256 || k < 1 || k > N) return DE_ERR_INVALID;
  if (!pred_idx || !uhat || !q || !out || budget < DE_BUDGET_CACHE || slots < 0 ||
      tau != tau)
    return DE_ERR_INVALID;
  if ((reinterpret_cast<uintptr_t>(uhat) & 7u) != 0) return DE_ERR_INVALID;
  de::ExpansionArgs a{};
  a.L = L;
  a.k = k;
  a.N = N;
  a.pred = pred_idx;
  a.uhat = reinterpret_cast<unsigned long long*>(uhat);
  a.first = first != 0;
  a.q = q;
  a.tau = tau;
  a.budget = budget;
  a.slots = slots;
  a.out = out;
  return hip_status(de::launch_expansion(a, stream));
}

int de_residual_target(const de_moe_desc* d, int T, const void* ws, size_t ws_bytes,
                       float* m_star, hipStream_t stream) {
  int rc = de_check_desc(d);
  if (rc != DE_OK) return rc;
  if ((rc = check_T(T)) != DE_OK) return rc;
  if (m_star == nullptr) return DE_ERR_INVALID;
  if ((rc = check_ws(*d, T, ws, ws_bytes)) != DE_OK) return rc;
  const Layout L = layout(*d, T);
  de::ResidualArgs a{};
  a.T = T;
  a.H = d->hidden;
  a.kk = d->top_k;
  a.pairs_max = T * d->top_k;
  a.p_r = at<float>(const_cast<void*>(ws), L.p_r);
  a.pair_pos = at<int32_t>(const_cast<void*>(ws), L.ppos);
  a.out = m_star;
  return hip_status(de::launch_residual(a, stream));
}

int de_layer_router_logits(const de_moe_desc* d, int T, const void* ws, size_t ws_bytes,
                           float* z, hipStream_t stream) {
  int rc = de_check_desc(d);
  if (rc != DE_OK) return rc;
  if ((rc = check_T(T)) != DE_OK) return rc;
  if (z == nullptr) return DE_ERR_INVALID;
  if ((rc = check_ws(*d, T, ws, ws_bytes)) != DE_OK) return rc;
  const Layout L = layout(*d, T);
  return hip_status(hipMemcpyAsync(z, static_cast<const char*>(ws) + L.z,
                                   (size_t)T * d->n_experts * 4, hipMemcpyDeviceToDevice,
                                   stream));
}

int de_row_kl(int rows, int n, const float* a, int lda, const float* b, int ldb,
              const float* bias, int sigmoid, float tau, float* kl, float* ce,
              hipStream_t stream) {
  if (rows < 1 || rows > (1 << 20) || n < 1 || lda < n || ldb < n) return DE_ERR_INVALID;
  if (!a || !b || !kl || !(tau > 0.f) || !std::isfinite(tau)) return DE_ERR_INVALID;
  if (sigmoid != 0 && (bias != nullptr || ce != nullptr || tau != 1.f)) return DE_ERR_INVALID;
  de::RowKlArgs r{};
  r.rows = rows;
  r.n = n;
  r.a = a;
  r.lda = lda;
  r.b = b;
  r.ldb = ldb;
  r.bias = bias;
  r.sigmoid = sigmoid != 0;
  r.tau = tau;
  r.kl = kl;
  r.ce = ce;
  return hip_status(de::launch_rowkl(r, stream));
}

int de_stream_probe(const void* buf, size_t bytes, float* sink, hipStream_t stream) {
  if (!buf || !sink || bytes == 0 || bytes % 16 || !aligned16(buf)) return DE_ERR_INVALID;
  return hip_status(de::launch_stream_probe(buf, bytes, sink, stream));
}

}  // extern "C"
