// The fixed-footprint draft pass (Eq. 5) of one block position through a run
// of consecutive MoE layers in a single launch.
//
// A draft layer streams about 70 MB (V2-Lite: router 0.5 MB, two shared
// experts, the top-1 expert and the draft expert), which the separate
// gate/up, down and combine launches spread over three launch boundaries,
// prologues and tails.  Here one block per CU stays resident for all the
// layers, and three device-wide points order the work of a layer:
//
//   sel  the layer's router logits are written: each is a 64-bit word
//        (value, layer tag) that the selecting wave of every block polls;
//   S2   every gate/up output A of the layer is written;
//   S3   every row of the layer's down projection is written: each row is a
//        (value, layer tag) word that every block's combine polls.
//
// The next layer's router rows and each wave's first shared or draft
// gate/up pair, which depend on no result, go out between S3's arrival and
// its wait; the other gate/up pairs when the wave reaches them, the down
// rows of the shared and draft experts at S2 with the top-1 expert's.  A
// wave's loads complete in issue order and the memory queues are shared, so
// every byte in flight at a device-wide point delays that point's polls:
// prefetching less (one pair instead of two, the down rows at S2 instead of
// S3) made a V2-Lite draft position 14% faster.  On the same path, the
// selecting wave selects before its own gate/up work, and publishes the
// top-1 expert (the top-k's first entry) before it completes the list and
// the gates, so that the top-1 rows load while it finishes.  A draft
// position runs the whole stack in one launch; a single layer call runs as a
// one-layer launch, which is also faster than its separate launches.
//
// The arithmetic is the one of the separate launches, operation for
// operation (lane l owns the 16-byte weight units l, l + 64, ...; fp32 FMAs in
// element order; the same wave reductions; the combine's summation order and
// RMSNorm reduction; the same router dot product and top-k selection), so the
// results are bit-identical to theirs.
//
// Blocks exchange data through agent-scope atomic loads and stores, which
// stay coherent across the XCDs' L2 caches without a cache-wide write-back,
// and per-block arrival flags, logit and down-row words tagged with the
// launch's epoch (nothing is reset between launches).  Every wait is bounded: a wait that runs out
// records kStatusSyncTimeout in the status word, and every later wait of the
// block returns at once, so the launch always ends.
#include "de_common.h"
#include "draft_persistent.h"
#include "topk_union.h"

#include <cstddef>
#include <cstdlib>

namespace de {
namespace {

constexpr int kPB = 512;           // threads per block: one block per CU
constexpr int kPW = kPB / kWave;   // waves per block
constexpr int kSelWave = kPW - 1;  // the wave that selects the top-k in each block
constexpr int kGUSlots = 3;        // (G, U) row pairs per wave and layer
constexpr int kGUPre = 1;          // of which issued ahead of the layer's input
constexpr int kDnSlots = 4;        // (row, source) down dot products per wave and layer
// The combine reproduces the 1024-thread combine launch: virtual thread v
// holds elements v and v + 1024, virtual wave w its 64 threads; real thread t
// plays virtual threads t and t + kPB.
constexpr int kCombVT = 1024;
constexpr int kCombVW = kCombVT / kWave;
constexpr int kMaxSrc = 5;         // down sources: shared chunks, draft expert, top-1 expert
constexpr int kMaxRows = 16;       // down rows per block
constexpr int kPDMaxA = 6144;      // gate/up outputs of a layer (Is + Id + I)
constexpr int kPDMaxLogit = 32;    // blocks computing router logits (one expert per wave)

typedef __attribute__((address_space(4))) const char kchar;

// Values that are the same in every lane, moved to scalar registers.
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
template <typename P>
__device__ __forceinline__ P* uni(P* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<P*>(((uint64_t)hi << 32) | lo);
}

// Layer l's descriptor, read from the kernel argument segment with a uniform
// index (scalar loads; a run-time index into a by-value argument would make a
// per-lane copy of the whole argument).
template <typename T>
__device__ __forceinline__ T karg(kchar* p) {
  return *(__attribute__((address_space(4))) const T*)p;
}

__device__ __forceinline__ PDLayer layer_at(int l) {
  kchar* p = (kchar*)__builtin_amdgcn_kernarg_segment_ptr() + offsetof(PDArgs, layers) +
             (size_t)l * sizeof(PDLayer);
  PDLayer d;
  d.w_router = karg<const float*>(p + offsetof(PDLayer, w_router));
  d.bias = karg<const float*>(p + offsetof(PDLayer, bias));
  d.routed = karg<const char*>(p + offsetof(PDLayer, routed));
  d.stride = karg<int64_t>(p + offsetof(PDLayer, stride));
  d.slot_of_expert = karg<const int32_t*>(p + offsetof(PDLayer, slot_of_expert));
  d.shared = karg<const char*>(p + offsetof(PDLayer, shared));
  d.draft = karg<const char*>(p + offsetof(PDLayer, draft));
  d.n_slots = karg<int32_t>(p + offsetof(PDLayer, n_slots));
  d.gamma = karg<float>(p + offsetof(PDLayer, gamma));
  return d;
}

__device__ __forceinline__ float ld_coherent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_coherent64(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_flag(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Waits for every memory operation of the wave to complete (its stores are
// then visible at agent scope).
__device__ __forceinline__ void drain() { __builtin_amdgcn_s_waitcnt(0); }

// Records a timeout once per block; later waits of the block return at once.
__device__ void give_up(const PDArgs& a, int* s_abort) {
  if (!*(volatile int*)s_abort) {
    *(volatile int*)s_abort = 1;
    __hip_atomic_fetch_or(a.status, kStatusSyncTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Waits (one whole wave) until flags[0..n) all reach `target`: lane j watches
// flags j, j + 64, ...  False on a timeout, or at once when an earlier wait
// of the block timed out.
__device__ bool wait_flags(const PDArgs& a, const uint64_t* flags, int n, uint64_t target,
                           int* s_abort) {
  const int lane = threadIdx.x & 63;
  for (unsigned i = 0; i < a.spin_limit; ++i) {
    if (*(volatile int*)s_abort) return false;
    uint64_t mn = ~0ull;
    for (int j = lane; j < n; j += kWave) {
      const uint64_t f = ld_coherent64(flags + j);
      mn = f < mn ? f : mn;
    }
    if (__builtin_amdgcn_ballot_w64(mn < target) == 0ull) return true;
    __builtin_amdgcn_s_sleep(2);
  }
  if (lane == 0) give_up(a, s_abort);
  return false;
}

// Device-wide point n, in two halves so that loads can be issued between
// them: arrive (the block's stores complete, then its flag), ...
__device__ void grid_arrive(const PDArgs& a, unsigned n) {
  drain();
  __syncthreads();
  if (threadIdx.x == 0) st_flag(a.grid_flags + blockIdx.x, ((uint64_t)a.epoch << 32) | n);
}
// ... and wait until every block has arrived.
__device__ void grid_wait(const PDArgs& a, unsigned n, int* s_abort) {
  if (threadIdx.x < kWave)
    wait_flags(a, a.grid_flags, gridDim.x, ((uint64_t)a.epoch << 32) | n, s_abort);
  __syncthreads();
}

// The tag of layer l's logit and down-row words in this launch: never 0 (a
// zeroed word is never taken) and different for every layer of the last
// 2^26 launches.
__device__ __forceinline__ uint32_t layer_tag(const PDArgs& a, int l) {
  return (a.epoch << 6) + (uint32_t)l + 1u;
}

// Layer l's N logits (z[0][q]: expert lane + 64 q), once every word carries
// the layer's tag (one wave).  Bounded: a timeout is recorded and the words
// are used as they are.
__device__ void wait_logits(const PDArgs& a, int l, float (&z)[1][4], int* s_abort) {
  const int lane = threadIdx.x & 63;
  const uint32_t tag = layer_tag(a, l);
  uint64_t w[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = lane + q * kWave;
    w[q] = e < a.N ? ld_coherent64(a.z_tag + e) : (uint64_t)tag << 32;
  }
  for (unsigned it = 0;; ++it) {
    bool ok = true;
#pragma unroll
    for (int q = 0; q < 4; ++q) ok = ok && (uint32_t)(w[q] >> 32) == tag;
    if (__builtin_amdgcn_ballot_w64(!ok) == 0ull) break;
    if (*(volatile int*)s_abort) break;
    if (it >= a.spin_limit) {
      if (lane == 0) give_up(a, s_abort);
      break;
    }
    __builtin_amdgcn_s_sleep(2);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane + q * kWave;
      if ((uint32_t)(w[q] >> 32) != tag && e < a.N) w[q] = ld_coherent64(a.z_tag + e);
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = lane + q * kWave;
    z[0][q] = e < a.N ? __uint_as_float((uint32_t)w[q]) : 0.f;
  }
}

// A (G, U) row pair of the layer: which source, and its row.
struct GURow {
  int src;  // 0 shared, 1 draft, 2 top-1 expert, -1 none
  int row;
  int p;    // index in the concatenated gate/up output [shared | draft | top-1]
};

__device__ __forceinline__ GURow gu_row(const PDArgs& a, int p) {
  GURow g{-1, 0, p};
  if (p < 0 || p >= a.Is + a.Id + a.I) return g;
  if (p < a.Is) {
    g.src = 0;
    g.row = p;
  } else if (p < a.Is + a.Id) {
    g.src = 1;
    g.row = p - a.Is;
  } else {
    g.src = 2;
    g.row = p - a.Is - a.Id;
  }
  return g;
}

// A down dot product: row h of source s (shared chunk c < n_chunks, then the
// draft expert if any, then the top-1 expert).
struct DnDot {
  int i;    // block-local row index; -1 none
  int src;
};

template <int GU_IT>
struct GURegs {
  u32x4 g[GU_IT], u[GU_IT];
};

// Issues the loads of one (G, U) row pair whose G matrix starts at `blk`
// (the block's [G|U|D] layout with intermediate `inter`).
template <int GU_IT>
__device__ __forceinline__ void issue_gu(const PDArgs& a, const char* blk, int inter, int row,
                                         GURegs<GU_IT>& r, int lane) {
  const int L = a.H / 8;  // 16-byte units per row
  const size_t rb = (size_t)a.H * 2;
  const char* G = uni(blk + (size_t)row * rb);
  const char* U = uni(blk + (size_t)inter * rb + (size_t)row * rb);
#pragma unroll
  for (int it = 0; it < GU_IT; ++it) {
    const uint32_t u = (uint32_t)min(it * kWave + lane, L - 1);
    r.g[it] = load_stream16(G + u * 16u);
    r.u[it] = load_stream16(U + u * 16u);
  }
}

// silu(G x) * (U x) with x from LDS, in the lane order and FMA order of the
// grouped gate/up kernel.
template <int GU_IT>
__device__ __forceinline__ float fma_gu(const PDArgs& a, const GURegs<GU_IT>& r, const float* xs,
                                        int lane) {
  const int L = a.H / 8;
  float ag = 0.f, au = 0.f;
#pragma unroll
  for (int it = 0; it < GU_IT; ++it) {
    const int u = it * kWave + lane;
    const bool ok = u < L;
    const int uc = ok ? u : L - 1;
    const float4 x0 = reinterpret_cast<const float4*>(xs)[uc * 2];
    const float4 x1 = reinterpret_cast<const float4*>(xs)[uc * 2 + 1];
    const float xv[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
    const u32x4 z{0u, 0u, 0u, 0u};
    float wg[8], wu[8];
    const u32x4 rg = ok ? r.g[it] : z, ru = ok ? r.u[it] : z;
    wg[0] = bf16_lo(rg.x); wg[1] = bf16_hi(rg.x); wg[2] = bf16_lo(rg.y); wg[3] = bf16_hi(rg.y);
    wg[4] = bf16_lo(rg.z); wg[5] = bf16_hi(rg.z); wg[6] = bf16_lo(rg.w); wg[7] = bf16_hi(rg.w);
    wu[0] = bf16_lo(ru.x); wu[1] = bf16_hi(ru.x); wu[2] = bf16_lo(ru.y); wu[3] = bf16_hi(ru.y);
    wu[4] = bf16_lo(ru.z); wu[5] = bf16_hi(ru.z); wu[6] = bf16_lo(ru.w); wu[7] = bf16_hi(ru.w);
#pragma unroll
    for (int v = 0; v < 8; ++v) ag = fmaf(wg[v], xv[v], ag);
#pragma unroll
    for (int v = 0; v < 8; ++v) au = fmaf(wu[v], xv[v], au);
  }
  const float g = wave_sum(ag);
  const float u = wave_sum(au);
  return silu_f(g) * u;
}

template <int DN_IT>
struct DnRegs {
  u32x4 w[DN_IT];
};

// Down row pointer, length and A offset of dot d for layer descriptor ld.
struct DnRow {
  const char* w;  // first element of the row segment
  int len;        // elements
  int aoff;       // offset of its input in the concatenated A
  int routed;     // 1: the top-1 expert (gate g_e1)
};

__device__ __forceinline__ DnRow dn_row(const PDArgs& a, const PDLayer& ld, int h, int src,
                                        const char* e1blk) {
  DnRow r{nullptr, 0, 0, 0};
  if (src < a.n_chunks) {
    const char* D = ld.shared + (size_t)4 * a.Is * a.H;  // after G and U (bf16)
    r.w = D + ((size_t)h * a.Is + (size_t)src * a.chunk) * 2;
    r.len = a.chunk;
    r.aoff = src * a.chunk;
  } else if (a.has_draft && src == a.n_chunks) {
    const char* D = ld.draft + (size_t)4 * a.Id * a.H;
    r.w = D + (size_t)h * a.Id * 2;
    r.len = a.Id;
    r.aoff = a.Is;
  } else {
    r.w = e1blk == nullptr ? nullptr : e1blk + (size_t)4 * a.I * a.H + (size_t)h * a.I * 2;
    r.len = a.I;
    r.aoff = a.Is + a.Id;
    r.routed = 1;
  }
  return r;
}

template <int DN_IT>
__device__ __forceinline__ void issue_dn(const DnRow& r, DnRegs<DN_IT>& w, int lane) {
  const int L = r.len / 8;
  const char* base = uni(r.w);
#pragma unroll
  for (int it = 0; it < DN_IT; ++it) {
    const uint32_t u = (uint32_t)min(it * kWave + lane, L - 1);
    w.w[it] = load_stream16(base + u * 16u);
  }
}

// The dot product of a down row with its A segment (LDS), in the lane order
// and FMA order of the grouped down kernel; every lane gets the sum.
template <int DN_IT>
__device__ __forceinline__ float fma_dn(const DnRow& r, const DnRegs<DN_IT>& w, const float* as,
                                        int lane) {
  const int L = r.len / 8;
  float acc = 0.f;
#pragma unroll
  for (int it = 0; it < DN_IT; ++it) {
    const int u = it * kWave + lane;
    const bool ok = u < L;
    const int uc = ok ? u : L - 1;
    const float4 x0 = reinterpret_cast<const float4*>(as + r.aoff)[uc * 2];
    const float4 x1 = reinterpret_cast<const float4*>(as + r.aoff)[uc * 2 + 1];
    const float xv[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
    const u32x4 rr = ok ? w.w[it] : u32x4{0u, 0u, 0u, 0u};
    float wv[8];
    wv[0] = bf16_lo(rr.x); wv[1] = bf16_hi(rr.x); wv[2] = bf16_lo(rr.y); wv[3] = bf16_hi(rr.y);
    wv[4] = bf16_lo(rr.z); wv[5] = bf16_hi(rr.z); wv[6] = bf16_lo(rr.w); wv[7] = bf16_hi(rr.w);
#pragma unroll
    for (int v = 0; v < 8; ++v) acc = fmaf(wv[v], xv[v], acc);
  }
  return wave_sum(acc);
}

template <int GU_IT, int DN_IT>
__global__ __launch_bounds__(kPB) void draft_persistent_kernel(PDArgs a) {
  extern __shared__ __align__(16) float s_a[];  // the layer's gate/up outputs, staged
  __shared__ __align__(16) float s_x[kPDMaxH];  // normed input of the current layer
  __shared__ float s_h[kPDMaxH];                // residual stream
  __shared__ float s_red[kCombVW];
  __shared__ float s_part[kMaxRows * kMaxSrc];
  __shared__ int32_t s_idx[32];
  __shared__ float s_sc[32];
  __shared__ int s_e1;
  __shared__ float s_g1;
  __shared__ int s_sel_layer;
  __shared__ int s_abort;
  __shared__ int s_missing;

  const int b = blockIdx.x, G = gridDim.x;
  int lane = threadIdx.x & 63;
  const int wave = uni((int)(threadIdx.x >> 6));
  const int H = a.H;
  const int P = a.Is + a.Id + a.I;
  const int nsrc = a.n_chunks + a.has_draft + 1;
  const int rpb = (H + G - 1) / G;
  const int nlogit = (a.N + kPW - 1) / kPW;  // blocks computing router logits
  const bool logit_block = b < nlogit;

  if (threadIdx.x == 0) {
    s_sel_layer = 0;
    s_abort = 0;
    s_missing = 0;
  }

  // This wave's gate/up rows and down dot products (the same in every layer).
  GURow gr[kGUSlots];
#pragma unroll
  for (int t = 0; t < kGUSlots; ++t) {
    const int j = wave + kPW * t;
    gr[t] = gu_row(a, b + G * j);
    gr[t].src = uni(gr[t].src);
    gr[t].row = uni(gr[t].row);
    gr[t].p = uni(gr[t].p);
  }
  DnDot dd[kDnSlots];
#pragma unroll
  for (int q = 0; q < kDnSlots; ++q) {
    const int qq = wave + kPW * q;
    const int i = qq / nsrc, s = qq - i * nsrc;
    dd[q].i = uni((i < rpb && b + G * i < H) ? i : -1);
    dd[q].src = uni(s);
  }

  GURegs<GU_IT> gw[kGUPre];
  DnRegs<DN_IT> dw[kDnSlots];

  const auto issue_gu_slot = [&](int t, const PDLayer& ld, GURegs<GU_IT>& r) {
    if (gr[t].src == 0) issue_gu<GU_IT>(a, ld.shared, a.Is, gr[t].row, r, lane);
    if (gr[t].src == 1) issue_gu<GU_IT>(a, ld.draft, a.Id, gr[t].row, r, lane);
  };
  // The wave's first kGUPre dense gate/up row pairs of a layer are issued
  // ahead of the layer's input.
  const auto issue_dense = [&](int l) {
    const PDLayer ld = layer_at(l);
#pragma unroll
    for (int t = 0; t < kGUPre; ++t) issue_gu_slot(t, ld, gw[t]);
  };
  const int H4 = H >> 2;
  // A logit block's router rows (expert b * kPW + wave) of layer l, loaded
  // ahead of the layer's input (H <= 2048: 8 float4 per lane).
  float4 wr[8];
  const auto issue_router = [&](int l) {
    const int e = min(b * kPW + wave, a.N - 1);
    const float4* w4 = uni(reinterpret_cast<const float4*>(layer_at(l).w_router) + (size_t)e * H4);
#pragma unroll
    for (int j = 0; j < 8; ++j) wr[j] = w4[min(lane + j * kWave, H4 - 1)];
  };
  // Router logits of layer l from s_x (logit blocks), each published as a
  // (value, tag) word: no drain and no flag, so the logits do not wait for
  // the wave's weight loads in flight.
  const auto logits = [&](int l) {
    const int e = b * kPW + wave;
    if (e < a.N) {
      const float4* xs4 = reinterpret_cast<const float4*>(s_x);
      const float z = router_dot_pre(wr, H4, lane, [&](int h) { return xs4[h]; });
      if (lane == 0)
        st_flag(a.z_tag + e, ((uint64_t)layer_tag(a, l) << 32) | __float_as_uint(z));
    }
  };
  // The top-1 expert of layer l's weight block, or NULL when it has no valid slot.
  const auto e1_block = [&](const PDLayer& ld) -> const char* {
    const int e1 = uni(s_e1);
    const int slot =
        uni((e1 >= 0 && e1 < a.N) ? (ld.slot_of_expert ? ld.slot_of_expert[e1] : e1) : -1);
    if (slot < 0 || slot >= ld.n_slots) return nullptr;
    return ld.routed + (size_t)slot * ld.stride;
  };

  // ---- prologue: layer 0's first gate/up pairs in flight, its input in LDS, its logits
  issue_dense(0);
  if (logit_block && a.z_in == nullptr) issue_router(0);
  for (int i = threadIdx.x; i < H; i += kPB) {
    s_x[i] = a.x_in[i];
    s_h[i] = a.h_in != nullptr ? a.h_in[i] : 0.f;
  }
  __syncthreads();
  if (a.z_in == nullptr && logit_block) logits(0);

  for (int l = 0; l < a.L; ++l) {
    // Opaque to the compiler: per-lane offsets and masks are recomputed in
    // every layer instead of being kept live across the whole run.
    asm volatile("" : "+v"(lane));
    const bool more = l + 1 < a.L;
    const PDLayer ld = layer_at(l);
    // Top-k of the layer (one wave per block), published in LDS.  Layer 0's
    // logits may come from the previous launch (z_in).
    const auto select = [&]() {
      const bool given = l == 0 && a.z_in != nullptr;  // layer 0's logits from the caller
      TopkUnionArgs sel{};
      sel.T = 1;
      sel.N = a.N;
      sel.k = a.k;
      sel.bias = ld.bias;
      sel.score_func = a.score_func;
      sel.norm_topk = a.norm_topk;
      sel.routed_scale = a.routed_scale;
      float z[1][4];
      if (given) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int e = lane + q * kWave;
          z[0][q] = e < a.N ? ld_coherent(a.z_in + e) : 0.f;
        }
      } else {
        wait_logits(a, l, z, &s_abort);
        if (b == 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (lane + q * kWave < a.N) a.z_plain[lane + q * kWave] = z[0][q];
        }
      }
      // The top-1 expert first, published at once so that its rows load while
      // the rest of the selection runs: the first round of topk_regs (the
      // largest key, ties to the lower id), computed the same way, so it is
      // the list's first entry.
      {
        float bk = -INFINITY;
        int bid = INT_MAX;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int e = lane + q * kWave;
          if (e >= a.N) continue;
          const float bias = sel.bias != nullptr ? sel.bias[e] : 0.f;
          float kk = sel.score_func == 0 ? z[0][q] + bias : 1.0f / (1.0f + expf(-z[0][q])) + bias;
          if (!(kk == kk)) kk = -INFINITY;
          if (kk > bk || (kk == bk && e < bid)) {
            bk = kk;
            bid = e;
          }
        }
        const float m = wave_max(bk);
        const int win = wave_min_i32(bk == m ? bid : INT_MAX);
        if (lane == 0) s_e1 = win;
        __hip_atomic_store(&s_sel_layer, l + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
      // The whole list and the gates (g1 is read after the S2 barrier).
      topk_regs<1>(sel, z, s_idx, s_sc);
      if (lane < a.k) {
        const float g = topk_gate(sel, s_sc, lane);
        if (lane == 0) s_g1 = g;
        if (b == 0 && a.pred_idx != nullptr) a.pred_idx[(size_t)l * a.k + lane] = s_idx[lane];
        if (b == 0 && a.pred_gate != nullptr) a.pred_gate[(size_t)l * a.k + lane] = g;
      }
    };
    const auto wait_selected = [&]() {
      for (unsigned i = 0; i < 16 * a.spin_limit; ++i) {
        if (__hip_atomic_load(&s_sel_layer, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) > l) return;
        if (*(volatile int*)&s_abort) return;
        __builtin_amdgcn_s_sleep(2);
      }
      if (lane == 0) give_up(a, &s_abort);
    };

    // ---- the selection first (the selecting wave's own gate/up loads would
    // delay it), then gate/up: dense rows, then the top-1 expert's
    if (wave == kSelWave) select();
#pragma unroll
    for (int t = 0; t < kGUSlots; ++t) {
      if (gr[t].src < 0) continue;
      if (gr[t].src == 2) {
        if (wave != kSelWave) wait_selected();
        const char* blk = e1_block(ld);
        if (blk == nullptr) {
          if (lane == 0) st_coherent(a.a_buf + gr[t].p, 0.f);
          continue;
        }
        issue_gu<GU_IT>(a, blk, a.I, gr[t].row, gw[t % kGUPre], lane);
      } else if (t >= kGUPre) {
        issue_gu_slot(t, ld, gw[t % kGUPre]);
      }
      const float v = fma_gu<GU_IT>(a, gw[t % kGUPre], s_x, lane);
      if (lane == 0) st_coherent(a.a_buf + gr[t].p, v);
    }

    // ---- S2: arrive, put the shared / draft and top-1 down rows in flight, wait
    grid_arrive(a, 2 * l + 1);
    {
#pragma unroll
      for (int q = 0; q < kDnSlots; ++q) {
        if (dd[q].i < 0 || dd[q].src == nsrc - 1) continue;
        issue_dn<DN_IT>(dn_row(a, ld, b + G * dd[q].i, dd[q].src, nullptr), dw[q], lane);
      }
    }
    bool need_e1 = false;
#pragma unroll
    for (int q = 0; q < kDnSlots; ++q) need_e1 |= dd[q].i >= 0 && dd[q].src == nsrc - 1;
    const char* e1blk = e1_block(ld);  // selected: every wave passed the block barrier
    if (need_e1 && e1blk != nullptr) {
#pragma unroll
      for (int q = 0; q < kDnSlots; ++q) {
        if (dd[q].i < 0 || dd[q].src != nsrc - 1) continue;
        issue_dn<DN_IT>(dn_row(a, ld, b + G * dd[q].i, dd[q].src, e1blk), dw[q], lane);
      }
    }
    grid_wait(a, 2 * l + 1, &s_abort);

    // ---- the layer's A, staged for the down dot products
    {
      const uint64_t* src = reinterpret_cast<const uint64_t*>(a.a_buf);
      uint64_t* dst = reinterpret_cast<uint64_t*>(s_a);
      for (int i = threadIdx.x; i < P / 2; i += kPB) dst[i] = ld_coherent64(src + i);
      if ((P & 1) && threadIdx.x == 0) s_a[P - 1] = ld_coherent(a.a_buf + P - 1);
    }
    if (wave == kSelWave && lane == 0 && e1blk == nullptr) s_missing = 1;
    __syncthreads();
    const float g1 = s_g1;
#pragma unroll
    for (int q = 0; q < kDnSlots; ++q) {
      if (dd[q].i < 0) continue;
      const DnRow r = dn_row(a, ld, b + G * dd[q].i, dd[q].src, e1blk);
      float v = 0.f;
      if (r.w != nullptr) {
        const float dot = fma_dn<DN_IT>(r, dw[q], s_a, lane);
        const float gm = r.routed ? g1 : (dd[q].src < a.n_chunks ? 1.0f : ld.gamma);
        v = gm * dot;
      }
      if (lane == 0) s_part[dd[q].i * nsrc + dd[q].src] = v;
    }
    __syncthreads();
    // Per row: the dense partials in source order, then the routed one.
    if (threadIdx.x < rpb && b + G * (int)threadIdx.x < H) {
      float x = 0.f;
      for (int s = 0; s < nsrc; ++s) x += s_part[threadIdx.x * nsrc + s];
      st_flag(a.d_tag + b + G * threadIdx.x,
              ((uint64_t)layer_tag(a, l) << 32) | __float_as_uint(x));
    }

    // ---- S3 (every down row written) is the row words' tags: put the next
    // layer's router rows and first gate/up pair in flight, then gather.  The
    // words also order the reuse of A: a block writes the next layer's A only
    // after its combine, which needs every block's rows, which each block
    // writes after it staged this layer's A.
    if (more) {
      if (logit_block) issue_router(l + 1);
      // A logit block's gate/up pair goes out after its logits (below): its
      // logit words then do not queue behind it.
      if (!logit_block) issue_dense(l + 1);
    }

    // ---- combine: y = residual + the row sums; RMSNorm(y) (the combine
    // launch's element order and reduction order).  Virtual thread
    // vt = threadIdx.x + kPB * j (j = 0, 1) holds elements vt + kCombVT * i
    // (i = 0, 1), its squares summed in that order.
    const bool has_res = l > 0 || a.h_in != nullptr;
    const bool want_norm = more || a.normed_out != nullptr;
    constexpr int kVT = kCombVT / kPB, kPer = kPDMaxH / kCombVT;
    uint64_t dwd[kVT][kPer];
    {
      const uint32_t tag = layer_tag(a, l);
#pragma unroll
      for (int j = 0; j < kVT; ++j)
#pragma unroll
        for (int i = 0; i < kPer; ++i) {
          const int h = threadIdx.x + kPB * j + kCombVT * i;
          dwd[j][i] = h < H ? ld_coherent64(a.d_tag + h) : (uint64_t)tag << 32;
        }
      for (unsigned it = 0;; ++it) {
        bool ok = true;
#pragma unroll
        for (int j = 0; j < kVT; ++j)
#pragma unroll
          for (int i = 0; i < kPer; ++i) ok = ok && (uint32_t)(dwd[j][i] >> 32) == tag;
        if (__builtin_amdgcn_ballot_w64(!ok) == 0ull) break;
        if (*(volatile int*)&s_abort) break;
        if (it >= a.spin_limit) {
          if (lane == 0) give_up(a, &s_abort);
          break;
        }
        __builtin_amdgcn_s_sleep(2);
#pragma unroll
        for (int j = 0; j < kVT; ++j)
#pragma unroll
          for (int i = 0; i < kPer; ++i) {
            const int h = threadIdx.x + kPB * j + kCombVT * i;
            if ((uint32_t)(dwd[j][i] >> 32) != tag && h < H) dwd[j][i] = ld_coherent64(a.d_tag + h);
          }
      }
    }
    float v[kVT][kPer];
    float ss[kVT];
#pragma unroll
    for (int j = 0; j < kVT; ++j) {
      ss[j] = 0.f;
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        const int h = threadIdx.x + kPB * j + kCombVT * i;
        v[j][i] = 0.f;
        if (h < H) {
          float x = __uint_as_float((uint32_t)dwd[j][i]);
          if (has_res) x = s_h[h] + x;
          v[j][i] = x;
          ss[j] = fmaf(x, x, ss[j]);
        }
      }
    }
    float r = 0.f;
    if (want_norm) {
#pragma unroll
      for (int j = 0; j < kVT; ++j) {
        const float t = wave_sum(ss[j]);
        if (lane == 0) s_red[wave + kPW * j] = t;
      }
      __syncthreads();
      float tot = 0.f;
      for (int w = 0; w < kCombVW; ++w) tot += s_red[w];
      r = 1.0f / sqrtf(tot / (float)H + a.eps);
    }
#pragma unroll
    for (int j = 0; j < kVT; ++j) {
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        const int h = threadIdx.x + kPB * j + kCombVT * i;
        if (h < H) {
          s_h[h] = v[j][i];
          if (want_norm) s_x[h] = v[j][i] * r;
          if (!more && b == 0) {
            a.y_out[h] = v[j][i];
            if (a.normed_out != nullptr) a.normed_out[h] = v[j][i] * r;
          }
        }
      }
    }
    __syncthreads();
    if (more && logit_block) {
      logits(l + 1);
      issue_dense(l + 1);
    }
  }

  if (b == 0 && threadIdx.x == 0 && s_missing)
    __hip_atomic_fetch_or(a.status, kStatusNotResident, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int GU_IT, int DN_IT>
hipError_t launch_typed(const PDArgs& a, hipStream_t s) {
  const void* fn = reinterpret_cast<const void*>(draft_persistent_kernel<GU_IT, DN_IT>);
  // At least half of a CU's LDS, so that two blocks never share a CU.
  const size_t lds = a.lds_bytes;
  hipError_t e = allow_lds(fn, lds);
  if (e != hipSuccess) return note_hip(e);
  int occ = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, draft_persistent_kernel<GU_IT, DN_IT>, kPB,
                                                   lds);
  if (e != hipSuccess) return note_hip(e);
  if (occ < 1 || a.grid > occ * dev_info().num_cus) return note_hip(hipErrorCooperativeLaunchTooLarge);
  PDArgs args = a;
  void* params[] = {&args};
  // The grid is one block per CU with at least half of a CU's LDS each, so on
  // a device the stream has to itself every block is resident at once, and
  // every wait is bounded in any case.  A cooperative launch guarantees
  // residency also beside other streams' kernels, at the cost of a
  // synchronisation before and after the launch; DE_PD_COOPERATIVE=1 asks
  // for it.
  const char* env = std::getenv("DE_PD_COOPERATIVE");
  const bool coop = env != nullptr && env[0] == '1';
  e = coop ? hipLaunchCooperativeKernel(fn, dim3(a.grid), dim3(kPB), params, (unsigned)lds, s)
           : hipLaunchKernel(fn, dim3(a.grid), dim3(kPB), params, lds, s);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return note_hip(e);
  }
  return note_hip(hipGetLastError());
}

}  // namespace

bool draft_persistent_fits(const PDShape& s, int grid, int* gu_it, int* dn_it) {
  if (grid < 1 || grid > kPDMaxGrid || s.H < 512 || s.H > kPDMaxH || s.H % 512 != 0) return false;
  if (s.N < 1 || s.N > 256 || s.k < 1 || s.k > 32 || s.k > s.N) return false;
  if (s.I < 8 || s.I % 8 || s.Is < 0 || s.Is % 8 || s.Id < 0 || s.Id % 8) return false;
  if (s.n_chunks < 0 || s.n_chunks > 3 || (s.n_chunks > 0 && (s.chunk % 8 || s.chunk * s.n_chunks != s.Is)))
    return false;
  if (s.n_chunks == 0 && s.Is != 0) return false;
  const int P = s.Is + s.Id + s.I;
  if (P > kPDMaxA || (P + grid - 1) / grid > kGUSlots * kPW) return false;
  const int nsrc = s.n_chunks + (s.Id > 0 ? 1 : 0) + 1;
  const int rpb = (s.H + grid - 1) / grid;
  if (rpb > kMaxRows || nsrc > kMaxSrc || rpb * nsrc > kDnSlots * kPW) return false;
  // Router logits: one wave per expert in the first blocks.
  const int nlogit = (s.N + kPW - 1) / kPW;
  if (nlogit > grid || nlogit > kPDMaxLogit) return false;
  int len = s.I;
  if (s.Id > len) len = s.Id;
  if (s.chunk > len) len = s.chunk;
  const int dn = (len / 8 + kWave - 1) / kWave;
  const int gu = s.H / 512;
  if (dn < 1 || dn > 4 || gu < 1 || gu > 4) return false;
  if (gu_it) *gu_it = gu;
  if (dn_it) *dn_it = dn;
  return true;
}

size_t draft_persistent_lds(const PDShape& s) {
  const size_t need = (size_t)(s.Is + s.Id + s.I) * sizeof(float);
  return need > (size_t)84 * 1024 ? need : (size_t)84 * 1024;
}

hipError_t launch_draft_persistent(const PDArgs& a, hipStream_t s) {
  PDShape sh{a.H, a.N, a.k, a.I, a.Is, a.Id, a.n_chunks, a.chunk};
  int gu = 0, dn = 0;
  if (!draft_persistent_fits(sh, a.grid, &gu, &dn) || a.L < 1 || a.L > kPDMaxLayers)
    return note_hip(hipErrorInvalidValue);
  // Extra iterations past a row's end add exact zeros, so a larger
  // instantiation gives the same bits.
  if (gu > 2 && dn <= 3) return launch_typed<4, 3>(a, s);
  if (gu > 2) return launch_typed<4, 4>(a, s);
  if (gu == 2) return launch_typed<2, 4>(a, s);
  return launch_typed<1, 4>(a, s);
}

}  // namespace de
