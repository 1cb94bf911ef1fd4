// The verify layer of a block of positions (Eq. 4 over the expert union of
// Eq. 2-3, with the shared path) in one launch.
//
// As separate launches (routing, gate/up, down, combine) about a quarter of
// the layer's time goes to launch boundaries: the down launch cannot start
// until the last gate/up wave ends, and CUs idle through the gate/up tail and
// the down prologue.  Here one launch holds, in block order,
//
//   1. G1 gate/up blocks (two per CU): the gate/up launch's blocks, each with
//      its prologue (positions staged in LDS, top-k of every position from
//      the router logits, the union; block 0 also publishes the lists) and
//      its tiles of the shared block and the union members;
//   2. down blocks: the shared down chunks' tiles, then each union member's,
//      in runs of kDownRun tiles of one source, a block per run;
//   3. T combine blocks, one per position.
//
// Workgroups are dispatched in index order, so down blocks start on CUs as
// gate/up blocks finish: the gate/up tail fills with down work, and CUs that
// stream faster take more down runs.  Every wait in the launch is for a block
// of lower index, which is already running or done (the G1 gate/up blocks
// are all resident from the start and wait for nothing), so the launch
// always makes progress.
//
// Blocks meet through tagged values.  Every gate/up output, every down
// partial and the published lists are also stored as 64-bit words (value,
// launch epoch) with agent-scope stores, which are written through to
// memory, and a reader loads a word with agent-scope loads until it carries
// this launch's epoch.  A value is ready exactly when its word says so: no
// flag, fence or device-wide barrier, and nothing is reset between launches
// (a word left by an earlier launch carries an older epoch).  Every wait is
// bounded: one that runs out records kStatusSyncTimeout in the status word.
//
// Every output value is computed by the functions of the separate launches
// (grouped_core.h for the tiles, the combine's summation order and
// reduction), so the results are bit-identical to theirs.
#include "verify_fused.h"

#include "grouped_core.h"
#include "topk_union.h"

namespace de {
namespace {

constexpr int kFB = kBlock;        // threads per block (two blocks per CU)
constexpr int kFW = kFB / kWave;   // waves per block
constexpr int kFRT = kNS;          // weight rows per tile
constexpr int kFEPU = 8;           // bf16 weights per 16-byte unit
constexpr unsigned kSpinLimit = 1u << 20;  // polls of one word before a wait gives up
constexpr int kVT = kCombThreads / kFB;    // combine: virtual threads per thread
constexpr int kDownRun = 16;       // down tiles per down block

__device__ __forceinline__ uint64_t ld_tag(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ bool tag_ok(uint64_t w, uint32_t epoch) {
  return (uint32_t)(w >> 32) == epoch;
}

__device__ __forceinline__ float tag_value(uint64_t w) { return __uint_as_float((uint32_t)w); }

// What a wait needs: the epoch, where to record a timeout, and the block's
// flag that makes later waits return at once.
struct Waiter {
  uint32_t epoch;
  int32_t* status;
  int* s_abort;

  // Reloads the words p[i] with need[i] (w[i]: as first loaded) until all of
  // them carry the epoch, or the poll budget runs out (then the timeout is
  // recorded and the words are used as they are).
  template <int N>
  __device__ __forceinline__ void await(const uint64_t* const (&p)[N], uint64_t (&w)[N],
                                        const bool (&need)[N]) const {
    bool ok = true;
#pragma unroll
    for (int i = 0; i < N; ++i) ok = ok && (!need[i] || tag_ok(w[i], epoch));
    if (ok) return;
    for (unsigned it = 0; it < kSpinLimit && !ok; ++it) {
      if (*(volatile int*)s_abort) return;
      __builtin_amdgcn_s_sleep(2);
      ok = true;
#pragma unroll
      for (int i = 0; i < N; ++i) {
        if (need[i] && !tag_ok(w[i], epoch)) {
          w[i] = ld_tag(p[i]);
          ok = ok && tag_ok(w[i], epoch);
        }
      }
    }
    if (!ok && atomicExch(s_abort, 1) == 0 && status != nullptr)
      __hip_atomic_fetch_or(status, kStatusSyncTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // One word once it carries the epoch.
  __device__ __forceinline__ uint64_t word(const uint64_t* p) const {
    const uint64_t* q[1] = {p};
    uint64_t w[1] = {ld_tag(p)};
    const bool need[1] = {true};
    await(q, w, need);
    return w[0];
  }
};

// rows x len tagged values (row stride rstride) into LDS at dst in the
// staged layout of the grouped kernels (all threads; the caller
// synchronises).  Two float4 groups per thread are loaded before any is
// checked.
__device__ __forceinline__ void copy_tagged(const Waiter& wt, float* dst, const uint64_t* src,
                                            int rstride, int rows, int len) {
  const int l4 = len >> 2;
  const int sst = staged_stride<kFEPU>(len);
  const int n = rows * l4;
  for (int i0 = threadIdx.x; i0 < n; i0 += 2 * kFB) {
    uint64_t w[8];
    const uint64_t* p[8];
    bool need[8];
    int o[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int i = min(i0 + u * kFB, n - 1);
      const int t = i / l4, h4 = i - t * l4;
      o[u] = t * sst + staged_f4<kFEPU>(h4);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        p[4 * u + j] = src + (size_t)t * rstride + h4 * 4 + j;
        w[4 * u + j] = ld_tag(p[4 * u + j]);
        need[4 * u + j] = i0 + u * kFB < n;
      }
    }
    wt.await(p, w, need);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      if (need[4 * u]) {
        const f32x4 v{tag_value(w[4 * u]), tag_value(w[4 * u + 1]), tag_value(w[4 * u + 2]),
                      tag_value(w[4 * u + 3])};
        *reinterpret_cast<f32x4*>(dst + o[u]) = v;
      }
    }
  }
}

// A down block's tiles, lo + [0, n), handed out in order from an LDS counter
// (a wave takes the next tile when it is ready for one).
struct TileQueue {
  int* cnt;
  int lo, n;

  __device__ __forceinline__ int grab() const {
    int q = 0;
    if ((threadIdx.x & 63) == 0) q = atomicAdd(cnt, 1);
    q = __builtin_amdgcn_readfirstlane(q);
    return q < n ? lo + q : -1;
  }
};

// run_stream with the tiles taken from a queue.  The loader takes the next
// tile when it starts issuing it and queues it for the consumer (the loader
// is at most RING iterations ahead, which spans at most two tiles: every
// tile has at least two iterations); tiles of a member without a slot are
// skipped by the loader.
template <typename WT, bool GATEUP, int NT, int RING, int RT, class Q>
__device__ __forceinline__ void run_stream_dyn(const GroupedArgs& a,
                                               const Walker<WT, GATEUP, NT, RT, true> wk,
                                               const Q& tq, int lane) {
  int f0 = -1, f1 = -1, nf = 0;  // taken by the loader, not yet reached by the consumer
  Cursor lc{0, 0, 0}, cc{0, 0, 0};
  Pass<NT> lp, cp;
  const auto grab = [&]() -> bool {
    for (;;) {
      const int t = tq.grab();
      if (t < 0) return false;
      lc.tile = t;
      lc.m0 = 0;
      if (wk.make(a, lc, lp) && lc.ntok > 0) {
        if (nf == 0) f0 = t; else f1 = t;
        ++nf;
        return true;
      }
    }
  };
  const auto pop = [&]() -> bool {
    if (nf == 0) return false;
    cc.tile = f0;
    cc.m0 = 0;
    f0 = f1;
    --nf;
    wk.make(a, cc, cp);
    return true;
  };
  const auto advance_loader = [&](bool& l_ok, int& l_it) {
    if (++l_it == lp.nit) {
      l_it = 0;
      lc.m0 += NT;
      if (lc.m0 < lc.ntok)
        wk.make(a, lc, lp);
      else
        l_ok = grab();
    }
  };
  bool l_ok = grab();
  bool c_ok = pop();
  int l_it = 0, c_it = 0;
  u32x4 raw[RING][RT];
  uint32_t sraw[RING][RT];
#pragma unroll
  for (int q = 0; q < RING; ++q) {
    if (l_ok) {
      issue<WT>(lp, l_it, raw[q], sraw[q], lane);
      advance_loader(l_ok, l_it);
    }
  }
  float acc[RT][NT];
#pragma unroll
  for (int k = 0; k < RT; ++k)
#pragma unroll
    for (int m = 0; m < NT; ++m) acc[k][m] = 0.f;
  while (c_ok) {
#pragma unroll
    for (int q = 0; q < RING; ++q) {
      if (c_ok) {
        consume<WT, NT, RT>(cp, c_it, raw[q], sraw[q], lane, acc);
        if (++c_it == cp.nit) {
          finish<GATEUP, NT, RT, true>(cp, wk.tb, lane, acc, a.epoch);
          c_it = 0;
          cc.m0 += NT;
          if (cc.m0 < cc.ntok)
            wk.make(a, cc, cp);
          else
            c_ok = pop();
        }
        if (l_ok) {
          issue<WT>(lp, l_it, raw[q], sraw[q], lane);
          advance_loader(l_ok, l_it);
        }
      }
    }
  }
}

// The published lists (tagged words): n_union, union_ids[N], offsets[N + 1],
// gate_list[T k], pair_pos[T k], top-k ids[T k].
struct Pub {
  uint64_t* base;
  int N, tk;
  __device__ __forceinline__ uint64_t* nu() const { return base; }
  __device__ __forceinline__ uint64_t* uids() const { return base + 1; }
  __device__ __forceinline__ uint64_t* offs() const { return base + 1 + N; }
  __device__ __forceinline__ uint64_t* gates() const { return base + 2 + 2 * N; }
  __device__ __forceinline__ uint64_t* ppos() const { return base + 2 + 2 * N + tk; }
  __device__ __forceinline__ uint64_t* ids() const { return base + 2 + 2 * N + 2 * tk; }
};

__device__ __forceinline__ void put_tag(uint64_t* p, uint32_t bits, uint32_t epoch) {
  __hip_atomic_store(p, ((uint64_t)epoch << 32) | bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------------ gate/up block

__device__ __forceinline__ void gateup_block(const FusedArgs& f, int b, int lane, int wave,
                                             int* s_absent, DenseSrc* s_dense) {
  const GroupedArgs& a = f.gu;
  const int T = a.T, H = a.H, k = a.sel.k, N = a.sel.N;
  Tables tb = tables_at(a, T * staged_stride<kFEPU>(H));
  tb.dense = s_dense;
  const SelView v = sel_at(a, tb);
  // The wave's first two positions' logits are loaded before the staging so
  // that their latency overlaps it.
  float z0[2][4];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int t = min(wave + r * kFW, T - 1);  // clamped: in bounds, never selected past T
    topk_load(a.sel, a.sel.z + (size_t)t * N, z0[r]);
  }
  stage_rows<kFEPU>(a.x, H, T, H);
  // Wave w selects positions w, w + 8 (two interleaved), then w + 16, ...
  for (int t = wave; t < T; t += 2 * kFW) {
    const int t1 = t + kFW;
    if (t != wave) {
      topk_load(a.sel, a.sel.z + (size_t)t * N, z0[0]);
      if (t1 < T) topk_load(a.sel, a.sel.z + (size_t)t1 * N, z0[1]);
    }
    if (t1 < T) {
      topk_regs<2>(a.sel, z0, v.idx + t * k, v.sc + t * k, v.idx + t1 * k, v.sc + t1 * k);
    } else {
      float z1[1][4];
#pragma unroll
      for (int q = 0; q < 4; ++q) z1[0][q] = z0[0][q];
      topk_regs<1>(a.sel, z1, v.idx + t * k, v.sc + t * k);
    }
    const int kr = a.sel.rounds > 0 ? min(a.sel.rounds, k) : k;
    for (int r = 0; r < 2; ++r) {
      const int tt = t + r * kFW;
      if (tt < T && lane < kr) {
        const float g = topk_gate(a.sel, v.sc + tt * k, lane);
        v.gate[tt * k + lane] = g;
        if (b == 0) {
          a.sel.idx_out[tt * k + lane] = v.idx[tt * k + lane];
          a.sel.gate_out[tt * k + lane] = g;
        }
      }
    }
  }
  __syncthreads();
  if (wave == 0) {
    build_union_wave(a.sel, v, b == 0, tb.tok, tb.gate);
    const int n = uni(v.misc[1]);
    if (n > 0) members_from_union(a, tb, v, lane, kWave, s_absent);
  }
  __syncthreads();
  const int nu_raw = uni(v.misc[1]);
  const int nu = nu_raw < 0 ? 0 : min(nu_raw, a.r.max_union);
  const uint32_t ep = a.epoch;
  if (b == 0) {
    // The lists for the down and combine blocks.
    const Pub pub{f.pub, N, a.r.pairs_max};
    const int tk = T * k;
    if (nu_raw > 0) {
      for (int e = threadIdx.x; e < N; e += kFB) {
        if (v.mask[e] != 0ull) {
          put_tag(pub.uids() + v.upos[e], (uint32_t)e, ep);
          put_tag(pub.offs() + v.upos[e], (uint32_t)v.off[e], ep);
        }
      }
      if (threadIdx.x == 0) put_tag(pub.offs() + nu, (uint32_t)v.misc[2], ep);
      for (int i = threadIdx.x; i < v.misc[2]; i += kFB)
        put_tag(pub.gates() + i, __float_as_uint(tb.gate[i]), ep);
      for (int i = threadIdx.x; i < tk; i += kFB) {
        const int t = i / k, e = v.idx[i];
        const unsigned long long below = t == 0 ? 0ull : (v.mask[e] & (~0ull >> (64 - t)));
        put_tag(pub.ppos() + i, (uint32_t)(v.off[e] + (int)__popcll(below)), ep);
        put_tag(pub.ids() + i, (uint32_t)e, ep);
      }
    }
    // The union size last.  Readers wait for every word they use by its own
    // tag, so the order only matters for how soon they find them.
    if (threadIdx.x == 0) put_tag(pub.nu(), (uint32_t)nu_raw, ep);
  }
  // A needed member without a slot: reported once per launch; its plain
  // partial rows are written as zeros (the combine adds zeros for it).
  if (*s_absent) {
    if (b == 0 && threadIdx.x == 0 && a.r.status != nullptr)
      __hip_atomic_fetch_or(a.r.status, kStatusNotResident, __ATOMIC_RELAXED,
                            __HIP_MEMORY_SCOPE_AGENT);
    const size_t gstride = (size_t)f.g1 * kFB;
    for (int j = 0; j < nu; ++j) {
      const Member m = tb.mem[j];
      if (m.blk != nullptr || m.ntok <= 0) continue;
      float* p = f.dn.r.p + (size_t)m.off * H;
      const size_t n = (size_t)m.ntok * H;
      for (size_t i = (size_t)b * kFB + threadIdx.x; i < n; i += gstride)
        *(DE_GLOBAL float*)(p + i) = 0.f;
    }
  }
  // The tiles: the separate gate/up launch's split over the G1 gate/up blocks.
  const Layout ly = make_layout<kFRT>(a, nu, true);
  const int step = f.g1 * kFW, first = b * kFW + wave;
  NoHook h;
  if (first < ly.ndt) {
    constexpr int DNT = kDenseNTOf<uint16_t>;
    const Walker<uint16_t, true, DNT, kFRT, true> wd{ly, tb, step, 0, ly.ndt,
                                                     staged_stride<kFEPU>(H), true};
    run_stream<uint16_t, true, DNT, kDenseRing, kFRT>(a, wd, first, lane, h);
  }
  __builtin_amdgcn_s_setprio(0);
  if (ly.nr > 0) {
    const int f2 = first >= ly.ndt ? first : first + cdiv(ly.ndt - first, step) * step;
    constexpr int RNT = kRoutedNTOf<uint16_t>;
    const Walker<uint16_t, true, RNT, kFRT, true> wr{ly, tb, step, ly.ndt, ly.total,
                                                     staged_stride<kFEPU>(H), true};
    run_stream<uint16_t, true, RNT, kRingOf<uint16_t>, kFRT>(a, wr, f2, lane, h);
  }
}

// ------------------------------------------------------------------ down block

// Down block d: run d % runs of source d / runs (the shared down chunks, then
// the union members in union order).
__device__ __forceinline__ void down_block(const FusedArgs& f, int d, int lane, int* s_cnt,
                                           int* s_abort, DenseSrc* s_dense) {
  const GroupedArgs& a = f.dn;
  const int T = a.T, H = a.H;
  const Waiter wt{a.epoch, f.status, s_abort};
  const Pub pub{f.pub, a.sel.N, a.r.pairs_max};
  const int src = d / f.runs, run = d - src * f.runs;
  const int nd = a.n_dense;
  const int tps = cdiv(H, kFRT);  // tiles per source
  // The union size (published by gate/up block 0).
  const int nu_raw = (int)(uint32_t)wt.word(pub.nu());
  const int nu = nu_raw < 0 ? 0 : min(nu_raw, a.r.max_union);
  if (src >= nd + nu) return;
  // LDS: staged input rows, then the tables (dense descriptors, members,
  // token and gate lists) and the dense sources' staged offsets.
  Tables tb = tables_at(a, f.region_floats);
  int* dact = reinterpret_cast<int*>(tb.gate + a.r.pairs_max);
  tb.dact = dact;
  tb.dense = s_dense;
  if (threadIdx.x < 3) dact[threadIdx.x] = 0;
  if (threadIdx.x == 0) *s_cnt = 0;
  const Layout ly = make_layout<kFRT>(a, nu, false);
  int lo, hi;
  if (src < nd) {
    lo = src * tps + run * f.run_tiles;
    hi = min((src + 1) * tps, lo + f.run_tiles);
    const DenseSrc& ds = tb.dense[src];
    copy_tagged(wt, s_dyn, uni(ds.vin_tag), uni(ds.vin_stride), T, uni(ds.inter));
  } else {
    const int j = src - nd;
    lo = ly.ndt + j * ly.tr + run * f.run_tiles;
    hi = min(ly.ndt + (j + 1) * ly.tr, lo + f.run_tiles);
    const int e = (int)(uint32_t)wt.word(pub.uids() + j);
    const int off = (int)(uint32_t)wt.word(pub.offs() + j);
    const int ntok = (int)(uint32_t)wt.word(pub.offs() + j + 1) - off;
    const int slot = (e >= 0 && e < a.r.n_experts)
                         ? (a.r.slot_of_expert ? a.r.slot_of_expert[e] : e)
                         : -1;
    // A member without a slot: its partials are zero (the combine adds zeros
    // for it; the plain rows are written by the gate/up blocks).
    if (slot < 0 || slot >= a.r.n_slots || ntok <= 0 || off < 0 || off + ntok > a.r.pairs_max)
      return;
    if (threadIdx.x == 0)
      tb.mem[j] = Member{a.r.base + (size_t)slot * a.r.stride, off, ntok, 0, 0};
    for (int i = threadIdx.x; i < ntok; i += kFB)
      tb.gate[off + i] = tag_value(wt.word(pub.gates() + off + i));
    copy_tagged(wt, s_dyn, a.r.a_tag + (size_t)off * a.r.inter, a.r.inter, ntok, a.r.inter);
  }
  __syncthreads();
  const TileQueue q{s_cnt, lo, hi - lo};
  if (src < nd) {
    constexpr int DNT = kDenseNTOf<uint16_t>;
    const Walker<uint16_t, false, DNT, kFRT, true> w{ly, tb, 1, 0, ly.ndt, 0, false};
    run_stream_dyn<uint16_t, false, DNT, kDenseRing, kFRT>(a, w, q, lane);
  } else {
    constexpr int RNT = kRoutedNTOf<uint16_t>;
    const Walker<uint16_t, false, RNT, kFRT, true> w{ly, tb, 1, ly.ndt, ly.total, 0, false};
    run_stream_dyn<uint16_t, false, RNT, kRingOf<uint16_t>, kFRT>(a, w, q, lane);
  }
}

// ------------------------------------------------------------------ combine block

// The combine of position t: combine_row of the separate launches (its
// kCombThreads threads played by kFB threads, thread i as the virtual
// threads i + j kFB, so the element order, the summation order and the
// reduction order are the same), with the partials read from the tagged
// buffers: first every word a thread sums is awaited, then all are loaded
// again and summed.
__device__ __forceinline__ void combine_block(const FusedArgs& f, int t, float* red, int* s_abort) {
  const CombineArgs& a = f.c;
  const Waiter wt{f.gu.epoch, f.status, s_abort};
  const Pub pub{f.pub, f.gu.sel.N, f.gu.r.pairs_max};
  const int H = a.H, k = f.gu.sel.k;
  const size_t rowoff = (size_t)t * H;
  const int nd = a.n_dense;
  const uint64_t* dt0 = f.dn.dense[0].out_tag;
  const uint64_t* dt1 = f.dn.dense[1].out_tag;
  const uint64_t* dt2 = f.dn.dense[2].out_tag;
  const uint64_t* pt = f.dn.r.p_tag;
  const RoutedSrc& r = f.gu.r;
  const int nu_raw = (int)(uint32_t)wt.word(pub.nu());
  const int kk = nu_raw >= 0 ? a.kk : 0;
  // Pair j of the position: its pair index, and whether its member has no
  // slot (then its partial is zero).
  const auto pair_of = [&](int j, bool& zero) {
    const int e = (int)(uint32_t)wt.word(pub.ids() + t * k + j);
    const int slot =
        (e >= 0 && e < r.n_experts) ? (r.slot_of_expert ? r.slot_of_expert[e] : e) : -1;
    zero = slot < 0 || slot >= r.n_slots;
    return (int)(uint32_t)wt.word(pub.ppos() + t * k + j);
  };
  int pp[8];
  bool pz[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    pp[j] = 0;
    pz[j] = true;
    if (j < kk) pp[j] = pair_of(j, pz[j]);
  }
  const auto dtag = [&](int s) { return s == 0 ? dt0 : (s == 1 ? dt1 : dt2); };
#pragma unroll 1
  for (int i = 0; i < kVT * kCombPer; ++i) {
    const int h = threadIdx.x + i * kFB;
    if (h >= H) break;
#pragma unroll
    for (int s = 0; s < 3; ++s)
      if (s < nd) wt.word(dtag(s) + rowoff + h);
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (j < kk && !pz[j]) wt.word(pt + (size_t)pp[j] * H + h);
    for (int j = 8; j < kk; ++j) {
      bool z = true;
      const int p = pair_of(j, z);
      if (!z) wt.word(pt + (size_t)p * H + h);
    }
  }
  const auto val = [&](const uint64_t* p) { return tag_value(ld_tag(p)); };
  float ss[kVT];
  float vv[kVT][kCombPer];
#pragma unroll
  for (int jv = 0; jv < kVT; ++jv) {
    ss[jv] = 0.f;
    const int vt = (int)threadIdx.x + jv * kFB;  // the virtual thread
#pragma unroll
    for (int i = 0; i < kCombPer; ++i) {
      const int h = vt + i * kCombThreads;
      float x = 0.f;
      if (h < H) {
#pragma unroll
        for (int s = 0; s < 3; ++s)
          if (s < nd) x += val(dtag(s) + rowoff + h);
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (j < kk) x += pz[j] ? 0.f : val(pt + (size_t)pp[j] * H + h);
        for (int j = 8; j < kk; ++j) {
          bool z = true;
          const int p = pair_of(j, z);
          x += z ? 0.f : val(pt + (size_t)p * H + h);
        }
        if (a.residual) x = a.residual[rowoff + h] + x;
        a.y[rowoff + h] = x;
        ss[jv] = fmaf(x, x, ss[jv]);
      }
      vv[jv][i] = x;
    }
  }
  if (a.normed) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int jv = 0; jv < kVT; ++jv) {
      const float w = wave_sum(ss[jv]);
      if (lane == 0) red[wave + jv * kFW] = w;
    }
    __syncthreads();
    float tot = 0.f;
    for (int w = 0; w < kCombThreads / kWave; ++w) tot += red[w];
    const float rr = 1.0f / sqrtf(tot / (float)H + a.eps);
#pragma unroll
    for (int jv = 0; jv < kVT; ++jv)
#pragma unroll
      for (int i = 0; i < kCombPer; ++i) {
        const int h = (int)threadIdx.x + jv * kFB + i * kCombThreads;
        if (h < H) a.normed[rowoff + h] = vv[jv][i] * rr;
      }
  }
}

__global__ __launch_bounds__(kFB) __attribute__((amdgpu_waves_per_eu(4))) void verify_fused_kernel(
    FusedArgs f) {
  const int lane = threadIdx.x & 63, wave = uni((int)(threadIdx.x >> 6));
  const int b = (int)blockIdx.x;
  __shared__ int s_absent, s_abort, s_cnt;
  __shared__ float s_red[kCombThreads / kWave];
  __shared__ DenseSrc s_dense[3];  // the role's dense-source descriptors
  // The descriptors first, by one thread with constant indices: copied later,
  // the compiler keeps the kernel argument's values alive in per-lane scratch
  // memory until then.
  if (threadIdx.x == 0) {
    s_absent = 0;
    s_abort = 0;
    const GroupedArgs& g = b < f.g1 ? f.gu : f.dn;
    if (g.n_dense > 0) s_dense[0] = g.dense[0];
    if (g.n_dense > 1) s_dense[1] = g.dense[1];
    if (g.n_dense > 2) s_dense[2] = g.dense[2];
  }
  __syncthreads();
  if (b < f.g1)
    gateup_block(f, b, lane, wave, &s_absent, s_dense);
  else if (b < f.g1 + f.g2)
    down_block(f, b - f.g1, lane, &s_cnt, &s_abort, s_dense);
  else
    combine_block(f, b - f.g1 - f.g2, s_red, &s_abort);
}

}  // namespace

int verify_fused_region(int T, int H, int I, int Is, int chunks) {
  const int x = T * staged_stride<kFEPU>(H);
  int len = I;
  if (chunks > 0 && Is / chunks > len) len = Is / chunks;
  const int st = T * staged_stride<kFEPU>(len);
  return x > st ? x : st;
}

size_t verify_fused_lds(int T, int H, int N, int k, int I, int Is, int chunks) {
  if (T < 2 || T > 64 || H % 8 || I % 8 || Is % 8 || chunks < 0 || chunks > 3) return 0;
  if (chunks > 0 && (Is % chunks || (Is / chunks) % 8)) return 0;
  if (H > kCombThreads * kCombPer) return 0;  // the combine keeps a row's elements in registers
  // Every tile has at least two 16-byte iterations per lane (rows longer than
  // 512 bf16), so a loader is never more than two tiles ahead.
  if (H <= 512 || I <= 512 || (chunks > 0 && Is / chunks <= 512)) return 0;
  const int tk = T * k;
  const int max_union = tk < N ? tk : N;
  size_t b = (size_t)verify_fused_region(T, H, I, Is, chunks) * sizeof(float);
  b += 3 * sizeof(DenseSrc) + (size_t)max_union * sizeof(Member) + (size_t)tk * 8;
  b += sel_view_bytes(T, k, N);
  b += 4 * sizeof(int);
  // Two blocks per CU (160 KB of LDS), less the kernel's static LDS.
  return b <= 80 * 1024 - 512 ? b : 0;
}

size_t verify_fused_pub_words(int T, int N, int k) { return 2 + 2 * (size_t)N + 3 * (size_t)T * k; }

hipError_t launch_verify_fused(const FusedArgs& f, size_t lds, hipStream_t s) {
  const hipError_t e = allow_lds(reinterpret_cast<const void*>(verify_fused_kernel), lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return note_hip(e);
  }
  FusedArgs a = f;
  a.g1 = 2 * dev_info().num_cus;
  const int tps = (f.dn.H + kFRT - 1) / kFRT;
  a.run_tiles = kDownRun;
  a.runs = (tps + kDownRun - 1) / kDownRun;
  a.g2 = (f.dn.n_dense + f.dn.r.max_union) * a.runs;
  const int grid = a.g1 + a.g2 + f.c.T;
  hipLaunchKernelGGL(verify_fused_kernel, dim3(grid), dim3(kFB), lds, s, a);
  return note_hip(hipGetLastError());
}

}  // namespace de
