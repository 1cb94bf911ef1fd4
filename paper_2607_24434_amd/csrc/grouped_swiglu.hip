// Grouped SwiGLU over the expert union plus the shared / draft / dense
// sources (Eq. 4 and Eq. 5 without the routing), the fixed-order combine, and
// the row-dot used for the LM head.
//
// The separate launches: 512-thread blocks (two per CU), the pass stream of
// grouped_core.h.  The union size stays in device memory; the member table
// (weight block, first pair, positions) and the token / gate lists are copied
// to LDS at the start.  Activations come from LDS: gate/up stages the block of
// positions once, in a bank-conflict-free order; down stages the input rows
// of the sources a block visits, as far as they fit.  A single position, and
// rows that do not fit, are read from global memory.
#include "de_common.h"
#include "draftexpert.h"
#include "topk_union.h"

#include <mutex>
#include <type_traits>
#include <utility>
#include <vector>

#include "grouped_core.h"

namespace de {
namespace {

// ------------------------------------------------------------------ kernels


// Gate/up: A = silu(G x) * (U x) for the dense sources and the union members'
// pairs.  LDSX: the block of positions is staged in LDS.
template <typename WT, bool LDSX, int RT>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void gateup_kernel(
    GroupedArgs a) {
  constexpr int EPU = WTr<WT>::EPU;
  const int lane = threadIdx.x & 63, wave = uni((int)(threadIdx.x >> 6));
  const int act_floats = LDSX ? a.T * staged_stride<EPU>(a.H) : 0;
  const Tables tb = tables_at(a, act_floats);
  // Fused selection: the wave's first two positions' logits are loaded
  // before the staging so that their latency overlaps it.
  const bool sel = a.fuse_route && a.fuse_select;
  __shared__ int s_absent;
  if (threadIdx.x == 0) s_absent = 0;
  float z0[2][4];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    // Clamped position: in bounds; a position past T is never selected.
    const int t = min(wave + r * kWavesPB, a.T - 1);
    if (sel) {
      topk_load(a.sel, a.sel.z + (size_t)t * a.sel.N, z0[r]);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) z0[r][q] = 0.f;
    }
  }
  if constexpr (LDSX) stage_rows<EPU>(a.x, a.H, a.T, a.H);
  fill_dense(a, tb);
  int nu;
  if (a.fuse_route) {
    // The top-k lists (selected here from the logits, or given), then their
    // union, in every block; block 0 also publishes both for the down and
    // combine launches.
    const SelView v = sel_at(a, tb);
    const int k = a.sel.k;
    if (sel) {
      // Wave w selects positions w, w + 8 (two interleaved), then w + 16, ...
      for (int t = wave; t < a.T; t += 2 * kWavesPB) {
        const int t1 = t + kWavesPB;
        if (t != wave) {
          topk_load(a.sel, a.sel.z + (size_t)t * a.sel.N, z0[0]);
          if (t1 < a.T) topk_load(a.sel, a.sel.z + (size_t)t1 * a.sel.N, z0[1]);
        }
        if (t1 < a.T) {
          topk_regs<2>(a.sel, z0, v.idx + t * k, v.sc + t * k, v.idx + t1 * k, v.sc + t1 * k);
        } else {
          float z1[1][4];
#pragma unroll
          for (int q = 0; q < 4; ++q) z1[0][q] = z0[0][q];
          topk_regs<1>(a.sel, z1, v.idx + t * k, v.sc + t * k);
        }
        const int kr = a.sel.rounds > 0 ? min(a.sel.rounds, k) : k;
        for (int r = 0; r < 2; ++r) {
          const int tt = t + r * kWavesPB;
          if (tt < a.T && lane < kr) {
            const float g = topk_gate(a.sel, v.sc + tt * k, lane);
            v.gate[tt * k + lane] = g;
            if (blockIdx.x == 0) {
              a.sel.idx_out[tt * k + lane] = v.idx[tt * k + lane];
              a.sel.gate_out[tt * k + lane] = g;
            }
          }
        }
      }
    } else {
      for (int i = threadIdx.x; i < a.T * k; i += kBlock) {
        v.idx[i] = a.sel.idx_out[i];
        v.gate[i] = a.sel.gate_out[i];
      }
    }
    __syncthreads();
    if (wave == 0) {
      build_union_wave(a.sel, v, blockIdx.x == 0, tb.tok, tb.gate);
      const int n = uni(v.misc[1]);
      if (n > 0) members_from_union(a, tb, v, lane, kWave, &s_absent);
    }
    __syncthreads();
    nu = uni(v.misc[1]);
    nu = nu < 0 ? 0 : min(nu, a.r.max_union);
  } else {
    nu = routed_count(a);
    __syncthreads();  // s_absent is initialised
    if (a.has_routed) fill_tables(a, tb, nu, &s_absent);
    __syncthreads();
  }
  // A needed member without a slot: reported once per launch.
  if (blockIdx.x == 0 && threadIdx.x == 0 && s_absent && !a.r.absent_ok && a.r.status != nullptr)
    *(DE_GLOBAL int32_t*)a.r.status |= kStatusNotResident;
  const Layout ly = make_layout<RT>(a, nu, true);
  run_tiles<WT, true, RT>(a, ly, tb, LDSX ? staged_stride<EPU>(a.H) : a.H, LDSX, lane, wave);
}

// Down projection / row-dot: out = gate * (M v) for the dense sources and the
// union members' D rows.  A block stages in LDS the input rows of the members
// its tiles visit (one or two per sweep of the grid) and of the dense sources
// it meets, as far as they fit; the rest are read from global memory.
template <typename WT, int RT>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void down_kernel(
    GroupedArgs a) {
  constexpr int EPU = WTr<WT>::EPU;
  const int lane = threadIdx.x & 63, wave = uni((int)(threadIdx.x >> 6));
  const int nu = routed_count(a);
  const Tables tb = tables_at(a, a.lds_floats);
  __shared__ int s_absent;
  if (threadIdx.x == 0) s_absent = 0;
  // The dense descriptors are copied before the first barrier: copied after
  // it, the compiler keeps the whole argument in per-lane scratch memory, and
  // a launch that uses scratch costs several µs more.
  fill_dense(a, tb);
  __syncthreads();  // s_absent is initialised
  if (a.has_routed) fill_tables(a, tb, nu, &s_absent);
  __syncthreads();
  if (s_absent && !a.r.absent_ok) {
    // A needed member without a slot contributes zero partials (the combine
    // sums its pairs like any other), spread over the grid.
    const size_t gstride = (size_t)gridDim.x * kBlock;
    for (int j = 0; j < nu; ++j) {
      const Member m = tb.mem[j];
      if (m.blk != nullptr || m.ntok <= 0) continue;
      float* p = a.r.p + (size_t)m.off * a.H;
      const size_t n = (size_t)m.ntok * a.H;
      for (size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += gstride)
        *(DE_GLOBAL float*)(p + i) = 0.f;
    }
  }
  Layout ly = make_layout<RT>(a, nu, false);
  __shared__ int s_dact[3];
  __shared__ int s_list[kMaxStaged + 1];
  __shared__ int s_nlist;
  if (threadIdx.x == 0) {
    const int step = (int)gridDim.x * kWavesPB;
    // A single position's inputs are read from global memory (their loads
    // overlap the weight loads; staging them first measured slower).
    int used = a.T == 1 ? a.lds_floats + 1 : 0, n = 0;
    // Dense sources whose tiles this block visits.
    for (int s = 0; s < 3; ++s) s_dact[s] = -1;
    for (int t = blockIdx.x * kWavesPB; t < ly.ndt; t += step) {
      for (int w = 0; w < kWavesPB && t + w < ly.ndt; w += kWavesPB - 1) {
        int start = 0, unused = 0;
        const int s = ly.source(t + w, start, unused);
        const int len = s == 0 ? a.dense[0].inter : (s == 1 ? a.dense[1].inter : a.dense[2].inter);
        const int need = a.T * staged_stride<EPU>(len);
        if (s_dact[s] < 0 && used + need <= a.lds_floats) {
          s_dact[s] = used;
          used += need;
        }
      }
    }
    // Members whose tiles this block visits, in visiting order.
    int last = -1;
    for (int t = blockIdx.x * kWavesPB + (ly.ndt > 0 ? cdiv(ly.ndt - (int)blockIdx.x * kWavesPB, step) * step : 0);
         t < ly.total; t += step) {
      const int t0 = max(t, ly.ndt), t1 = min(t + kWavesPB - 1, ly.total - 1);
      if (t0 > t1) continue;
      for (int j = (t0 - ly.ndt) / ly.tr; j <= (t1 - ly.ndt) / ly.tr; ++j) {
        if (j == last || n >= kMaxStaged) continue;
        last = j;
        Member& m = tb.mem[j];
        const int need = m.ntok * staged_stride<EPU>(a.r.inter);
        if (m.blk != nullptr && m.ntok > 0 && used + need <= a.lds_floats) {
          m.act = used;
          used += need;
          s_list[n++] = j;
        }
      }
    }
    s_nlist = n;
  }
  __syncthreads();
  for (int i = 0; i < s_nlist; ++i) {
    const Member m = tb.mem[s_list[i]];
    stage_rows_at<EPU>(s_dyn + m.act, a.r.a + (size_t)m.off * a.r.inter, a.r.inter, m.ntok,
                       a.r.inter);
  }
  // Static indices only: a run-time index into the kernel argument would make
  // the compiler copy the whole argument to scratch memory.
  if (a.n_dense > 0 && s_dact[0] >= 0)
    stage_rows_at<EPU>(s_dyn + s_dact[0], a.dense[0].vin, a.dense[0].vin_stride, a.T,
                       a.dense[0].inter);
  if (a.n_dense > 1 && s_dact[1] >= 0)
    stage_rows_at<EPU>(s_dyn + s_dact[1], a.dense[1].vin, a.dense[1].vin_stride, a.T,
                       a.dense[1].inter);
  if (a.n_dense > 2 && s_dact[2] >= 0)
    stage_rows_at<EPU>(s_dyn + s_dact[2], a.dense[2].vin, a.dense[2].vin_stride, a.T,
                       a.dense[2].inter);
  __syncthreads();
  ly.act0 = uni(s_dact[0]);
  ly.act1 = uni(s_dact[1]);
  ly.act2 = uni(s_dact[2]);
  run_tiles<WT, false, RT>(a, ly, tb, 0, false, lane, wave);
}

// ------------------------------------------------------------------ combine

// y[t] = sum of the dense partials + sum_j P_r[pair_pos[t, j]] (+ residual),
// in that fixed order; optionally also RMSNorm(y).  One block of NTH threads
// per position; each thread's kCombPer elements are loaded independently and,
// for a row of at most NTH * kCombPer elements, stay in registers for the
// normalisation.  xs (LDS, may be null) also receives the normalised row;
// without `write` (only with a row of at most NTH * kCombPer elements and
// xs) nothing is written to global memory.
template <int NTH>
__device__ __forceinline__ void combine_row(const CombineArgs& a, int t, float* red,
                                            float* xs = nullptr, bool write = true) {
  const size_t rowoff = (size_t)t * a.H;
  int pp[8];
  const int kk = a.p_r ? min(a.kk, 8) : 0;
  for (int j = 0; j < kk; ++j) {
    const int p = a.pair_pos[(size_t)t * a.kk + j];
    pp[j] = (p >= 0 && p < a.pairs_max) ? p : -1;
  }
  float ss = 0.f;
  float v[kCombPer];
  for (int h0 = threadIdx.x; h0 < a.H; h0 += NTH * kCombPer) {
    // All of an element's partials are loaded before any is added (fixed
    // maxima, predicated), so the loads overlap; the sum keeps the fixed order.
    float dv[kCombPer][3], rv[kCombPer][8], res[kCombPer];
#pragma unroll
    for (int i = 0; i < kCombPer; ++i) {
      const int h = min(h0 + i * NTH, a.H - 1);
#pragma unroll
      for (int s = 0; s < 3; ++s) dv[i][s] = s < a.n_dense ? a.dense_p[s][rowoff + h] : 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        rv[i][j] = (j < kk && pp[j] >= 0) ? a.p_r[(size_t)pp[j] * a.H + h] : 0.f;
      res[i] = a.residual ? a.residual[rowoff + h] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < kCombPer; ++i) {
      const int h = h0 + i * NTH;
      float x = 0.f;
      if (h < a.H) {
#pragma unroll
        for (int s = 0; s < 3; ++s)
          if (s < a.n_dense) x += dv[i][s];
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (j < kk && pp[j] >= 0) x += rv[i][j];
        for (int j = kk; j < (a.p_r ? a.kk : 0); ++j) {
          const int p = a.pair_pos[(size_t)t * a.kk + j];
          if (p >= 0 && p < a.pairs_max) x += a.p_r[(size_t)p * a.H + h];
        }
        if (a.residual) x = res[i] + x;
      }
      v[i] = x;
    }
#pragma unroll
    for (int i = 0; i < kCombPer; ++i) {
      const int h = h0 + i * NTH;
      if (h < a.H) {
        if (write) a.y[rowoff + h] = v[i];
        ss = fmaf(v[i], v[i], ss);
      }
    }
  }
  if (a.normed) {
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    float tot = 0.f;
    for (int w = 0; w < NTH / 64; ++w) tot += red[w];
    const float r = 1.0f / sqrtf(tot / (float)a.H + a.eps);
    if (a.H <= NTH * kCombPer) {
#pragma unroll
      for (int i = 0; i < kCombPer; ++i) {
        const int h = threadIdx.x + i * NTH;
        if (h < a.H) {
          const float n = v[i] * r;
          if (write) a.normed[rowoff + h] = n;
          if (xs != nullptr) xs[h] = n;
        }
      }
    } else {
      for (int h = threadIdx.x; h < a.H; h += NTH) a.normed[rowoff + h] = a.y[rowoff + h] * r;
    }
    __syncthreads();  // red is reused by the next row
  }
}

__global__ __launch_bounds__(kCombThreads) void combine_kernel(CombineArgs a) {
  __shared__ float red[kCombThreads / 64];
  combine_row<kCombThreads>(a, blockIdx.x, red);
}

// The combine of one layer and the router logits of the next (Eq. 1) in one
// launch.  Block L = t G + g combines position t (the g = 0 blocks write y and
// RMSNorm(y); every block keeps the normalised row in LDS) and computes the
// next layer's logits of experts 16 g .. 16 g + 15, one per wave, with the
// same arithmetic as the routing launch.  (The expert group varies fastest:
// workgroups go to the XCDs round-robin, so one group's router rows are read
// from memory by a few XCDs' L2 caches instead of one per position.)
__global__ __launch_bounds__(kCombThreads) void combine_route_kernel(CombineArgs a, RouteArgs r) {
  __shared__ float red[kCombThreads / 64];
  const int G = (r.sel.N + kCombThreads / kWave - 1) / (kCombThreads / kWave);
  const int t = blockIdx.x / G, grp = blockIdx.x - t * G;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int e = grp * (kCombThreads / kWave) + wave;
  const int H4 = r.H >> 2;
  const float4* w4 = reinterpret_cast<const float4*>(r.w) + (size_t)min(e, r.sel.N - 1) * H4;
  // A router row of at most 2048 floats is loaded before the combine (it does
  // not depend on it), so its latency overlaps the combine's.
  const bool pre = H4 <= kWave * 8;
  float4 wp[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) wp[j] = pre ? w4[min(lane + j * kWave, H4 - 1)] : float4{};
  combine_row<kCombThreads>(a, t, red, s_dyn, grp == 0);
  __syncthreads();
  if (e < r.sel.N) {
    const float4* xs4 = reinterpret_cast<const float4*>(s_dyn);
    const auto xf = [&](int h) { return xs4[h]; };
    const float acc = pre ? router_dot_pre(wp, H4, lane, xf) : router_dot(w4, H4, lane, xf);
    if (lane == 0) r.z[(size_t)t * r.sel.N + e] = acc;
  }
}

// ------------------------------------------------------------------ launch

template <typename K>
int occupancy_blocks(K kernel, size_t lds) {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kBlock, lds) != hipSuccess || n < 1)
    n = 1;
  return n;
}

// Grid: enough blocks to fill the device at the kernel's occupancy, never more
// than one wave per tile.
template <typename K>
hipError_t launch_persistent(K kernel, int max_tiles, size_t lds, const GroupedArgs& a,
                             hipStream_t s) {
  const hipError_t e = allow_lds(reinterpret_cast<const void*>(kernel), lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();  // the failure is returned here, not left for a later check
    return note_hip(e);
  }
  const int occ = occupancy_blocks(kernel, lds);
  const int cap = dev_info().num_cus * occ;
  const int want = cdiv(max_tiles, kWavesPB);
  const int g = want < 1 ? 1 : (want < cap ? want : cap);
  hipLaunchKernelGGL(kernel, dim3(g), dim3(kBlock), lds, s, a);
  return note_hip(hipGetLastError());
}

int max_tiles(const GroupedArgs& a, bool gateup, int rt) {
  const int per = gateup ? rt / 2 : rt;
  int t = a.has_routed ? a.r.max_union * cdiv(gateup ? a.r.inter : a.H, per) : 0;
  for (int s = 0; s < a.n_dense; ++s) t += cdiv(gateup ? a.dense[s].inter : a.dense[s].rows, per);
  return t;
}

template <typename WT>
size_t staged_bytes(int rows, int len) {
  return (size_t)rows * staged_stride<WTr<WT>::EPU>(len) * sizeof(float);
}

// The whole block of positions is staged in LDS when it fits the budget and
// holds more than one position.
// Small launches (fewer full tiles than the device has waves) use tiles of
// one (G, U) pair or two rows, so that more waves share the rows (one row per
// down tile measured slower, also for a single position, whose input is not
// staged: the dense layer at T = 1 took 54 instead of 48 us).
bool small_launch(const GroupedArgs& a, bool gateup) {
  return max_tiles(a, gateup, kNS) < dev_info().num_cus * 2 * kWavesPB;
}

// Two-row tiles for small launches and for a single position (read from
// global memory): the 2 x 10944 gate/up rows of a dense layer at T = 1 are
// 1.34 rounds of four-row tiles over the grid's waves (a second round a
// third full) and 1.78 rounds of two-row tiles.
template <typename WT, bool LDSX>
hipError_t gateup_tiles(const GroupedArgs& a, size_t lds, hipStream_t s) {
  if (small_launch(a, true) || !LDSX)
    return launch_persistent(gateup_kernel<WT, LDSX, 2>, max_tiles(a, true, 2), lds, a, s);
  return launch_persistent(gateup_kernel<WT, LDSX, kNS>, max_tiles(a, true, kNS), lds, a, s);
}

template <typename WT>
hipError_t gateup_typed(const GroupedArgs& a, hipStream_t s) {
  if (max_tiles(a, true, kNS) == 0) return hipSuccess;
  const size_t tabs = tables_bytes(a);
  const size_t lds = staged_bytes<WT>(a.T, a.H);
  // Staged unless a single position (read from global memory alongside the
  // weights, as in the down pass).
  if (lds + tabs <= (size_t)kLdsBudget && a.T > 1) return gateup_tiles<WT, true>(a, lds + tabs, s);
  return gateup_tiles<WT, false>(a, tabs, s);
}

// The down kernel stages the inputs of the sources a block visits: a fixed
// budget per block (two blocks per CU), which holds a row-dot's T input rows
// and the few members' rows of the grouped down in the common case.
template <typename WT>
hipError_t down_typed(GroupedArgs a, hipStream_t s) {
  if (max_tiles(a, false, kNS) == 0) return hipSuccess;
  const size_t tabs = tables_bytes(a);
  const size_t budget = (size_t)kDownLds > tabs + 4096 ? (size_t)kDownLds - tabs : 4096;
  a.lds_floats = (int)(budget / sizeof(float)) & ~3;
  const size_t lds = (size_t)a.lds_floats * sizeof(float) + tabs;
  if (small_launch(a, false))
    return launch_persistent(down_kernel<WT, 2>, max_tiles(a, false, 2), lds, a, s);
  return launch_persistent(down_kernel<WT, kNS>, max_tiles(a, false, kNS), lds, a, s);
}

}  // namespace

// Raises a kernel's dynamic LDS limit to `lds` when a launch needs more than
// the default 64 KB (once per kernel and size; the limit counts the kernel's
// static LDS too, so the request is the exact size, never a blanket maximum).
hipError_t allow_lds(const void* fn, size_t lds) {
  if (lds <= 64 * 1024) return hipSuccess;
  static std::mutex mu;
  static std::vector<std::pair<const void*, size_t>> granted;
  std::lock_guard<std::mutex> lock(mu);
  for (auto& g : granted)
    if (g.first == fn && g.second >= lds) return hipSuccess;
  const hipError_t e =
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  granted.emplace_back(fn, lds);
  return hipSuccess;
}

hipError_t launch_gateup(const GroupedArgs& a, int wdtype, hipStream_t s) {
  if (wdtype == DE_Q4_0) return gateup_typed<q4_t>(a, s);
  return wdtype == DE_BF16 ? gateup_typed<uint16_t>(a, s) : gateup_typed<float>(a, s);
}

hipError_t launch_down(const GroupedArgs& a, int wdtype, hipStream_t s) {
  if (wdtype == DE_Q4_0) return down_typed<q4_t>(a, s);
  return wdtype == DE_BF16 ? down_typed<uint16_t>(a, s) : down_typed<float>(a, s);
}

bool combine_route_fits(int H) { return H <= kCombThreads * kCombPer && H % 4 == 0; }

// True when the [T, H] fp32 rows at p and q share any byte.
static bool rows_overlap(const float* p, const float* q, int T, int H) {
  if (p == nullptr || q == nullptr) return false;
  const uintptr_t a = reinterpret_cast<uintptr_t>(p), b = reinterpret_cast<uintptr_t>(q);
  const uintptr_t n = (uintptr_t)T * H * sizeof(float);
  return a < b + n && b < a + n;
}

hipError_t launch_combine_route(const CombineArgs& a, const RouteArgs& r, hipStream_t s) {
  // The normalised row is held in LDS: a row that does not fit is an error.
  if (!combine_route_fits(a.H) || r.H != a.H) return note_hip(hipErrorInvalidValue);
  // Every block of a position re-reads its residual row while block 0 of the
  // position writes y and the normalised row: none of them may share memory.
  if (rows_overlap(a.residual, a.y, a.T, a.H) || rows_overlap(a.residual, a.normed, a.T, a.H) ||
      rows_overlap(a.y, a.normed, a.T, a.H))
    return note_hip(hipErrorInvalidValue);
  const int G = (r.sel.N + kCombThreads / kWave - 1) / (kCombThreads / kWave);
  hipLaunchKernelGGL(combine_route_kernel, dim3(a.T * G), dim3(kCombThreads), (size_t)a.H * 4, s,
                     a, r);
  return note_hip(hipGetLastError());
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(combine_kernel, dim3(a.T), dim3(kCombThreads), 0, s, a);
  return note_hip(hipGetLastError());
}

}  // namespace de
