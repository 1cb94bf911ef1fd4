// Router scoring (Eq. 1) with the top-k and gates (Eq. 1, Eq. 4) in one
// launch, and the standalone union launch (Eq. 2, Eq. 3).
//
// route_split_kernel: (position, 16 experts) blocks compute the logits; the
//   last block of each position selects its ordered top-k (the grouped
//   gate/up kernel's prologue then builds the union from the lists in every
//   block).
// union_kernel: the union from caller-supplied top-k lists.
#include "de_common.h"
#include "topk_union.h"

#include <climits>

namespace de {
namespace {

constexpr int kSelThreads = 1024;                 // union kernel
constexpr int kRsThreads = 1024;                  // route: 16 experts per block, one per wave
constexpr int kRsWaves = kRsThreads / kWave;
constexpr int kMaxT = 64;
constexpr int kMaxK = 32;
constexpr int kMaxN = 256;


// Fixed-size selection state of the standalone kernels (T <= 64, k <= 32,
// N <= 256).
struct SelShared {
  int32_t idx[kMaxT * kMaxK];
  float sc[kMaxT * kMaxK];
  float gate[kMaxT * kMaxK];
  unsigned long long mask[kMaxN];
  int32_t off[kMaxN];
  int32_t upos[kMaxN];
  int32_t misc[4];
};

__device__ inline SelView view_of(SelShared& s) {
  return SelView{s.idx, s.sc, s.gate, s.mask, s.off, s.upos, s.misc};
}

// Block (t, g) (see the index map below): router logits of position t
// (Eq. 1) for experts 16g .. 16g+15, one per wave, each router row's and x_t's loads in flight
// together.  The logits go to z.  With r.select, the last of the position's
// blocks to finish (device-scope counter, release / acquire fences so logits
// written on other XCDs are visible; the counter is left at zero) selects the
// position's ordered top-k and gates.
__global__ __launch_bounds__(kRsThreads) void route_split_kernel(RouteArgs r) {
  __shared__ int32_t lidx[kMaxK];
  __shared__ float lsc[kMaxK];
  __shared__ int s_last;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // Block L is (position L / G, expert group L % G): workgroups go to the
  // XCDs round-robin by index, so the blocks of one expert group share a
  // few XCDs' L2 caches and read its router rows from memory once per XCD
  // instead of once per position.
  const int G = (r.sel.N + kRsWaves - 1) / kRsWaves;
  const int t = blockIdx.x / G, grp = blockIdx.x - t * G;
  const int H4 = r.H >> 2, N = r.sel.N, k = r.sel.k;
  const float4* xg = reinterpret_cast<const float4*>(r.x) + (size_t)t * H4;
  const float4* w4 = reinterpret_cast<const float4*>(r.w);
  const int e = grp * kRsWaves + wave;
  if (e < N) {
    const float acc = router_dot(w4 + (size_t)e * H4, H4, lane, [&](int h) { return xg[h]; });
    if (lane == 0) r.z[(size_t)t * N + e] = acc;
  }
  if (!r.select) return;
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    const unsigned prev = __hip_atomic_fetch_add(r.counter + t, 1u, __ATOMIC_ACQ_REL,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    s_last = prev == (unsigned)G - 1;
    if (s_last) __hip_atomic_store(r.counter + t, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!s_last) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  if (wave == 0) topk_row(r.sel, r.z + (size_t)t * N, lidx, lsc);
  __syncthreads();
  if (threadIdx.x < k) {
    const int i = t * k + threadIdx.x;
    r.sel.idx_out[i] = lidx[threadIdx.x];
    r.sel.gate_out[i] = topk_gate(r.sel, lsc, threadIdx.x);
  }
}

__global__ __launch_bounds__(kSelThreads) void union_kernel(TopkUnionArgs a) {
  __shared__ SelShared sel;
  const SelView v = view_of(sel);
  for (int i = threadIdx.x; i < a.T * a.k; i += kSelThreads) {
    sel.idx[i] = a.idx_in[i];
    sel.gate[i] = a.gate_in[i];
  }
  __syncthreads();
  build_union(a, v, true, nullptr, nullptr);
}

}  // namespace

// Grid (T, ceil(N / 16)): every (position, 16 experts) pair in its own block,
// so all the router rows of a position stream in parallel and each position's
// selection (when r.select) runs in its own last block.
hipError_t launch_route(const RouteArgs& r, hipStream_t s) {
  const int G = (r.sel.N + kRsWaves - 1) / kRsWaves;
  hipLaunchKernelGGL(route_split_kernel, dim3(r.sel.T * G), dim3(kRsThreads), 0, s, r);
  return note_hip(hipGetLastError());
}

hipError_t launch_union(const TopkUnionArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(union_kernel, dim3(1), dim3(kSelThreads), 0, s, a);
  return note_hip(hipGetLastError());
}

}  // namespace de
