// Router scoring (Eq. 1), top-k with gates (Eq. 4) and the block union with
// per-expert token lists (Eq. 2, Eq. 3), in one launch.
//
// route_kernel: ceil(N/16) blocks of 16 waves, one wave per expert.  A block
//   stages the block's activations in LDS, each wave streams its expert's
//   fp32 router row once (all of its float4 loads issued together) and dots
//   it with every position.  The last block to finish (device-scope counter,
//   release/acquire fences so logits written on other XCDs are visible) then
//   selects the top-k of every position, one wave per position, by repeated
//   wave-wide (key, id) argmax with ties to the lower id, and builds the union
//   with integer work only: a 64-bit position mask per expert, a wave prefix
//   scan over the experts for the list offsets, rank = popcount of the mask
//   below the position.  No floating-point arithmetic touches the union, so
//   it is bit-exact and deterministic.
// union_kernel: the same union build from caller-supplied top-k lists.
#include "de_common.h"

#include <climits>

namespace de {
namespace {

constexpr int kRouteThreads = 1024;
constexpr int kRouteWaves = kRouteThreads / kWave;  // experts per block
constexpr int kRouteLds = 136 * 1024;  // + ~20 KB of static selection state <= 160 KB
constexpr int kRouterTok = 16;                      // positions per accumulator pass
constexpr int kMaxT = 64;
constexpr int kMaxK = 32;
constexpr int kMaxN = 256;

extern __shared__ __align__(16) float s_x[];

// (key, id) candidate ordering: larger key first, equal keys to the lower id.
// id == INT_MAX marks "no candidate".
__device__ __forceinline__ bool better(float ka, int ea, float kb, int eb) {
  if (ea == INT_MAX) return false;
  if (eb == INT_MAX) return true;
  return ka > kb || (ka == kb && ea < eb);
}

struct SelShared {
  int32_t idx[kMaxT * kMaxK];
  float gate[kMaxT * kMaxK];
  unsigned long long mask[kMaxN];
  int32_t off[kMaxN];
  int32_t upos[kMaxN];
  int bad, nu, total;
};

// Top-k of every position from the logits z [T, N] (one wave per position),
// into s.idx / s.gate and the optional global outputs.
__device__ void select_topk(const TopkUnionArgs& a, SelShared& s) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const int T = a.T, N = a.N, k = a.k;
  for (int t = wave; t < T; t += nwaves) {
    float key[4], sc[4];
    bool taken[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane + q * kWave;
      const bool valid = e < N;
      const float zz = valid ? a.z[(size_t)t * N + e] : 0.f;
      const float b = (valid && a.bias != nullptr) ? a.bias[e] : 0.f;
      float kk, sv;
      if (a.score_func == 0) {  // softmax(z + b): key z + b
        kk = zz + b;
        sv = 0.f;
      } else {                  // sigmoid(z): key sigmoid(z) + b
        sv = 1.0f / (1.0f + expf(-zz));
        kk = sv + b;
      }
      if (!(kk == kk)) kk = -INFINITY;  // a NaN never wins
      key[q] = valid ? kk : -INFINITY;
      sc[q] = sv;
      taken[q] = !valid;
    }
    if (a.score_func == 0) {
      float m = -INFINITY;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (!taken[q]) m = fmaxf(m, key[q]);
      m = wave_max(m);
      float ex[4], sum = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        ex[q] = taken[q] ? 0.f : expf(key[q] - m);
        sum += ex[q];
      }
      sum = wave_sum(sum);
#pragma unroll
      for (int q = 0; q < 4; ++q) sc[q] = ex[q] / sum;
    }
    int my_e = 0;
    float my_s = 0.f, gsum = 0.f;
    for (int j = 0; j < k; ++j) {
      float bk = -INFINITY, bs = 0.f;
      int be = INT_MAX;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = lane + q * kWave;
        if (!taken[q] && better(key[q], e, bk, be)) {
          bk = key[q];
          be = e;
          bs = sc[q];
        }
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const float ok = __shfl_xor(bk, o, kWave);
        const int oe = __shfl_xor(be, o, kWave);
        const float os = __shfl_xor(bs, o, kWave);
        if (better(ok, oe, bk, be)) {
          bk = ok;
          be = oe;
          bs = os;
        }
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (lane + q * kWave == be) taken[q] = true;
      if (lane == j) {
        my_e = be;
        my_s = bs;
      }
      gsum += bs;
    }
    if (lane < k) {
      float g = my_s;
      if (a.norm_topk) g = g / gsum;
      g *= a.routed_scale;
      s.idx[t * k + lane] = my_e;
      s.gate[t * k + lane] = g;
      if (a.idx_out) a.idx_out[(size_t)t * k + lane] = my_e;
      if (a.gate_out) a.gate_out[(size_t)t * k + lane] = g;
    }
  }
}

// Union of the first ucols entries of every position's list in s.idx.
// Integer only.  Writes n_union = -1 for an id outside [0, N) or an id that
// repeats within one position.
__device__ void build_union(const TopkUnionArgs& a, SelShared& s) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nthreads = blockDim.x;
  const int T = a.T, N = a.N, k = a.k, uc = a.ucols;
  if (tid == 0) s.bad = 0;
  __syncthreads();
  for (int i = tid; i < T * uc; i += nthreads) {
    const int e = s.idx[(i / uc) * k + (i % uc)];
    if (e < 0 || e >= N) s.bad = 1;
  }
  for (int e = tid; e < N; e += nthreads) {
    unsigned long long mask = 0ull;
    bool dup = false;
    for (int t = 0; t < T; ++t) {
      for (int j = 0; j < uc; ++j) {
        if (s.idx[t * k + j] == e) {
          if ((mask >> t) & 1ull) dup = true;
          mask |= 1ull << t;
        }
      }
    }
    s.mask[e] = mask;
    if (dup) s.bad = 1;
  }
  __syncthreads();
  if (s.bad) {
    if (tid == 0) *a.n_union = -1;
    return;
  }
  // exclusive scans over experts in ascending id (wave 0, four ids per lane)
  if (wave == 0) {
    int cnt[4], flg[4], csum = 0, fsum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane * 4 + q;
      const unsigned long long m = e < N ? s.mask[e] : 0ull;
      cnt[q] = __popcll(m);
      flg[q] = m != 0ull;
      csum += cnt[q];
      fsum += flg[q];
    }
    int ci = csum, fi = fsum;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int cu = __shfl_up(ci, o, kWave);
      const int fu = __shfl_up(fi, o, kWave);
      if (lane >= o) {
        ci += cu;
        fi += fu;
      }
    }
    int cbase = ci - csum, fbase = fi - fsum;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane * 4 + q;
      if (e < N) {
        s.off[e] = cbase;
        s.upos[e] = fbase;
      }
      cbase += cnt[q];
      fbase += flg[q];
    }
    if (lane == kWave - 1) {
      s.nu = fi;
      s.total = ci;
    }
  }
  __syncthreads();
  const int nu = s.nu, total = s.total;
  for (int e = tid; e < N; e += nthreads) {
    if (s.mask[e] != 0ull) {
      a.union_ids[s.upos[e]] = e;
      a.offsets[s.upos[e]] = s.off[e];
    }
  }
  for (int u = nu + tid; u < N; u += nthreads) a.union_ids[u] = -1;
  for (int u = nu + tid; u <= N; u += nthreads) a.offsets[u] = total;
  if (tid == 0) *a.n_union = nu;
  for (int i = tid; i < T * uc; i += nthreads) {
    const int t = i / uc, j = i % uc;
    const int e = s.idx[t * k + j];
    const unsigned long long below = t == 0 ? 0ull : (s.mask[e] & (~0ull >> (64 - t)));
    const int p = s.off[e] + __popcll(below);
    a.tok_list[p] = t;
    a.gate_list[p] = s.gate[t * k + j];
    a.pair_pos[i] = p;
  }
}

template <bool XLDS>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(RouteArgs r) {
  __shared__ SelShared sel;
  __shared__ int s_last;
  const TopkUnionArgs& a = r.sel;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int T = a.T, H = r.H, N = a.N, H4 = H >> 2;
  if constexpr (XLDS) {
    for (int i = threadIdx.x; i < T * H4; i += kRouteThreads)
      reinterpret_cast<float4*>(s_x)[i] = reinterpret_cast<const float4*>(r.x)[i];
    __syncthreads();
  }
  const int e = blockIdx.x * kRouteWaves + wave;
  if (e < N) {
    const float4* wr = reinterpret_cast<const float4*>(r.w + (size_t)e * H);
    for (int h0 = 0; h0 < H4; h0 += kWave * 8) {
      float4 wv[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int h = h0 + lane + i * kWave;
        wv[i] = h < H4 ? wr[h] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
      for (int t0 = 0; t0 < T; t0 += kRouterTok) {
        float acc[kRouterTok];
#pragma unroll
        for (int m = 0; m < kRouterTok; ++m) acc[m] = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int h = h0 + lane + i * kWave;
          if (h < H4) {
#pragma unroll
            for (int m = 0; m < kRouterTok; ++m) {
              if (t0 + m < T) {
                const float4 xv = XLDS ? reinterpret_cast<const float4*>(s_x)[(t0 + m) * H4 + h]
                                       : reinterpret_cast<const float4*>(r.x)[(size_t)(t0 + m) * H4 + h];
                float v = acc[m];
                v = fmaf(wv[i].x, xv.x, v);
                v = fmaf(wv[i].y, xv.y, v);
                v = fmaf(wv[i].z, xv.z, v);
                v = fmaf(wv[i].w, xv.w, v);
                acc[m] = v;
              }
            }
          }
        }
#pragma unroll
        for (int m = 0; m < kRouterTok; ++m) {
          if (t0 + m < T) {
            const float sm = wave_sum(acc[m]);
            // Partial sums over h0 chunks accumulate in z (H > 2048 only).
            if (lane == 0) {
              float* zp = r.z + (size_t)(t0 + m) * N + e;
              *zp = h0 == 0 ? sm : *zp + sm;
            }
          }
        }
      }
    }
  }
  // ---- the last block to finish selects and builds the union.  The barrier
  // orders the block's logit stores before thread 0's device-scope release;
  // one fence per block (each is an L2 write-back on this part).
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    const unsigned prev = __hip_atomic_fetch_add(r.counter, 1u, __ATOMIC_ACQ_REL,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    s_last = prev == gridDim.x - 1;
    if (s_last) {
      __threadfence();
      __hip_atomic_store(r.counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  if (!s_last) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");  // every wave reads other blocks' logits
  select_topk(a, sel);
  if (a.n_union == nullptr) return;
  __syncthreads();
  build_union(a, sel);
}

__global__ __launch_bounds__(kRouteThreads) void union_kernel(TopkUnionArgs a) {
  __shared__ SelShared sel;
  for (int i = threadIdx.x; i < a.T * a.k; i += kRouteThreads) {
    sel.idx[i] = a.idx_in[i];
    sel.gate[i] = a.gate_in[i];
  }
  __syncthreads();
  build_union(a, sel);
}

}  // namespace

hipError_t launch_route(const RouteArgs& r, hipStream_t s) {
  const int grid = (r.sel.N + kRouteWaves - 1) / kRouteWaves;
  const size_t lds = (size_t)r.sel.T * r.H * sizeof(float);
  if (lds <= (size_t)kRouteLds) {
    static bool attr = false;
    if (!attr) {
      hipFuncSetAttribute(reinterpret_cast<const void*>(route_kernel<true>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kRouteLds);
      attr = true;
    }
    hipLaunchKernelGGL(route_kernel<true>, dim3(grid), dim3(kRouteThreads), lds, s, r);
  } else {
    hipLaunchKernelGGL(route_kernel<false>, dim3(grid), dim3(kRouteThreads), 0, s, r);
  }
  return hipGetLastError();
}

hipError_t launch_union(const TopkUnionArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(union_kernel, dim3(1), dim3(kRouteThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace de
