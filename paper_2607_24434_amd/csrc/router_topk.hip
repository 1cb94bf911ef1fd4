// Router scoring (Eq. 1), top-k with gates (Eq. 4) and the block union with
// per-expert token lists (Eq. 2, Eq. 3).
//
// router_logits_kernel: one wave per expert; the wave streams that expert's
//   fp32 router row once (coalesced float4 loads) and dots it with every
//   block position; 64-lane shuffle reduction.
// topk_union_kernel: one workgroup.  One wave per block position selects the
//   top-k by repeated wave-wide (key, id) argmax with ties to the lower id;
//   then the union is built with integer work only: a 64-bit position mask
//   per expert, a wave prefix scan over the experts for the list offsets, and
//   rank = popcount of the mask below the position.  No floating-point
//   arithmetic touches the union, so it is bit-exact and deterministic.
#include "de_common.h"

#include <climits>

namespace de {
namespace {

constexpr int kRouterTok = 8;

__global__ __launch_bounds__(256) void router_logits_kernel(const float* __restrict__ x,
                                                            const float* __restrict__ w, int T,
                                                            int H, int N, float* __restrict__ z) {
  const int lane = threadIdx.x & 63;
  const int e = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (e >= N) return;
  const float4* wr = reinterpret_cast<const float4*>(w + (size_t)e * H);
  const int H4 = H >> 2;
  for (int t0 = 0; t0 < T; t0 += kRouterTok) {
    const int nt = min(kRouterTok, T - t0);
    float acc[kRouterTok];
#pragma unroll
    for (int m = 0; m < kRouterTok; ++m) acc[m] = 0.f;
    for (int h = lane; h < H4; h += kWave) {
      const float4 wv = wr[h];
#pragma unroll
      for (int m = 0; m < kRouterTok; ++m) {
        if (m < nt) {
          const float4 xv = reinterpret_cast<const float4*>(x + (size_t)(t0 + m) * H)[h];
          float a = acc[m];
          a = fmaf(wv.x, xv.x, a);
          a = fmaf(wv.y, xv.y, a);
          a = fmaf(wv.z, xv.z, a);
          a = fmaf(wv.w, xv.w, a);
          acc[m] = a;
        }
      }
    }
#pragma unroll
    for (int m = 0; m < kRouterTok; ++m) {
      if (m < nt) {
        const float s = wave_sum(acc[m]);
        if (lane == 0) z[(size_t)(t0 + m) * N + e] = s;
      }
    }
  }
}

constexpr int kMaxT = 64;
constexpr int kMaxK = 32;
constexpr int kMaxN = 256;
constexpr int kTopkThreads = 256;

// (key, id) candidate ordering: larger key first, equal keys to the lower id.
// id == INT_MAX marks "no candidate".
__device__ __forceinline__ bool better(float ka, int ea, float kb, int eb) {
  if (ea == INT_MAX) return false;
  if (eb == INT_MAX) return true;
  return ka > kb || (ka == kb && ea < eb);
}

__global__ __launch_bounds__(kTopkThreads) void topk_union_kernel(TopkUnionArgs a) {
  __shared__ int32_t s_idx[kMaxT * kMaxK];
  __shared__ float s_gate[kMaxT * kMaxK];
  __shared__ unsigned long long s_mask[kMaxN];
  __shared__ int32_t s_off[kMaxN];
  __shared__ int32_t s_upos[kMaxN];
  __shared__ int s_bad, s_nu, s_total;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int T = a.T, N = a.N, k = a.k;
  if (tid == 0) s_bad = 0;

  if (a.z != nullptr) {
    // ---- selection: one wave per block position
    for (int t = wave; t < T; t += kTopkThreads / kWave) {
      float key[4], sc[4];
      bool taken[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = lane + q * kWave;
        const bool valid = e < N;
        const float zz = valid ? a.z[(size_t)t * N + e] : 0.f;
        const float b = (valid && a.bias != nullptr) ? a.bias[e] : 0.f;
        float kk, s;
        if (a.score_func == 0) {  // softmax(z + b): key z + b
          kk = zz + b;
          s = 0.f;
        } else {                  // sigmoid(z): key sigmoid(z) + b
          s = 1.0f / (1.0f + expf(-zz));
          kk = s + b;
        }
        if (!(kk == kk)) kk = -INFINITY;  // a NaN never wins
        key[q] = valid ? kk : -INFINITY;
        sc[q] = s;
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
        s_idx[t * k + lane] = my_e;
        s_gate[t * k + lane] = g;
        if (a.idx_out) a.idx_out[(size_t)t * k + lane] = my_e;
        if (a.gate_out) a.gate_out[(size_t)t * k + lane] = g;
      }
    }
  } else {
    for (int i = tid; i < T * k; i += kTopkThreads) {
      s_idx[i] = a.idx_in[i];
      s_gate[i] = a.gate_in[i];
    }
  }
  if (a.n_union == nullptr) return;
  __syncthreads();

  // ---- union: per-expert position masks
  const int uc = a.ucols;
  for (int i = tid; i < T * uc; i += kTopkThreads) {
    const int e = s_idx[(i / uc) * k + (i % uc)];
    if (e < 0 || e >= N) s_bad = 1;
  }
  for (int e = tid; e < N; e += kTopkThreads) {
    unsigned long long mask = 0ull;
    bool dup = false;
    for (int t = 0; t < T; ++t) {
      for (int j = 0; j < uc; ++j) {
        if (s_idx[t * k + j] == e) {
          if ((mask >> t) & 1ull) dup = true;
          mask |= 1ull << t;
        }
      }
    }
    s_mask[e] = mask;
    if (dup) s_bad = 1;
  }
  __syncthreads();
  if (s_bad) {
    if (tid == 0) *a.n_union = -1;
    return;
  }

  // ---- exclusive scans over experts (ascending id) in wave 0
  if (wave == 0) {
    int cnt[4], flg[4], csum = 0, fsum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane * 4 + q;
      const unsigned long long m = e < N ? s_mask[e] : 0ull;
      cnt[q] = __popcll(m);
      flg[q] = m != 0ull;
      csum += cnt[q];
      fsum += flg[q];
    }
    int ci = csum, fi = fsum;  // inclusive wave scans
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
        s_off[e] = cbase;
        s_upos[e] = fbase;
      }
      cbase += cnt[q];
      fbase += flg[q];
    }
    if (lane == kWave - 1) {
      s_nu = fi;
      s_total = ci;
    }
  }
  __syncthreads();
  const int nu = s_nu, total = s_total;
  for (int e = tid; e < N; e += kTopkThreads) {
    if (s_mask[e] != 0ull) {
      a.union_ids[s_upos[e]] = e;
      a.offsets[s_upos[e]] = s_off[e];
    }
  }
  for (int u = nu + tid; u < N; u += kTopkThreads) a.union_ids[u] = -1;
  for (int u = nu + tid; u <= N; u += kTopkThreads) a.offsets[u] = total;
  if (tid == 0) *a.n_union = nu;
  for (int i = tid; i < T * uc; i += kTopkThreads) {
    const int t = i / uc, j = i % uc;
    const int e = s_idx[t * k + j];
    const unsigned long long below = t == 0 ? 0ull : (s_mask[e] & (~0ull >> (64 - t)));
    const int p = s_off[e] + __popcll(below);
    a.tok_list[p] = t;
    a.gate_list[p] = s_gate[t * k + j];
    a.pair_pos[i] = p;
  }
}

}  // namespace

hipError_t launch_router_logits(const float* x, const float* w, int T, int H, int N, float* z,
                                hipStream_t s) {
  hipLaunchKernelGGL(router_logits_kernel, dim3((N + 3) / 4), dim3(256), 0, s, x, w, T, H, N, z);
  return hipGetLastError();
}

hipError_t launch_topk_union(const TopkUnionArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(topk_union_kernel, dim3(1), dim3(kTopkThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace de
