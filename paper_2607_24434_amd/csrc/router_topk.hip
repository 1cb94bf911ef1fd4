// Router scoring (Eq. 1), top-k with gates (Eq. 4) and the block union with
// per-expert token lists (Eq. 2, Eq. 3).
//
// scores_kernel: a 2-D grid of (4 experts) x (up to 8 positions) blocks.  A
//   block issues its experts' router-row loads, stages its positions'
//   activations in LDS with all loads in flight at once, and each wave dots
//   one expert's row with every staged position.  Logits go to z [T, N].
// select_kernel: one block.  Each wave takes one position: lane l holds the
//   candidates l, l+64, ...; a candidate's rank is the number of candidates
//   with a larger key (ties to the lower id), counted against every key
//   broadcast with readlane, so no chain of cross-lane shuffles is needed.
//   Rank < k places the candidate in the ordered top-k list.  The gates are
//   then normalised in list order and the union is built with integer work
//   only: a 64-bit position mask per expert, a wave prefix scan over the
//   experts for the list offsets, rank of a position = popcount of the mask
//   below it.  No floating-point arithmetic touches the union, so it is
//   bit-exact and deterministic.  The kernel boundary between the two
//   launches orders the logits before the selection.
// union_kernel: the same union build from caller-supplied top-k lists.
#include "de_common.h"

#include <climits>

namespace de {
namespace {

constexpr int kSelThreads = 1024;                 // select / union: one wave per position
constexpr int kScoreWaves = 4;                    // experts per scores block
constexpr int kScoreThreads = kScoreWaves * kWave;
constexpr int kScoreTok = 8;                      // positions per scores block (max)
constexpr int kScoreLds = 64 * 1024;              // staged activations per scores block
constexpr int kStageBatch = 16;                   // float4 loads in flight per thread
constexpr int kMaxT = 64;
constexpr int kMaxK = 32;
constexpr int kMaxN = 256;

extern __shared__ __align__(16) float s_x[];

struct SelShared {
  int32_t idx[kMaxT * kMaxK];
  float sc[kMaxT * kMaxK];    // score of each list entry
  float gate[kMaxT * kMaxK];
  unsigned long long mask[kMaxN];
  int32_t off[kMaxN];
  int32_t upos[kMaxN];
  int bad, nu, total;
};

// Top-k of every position from the logits z [T, N] (one wave per position),
// into s.idx / s.gate and the optional global outputs.  All threads.
__device__ void select_topk(const TopkUnionArgs& a, SelShared& s) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const int T = a.T, N = a.N, k = a.k;
  for (int t = wave; t < T; t += nwaves) {
    float key[4], sc[4];
    bool valid[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane + q * kWave;
      valid[q] = e < N;
      const float zz = valid[q] ? a.z[(size_t)t * N + e] : 0.f;
      const float b = (valid[q] && a.bias != nullptr) ? a.bias[e] : 0.f;
      float kk, sv;
      if (a.score_func == 0) {  // softmax(z + b): key z + b
        kk = zz + b;
        sv = 0.f;
      } else {                  // sigmoid(z): key sigmoid(z) + b
        sv = 1.0f / (1.0f + expf(-zz));
        kk = sv + b;
      }
      if (!(kk == kk)) kk = -INFINITY;  // a NaN never wins
      key[q] = valid[q] ? kk : -INFINITY;
      sc[q] = sv;
    }
    if (a.score_func == 0) {
      float m = -INFINITY;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (valid[q]) m = fmaxf(m, key[q]);
      m = wave_max(m);
      float ex[4], sum = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        ex[q] = valid[q] ? expf(key[q] - m) : 0.f;
        sum += ex[q];
      }
      sum = wave_sum(sum);
#pragma unroll
      for (int q = 0; q < 4; ++q) sc[q] = ex[q] / sum;
    }
    // rank[q] = number of candidates that beat candidate (key[q], id).
    int rank[4] = {0, 0, 0, 0};
#pragma unroll
    for (int q2 = 0; q2 < 4; ++q2) {
      if (q2 * kWave >= N) break;
      const int n2 = min(kWave, N - q2 * kWave);
      for (int l = 0; l < n2; ++l) {
        const float kb = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(key[q2]), l));
        const int eb = q2 * kWave + l;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int e = lane + q * kWave;
          rank[q] += (kb > key[q] || (kb == key[q] && eb < e)) ? 1 : 0;
        }
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (valid[q] && rank[q] < k) {
        s.idx[t * k + rank[q]] = lane + q * kWave;
        s.sc[t * k + rank[q]] = sc[q];
      }
    }
  }
  __syncthreads();
  // Gates in list order: g_j = score_j (/ sum of the k scores) * routed_scale.
  for (int i = threadIdx.x; i < T * k; i += blockDim.x) {
    const int t = i / k;
    float g = s.sc[i];
    if (a.norm_topk) {
      float gsum = 0.f;
      for (int j = 0; j < k; ++j) gsum += s.sc[t * k + j];
      g = g / gsum;
    }
    g *= a.routed_scale;
    s.gate[i] = g;
    if (a.idx_out) a.idx_out[i] = s.idx[i];
    if (a.gate_out) a.gate_out[i] = g;
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

// z[t0 + m, e] = W_r[e] . x[t0 + m] for the block's experts (one per wave) and
// positions.  With XLDS the positions are staged in LDS (all loads of a batch
// in flight before any store); otherwise they are read from global memory.
template <bool XLDS>
__global__ __launch_bounds__(kScoreThreads) void scores_kernel(RouteArgs r) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int T = r.sel.T, H = r.H, N = r.sel.N, H4 = H >> 2;
  const int t0 = blockIdx.y * r.tok_per_block;
  const int nt = min(r.tok_per_block, T - t0);
  const float4* xg = reinterpret_cast<const float4*>(r.x) + (size_t)t0 * H4;
  if constexpr (XLDS) {
    float4* sx = reinterpret_cast<float4*>(s_x);
    const int n4 = nt * H4;
    for (int i0 = 0; i0 < n4; i0 += kScoreThreads * kStageBatch) {
      float4 v[kStageBatch];
#pragma unroll
      for (int j = 0; j < kStageBatch; ++j)  // clamped: every load is in bounds, none is skipped
        v[j] = xg[min(i0 + j * kScoreThreads + (int)threadIdx.x, n4 - 1)];
#pragma unroll
      for (int j = 0; j < kStageBatch; ++j) {
        const int i = i0 + j * kScoreThreads + threadIdx.x;
        if (i < n4) sx[i] = v[j];
      }
    }
    __syncthreads();
  }
  const int e = blockIdx.x * kScoreWaves + wave;
  if (e >= N) return;
  const float4* wr = reinterpret_cast<const float4*>(r.w + (size_t)e * H);
  float acc[kScoreTok];
#pragma unroll
  for (int m = 0; m < kScoreTok; ++m) acc[m] = 0.f;
  for (int h0 = 0; h0 < H4; h0 += kWave * 8) {
    float4 wv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int h = h0 + lane + i * kWave;
      wv[i] = h < H4 ? wr[h] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int m = 0; m < kScoreTok; ++m) {
      if (m < nt) {
        float v = acc[m];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int h = h0 + lane + i * kWave;
          if (h < H4) {
            const float4 xv = XLDS ? reinterpret_cast<const float4*>(s_x)[m * H4 + h]
                                   : xg[(size_t)m * H4 + h];
            v = fmaf(wv[i].x, xv.x, v);
            v = fmaf(wv[i].y, xv.y, v);
            v = fmaf(wv[i].z, xv.z, v);
            v = fmaf(wv[i].w, xv.w, v);
          }
        }
        acc[m] = v;
      }
    }
  }
#pragma unroll
  for (int m = 0; m < kScoreTok; ++m) {
    if (m < nt) {
      const float sm = wave_sum(acc[m]);
      if (lane == 0) r.z[(size_t)(t0 + m) * N + e] = sm;
    }
  }
}

// Top-k of every position, then (when asked) the union.  One block.
__global__ __launch_bounds__(kSelThreads) void select_kernel(TopkUnionArgs a) {
  __shared__ SelShared sel;
  select_topk(a, sel);
  if (a.n_union == nullptr) return;
  __syncthreads();
  build_union(a, sel);
}

__global__ __launch_bounds__(kSelThreads) void union_kernel(TopkUnionArgs a) {
  __shared__ SelShared sel;
  for (int i = threadIdx.x; i < a.T * a.k; i += kSelThreads) {
    sel.idx[i] = a.idx_in[i];
    sel.gate[i] = a.gate_in[i];
  }
  __syncthreads();
  build_union(a, sel);
}

}  // namespace

hipError_t launch_route(const RouteArgs& r0, hipStream_t s) {
  RouteArgs r = r0;
  const int T = r.sel.T;
  // Positions per scores block: at most kScoreTok, fewer when a row is long,
  // spread evenly over the position chunks.
  const int fit = (int)(kScoreLds / ((size_t)r.H * sizeof(float)));
  const int cap = fit < 1 ? kScoreTok : (fit < kScoreTok ? fit : kScoreTok);
  const int chunks = (T + cap - 1) / cap;
  r.tok_per_block = (T + chunks - 1) / chunks;
  const dim3 grid((r.sel.N + kScoreWaves - 1) / kScoreWaves, chunks);
  if (fit >= 1) {
    const size_t lds = (size_t)r.tok_per_block * r.H * sizeof(float);
    hipLaunchKernelGGL(scores_kernel<true>, grid, dim3(kScoreThreads), lds, s, r);
  } else {
    hipLaunchKernelGGL(scores_kernel<false>, grid, dim3(kScoreThreads), 0, s, r);
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(select_kernel, dim3(1), dim3(kSelThreads), 0, s, r.sel);
  return hipGetLastError();
}

hipError_t launch_union(const TopkUnionArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(union_kernel, dim3(1), dim3(kSelThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace de
