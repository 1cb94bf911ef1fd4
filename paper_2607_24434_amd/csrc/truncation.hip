// Confidence-expansion truncation of the draft loop (Section 3.4, Eqs. 12-14;
// Algorithm 1): the confidence of a draft token's logits, and the predicted
// verifier set with the token's marginal expansion and the stop rule.
#include "de_common.h"

#include <climits>

namespace de {
namespace {

constexpr int kConfThreads = 1024;

// Running (max, sum of exp(l - max)) pair of a softmax denominator; a NaN
// logit counts as -infinity, as in the argmax.
struct SoftAcc {
  float m, s;
};

__device__ __forceinline__ SoftAcc soft_add(SoftAcc a, float v) {
  if (!(v == v) || v == -INFINITY) return a;
  if (v > a.m) {
    a.s = a.s * expf(a.m - v) + 1.f;
    a.m = v;
  } else {
    a.s += expf(v - a.m);
  }
  return a;
}

__device__ __forceinline__ SoftAcc soft_merge(SoftAcc a, SoftAcc b) {
  if (b.s == 0.f) return a;
  if (a.s == 0.f) return b;
  const float m = fmaxf(a.m, b.m);
  return SoftAcc{m, a.s * expf(a.m - m) + b.s * expf(b.m - m)};
}

// One block per row: q = 1 / sum_v exp(l_v - max l), the largest softmax
// probability.  A row without a finite-or-+inf logit gives q = NaN.
__global__ __launch_bounds__(kConfThreads) void confidence_kernel(const float* logits, int V,
                                                                  float* q) {
  __shared__ SoftAcc part[kConfThreads / 64];
  const float* p = logits + (size_t)blockIdx.x * V;
  SoftAcc acc{-INFINITY, 0.f};
  if ((reinterpret_cast<uintptr_t>(p) & 15u) == 0) {
    const int v4 = V / 4;
    const float4* p4 = reinterpret_cast<const float4*>(p);
    for (int i = threadIdx.x; i < v4; i += kConfThreads) {
      const float4 f = p4[i];
      acc = soft_add(acc, f.x);
      acc = soft_add(acc, f.y);
      acc = soft_add(acc, f.z);
      acc = soft_add(acc, f.w);
    }
    for (int i = v4 * 4 + threadIdx.x; i < V; i += kConfThreads) acc = soft_add(acc, p[i]);
  } else {
    for (int i = threadIdx.x; i < V; i += kConfThreads) acc = soft_add(acc, p[i]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const SoftAcc b{__shfl_xor(acc.m, o, kWave), __shfl_xor(acc.s, o, kWave)};
    acc = soft_merge(acc, b);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) part[wave] = acc;
  __syncthreads();
  if (threadIdx.x != 0) return;
  SoftAcc t = part[0];
  for (int w = 1; w < kConfThreads / 64; ++w) t = soft_merge(t, part[w]);
  q[blockIdx.x] = t.s > 0.f ? 1.f / t.s : __int_as_float(0x7fc00000);
}

constexpr int kExpThreads = 256;
constexpr int kMaxWords = 4;   // 256 experts per layer

__device__ __forceinline__ int block_sum(int v, int* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  int t = 0;
#pragma unroll
  for (int w = 0; w < kExpThreads / 64; ++w) t += red[w];
  return t;
}

// One block.  Layer l's predicted experts pred[l, 0..k) as a bit set against
// the layer's bits of the block-level set uhat (empty when `first`): the
// token's expansion (new pairs), the cache room (sum_l max(0, slots - set
// size of l)), the stop rule q < tau and expansion > budget (the room when
// budget < 0); the set grows only for a kept token.  out = (expansion, stop,
// budget used, set size after, ids out of range).
__global__ __launch_bounds__(kExpThreads) void expansion_kernel(ExpansionArgs a) {
  __shared__ int red[kExpThreads / 64];
  const int words = (a.N + 63) / 64;
  int delta = 0, room = 0, before = 0, grown = 0, bad = 0;
  for (int l = threadIdx.x; l < a.L; l += kExpThreads) {
    unsigned long long nw[kMaxWords] = {0ull, 0ull, 0ull, 0ull};
    for (int j = 0; j < a.k; ++j) {
      const int e = a.pred[(size_t)l * a.k + j];
      if (e < 0 || e >= a.N) {
        ++bad;
        continue;
      }
#pragma unroll
      for (int w = 0; w < kMaxWords; ++w)
        if ((e >> 6) == w) nw[w] |= 1ull << (e & 63);
    }
    int nb = 0, ng = 0;
#pragma unroll
    for (int w = 0; w < kMaxWords; ++w) {
      if (w < words) {
        const unsigned long long ow = a.first ? 0ull : a.uhat[(size_t)l * words + w];
        nb += __popcll(ow);
        ng += __popcll(ow | nw[w]);
      }
    }
    delta += ng - nb;
    before += nb;
    grown += ng;
    room += max(0, a.slots - nb);
  }
  delta = block_sum(delta, red);
  room = block_sum(room, red);
  before = block_sum(before, red);
  grown = block_sum(grown, red);
  bad = block_sum(bad, red);
  const float q = *a.q;
  const int budget = a.budget >= 0 ? a.budget : room;
  const bool stop = q < a.tau && delta > budget;
  // Commit (or, for the first token, clear) the set.
  for (int l = threadIdx.x; l < a.L; l += kExpThreads) {
    unsigned long long nw[kMaxWords] = {0ull, 0ull, 0ull, 0ull};
    if (!stop) {
      for (int j = 0; j < a.k; ++j) {
        const int e = a.pred[(size_t)l * a.k + j];
        if (e < 0 || e >= a.N) continue;
#pragma unroll
        for (int w = 0; w < kMaxWords; ++w)
          if ((e >> 6) == w) nw[w] |= 1ull << (e & 63);
      }
    }
#pragma unroll
    for (int w = 0; w < kMaxWords; ++w) {
      if (w < words) {
        const unsigned long long ow = a.first ? 0ull : a.uhat[(size_t)l * words + w];
        a.uhat[(size_t)l * words + w] = ow | nw[w];
      }
    }
  }
  if (threadIdx.x == 0) {
    a.out[0] = delta;
    a.out[1] = stop ? 1 : 0;
    a.out[2] = budget;
    a.out[3] = stop ? before : grown;
    a.out[4] = bad;
  }
}

}  // namespace

hipError_t launch_confidence(int T, int V, const float* logits, float* q, hipStream_t s) {
  hipLaunchKernelGGL(confidence_kernel, dim3(T), dim3(kConfThreads), 0, s, logits, V, q);
  return note_hip(hipGetLastError());
}

hipError_t launch_expansion(const ExpansionArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(expansion_kernel, dim3(1), dim3(kExpThreads), 0, s, a);
  return note_hip(hipGetLastError());
}

}  // namespace de
