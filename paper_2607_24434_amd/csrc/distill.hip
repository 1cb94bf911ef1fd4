// Self-distillation signals as by-products of a verify pass (Section 3.3,
// Eqs. 6-10): the residual target from the layer's routed partials, and row
// divergences between target and draft distributions (router agreement,
// temperature-scaled logit KL, token cross entropy).
#include "de_common.h"

#include <climits>

namespace de {
namespace {

constexpr int kResThreads = 256;

// m*[t] = sum_{j = 1 .. kk-1} P[pair_pos[t, j]]: the routed partials of
// position t without its top-1 expert's, in list order (entries outside the
// partial rows are skipped).  Grid (T, column chunks).
__global__ __launch_bounds__(kResThreads) void residual_kernel(ResidualArgs a) {
  const int t = blockIdx.x;
  const int h = blockIdx.y * kResThreads + threadIdx.x;
  if (h >= a.H) return;
  float m = 0.f;
  for (int j = 1; j < a.kk; ++j) {
    const int p = a.pair_pos[(size_t)t * a.kk + j];
    if (p >= 0 && p < a.pairs_max) m += a.p_r[(size_t)p * a.H + h];
  }
  a.out[(size_t)t * a.H + h] = m;
}

constexpr int kKlThreads = 256;

// Running (max, sum exp(v - max)).
struct Lse {
  float m, s;
};

__device__ __forceinline__ Lse lse_add(Lse a, float v) {
  if (v > a.m) {
    a.s = a.s * expf(a.m - v) + 1.f;
    a.m = v;
  } else {
    a.s += expf(v - a.m);
  }
  return a;
}

__device__ __forceinline__ Lse lse_merge(Lse a, Lse b) {
  if (b.s == 0.f) return a;
  if (a.s == 0.f) return b;
  const float m = fmaxf(a.m, b.m);
  return Lse{m, a.s * expf(a.m - m) + b.s * expf(b.m - m)};
}

__device__ __forceinline__ float lse_val(Lse a) { return a.m + logf(a.s); }

// log sigmoid(z) without overflow.
__device__ __forceinline__ float log_sigmoid(float z) {
  return z < 0.f ? z - log1pf(expf(z)) : -log1pf(expf(-z));
}

// Reduces v over the block with op (every thread receives the result); the
// members of V are floats.
template <typename V, typename Op>
__device__ __forceinline__ V block_reduce(V v, V* red, Op op, V zero) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    V w;
    w = v;
    // Shuffle each float member.
    float* pv = reinterpret_cast<float*>(&w);
#pragma unroll
    for (int i = 0; i < (int)(sizeof(V) / 4); ++i) pv[i] = __shfl_xor(pv[i], o, kWave);
    v = op(v, w);
  }
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  V t = zero;
  for (int w = 0; w < kKlThreads / 64; ++w) t = op(t, red[w]);
  return t;
}

struct LseOp {
  __device__ Lse operator()(Lse a, Lse b) const { return lse_merge(a, b); }
};

struct Best {
  float v;
  float i;  // index as float bits (shuffled as a float)
};

// Larger value, then lower index; index INT_MAX marks "none".
struct BestOp {
  __device__ Best operator()(Best a, Best b) const {
    const int ia = __float_as_int(a.i), ib = __float_as_int(b.i);
    if (ib == INT_MAX) return a;
    if (ia == INT_MAX) return b;
    return (b.v > a.v || (b.v == a.v && ib < ia)) ? b : a;
  }
};

struct Sum {
  float s;
};
struct SumOp {
  __device__ Sum operator()(Sum a, Sum b) const { return Sum{a.s + b.s}; }
};

// One block per row r: a = target row, b = draft row (n values each).
// softmax mode (sigmoid == 0): p = softmax((a + bias) / tau), q likewise from
// b; kl = tau^2 KL(p || q).  sigmoid mode: p = sigmoid(a) normalised to sum
// one, q likewise; kl = KL(p || q).  ce (optional) = -log softmax(b + bias)
// at the argmax of a + bias (ties to the lower index).
__global__ __launch_bounds__(kKlThreads) void rowkl_kernel(RowKlArgs a) {
  __shared__ Lse rl[kKlThreads / 64];
  __shared__ Best rb[kKlThreads / 64];
  __shared__ Sum rs[kKlThreads / 64];
  const float* pa = a.a + (size_t)blockIdx.x * a.lda;
  const float* pb = a.b + (size_t)blockIdx.x * a.ldb;
  const float it = 1.f / a.tau;
  Lse la{-INFINITY, 0.f}, lb{-INFINITY, 0.f}, lb1{-INFINITY, 0.f};
  Best best{-INFINITY, __int_as_float(INT_MAX)};
  for (int i = threadIdx.x; i < a.n; i += kKlThreads) {
    const float bias = a.bias ? a.bias[i] : 0.f;
    const float va = pa[i], vb = pb[i];
    if (a.sigmoid) {
      la = lse_add(la, log_sigmoid(va));
      lb = lse_add(lb, log_sigmoid(vb));
    } else {
      la = lse_add(la, (va + bias) * it);
      lb = lse_add(lb, (vb + bias) * it);
      lb1 = lse_add(lb1, vb + bias);
    }
    // Argmax of a + bias; a NaN counts as -infinity, as in the argmax.
    const float vc = va == va ? va + bias : -INFINITY;
    const int bi = __float_as_int(best.i);
    if (bi == INT_MAX || vc > best.v) best = Best{vc, __int_as_float(i)};
  }
  la = block_reduce(la, rl, LseOp{}, Lse{-INFINITY, 0.f});
  lb = block_reduce(lb, rl, LseOp{}, Lse{-INFINITY, 0.f});
  lb1 = block_reduce(lb1, rl, LseOp{}, Lse{-INFINITY, 0.f});
  best = block_reduce(best, rb, BestOp{}, Best{-INFINITY, __int_as_float(INT_MAX)});
  const float lsa = lse_val(la), lsb = lse_val(lb);
  float acc = 0.f;
  for (int i = threadIdx.x; i < a.n; i += kKlThreads) {
    const float bias = a.bias ? a.bias[i] : 0.f;
    float xa, xb;
    if (a.sigmoid) {
      xa = log_sigmoid(pa[i]) - lsa;
      xb = log_sigmoid(pb[i]) - lsb;
    } else {
      xa = (pa[i] + bias) * it - lsa;
      xb = (pb[i] + bias) * it - lsb;
    }
    acc += expf(xa) * (xa - xb);
  }
  const Sum tot = block_reduce(Sum{acc}, rs, SumOp{}, Sum{0.f});
  if (threadIdx.x == 0) {
    a.kl[blockIdx.x] = a.sigmoid ? tot.s : a.tau * a.tau * tot.s;
    if (a.ce != nullptr) {
      const int t = __float_as_int(best.i);
      const float bias = (a.bias && t != INT_MAX) ? a.bias[t] : 0.f;
      a.ce[blockIdx.x] = t == INT_MAX ? __int_as_float(0x7fc00000)
                                      : lse_val(lb1) - (pb[t] + bias);
    }
  }
}

}  // namespace

hipError_t launch_residual(const ResidualArgs& a, hipStream_t s) {
  const dim3 grid(a.T, (a.H + kResThreads - 1) / kResThreads);
  hipLaunchKernelGGL(residual_kernel, grid, dim3(kResThreads), 0, s, a);
  return note_hip(hipGetLastError());
}

hipError_t launch_rowkl(const RowKlArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(rowkl_kernel, dim3(a.rows), dim3(kKlThreads), 0, s, a);
  return note_hip(hipGetLastError());
}

}  // namespace de
