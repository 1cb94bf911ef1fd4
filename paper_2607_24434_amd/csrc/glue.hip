// Acceptance (Algorithm 1, verify and accept), row argmax, RMSNorm,
// embedding gather and the streaming-read probe.
#include "de_common.h"

#include <climits>

namespace de {
namespace {

constexpr int kAmThreads = 256;
constexpr int kAmPer = 16;                        // logits per thread
constexpr int kAmChunk = kAmThreads * kAmPer;     // logits per block

// (value, index) ordering for argmax: larger value, then lower index; a NaN
// counts as -infinity; index INT_MAX marks "none".
__device__ __forceinline__ bool am_better(float va, int ia, float vb, int ib) {
  if (ia == INT_MAX) return false;
  if (ib == INT_MAX) return true;
  return va > vb || (va == vb && ia < ib);
}

constexpr int kRowThreads = 1024;

// K = 0: the argmax of the single row by one block (each thread scans a
// strided slice in 16-byte loads when the row allows), with no cross-block
// step; out = (0, argmax).
__global__ __launch_bounds__(kRowThreads) void argmax_row_kernel(AcceptArgs a) {
  __shared__ float sv[kRowThreads / 64];
  __shared__ int si[kRowThreads / 64];
  const float* p = a.logits;
  float bv = -INFINITY;
  int bi = INT_MAX;
  const auto offer = [&](float xv, int v) {
    if (!(xv == xv)) xv = -INFINITY;
    if (am_better(xv, v, bv, bi)) {
      bv = xv;
      bi = v;
    }
  };
  if ((a.V & 3) == 0 && (reinterpret_cast<uintptr_t>(p) & 15u) == 0) {
    const float4* p4 = reinterpret_cast<const float4*>(p);
    const int n4 = a.V >> 2;
#pragma unroll 4
    for (int j = threadIdx.x; j < n4; j += kRowThreads) {
      const float4 q = p4[j];
      offer(q.x, 4 * j);
      offer(q.y, 4 * j + 1);
      offer(q.z, 4 * j + 2);
      offer(q.w, 4 * j + 3);
    }
  } else {
    for (int v = threadIdx.x; v < a.V; v += kRowThreads) offer(p[v], v);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o, kWave);
    const int oi = __shfl_xor(bi, o, kWave);
    if (am_better(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    sv[wave] = bv;
    si[wave] = bi;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  for (int w = 1; w < kRowThreads / 64; ++w)
    if (am_better(sv[w], si[w], sv[0], si[0])) {
      sv[0] = sv[w];
      si[0] = si[w];
    }
  const int t = si[0] == INT_MAX ? 0 : si[0];
  a.amax[0] = t;
  a.out[0] = 0;
  a.out[1] = t;
}

// Grid (chunks, K+1).  Each block finds the argmax of one 4096-logit chunk of
// one row; the last block of a row (device-scope counter) reduces the row's
// chunk results in chunk order, and the last row to finish applies the greedy
// accept rule.  Counters are left at zero.
__global__ __launch_bounds__(kAmThreads) void argmax_accept_kernel(AcceptArgs a) {
  __shared__ float sv[kAmThreads / 64];
  __shared__ int si[kAmThreads / 64];
  __shared__ int s_flag;
  const int row = blockIdx.y, chunk = blockIdx.x, nch = gridDim.x;
  const float* p = a.logits + (size_t)row * a.V;
  const int base = chunk * kAmChunk;
  float x[kAmPer];
#pragma unroll
  for (int i = 0; i < kAmPer; ++i) {
    const int v = base + threadIdx.x + i * kAmThreads;
    x[i] = v < a.V ? p[v] : -INFINITY;
  }
  float bv = -INFINITY;
  int bi = INT_MAX;
#pragma unroll
  for (int i = 0; i < kAmPer; ++i) {
    const int v = base + threadIdx.x + i * kAmThreads;
    float xv = x[i];
    if (!(xv == xv)) xv = -INFINITY;
    if (v < a.V && am_better(xv, v, bv, bi)) {
      bv = xv;
      bi = v;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o, kWave);
    const int oi = __shfl_xor(bi, o, kWave);
    if (am_better(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    sv[wave] = bv;
    si[wave] = bi;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  for (int w = 1; w < kAmThreads / 64; ++w)
    if (am_better(sv[w], si[w], sv[0], si[0])) {
      sv[0] = sv[w];
      si[0] = si[w];
    }
  a.part_v[row * nch + chunk] = sv[0];
  a.part_i[row * nch + chunk] = si[0];
  __threadfence();
  const unsigned prev = __hip_atomic_fetch_add(&a.row_cnt[row], 1u, __ATOMIC_ACQ_REL,
                                               __HIP_MEMORY_SCOPE_AGENT);
  if (prev != (unsigned)nch - 1) return;
  __threadfence();
  float v = -INFINITY;
  int i = INT_MAX;
  for (int c = 0; c < nch; ++c)
    if (am_better(a.part_v[row * nch + c], a.part_i[row * nch + c], v, i)) {
      v = a.part_v[row * nch + c];
      i = a.part_i[row * nch + c];
    }
  a.amax[row] = i == INT_MAX ? 0 : i;
  __hip_atomic_store(&a.row_cnt[row], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __threadfence();
  const unsigned done = __hip_atomic_fetch_add(a.done_cnt, 1u, __ATOMIC_ACQ_REL,
                                               __HIP_MEMORY_SCOPE_AGENT);
  if (done != (unsigned)gridDim.y - 1) return;
  __threadfence();
  __hip_atomic_store(a.done_cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  int n = 0;
  while (n < a.K && a.drafts[n] == a.amax[n]) ++n;
  a.out[0] = n;
  a.out[1] = a.amax[n];
  (void)s_flag;
}

__device__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const float t = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return t;
}

__global__ __launch_bounds__(256) void rmsnorm_kernel(int H, const float* __restrict__ x, float eps,
                                                      float* out) {
  __shared__ float red[4];
  const size_t off = (size_t)blockIdx.x * H;
  float ss = 0.f;
  for (int h = threadIdx.x; h < H; h += 256) ss = fmaf(x[off + h], x[off + h], ss);
  ss = block_sum256(ss, red);
  const float r = 1.0f / sqrtf(ss / (float)H + eps);
  for (int h = threadIdx.x; h < H; h += 256) out[off + h] = x[off + h] * r;
}

// A token id outside [0, V) reads no embedding row: its h (and normed) row is
// NaN, so nothing downstream passes for a real token, and *status (when not
// NULL) receives kStatusBadToken.
__global__ __launch_bounds__(256) void embed_kernel(int H, int V, const int32_t* __restrict__ tokens,
                                                    const uint16_t* __restrict__ emb, float* h,
                                                    float* normed, float eps, int32_t* status) {
  __shared__ float red[4];
  const int tok = tokens[blockIdx.x];
  const size_t off = (size_t)blockIdx.x * H;
  if (tok < 0 || tok >= V) {
    for (int i = threadIdx.x; i < H; i += 256) {
      h[off + i] = __builtin_nanf("");
      if (normed) normed[off + i] = __builtin_nanf("");
    }
    if (threadIdx.x == 0 && status != nullptr)
      __hip_atomic_fetch_or(status, kStatusBadToken, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  const uint16_t* row = emb + (size_t)tok * H;
  float ss = 0.f;
  for (int i = threadIdx.x; i < H; i += 256) {
    const float v = __uint_as_float((uint32_t)row[i] << 16);
    h[off + i] = v;
    ss = fmaf(v, v, ss);
  }
  if (normed) {
    ss = block_sum256(ss, red);
    const float r = 1.0f / sqrtf(ss / (float)H + eps);
    for (int i = threadIdx.x; i < H; i += 256) normed[off + i] = h[off + i] * r;
  }
}

__global__ __launch_bounds__(256) void stream_probe_kernel(const u32x4* __restrict__ p, size_t n,
                                                           float* sink) {
  uint32_t acc = 0;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const u32x4 a = __builtin_nontemporal_load(p + i);
    const u32x4 b = __builtin_nontemporal_load(p + i + stride);
    const u32x4 c = __builtin_nontemporal_load(p + i + 2 * stride);
    const u32x4 d = __builtin_nontemporal_load(p + i + 3 * stride);
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < n; i += stride) {
    const u32x4 a = __builtin_nontemporal_load(p + i);
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  // The store is never taken for real data, but the loads cannot be dropped.
  if (acc == 0x9E3779B9u) sink[0] = (float)acc;
}

}  // namespace

int accept_chunks(int V) { return (V + kAmChunk - 1) / kAmChunk; }

hipError_t launch_argmax_accept(const AcceptArgs& a, hipStream_t s) {
  if (a.K == 0) {
    hipLaunchKernelGGL(argmax_row_kernel, dim3(1), dim3(kRowThreads), 0, s, a);
    return note_hip(hipGetLastError());
  }
  hipLaunchKernelGGL(argmax_accept_kernel, dim3(accept_chunks(a.V), a.K + 1), dim3(kAmThreads), 0,
                     s, a);
  return note_hip(hipGetLastError());
}

hipError_t launch_rmsnorm(int T, int H, const float* x, float eps, float* out, hipStream_t s) {
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(T), dim3(256), 0, s, H, x, eps, out);
  return note_hip(hipGetLastError());
}

hipError_t launch_embed(int T, int H, int V, const int32_t* tokens, const uint16_t* emb, float* h,
                        float* normed, float eps, int32_t* status, hipStream_t s) {
  hipLaunchKernelGGL(embed_kernel, dim3(T), dim3(256), 0, s, H, V, tokens, emb, h, normed, eps,
                     status);
  return note_hip(hipGetLastError());
}

hipError_t launch_stream_probe(const void* buf, size_t bytes, float* sink, hipStream_t s) {
  const size_t n = bytes / 16;
  const int grid = dev_info().num_cus * 8;
  hipLaunchKernelGGL(stream_probe_kernel, dim3(grid), dim3(256), 0, s,
                     static_cast<const u32x4*>(buf), n, sink);
  return note_hip(hipGetLastError());
}

}  // namespace de
