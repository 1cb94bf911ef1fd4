// Acceptance (Algorithm 1, verify and accept), row argmax, RMSNorm,
// embedding gather and the streaming-read probe.
#include "de_common.h"

#include <climits>

namespace de {
namespace {

constexpr int kArgmaxThreads = 1024;

// (value, index) ordering for argmax: larger value, then lower index; a NaN
// counts as -infinity.
__device__ __forceinline__ bool am_better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

__global__ __launch_bounds__(kArgmaxThreads) void argmax_rows_kernel(const float* __restrict__ logits,
                                                                     int V, int32_t* __restrict__ amax) {
  __shared__ float sv[kArgmaxThreads / 64];
  __shared__ int si[kArgmaxThreads / 64];
  const int row = blockIdx.x;
  const float* p = logits + (size_t)row * V;
  float bv = -INFINITY;
  int bi = INT_MAX;
  for (int v = threadIdx.x; v < V; v += blockDim.x) {
    float x = p[v];
    if (!(x == x)) x = -INFINITY;
    if (bi == INT_MAX || am_better(x, v, bv, bi)) {
      bv = x;
      bi = v;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o, kWave);
    const int oi = __shfl_xor(bi, o, kWave);
    if (oi != INT_MAX && (bi == INT_MAX || am_better(ov, oi, bv, bi))) {
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
  if (threadIdx.x == 0) {
    float v = sv[0];
    int i = si[0];
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w)
      if (si[w] != INT_MAX && (i == INT_MAX || am_better(sv[w], si[w], v, i))) {
        v = sv[w];
        i = si[w];
      }
    amax[row] = i == INT_MAX ? 0 : i;
  }
}

__global__ void accept_kernel(int K, const int32_t* __restrict__ amax,
                              const int32_t* __restrict__ drafts, int32_t* __restrict__ out) {
  if (threadIdx.x != 0) return;
  int n = 0;
  while (n < K && drafts[n] == amax[n]) ++n;
  out[0] = n;
  out[1] = amax[n];
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

__global__ __launch_bounds__(256) void embed_kernel(int H, int V, const int32_t* __restrict__ tokens,
                                                    const uint16_t* __restrict__ emb, float* h,
                                                    float* normed, float eps) {
  __shared__ float red[4];
  int tok = tokens[blockIdx.x];
  tok = tok < 0 ? 0 : (tok >= V ? V - 1 : tok);
  const uint16_t* row = emb + (size_t)tok * H;
  const size_t off = (size_t)blockIdx.x * H;
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

hipError_t launch_argmax_rows(const float* logits, int rows, int V, int32_t* amax, hipStream_t s) {
  hipLaunchKernelGGL(argmax_rows_kernel, dim3(rows), dim3(kArgmaxThreads), 0, s, logits, V, amax);
  return hipGetLastError();
}

hipError_t launch_accept(int K, const int32_t* amax, const int32_t* drafts, int32_t* out,
                         hipStream_t s) {
  hipLaunchKernelGGL(accept_kernel, dim3(1), dim3(64), 0, s, K, amax, drafts, out);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(int T, int H, const float* x, float eps, float* out, hipStream_t s) {
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(T), dim3(256), 0, s, H, x, eps, out);
  return hipGetLastError();
}

hipError_t launch_embed(int T, int H, int V, const int32_t* tokens, const uint16_t* emb, float* h,
                        float* normed, float eps, hipStream_t s) {
  hipLaunchKernelGGL(embed_kernel, dim3(T), dim3(256), 0, s, H, V, tokens, emb, h, normed, eps);
  return hipGetLastError();
}

hipError_t launch_stream_probe(const void* buf, size_t bytes, float* sink, hipStream_t s) {
  const size_t n = bytes / 16;
  const int grid = dev_info().num_cus * 8;
  hipLaunchKernelGGL(stream_probe_kernel, dim3(grid), dim3(256), 0, s,
                     static_cast<const u32x4*>(buf), n, sink);
  return hipGetLastError();
}

}  // namespace de
