// GPU fill of the seeded synthetic streams of workloads/rng.py, bit for bit.
//
// Element i of the stream with key k is mix64(k + (i + 1) * GAMMA) (SplitMix64
// in counter mode); its four 16-bit fields are summed and centred
// (Irwin-Hall, n = 4), scaled by one fp64 multiply, rounded to fp32 and, for
// bf16 output, rounded to nearest-even bf16.  Every step is either integer or
// a single correctly rounded IEEE operation, so the CPU and GPU agree exactly.
// This library only draws inputs; it is not part of the hot path.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ void fill_normal_kernel(void* out, int64_t n, int bf16, uint64_t key, uint64_t start,
                                   double scale) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint64_t z = mix64(key + (start + (uint64_t)i + 1ull) * kGamma);
    const int s = (int)(z & 0xffffu) + (int)((z >> 16) & 0xffffu) + (int)((z >> 32) & 0xffffu) +
                  (int)(z >> 48) - 131070;
    const float f = (float)((double)s * scale);
    if (bf16) {
      const uint32_t u = __float_as_uint(f);
      const uint32_t r = ((u >> 16) & 1u) + 0x7FFFu;
      static_cast<uint16_t*>(out)[i] = (uint16_t)((u + r) >> 16);
    } else {
      static_cast<float*>(out)[i] = f;
    }
  }
}

// Raw bytes: byte i is byte (i % 8), little-endian, of output start_word + i / 8.
__global__ void fill_bytes_kernel(uint8_t* out, int64_t n, uint64_t key, uint64_t start_word) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint64_t z = mix64(key + (start_word + (uint64_t)(i >> 3) + 1ull) * kGamma);
    out[i] = (uint8_t)(z >> (8 * (i & 7)));
  }
}

// Q4_0 scale bits: exponent field 7, mantissa the low 10 bits of output i.
__global__ void fill_q4scale_kernel(uint16_t* out, int64_t n, uint64_t key, uint64_t start) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint64_t z = mix64(key + (start + (uint64_t)i + 1ull) * kGamma);
    out[i] = (uint16_t)((7u << 10) | (uint32_t)(z & 0x3FFu));
  }
}

unsigned grid_for(int64_t n) {
  int64_t blocks = (n + 255) / 256;
  return (unsigned)(blocks > 65536 ? 65536 : blocks);
}

}  // namespace

extern "C" int synth_fill_bytes(void* out, int64_t n, uint64_t key, uint64_t start_word,
                                hipStream_t stream) {
  if (out == nullptr || n < 0) return -1;
  if (n == 0) return 0;
  hipLaunchKernelGGL(fill_bytes_kernel, dim3(grid_for(n)), dim3(256), 0, stream,
                     static_cast<uint8_t*>(out), n, key, start_word);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int synth_fill_q4scale(void* out, int64_t n, uint64_t key, uint64_t start,
                                  hipStream_t stream) {
  if (out == nullptr || n < 0) return -1;
  if (n == 0) return 0;
  hipLaunchKernelGGL(fill_q4scale_kernel, dim3(grid_for(n)), dim3(256), 0, stream,
                     static_cast<uint16_t*>(out), n, key, start);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int synth_fill_normal(void* out, int64_t n, int bf16, uint64_t key, uint64_t start,
                                 double scale, hipStream_t stream) {
  if (out == nullptr || n < 0) return -1;
  if (n == 0) return 0;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(fill_normal_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, out, n, bf16,
                     key, start, scale);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
