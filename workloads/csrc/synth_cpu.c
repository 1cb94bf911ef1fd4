/* CPU fill of the seeded synthetic streams of workloads/rng.py, bit for bit
 * (SplitMix64 in counter mode, Irwin-Hall(4) of 16-bit fields, one fp64
 * multiply, fp32 rounding, optional bf16 round-to-nearest-even).
 * A fast path for large tensors; rng.py is the definition it is tested against. */
#include <stdint.h>
#include <string.h>

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static inline float one(uint64_t key, uint64_t ctr, double scale) {
  const uint64_t z = mix64(key + ctr * 0x9E3779B97F4A7C15ull);
  const int s = (int)(z & 0xffffu) + (int)((z >> 16) & 0xffffu) + (int)((z >> 32) & 0xffffu) +
                (int)(z >> 48) - 131070;
  return (float)((double)s * scale);
}

void synth_normal_f32(float* out, int64_t n, uint64_t key, uint64_t start, double scale) {
  for (int64_t i = 0; i < n; ++i) out[i] = one(key, start + (uint64_t)i + 1ull, scale);
}

void synth_normal_bf16(uint16_t* out, int64_t n, uint64_t key, uint64_t start, double scale) {
  for (int64_t i = 0; i < n; ++i) {
    const float f = one(key, start + (uint64_t)i + 1ull, scale);
    uint32_t u;
    memcpy(&u, &f, 4);
    const uint32_t r = ((u >> 16) & 1u) + 0x7FFFu;
    out[i] = (uint16_t)((u + r) >> 16);
  }
}
