// The LM head's row-dot (out[t, v] = sum_h W[v, h] x[t, h], §3.3: the
// target's logits at every block position) for a block of 5 to 12 positions
// on the matrix cores.
//
// With bf16 weights and a handful of positions the vector-ALU row-dot does
// 8 FMAs per position for every 16 weight bytes, which at 9 positions keeps
// it arithmetic-bound at about half of the HBM rate.  v_mfma_f32_16x16x32_bf16
// takes 16 weight rows x 32 columns against 32 columns x 16 positions per
// instruction.  The fp32 activations are split exactly into three bf16 parts
// (hi = bf16(x), mid = bf16(x - hi), lo = bf16(x - hi - mid): 24 mantissa bits,
// the whole fp32 mantissa), and every weight fragment meets all three, so
// each product is exact and only the fp32 accumulation order differs from the
// FMA row-dot.
//
// Operand layout (per 64-lane wave, lane l, group g = l / 16): A holds weight
// row l % 16, columns 8g .. 8g + 7 of the 32-column step (one 16-byte load);
// B holds the same 8 columns of position l % 16 (zero past the block's
// positions); D holds rows 4g .. 4g + 3 of position l % 16.  A and B use the
// same column assignment, which is all the product needs.
//
// A block owns a contiguous range of tiles of 16 weight rows, one block per
// CU on every CU; its waves take the tiles round-robin and stream them as one
// flat sequence of 32-column steps with kMRing steps of loads in flight,
// across tile boundaries.  (Giving every wave the same number of tiles
// instead left 56 of 256 CUs idle at V = 102400.)
#include "de_common.h"

namespace de {
namespace {

constexpr int kMThreads = 1024;  // 16 waves: one block per CU holds the split activations
constexpr int kMWaves = kMThreads / kWave;
constexpr int kMRing = 8;        // 32-column steps of weights in flight per wave
constexpr int kMPad = 8;         // bf16 elements of padding per activation row (16 bytes)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4v __attribute__((ext_vector_type(4)));

// Round-to-nearest-even fp32 -> bf16 bits (finite inputs; a NaN stays a NaN).
__device__ __forceinline__ uint32_t bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u) return (u >> 16) | ((u & 0xffffu) ? 0x40u : 0u);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ float bf16_value(uint32_t b) { return __uint_as_float(b << 16); }

__global__ __launch_bounds__(kMThreads) void rowdot_mfma_kernel(const uint16_t* __restrict__ w,
                                                                const float* __restrict__ x,
                                                                float* __restrict__ out, int T,
                                                                int H, int V, int tiles_per_block) {
  extern __shared__ __align__(16) uint16_t xs[];  // [3][T][H + kMPad]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ld = H + kMPad;
  // Split the block of positions into three bf16 parts.
  for (int i = threadIdx.x; i < T * H; i += kMThreads) {
    const int t = i / H, h = i - t * H;
    const float v = x[i];
    uint32_t hi = bf16_bits(v), mid = 0u, lo = 0u;
    if ((hi & 0x7f80u) == 0x7f80u && (__float_as_uint(v) & 0x7f800000u) != 0x7f800000u)
      hi = __float_as_uint(v) >> 16;  // rounding would overflow: truncate instead
    if ((hi & 0x7f80u) != 0x7f80u) {  // an infinite or NaN x is carried by hi alone
      const float r1 = v - bf16_value(hi);
      mid = bf16_bits(r1);
      lo = bf16_bits(r1 - bf16_value(mid));
    }
    xs[(0 * T + t) * ld + h] = (uint16_t)hi;
    xs[(1 * T + t) * ld + h] = (uint16_t)mid;
    xs[(2 * T + t) * ld + h] = (uint16_t)lo;
  }
  __syncthreads();
  const int n = lane & 15, g = lane >> 4;
  const bool has_pos = n < T;
  const int nk = H / 32;
  const int tiles = (V + 15) / 16;
  // The block's tiles [b0, b1); the wave's are t0, t0 + kMWaves, ...
  const int b0 = blockIdx.x * tiles_per_block;
  const int b1 = min(b0 + tiles_per_block, tiles);
  const int t0 = b0 + wave;
  const int ntile = t0 < b1 ? (b1 - t0 + kMWaves - 1) / kMWaves : 0;
  if (ntile <= 0) return;
  const int steps = ntile * nk;
  // Lane's weight row pointer for the tile of step s (rows clamped into the
  // matrix; rows past V are computed and not stored).
  const auto row_ptr = [&](int s) {
    const int tile = t0 + (s / nk) * kMWaves;
    const int row = min(tile * 16 + n, V - 1);
    return w + (size_t)row * H + (size_t)(s % nk) * 32 + 8 * g;
  };
  u32x4 ring[kMRing];
#pragma unroll
  for (int q = 0; q < kMRing; ++q)
    if (q < steps) ring[q] = __builtin_nontemporal_load((const DE_GLOBAL u32x4*)row_ptr(q));
  const uint16_t* xh = xs + (size_t)(0 * T + n) * ld + 8 * g;
  const uint16_t* xm = xs + (size_t)(1 * T + n) * ld + 8 * g;
  const uint16_t* xl = xs + (size_t)(2 * T + n) * ld + 8 * g;
  f32x4v acc = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < steps; s0 += kMRing) {
#pragma unroll
    for (int q = 0; q < kMRing; ++q) {
      const int s = s0 + q;
      if (s < steps) {
        const int k0 = (s % nk) * 32;
        bf16x8 bh, bm, bl;
        if (has_pos) {
          bh = *reinterpret_cast<const bf16x8*>(xh + k0);
          bm = *reinterpret_cast<const bf16x8*>(xm + k0);
          bl = *reinterpret_cast<const bf16x8*>(xl + k0);
        } else {
          bh = bm = bl = bf16x8{};
        }
        const bf16x8 a = __builtin_bit_cast(bf16x8, ring[q]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bh, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bm, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bl, acc, 0, 0, 0);
        if (s + kMRing < steps)
          ring[q] = __builtin_nontemporal_load((const DE_GLOBAL u32x4*)row_ptr(s + kMRing));
        if (s % nk == nk - 1) {
          // Rows 4g .. 4g + 3 of the tile, position n.
          const int r = (t0 + (s / nk) * kMWaves) * 16 + 4 * g;
          if (has_pos) {
            float* o = out + (size_t)n * V + r;
            if (r + 3 < V) {
              o[0] = acc[0];
              o[1] = acc[1];
              o[2] = acc[2];
              o[3] = acc[3];
            } else {
              for (int i = 0; i < 4; ++i)
                if (r + i < V) o[i] = acc[i];
            }
          }
          acc = f32x4v{0.f, 0.f, 0.f, 0.f};
        }
      }
    }
  }
}

}  // namespace

size_t rowdot_mfma_lds(int T, int H) { return (size_t)3 * T * (H + kMPad) * sizeof(uint16_t); }

bool rowdot_mfma_fits(int T, int H) {
  // Below 5 positions the vector-ALU row-dot is as fast (measured at
  // V = 102400, H = 2048: 86 us against 103 us at 2 positions, 113 against
  // 106 at 5); the kernel itself is correct for any T from 1 to 16.
  return T >= 5 && T <= 12 && H >= 32 && H % 32 == 0 && rowdot_mfma_lds(T, H) <= 160 * 1024;
}

hipError_t launch_rowdot_mfma(int T, int H, int V, const float* x, const void* w, float* out,
                              hipStream_t s) {
  if (!rowdot_mfma_fits(T, H) || V < 1) return note_hip(hipErrorInvalidValue);
  const size_t lds = rowdot_mfma_lds(T, H);
  const hipError_t e = allow_lds(reinterpret_cast<const void*>(rowdot_mfma_kernel), lds);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return note_hip(e);
  }
  const int tiles = (V + 15) / 16;
  const int cus = dev_info().num_cus;
  const int tpb = (tiles + cus - 1) / cus;
  const int blocks = (tiles + tpb - 1) / tpb;
  hipLaunchKernelGGL(rowdot_mfma_kernel, dim3(blocks), dim3(kMThreads), lds, s,
                     static_cast<const uint16_t*>(w), x, out, T, H, V, tpb);
  return note_hip(hipGetLastError());
}

}  // namespace de
