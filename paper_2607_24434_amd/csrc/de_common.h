// Internal declarations shared by the HIP kernels and the C ABI layer.
// gfx950 only: wave64, 16-lane DPP rows, 128-bit global loads.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace de {

constexpr int kWave = 64;

// ---------------------------------------------------------------- device helpers

// A uint32 holding two bf16 values: element 0 in the low half.
__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

// Sum over the 16 lanes of a DPP row; every lane of the row ends with the
// same total (each step adds a mirrored partner, so both partners compute
// a+b and b+a, which are equal bit for bit).
__device__ __forceinline__ float row16_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));  // quad_perm 1,0,3,2
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));  // quad_perm 2,3,0,1
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false)); // row_half_mirror
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false)); // row_mirror
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

__device__ __forceinline__ float silu_f(float v) { return v / (1.0f + expf(-v)); }

// Native 128-bit vector (the builtins below need a clang vector type).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte load of weights that are streamed once (non-temporal hint).
__device__ __forceinline__ u32x4 load_stream16(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

// ---------------------------------------------------------------- kernel arguments

// A weight source of the grouped kernels that is applied to every block
// position with one scalar gate: the shared path, the draft expert, a dense
// layer or the LM head.
struct DenseSrc {
  const void* w;     // gate/up: the [G|U|D] block; down/rowdot: the [rows, len] matrix
  int inter;         // gate/up: rows of G and U.  down: reduction length
  int rows;          // down: output rows (H for experts, V for the LM head)
  float gate;        // down: scale of the result
  const float* vin;  // down: input vectors [T, vin_stride]
  int vin_stride;
  float* out;        // gate/up: A [T, inter]; down: P [T, out_stride]
  int out_stride;
};

// The routed part of a grouped launch: the union members and their lists.
struct RoutedSrc {
  const char* base;            // expert table base
  int64_t stride;              // bytes per slot
  const int32_t* slot_of_expert;
  int n_slots;
  const int32_t* n_union;      // device scalar; < 0 means "no routed work"
  const int32_t* union_ids;
  const int32_t* offsets;
  const int32_t* tok_list;
  const float* gate_list;
  int max_union;               // N: bound on the union size and on expert ids
  int pairs_max;               // T*k: capacity of the token lists, A_r and P_r
  int inter;                   // I
  float* a;                    // A_r [pairs, I]
  float* p;                    // P_r [pairs, H]
};

struct GroupedArgs {
  int T;
  int H;
  const float* x;      // [T, H]
  int has_routed;
  RoutedSrc r;
  int n_dense;
  DenseSrc dense[3];
};

// ---------------------------------------------------------------- launchers (HIP side)

struct DevInfo {
  int device;
  int num_cus;
};
const DevInfo& dev_info();

hipError_t launch_router_logits(const float* x, const float* w, int T, int H, int N, float* z,
                                hipStream_t s);

struct TopkUnionArgs {
  int T, N, k;
  const float* z;          // [T, N] logits; NULL: read idx_in/gate_in instead
  const float* bias;       // [N] or NULL
  int score_func, norm_topk;
  float routed_scale;
  const int32_t* idx_in;   // union-only mode
  const float* gate_in;
  int32_t* idx_out;        // [T, k] (may be NULL in union-only mode)
  float* gate_out;
  int ucols;               // union over the first ucols columns of each row (k or 1)
  int32_t* n_union;        // NULL: skip the union
  int32_t* union_ids;
  int32_t* offsets;
  int32_t* tok_list;
  float* gate_list;
  int32_t* pair_pos;       // [T, ucols]
};
hipError_t launch_topk_union(const TopkUnionArgs& a, hipStream_t s);

hipError_t launch_gateup(const GroupedArgs& a, int wdtype, hipStream_t s);
hipError_t launch_down(const GroupedArgs& a, int wdtype, hipStream_t s);

struct CombineArgs {
  int T, H;
  int n_dense;
  const float* dense_p[3];     // [T, H] partials with their gates applied
  const float* p_r;            // [pairs, H] routed partials or NULL
  const int32_t* pair_pos;     // [T, kk]
  int kk;
  int pairs_max;               // rows of p_r
  const float* residual;       // [T, H] or NULL
  float* y;                    // [T, H]
  float* normed;               // [T, H] or NULL
  float eps;
};
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);

hipError_t launch_argmax_rows(const float* logits, int rows, int V, int32_t* amax, hipStream_t s);
hipError_t launch_accept(int K, const int32_t* amax, const int32_t* drafts, int32_t* out,
                         hipStream_t s);
hipError_t launch_rmsnorm(int T, int H, const float* x, float eps, float* out, hipStream_t s);
hipError_t launch_embed(int T, int H, int V, const int32_t* tokens, const uint16_t* emb, float* h,
                        float* normed, float eps, hipStream_t s);
hipError_t launch_stream_probe(const void* buf, size_t bytes, float* sink, hipStream_t s);

}  // namespace de
