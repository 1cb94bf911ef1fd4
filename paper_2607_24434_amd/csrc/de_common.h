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

// Whole-wave reductions without LDS: the 16-lane row steps above, then
// row_bcast:15 (rows 1 and 3 take the row below's lane 15) and row_bcast:31
// (rows 2 and 3 take lane 31), which leaves the total in lane 63; readlane
// hands it to every lane.  A sum pairs the rows as (r3 + r2) + (r1 + r0).
__device__ __forceinline__ float wave_sum(float v) {
  v = row16_sum(v);
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x142, 0xA, 0xF, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x143, 0xC, 0xF, false));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ float wave_max(float v) {
  const int ni = __float_as_int(-INFINITY);
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(ni, __float_as_int(v), 0xB1, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(ni, __float_as_int(v), 0x4E, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(ni, __float_as_int(v), 0x141, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(ni, __float_as_int(v), 0x140, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(ni, __float_as_int(v), 0x142, 0xA, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(ni, __float_as_int(v), 0x143, 0xC, 0xF, false)));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ int wave_min_i32(int v) {
  const int big = 0x7fffffff;
  v = min(v, __builtin_amdgcn_update_dpp(big, v, 0xB1, 0xF, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(big, v, 0x4E, 0xF, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(big, v, 0x141, 0xF, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(big, v, 0x140, 0xF, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(big, v, 0x142, 0xA, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(big, v, 0x143, 0xC, 0xF, false));
  return __builtin_amdgcn_readlane(v, 63);
}

__device__ __forceinline__ float silu_f(float v) { return v / (1.0f + expf(-v)); }

// Native 128-bit vectors (the builtins and address-space casts below need
// clang vector types rather than HIP's vector classes).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Pointers known to be in global memory.  Loads through generic pointers
// compile to flat loads, which also count against the LDS wait counter and so
// serialise with LDS reads; every weight and activation stream here is global.
#define DE_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ const DE_GLOBAL T* gptr(const void* p) {
  return (const DE_GLOBAL T*)(p);
}

// 16-byte load of weights that are streamed once (non-temporal hint).
__device__ __forceinline__ u32x4 load_stream16(const void* p) {
  return __builtin_nontemporal_load(gptr<u32x4>(p));
}

// ---------------------------------------------------------------- kernel arguments

// A weight source of the grouped kernels that is applied to every block
// position with one scalar gate: the shared path, the draft expert, a dense
// layer or the LM head.
struct DenseSrc {
  const void* w;     // gate/up: the [G|U|D] block; down/rowdot: the [rows, len] matrix
  int inter;         // gate/up: rows of G and U.  down: reduction length
  int ld;            // down: row stride of the matrix in elements (0: inter)
  int rows;          // down: output rows (H for experts, V for the LM head)
  float gate;        // down: scale of the result
  const float* vin;  // down: input vectors [T, vin_stride]
  int vin_stride;
  float* out;        // gate/up: A [T, inter]; down: P [T, out_stride]
  int out_stride;
  const void* ws;    // down, Q4_0 weights: the scales of the matrix's first row
  // The single-launch verify layer only: every output value also goes to
  // out_tag (same indexing as out) as a 64-bit (value, launch epoch) pair, and
  // the down pass reads its input pairs from vin_tag (same indexing as vin).
  uint64_t* out_tag;
  const uint64_t* vin_tag;
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
  int max_union;               // bound on the union size: min(N, T * entries per position)
  int n_experts;               // N: bound on expert ids
  int pairs_max;               // T*k: capacity of the token lists, A_r and P_r
  int inter;                   // I
  float* a;                    // A_r [pairs, I]
  float* p;                    // P_r [pairs, H]
  // A union member whose slot is outside [0, n_slots): with absent_ok (the
  // expert cache's chunked calls, which mark the other chunks' members absent
  // on purpose) its work is skipped; otherwise its partial rows are written as
  // zeros (its term drops out of y) and block 0 of the gate/up launch stores
  // kStatusNotResident into *status (when not NULL).
  int absent_ok;
  int32_t* status;
  // The single-launch verify layer only: (value, launch epoch) pairs of A_r and
  // P_r, indexed as a and p.
  uint64_t* a_tag;
  uint64_t* p_tag;
};

// Bits of the device status word of a workspace.
constexpr int32_t kStatusNotResident = 1;
constexpr int32_t kStatusBadToken = 2;
constexpr int32_t kStatusSyncTimeout = 4;  // a bounded device-wide wait ran out

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
  int rounds;              // fused selection: leading entries selected per row
                           // (0: all k; fewer only when nothing reads the rest)
  int32_t* n_union;        // NULL: skip the union
  int32_t* union_ids;
  int32_t* offsets;
  int32_t* tok_list;
  float* gate_list;
  int32_t* pair_pos;       // [T, ucols]
};

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

struct GroupedArgs {
  int T;
  int H;
  const float* x;      // [T, H]
  int has_routed;
  RoutedSrc r;
  int n_dense;
  DenseSrc dense[3];
  int lds_floats;      // set by the launcher: staged-input capacity of a block
  // Gate/up only: build the union in every block (block 0 also writes sel's
  // outputs); r.n_union ... r.gate_list are then not read.  The lists come
  // from sel.idx_out / sel.gate_out, or with fuse_select every block selects
  // them itself from the logits sel.z (block 0 writes them out).
  int fuse_route;
  int fuse_select;
  TopkUnionArgs sel;
  uint32_t epoch;      // the single-launch verify layer: this launch's tag
};

// ---------------------------------------------------------------- launchers (HIP side)

struct DevInfo {
  int device;
  int num_cus;
};
const DevInfo& dev_info();

// Records a failed HIP call for de_hip_error_detail (per host thread) and
// returns its code.
hipError_t note_hip(hipError_t e);


// Router logits and top-k of every position (one block per position).
struct RouteArgs {
  TopkUnionArgs sel;       // top-k options and the idx_out / gate_out lists
  const float* x;          // [T, H]
  const float* w;          // [N, H] fp32 router
  int H;
  float* z;                // [T, N] logits out (each position's last block reads them back)
  unsigned* counter;       // [T] arrival counters, zero between calls
  int select;              // 0: logits only (the gate/up prologue selects)
};
hipError_t launch_route(const RouteArgs& r, hipStream_t s);
hipError_t launch_combine_route(const CombineArgs& a, const RouteArgs& r, hipStream_t s);
// Union only, from caller-supplied lists (sel.idx_in / sel.gate_in).
hipError_t launch_union(const TopkUnionArgs& a, hipStream_t s);

hipError_t launch_gateup(const GroupedArgs& a, int wdtype, hipStream_t s);
// The LM head row-dot on the matrix cores (bf16 weights [V, H], fp32 x [T, H],
// out [T, V]) for the shapes rowdot_mfma_fits accepts.
bool rowdot_mfma_fits(int T, int H);
hipError_t launch_rowdot_mfma(int T, int H, int V, const float* x, const void* w, float* out,
                              hipStream_t s);
// Raises a kernel's dynamic LDS limit to `lds` bytes when above the default.
hipError_t allow_lds(const void* fn, size_t lds);
hipError_t launch_down(const GroupedArgs& a, int wdtype, hipStream_t s);


hipError_t launch_combine(const CombineArgs& a, hipStream_t s);
// The combine (with RMSNorm) fused with the next layer's router logits:
// r.w, r.H, r.z, r.sel.N are read.  Needs a.normed and combine_route_fits(H).
bool combine_route_fits(int H);

struct AcceptArgs {
  int K, V;
  const float* logits;     // [K+1, V]
  const int32_t* drafts;   // [K]
  int32_t* amax;           // [K+1]
  int32_t* out;            // [2]: n, bonus
  float* part_v;           // [K+1, chunks] scratch
  int32_t* part_i;
  unsigned* row_cnt;       // [K+1], zero between calls
  unsigned* done_cnt;      // [1], zero between calls
  // Optional (emb not NULL): the bonus token's bf16 embedding row [H] goes to
  // h and its RMSNorm (eps) to normed, as one position of the embedding gather.
  const uint16_t* emb;
  float* h;
  float* normed;
  float eps;
  int H;
};
int accept_chunks(int V);
hipError_t launch_argmax_accept(const AcceptArgs& a, hipStream_t s);
hipError_t launch_rmsnorm(int T, int H, const float* x, float eps, float* out, hipStream_t s);
hipError_t launch_embed(int T, int H, int V, const int32_t* tokens, const uint16_t* emb, float* h,
                        float* normed, float eps, int32_t* status, hipStream_t s);
hipError_t launch_stream_probe(const void* buf, size_t bytes, float* sink, hipStream_t s);

// Truncation of the draft loop.
struct ExpansionArgs {
  int L, k, N;                 // layers, predicted experts per layer, experts per layer (<= 256)
  const int32_t* pred;         // [L, k] the token's predicted experts
  unsigned long long* uhat;    // [L, ceil(N / 64)] the block-level predicted set
  int first;                   // the set is empty before this token
  const float* q;              // the token's confidence (device scalar)
  float tau;
  int budget;                  // >= 0 fixed; < 0 the cache room
  int slots;
  int32_t* out;                // [5]
};
hipError_t launch_confidence(int T, int V, const float* logits, float* q, hipStream_t s);

// Self-distillation signals.
struct ResidualArgs {
  int T, H, kk, pairs_max;
  const float* p_r;            // [pairs, H] routed partials (gates applied)
  const int32_t* pair_pos;     // [T, kk]
  float* out;                  // [T, H]
};
struct RowKlArgs {
  int rows, n;
  const float* a;              // target rows [rows, lda]
  int lda;
  const float* b;              // draft rows [rows, ldb]
  int ldb;
  const float* bias;           // [n] or NULL (softmax mode)
  int sigmoid;
  float tau;
  float* kl;                   // [rows]
  float* ce;                   // [rows] or NULL (softmax mode only)
};
hipError_t launch_residual(const ResidualArgs& a, hipStream_t s);
hipError_t launch_rowkl(const RowKlArgs& a, hipStream_t s);
hipError_t launch_expansion(const ExpansionArgs& a, hipStream_t s);

}  // namespace de
