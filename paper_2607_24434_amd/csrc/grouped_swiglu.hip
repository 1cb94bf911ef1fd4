// Grouped SwiGLU over the expert union plus the shared / draft / dense
// sources (Eq. 4 and Eq. 5 without the routing), the fixed-order combine, and
// the row-dot kernel used for the LM head.
//
// With a few block positions per expert the work is a batch of skinny GEMVs:
// every weight byte meets only |T_e| positions, so the kernels are bound by
// HBM bandwidth, not arithmetic.  The design keeps many 128-bit loads in
// flight and touches each weight byte once:
//
//  * Persistent 512-thread blocks.  The tiles of a launch (union members
//    first, then the dense sources) form segments; block b owns a contiguous
//    tile range whose cost (bytes x position passes) is 1/grid of the total,
//    so the blocks finish together.  Within a range the 8 waves take every
//    8th tile.  The number of union members stays in device memory.
//  * A wave tile is NS weight rows streamed by all four 16-lane groups of the
//    wave (GR = 4 groups per row): each wave load reads 1 KB of one row, and
//    a lane issues the loads of MI 16-byte iterations before using them.
//  * Activations are staged in LDS per block in a bank-conflict-free order
//    (gate/up: the whole block of positions once; down: the segment's input
//    rows), so only weights come from HBM.
//  * bf16 -> fp32 by a shift or mask, fp32 accumulation; per-row sums use
//    four DPP steps inside a 16-lane row and two cross-group shuffles, and are
//    identical in every lane.  No float atomics: results are bitwise
//    reproducible.
#include "de_common.h"

// Build-time tuning knobs (kept at the measured best by default).
#ifndef DE_NT_LOADS
#define DE_NT_LOADS 1
#endif
#ifndef DE_GU_STRIDED
#define DE_GU_STRIDED 1
#endif
#ifndef DE_DN_STRIDED
#define DE_DN_STRIDED 1
#endif
#ifndef DE_GU_PAIRS
#define DE_GU_PAIRS 2
#endif
#ifndef DE_DN_ROWS
#define DE_DN_ROWS 4
#endif
#ifndef DE_RD_ROWS
#define DE_RD_ROWS 4
#endif
#ifndef DE_DENSE_NT
#define DE_DENSE_NT 4
#endif
#ifndef DE_TOK_GROUP
#define DE_TOK_GROUP 4
#endif
#ifndef DE_REG_BUDGET
#define DE_REG_BUDGET 96
#endif

namespace de {
namespace {

constexpr int kBlock = 512;                 // 8 waves share the staged activations
constexpr int kWavesPB = kBlock / kWave;
constexpr int kTokGroup = DE_TOK_GROUP;               // positions whose activation loads may be hoisted together
constexpr int kLdsBudget = 144 * 1024;      // staged activations per block (gate/up)
constexpr int kDownLds = 72 * 1024;         // staged input rows per block (down): two blocks/CU

// Wave tiles: every lane of a wave streams the same NS rows, 1 KB of one row
// per load instruction.
constexpr int kGuPairs = DE_GU_PAIRS;       // gate/up: (G row, U row) pairs
constexpr int kDnRows = DE_DN_ROWS;         // grouped down: D rows
constexpr int kRdRows = DE_RD_ROWS;         // row-dot (LM head, dense down): rows
constexpr int kRoutedNT = 4;                // positions per pass of a union member
constexpr int kDenseNT = DE_DENSE_NT;       // positions per pass of a dense source (cap)

// 16-byte iterations whose weight loads are issued together (NS*MI loads in
// flight per lane): what the register budget leaves after the NS*NT
// accumulators and one group of activations.
template <int NS, int NT, int EPU>
struct InFlight {
  static constexpr int TG = NT < kTokGroup ? NT : kTokGroup;
  static constexpr int free_regs = DE_REG_BUDGET - NS * NT - TG * EPU - EPU;
  static constexpr int MI = free_regs / (4 * NS) > 4 ? 4 : (free_regs / (4 * NS) < 1 ? 1 : free_regs / (4 * NS));
};

// Dynamic LDS: the block's staged activation rows.
extern __shared__ __align__(16) float s_act[];

template <typename WT>
struct WTr;
template <>
struct WTr<uint16_t> {
  static constexpr int EPU = 8;  // elements per 16 bytes
};
template <>
struct WTr<float> {
  static constexpr int EPU = 4;
};

__device__ __forceinline__ u32x4 load_w16(const void* p) {
#if DE_NT_LOADS
  return load_stream16(p);
#else
  return *gptr<u32x4>(p);
#endif
}

__device__ __forceinline__ void unpack(const u32x4& r, float (&f)[8]) {
  f[0] = bf16_lo(r.x);
  f[1] = bf16_hi(r.x);
  f[2] = bf16_lo(r.y);
  f[3] = bf16_hi(r.y);
  f[4] = bf16_lo(r.z);
  f[5] = bf16_hi(r.z);
  f[6] = bf16_lo(r.w);
  f[7] = bf16_hi(r.w);
}
__device__ __forceinline__ void unpack(const u32x4& r, float (&f)[4]) {
  f[0] = __uint_as_float(r.x);
  f[1] = __uint_as_float(r.y);
  f[2] = __uint_as_float(r.z);
  f[3] = __uint_as_float(r.w);
}

// Staged layout of one activation row for bf16 weights: the 8 floats that
// meet weight unit u (16 bytes = 8 bf16) are split into two float4 halves
// stored at ((u/16)*2 + half)*16 + u%16, so the 16 lanes of a group read 256
// contiguous bytes per ds_read_b128 (no bank conflicts).  Rows are padded to a
// multiple of 128 floats.  fp32 weights (4 per unit) keep the natural order.
__device__ __forceinline__ int perm_index(int u, int half) {
  return (((u >> 4) * 2 + half) * 16 + (u & 15)) * 4;
}

template <int EPU>
__host__ __device__ __forceinline__ int staged_stride(int len) {
  return EPU == 8 ? ((len + 127) / 128) * 128 : len;
}

// The EPU activations that meet weight unit u of one row, from LDS (staged
// layout, row at float offset `off`) or from global memory (natural layout).
template <int EPU, bool LDSX>
__device__ __forceinline__ void act_frag(const float* g, int off, int u, float (&v)[EPU]) {
  if constexpr (LDSX) {
    if constexpr (EPU == 8) {
      const float4 a = *reinterpret_cast<const float4*>(&s_act[off + perm_index(u, 0)]);
      const float4 b = *reinterpret_cast<const float4*>(&s_act[off + perm_index(u, 1)]);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
      v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
      const float4 a = *reinterpret_cast<const float4*>(&s_act[off + u * 4]);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    }
  } else {
    const DE_GLOBAL f32x4* q = gptr<f32x4>(g + off + u * EPU);
#pragma unroll
    for (int i = 0; i < EPU / 4; ++i) {
      const f32x4 t = q[i];
      v[4 * i + 0] = t.x;
      v[4 * i + 1] = t.y;
      v[4 * i + 2] = t.z;
      v[4 * i + 3] = t.w;
    }
  }
}

// Copies `rows` activation rows of length len (fp32, row stride gstride) into
// LDS in the staged layout (row stride staged_stride(len)).  All threads; the
// caller synchronises before the rows are read.
template <int EPU>
__device__ __forceinline__ void stage_rows(const float* g, int gstride, int rows, int len) {
  const int l4 = len >> 2;
  const int sst = staged_stride<EPU>(len);
  for (int i = threadIdx.x; i < rows * l4; i += kBlock) {
    const int t = i / l4, h4 = i - t * l4;
    const f32x4 v = gptr<f32x4>(g + (size_t)t * gstride)[h4];
    const int dst = t * sst + (EPU == 8 ? perm_index(h4 >> 1, h4 & 1) : h4 * 4);
    *reinterpret_cast<f32x4*>(&s_act[dst]) = v;
  }
}

// Dot products of NS weight rows (L 16-byte units each) with up to NT
// activation rows.  Lane l owns the units it*64 + l; loads of MI iterations are
// issued together, then consumed.  Past the row end a lane re-reads the last
// unit (always in bounds) and zeroes it.  Activation row m starts at float
// offset voff[m] (LDS or global).  The sums are partial per lane; row_total()
// finishes them.
template <typename WT, int NS, int NT, bool LDSX>
__device__ __forceinline__ void rows_dot(const char* const (&rowp)[NS], int L, int lane,
                                         const float* gact, const int (&voff)[NT], int nt,
                                         float (&acc)[NS][NT]) {
  constexpr int EPU = WTr<WT>::EPU;
  constexpr int MI = InFlight<NS, NT, EPU>::MI;
  constexpr int TG = InFlight<NS, NT, EPU>::TG;
  const int nit = (L + kWave - 1) / kWave;
  for (int i0 = 0; i0 < nit; i0 += MI) {
    u32x4 raw[MI][NS];
#pragma unroll
    for (int q = 0; q < MI; ++q) {
      if (i0 + q < nit) {
        const uint32_t uc = (uint32_t)min((i0 + q) * kWave + lane, L - 1) * 16u;
#pragma unroll
        for (int s = 0; s < NS; ++s) raw[q][s] = load_w16(rowp[s] + uc);
      }
    }
#pragma unroll
    for (int q = 0; q < MI; ++q) {
      if (i0 + q < nit) {
        const int u = (i0 + q) * kWave + lane;
        const bool ok = u < L;
        const int uc = ok ? u : L - 1;
        // Positions in groups of TG: the group's activations are loaded once
        // and meet every row; a row's weights are unpacked when used.
#pragma unroll
        for (int mg = 0; mg < NT; mg += TG) {
          if (mg < nt) {
            float xv[TG][EPU];
#pragma unroll
            for (int m = 0; m < TG; ++m) {
              if (mg + m < nt) {
                act_frag<EPU, LDSX>(gact, voff[mg + m], uc, xv[m]);
              } else {
#pragma unroll
                for (int v = 0; v < EPU; ++v) xv[m][v] = 0.f;
              }
            }
#pragma unroll
            for (int s = 0; s < NS; ++s) {
              const u32x4 r = ok ? raw[q][s] : u32x4{0u, 0u, 0u, 0u};
              float w[EPU];
              unpack(r, w);
#pragma unroll
              for (int m = 0; m < TG; ++m)
#pragma unroll
                for (int v = 0; v < EPU; ++v) acc[s][mg + m] = fmaf(w[v], xv[m][v], acc[s][mg + m]);
            }
          }
          // Keeps the next group's (or iteration's) activation loads from
          // being hoisted above this one's arithmetic.
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  }
}

// Total of a per-lane partial over the 64 lanes of a wave; every lane receives
// the same bits.
__device__ __forceinline__ float row_total(float v) {
  v = row16_sum(v);
  v += __shfl_xor(v, 16, kWave);
  v += __shfl_xor(v, 32, kWave);
  return v;
}

__device__ __forceinline__ int cdiv(int a, int b) { return (a + b - 1) / b; }

// Values that are the same in every lane (tile and segment metadata, read from
// memory) are moved to scalar registers; the compiler cannot prove it itself
// for loaded values, and keeping them in vector registers causes spills.
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
template <typename P>
__device__ __forceinline__ P* uni(P* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<P*>(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ int routed_count(const GroupedArgs& a) {
  if (!a.has_routed) return 0;
  const int nu = uni(*a.r.n_union);
  return nu < 0 ? 0 : min(nu, a.r.max_union);
}

// Resolves union member j to its weight block and token-list span; nullptr
// when the expert is not resident or the lists are malformed (lists built by
// the union kernel always pass; caller-supplied ones are checked so that a
// bad list can only drop work, never read or write out of bounds).
__device__ __forceinline__ const char* member_block(const RoutedSrc& r, int j, int& off,
                                                    int& ntok) {
  const int e = uni(r.union_ids[j]);
  if (e < 0 || e >= r.max_union) return nullptr;
  const int slot = uni(r.slot_of_expert ? r.slot_of_expert[e] : e);
  if (slot < 0 || slot >= r.n_slots) return nullptr;
  off = uni(r.offsets[j]);
  const int end = uni(r.offsets[j + 1]);
  if (off < 0 || end < off || end > r.pairs_max) return nullptr;
  ntok = end - off;
  return uni(r.base + (size_t)slot * r.stride);
}

// a.dense[s] with a run-time s would copy the kernel-argument array to scratch
// memory; an explicit select keeps everything in scalar registers.
__device__ __forceinline__ DenseSrc pick_dense(const GroupedArgs& a, int s) {
  return s == 0 ? a.dense[0] : (s == 1 ? a.dense[1] : a.dense[2]);
}

// Tiles are laid out as consecutive segments (the union members, then each
// dense source); every tile of a segment has the same cost.  Block b owns the
// contiguous tile range whose cost covers [b, b+1) * total / grid.
struct Segments {
  int n;
  int tiles[4];
  long long cost[4];  // per tile
};

__device__ __forceinline__ int tile_at_cost(const Segments& sg, long long c) {
  int t0 = 0;
  long long c0 = 0;
  for (int i = 0; i < sg.n; ++i) {
    const long long seg = (long long)sg.tiles[i] * sg.cost[i];
    if (c < c0 + seg) return t0 + (int)((c - c0 + sg.cost[i] - 1) / sg.cost[i]);
    t0 += sg.tiles[i];
    c0 += seg;
  }
  return t0;
}

// Integer division has no scalar instruction, so its results land in vector
// registers; lo and hi are moved back to scalar ones.
__device__ __forceinline__ void block_range(const Segments& sg, int& lo, int& hi) {
  long long total = 0;
  for (int i = 0; i < sg.n; ++i) total += (long long)sg.tiles[i] * sg.cost[i];
  lo = uni(tile_at_cost(sg, total * blockIdx.x / gridDim.x));
  hi = uni(tile_at_cost(sg, total * (blockIdx.x + 1) / gridDim.x));
}

// ------------------------------------------------------------------ gate/up

constexpr int kGuRows = kGuPairs;  // (G, U) row pairs per wave tile

// One pass (up to NT positions) over the (G, U) row pairs r0 .. r0+kGuPairs-1:
// A[arow0 + m][r] = silu(G_r . x_m) * (U_r . x_m).
template <typename WT, int NT, bool LDSX>
__device__ __forceinline__ void gateup_pass(const char* G, const char* U, int inter, int H, int r0,
                                            int lane, const float* gx, const int (&voff)[NT],
                                            int nt, float* A, int arow0) {
  constexpr int NS = 2 * kGuPairs;
  const size_t rb = (size_t)H * sizeof(WT);
  const char* rowp[NS];
#pragma unroll
  for (int p = 0; p < kGuPairs; ++p) {
    const size_t rc = (size_t)min(r0 + p, inter - 1);
    rowp[2 * p] = G + rc * rb;
    rowp[2 * p + 1] = U + rc * rb;
  }
  float acc[NS][NT];
#pragma unroll
  for (int k = 0; k < NS; ++k)
#pragma unroll
    for (int m = 0; m < NT; ++m) acc[k][m] = 0.f;
  rows_dot<WT, NS, NT, LDSX>(rowp, (int)(rb / 16), lane, gx, voff, nt, acc);
#pragma unroll
  for (int m = 0; m < NT; ++m) {
    if (m < nt) {
#pragma unroll
      for (int p = 0; p < kGuPairs; ++p) {
        const float g = row_total(acc[2 * p][m]);
        const float u = row_total(acc[2 * p + 1][m]);
        if (lane == m && r0 + p < inter) A[(size_t)(arow0 + m) * inter + r0 + p] = silu_f(g) * u;
      }
    }
  }
}

// Activation offsets of one pass (token list or consecutive positions).
template <int NT>
__device__ __forceinline__ void pass_offsets(int (&voff)[NT], const int32_t* tok, int tok_base,
                                             int nt, int T, int stride) {
#pragma unroll
  for (int m = 0; m < NT; ++m) {
    int t = uni(m < nt ? (tok ? tok[m] : tok_base + m) : tok_base);
    t = t < 0 ? 0 : (t >= T ? T - 1 : t);  // a position outside the block never indexes x
    voff[m] = t * stride;
  }
}

// Every pass over one wave tile of a source: its ntok positions (token list
// tok, or 0..ntok-1) in passes of NTP, a single remaining position by the
// one-position variant.  The passes run back to back, so the later ones find
// the rows in cache.
template <typename WT, int NTP, bool LDSX>
__device__ __forceinline__ void gateup_tile(const char* G, const char* U, int inter, int H, int r0,
                                            int lane, const float* gx, int xstride, int T,
                                            const int32_t* tok, int ntok, float* A, int arow0) {
  for (int m0 = 0; m0 < ntok; m0 += NTP) {
    const int nt = min(NTP, ntok - m0);
    const int32_t* tk = tok ? tok + m0 : nullptr;
    if (nt == 1) {
      int voff[1];
      pass_offsets<1>(voff, tk, m0, 1, T, xstride);
      gateup_pass<WT, 1, LDSX>(G, U, inter, H, r0, lane, gx, voff, 1, A, arow0 + m0);
    } else {
      int voff[NTP];
      pass_offsets<NTP>(voff, tk, m0, nt, T, xstride);
      gateup_pass<WT, NTP, LDSX>(G, U, inter, H, r0, lane, gx, voff, nt, A, arow0 + m0);
    }
  }
}

// Persistent gate/up kernel over the union members and the dense sources.
// Tiles: union member j covers tiles [j*tr, (j+1)*tr), then each dense source.
template <typename WT, bool LDSX>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void gateup_kernel(
    GroupedArgs a) {
  constexpr int EPU = WTr<WT>::EPU;
  const int lane = threadIdx.x & 63, wave = uni((int)(threadIdx.x >> 6));
  int xstride = a.H;
  if constexpr (LDSX) {
    stage_rows<EPU>(a.x, a.H, a.T, a.H);
    __syncthreads();
    xstride = staged_stride<EPU>(a.H);
  }
  const int nu = routed_count(a);
  const int tr = uni(a.has_routed ? cdiv(a.r.inter, kGuRows) : 0);
  const int nr = nu * tr;
  const size_t esz = sizeof(WT);
  int dstart[4];
  int total = nr;
  for (int s = 0; s < a.n_dense; ++s) {
    dstart[s] = total;
    total += uni(cdiv(a.dense[s].inter, kGuRows));
  }
  dstart[a.n_dense] = total;
#if DE_GU_STRIDED
  // Grid-strided tile order: at any moment the whole grid streams a narrow
  // window of consecutive rows.
  int cur_j = -1, off = 0, ntok = 0;
  const char* blk = nullptr;
  for (int tile = blockIdx.x * kWavesPB + wave; tile < total; tile += gridDim.x * kWavesPB) {
    if (tile < nr) {
      const int j = uni(tile / tr);
      if (j != cur_j) {
        blk = member_block(a.r, j, off, ntok);
        cur_j = j;
      }
      if (blk == nullptr) continue;
      gateup_tile<WT, kRoutedNT, LDSX>(blk, blk + (size_t)a.r.inter * a.H * esz, a.r.inter, a.H,
                                       (tile - j * tr) * kGuRows, lane, a.x, xstride, a.T,
                                       a.r.tok_list + off, ntok, a.r.a, off);
    } else {
      int s = 0;
      while (s + 1 < a.n_dense && tile >= dstart[s + 1]) ++s;
      const DenseSrc d = pick_dense(a, s);
      const char* G = static_cast<const char*>(d.w);
      gateup_tile<WT, kDenseNT, LDSX>(G, G + (size_t)d.inter * a.H * esz, d.inter, a.H,
                                      (tile - dstart[s]) * kGuRows, lane, a.x, xstride, a.T,
                                      nullptr, a.T, d.out, 0);
    }
  }
#else
  // Contiguous order: block b owns the tile range whose cost (bytes x passes)
  // is 1/grid of the total; its waves take every 8th tile of the range.
  Segments sg;
  const long long row_cost = (long long)a.H * sizeof(WT) * 2 * kGuRows;
  sg.n = 0;
  sg.tiles[sg.n] = nr;
  sg.cost[sg.n++] = row_cost;  // one pass for a member in the common case
  for (int s = 0; s < a.n_dense; ++s) {
    sg.tiles[sg.n] = dstart[s + 1] - dstart[s];
    sg.cost[sg.n++] = row_cost * ((a.T + kDenseNT - 1) / kDenseNT);
  }
  int lo, hi;
  block_range(sg, lo, hi);
  int t = lo;
  while (t < hi) {
    if (t < nr) {
      const int j = uni(t / tr), seg0 = j * tr, t1 = min(hi, seg0 + tr);
      int off = 0, ntok = 0;
      const char* blk = member_block(a.r, j, off, ntok);
      if (blk != nullptr)
        for (int tile = t + wave; tile < t1; tile += kWavesPB)
          gateup_tile<WT, kRoutedNT, LDSX>(blk, blk + (size_t)a.r.inter * a.H * esz, a.r.inter,
                                           a.H, (tile - seg0) * kGuRows, lane, a.x, xstride, a.T,
                                           a.r.tok_list + off, ntok, a.r.a, off);
      t = t1;
    } else {
      int s = 0;
      while (s + 1 < a.n_dense && t >= dstart[s + 1]) ++s;
      const DenseSrc d = pick_dense(a, s);
      const int seg0 = dstart[s], t1 = min(hi, dstart[s + 1]);
      const char* G = static_cast<const char*>(d.w);
      for (int tile = t + wave; tile < t1; tile += kWavesPB)
        gateup_tile<WT, kDenseNT, LDSX>(G, G + (size_t)d.inter * a.H * esz, d.inter, a.H,
                                        (tile - seg0) * kGuRows, lane, a.x, xstride, a.T, nullptr,
                                        a.T, d.out, 0);
      t = t1;
    }
  }
#endif
}

// ------------------------------------------------------------------ down / row-dot

// One pass over the NS rows r0.. of a [rows, len] matrix for up to NT inputs:
// out[orow0 + m][r] = gate_m * (M_r . v_m).
template <typename WT, int NS, int NT, bool LDSX>
__device__ __forceinline__ void down_pass(const char* M, int rows, int len, int r0, int lane,
                                          const float* gv, const int (&voff)[NT], int nt,
                                          const float* gates, float gscalar, float* out,
                                          int ostride, int orow0) {
  const size_t rb = (size_t)len * sizeof(WT);
  const char* rowp[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) rowp[k] = M + (size_t)min(r0 + k, rows - 1) * rb;
  float acc[NS][NT];
#pragma unroll
  for (int k = 0; k < NS; ++k)
#pragma unroll
    for (int m = 0; m < NT; ++m) acc[k][m] = 0.f;
  rows_dot<WT, NS, NT, LDSX>(rowp, (int)(rb / 16), lane, gv, voff, nt, acc);
#pragma unroll
  for (int m = 0; m < NT; ++m) {
    if (m < nt) {
      const float gm = gates ? gates[m] : gscalar;
#pragma unroll
      for (int k = 0; k < NS; ++k) {
        const float v = row_total(acc[k][m]);
        if (lane == m && r0 + k < rows) out[(size_t)(orow0 + m) * ostride + r0 + k] = gm * v;
      }
    }
  }
}

// Every pass over one wave tile for the inputs vrow0 .. vrow0+n-1 (rows of
// length len at stride vstride, LDS or global), NTP per pass, a single
// remaining input by the one-input variant.
template <typename WT, int NS, int NTP, bool LDSX>
__device__ __forceinline__ void down_tile(const char* M, int rows, int len, int r0, int lane,
                                          const float* gv, int vstride, int vrow0, int n,
                                          const float* gates, float gscalar, float* out,
                                          int ostride, int orow0) {
  for (int m0 = 0; m0 < n; m0 += NTP) {
    const int nt = min(NTP, n - m0);
    const float* gt = gates ? gates + m0 : nullptr;
    if (nt == 1) {
      const int voff[1] = {(vrow0 + m0) * vstride};
      down_pass<WT, NS, 1, LDSX>(M, rows, len, r0, lane, gv, voff, 1, gt, gscalar, out, ostride,
                                 orow0 + m0);
    } else {
      int voff[NTP];
#pragma unroll
      for (int m = 0; m < NTP; ++m) voff[m] = (vrow0 + m0 + (m < nt ? m : 0)) * vstride;
      down_pass<WT, NS, NTP, LDSX>(M, rows, len, r0, lane, gv, voff, nt, gt, gscalar, out,
                                   ostride, orow0 + m0);
    }
  }
}

// One source of the down kernel, resolved for tile t.
struct DownSeg {
  const char* M;
  const float* vin;
  const float* gates;
  float* out;
  float gscalar;
  int rows, len, vstride, vrow0, ntok, ostride, orow0, seg0, seg1;
  bool routed, valid;
};

template <typename WT>
__device__ __forceinline__ DownSeg down_seg(const GroupedArgs& a, int t, int nr, int tr,
                                            const int (&dstart)[4]) {
  DownSeg g;
  const size_t esz = sizeof(WT);
  if (t < nr) {
    const int j = uni(t / tr);
    int off = 0, ntok = 0;
    const char* blk = member_block(a.r, j, off, ntok);
    g.valid = blk != nullptr;
    g.routed = true;
    g.seg0 = j * tr;
    g.seg1 = g.seg0 + tr;
    g.M = blk + 2 * (size_t)a.r.inter * a.H * esz;
    g.rows = a.H;
    g.len = a.r.inter;
    g.vin = a.r.a;
    g.vstride = a.r.inter;
    g.vrow0 = off;
    g.ntok = ntok;
    g.gates = a.r.gate_list + off;
    g.gscalar = 0.f;
    g.out = a.r.p;
    g.ostride = a.H;
    g.orow0 = off;
  } else {
    int s = 0;
    while (s + 1 < a.n_dense && t >= dstart[s + 1]) ++s;
    const DenseSrc d = pick_dense(a, s);
    g.valid = true;
    g.routed = false;
    g.seg0 = dstart[s];
    g.seg1 = dstart[s + 1];
    g.M = static_cast<const char*>(d.w);
    g.rows = d.rows;
    g.len = d.inter;
    g.vin = d.vin;
    g.vstride = d.vin_stride;
    g.vrow0 = 0;
    g.ntok = a.T;
    g.gates = nullptr;
    g.gscalar = d.gate;
    g.out = d.out;
    g.ostride = d.out_stride;
    g.orow0 = 0;
  }
  return g;
}

// Persistent down-projection / row-dot kernel (NS rows per wave tile).
template <typename WT, bool LDSX, int NS>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void down_kernel(
    GroupedArgs a) {
  constexpr int EPU = WTr<WT>::EPU;
  const int lane = threadIdx.x & 63, wave = uni((int)(threadIdx.x >> 6));
  const int nu = routed_count(a);
  const int tr = uni(a.has_routed ? cdiv(a.H, NS) : 0);
  const int nr = nu * tr;
  int dstart[4];
  int total = nr;
  for (int s = 0; s < a.n_dense; ++s) {
    dstart[s] = total;
    total += uni(cdiv(a.dense[s].rows, NS));
  }
  dstart[a.n_dense] = total;
#if DE_DN_STRIDED
  // Grid-strided tile order.  Inputs: a single dense source (the row-dot)
  // stages all T input rows in LDS at the start when LDSX; otherwise they are
  // read from global memory (they are small and stay in cache).
  int sstride = 0;
  if constexpr (LDSX) {
    const DenseSrc d0 = a.dense[0];
    stage_rows<EPU>(d0.vin, d0.vin_stride, a.T, d0.inter);
    __syncthreads();
    sstride = staged_stride<EPU>(d0.inter);
  }
  int cur = -1;
  DownSeg g;
  for (int tile = blockIdx.x * kWavesPB + wave; tile < total; tile += gridDim.x * kWavesPB) {
    if (tile >= cur) {  // tiles only increase: a new segment starts at or after seg1
      g = down_seg<WT>(a, tile, nr, tr, dstart);
      cur = g.seg1;
    }
    if (!g.valid) continue;
    const int r0 = (tile - g.seg0) * NS;
    if (LDSX && !g.routed)
      down_tile<WT, NS, kDenseNT, LDSX>(g.M, g.rows, g.len, r0, lane, nullptr, sstride, 0, g.ntok,
                                        nullptr, g.gscalar, g.out, g.ostride, 0);
    else if (g.routed)
      down_tile<WT, NS, kRoutedNT, false>(g.M, g.rows, g.len, r0, lane, g.vin, g.vstride, g.vrow0,
                                          g.ntok, g.gates, 0.f, g.out, g.ostride, g.orow0);
    else
      down_tile<WT, NS, kDenseNT, false>(g.M, g.rows, g.len, r0, lane, g.vin, g.vstride, 0, g.ntok,
                                         nullptr, g.gscalar, g.out, g.ostride, 0);
  }
#else
  // Contiguous order: block b owns the tile range whose cost is 1/grid of the
  // total and walks it segment by segment; with LDSX each segment's input
  // rows are staged in LDS (as many as fit at once, all of them normally).
  Segments sg;
  sg.n = 0;
  sg.tiles[sg.n] = nr;
  sg.cost[sg.n++] = (long long)(a.has_routed ? a.r.inter : 0) * sizeof(WT) * NS + 1;
  for (int s = 0; s < a.n_dense; ++s) {
    sg.tiles[sg.n] = dstart[s + 1] - dstart[s];
    sg.cost[sg.n++] =
        (long long)a.dense[s].inter * sizeof(WT) * NS * ((a.T + kDenseNT - 1) / kDenseNT);
  }
  int lo, hi;
  block_range(sg, lo, hi);
  int t = lo;
  while (t < hi) {
    const DownSeg g = down_seg<WT>(a, t, nr, tr, dstart);
    const int t1 = min(hi, g.seg1);
    if (g.valid) {
      if constexpr (LDSX) {
        const int sst = staged_stride<EPU>(g.len);
        const int cap = uni(max(1, a.lds_floats / sst));
        for (int c0 = 0; c0 < g.ntok; c0 += cap) {
          const int nc = min(cap, g.ntok - c0);
          __syncthreads();  // the previous rows are no longer read
          stage_rows<EPU>(g.vin + (size_t)(g.vrow0 + c0) * g.vstride, g.vstride, nc, g.len);
          __syncthreads();
          for (int tile = t + wave; tile < t1; tile += kWavesPB) {
            const int r0 = (tile - g.seg0) * NS;
            if (g.routed)
              down_tile<WT, NS, kRoutedNT, true>(g.M, g.rows, g.len, r0, lane, nullptr, sst, 0, nc,
                                                 g.gates + c0, 0.f, g.out, g.ostride,
                                                 g.orow0 + c0);
            else
              down_tile<WT, NS, kDenseNT, true>(g.M, g.rows, g.len, r0, lane, nullptr, sst, 0, nc,
                                                nullptr, g.gscalar, g.out, g.ostride, c0);
          }
        }
      } else {
        for (int tile = t + wave; tile < t1; tile += kWavesPB) {
          const int r0 = (tile - g.seg0) * NS;
          if (g.routed)
            down_tile<WT, NS, kRoutedNT, false>(g.M, g.rows, g.len, r0, lane, g.vin, g.vstride,
                                                g.vrow0, g.ntok, g.gates, 0.f, g.out, g.ostride,
                                                g.orow0);
          else
            down_tile<WT, NS, kDenseNT, false>(g.M, g.rows, g.len, r0, lane, g.vin, g.vstride, 0,
                                               g.ntok, nullptr, g.gscalar, g.out, g.ostride, 0);
        }
      }
    }
    t = t1;
  }
#endif
}

// ------------------------------------------------------------------ combine

constexpr int kCombThreads = 1024;
constexpr int kCombPer = 4;

// y[t] = sum of the dense partials + sum_j P_r[pair_pos[t, j]] (+ residual),
// in that fixed order; optionally also RMSNorm(y).  One block per position;
// each thread's kCombPer elements are loaded independently.
__global__ __launch_bounds__(kCombThreads) void combine_kernel(CombineArgs a) {
  __shared__ float red[kCombThreads / 64];
  const int t = blockIdx.x;
  const size_t rowoff = (size_t)t * a.H;
  int pp[8];
  const int kk = a.p_r ? min(a.kk, 8) : 0;
  for (int j = 0; j < kk; ++j) {
    const int p = a.pair_pos[(size_t)t * a.kk + j];
    pp[j] = (p >= 0 && p < a.pairs_max) ? p : -1;
  }
  float ss = 0.f;
  for (int h0 = threadIdx.x; h0 < a.H; h0 += kCombThreads * kCombPer) {
    float v[kCombPer];
#pragma unroll
    for (int i = 0; i < kCombPer; ++i) {
      const int h = h0 + i * kCombThreads;
      float x = 0.f;
      if (h < a.H) {
        for (int s = 0; s < a.n_dense; ++s) x += a.dense_p[s][rowoff + h];
        for (int j = 0; j < kk; ++j)
          if (pp[j] >= 0) x += a.p_r[(size_t)pp[j] * a.H + h];
        for (int j = kk; j < (a.p_r ? a.kk : 0); ++j) {
          const int p = a.pair_pos[(size_t)t * a.kk + j];
          if (p >= 0 && p < a.pairs_max) x += a.p_r[(size_t)p * a.H + h];
        }
        if (a.residual) x = a.residual[rowoff + h] + x;
      }
      v[i] = x;
    }
#pragma unroll
    for (int i = 0; i < kCombPer; ++i) {
      const int h = h0 + i * kCombThreads;
      if (h < a.H) {
        a.y[rowoff + h] = v[i];
        ss = fmaf(v[i], v[i], ss);
      }
    }
  }
  if (a.normed) {
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    float tot = 0.f;
    for (int w = 0; w < kCombThreads / 64; ++w) tot += red[w];
    const float r = 1.0f / sqrtf(tot / (float)a.H + a.eps);
    for (int h = threadIdx.x; h < a.H; h += kCombThreads) a.normed[rowoff + h] = a.y[rowoff + h] * r;
  }
}

// ------------------------------------------------------------------ launch

template <typename K>
int occupancy_blocks(K kernel, size_t lds) {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kBlock, lds) != hipSuccess || n < 1)
    n = 1;
  return n;
}

// Grid: enough blocks to fill the device at the kernel's occupancy, never more
// than max_blocks (a block has work for up to 8 tiles at a time).
template <typename K>
hipError_t launch_persistent(K kernel, int max_blocks, size_t lds, const GroupedArgs& a,
                             hipStream_t s) {
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    attr_set = true;
  }
  const int occ = occupancy_blocks(kernel, lds);
  const int cap = dev_info().num_cus * occ;
  int g = max_blocks < cap ? max_blocks : cap;
  if (g < 1) g = 1;
  hipLaunchKernelGGL(kernel, dim3(g), dim3(kBlock), lds, s, a);
  return hipGetLastError();
}

int gateup_max_tiles(const GroupedArgs& a) {
  int t = a.has_routed ? a.r.max_union * ((a.r.inter + kGuRows - 1) / kGuRows) : 0;
  for (int s = 0; s < a.n_dense; ++s) t += (a.dense[s].inter + kGuRows - 1) / kGuRows;
  return t;
}

int down_max_tiles(const GroupedArgs& a, int rows_per_tile) {
  int t = a.has_routed ? a.r.max_union * ((a.H + rows_per_tile - 1) / rows_per_tile) : 0;
  for (int s = 0; s < a.n_dense; ++s) t += (a.dense[s].rows + rows_per_tile - 1) / rows_per_tile;
  return t;
}

template <typename WT>
size_t staged_bytes(int rows, int len) {
  return (size_t)rows * staged_stride<WTr<WT>::EPU>(len) * sizeof(float);
}

// The whole block of positions is staged in LDS when it fits the budget.
template <typename WT>
hipError_t gateup_typed(const GroupedArgs& a, hipStream_t s) {
  const int tiles = gateup_max_tiles(a);
  if (tiles == 0) return hipSuccess;
  const size_t lds = staged_bytes<WT>(a.T, a.H);
  if (lds <= (size_t)kLdsBudget)
    return launch_persistent(gateup_kernel<WT, true>, (tiles + kWavesPB - 1) / kWavesPB, lds, a, s);
  return launch_persistent(gateup_kernel<WT, false>, (tiles + kWavesPB - 1) / kWavesPB, 0, a, s);
}

#if DE_DN_STRIDED
// Strided order: a single dense source (the row-dot) stages all T input rows
// once when they fit; the grouped down reads its inputs directly.
template <typename WT, int NS>
hipError_t down_launch(GroupedArgs a, hipStream_t s) {
  const int tiles = (down_max_tiles(a, NS) + kWavesPB - 1) / kWavesPB;
  if (tiles == 0) return hipSuccess;
  if (!a.has_routed && a.n_dense == 1) {
    const size_t lds = staged_bytes<WT>(a.T, a.dense[0].inter);
    if (lds <= (size_t)kLdsBudget) {
      a.lds_floats = (int)(lds / sizeof(float));
      return launch_persistent(down_kernel<WT, true, NS>, tiles, lds, a, s);
    }
  }
  a.lds_floats = 0;
  return launch_persistent(down_kernel<WT, false, NS>, tiles, 0, a, s);
}
#else
// Inputs are staged in LDS when at least min(T, 4) rows of the longest input
// fit the per-block budget (two blocks per CU); otherwise (rows as long as a
// 10944-wide dense layer) they are read from global memory.
template <typename WT, int NS>
hipError_t down_launch(GroupedArgs a, hipStream_t s) {
  constexpr int EPU = WTr<WT>::EPU;
  const int tiles = (down_max_tiles(a, NS) + kWavesPB - 1) / kWavesPB;
  if (tiles == 0) return hipSuccess;
  int maxlen = a.has_routed ? a.r.inter : 0;
  for (int i = 0; i < a.n_dense; ++i) maxlen = maxlen > a.dense[i].inter ? maxlen : a.dense[i].inter;
  const int want = a.T < 4 ? a.T : 4;
  const size_t row_bytes = (size_t)staged_stride<EPU>(maxlen) * sizeof(float);
  if ((size_t)want * row_bytes <= (size_t)kDownLds) {
    size_t lds = (size_t)kDownLds;
    const size_t all = (size_t)a.T * row_bytes;
    if (all < lds) lds = all;
    a.lds_floats = (int)(lds / sizeof(float));
    return launch_persistent(down_kernel<WT, true, NS>, tiles, lds, a, s);
  }
  a.lds_floats = 0;
  return launch_persistent(down_kernel<WT, false, NS>, tiles, 0, a, s);
}
#endif

template <typename WT>
hipError_t down_typed(const GroupedArgs& a, hipStream_t s) {
  // One dense source and no routed part is a plain row-dot (the LM head, the
  // down projection of a dense layer).
  if (!a.has_routed && a.n_dense == 1) return down_launch<WT, kRdRows>(a, s);
  return down_launch<WT, kDnRows>(a, s);
}

}  // namespace

hipError_t launch_gateup(const GroupedArgs& a, int wdtype, hipStream_t s) {
  return wdtype == 1 ? gateup_typed<uint16_t>(a, s) : gateup_typed<float>(a, s);
}

hipError_t launch_down(const GroupedArgs& a, int wdtype, hipStream_t s) {
  return wdtype == 1 ? down_typed<uint16_t>(a, s) : down_typed<float>(a, s);
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(combine_kernel, dim3(a.T), dim3(kCombThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace de
