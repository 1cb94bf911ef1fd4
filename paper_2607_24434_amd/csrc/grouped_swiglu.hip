// Grouped SwiGLU over the expert union plus the shared / draft / dense
// sources (Eq. 4 and Eq. 5 without the routing), and the fixed-order combine.
//
// With at most a few block positions per expert the work is a batch of skinny
// GEMVs: every weight byte is used by only |T_e| tokens, so the kernels are
// bound by HBM bandwidth, not arithmetic.  The design is therefore about
// keeping enough 128-bit loads in flight:
//
//  * A block of 256 threads (4 waves) owns a tile of rows of one source.
//    Within a wave, four 16-lane groups each own RG rows; the reduction
//    dimension is split across the four waves (interleaved 16-byte units),
//    so a tile exposes 4x more independent loads than one wave could hold.
//  * Each lane issues all the loads of its slice up front (MAXI iterations x
//    streams x 16 B), then does the FMAs: bf16 -> fp32 by a shift or mask,
//    fp32 accumulation, activations fp32.
//  * Per-group sums use four DPP steps inside a 16-lane row; the four waves'
//    partials meet in LDS and are added in a fixed order.  No float atomics
//    anywhere, so results are bitwise reproducible.
//  * Persistent grid: the number of routed tiles depends on the union size,
//    which stays on the device; blocks stride over tiles and exit when done.
//  * Weight loads are non-temporal: each byte is read once per pass.
#include "de_common.h"

namespace de {
namespace {

constexpr int kBlock = 512;                 // 8 waves share the staged activations
constexpr int kWavesPB = kBlock / kWave;
constexpr int kGroups = kWave / 16;         // 16-lane groups per wave
constexpr int kDnRG = 2;                    // rows per group in the down / row-dot kernel
constexpr int kMaxNT = 8;                   // positions per pass
constexpr int kTokGroup = 4;                // positions whose activation loads may be hoisted together
constexpr int kMaxNTDown = 4;               // positions per pass in the down kernel
constexpr int kLdsBudget = 144 * 1024;      // staged activations per block (gate/up)
constexpr int kDownLds = 72 * 1024;         // staged input rows per block (down), two blocks/CU

// 16-byte iterations whose weight loads are issued together, by positions per
// pass: more positions need more accumulators, leaving fewer registers.
// Activations read from global memory are hoisted further (longer latency),
// so that path keeps fewer weight iterations in flight.
template <int NT, bool LDSX>
struct InFlight {
  static constexpr int MI = LDSX ? (NT <= 4 ? 4 : 2) : (NT <= 2 ? 4 : 2);
};

// Dynamic LDS: the block's activation rows (gate/up: x; row-dot: its inputs).
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

// Dot products of NS weight rows with up to NT activation rows.  The GR
// groups of one row set split each row: group `sub` owns the 16-unit
// iterations it = sub, sub+GR, ... and lane lg the unit u = it*16 + lg, so a
// wave instruction reads GR contiguous 256-byte pieces of one row.  Loads of
// kMI iterations are issued together, then consumed.  Activation row m of the
// pass starts at float offset voff[m] (LDS or global).  The sums are partial
// per lane; row_total() finishes them.
template <typename WT, int NS, int NT, bool LDSX, int GR>
__device__ __forceinline__ void rows_dot(const char* const (&rowp)[NS], int L, int sub, int lg,
                                         const float* gact, const int (&voff)[NT], int nt,
                                         float (&acc)[NS][NT]) {
  constexpr int EPU = WTr<WT>::EPU;
  constexpr int kMI = InFlight<NT, LDSX>::MI;
  const int nit = (L + 15) >> 4;
  const int my_nit = nit > sub ? (nit - sub + GR - 1) / GR : 0;
  for (int i0 = 0; i0 < my_nit; i0 += kMI) {
    u32x4 raw[kMI][NS];
#pragma unroll
    for (int q = 0; q < kMI; ++q) {
      const int u = (sub + GR * (i0 + q)) * 16 + lg;
      const bool ok = i0 + q < my_nit && u < L;
#pragma unroll
      for (int s = 0; s < NS; ++s)
        raw[q][s] = ok ? load_stream16(rowp[s] + (size_t)u * 16) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int q = 0; q < kMI; ++q) {
      if (i0 + q >= my_nit) break;
      const int u = (sub + GR * (i0 + q)) * 16 + lg;
      const bool ok = u < L;
      float w[NS][EPU];
#pragma unroll
      for (int s = 0; s < NS; ++s) unpack(raw[q][s], w[s]);
#pragma unroll
      for (int m = 0; m < NT; ++m) {
        if (m < nt) {
          float xv[EPU];
          if (ok) {
            act_frag<EPU, LDSX>(gact, voff[m], u, xv);
          } else {
#pragma unroll
            for (int v = 0; v < EPU; ++v) xv[v] = 0.f;
          }
#pragma unroll
          for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int v = 0; v < EPU; ++v) acc[s][m] = fmaf(w[s][v], xv[v], acc[s][m]);
        }
        // Keep the scheduler from hoisting every position's activation loads
        // at once: that would exceed the register budget and spill.
        if ((m + 1) % kTokGroup == 0 && m + 1 < NT) __builtin_amdgcn_sched_barrier(0);
      }
      if (NT > kTokGroup) __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// Total of a per-lane partial over the 16 lanes of a group and the GR groups
// of its row set; every lane of the row set receives the same bits.
template <int GR>
__device__ __forceinline__ float row_total(float v) {
  v = row16_sum(v);
  if (GR >= 2) v += __shfl_xor(v, 16, kWave);
  if (GR >= 4) v += __shfl_xor(v, 32, kWave);
  return v;
}

__device__ __forceinline__ int cdiv(int a, int b) { return (a + b - 1) / b; }

// Values that are the same in every lane (tile and segment metadata, read from
// memory) are moved to scalar registers; the compiler cannot prove it itself
// for loaded values, and keeping them in vector registers causes spills.
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ float uni(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}
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

// Tiles are laid out as consecutive segments (the union members, then each
// dense source); every tile of a segment has the same cost (bytes streamed
// times position passes).  Block b owns the contiguous tile range whose cost
// covers [b, b+1) * total_cost / grid, so blocks finish together even when
// some segments (the shared path with 9+ positions, rows twice as long) are
// several times more expensive per tile than the routed ones.
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
    if (c < c0 + seg) {
      const long long k = (c - c0 + sg.cost[i] - 1) / sg.cost[i];
      return t0 + (int)k;
    }
    t0 += sg.tiles[i];
    c0 += seg;
  }
  return t0;
}

__device__ __forceinline__ void block_range(const Segments& sg, int& lo, int& hi) {
  long long total = 0;
  for (int i = 0; i < sg.n; ++i) total += (long long)sg.tiles[i] * sg.cost[i];
  const long long a = total * blockIdx.x / gridDim.x;
  const long long b = total * (blockIdx.x + 1) / gridDim.x;
  lo = tile_at_cost(sg, a);
  hi = tile_at_cost(sg, b);
}

__device__ __forceinline__ long long passes(int ntok) { return (ntok + kMaxNT - 1) / kMaxNT; }

// a.dense[s] with a run-time s would copy the kernel-argument array to scratch
// memory; an explicit select keeps everything in scalar registers.
__device__ __forceinline__ DenseSrc pick_dense(const GroupedArgs& a, int s) {
  return s == 0 ? a.dense[0] : (s == 1 ? a.dense[1] : a.dense[2]);
}

// ------------------------------------------------------------------ gate/up

// One pass (up to NT positions) over the (G, U) row pair r of one group:
// A[arow0 + m][r] = silu(G_r . x_m) * (U_r . x_m).
template <typename WT, int NT, bool LDSX, int GR>
__device__ __forceinline__ void gateup_pass(const char* G, const char* U, int inter, int H, int r,
                                            int sub, int lg, int xstride, const float* gx, int T,
                                            const int32_t* tok, int tok_base, int nt, float* A,
                                            int arow0) {
  const size_t rb = (size_t)H * sizeof(WT);
  const int rc = min(r, inter - 1);
  const char* rowp[2] = {G + (size_t)rc * rb, U + (size_t)rc * rb};
  int voff[NT];
#pragma unroll
  for (int m = 0; m < NT; ++m) {
    int t = uni(m < nt ? (tok ? tok[m] : tok_base + m) : tok_base);
    t = t < 0 ? 0 : (t >= T ? T - 1 : t);  // a position outside the block never indexes x
    voff[m] = t * xstride;
  }
  float acc[2][NT];
#pragma unroll
  for (int m = 0; m < NT; ++m) acc[0][m] = acc[1][m] = 0.f;
  rows_dot<WT, 2, NT, LDSX, GR>(rowp, (int)(rb / 16), sub, lg, gx, voff, nt, acc);
#pragma unroll
  for (int m = 0; m < NT; ++m) {
    if (m < nt) {
      const float g = row_total<GR>(acc[0][m]);
      const float u = row_total<GR>(acc[1][m]);
      if (sub == 0 && lg == m && r < inter) A[(size_t)(arow0 + m) * inter + r] = silu_f(g) * u;
    }
  }
}

template <typename WT, bool LDSX, int GR>
__device__ __forceinline__ void gateup_rows(const char* G, const char* U, int inter, int H, int r,
                                            int sub, int lg, int xstride, const float* gx, int T,
                                            const int32_t* tok, int ntok, float* A, int arow0) {
  for (int m0 = 0; m0 < ntok; m0 += kMaxNT) {
    const int nt = min(kMaxNT, ntok - m0);
    const int32_t* tk = tok ? tok + m0 : nullptr;
#define DE_GU(NTV) \
  gateup_pass<WT, NTV, LDSX, GR>(G, U, inter, H, r, sub, lg, xstride, gx, T, tk, m0, nt, A, arow0 + m0)
    if (nt <= 1)
      DE_GU(1);
    else if (nt <= 2)
      DE_GU(2);
    else if (nt <= 4)
      DE_GU(4);
    else
      DE_GU(8);
#undef DE_GU
  }
}

// Persistent gate/up kernel.  Tiles: kGuRows consecutive (G, U) row pairs of
// one source (union members first, then the dense sources); block b owns a
// contiguous tile range and its waves take every 8th tile of it.
template <typename WT, bool LDSX, int GR>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void gateup_kernel(
    GroupedArgs a) {
  constexpr int EPU = WTr<WT>::EPU;
  constexpr int kGuRows = kGroups / GR;  // (G, U) row pairs per wave tile
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane >> 4, lg = lane & 15;
  const int rset = grp / GR, sub = grp % GR;
  int xstride = a.H;
  if constexpr (LDSX) {
    stage_rows<EPU>(a.x, a.H, a.T, a.H);
    __syncthreads();
    xstride = staged_stride<EPU>(a.H);
  }
  const int nu = routed_count(a);
  const int tr = a.has_routed ? cdiv(a.r.inter, kGuRows) : 0;
  const int nr = nu * tr;
  const long long row_cost = (long long)a.H * sizeof(WT) * 2 * kGuRows;
  Segments sg;
  sg.n = 0;
  sg.tiles[sg.n] = nr;
  sg.cost[sg.n++] = row_cost;  // a union member has one pass in the common case
  int dstart[3];
  int total = nr;
  for (int s = 0; s < a.n_dense; ++s) {
    dstart[s] = total;
    sg.tiles[sg.n] = cdiv(a.dense[s].inter, kGuRows);
    sg.cost[sg.n++] = row_cost * passes(a.T);
    total += sg.tiles[sg.n - 1];
  }
  int lo, hi;
  block_range(sg, lo, hi);
  const size_t esz = sizeof(WT);
  int cur_j = -1, off = 0, ntok = 0;  // member metadata, reused while the wave stays in it
  const char* blk = nullptr;
  for (int tile = lo + wave; tile < hi; tile += kWavesPB) {
    if (tile < nr) {
      const int j = tile / tr, rt = tile - j * tr;
      if (j != cur_j) {
        blk = member_block(a.r, j, off, ntok);
        cur_j = j;
      }
      if (blk == nullptr) continue;
      const char* U = blk + (size_t)a.r.inter * a.H * esz;
      gateup_rows<WT, LDSX, GR>(blk, U, a.r.inter, a.H, rt * kGuRows + rset, sub, lg, xstride, a.x,
                                a.T, a.r.tok_list + off, ntok, a.r.a, off);
    } else {
      int s = 0;
      while (s + 1 < a.n_dense && tile >= dstart[s + 1]) ++s;
      const DenseSrc d = pick_dense(a, s);
      const char* G = static_cast<const char*>(d.w);
      const char* U = G + (size_t)d.inter * a.H * esz;
      gateup_rows<WT, LDSX, GR>(G, U, d.inter, a.H, (tile - dstart[s]) * kGuRows + rset, sub, lg,
                                xstride, a.x, a.T, nullptr, a.T, d.out, 0);
    }
  }
}

// ------------------------------------------------------------------ down / row-dot

// One pass over the kDnRG rows r0.. of one group of a [rows, len] matrix:
// out[orow0 + m][r] = gate_m * (M_r . v_m).
template <typename WT, int NT, bool LDSX, int GR>
__device__ __forceinline__ void down_pass(const char* M, int rows, int len, int r0, int sub, int lg,
                                          const float* gv, int vstride, int vrow0, int nt,
                                          const float* gates, float gscalar, float* out,
                                          int ostride, int orow0) {
  const size_t rb = (size_t)len * sizeof(WT);
  const char* rowp[kDnRG];
#pragma unroll
  for (int k = 0; k < kDnRG; ++k) rowp[k] = M + (size_t)min(r0 + k, rows - 1) * rb;
  int voff[NT];
#pragma unroll
  for (int m = 0; m < NT; ++m) voff[m] = (vrow0 + (m < nt ? m : 0)) * vstride;
  float acc[kDnRG][NT];
#pragma unroll
  for (int k = 0; k < kDnRG; ++k)
#pragma unroll
    for (int m = 0; m < NT; ++m) acc[k][m] = 0.f;
  rows_dot<WT, kDnRG, NT, LDSX, GR>(rowp, (int)(rb / 16), sub, lg, gv, voff, nt, acc);
#pragma unroll
  for (int m = 0; m < NT; ++m) {
    if (m < nt) {
#pragma unroll
      for (int k = 0; k < kDnRG; ++k) {
        const float v = row_total<GR>(acc[k][m]);
        if (sub == 0 && lg == m && r0 + k < rows)
          out[(size_t)(orow0 + m) * ostride + r0 + k] = (gates ? gates[m] : gscalar) * v;
      }
    }
  }
}

template <typename WT, bool LDSX, int GR>
__device__ __forceinline__ void down_rows(const char* M, int rows, int len, int r0, int sub, int lg,
                                          const float* gv, int vstride, int vrow0, int ntok,
                                          const float* gates, float gscalar, float* out,
                                          int ostride, int orow0) {
  for (int m0 = 0; m0 < ntok; m0 += kMaxNTDown) {
    const int nt = min(kMaxNTDown, ntok - m0);
    const float* gg = gates ? gates + m0 : nullptr;
#define DE_DN(NTV)                                                                              \
  down_pass<WT, NTV, LDSX, GR>(M, rows, len, r0, sub, lg, gv, vstride, vrow0 + m0, nt, gg, gscalar, out, \
                           ostride, orow0 + m0)
    if (nt <= 1)
      DE_DN(1);
    else if (nt <= 2)
      DE_DN(2);
    else
      DE_DN(4);
#undef DE_DN
  }
}

// Persistent down-projection / row-dot kernel over the union members and the
// dense sources.  A block walks its tile range segment by segment (a segment
// is the part of one source inside the range); with LDSX the segment's input
// rows (the member's A rows, a dense source's rows) are staged in LDS once,
// in passes of at most `npass` positions, and every wave of the block reads
// them from there.
template <typename WT, bool LDSX, int GR>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void down_kernel(
    GroupedArgs a) {
  constexpr int EPU = WTr<WT>::EPU;
  constexpr int kDnRows = (kGroups / GR) * kDnRG;  // rows per wave tile
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane >> 4, lg = lane & 15;
  const int rset = grp / GR, sub = grp % GR;
  const int nu = routed_count(a);
  const int tr = a.has_routed ? cdiv(a.H, kDnRows) : 0;
  const int nr = nu * tr;
  Segments sg;
  sg.n = 0;
  sg.tiles[sg.n] = nr;
  sg.cost[sg.n++] = (long long)(a.has_routed ? a.r.inter : 0) * sizeof(WT) * kDnRows + 1;
  int dstart[4];
  int total = nr;
  for (int s = 0; s < a.n_dense; ++s) {
    dstart[s] = total;
    sg.tiles[sg.n] = cdiv(a.dense[s].rows, kDnRows);
    sg.cost[sg.n++] = (long long)a.dense[s].inter * sizeof(WT) * kDnRows *
                      ((a.T + kMaxNTDown - 1) / kMaxNTDown);
    total += sg.tiles[sg.n - 1];
  }
  dstart[a.n_dense] = total;
  int lo, hi;
  block_range(sg, lo, hi);
  const size_t esz = sizeof(WT);
  int t = lo;
  while (t < hi) {
    // ---- the segment containing tile t
    const char* M;
    const float* vin;
    const float* gates;
    float* out;
    int rows, len, vstride, vrow0, ntok, ostride, orow0, seg0, seg1;
    float gscalar = 0.f;
    if (t < nr) {
      const int j = t / tr;
      seg0 = j * tr;
      seg1 = min(hi, seg0 + tr);
      int off = 0;
      ntok = 0;
      const char* blk = member_block(a.r, j, off, ntok);
      if (blk == nullptr) {
        t = seg1;
        continue;
      }
      M = blk + 2 * (size_t)a.r.inter * a.H * esz;
      rows = a.H;
      len = a.r.inter;
      vin = a.r.a;
      vstride = a.r.inter;
      vrow0 = off;
      gates = a.r.gate_list + off;
      out = a.r.p;
      ostride = a.H;
      orow0 = off;
    } else {
      int s = 0;
      while (s + 1 < a.n_dense && t >= dstart[s + 1]) ++s;
      const DenseSrc d = pick_dense(a, s);
      seg0 = dstart[s];
      seg1 = min(hi, dstart[s + 1]);
      M = static_cast<const char*>(d.w);
      rows = d.rows;
      len = d.inter;
      vin = d.vin;
      vstride = d.vin_stride;
      vrow0 = 0;
      ntok = a.T;
      gates = nullptr;
      gscalar = d.gate;
      out = d.out;
      ostride = d.out_stride;
      orow0 = 0;
    }
    if constexpr (LDSX) {
      const int sst = staged_stride<EPU>(len);
      const int npass = max(1, min(kMaxNTDown, a.lds_floats / sst));
      for (int m0 = 0; m0 < ntok; m0 += npass) {
        const int np = min(npass, ntok - m0);
        __syncthreads();  // the previous rows are no longer read
        stage_rows<EPU>(vin + (size_t)(vrow0 + m0) * vstride, vstride, np, len);
        __syncthreads();
        for (int tile = t + wave; tile < seg1; tile += kWavesPB) {
          const int r0 = (tile - seg0) * kDnRows + rset * kDnRG;
          down_rows<WT, true, GR>(M, rows, len, r0, sub, lg, nullptr, sst, 0, np,
                                  gates ? gates + m0 : nullptr, gscalar, out, ostride,
                                  orow0 + m0);
        }
      }
    } else {
      for (int tile = t + wave; tile < seg1; tile += kWavesPB) {
        const int r0 = (tile - seg0) * kDnRows + rset * kDnRG;
        down_rows<WT, false, GR>(M, rows, len, r0, sub, lg, vin, vstride, vrow0, ntok, gates,
                                 gscalar, out, ostride, orow0);
      }
    }
    t = seg1;
  }
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

template <typename K>
int occupancy_blocks(K kernel, size_t lds) {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kBlock, lds) != hipSuccess || n < 1)
    n = 1;
  return n;
}

template <typename K>
hipError_t launch_persistent(K kernel, int max_tiles, size_t lds, const GroupedArgs& a,
                             hipStream_t s) {
  static bool attr_set = false;
  if (!attr_set) {
    hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    attr_set = true;
  }
  const int occ = occupancy_blocks(kernel, lds);
  const int cap = dev_info().num_cus * occ;
  int g = max_tiles < cap ? max_tiles : cap;
  if (g < 1) g = 1;
  hipLaunchKernelGGL(kernel, dim3(g), dim3(kBlock), lds, s, a);
  return hipGetLastError();
}

// Groups per row: all four groups of a wave stream the same rows (1 KB per
// wave load, 4x more tiles than one group per row), which keeps every wave
// of the grid busy even for the one-position draft layer.
constexpr int kGR = 4;

int gateup_max_tiles(const GroupedArgs& a) {
  const int rows = kGroups / kGR;
  int t = a.has_routed ? a.r.max_union * ((a.r.inter + rows - 1) / rows) : 0;
  for (int s = 0; s < a.n_dense; ++s) t += (a.dense[s].inter + rows - 1) / rows;
  return t;
}

int down_max_tiles(const GroupedArgs& a) {
  const int rows = (kGroups / kGR) * kDnRG;
  int t = a.has_routed ? a.r.max_union * ((a.H + rows - 1) / rows) : 0;
  for (int s = 0; s < a.n_dense; ++s) t += (a.dense[s].rows + rows - 1) / rows;
  return t;
}

template <typename WT>
size_t staged_bytes(int rows, int len) {
  return (size_t)rows * staged_stride<WTr<WT>::EPU>(len) * sizeof(float);
}

template <typename WT>
hipError_t gateup_typed(const GroupedArgs& a, hipStream_t s) {
  const int tiles = gateup_max_tiles(a);
  if (tiles == 0) return hipSuccess;
  const size_t lds = staged_bytes<WT>(a.T, a.H);
  if (lds <= (size_t)kLdsBudget)
    return launch_persistent(gateup_kernel<WT, true, kGR>, tiles, lds, a, s);
  return launch_persistent(gateup_kernel<WT, false, kGR>, tiles, 0, a, s);
}

template <typename WT>
hipError_t down_typed(GroupedArgs a, hipStream_t s) {
  const int tiles = down_max_tiles(a);
  if (tiles == 0) return hipSuccess;
  // Stage inputs in LDS when a pass of min(T, 4) positions of the longest
  // input row fits the per-block budget (two blocks per CU); otherwise
  // (long rows such as a 10944-wide dense layer) read them from global memory.
  constexpr int EPU = WTr<WT>::EPU;
  int maxlen = a.has_routed ? a.r.inter : 0;
  for (int i = 0; i < a.n_dense; ++i) maxlen = maxlen > a.dense[i].inter ? maxlen : a.dense[i].inter;
  const int want = a.T < 4 ? a.T : 4;
  int rows_cap = a.has_routed ? a.T : 0;  // positions per member (at most T)
  for (int i = 0; i < a.n_dense; ++i) rows_cap = a.T;
  const size_t need = (size_t)want * staged_stride<EPU>(maxlen) * sizeof(float);
  if (need <= (size_t)kDownLds) {
    size_t lds = (size_t)kDownLds;
    const size_t all = (size_t)rows_cap * staged_stride<EPU>(maxlen) * sizeof(float);
    if (all < lds) lds = all;
    a.lds_floats = (int)(lds / sizeof(float));
    return launch_persistent(down_kernel<WT, true, kGR>, tiles, lds, a, s);
  }
  a.lds_floats = 0;
  return launch_persistent(down_kernel<WT, false, kGR>, tiles, 0, a, s);
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
