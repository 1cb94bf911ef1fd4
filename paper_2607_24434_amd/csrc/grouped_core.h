// The pass stream of the grouped SwiGLU kernels (internal): weight tiles of
// union members and dense sources, each lane's 16-byte units, the register
// ring of weight loads, the FMA order and the row reductions.  Shared by the
// separate gate/up and down launches and by the single-launch verify layer,
// which therefore compute every output value with the same operations.
//
// With a few block positions per expert the work is a batch of skinny GEMVs:
// every weight byte meets only |T_e| positions, so the kernels are bound by
// HBM bandwidth, not arithmetic.  The design keeps the memory system busy
// without pause and touches each weight byte once:
//
//  * Persistent blocks over a tile list: each dense source's row tiles, then
//    the union members'.  Wave w of block b takes the tiles b*W + w (W waves
//    per block), then every (grid*W)-th one, so at any moment the whole grid
//    streams a narrow window of consecutive rows.
//  * A tile is 4 weight rows (gate/up: two (G, U) row pairs) and expands into
//    passes of up to 4 positions.  All 64 lanes of a wave stream the same
//    rows: lane l owns the 16-byte units it*64 + l, so one load instruction
//    reads 1 KB of a row (128-bit non-temporal loads).
//  * The wave's passes form one flat sequence of 16-byte iterations.  A ring
//    of kRing iterations (x 4 rows) of weights lives in registers: the loader
//    runs kRing iterations ahead of the consumer across pass and tile
//    boundaries, so the next tile's first loads are in flight while the
//    current one finishes and its sums are reduced.
//  * bf16 -> fp32 by a shift or mask, fp32 accumulation; a row sum is four DPP
//    steps inside 16 lanes and two cross-row shuffles, identical in every
//    lane.  No float atomics: results are bitwise reproducible.
#pragma once

#include "de_common.h"
#include "draftexpert.h"
#include "topk_union.h"

#include <type_traits>

// Build-time tuning knobs (kept at the measured best by default).
#ifndef DE_NT_LOADS
#define DE_NT_LOADS 1
#endif
#ifndef DE_RING
#define DE_RING 4
#endif
#ifndef DE_DENSE_RING
#define DE_DENSE_RING 2
#endif
#ifndef DE_DENSE_NT
#define DE_DENSE_NT 9
#endif

namespace de {
namespace {

constexpr int kBlock = 512;                 // 8 waves share the staged activations
constexpr int kWavesPB = kBlock / kWave;
constexpr int kNS = 4;                      // weight rows per tile
constexpr int kRoutedNT = 4;                // positions per pass of a union member
constexpr int kDenseNT = DE_DENSE_NT;       // positions per pass of a dense source
constexpr int kMaxStaged = 32;              // union members with input rows staged per block (down)
constexpr int kRing = DE_RING;              // 16-byte iterations in flight per lane (x kNS), members
constexpr int kDenseRing = DE_DENSE_RING;   // the same, dense sources
constexpr int kCombThreads = 1024;             // the combine: threads per position
constexpr int kCombPer = 4;                 // row elements per combine thread held in registers
constexpr int kLdsBudget = 144 * 1024;      // staged activations + tables per block (gate/up)
constexpr int kDownLds = 76 * 1024;         // staged inputs + tables per block (down): two blocks/CU

// Dynamic LDS: staged activation rows, then the member table and the lists.
extern __shared__ __align__(16) float s_dyn[];

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

// Q4_0 weights: blocks of 32 weights of a row, 16 bytes of 4-bit codes q
// (byte j: weight j in the low nibble, weight j + 16 in the high one) and an
// fp16 scale d; weight = d (q - 8).  A [rows, cols] matrix holds every row's
// codes (cols / 2 bytes per row), then every row's scales (cols / 16 bytes).
struct q4_t {};
template <>
struct WTr<q4_t> {
  static constexpr int EPU = 32;
};

template <typename WT>
constexpr bool kQ4 = std::is_same_v<WT, q4_t>;

// Positions per pass and ring depth.  Q4_0 units carry four times the
// weights of a bf16 unit (and its arithmetic): fewer positions per pass and a
// shallower ring keep the unrolled stream in registers, and the 16-byte loads
// in flight per wave (2 x 4 KB) still cover the memory latency.
template <typename WT>
constexpr int kDenseNTOf = kQ4<WT> ? 3 : kDenseNT;
template <typename WT>
constexpr int kRoutedNTOf = kQ4<WT> ? 2 : kRoutedNT;
template <typename WT>
constexpr int kRingOf = kQ4<WT> ? 2 : kRing;

// Bytes per row of a matrix's codes (or plain values).
template <typename WT>
__host__ __device__ __forceinline__ size_t qrow_bytes(int cols) {
  if constexpr (kQ4<WT>)
    return (size_t)cols / 2;
  else
    return (size_t)cols * sizeof(WT);
}

// Bytes of a [rows, cols] matrix.
template <typename WT>
__host__ __device__ __forceinline__ size_t mat_bytes(int rows, int cols) {
  if constexpr (kQ4<WT>)
    return (size_t)rows * cols * 9 / 16;
  else
    return (size_t)rows * cols * sizeof(WT);
}

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
// stored at ((u/16)*2 + half)*16 + u%16, so the 16 lanes of a row group read
// 256 contiguous bytes per ds_read_b128 (no bank conflicts).  Rows are padded
// to a multiple of 128 floats.  fp32 weights (4 per unit) keep the natural
// order.
__device__ __forceinline__ int perm_index(int u, int half) {
  return (((u >> 4) * 2 + half) * 16 + (u & 15)) * 4;
}

// Q4_0 weights (32 per unit): unit u's 32 floats stay in its own 128 bytes,
// its float4 j stored at slot (j + u / 2) mod 8, so that 16 lanes reading
// float4 j of 16 consecutive units hit 64 distinct banks (no padding: the
// rows of a 9-position block still fit two blocks per CU).
template <int EPU>
__host__ __device__ __forceinline__ int staged_stride(int len) {
  return EPU == 8 ? ((len + 127) / 128) * 128 : len;
}

__device__ __forceinline__ int q4_slot(int u, int j) { return u * 32 + 4 * ((j + (u >> 1)) & 7); }

// LDS float offset of float4 h4 of a staged row.
template <int EPU>
__device__ __forceinline__ int staged_f4(int h4) {
  if constexpr (EPU == 8) return perm_index(h4 >> 1, h4 & 1);
  if constexpr (EPU == 32) return q4_slot(h4 >> 3, h4 & 7);
  return h4 * 4;
}

// The EPU activations that meet weight unit u of one row: from LDS (staged
// layout, row at float offset `off`) when g is null, else from global memory
// (natural layout).
// Staged offsets are multiples of 4 floats; indexing LDS as float4 lets the
// compiler use 16-byte reads (a float pointer plus an offset it cannot prove
// aligned is read as pairs of dwords).
__device__ __forceinline__ float4 lds4(int off_floats) {
  return reinterpret_cast<const float4*>(s_dyn)[off_floats >> 2];
}

template <int EPU>
__device__ __forceinline__ void act_frag(const float* g, int off, int u, float (&v)[EPU]) {
  if (g == nullptr) {
    if constexpr (EPU == 8) {
      const float4 a = lds4(off + perm_index(u, 0));
      const float4 b = lds4(off + perm_index(u, 1));
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
      v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
      const float4 a = lds4(off + u * 4);
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

// Half h (weights 16 h .. 16 h + 15) of the 32 activations that meet Q4_0
// unit u: from LDS (staged layout) when g is null, else from global memory.
__device__ __forceinline__ void act_half_q4(const float* g, int off, int u, int h,
                                            float (&v)[16]) {
  if (g == nullptr) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float4 a = lds4(off + q4_slot(u, 4 * h + i));
      v[4 * i + 0] = a.x; v[4 * i + 1] = a.y; v[4 * i + 2] = a.z; v[4 * i + 3] = a.w;
    }
  } else {
    const DE_GLOBAL f32x4* q = gptr<f32x4>(g + off + u * 32 + 16 * h);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x4 t = q[i];
      v[4 * i + 0] = t.x; v[4 * i + 1] = t.y; v[4 * i + 2] = t.z; v[4 * i + 3] = t.w;
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
    const int dst = t * sst + staged_f4<EPU>(h4);
    *reinterpret_cast<f32x4*>(&s_dyn[dst]) = v;
  }
}

// The same, into LDS at dst.
template <int EPU>
__device__ __forceinline__ void stage_rows_at(float* dst, const float* g, int gstride, int rows,
                                              int len) {
  const int l4 = len >> 2;
  const int sst = staged_stride<EPU>(len);
  for (int i = threadIdx.x; i < rows * l4; i += kBlock) {
    const int t = i / l4, h4 = i - t * l4;
    const f32x4 v = gptr<f32x4>(g + (size_t)t * gstride)[h4];
    const int o = t * sst + staged_f4<EPU>(h4);
    *reinterpret_cast<f32x4*>(dst + o) = v;
  }
}

// Total of a per-lane partial over the 64 lanes of a wave; every lane receives
// the same bits.
__device__ __forceinline__ float row_total(float v) { return wave_sum(v); }

__host__ __device__ __forceinline__ int cdiv(int a, int b) { return (a + b - 1) / b; }

// Values that are the same in every lane (tile and pass metadata, read from
// memory or produced by integer division, which has no scalar instruction)
// are moved to scalar registers; the compiler cannot prove it itself, and
// keeping them in vector registers causes spills.
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
template <typename P>
__device__ __forceinline__ P* uni(P* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<P*>(((uint64_t)hi << 32) | lo);
}

// The dense sources are read from an LDS copy (Tables::dense): a run-time
// index into the kernel argument (a.dense[s]) makes the compiler copy the
// whole argument to per-lane scratch memory.

// ------------------------------------------------------------------ block tables

// A union member as a block sees it: its weight block (null when the expert
// is not resident or the lists are malformed), first pair, positions, and the
// LDS float offset of its staged input rows (down only; -1: global memory).
struct Member {
  const char* blk;
  int off;
  int ntok;
  int act;
  int pad;
};

// LDS layout: [staged activations: act_floats][dense: 3][members: max_union]
//             [tok: pairs_max][gate: pairs_max]
struct Tables {
  DenseSrc* dense;
  Member* mem;
  int32_t* tok;
  float* gate;
  int* dact;  // single-launch verify layer: LDS offsets of the dense sources' staged inputs
};

size_t tables_bytes(const GroupedArgs& a) {
  size_t b = 3 * sizeof(DenseSrc);
  if (a.has_routed) b += (size_t)a.r.max_union * sizeof(Member) + (size_t)a.r.pairs_max * 8;
  if (a.fuse_route) b += sel_view_bytes(a.T, a.sel.k, a.sel.N);
  return b;
}

// The selection state after the tables (fused routing only).
__device__ __forceinline__ SelView sel_at(const GroupedArgs& a, const Tables& tb) {
  char* p = reinterpret_cast<char*>(tb.gate + (a.has_routed ? a.r.pairs_max : 0));
  return sel_view_at(p, a.T, a.sel.k, a.sel.N);
}

// The member table from a union built in LDS: member j = the expert with
// union index j.  All threads; the caller synchronises.
__device__ __forceinline__ void members_from_union(const GroupedArgs& a, const Tables& tb,
                                                   const SelView& v, int first, int stride,
                                                   int* absent) {
  const RoutedSrc& r = a.r;
  for (int e = first; e < a.sel.N; e += stride) {
    const unsigned long long m = v.mask[e];
    if (m == 0ull) continue;
    const int slot = e < r.n_experts ? (r.slot_of_expert ? r.slot_of_expert[e] : e) : -1;
    Member mb{nullptr, v.off[e], (int)__popcll(m), -1, 0};
    if (slot >= 0 && slot < r.n_slots)
      mb.blk = r.base + (size_t)slot * r.stride;
    else
      *absent = 1;
    tb.mem[v.upos[e]] = mb;
  }
}

__device__ __forceinline__ Tables tables_at(const GroupedArgs& a, int act_floats) {
  Tables tb;
  char* p = reinterpret_cast<char*>(s_dyn + act_floats);
  tb.dense = reinterpret_cast<DenseSrc*>(p);
  p += 3 * sizeof(DenseSrc);
  tb.mem = reinterpret_cast<Member*>(p);
  const int nm = a.has_routed ? a.r.max_union : 0;
  tb.tok = reinterpret_cast<int32_t*>(p + (size_t)nm * sizeof(Member));
  tb.gate = reinterpret_cast<float*>(tb.tok + (a.has_routed ? a.r.pairs_max : 0));
  tb.dact = nullptr;
  return tb;
}

// Dense source s from the LDS copy, in scalar registers.
__device__ __forceinline__ DenseSrc dense_at(const Tables& tb, int s) {
  const DenseSrc& g = tb.dense[s];
  DenseSrc d;
  d.w = uni(g.w);
  d.inter = uni(g.inter);
  d.ld = uni(g.ld);
  d.rows = uni(g.rows);
  d.gate = __int_as_float(uni(__float_as_int(g.gate)));
  d.vin = uni(g.vin);
  d.vin_stride = uni(g.vin_stride);
  d.out = uni(g.out);
  d.out_stride = uni(g.out_stride);
  d.ws = uni(g.ws);
  d.out_tag = uni(g.out_tag);
  return d;
}

// Copies the dense-source descriptors to LDS (static indices only).  The
// caller synchronises.
__device__ __forceinline__ void fill_dense(const GroupedArgs& a, const Tables& tb) {
  if (threadIdx.x == 0 && a.n_dense > 0) tb.dense[0] = a.dense[0];
  if (threadIdx.x == 1 && a.n_dense > 1) tb.dense[1] = a.dense[1];
  if (threadIdx.x == 2 && a.n_dense > 2) tb.dense[2] = a.dense[2];
}

// Resolves the union members into LDS.  Lists built by the union kernel always
// pass; caller-supplied ones are checked so that a bad list can only drop
// work, never read or write out of bounds.  A member with a valid list and no
// valid slot keeps its list (blk NULL) and sets *absent.  All threads; the
// caller synchronises.
__device__ __forceinline__ void fill_tables(const GroupedArgs& a, const Tables& tb, int nu,
                                            int* absent) {
  const RoutedSrc& r = a.r;
  for (int j = threadIdx.x; j < nu; j += kBlock) {
    Member m{nullptr, 0, 0, -1, 0};
    const int e = r.union_ids[j];
    const int slot =
        (e >= 0 && e < r.n_experts) ? (r.slot_of_expert ? r.slot_of_expert[e] : e) : -1;
    const int off = r.offsets[j], end = r.offsets[j + 1];
    if (off >= 0 && end >= off && end <= r.pairs_max) {
      m.off = off;
      m.ntok = end - off;
      if (slot >= 0 && slot < r.n_slots)
        m.blk = r.base + (size_t)slot * r.stride;
      else if (m.ntok > 0)
        *absent = 1;
    }
    tb.mem[j] = m;
  }
  for (int i = threadIdx.x; i < r.pairs_max; i += kBlock) {
    const int t = r.tok_list[i];
    tb.tok[i] = t < 0 ? 0 : (t >= a.T ? a.T - 1 : t);  // a position outside the block never indexes x
    tb.gate[i] = r.gate_list[i];
  }
}

__device__ __forceinline__ int routed_count(const GroupedArgs& a) {
  if (!a.has_routed) return 0;
  const int nu = uni(*a.r.n_union);
  return nu < 0 ? 0 : min(nu, a.r.max_union);
}

// ------------------------------------------------------------------ the pass stream

// One pass: kNS weight rows against up to NT activation rows.
template <int NT>
struct Pass {
  const char* row[kNS];
  const char* srow[kNS];  // Q4_0: the rows' scales
  int L;               // 16-byte units per row
  int nit;             // wave iterations: ceil(L / 64)
  int nt;              // positions
  const float* act;    // activation base; null: LDS
  int vo[NT];          // activation offsets (floats)
  int r0;              // gate/up: first (G, U) pair; down: first row
  int rows;            // rows (pairs) of the source
  float* out;
  int ostride;
  int orow0;           // output row of the pass's first position
  int goff;            // routed down: gate-list index of the first position; -1: gscalar
  float gscalar;
  uint64_t* tout;      // single-launch verify layer: tagged outputs, indexed as out
};

// Tile list of a launch: the dense sources' tiles first (source s from ds[s]),
// then the union members' tiles from ndt (member j: tr tiles).  Named fields:
// an array indexed at run time would live in per-lane scratch memory.
struct Layout {
  int ndt, tr, nr, total, nd;
  int ds1, ds2;
  int act0, act1, act2;  // down: LDS offsets of the dense sources' staged inputs (-1: global)

  __device__ __forceinline__ int source(int t, int& start, int& act) const {
    if (nd > 2 && t >= ds2) {
      start = ds2;
      act = act2;
      return 2;
    }
    if (nd > 1 && t >= ds1) {
      start = ds1;
      act = act1;
      return 1;
    }
    start = 0;
    act = act0;
    return 0;
  }
};

// Tiles of RT weight rows (gate/up: RT / 2 (G, U) pairs).
template <int RT>
__device__ __forceinline__ Layout make_layout(const GroupedArgs& a, int nu, bool gateup) {
  Layout ly;
  const int per = gateup ? RT / 2 : RT;
  const int n0 = a.n_dense > 0 ? uni(cdiv(gateup ? a.dense[0].inter : a.dense[0].rows, per)) : 0;
  const int n1 = a.n_dense > 1 ? uni(cdiv(gateup ? a.dense[1].inter : a.dense[1].rows, per)) : 0;
  const int n2 = a.n_dense > 2 ? uni(cdiv(gateup ? a.dense[2].inter : a.dense[2].rows, per)) : 0;
  ly.nd = a.n_dense;
  ly.ds1 = n0;
  ly.ds2 = n0 + n1;
  ly.ndt = n0 + n1 + n2;
  ly.tr = a.has_routed ? uni(cdiv(gateup ? a.r.inter : a.H, per)) : 0;
  ly.nr = nu * ly.tr;
  ly.total = ly.ndt + ly.nr;
  ly.act0 = ly.act1 = ly.act2 = -1;
  return ly;
}

// A wave's position in its sequence of passes: tile, first position of the
// pass, positions of the tile.
struct Cursor {
  int tile, m0, ntok;
};

// The passes of a wave's tiles in [lo, hi) (tiles b*W + w + k * step).
// FUSED (the single-launch verify layer): outputs also go to the tagged
// buffers, and a dense source's staged input offset comes from tb.dact.
template <typename WT, bool GATEUP, int NT, int RT, bool FUSED = false>
struct Walker {
  Layout ly;      // by value: a reference to a local would live in per-lane scratch
  Tables tb;
  int step;       // grid * waves
  int lo, hi;
  int xstride;    // gate/up: row stride of the staged (or global) x
  bool xlds;      // gate/up: x is staged in LDS

  // Fills p for tile c.tile at position c.m0; c.ntok receives the tile's
  // position count.  False when the tile's member is not resident.
  __device__ __forceinline__ bool make(const GroupedArgs& a, Cursor& c, Pass<NT>& p) const {
    constexpr int EPU = WTr<WT>::EPU;
    const int H = a.H;
    if (c.tile >= ly.ndt) {
      const int j = uni((c.tile - ly.ndt) / ly.tr);
      const int rg = c.tile - ly.ndt - j * ly.tr;
      const Member mb = tb.mem[j];
      const char* blk = uni(mb.blk);
      if (blk == nullptr) return false;
      const int off = uni(mb.off);
      c.ntok = uni(mb.ntok);
      const int I = a.r.inter;
      p.nt = min(NT, c.ntok - c.m0);
      p.orow0 = off + c.m0;
      if constexpr (GATEUP) {
        const size_t rb = qrow_bytes<WT>(H);
        const char* U = blk + mat_bytes<WT>(I, H);
        p.r0 = rg * (RT / 2);
        p.rows = I;
#pragma unroll
        for (int q = 0; q < RT / 2; ++q) {
          const size_t rc = (size_t)min(p.r0 + q, I - 1);
          p.row[2 * q] = blk + rc * rb;
          p.row[2 * q + 1] = U + rc * rb;
          if constexpr (kQ4<WT>) {
            p.srow[2 * q] = blk + (size_t)I * rb + rc * (H / 16);
            p.srow[2 * q + 1] = U + (size_t)I * rb + rc * (H / 16);
          }
        }
        p.L = (int)(rb / 16);
        p.act = xlds ? nullptr : a.x;
#pragma unroll
        for (int m = 0; m < NT; ++m) p.vo[m] = uni(tb.tok[p.orow0 + min(m, p.nt - 1)]) * xstride;
        p.out = a.r.a;
        p.ostride = I;
        p.goff = -1;
        if constexpr (FUSED) p.tout = a.r.a_tag;
      } else {
        const size_t rb = qrow_bytes<WT>(I);
        const char* D = blk + 2 * mat_bytes<WT>(I, H);
        p.r0 = rg * RT;
        p.rows = H;
#pragma unroll
        for (int k = 0; k < RT; ++k) {
          const size_t r = (size_t)min(p.r0 + k, H - 1);
          p.row[k] = D + r * rb;
          if constexpr (kQ4<WT>) p.srow[k] = D + (size_t)H * rb + r * (I / 16);
        }
        p.L = (int)(rb / 16);
        const int act = uni(mb.act);
        if (act >= 0) {
          const int sst = staged_stride<EPU>(I);
          p.act = nullptr;
#pragma unroll
          for (int m = 0; m < NT; ++m) p.vo[m] = act + (c.m0 + min(m, p.nt - 1)) * sst;
        } else {
          p.act = a.r.a;
#pragma unroll
          for (int m = 0; m < NT; ++m) p.vo[m] = (p.orow0 + min(m, p.nt - 1)) * I;
        }
        p.out = a.r.p;
        p.ostride = H;
        p.goff = p.orow0;
        if constexpr (FUSED) p.tout = a.r.p_tag;
      }
      p.gscalar = 0.f;
    } else {
      int start = 0, dact = -1;
      const int s = ly.source(c.tile, start, dact);
      const DenseSrc d = dense_at(tb, s);
      const int rg = c.tile - start;
      c.ntok = a.T;
      p.nt = min(NT, a.T - c.m0);
      p.orow0 = c.m0;
      const char* W = static_cast<const char*>(d.w);
      if constexpr (GATEUP) {
        const size_t rb = qrow_bytes<WT>(H);
        const char* U = W + mat_bytes<WT>(d.inter, H);
        p.r0 = rg * (RT / 2);
        p.rows = d.inter;
#pragma unroll
        for (int q = 0; q < RT / 2; ++q) {
          const size_t rc = (size_t)min(p.r0 + q, d.inter - 1);
          p.row[2 * q] = W + rc * rb;
          p.row[2 * q + 1] = U + rc * rb;
          if constexpr (kQ4<WT>) {
            p.srow[2 * q] = W + (size_t)d.inter * rb + rc * (H / 16);
            p.srow[2 * q + 1] = U + (size_t)d.inter * rb + rc * (H / 16);
          }
        }
        p.L = (int)(rb / 16);
        p.act = xlds ? nullptr : a.x;
#pragma unroll
        for (int m = 0; m < NT; ++m) p.vo[m] = (c.m0 + min(m, p.nt - 1)) * xstride;
        p.out = d.out;
        p.ostride = d.inter;
        if constexpr (FUSED) p.tout = d.out_tag;
      } else {
        const int ldc = d.ld > 0 ? d.ld : d.inter;
        const size_t rb = qrow_bytes<WT>(ldc);
        p.r0 = rg * RT;
        p.rows = d.rows;
#pragma unroll
        for (int k = 0; k < RT; ++k) {
          const size_t r = (size_t)min(p.r0 + k, d.rows - 1);
          p.row[k] = W + r * rb;
          if constexpr (kQ4<WT>) p.srow[k] = static_cast<const char*>(d.ws) + r * (ldc / 16);
        }
        p.L = (int)(qrow_bytes<WT>(d.inter) / 16);
        const int act = FUSED ? uni(tb.dact[s]) : dact;
        if (act >= 0) {
          const int sst = staged_stride<EPU>(d.inter);
          p.act = nullptr;
#pragma unroll
          for (int m = 0; m < NT; ++m) p.vo[m] = act + (c.m0 + min(m, p.nt - 1)) * sst;
        } else {
          p.act = d.vin;
#pragma unroll
          for (int m = 0; m < NT; ++m) p.vo[m] = (c.m0 + min(m, p.nt - 1)) * d.vin_stride;
        }
        p.out = d.out;
        p.ostride = d.out_stride;
        if constexpr (FUSED) p.tout = d.out_tag;
      }
      p.goff = -1;
      p.gscalar = d.gate;
    }
    p.nit = (p.L + kWave - 1) / kWave;
    return true;
  }

  // The first pass at or after tile c.tile; false at the end of the range.
  __device__ __forceinline__ bool seek(const GroupedArgs& a, Cursor& c, Pass<NT>& p) const {
    c.m0 = 0;
    while (c.tile < hi) {
      if (make(a, c, p) && c.ntok > 0) return true;
      c.tile += step;
    }
    return false;
  }

  // The pass after c; false at the end of the range.
  __device__ __forceinline__ bool next(const GroupedArgs& a, Cursor& c, Pass<NT>& p) const {
    c.m0 += NT;
    if (c.m0 < c.ntok) return make(a, c, p);
    c.tile += step;
    return seek(a, c, p);
  }
};

// Loads iteration `it` of pass p (RT rows) into r (Q4_0: the units' scales
// into sc).  Past a row's end the lane re-reads the last unit (always in
// bounds); consume() zeroes it.
template <typename WT, int NT, int RT>
__device__ __forceinline__ void issue(const Pass<NT>& p, int it, u32x4 (&r)[RT],
                                      uint32_t (&sc)[RT], int lane) {
  const uint32_t u = (uint32_t)min(it * kWave + lane, p.L - 1);
#pragma unroll
  for (int k = 0; k < RT; ++k) {
    r[k] = load_w16(p.row[k] + u * 16u);
    if constexpr (kQ4<WT>) sc[k] = *gptr<uint16_t>(p.srow[k] + u * 2u);
  }
}

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return (float)__builtin_bit_cast(_Float16, (unsigned short)h);
}

// Accumulates iteration `it` of pass p.
// HOIST (bf16 / fp32 weights): each weight unit is converted once and met
// by every position, instead of once per position; the same FMAs in the same
// order.  It needs RT x EPU more registers, which the down passes have.
template <typename WT, int NT, int RT, bool HOIST = false>
__device__ __forceinline__ void consume(const Pass<NT>& p, int it, const u32x4 (&r)[RT],
                                        const uint32_t (&sc)[RT], int lane,
                                        float (&acc)[RT][NT]) {
  constexpr int EPU = WTr<WT>::EPU;
  const int u = it * kWave + lane;
  const bool ok = u < p.L;
  const int uc = ok ? u : p.L - 1;
  if constexpr (kQ4<WT> || !HOIST) {
#pragma unroll
    for (int m = 0; m < NT; ++m) {
      if (m < p.nt) {
        if constexpr (kQ4<WT>) {
            // sum_e d (q_e - 8) x_e = d (sum_e q_e x_e - 8 sum_e x_e), in two
            // halves: weights 0..15 of the unit are the low nibbles of its 16
            // bytes, weights 16..31 the high nibbles.
            float qx[RT], xs = 0.f;
    #pragma unroll
            for (int k = 0; k < RT; ++k) qx[k] = 0.f;
    #pragma unroll
            for (int h = 0; h < 2; ++h) {
              float xv[16];
              act_half_q4(p.act, p.vo[m], uc, h, xv);
    #pragma unroll
              for (int v = 0; v < 16; ++v) xs += xv[v];
    #pragma unroll
              for (int k = 0; k < RT; ++k) {
                const uint32_t wd[4] = {r[k].x, r[k].y, r[k].z, r[k].w};
                uint32_t nib[4];
    #pragma unroll
                for (int w = 0; w < 4; ++w) nib[w] = (h ? wd[w] >> 4 : wd[w]) & 0x0F0F0F0Fu;
                // Opaque to the compiler: the codes are converted again for every
                // position (4 x 32 converted floats would not fit in registers),
                // and each byte is converted by one byte-select conversion
                // instead of a bit-field extract and a conversion.
                asm volatile("" : "+v"(nib[0]), "+v"(nib[1]), "+v"(nib[2]), "+v"(nib[3]));
    #pragma unroll
                for (int w = 0; w < 4; ++w) {
    #pragma unroll
                  for (int b = 0; b < 4; ++b)
                    qx[k] = fmaf((float)((nib[w] >> (8 * b)) & 0xFFu), xv[4 * w + b], qx[k]);
                }
              }
            }
    #pragma unroll
            for (int k = 0; k < RT; ++k) {
              // A lane past the row's end re-read the last unit: scale 0.
              const float d = ok ? half_bits_to_float(sc[k]) : 0.f;
              acc[k][m] = fmaf(d, fmaf(-8.f, xs, qx[k]), acc[k][m]);
            }
        } else {
          float xv[EPU];
          act_frag<EPU>(p.act, p.vo[m], uc, xv);
#pragma unroll
          for (int k = 0; k < RT; ++k) {
            const u32x4 rr = ok ? r[k] : u32x4{0u, 0u, 0u, 0u};
            float w[EPU];
            unpack(rr, w);
#pragma unroll
            for (int v = 0; v < EPU; ++v) acc[k][m] = fmaf(w[v], xv[v], acc[k][m]);
          }
        }
      }
      // Keeps the next position's activation loads from being hoisted above
      // this one's arithmetic.
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
    // Each weight unit is converted once and met by every position (the
    // conversion is as much arithmetic as the unit's FMAs).
    float w[RT][EPU];
#pragma unroll
    for (int k = 0; k < RT; ++k) unpack(ok ? r[k] : u32x4{0u, 0u, 0u, 0u}, w[k]);
#pragma unroll
    for (int m = 0; m < NT; ++m) {
      if (m < p.nt) {
        float xv[EPU];
        act_frag<EPU>(p.act, p.vo[m], uc, xv);
#pragma unroll
        for (int k = 0; k < RT; ++k)
#pragma unroll
          for (int v = 0; v < EPU; ++v) acc[k][m] = fmaf(w[k][v], xv[v], acc[k][m]);
      }
      // Keeps the next position's activation loads from being hoisted above
      // this one's arithmetic.
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// Stores v with this launch's epoch as one 64-bit value (agent scope: written
// through to memory, so a block on another XCD that reads it with an
// agent-scope load sees the value and its epoch together).
__device__ __forceinline__ void st_tag(uint64_t* p, float v, uint32_t epoch) {
  __hip_atomic_store(p, ((uint64_t)epoch << 32) | (uint64_t)__float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

// One output value of a pass: to out (plain) and, with TAGGED, to the tagged
// buffer (either may be null in that mode).
template <bool TAGGED, int NT>
__device__ __forceinline__ void put(const Pass<NT>& p, size_t o, float v, uint32_t epoch) {
  if constexpr (TAGGED) {
    if (p.tout != nullptr) st_tag(p.tout + o, v, epoch);
    if (p.out != nullptr) *(DE_GLOBAL float*)(p.out + o) = v;
  } else {
    // A global (not flat) store: a flat store also counts against the LDS wait
    // counter and would hold up the activation reads behind it.
    *(DE_GLOBAL float*)(p.out + o) = v;
  }
}

// Reduces the pass's sums and writes them; clears acc.
template <bool GATEUP, int NT, int RT, bool TAGGED = false>
__device__ __forceinline__ void finish(const Pass<NT>& p, const Tables& tb, int lane,
                                       float (&acc)[RT][NT], uint32_t epoch = 0) {
#pragma unroll
  for (int m = 0; m < NT; ++m) {
    if (m < p.nt) {
      if constexpr (GATEUP) {
#pragma unroll
        for (int q = 0; q < RT / 2; ++q) {
          const float g = row_total(acc[2 * q][m]);
          const float u = row_total(acc[2 * q + 1][m]);
          if (lane == m && p.r0 + q < p.rows)
            put<TAGGED>(p, (size_t)(p.orow0 + m) * p.ostride + p.r0 + q, silu_f(g) * u, epoch);
        }
      } else {
        const float gm = p.goff >= 0 ? tb.gate[p.goff + m] : p.gscalar;
#pragma unroll
        for (int k = 0; k < RT; ++k) {
          const float v = row_total(acc[k][m]);
          if (lane == m && p.r0 + k < p.rows)
            put<TAGGED>(p, (size_t)(p.orow0 + m) * p.ostride + p.r0 + k, gm * v, epoch);
        }
      }
    }
  }
#pragma unroll
  for (int k = 0; k < RT; ++k)
#pragma unroll
    for (int m = 0; m < NT; ++m) acc[k][m] = 0.f;
}

// Called by the consumer before the first pass of each of its tiles (the
// pass is already made and may be remade).  The separate launches need
// nothing there.
struct NoHook {
  template <class WK, class P>
  __device__ __forceinline__ void enter(const GroupedArgs&, const WK&, Cursor&, P&) {}
};

// Streams the wave's pass sequence: the loader runs RING iterations ahead of
// the consumer, across pass and tile boundaries.
template <typename WT, bool GATEUP, int NT, int RING, int RT, bool FUSED, class Hook>
__device__ __forceinline__ void run_stream(const GroupedArgs& a,
                                           const Walker<WT, GATEUP, NT, RT, FUSED> wk,
                                           int first_tile, int lane, Hook& hk) {
  Cursor lc{first_tile, 0, 0}, cc{first_tile, 0, 0};
  Pass<NT> lp, cp;
  bool l_ok = wk.seek(a, lc, lp);
  bool c_ok = wk.seek(a, cc, cp);
  int l_it = 0, c_it = 0;
  u32x4 raw[RING][RT];
  uint32_t sraw[RING][RT];
#pragma unroll
  for (int q = 0; q < RING; ++q) {
    if (l_ok) {
      issue<WT>(lp, l_it, raw[q], sraw[q], lane);
      if (++l_it == lp.nit) {
        l_ok = wk.next(a, lc, lp);
        l_it = 0;
      }
    }
  }
  float acc[RT][NT];
#pragma unroll
  for (int k = 0; k < RT; ++k)
#pragma unroll
    for (int m = 0; m < NT; ++m) acc[k][m] = 0.f;
  if (c_ok) hk.enter(a, wk, cc, cp);
  while (c_ok) {
#pragma unroll
    for (int q = 0; q < RING; ++q) {
      if (c_ok) {
        consume<WT, NT, RT, !GATEUP>(cp, c_it, raw[q], sraw[q], lane, acc);
        if (++c_it == cp.nit) {
          finish<GATEUP, NT, RT, FUSED>(cp, wk.tb, lane, acc, a.epoch);
          const int prev_tile = cc.tile;
          c_ok = wk.next(a, cc, cp);
          c_it = 0;
          if (c_ok && cc.tile != prev_tile) hk.enter(a, wk, cc, cp);
          // Dense sources over many positions are arithmetic-heavy: a wave
          // with more tiles left gets a higher issue priority, so the waves
          // of a CU finish together instead of the oldest first.
          if (NT == kDenseNTOf<WT> && a.T >= 8 && c_ok && cc.tile != prev_tile) {
            const int rem = (wk.hi - 1 - cc.tile) / wk.step;
            if (rem >= 3)
              __builtin_amdgcn_s_setprio(3);
            else if (rem == 2)
              __builtin_amdgcn_s_setprio(2);
            else if (rem == 1)
              __builtin_amdgcn_s_setprio(1);
            else
              __builtin_amdgcn_s_setprio(0);
          }
        }
        if (l_ok) {
          issue<WT>(lp, l_it, raw[q], sraw[q], lane);
          if (++l_it == lp.nit) {
            l_ok = wk.next(a, lc, lp);
            l_it = 0;
          }
        }
      }
    }
  }
}

// A wave's tiles: first, first + step, ...  The dense tiles [0, ndt) run with
// passes of kDenseNT positions, the members' tiles with kRoutedNT.  WPB waves
// per block; FUSED and the hook as in Walker and run_stream.
template <typename WT, bool GATEUP, int RT, int WPB, bool FUSED, class Hook>
__device__ __forceinline__ void run_tiles(const GroupedArgs& a, const Layout ly, const Tables& tb,
                                          int xstride, bool xlds, int lane, int wave, Hook& hk) {
  const int step = (int)gridDim.x * WPB;
  const int first = (int)blockIdx.x * WPB + wave;
  if (first < ly.ndt) {
    constexpr int DNT = kDenseNTOf<WT>;
    const Walker<WT, GATEUP, DNT, RT, FUSED> wd{ly, tb, step, 0, ly.ndt, xstride, xlds};
    run_stream<WT, GATEUP, DNT, kDenseRing, RT>(a, wd, first, lane, hk);
  }
  __builtin_amdgcn_s_setprio(0);
  if (ly.nr > 0) {
    const int f2 = first >= ly.ndt ? first : first + cdiv(ly.ndt - first, step) * step;
    constexpr int RNT = kRoutedNTOf<WT>;
    const Walker<WT, GATEUP, RNT, RT, FUSED> wr{ly, tb, step, ly.ndt, ly.total, xstride, xlds};
    run_stream<WT, GATEUP, RNT, kRingOf<WT>, RT>(a, wr, f2, lane, hk);
  }
}

template <typename WT, bool GATEUP, int RT>
__device__ __forceinline__ void run_tiles(const GroupedArgs& a, const Layout ly, const Tables& tb,
                                          int xstride, bool xlds, int lane, int wave) {
  NoHook h;
  run_tiles<WT, GATEUP, RT, kWavesPB, false>(a, ly, tb, xstride, xlds, lane, wave, h);
}

}  // namespace
}  // namespace de
