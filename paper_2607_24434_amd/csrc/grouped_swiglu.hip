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

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / kWave;
constexpr int kGroups = kWave / 16;
constexpr int kGuRG = 1;                  // (G row, U row) pairs per 16-lane group
constexpr int kGuTile = kGroups * kGuRG;  // row pairs per gate/up tile
constexpr int kDnRG = 2;                  // rows per group (down and row-dot)
constexpr int kDnTile = kGroups * kDnRG;  // rows per down tile
constexpr int kMaxNT = 16;                // positions per pass

// 16-byte iterations whose loads are issued together, by positions per pass:
// fewer positions leave registers for more loads in flight.
template <int NT>
struct InFlight {
  static constexpr int MI = NT <= 4 ? 4 : (NT <= 8 ? 2 : 1);
};

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

template <int EPU>
__device__ __forceinline__ void load_vec(const float* p, float (&v)[EPU]) {
  const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
  for (int i = 0; i < EPU / 4; ++i) {
    const float4 t = q[i];
    v[4 * i + 0] = t.x;
    v[4 * i + 1] = t.y;
    v[4 * i + 2] = t.z;
    v[4 * i + 3] = t.w;
  }
}

// Dot products of NS weight rows with up to NT input vectors over the
// 16-byte units this lane owns: unit u = it*16 + lg for iterations it =
// wave, wave+4, ...  (L = units per row).  Input vector m starts at
// vbase + voff[m] (32-bit float offsets keep the address math in one VGPR).
template <typename WT, int NS, int NT>
__device__ __forceinline__ void slice_dot(const char* const (&rowp)[NS], int L, int wave, int lg,
                                          const float* vbase, const int (&voff)[NT], int nt,
                                          float (&acc)[NS][NT]) {
  constexpr int EPU = WTr<WT>::EPU;
  constexpr int MI = InFlight<NT>::MI;
  const int nit = (L + 15) >> 4;
  for (int it0 = wave; it0 < nit; it0 += kWaves * MI) {
    u32x4 raw[MI][NS];
#pragma unroll
    for (int q = 0; q < MI; ++q) {
      const int it = it0 + q * kWaves;
      const int u = it * 16 + lg;
      const bool ok = it < nit && u < L;
#pragma unroll
      for (int s = 0; s < NS; ++s)
        raw[q][s] = ok ? load_stream16(rowp[s] + (size_t)u * 16) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int q = 0; q < MI; ++q) {
      const int it = it0 + q * kWaves;
      if (it >= nit) break;
      const int u = it * 16 + lg;
      const bool ok = u < L;
      float w[NS][EPU];
#pragma unroll
      for (int s = 0; s < NS; ++s) unpack(raw[q][s], w[s]);
#pragma unroll
      for (int m = 0; m < NT; ++m) {
        if (m < nt) {
          float xv[EPU];
          if (ok) {
            load_vec<EPU>(vbase + voff[m] + u * EPU, xv);
          } else {
#pragma unroll
            for (int v = 0; v < EPU; ++v) xv[v] = 0.f;
          }
#pragma unroll
          for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int v = 0; v < EPU; ++v) acc[s][m] = fmaf(w[s][v], xv[v], acc[s][m]);
        }
      }
    }
  }
}

// ------------------------------------------------------------------ gate/up

// One tile of kGuTile (G row, U row) pairs of one source for up to NT
// positions: A[arow0 + m][r] = silu(G_r . x_m) * (U_r . x_m).
template <typename WT, int NT>
__device__ void gateup_tile(const char* G, const char* U, int inter, int H, int T, int row_base,
                            const float* x, const int32_t* tok, int tok_base, int nt, float* A,
                            int arow0, float* lds) {
  constexpr int NS = 2 * kGuRG;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane >> 4, lg = lane & 15;
  const size_t rb = (size_t)H * sizeof(WT);
  const char* rowp[NS];
#pragma unroll
  for (int k = 0; k < kGuRG; ++k) {
    const int r = min(row_base + grp * kGuRG + k, inter - 1);
    rowp[2 * k] = G + (size_t)r * rb;
    rowp[2 * k + 1] = U + (size_t)r * rb;
  }
  int voff[NT];
#pragma unroll
  for (int m = 0; m < NT; ++m) {
    int t = m < nt ? (tok ? tok[m] : tok_base + m) : (tok ? tok[0] : tok_base);
    t = t < 0 ? 0 : (t >= T ? T - 1 : t);  // a position outside the block never indexes x
    voff[m] = t * H;
  }
  float acc[NS][NT];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int m = 0; m < NT; ++m) acc[s][m] = 0.f;
  slice_dot<WT, NS, NT>(rowp, (int)(rb / 16), wave, lg, x, voff, nt, acc);
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int m = 0; m < NT; ++m) {
      if (m < nt) {
        const float v = row16_sum(acc[s][m]);
        if (lg == m) lds[((wave * kGroups + grp) * NS + s) * kMaxNT + m] = v;
      }
    }
  __syncthreads();
  if (wave == 0 && lg < nt) {
#pragma unroll
    for (int k = 0; k < kGuRG; ++k) {
      const int r = row_base + grp * kGuRG + k;
      if (r < inter) {
        float g = 0.f, u = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
          g += lds[((w * kGroups + grp) * NS + 2 * k) * kMaxNT + lg];
          u += lds[((w * kGroups + grp) * NS + 2 * k + 1) * kMaxNT + lg];
        }
        A[(size_t)(arow0 + lg) * inter + r] = silu_f(g) * u;
      }
    }
  }
  __syncthreads();
}

template <typename WT>
__device__ void gateup_dispatch(const char* G, const char* U, int inter, int H, int T, int row_base,
                                const float* x, const int32_t* tok, int tok_base, int ntok,
                                float* A, int arow0, float* lds) {
  for (int m0 = 0; m0 < ntok; m0 += kMaxNT) {
    const int nt = min(kMaxNT, ntok - m0);
    const int32_t* tk = tok ? tok + m0 : nullptr;
    if (nt <= 1)
      gateup_tile<WT, 1>(G, U, inter, H, T, row_base, x, tk, tok_base + m0, nt, A, arow0 + m0, lds);
    else if (nt <= 2)
      gateup_tile<WT, 2>(G, U, inter, H, T, row_base, x, tk, tok_base + m0, nt, A, arow0 + m0, lds);
    else if (nt <= 4)
      gateup_tile<WT, 4>(G, U, inter, H, T, row_base, x, tk, tok_base + m0, nt, A, arow0 + m0, lds);
    else if (nt <= 8)
      gateup_tile<WT, 8>(G, U, inter, H, T, row_base, x, tk, tok_base + m0, nt, A, arow0 + m0, lds);
    else
      gateup_tile<WT, 16>(G, U, inter, H, T, row_base, x, tk, tok_base + m0, nt, A, arow0 + m0, lds);
  }
}

__device__ __forceinline__ int cdiv(int a, int b) { return (a + b - 1) / b; }

__device__ __forceinline__ int routed_count(const GroupedArgs& a) {
  if (!a.has_routed) return 0;
  const int nu = *a.r.n_union;
  return nu < 0 ? 0 : min(nu, a.r.max_union);
}

// Resolves union member j to its weight block and token-list span; nullptr
// when the expert is not resident or the lists are malformed (lists built by
// the union kernel always pass; caller-supplied ones are checked so that a
// bad list can only drop work, never read or write out of bounds).
__device__ __forceinline__ const char* member_block(const RoutedSrc& r, int j, int& off,
                                                    int& ntok) {
  const int e = r.union_ids[j];
  if (e < 0 || e >= r.max_union) return nullptr;
  const int slot = r.slot_of_expert ? r.slot_of_expert[e] : e;
  if (slot < 0 || slot >= r.n_slots) return nullptr;
  off = r.offsets[j];
  const int end = r.offsets[j + 1];
  if (off < 0 || end < off || end > r.pairs_max) return nullptr;
  ntok = end - off;
  return r.base + (size_t)slot * r.stride;
}

template <typename WT>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void gateup_kernel(GroupedArgs a) {
  __shared__ float lds[kWaves * kGroups * 2 * kGuRG * kMaxNT];
  const int nu = routed_count(a);
  const int tr = a.has_routed ? cdiv(a.r.inter, kGuTile) : 0;
  const int nr = nu * tr;
  int total = nr;
  int dstart[3];
  for (int s = 0; s < a.n_dense; ++s) {
    dstart[s] = total;
    total += cdiv(a.dense[s].inter, kGuTile);
  }
  const size_t esz = sizeof(WT);
  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    if (tile < nr) {
      const int j = tile / tr, rt = tile - j * tr;
      int off = 0, ntok = 0;
      const char* blk = member_block(a.r, j, off, ntok);
      if (blk == nullptr) continue;
      const char* G = blk;
      const char* U = blk + (size_t)a.r.inter * a.H * esz;
      gateup_dispatch<WT>(G, U, a.r.inter, a.H, a.T, rt * kGuTile, a.x, a.r.tok_list + off, 0, ntok,
                          a.r.a, off, lds);
    } else {
      int s = 0;
      while (s + 1 < a.n_dense && tile >= dstart[s + 1]) ++s;
      const DenseSrc& d = a.dense[s];
      const int rt = tile - dstart[s];
      const char* G = static_cast<const char*>(d.w);
      const char* U = G + (size_t)d.inter * a.H * esz;
      gateup_dispatch<WT>(G, U, d.inter, a.H, a.T, rt * kGuTile, a.x, nullptr, 0, a.T, d.out, 0, lds);
    }
  }
}

// ------------------------------------------------------------------ down / row-dot

// One tile of kDnTile rows of a [rows, len] matrix for up to NT input
// vectors: out[orow0 + m][r] = gate_m * (M_r . v_m).
template <typename WT, int NT>
__device__ void down_tile(const char* M, int rows, int len, int row_base, const float* vin,
                          int vstride, int vrow0, int nt, const float* gates, float gscalar,
                          float* out, int ostride, int orow0, float* lds) {
  constexpr int NS = kDnRG;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane >> 4, lg = lane & 15;
  const size_t rb = (size_t)len * sizeof(WT);
  const char* rowp[NS];
#pragma unroll
  for (int k = 0; k < NS; ++k) {
    const int r = min(row_base + grp * NS + k, rows - 1);
    rowp[k] = M + (size_t)r * rb;
  }
  int voff[NT];
#pragma unroll
  for (int m = 0; m < NT; ++m) voff[m] = (vrow0 + (m < nt ? m : 0)) * vstride;
  float acc[NS][NT];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int m = 0; m < NT; ++m) acc[s][m] = 0.f;
  slice_dot<WT, NS, NT>(rowp, (int)(rb / 16), wave, lg, vin, voff, nt, acc);
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int m = 0; m < NT; ++m) {
      if (m < nt) {
        const float v = row16_sum(acc[s][m]);
        if (lg == m) lds[((wave * kGroups + grp) * NS + s) * kMaxNT + m] = v;
      }
    }
  __syncthreads();
  if (wave == 0 && lg < nt) {
    const float g = gates ? gates[lg] : gscalar;
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const int r = row_base + grp * NS + k;
      if (r < rows) {
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) v += lds[((w * kGroups + grp) * NS + k) * kMaxNT + lg];
        out[(size_t)(orow0 + lg) * ostride + r] = g * v;
      }
    }
  }
  __syncthreads();
}

template <typename WT>
__device__ void down_dispatch(const char* M, int rows, int len, int row_base, const float* vin,
                              int vstride, int vrow0, int ntok, const float* gates, float gscalar,
                              float* out, int ostride, int orow0, float* lds) {
  for (int m0 = 0; m0 < ntok; m0 += kMaxNT) {
    const int nt = min(kMaxNT, ntok - m0);
    const float* gg = gates ? gates + m0 : nullptr;
#define DE_DOWN(NTV)                                                                            \
  down_tile<WT, NTV>(M, rows, len, row_base, vin, vstride, vrow0 + m0, nt, gg, gscalar, out, \
                     ostride, orow0 + m0, lds)
    if (nt <= 1)
      DE_DOWN(1);
    else if (nt <= 2)
      DE_DOWN(2);
    else if (nt <= 4)
      DE_DOWN(4);
    else if (nt <= 8)
      DE_DOWN(8);
    else
      DE_DOWN(16);
#undef DE_DOWN
  }
}

template <typename WT>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) void down_kernel(GroupedArgs a) {
  __shared__ float lds[kWaves * kGroups * kDnRG * kMaxNT];
  const int nu = routed_count(a);
  const int tr = a.has_routed ? cdiv(a.H, kDnTile) : 0;
  const int nr = nu * tr;
  int total = nr;
  int dstart[3];
  for (int s = 0; s < a.n_dense; ++s) {
    dstart[s] = total;
    total += cdiv(a.dense[s].rows, kDnTile);
  }
  const size_t esz = sizeof(WT);
  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    if (tile < nr) {
      const int j = tile / tr, rt = tile - j * tr;
      int off = 0, ntok = 0;
      const char* blk = member_block(a.r, j, off, ntok);
      if (blk == nullptr) continue;
      const char* D = blk + 2 * (size_t)a.r.inter * a.H * esz;
      down_dispatch<WT>(D, a.H, a.r.inter, rt * kDnTile, a.r.a, a.r.inter, off, ntok,
                        a.r.gate_list + off, 0.f, a.r.p, a.H, off, lds);
    } else {
      int s = 0;
      while (s + 1 < a.n_dense && tile >= dstart[s + 1]) ++s;
      const DenseSrc& d = a.dense[s];
      const int rt = tile - dstart[s];
      down_dispatch<WT>(static_cast<const char*>(d.w), d.rows, d.inter, rt * kDnTile, d.vin,
                        d.vin_stride, 0, a.T, nullptr, d.gate, d.out, d.out_stride, 0, lds);
    }
  }
}

// ------------------------------------------------------------------ combine

__device__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float t = 0.f;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) t += red[w];
  __syncthreads();
  return t;
}

// y[t] = sum of the dense partials + sum_j P_r[pair_pos[t, j]] (+ residual),
// in that fixed order; optionally also RMSNorm(y).
__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
  __shared__ float red[4];
  const int t = blockIdx.x;
  const size_t rowoff = (size_t)t * a.H;
  float ss = 0.f;
  for (int h = threadIdx.x; h < a.H; h += blockDim.x) {
    float v = 0.f;
    for (int s = 0; s < a.n_dense; ++s) v += a.dense_p[s][rowoff + h];
    if (a.p_r) {
      for (int j = 0; j < a.kk; ++j) {
        const int p = a.pair_pos[(size_t)t * a.kk + j];
        if (p >= 0 && p < a.pairs_max) v += a.p_r[(size_t)p * a.H + h];
      }
    }
    if (a.residual) v = a.residual[rowoff + h] + v;
    a.y[rowoff + h] = v;
    ss = fmaf(v, v, ss);
  }
  if (a.normed) {
    ss = block_sum(ss, red);
    const float r = 1.0f / sqrtf(ss / (float)a.H + a.eps);
    for (int h = threadIdx.x; h < a.H; h += blockDim.x) a.normed[rowoff + h] = a.y[rowoff + h] * r;
  }
}

template <typename K>
int occupancy_blocks(K kernel) {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, kBlock, 0) != hipSuccess || n < 1)
    n = 1;
  return n;
}

int grid_for(int max_tiles, int occ) {
  const int cap = dev_info().num_cus * occ;
  int g = max_tiles < cap ? max_tiles : cap;
  return g < 1 ? 1 : g;
}

int gateup_max_tiles(const GroupedArgs& a) {
  int t = a.has_routed ? a.r.max_union * ((a.r.inter + kGuTile - 1) / kGuTile) : 0;
  for (int s = 0; s < a.n_dense; ++s) t += (a.dense[s].inter + kGuTile - 1) / kGuTile;
  return t;
}

int down_max_tiles(const GroupedArgs& a) {
  int t = a.has_routed ? a.r.max_union * ((a.H + kDnTile - 1) / kDnTile) : 0;
  for (int s = 0; s < a.n_dense; ++s) t += (a.dense[s].rows + kDnTile - 1) / kDnTile;
  return t;
}

}  // namespace

hipError_t launch_gateup(const GroupedArgs& a, int wdtype, hipStream_t s) {
  const int tiles = gateup_max_tiles(a);
  if (tiles == 0) return hipSuccess;
  if (wdtype == 1) {
    static int occ = occupancy_blocks(gateup_kernel<uint16_t>);
    hipLaunchKernelGGL(gateup_kernel<uint16_t>, dim3(grid_for(tiles, occ)), dim3(kBlock), 0, s, a);
  } else {
    static int occ = occupancy_blocks(gateup_kernel<float>);
    hipLaunchKernelGGL(gateup_kernel<float>, dim3(grid_for(tiles, occ)), dim3(kBlock), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_down(const GroupedArgs& a, int wdtype, hipStream_t s) {
  const int tiles = down_max_tiles(a);
  if (tiles == 0) return hipSuccess;
  if (wdtype == 1) {
    static int occ = occupancy_blocks(down_kernel<uint16_t>);
    hipLaunchKernelGGL(down_kernel<uint16_t>, dim3(grid_for(tiles, occ)), dim3(kBlock), 0, s, a);
  } else {
    static int occ = occupancy_blocks(down_kernel<float>);
    hipLaunchKernelGGL(down_kernel<float>, dim3(grid_for(tiles, occ)), dim3(kBlock), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(combine_kernel, dim3(a.T), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace de
