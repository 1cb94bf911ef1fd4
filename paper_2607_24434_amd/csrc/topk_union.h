// Top-k selection with gates (Eq. 1, Eq. 4) and the block union with
// per-expert position lists (Eq. 2, Eq. 3), as device functions over LDS
// arrays.  The routing launch selects; the union kernel and the prologue of
// the grouped gate/up kernel (in every block, from the selected lists) build
// the union.
//
// Selection: one wave per position, k rounds of a wave-wide argmax (largest
// key, ties to the lower id).  Gates are normalised in list order.
//
// Union: integer work only.  Every (position, slot) entry sets its position
// bit in the expert's 64-bit mask with an LDS atomic OR (a bit already set
// means the id repeats within a position); a wave scan over the experts in
// ascending id gives each member's list offset and union index; the rank of
// a position in its expert's list is the popcount of the mask below it.
#pragma once

#include "de_common.h"

#include <climits>

namespace de {

// LDS arrays of the selection and union (sizes: T*k, T*k, T*k, N, N, N, 4).
struct SelView {
  int32_t* idx;              // ordered top-k ids [T, k]
  float* sc;                 // their scores
  float* gate;               // their gates
  unsigned long long* mask;  // position mask per expert [N]
  int32_t* off;              // list offset per expert
  int32_t* upos;             // union index per expert
  int32_t* misc;             // [0] bad, [1] n_union, [2] pairs
};

__host__ __device__ inline size_t sel_view_bytes(int T, int k, int N) {
  const size_t tk = (size_t)T * k;
  return ((tk * 12 + 7) & ~(size_t)7) + (size_t)N * 16 + 16;
}

__device__ inline SelView sel_view_at(char* p, int T, int k, int N) {
  SelView v;
  const size_t tk = (size_t)T * k;
  v.idx = reinterpret_cast<int32_t*>(p);
  v.sc = reinterpret_cast<float*>(v.idx + tk);
  v.gate = v.sc + tk;
  p += (tk * 12 + 7) & ~(size_t)7;
  v.mask = reinterpret_cast<unsigned long long*>(p);
  v.off = reinterpret_cast<int32_t*>(v.mask + N);
  v.upos = v.off + N;
  v.misc = v.upos + N;
  return v;
}

// Loads a position's N logits into the lane layout of the selection: lane l
// holds candidates l, l + 64, ... (N <= 256; zrow in LDS or global memory).
__device__ __forceinline__ void topk_load(const TopkUnionArgs& a, const float* zrow,
                                          float (&z)[4]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = lane + q * kWave;
    z[q] = e < a.N ? zrow[e] : 0.f;
  }
}

// Ordered top-k of R positions at once from their logits in registers (R
// independent chains interleaved, so their reduction latencies overlap):
// ids into idx0 / idx1 [0..k), scores into sc0 / sc1 [0..k).  Each of the k rounds
// takes the largest remaining key, ties to the lower id: every lane offers
// its best remaining candidate, a wave max finds the key, a wave min the
// lowest id offering it, and the owning lane records and retires it.  A NaN
// key counts as -inf; a candidate id >= N never competes.  With a.rounds
// set, only that many leading entries are selected.  One wave.
template <int R>
__device__ __forceinline__ void topk_regs(const TopkUnionArgs& a, const float (&z)[R][4],
                                          int32_t* idx0, float* sc0, int32_t* idx1 = nullptr,
                                          float* sc1 = nullptr) {
  const int lane = threadIdx.x & 63;
  const int N = a.N, k = a.k;
  float key[R][4], sc[R][4];
  bool left[R][4];
#pragma unroll
  for (int r = 0; r < R; ++r) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane + q * kWave;
      left[r][q] = e < N;
      const float b = (left[r][q] && a.bias != nullptr) ? a.bias[e] : 0.f;
      float kk, sv;
      if (a.score_func == 0) {  // softmax(z + b): key z + b
        kk = z[r][q] + b;
        sv = 0.f;
      } else {                  // sigmoid(z): key sigmoid(z) + b
        sv = 1.0f / (1.0f + expf(-z[r][q]));
        kk = sv + b;
      }
      if (!(kk == kk)) kk = -INFINITY;  // a NaN never wins
      key[r][q] = left[r][q] ? kk : -INFINITY;
      sc[r][q] = sv;
    }
  }
  if (a.score_func == 0) {
    float m[R], sum[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      m[r] = -INFINITY;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (left[r][q]) m[r] = fmaxf(m[r], key[r][q]);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) m[r] = wave_max(m[r]);
    float ex[R][4];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      sum[r] = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        ex[r][q] = left[r][q] ? expf(key[r][q] - m[r]) : 0.f;
        sum[r] += ex[r][q];
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) sum[r] = wave_sum(sum[r]);
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int q = 0; q < 4; ++q) sc[r][q] = ex[r][q] / sum[r];
  }
  const int kr = a.rounds > 0 ? min(a.rounds, k) : k;
  for (int j = 0; j < kr; ++j) {
    float bk[R];
    int bid[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      bk[r] = -INFINITY;
      bid[r] = INT_MAX;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = lane + q * kWave;
        if (left[r][q] && (key[r][q] > bk[r] || (key[r][q] == bk[r] && e < bid[r]))) {
          bk[r] = key[r][q];
          bid[r] = e;
        }
      }
    }
    float m[R];
#pragma unroll
    for (int r = 0; r < R; ++r) m[r] = wave_max(bk[r]);
    int win[R];
#pragma unroll
    for (int r = 0; r < R; ++r) win[r] = wave_min_i32(bk[r] == m[r] ? bid[r] : INT_MAX);
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (bid[r] == win[r]) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (q == (win[r] >> 6)) {
            left[r][q] = false;
            (r == 0 ? idx0 : idx1)[j] = win[r];
            (r == 0 ? sc0 : sc1)[j] = sc[r][q];
          }
        }
      }
    }
  }
}

// Ordered top-k of one position from its N logits zrow (one wave).
__device__ inline void topk_row(const TopkUnionArgs& a, const float* zrow, int32_t* idx,
                                float* sc_out) {
  float z[1][4];
  topk_load(a, zrow, z[0]);
  topk_regs<1>(a, z, idx, sc_out);
}

// Gate of list entry j of a position from the list's scores: score_j
// (/ sum of the k scores in list order) * routed_scale.
__device__ inline float topk_gate(const TopkUnionArgs& a, const float* sc, int j) {
  float g = sc[j];
  if (a.norm_topk) {
    float gsum = 0.f;
    for (int i = 0; i < a.k; ++i) gsum += sc[i];
    g = g / gsum;
  }
  return g * a.routed_scale;
}

// Union of the first a.ucols entries of every position's list in s.idx /
// s.gate.  s.misc[1] receives n_union (-1 for an id outside [0, N) or an id
// that repeats within a position) and s.misc[2] the number of pairs.  With
// write_out the lists go to a.n_union / union_ids / offsets / tok_list /
// gate_list / pair_pos; with ptok / pgate the per-pair positions and gates
// also go to LDS.  All threads of the block; ends with a barrier.
__device__ inline void build_union(const TopkUnionArgs& a, const SelView& s, bool write_out,
                                   int32_t* ptok, float* pgate) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nthreads = blockDim.x;
  const int T = a.T, N = a.N, k = a.k, uc = a.ucols;
  for (int e = tid; e < N; e += nthreads) s.mask[e] = 0ull;
  if (tid == 0) s.misc[0] = 0;
  __syncthreads();
  for (int i = tid; i < T * uc; i += nthreads) {
    const int t = i / uc, j = i - t * uc;
    const int e = s.idx[t * k + j];
    if (e < 0 || e >= N) {
      s.misc[0] = 1;
    } else {
      const unsigned long long bit = 1ull << t;
      const unsigned long long old = atomicOr(&s.mask[e], bit);
      if (old & bit) s.misc[0] = 1;
    }
  }
  __syncthreads();
  if (s.misc[0]) {
    if (tid == 0) {
      s.misc[1] = -1;
      s.misc[2] = 0;
      if (write_out) *a.n_union = -1;
    }
    __syncthreads();
    return;
  }
  // Exclusive scans over the experts in ascending id (wave 0, four per lane).
  if (wave == 0) {
    int cnt[4], flg[4], csum = 0, fsum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane * 4 + q;
      const unsigned long long m = e < N ? s.mask[e] : 0ull;
      cnt[q] = __popcll(m);
      flg[q] = m != 0ull;
      csum += cnt[q];
      fsum += flg[q];
    }
    int ci = csum, fi = fsum;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int cu = __shfl_up(ci, o, kWave);
      const int fu = __shfl_up(fi, o, kWave);
      if (lane >= o) {
        ci += cu;
        fi += fu;
      }
    }
    int cbase = ci - csum, fbase = fi - fsum;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = lane * 4 + q;
      if (e < N) {
        s.off[e] = cbase;
        s.upos[e] = fbase;
      }
      cbase += cnt[q];
      fbase += flg[q];
    }
    if (lane == kWave - 1) {
      s.misc[1] = fi;
      s.misc[2] = ci;
    }
  }
  __syncthreads();
  const int nu = s.misc[1], total = s.misc[2];
  if (write_out) {
    for (int e = tid; e < N; e += nthreads) {
      if (s.mask[e] != 0ull) {
        a.union_ids[s.upos[e]] = e;
        a.offsets[s.upos[e]] = s.off[e];
      }
    }
    for (int u = nu + tid; u < N; u += nthreads) a.union_ids[u] = -1;
    for (int u = nu + tid; u <= N; u += nthreads) a.offsets[u] = total;
    if (tid == 0) *a.n_union = nu;
  }
  for (int i = tid; i < T * uc; i += nthreads) {
    const int t = i / uc, j = i - t * uc;
    const int e = s.idx[t * k + j];
    const unsigned long long below = t == 0 ? 0ull : (s.mask[e] & (~0ull >> (64 - t)));
    const int p = s.off[e] + __popcll(below);
    const float g = s.gate[t * k + j];
    if (write_out) {
      a.tok_list[p] = t;
      a.gate_list[p] = g;
      a.pair_pos[i] = p;
    }
    if (ptok != nullptr) {
      ptok[p] = t;
      pgate[p] = g;
    }
  }
  __syncthreads();
}

// The union of build_union by one wave, with no block barrier (the caller
// synchronises the block afterwards): position masks by LDS atomics, the
// expert scan, and the lists.  Same results as build_union.
__device__ inline void build_union_wave(const TopkUnionArgs& a, const SelView& s, bool write_out,
                                        int32_t* ptok, float* pgate) {
  const int lane = threadIdx.x & 63;
  const int T = a.T, N = a.N, k = a.k, uc = a.ucols;
  for (int e = lane; e < N; e += kWave) s.mask[e] = 0ull;
  bool bad = false;
  for (int i = lane; i < T * uc; i += kWave) {
    const int t = i / uc, j = i - t * uc;
    const int e = s.idx[t * k + j];
    if (e < 0 || e >= N) {
      bad = true;
    } else {
      const unsigned long long bit = 1ull << t;
      const unsigned long long old = atomicOr(&s.mask[e], bit);
      if (old & bit) bad = true;
    }
  }
  if (__ballot(bad) != 0ull) {
    if (lane == 0) {
      s.misc[1] = -1;
      s.misc[2] = 0;
      if (write_out) *a.n_union = -1;
    }
    return;
  }
  int cnt[4], flg[4], csum = 0, fsum = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = lane * 4 + q;
    const unsigned long long m = e < N ? s.mask[e] : 0ull;
    cnt[q] = (int)__popcll(m);
    flg[q] = m != 0ull;
    csum += cnt[q];
    fsum += flg[q];
  }
  int ci = csum, fi = fsum;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int cu = __shfl_up(ci, o, kWave);
    const int fu = __shfl_up(fi, o, kWave);
    if (lane >= o) {
      ci += cu;
      fi += fu;
    }
  }
  int cbase = ci - csum, fbase = fi - fsum;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = lane * 4 + q;
    if (e < N) {
      s.off[e] = cbase;
      s.upos[e] = fbase;
    }
    cbase += cnt[q];
    fbase += flg[q];
  }
  const int nu = __builtin_amdgcn_readlane(fi, 63), total = __builtin_amdgcn_readlane(ci, 63);
  if (lane == 0) {
    s.misc[1] = nu;
    s.misc[2] = total;
  }
  if (write_out) {
    for (int e = lane; e < N; e += kWave) {
      if (s.mask[e] != 0ull) {
        a.union_ids[s.upos[e]] = e;
        a.offsets[s.upos[e]] = s.off[e];
      }
    }
    for (int u = nu + lane; u < N; u += kWave) a.union_ids[u] = -1;
    for (int u = nu + lane; u <= N; u += kWave) a.offsets[u] = total;
    if (lane == 0) *a.n_union = nu;
  }
  for (int i = lane; i < T * uc; i += kWave) {
    const int t = i / uc, j = i - t * uc;
    const int e = s.idx[t * k + j];
    const unsigned long long below = t == 0 ? 0ull : (s.mask[e] & (~0ull >> (64 - t)));
    const int p = s.off[e] + (int)__popcll(below);
    const float g = s.gate[t * k + j];
    if (write_out) {
      a.tok_list[p] = t;
      a.gate_list[p] = g;
      a.pair_pos[i] = p;
    }
    if (ptok != nullptr) {
      ptok[p] = t;
      pgate[p] = g;
    }
  }
}

// Router logit of one expert (Eq. 1) by one wave: the dot product of the
// expert's fp32 router row w (H4 float4s) with x (xf(h) returns float4 h of
// the position's input), lane-strided in chunks of 8 float4 per lane whose
// loads are in flight together, then summed over the wave.  Every lane
// receives the same bits, whichever memory xf reads.
template <typename XF>
__device__ __forceinline__ float router_dot(const float4* w, int H4, int lane, XF xf) {
  float acc = 0.f;
  for (int h0 = 0; h0 < H4; h0 += kWave * 8) {
    float4 v0[8], xv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int h = min(h0 + lane + j * kWave, H4 - 1);  // clamped: in bounds, skipped below
      v0[j] = w[h];
      xv[j] = xf(h);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (h0 + lane + j * kWave < H4) {
        acc = fmaf(v0[j].x, xv[j].x, acc);
        acc = fmaf(v0[j].y, xv[j].y, acc);
        acc = fmaf(v0[j].z, xv[j].z, acc);
        acc = fmaf(v0[j].w, xv[j].w, acc);
      }
    }
  }
  return wave_sum(acc);
}

// router_dot for rows of at most kWave * 8 float4 (H <= 2048) with the row
// already loaded (w[j] = float4 lane + j * kWave, clamped as in router_dot):
// the same arithmetic, so the same bits.
template <typename XF>
__device__ __forceinline__ float router_dot_pre(const float4 (&w)[8], int H4, int lane, XF xf) {
  float acc = 0.f;
  float4 xv[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) xv[j] = xf(min(lane + j * kWave, H4 - 1));
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    if (lane + j * kWave < H4) {
      acc = fmaf(w[j].x, xv[j].x, acc);
      acc = fmaf(w[j].y, xv[j].y, acc);
      acc = fmaf(w[j].z, xv[j].z, acc);
      acc = fmaf(w[j].w, xv[j].w, acc);
    }
  }
  return wave_sum(acc);
}

}  // namespace de
