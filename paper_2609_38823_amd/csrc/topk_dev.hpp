// Wavefront Top-k primitives shared by the routing kernels (Eq. 10 and the
// prefix re-route of Sec. 3.3): a total order on (value, index) pairs, DPP
// arg-max and sum over a wavefront, and the selection of the k best of one
// token's first Klim logits with their softmax weights.
#pragma once

#include <float.h>

#include "common.hpp"

namespace decomoe {
namespace {

// (ov, oi) replaces (v, i) when its value is larger, or equal with a smaller
// index; evaluated without short-circuit so that it compiles to compares and
// selects (no exec-mask branches)
__device__ __forceinline__ void better(float& v, int& i, float ov, int oi) {
  const bool take = (ov > v) | ((ov == v) & (oi < i));
  v = take ? ov : v;
  i = take ? oi : i;
}

// (value, index) of lane l -> the wavefront's best pair in every lane
// without LDS round trips: DPP moves within each row of 16 lanes (quad
// swaps, then the half-row and row mirrors pair the groups), then the four
// row results are read with v_readlane and combined (the same in every
// lane).  `better` is a total order on pairs, so the pairing order does not
// change the result.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ void dpp_better(float& v, int& i) {
  better(v, i, dpp_f<CTRL>(v), __builtin_amdgcn_mov_dpp(i, CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float lane_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
__device__ __forceinline__ void wave_best(float& v, int& i) {
  dpp_better<0xB1>(v, i);   // quad_perm [1, 0, 3, 2]
  dpp_better<0x4E>(v, i);   // quad_perm [2, 3, 0, 1]
  dpp_better<0x141>(v, i);  // row_half_mirror
  dpp_better<0x140>(v, i);  // row_mirror
  float bv = lane_f(v, 0);
  int bi = __builtin_amdgcn_readlane(i, 0);
#pragma unroll
  for (int r = 1; r < 4; ++r) better(bv, bi, lane_f(v, 16 * r), __builtin_amdgcn_readlane(i, 16 * r));
  v = bv;
  i = bi;
}
// sum over the wavefront: row sums by DPP, then the four rows in order
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  v += dpp_f<0x141>(v);
  v += dpp_f<0x140>(v);
  return ((lane_f(v, 0) + lane_f(v, 16)) + lane_f(v, 32)) + lane_f(v, 48);
}

// The k largest of one token's logits [0, Klim), one wavefront: lane l
// holds experts l, l + 64, ... in vals[c] (expert l + 64 c); k rounds of a
// wavefront arg-max (value descending, index ascending on ties) pick the
// slots in order; the weights are the softmax of the k selected logits.
// Lane r < k writes slot r.  Values at experts >= Klim are never selected.
template <int MAXC>  // values per lane: E <= 64 MAXC
__device__ __forceinline__ void topk_select_vals(const float (&vals)[MAXC], int E, int k, int Klim, int lane,
                                                 int32_t* idx_t, float* w_t) {
  // a taken or absent candidate is (-inf, INT_MAX): `better` never prefers
  // it, so the rounds need no per-candidate branches
  float v[MAXC];
  int ix[MAXC];
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int e = lane + c * 64;
    v[c] = e < Klim ? vals[c] : -INFINITY;
    ix[c] = e < Klim ? e : 0x7fffffff;
  }
  float my_v = 0.f;
  int my_i = 0;
  for (int r = 0; r < k; ++r) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) better(bv, bi, v[c], ix[c]);
    wave_best(bv, bi);
#pragma unroll
    for (int c = 0; c < MAXC; ++c)
      if (ix[c] == bi) {
        v[c] = -INFINITY;
        ix[c] = 0x7fffffff;
      }
    if (lane == r) { my_v = bv; my_i = bi; }
  }
  const float v0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, my_v), 0));
  float ex = lane < k ? expf(my_v - v0) : 0.f;
  float sum = ex;
  sum = wave_sum(sum);
  if (lane < k) {
    idx_t[lane] = my_i;
    w_t[lane] = ex / sum;
  }
}

// the same on row[0, Klim) in memory
template <int MAXC>
__device__ __forceinline__ void topk_select(const float* row, int E, int k, int Klim, int lane,
                                            int32_t* idx_t, float* w_t) {
  float v[MAXC];
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int e = lane + c * 64;
    v[c] = e < Klim ? row[e] : 0.f;
  }
  topk_select_vals<MAXC>(v, E, k, Klim, lane, idx_t, w_t);
}

// ---- one token per row of 16 lanes (four tokens per wavefront) ---------
// the row's best pair in all 16 lanes: quad swaps, then the half-row and row
// mirrors (no value leaves the row)
__device__ __forceinline__ void row_best(float& v, int& i) {
  dpp_better<0xB1>(v, i);   // quad_perm [1, 0, 3, 2]
  dpp_better<0x4E>(v, i);   // quad_perm [2, 3, 0, 1]
  dpp_better<0x141>(v, i);  // row_half_mirror
  dpp_better<0x140>(v, i);  // row_mirror
}
__device__ __forceinline__ float row_sum(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  v += dpp_f<0x141>(v);
  v += dpp_f<0x140>(v);
  return v;
}

// The k best of one token's logits [0, Klim) held by the 16 lanes of a row:
// lane j holds experts j, j + 16, ... in v[c] (expert j + 16 c).  Each
// round's arg-max is a lane-local scan plus row_best; round r's winner is
// kept by lane r % 16 in slot r / 16 (k <= 32).  Same selection order, tie
// rule and weights as topk_select_vals: the slots' exponentials are summed
// by the same butterfly, so for k <= 16 the weights are bitwise equal.
template <int MAXC>
__device__ __forceinline__ void row_topk_select(const float (&v)[MAXC], int j, int E, int k, int Klim,
                                                int32_t* idx_t, float* w_t) {
  // candidates as in topk_select_vals: a taken or absent one is (-inf,
  // INT_MAX), which `better` never prefers
  float cv[MAXC];
  int ix[MAXC];
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int e = j + 16 * c;
    cv[c] = e < Klim ? v[c] : -INFINITY;
    ix[c] = e < Klim ? e : 0x7fffffff;
  }
  float my_v[2] = {0.f, 0.f};
  int my_i[2] = {0, 0};
  float v0 = 0.f;
  for (int r = 0; r < k; ++r) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int c = 0; c < MAXC; ++c) better(bv, bi, cv[c], ix[c]);
    row_best(bv, bi);
#pragma unroll
    for (int c = 0; c < MAXC; ++c)
      if (ix[c] == bi) {
        cv[c] = -INFINITY;
        ix[c] = 0x7fffffff;
      }
    if (r == 0) v0 = bv;
    if ((r & 15) == j) {
      my_v[r >> 4] = bv;
      my_i[r >> 4] = bi;
    }
  }
  float ex[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) ex[q] = j + 16 * q < k ? expf(my_v[q] - v0) : 0.f;
  // slots in order r = 0..k-1: lanes hold r = j and r = j + 16; the row sum
  // adds the k exponentials (the same total in every lane of the row)
  const float sum = row_sum(ex[0] + ex[1]);
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int r = j + 16 * q;
    if (r < k) {
      idx_t[r] = my_i[q];
      w_t[r] = ex[q] / sum;
    }
  }
}

}  // namespace
}  // namespace decomoe
