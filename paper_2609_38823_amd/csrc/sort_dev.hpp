// Stable counting sort of up to DS_MAX routing entries by expert in one
// workgroup of DS_THREADS threads (Algorithm 2's dispatch: the rows of one
// expert keep ascending (token, slot) order).  Device code shared by the
// dispatch kernel and the one-launch calibration of moe_route_rcep.
#pragma once

#include "common.hpp"

namespace decomoe {
namespace {

constexpr int DS_THREADS = 1024;
constexpr int DS_WAVES = DS_THREADS / kWave;
constexpr int DS_MAX = 8192;  // beyond this the multi-workgroup path is faster

// All DS_THREADS threads call it.  keys[a] is the expert of entry a (global
// or LDS memory); entries outside [0, E) are dropped (row_of_slot = -1).
// The 16 wavefronts take contiguous slices in entry order, count their slice
// per expert in LDS (wh: DS_WAVES rows of ld ints, ld >= E), one scan turns
// the counts into offsets and each wavefront's starting row per expert, and
// the wavefronts rank their slices: the ballots over the key bits find the
// lanes with the same expert and a popcount gives each its rank.
__device__ void sort_small(const int32_t* keys, int A, int E, int key_bits, int* wh, int ld, int* part,
                           int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
                           int32_t* __restrict__ src_of_row, int32_t* __restrict__ row_of_slot) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int per = (A + DS_WAVES - 1) / DS_WAVES;
  const int lo = min(A, wv * per), hi = min(A, lo + per);
  for (int i = tid; i < DS_WAVES * ld; i += DS_THREADS) wh[i] = 0;
  __syncthreads();
  for (int a = lo + lane; a < hi; a += kWave) {
    const int e = keys[a];
    if (e >= 0 && e < E) atomicAdd(&wh[wv * ld + e], 1);
  }
  __syncthreads();
  // thread e: total count, then an exclusive scan over the experts
  int cnt = 0;
  if (tid < E)
#pragma unroll
    for (int w = 0; w < DS_WAVES; ++w) cnt += wh[w * ld + tid];
  int incl = cnt;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_up(incl, off, kWave);
    if (lane >= off) incl += y;
  }
  if (lane == kWave - 1) part[wv] = incl;
  __syncthreads();
  int base = 0;
  for (int w = 0; w < wv; ++w) base += part[w];
  if (tid < E) {
    int r = base + incl - cnt;  // exclusive offset of expert tid
    counts[tid] = cnt;
    offsets[tid] = r;
    if (tid == E - 1) offsets[E] = r + cnt;
#pragma unroll
    for (int w = 0; w < DS_WAVES; ++w) {
      const int c = wh[w * ld + tid];
      wh[w * ld + tid] = r;
      r += c;
    }
  }
  __syncthreads();
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int a0 = lo; a0 < hi; a0 += kWave) {
    const int a = a0 + lane;
    const int e = a < hi ? keys[a] : -1;
    const bool valid = e >= 0 && e < E;
    uint64_t peers = __ballot(valid);
#pragma unroll 1
    for (int b = 0; b < key_bits; ++b) {
      const bool bit = (e >> b) & 1;
      const uint64_t msk = __ballot(bit);
      peers &= bit ? msk : ~msk;
    }
    if (valid) {
      const int r = wh[wv * ld + e] + __popcll(peers & lt_mask);
      src_of_row[r] = a;
      row_of_slot[a] = r;
      if ((63 - __clzll(peers)) == lane) wh[wv * ld + e] += __popcll(peers);
    } else if (a < hi) {
      row_of_slot[a] = -1;
    }
    __builtin_amdgcn_wave_barrier();
  }
}

}  // namespace
}  // namespace decomoe
