// Activated mass of one invocation and its prefix length (Eqs. 11, 12):
// device code shared by the calibration kernel and the fused calibration +
// prefix re-route kernel.  Every function here is called by all
// CAL_THREADS threads of the workgroup (they synchronise it).
//
//   mass_sorted   up to CAL_STAGE routing entries and E <= CAL_SORT_E: the
//                 entries are staged with one bulk load and grouped by
//                 expert with a stable counting sort in LDS (token order
//                 kept within an expert); thread e adds its expert's weights
//                 in that order
//   mass_chunked  larger invocations: chunks of tokens are scattered into a
//                 dense LDS table [token][expert] (float64) and thread e
//                 adds column e in ascending token order
// Either way one float64 running sum per expert over the tokens: the
// sequence of additions of the plain definition (unrouted tokens add zeros,
// which change nothing).
//   prefix_K      the running sum c_K over the experts by one thread, then
//                 the first K with c_K >= p * c_E by a ballot; K = max(k, K)
#pragma once

#include "common.hpp"

namespace decomoe {
namespace {

constexpr int CAL_THREADS = 1024;
constexpr int CAL_TABLE = 8192;  // doubles in the LDS table (64 KB)
constexpr int CAL_STAGE = 8192;  // routing entries staged per bulk load (64 KB)
constexpr int CAL_ENT = 1024;    // routing entries scattered per chunk (one per thread)
constexpr int CAL_WAVES = CAL_THREADS / kWave;
constexpr int CAL_SORT_E = 512;  // the sorted path keeps [waves][E] counts in half the table

// Tokens per chunk: the table holds ch x E doubles and a chunk holds at most
// CAL_ENT routing entries.
__host__ __device__ inline int cal_chunk(int E, int k) {
  int c = CAL_TABLE / E;
  if (c * k > CAL_ENT) c = CAL_ENT / k;
  return c < 64 ? c : 64;
}

struct CalLds {
  double table[CAL_TABLE];
  double smass[1024 + 32];  // zero past E (the c_K loop reads whole batches)
  int st_e[CAL_STAGE];
  float st_w[CAL_STAGE];
  int s_cnt[1024], s_off[1024];
  int part[CAL_WAVES];
  double s_tot;
  int s_K;
};

// sets L.smass[e] = the mass of expert e (zero past E) and returns it in
// thread e < E.  n_all = routing entries from idx + base (token-major).
__device__ double mass_sorted(const int32_t* __restrict__ idx, const float* __restrict__ w, size_t base,
                              int n_all, int E, int key_bits, CalLds& L) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  int* wh = reinterpret_cast<int*>(L.table);                                   // [waves][E]
  float* sorted = reinterpret_cast<float*>(L.table) + CAL_WAVES * CAL_SORT_E;  // [CAL_STAGE]
  {
    constexpr int SPT = CAL_STAGE / CAL_THREADS;
    int re[SPT];
    float rw[SPT];
#pragma unroll
    for (int q = 0; q < SPT; ++q) {
      const int i = tid + q * CAL_THREADS;
      re[q] = i < n_all ? idx[base + i] : -1;
      rw[q] = i < n_all ? w[base + i] : 0.f;
    }
#pragma unroll
    for (int q = 0; q < SPT; ++q) {  // only entries below n_all are read below
      if (tid + q * CAL_THREADS < n_all) {
        L.st_e[tid + q * CAL_THREADS] = re[q];
        L.st_w[tid + q * CAL_THREADS] = rw[q];
      }
    }
  }
  for (int i = tid; i < CAL_WAVES * E; i += CAL_THREADS) wh[i] = 0;
  __syncthreads();
  const int per = ((n_all + CAL_WAVES - 1) / CAL_WAVES + kWave - 1) / kWave * kWave;
  const int a_lo = min(n_all, wv * per), a_hi = min(n_all, a_lo + per);
  for (int a = a_lo + lane; a < a_hi; a += kWave) {
    const int e = L.st_e[a];
    if (e >= 0 && e < E) atomicAdd(&wh[wv * E + e], 1);
  }
  __syncthreads();
  int cnt = 0;
  if (tid < E)
    for (int q = 0; q < CAL_WAVES; ++q) cnt += wh[q * E + tid];
  int incl = cnt;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_up(incl, off, kWave);
    if (lane >= off) incl += y;
  }
  if (lane == kWave - 1) L.part[wv] = incl;
  __syncthreads();
  if (tid < E) {
    int r = incl - cnt;
    for (int q = 0; q < wv; ++q) r += L.part[q];
    L.s_cnt[tid] = cnt;
    L.s_off[tid] = r;
    for (int q = 0; q < CAL_WAVES; ++q) {  // per-wave starting positions
      const int c = wh[q * E + tid];
      wh[q * E + tid] = r;
      r += c;
    }
  }
  __syncthreads();
  const uint64_t lt_mask = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  for (int a0 = a_lo; a0 < a_hi; a0 += kWave) {
    const int a = a0 + lane;
    const int e = a < a_hi ? L.st_e[a] : -1;
    const bool valid = e >= 0 && e < E;
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < key_bits; ++b) {
      const bool bit = (e >> b) & 1;
      const uint64_t msk = __ballot(bit);
      peers &= bit ? msk : ~msk;
    }
    if (valid) {
      sorted[wh[wv * E + e] + __popcll(peers & lt_mask)] = L.st_w[a];
      if ((63 - __clzll(peers)) == lane) wh[wv * E + e] += __popcll(peers);
    }
    __builtin_amdgcn_wave_barrier();
  }
  __syncthreads();
  double a = 0.0;
  if (tid < E) {
    // one dependent float64 chain per expert (the latency of the
    // additions, not of the LDS reads, bounds it)
    const int b0 = L.s_off[tid], b1 = b0 + L.s_cnt[tid];
#pragma unroll 8
    for (int j = b0; j < b1; ++j) a += static_cast<double>(sorted[j]);
    L.smass[tid] = a;
  } else {
    L.smass[tid] = 0.0;
  }
  if (tid < 32) L.smass[1024 + tid] = 0.0;
  __syncthreads();
  return a;
}

// the same for the tokens [lo, hi), any size
__device__ double mass_chunked(const int32_t* __restrict__ idx, const float* __restrict__ w, int lo, int hi,
                               int E, int k, CalLds& L) {
  const int tid = threadIdx.x;
  const int ch = cal_chunk(E, k);
  const int super_t = (CAL_STAGE / k) / ch * ch;  // tokens staged per bulk load
  for (int i = tid; i < ch * E; i += CAL_THREADS) L.table[i] = 0.0;
  double acc = 0.0;
  for (int s0 = lo; s0 < hi; s0 += super_t) {
    // stage the routing entries of up to super_t tokens with one bulk load
    const int n_ent = min(super_t, hi - s0) * k;
    __syncthreads();  // previous stage fully consumed
    {
      constexpr int SPT = CAL_STAGE / CAL_THREADS;  // all loads in flight together
      int re[SPT];
      float rw[SPT];
#pragma unroll
      for (int q = 0; q < SPT; ++q) {
        const int i = tid + q * CAL_THREADS;
        re[q] = i < n_ent ? idx[(size_t)s0 * k + i] : -1;
        rw[q] = i < n_ent ? w[(size_t)s0 * k + i] : 0.f;
      }
#pragma unroll
      for (int q = 0; q < SPT; ++q) {
        L.st_e[tid + q * CAL_THREADS] = re[q];
        L.st_w[tid + q * CAL_THREADS] = rw[q];
      }
    }
    __syncthreads();
    for (int t0 = s0; t0 < min(s0 + super_t, hi); t0 += ch) {
      const int nt = min(ch, hi - t0);
      // scatter: a token's experts are distinct (Top-k), so each cell gets
      // one addition onto 0.0 and holds the weight exactly; a repeated
      // expert adds its weights into the cell
#pragma unroll
      for (int q = 0; q < CAL_ENT / CAL_THREADS; ++q) {
        const int j = tid + q * CAL_THREADS;
        if (j < nt * k) {
          const int i = (t0 - s0) * k + j;
          const int e = L.st_e[i];
          if (e >= 0 && e < E) atomicAdd(&L.table[(j / k) * E + e], static_cast<double>(L.st_w[i]));
        }
      }
      __syncthreads();
      // column sums: thread e adds column e in ascending token order, then
      // clears it for the next chunk
      if (tid < E) {
        double a = acc;
#pragma unroll 8
        for (int r = 0; r < nt; ++r) {
          a += L.table[r * E + tid];
          L.table[r * E + tid] = 0.0;
        }
        acc = a;
      }
      __syncthreads();
    }
  }
  if (tid < E) {
    L.smass[tid] = acc;
  } else {
    L.smass[tid] = 0.0;
  }
  if (tid < 32) L.smass[1024 + tid] = 0.0;
  __syncthreads();
  return acc;
}

// K = max(k, the first K with c_K >= p * c_E) from L.smass, in every thread.
// c_K: one running sum in expert order by a single thread (the same
// sequence of float64 additions as the definition).  The masses come from
// LDS in batches of 16, the next batch read while the current one is added,
// with no per-element conditions (the masses past E are zero, and adding
// +0.0 to the non-negative running sum changes no bit); the c_K go to LDS
// and wave 0 finds the first K with c_K >= p * tot by a ballot.
__device__ int prefix_K(int E, int k, double p, CalLds& L) {
  const int tid = threadIdx.x;
  double* cbuf = L.table;  // free once the masses are formed
  if (tid == 0) {
    constexpr int B = 16;
    const int Ep = (E + B - 1) / B * B;
    double run = 0.0, v[B], nv[B];
#pragma unroll
    for (int j = 0; j < B; ++j) v[j] = L.smass[j];
    for (int e0 = 0; e0 < Ep; e0 += B) {
#pragma unroll
      for (int j = 0; j < B; ++j) nv[j] = L.smass[e0 + B + j];
#pragma unroll
      for (int j = 0; j < B; ++j) {
        run += v[j];
        cbuf[e0 + j] = run;
      }
#pragma unroll
      for (int j = 0; j < B; ++j) v[j] = nv[j];
    }
    L.s_tot = run;  // tot = c_E
  }
  __syncthreads();
  if (tid < kWave) {
    const double thr = p * L.s_tot;
    int k_hat = E;
    for (int e0 = 0; e0 < E; e0 += kWave) {
      const unsigned long long hit = __ballot(e0 + tid < E && cbuf[e0 + tid] >= thr);
      if (hit) {
        k_hat = e0 + __ffsll((long long)hit);  // K = index + 1
        break;
      }
    }
    if (tid == 0) L.s_K = k_hat > k ? k_hat : k;
  }
  __syncthreads();
  return L.s_K;
}

}  // namespace
}  // namespace decomoe
