// Activated mass, prefix length and Mean-Mass order (Eqs. 8, 9, 11, 12).
//
// One workgroup per invocation (segment).  The segment's renormalised Top-k
// weights are scattered, up to 128 tokens per pass, into a dense LDS table
// [token][expert]; thread e then adds its column to a float64 running sum in
// ascending token order.  The next pass's entries are fetched into registers
// while the current pass is summed.  Every expert's mass is therefore one sequential
// float64 sum in token order (no atomics, no tree), and the running prefix
// sum over experts that decides K is sequential too.
#include "common.hpp"

namespace decomoe {
namespace {

constexpr int CAL_THREADS = 256;
constexpr int CAL_TABLE = 16384;  // doubles in the dense LDS table (128 KB)
constexpr int CAL_STAGE = 1024;   // routing entries staged per pass
constexpr int CAL_EPT = CAL_STAGE / CAL_THREADS;

// Tokens per pass: the table holds sub x E doubles and the stage sub x k entries.
__host__ __device__ inline int cal_sub(int E, int k) {
  int s = CAL_TABLE / E;
  if (s * k > CAL_STAGE) s = CAL_STAGE / k;
  return s < 128 ? s : 128;
}

__global__ __launch_bounds__(CAL_THREADS) void segment_mass_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ w, int T, int E, int k,
    const int32_t* __restrict__ seg_offsets, double p, double* __restrict__ mass,
    int32_t* __restrict__ K_out) {
  __shared__ double table[CAL_TABLE];
  __shared__ int stage_e[CAL_STAGE];
  __shared__ float stage_w[CAL_STAGE];
  __shared__ double smass[1024];
  const int seg = blockIdx.x;
  const int tid = threadIdx.x;
  int lo = 0, hi = T;
  if (seg_offsets) {
    lo = clampi(seg_offsets[seg], 0, T);
    hi = clampi(seg_offsets[seg + 1], lo, T);
  }
  const int sub = cal_sub(E, k);
  constexpr int EPT = 1024 / CAL_THREADS;  // experts per thread, at most 4
  double acc[EPT] = {};

  // one pass's entries, prefetched into registers one pass ahead
  int pe[CAL_EPT];
  float pw[CAL_EPT];
  auto fetch = [&](int t0) {
    const int n = min(sub, hi - t0) * k;
    const size_t base = (size_t)t0 * k;
#pragma unroll
    for (int j = 0; j < CAL_EPT; ++j) {
      const int i = tid + j * CAL_THREADS;
      pe[j] = i < n ? idx[base + i] : -1;
      pw[j] = i < n ? w[base + i] : 0.f;
    }
  };

  for (int i = tid; i < sub * E; i += CAL_THREADS) table[i] = 0.0;
  if (lo < hi) fetch(lo);
  for (int t0 = lo; t0 < hi; t0 += sub) {
    const int nt = min(sub, hi - t0);
#pragma unroll
    for (int j = 0; j < CAL_EPT; ++j) {
      stage_e[tid + j * CAL_THREADS] = pe[j];
      stage_w[tid + j * CAL_THREADS] = pw[j];
    }
    __syncthreads();
    if (t0 + sub < hi) fetch(t0 + sub);
    // one thread per token adds its slots in slot order
    if (tid < nt) {
      for (int j = 0; j < k; ++j) {
        const int e = stage_e[tid * k + j];
        if (e >= 0 && e < E) table[tid * E + e] += static_cast<double>(stage_w[tid * k + j]);
      }
    }
    __syncthreads();
    // expert columns: one float64 running sum per expert, ascending token
#pragma unroll
    for (int c = 0; c < EPT; ++c) {
      const int e = tid + c * CAL_THREADS;
      if (e < E)
        for (int r = 0; r < nt; ++r) acc[c] += table[r * E + e];
    }
    __syncthreads();
    if (tid < nt) {
      for (int j = 0; j < k; ++j) {
        const int e = stage_e[tid * k + j];
        if (e >= 0 && e < E) table[tid * E + e] = 0.0;
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int c = 0; c < EPT; ++c) {
    const int e = tid + c * CAL_THREADS;
    if (e < E) {
      mass[(size_t)seg * E + e] = acc[c];
      smass[e] = acc[c];
    }
  }
  __syncthreads();
  if (tid == 0 && K_out) {
    // c_K running sum in expert order; tot = c_E; first K with c_K >= p*tot
    double run = 0.0;
    for (int e = 0; e < E; ++e) {
      run += smass[e];
      table[e] = run;
    }
    const double thr = p * run;
    int k_hat = E;
    for (int K = 1; K <= E; ++K)
      if (table[K - 1] >= thr) { k_hat = K; break; }
    K_out[seg] = k_hat > k ? k_hat : k;
  }
}

// Mean-Mass order over the segments taken as calibration cases (Eqs. 8, 9):
// mean_e = (sum over non-empty segments, in order, of s_e / len) / n_cases;
// order = argsort descending, ties to the lower expert index.
__global__ __launch_bounds__(1024) void mean_mass_order_kernel(
    const double* __restrict__ mass, int T, int E, const int32_t* __restrict__ seg_offsets,
    int n_seg, int32_t* __restrict__ order) {
  __shared__ double mean[1024];
  const int e = threadIdx.x;
  if (e < E) {
    double tot = 0.0;
    int cases = 0;
    for (int s = 0; s < n_seg; ++s) {
      int lo = 0, hi = T;
      if (seg_offsets) {
        lo = clampi(seg_offsets[s], 0, T);
        hi = clampi(seg_offsets[s + 1], lo, T);
      }
      if (hi > lo) {
        tot += mass[(size_t)s * E + e] / static_cast<double>(hi - lo);
        ++cases;
      }
    }
    mean[e] = cases ? tot / static_cast<double>(cases) : 0.0;
  }
  __syncthreads();
  if (e < E) {
    const double me = mean[e];
    int rank = 0;
    for (int j = 0; j < E; ++j) {
      double mj = mean[j];
      rank += (mj > me) || (mj == me && j < e);
    }
    order[rank] = e;
  }
}
}  // namespace

hipError_t launch_calibrate(const int32_t* idx, const float* w, int T, int E, int k,
                            const int32_t* seg_offsets, int n_seg, double p, double* mass,
                            int32_t* K_out, int32_t* order, hipStream_t s) {
  segment_mass_kernel<<<n_seg, CAL_THREADS, 0, s>>>(idx, w, T, E, k, seg_offsets, p, mass, K_out);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || !order) return err;
  mean_mass_order_kernel<<<1, 1024, 0, s>>>(mass, T, E, seg_offsets, n_seg, order);
  return hipGetLastError();
}

}  // namespace decomoe
