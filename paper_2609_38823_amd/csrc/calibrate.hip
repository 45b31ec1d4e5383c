// Activated mass, prefix length and Mean-Mass order (Eqs. 8, 9, 11, 12).
//
//   mass     one workgroup per invocation (segment): the float64 running
//            sums per expert in token order and the prefix length K
//            (device code in mass_dev.hpp, shared with the fused
//            calibration + prefix re-route kernel)
//   order    Mean-Mass order over the segments taken as calibration cases
#include "common.hpp"
#include "mass_dev.hpp"

namespace decomoe {
namespace {

__global__ __launch_bounds__(CAL_THREADS) void segment_mass_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ w, int T, int E, int k, int key_bits,
    const int32_t* __restrict__ seg_offsets, double p, double* __restrict__ mass,
    int32_t* __restrict__ K_out, const Guard g) {
  if (guard_skip(g)) return;
  __shared__ CalLds L;
  const int seg = blockIdx.x;
  const int tid = threadIdx.x;
  int lo = 0, hi = T;
  if (seg_offsets) {
    lo = clampi(seg_offsets[seg], 0, T);
    hi = clampi(seg_offsets[seg + 1], lo, T);
  }
  const int n_all = (hi - lo) * k;
  const double a = n_all <= CAL_STAGE && E <= CAL_SORT_E
                       ? mass_sorted(idx, w, (size_t)lo * k, n_all, E, key_bits, L)
                       : mass_chunked(idx, w, lo, hi, E, k, L);
  if (tid < E) mass[(size_t)seg * E + tid] = a;
  if (K_out) {
    const int K = prefix_K(E, k, p, L);
    if (tid == 0) K_out[seg] = K;
  }
}

// Mean-Mass order over the segments taken as calibration cases (Eqs. 8, 9):
// mean_e = (sum over non-empty segments, in order, of s_e / len) / n_cases;
// order = argsort descending, ties to the lower expert index.
__global__ __launch_bounds__(1024) void mean_mass_order_kernel(
    const double* __restrict__ mass, int T, int E, const int32_t* __restrict__ seg_offsets,
    int n_seg, int32_t* __restrict__ order, const Guard g) {
  if (guard_skip(g)) return;
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

size_t calibrate_ws_bytes(int T, int E) {
  (void)T;
  (void)E;
  return 0;  // the dense table lives in LDS
}

hipError_t launch_calibrate(const int32_t* idx, const float* w, int T, int E, int k,
                            const int32_t* seg_offsets, int n_seg, double p, double* mass,
                            int32_t* K_out, int32_t* order, void* ws, hipStream_t s, Guard g) {
  (void)ws;
  int key_bits = 0;
  while ((1 << key_bits) < E) ++key_bits;
  segment_mass_kernel<<<n_seg, CAL_THREADS, 0, s>>>(idx, w, T, E, k, key_bits, seg_offsets, p, mass,
                                                    K_out, g);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || !order) return err;
  mean_mass_order_kernel<<<1, 1024, 0, s>>>(mass, T, E, seg_offsets, n_seg, order, g);
  return hipGetLastError();
}

}  // namespace decomoe
