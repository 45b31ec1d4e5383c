// Activated mass, prefix length and Mean-Mass order (Eqs. 8, 9, 11, 12).
//
//   mass     one workgroup per invocation (segment) stages the routing
//            entries with one bulk load.  Up to 8192 entries (and E <= 512):
//            a stable counting sort in LDS groups them by expert, token order
//            kept, and thread e adds its expert's weights in that order.
//            Larger segments are walked in chunks: the chunk's weights are
//            scattered into a dense LDS table [token][expert] (float64) and
//            thread e adds column e in ascending token order.  Either way one
//            float64 running sum per expert over the tokens: the sequence of
//            additions of the plain definition (unrouted tokens add zeros,
//            which change nothing).  One thread then forms the running sum
//            c_K over the experts and wave 0 finds K with a ballot.
//   order    Mean-Mass order over the segments taken as calibration cases
#include "common.hpp"

namespace decomoe {
namespace {

constexpr int CAL_THREADS = 1024;
constexpr int CAL_TABLE = 8192;  // doubles in the LDS table (64 KB)
constexpr int CAL_STAGE = 8192;  // routing entries staged per bulk load (64 KB)

constexpr int CAL_ENT = 1024;   // routing entries scattered per chunk (one per thread)

// Tokens per chunk: the table holds ch x E doubles and a chunk holds at most
// CAL_ENT routing entries.
__host__ __device__ inline int cal_chunk(int E, int k) {
  int c = CAL_TABLE / E;
  if (c * k > CAL_ENT) c = CAL_ENT / k;
  return c < 64 ? c : 64;
}

constexpr int CAL_WAVES = CAL_THREADS / kWave;
constexpr int CAL_SORT_E = 512;  // the sorted path keeps [waves][E] counts in half the table

__global__ __launch_bounds__(CAL_THREADS) void segment_mass_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ w, int T, int E, int k, int key_bits,
    const int32_t* __restrict__ seg_offsets, double p, double* __restrict__ mass,
    int32_t* __restrict__ K_out) {
  __shared__ double table[CAL_TABLE];
  __shared__ double smass[1024 + 32];  // zero past E (the c_K loop reads whole batches)
  __shared__ int st_e[CAL_STAGE];
  __shared__ float st_w[CAL_STAGE];
  __shared__ int s_cnt[1024], s_off[1024];
  __shared__ int part[CAL_WAVES];
  const int seg = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  int lo = 0, hi = T;
  if (seg_offsets) {
    lo = clampi(seg_offsets[seg], 0, T);
    hi = clampi(seg_offsets[seg + 1], lo, T);
  }
  const int n_all = (hi - lo) * k;
  if (n_all <= CAL_STAGE && E <= CAL_SORT_E) {
    // ---- sorted path: the segment's entries are grouped by expert with a
    // stable counting sort in LDS (token order kept within an expert), then
    // thread e adds its expert's weights in that order -- the sequence of
    // float64 additions of the definition minus the additions of zero
    int* wh = reinterpret_cast<int*>(table);                      // [waves][E]
    float* sorted = reinterpret_cast<float*>(table) + CAL_WAVES * CAL_SORT_E;  // [CAL_STAGE]
    {
      constexpr int SPT = CAL_STAGE / CAL_THREADS;
      int re[SPT];
      float rw[SPT];
#pragma unroll
      for (int q = 0; q < SPT; ++q) {
        const int i = tid + q * CAL_THREADS;
        re[q] = i < n_all ? idx[(size_t)lo * k + i] : -1;
        rw[q] = i < n_all ? w[(size_t)lo * k + i] : 0.f;
      }
#pragma unroll
      for (int q = 0; q < SPT; ++q) {
        st_e[tid + q * CAL_THREADS] = re[q];
        st_w[tid + q * CAL_THREADS] = rw[q];
      }
    }
    for (int i = tid; i < CAL_WAVES * E; i += CAL_THREADS) wh[i] = 0;
    __syncthreads();
    const int per = ((n_all + CAL_WAVES - 1) / CAL_WAVES + kWave - 1) / kWave * kWave;
    const int a_lo = min(n_all, wv * per), a_hi = min(n_all, a_lo + per);
    for (int a = a_lo + lane; a < a_hi; a += kWave) {
      const int e = st_e[a];
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
    if (lane == kWave - 1) part[wv] = incl;
    __syncthreads();
    if (tid < E) {
      int r = incl - cnt;
      for (int q = 0; q < wv; ++q) r += part[q];
      s_cnt[tid] = cnt;
      s_off[tid] = r;
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
      const int e = a < a_hi ? st_e[a] : -1;
      const bool valid = e >= 0 && e < E;
      uint64_t peers = __ballot(valid);
      for (int b = 0; b < key_bits; ++b) {
        const bool bit = (e >> b) & 1;
        const uint64_t msk = __ballot(bit);
        peers &= bit ? msk : ~msk;
      }
      if (valid) {
        sorted[wh[wv * E + e] + __popcll(peers & lt_mask)] = st_w[a];
        if ((63 - __clzll(peers)) == lane) wh[wv * E + e] += __popcll(peers);
      }
      __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    if (tid < E) {
      // one dependent float64 chain per expert (the latency of the
      // additions, not of the LDS reads, bounds it)
      double a = 0.0;
      const int b0 = s_off[tid], b1 = b0 + s_cnt[tid];
#pragma unroll 8
      for (int j = b0; j < b1; ++j) a += static_cast<double>(sorted[j]);
      mass[(size_t)seg * E + tid] = a;
      smass[tid] = a;
    } else {
      smass[tid] = 0.0;
    }
    if (tid < 32) smass[1024 + tid] = 0.0;
    __syncthreads();
  } else {
  const int ch = cal_chunk(E, k);
  const int super_t = (CAL_STAGE / k) / ch * ch;  // tokens staged per bulk load
  for (int i = tid; i < ch * E; i += CAL_THREADS) table[i] = 0.0;
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
        st_e[tid + q * CAL_THREADS] = re[q];
        st_w[tid + q * CAL_THREADS] = rw[q];
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
          const int e = st_e[i];
          if (e >= 0 && e < E) atomicAdd(&table[(j / k) * E + e], static_cast<double>(st_w[i]));
        }
      }
      __syncthreads();
      // column sums: thread e adds column e in ascending token order, then
      // clears it for the next chunk
      if (tid < E) {
        double a = acc;
#pragma unroll 8
        for (int r = 0; r < nt; ++r) {
          a += table[r * E + tid];
          table[r * E + tid] = 0.0;
        }
        acc = a;
      }
      __syncthreads();
    }
  }
  if (tid < E) {
    mass[(size_t)seg * E + tid] = acc;
    smass[tid] = acc;
  } else {
    smass[tid] = 0.0;
  }
  if (tid < 32) smass[1024 + tid] = 0.0;
  __syncthreads();
  }  // chunked path
  if (K_out) {
    // c_K: one running sum in expert order by a single thread (the same
    // sequence of float64 additions as the definition).  The masses come
    // from LDS in batches of 16, the next batch read while the current one
    // is added, with no per-element conditions (the masses past E are zero,
    // and adding +0.0 to the non-negative running sum changes no bit); the
    // c_K go to LDS and wave 0 finds the first K with c_K >= p * tot by a
    // ballot
    double* cbuf = table;  // the table is free now
    __shared__ double s_tot;
    if (tid == 0) {
      constexpr int B = 16;
      const int Ep = (E + B - 1) / B * B;
      double run = 0.0, v[B], nv[B];
#pragma unroll
      for (int j = 0; j < B; ++j) v[j] = smass[j];
      for (int e0 = 0; e0 < Ep; e0 += B) {
#pragma unroll
        for (int j = 0; j < B; ++j) nv[j] = smass[e0 + B + j];
#pragma unroll
        for (int j = 0; j < B; ++j) {
          run += v[j];
          cbuf[e0 + j] = run;
        }
#pragma unroll
        for (int j = 0; j < B; ++j) v[j] = nv[j];
      }
      s_tot = run;  // tot = c_E
    }
    __syncthreads();
    if (tid < kWave) {
      const double thr = p * s_tot;
      int k_hat = E;
      for (int e0 = 0; e0 < E; e0 += kWave) {
        const unsigned long long hit = __ballot(e0 + tid < E && cbuf[e0 + tid] >= thr);
        if (hit) {
          k_hat = e0 + __ffsll((long long)hit);  // K = index + 1
          break;
        }
      }
      if (tid == 0) K_out[seg] = k_hat > k ? k_hat : k;
    }
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

size_t calibrate_ws_bytes(int T, int E) {
  (void)T;
  (void)E;
  return 0;  // the dense table lives in LDS
}

hipError_t launch_calibrate(const int32_t* idx, const float* w, int T, int E, int k,
                            const int32_t* seg_offsets, int n_seg, double p, double* mass,
                            int32_t* K_out, int32_t* order, void* ws, hipStream_t s) {
  (void)ws;
  int key_bits = 0;
  while ((1 << key_bits) < E) ++key_bits;
  segment_mass_kernel<<<n_seg, CAL_THREADS, 0, s>>>(idx, w, T, E, k, key_bits, seg_offsets, p, mass,
                                                    K_out);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || !order) return err;
  mean_mass_order_kernel<<<1, 1024, 0, s>>>(mass, T, E, seg_offsets, n_seg, order);
  return hipGetLastError();
}

}  // namespace decomoe
