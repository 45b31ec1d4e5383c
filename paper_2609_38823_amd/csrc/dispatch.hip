// Dispatch: stable counting sort of the T*k (token, slot) assignments by
// expert, then a token-major row gather (Algorithm 2: only the selected
// experts see a token).
//
//   1. chunk histograms      one workgroup per 1024 assignments, LDS counters
//   2. scan                  counts, offsets and each chunk's base per expert
//   3. ranks                 per wavefront, 64 assignments per round: lanes
//                            holding the same expert are found with ballots
//                            over the key bits; rank = lanes below with the
//                            same key; stable because chunks, waves and
//                            rounds follow assignment order
//   4. gather                each token row is read once and written to its
//                            k dispatched rows with 16-byte stores
// Up to 8192 assignments, steps 1-3 run in one workgroup (one launch); up
// to 64 chunks, steps 2 and 3 run in one launch (every rank workgroup
// re-derives the totals and its chunk's bases from the histograms).
#include "common.hpp"
#include "sort_dev.hpp"

namespace decomoe {
namespace {

constexpr int DP_CHUNK = 1024;  // assignments per chunk
constexpr int DP_THREADS = 256;  // 4 wavefronts, 256 assignments each
constexpr int DP_PER_WAVE = DP_CHUNK / (DP_THREADS / kWave);

// zero[0, n_zero) <- 0, mark_val at mark_at: the counters of a launch that
// follows (the expert FFN's), set by the first workgroup
__device__ __forceinline__ void zero_ints(int* zero, int n_zero, int mark_at, int mark_val, int nthr) {
  if (blockIdx.x != 0) return;
  for (int i = threadIdx.x; i < n_zero; i += nthr) zero[i] = i == mark_at ? mark_val : 0;
}

__global__ __launch_bounds__(DP_THREADS) void dispatch_hist_kernel(const int32_t* __restrict__ idx,
                                                                   int A, int E,
                                                                   int32_t* __restrict__ hist, int* zero,
                                                                   int n_zero, int mark_at, int mark_val,
                                                                   const Guard g) {
  if (guard_skip(g)) return;
  zero_ints(zero, n_zero, mark_at, mark_val, DP_THREADS);
  __shared__ int h[1024];
  for (int e = threadIdx.x; e < E; e += DP_THREADS) h[e] = 0;
  __syncthreads();
  const int a0 = blockIdx.x * DP_CHUNK;
  for (int i = threadIdx.x; i < DP_CHUNK; i += DP_THREADS) {
    int a = a0 + i;
    if (a < A) {
      int e = idx[a];
      if (e >= 0 && e < E) atomicAdd(&h[e], 1);
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += DP_THREADS) hist[(size_t)blockIdx.x * E + e] = h[e];
}

// one workgroup of 1024 threads.  Thread (p, e), tid = p E + e, owns expert e
// and the p-th of P = 1024 / E contiguous ranges of chunks: it sums its
// range (16 independent loads in flight), the P partial sums of an expert
// are combined in LDS, the scan over the experts is a wavefront scan plus
// the wavefront totals, and each thread then writes the chunk bases of its
// range.  Every sum runs in chunk order, so the bases are those of a
// sequential scan.
__global__ __launch_bounds__(1024) void dispatch_scan_kernel(const int32_t* __restrict__ hist,
                                                             int n_chunks, int E,
                                                             int32_t* __restrict__ base,
                                                             int32_t* __restrict__ counts,
                                                             int32_t* __restrict__ offsets, const Guard g) {
  if (guard_skip(g)) return;
  __shared__ int s_cnt[1024];          // [p][e] partial sums, then prefixes over p
  __shared__ int s_off[1024];          // [e] exclusive offsets
  __shared__ int part[1024 / kWave];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int P = 1024 / E;              // E <= 1024
  const int p = tid / E, e = tid - p * E;
  const bool mine = p < P;
  const int per = (n_chunks + P - 1) / P;
  const int c0 = min(n_chunks, p * per), c1 = min(n_chunks, c0 + per);
  int cnt = 0;
  if (mine) {
#pragma unroll 16
    for (int c = c0; c < c1; ++c) cnt += hist[(size_t)c * E + e];
    s_cnt[tid] = cnt;
  }
  __syncthreads();
  // threads 0..E-1: the expert totals and the per-range prefixes
  int tot = 0;
  if (tid < E) {
    for (int q = 0; q < P; ++q) {
      const int v = s_cnt[q * E + tid];
      s_cnt[q * E + tid] = tot;
      tot += v;
    }
  }
  int incl = tot;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_up(incl, off, kWave);
    if (lane >= off) incl += y;
  }
  if (lane == kWave - 1) part[wv] = incl;
  __syncthreads();
  if (tid < E) {
    int run = incl - tot;  // exclusive within the wavefront
    for (int w = 0; w < wv; ++w) run += part[w];
    s_off[tid] = run;
    counts[tid] = tot;
    offsets[tid] = run;
    if (tid == E - 1) offsets[E] = run + tot;
  }
  __syncthreads();
  if (mine) {
    int run = s_off[e] + s_cnt[tid];
#pragma unroll 16
    for (int c = c0; c < c1; ++c) {
      const int h = hist[(size_t)c * E + e];
      base[(size_t)c * E + e] = run;
      run += h;
    }
  }
}

// Ranks of one chunk's assignments from its per-wave starting rows `run`
// (stable: waves and rounds follow assignment order).
__device__ __forceinline__ void rank_chunk(const int32_t* __restrict__ idx, int A, int E, int key_bits,
                                           int a_chunk, int (*run)[1024], int32_t* __restrict__ src_of_row,
                                           int32_t* __restrict__ row_of_slot) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int i = 0; i < DP_PER_WAVE; i += kWave) {
    int a = a_chunk + wv * DP_PER_WAVE + i + lane;
    int e = a < A ? idx[a] : -1;
    bool valid = e >= 0 && e < E;
    uint64_t peers = __ballot(valid);
#pragma unroll 1
    for (int b = 0; b < key_bits; ++b) {
      bool bit = (e >> b) & 1;
      uint64_t m = __ballot(bit);
      peers &= bit ? m : ~m;
    }
    if (valid) {
      int r = run[wv][e] + __popcll(peers & lt_mask);
      src_of_row[r] = a;
      row_of_slot[a] = r;
      // the highest lane of the group advances the expert's counter
      if ((63 - __clzll(peers)) == lane) run[wv][e] += __popcll(peers);
    } else if (a < A) {
      row_of_slot[a] = -1;
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// per-wave histograms of one chunk into run[w][e] (zeroed here)
__device__ __forceinline__ void wave_hists(const int32_t* __restrict__ idx, int A, int E, int a_chunk,
                                           int (*run)[1024]) {
  constexpr int NW = DP_THREADS / kWave;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < NW * 1024; i += DP_THREADS) (&run[0][0])[i] = 0;
  __syncthreads();
  for (int i = 0; i < DP_PER_WAVE; i += kWave) {
    int a = a_chunk + wv * DP_PER_WAVE + i + lane;
    if (a < A) {
      int e = idx[a];
      if (e >= 0 && e < E) atomicAdd(&run[wv][e], 1);
    }
  }
}

constexpr int DP_FUSE_CHUNKS = 64;  // scan folded into the ranks up to this many chunks

// Steps 2 and 3 in one launch: workgroup c sums every chunk histogram per
// expert in chunk order (the totals, and the part before chunk c), scans the
// totals over the experts, and ranks chunk c; workgroup 0 also writes counts
// and offsets.  Integer sums: the bases equal those of the scan kernel.
__global__ __launch_bounds__(DP_THREADS) void dispatch_scan_rank_kernel(
    const int32_t* __restrict__ idx, int A, int E, int key_bits, const int32_t* __restrict__ hist,
    int n_chunks, int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ src_of_row, int32_t* __restrict__ row_of_slot, const Guard g) {
  if (guard_skip(g)) return;
  constexpr int NW = DP_THREADS / kWave;
  __shared__ int run[NW][1024];
  __shared__ int s_tot[1024], s_base[1024];
  __shared__ int part[NW];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int chunk = blockIdx.x;
  for (int e = tid; e < E; e += DP_THREADS) {
    int tot = 0, pre = 0;
#pragma unroll 16
    for (int c = 0; c < n_chunks; ++c) {
      const int h = hist[(size_t)c * E + e];
      pre += c < chunk ? h : 0;
      tot += h;
    }
    s_tot[e] = tot;
    s_base[e] = pre;
  }
  wave_hists(idx, A, E, chunk * DP_CHUNK, run);  // its barrier also publishes s_tot
  // exclusive scan of the totals: thread t owns experts 4t .. 4t + 3 (E <= 1024)
  int v[4], sum = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = 4 * tid + j;
    v[j] = e < E ? s_tot[e] : 0;
    sum += v[j];
  }
  int incl = sum;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_up(incl, off, kWave);
    if (lane >= off) incl += y;
  }
  if (lane == kWave - 1) part[wv] = incl;
  __syncthreads();
  int r0 = incl - sum;
  for (int w = 0; w < wv; ++w) r0 += part[w];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = 4 * tid + j;
    if (e < E) {
      if (chunk == 0) {
        counts[e] = v[j];
        offsets[e] = r0;
      }
      s_base[e] += r0;
    }
    r0 += v[j];
  }
  if (chunk == 0 && tid == DP_THREADS - 1) offsets[E] = r0;
  __syncthreads();
  // each wave's starting row per expert
  for (int e = tid; e < E; e += DP_THREADS) {
    int r = s_base[e];
#pragma unroll
    for (int w2 = 0; w2 < NW; ++w2) {
      int c = run[w2][e];
      run[w2][e] = r;
      r += c;
    }
  }
  __syncthreads();
  rank_chunk(idx, A, E, key_bits, chunk * DP_CHUNK, run, src_of_row, row_of_slot);
}

__global__ __launch_bounds__(DP_THREADS) void dispatch_rank_kernel(
    const int32_t* __restrict__ idx, int A, int E, int key_bits, const int32_t* __restrict__ base,
    int32_t* __restrict__ src_of_row, int32_t* __restrict__ row_of_slot, const Guard g) {
  if (guard_skip(g)) return;
  constexpr int NW = DP_THREADS / kWave;
  __shared__ int run[NW][1024];
  const int a_chunk = blockIdx.x * DP_CHUNK;
  wave_hists(idx, A, E, a_chunk, run);
  __syncthreads();
  // turn them into each wave's starting row per expert
  for (int e = threadIdx.x; e < E; e += DP_THREADS) {
    int r = base[(size_t)blockIdx.x * E + e];
#pragma unroll
    for (int w2 = 0; w2 < NW; ++w2) {
      int c = run[w2][e];
      run[w2][e] = r;
      r += c;
    }
  }
  __syncthreads();
  rank_chunk(idx, A, E, key_bits, a_chunk, run, src_of_row, row_of_slot);
}

// ---------------------------------------------------------------------------
// Single-workgroup counting sort for up to DS_MAX assignments (one launch
// instead of histogram + scan + rank): the 16 wavefronts take contiguous
// slices in assignment order, count their slice per expert in LDS, one
// scan turns the counts into offsets and each wavefront's starting row per
// expert, and the wavefronts rank their slices with the ballot scheme
// above.  Same result as the multi-workgroup path (a stable sort).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(DS_THREADS) void dispatch_sort_small_kernel(
    const int32_t* __restrict__ idx, int A, int E, int key_bits, int32_t* __restrict__ counts,
    int32_t* __restrict__ offsets, int32_t* __restrict__ src_of_row,
    int32_t* __restrict__ row_of_slot, int* zero, int n_zero, int mark_at, int mark_val, const Guard g) {
  if (guard_skip(g)) return;
  zero_ints(zero, n_zero, mark_at, mark_val, DS_THREADS);
  __shared__ int wh[DS_WAVES][1024];  // per-wave counts, then per-wave starting rows
  __shared__ int part[DS_WAVES];
  sort_small(idx, A, E, key_bits, &wh[0][0], 1024, part, counts, offsets, src_of_row, row_of_slot);
}

// token-major gather: each token row is read once (VEC-sized vectors, rows
// of `chunks` vectors) and stored to its k dispatched rows.  A block covers
// one token when a row has >= 256 vectors, else `rpb` whole tokens.
template <typename VEC>
__global__ __launch_bounds__(256) void dispatch_gather_kernel(const VEC* __restrict__ x, int T,
                                                              int k, int chunks, int rpb,
                                                              const int32_t* __restrict__ row_of_slot,
                                                              VEC* __restrict__ x_perm, const Guard g) {
  if (guard_skip(g)) return;
  const int A = T * k;
  int t, c0, cstep;
  if (chunks >= 256) {
    t = blockIdx.x;
    c0 = threadIdx.x;
    cstep = 256;
  } else {
    int tl = threadIdx.x / chunks;
    if (tl >= rpb) return;
    t = blockIdx.x * rpb + tl;
    c0 = threadIdx.x % chunks;
    cstep = chunks;
  }
  if (t >= T) return;
  for (int c = c0; c < chunks; c += cstep) {
    VEC v = x[(size_t)t * chunks + c];
    for (int j = 0; j < k; ++j) {
      int r = row_of_slot[(size_t)t * k + j];
      if (r >= 0 && r < A) x_perm[(size_t)r * chunks + c] = v;
    }
  }
}

// Dense-equivalent routing (App. A.3, the convention of a dense batched
// product over every retained expert): slot j of token t is expert j for
// j < K (else dropped, -1), weighted by the routing weight the sparse
// routing gave expert j (0 when it was not selected).
__global__ __launch_bounds__(256) void expand_dense_kernel(const int32_t* __restrict__ idx,
                                                           const float* __restrict__ w, int T, int k,
                                                           int E, const int32_t* __restrict__ K_dev,
                                                           int32_t* __restrict__ idx_dense,
                                                           float* __restrict__ w_dense) {
  const size_t n = (size_t)T * E;
  const int K = K_dev ? clampi(K_dev[0], 0, E) : E;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) {
    const int t = (int)(i / E), j = (int)(i % E);
    float wj = 0.f;
    for (int s = 0; s < k; ++s)
      if (idx[(size_t)t * k + s] == j) wj += w[(size_t)t * k + s];
    idx_dense[i] = j < K ? j : -1;
    w_dense[i] = wj;
  }
}
}  // namespace

size_t dispatch_ws_bytes(int T, int k, int E) {
  size_t A = (size_t)T * k;
  size_t n_chunks = (A + DP_CHUNK - 1) / DP_CHUNK;
  return 2 * n_chunks * (size_t)E * sizeof(int32_t);
}

hipError_t launch_dispatch(const int32_t* idx, int T, int k, int E, const void* x, int elt, int d,
                           int32_t* counts, int32_t* offsets, int32_t* src_of_row,
                           int32_t* row_of_slot, void* x_perm, void* ws, hipStream_t s, Guard g,
                           const ZeroAfter& za) {
  const int A = T * k;
  const int n_chunks = (A + DP_CHUNK - 1) / DP_CHUNK;
  int32_t* hist = static_cast<int32_t*>(ws);
  int32_t* base = hist + (size_t)n_chunks * E;
  int key_bits = 0;
  while ((1 << key_bits) < E) ++key_bits;
  hipError_t err;
  if (A <= DS_MAX) {
    dispatch_sort_small_kernel<<<1, DS_THREADS, 0, s>>>(idx, A, E, key_bits, counts, offsets, src_of_row,
                                                        row_of_slot, za.p, za.n, za.mark_at, za.mark_val, g);
    err = hipGetLastError();
    if (err != hipSuccess || A == 0) return err;
  } else {
    dispatch_hist_kernel<<<n_chunks, DP_THREADS, 0, s>>>(idx, A, E, hist, za.p, za.n, za.mark_at, za.mark_val,
                                                         g);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    if (n_chunks <= DP_FUSE_CHUNKS) {
      dispatch_scan_rank_kernel<<<n_chunks, DP_THREADS, 0, s>>>(idx, A, E, key_bits, hist, n_chunks, counts,
                                                                 offsets, src_of_row, row_of_slot, g);
    } else {
      dispatch_scan_kernel<<<1, 1024, 0, s>>>(hist, n_chunks, E, base, counts, offsets, g);
      err = hipGetLastError();
      if (err != hipSuccess) return err;
      dispatch_rank_kernel<<<n_chunks, DP_THREADS, 0, s>>>(idx, A, E, key_bits, base, src_of_row,
                                                            row_of_slot, g);
    }
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  if (!x) return err;
  const size_t row_bytes = (size_t)d * elt;
  if (row_bytes % 16 == 0) {
    int chunks = (int)(row_bytes / 16);
    int rpb = chunks >= 256 ? 1 : 256 / chunks;
    dispatch_gather_kernel<uint4><<<(T + rpb - 1) / rpb, 256, 0, s>>>(
        static_cast<const uint4*>(x), T, k, chunks, rpb, row_of_slot, static_cast<uint4*>(x_perm), g);
  } else if (row_bytes % 4 == 0) {
    int chunks = (int)(row_bytes / 4);
    int rpb = chunks >= 256 ? 1 : 256 / chunks;
    dispatch_gather_kernel<uint32_t><<<(T + rpb - 1) / rpb, 256, 0, s>>>(
        static_cast<const uint32_t*>(x), T, k, chunks, rpb, row_of_slot, static_cast<uint32_t*>(x_perm), g);
  } else {
    int chunks = (int)(row_bytes / 2);
    int rpb = chunks >= 256 ? 1 : 256 / chunks;
    dispatch_gather_kernel<uint16_t><<<(T + rpb - 1) / rpb, 256, 0, s>>>(
        static_cast<const uint16_t*>(x), T, k, chunks, rpb, row_of_slot, static_cast<uint16_t*>(x_perm), g);
  }
  return hipGetLastError();
}

hipError_t launch_expand_dense(const int32_t* idx, const float* w, int T, int k, int E,
                               const int32_t* K_dev, int32_t* idx_dense, float* w_dense, hipStream_t s) {
  const size_t n = (size_t)T * E;
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  expand_dense_kernel<<<(unsigned)blocks, 256, 0, s>>>(idx, w, T, k, E, K_dev, idx_dense, w_dense);
  return hipGetLastError();
}

}  // namespace decomoe
