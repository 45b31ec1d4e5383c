// Router logits and wavefront Top-k (Eq. 1; Eq. 10; prefix re-route of
// Sec. 3.3 and Algorithm 2).
#include "common.hpp"
#include "mass_dev.hpp"
#include "topk_dev.hpp"
#include "sort_dev.hpp"

#include <float.h>

namespace decomoe {

// ---------------------------------------------------------------------------
// logits[T, E] = x[T, d] W_r[d, E] + b on float32 MFMA (v_mfma_f32_16x16x4f32).
// Workgroup tile: 16 tokens x 64 experts; the four wavefronts split the
// d-range into quarters and their partial tiles are added in LDS in the
// fixed order w0 + w1 + w2 + w3 (deterministic).  Within a 32-wide k chunk
// lane l (token l%16, lane group q = l/16) loads 8 consecutive x values and
// MFMA step s consumes k = 8q + s on both operands, so each x row is read
// with one 16-byte (bf16) or two 16-byte (f32) loads per chunk.
// Needs d % 128 == 0 (four quarters of whole chunks).
//
// Split-K (small T, too few tiles to fill the chip): blockIdx.z = c takes the
// d-range [c d/S, (c+1) d/S) and writes its partial tile, without bias, to
// part[c][T][E]; the Top-k kernel adds the S partials in order c = 0..S-1,
// adds the bias and writes the logits.  Needs d % (128 S) == 0.
// ---------------------------------------------------------------------------
namespace {
typedef float f32x4 __attribute__((ext_vector_type(4)));
constexpr int RM_T = 16, RM_E = 64;

template <bool XBF16>
__global__ __launch_bounds__(256) void router_logits_mfma_kernel(const void* __restrict__ xv,
                                                                 const float* __restrict__ w_r,
                                                                 const float* __restrict__ bias,
                                                                 int T, int d, int E,
                                                                 float* __restrict__ logits,
                                                                 float* __restrict__ split_part, const Guard g) {
  if (guard_skip(g)) return;
  __shared__ f32x4 part[4][4][64];  // [wave][n-frag][lane]
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int e0 = blockIdx.x * RM_E, t0 = blockIdx.y * RM_T;
  const int q = lane >> 4, r16 = lane & 15;
  const int t = min(t0 + r16, T - 1);  // padding tokens re-read the last row
  const int dch = d / gridDim.z;       // this split's d-range
  const int quarter = dch >> 2;
  const int kb = blockIdx.z * dch + wv * quarter, ke = kb + quarter;
  int ecol[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) ecol[j] = min(e0 + j * 16 + r16, E - 1);

  f32x4 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = kb; k0 < ke; k0 += 32) {
    const int kk = k0 + 8 * q;
    float xa[8];
    if constexpr (XBF16) {
      const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(xv) + (size_t)t * d + kk);
      const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        xa[2 * i] = __uint_as_float(u[i] << 16);
        xa[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
      }
    } else {
      const float4* src = reinterpret_cast<const float4*>(static_cast<const float*>(xv) + (size_t)t * d + kk);
      const float4 a0 = src[0], a1 = src[1];
      xa[0] = a0.x; xa[1] = a0.y; xa[2] = a0.z; xa[3] = a0.w;
      xa[4] = a1.x; xa[5] = a1.y; xa[6] = a1.z; xa[7] = a1.w;
    }
    float wb[4][8];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int s = 0; s < 8; ++s) wb[j][s] = w_r[(size_t)(kk + s) * E + ecol[j]];
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(xa[s], wb[j][s], acc[j], 0, 0, 0);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) part[wv][j][lane] = acc[j];
  __syncthreads();
  // 4 n-frags x 64 lanes = 256 threads; each adds the four quarters in order
  {
    const int j = threadIdx.x >> 6, l = threadIdx.x & 63;
    f32x4 s = part[0][j][l];
    s += part[1][j][l];
    s += part[2][j][l];
    s += part[3][j][l];
    const int e = e0 + j * 16 + (l & 15);
    if (e < E) {
      if (split_part) {  // partial tile of split blockIdx.z, no bias
        float* dst = split_part + (size_t)blockIdx.z * T * E;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tt = t0 + 4 * (l >> 4) + i;
          if (tt < T) dst[(size_t)tt * E + e] = s[i];
        }
      } else {
        const float b = bias ? bias[e] : 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tt = t0 + 4 * (l >> 4) + i;
          if (tt < T) logits[(size_t)tt * E + e] = s[i] + b;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Fallback for d % 128 != 0: LDS-tiled float32 SIMT kernel, 32 tokens x 64
// experts per workgroup, 2 x 4 outputs per thread.  Loads are clamped to
// valid addresses instead of branched around.
// ---------------------------------------------------------------------------
constexpr int RT_T = 32, RT_E = 64, RT_K = 32;

template <bool XBF16>
__global__ __launch_bounds__(256) void router_logits_simt_kernel(const void* __restrict__ xv,
                                                                 const float* __restrict__ w_r,
                                                                 const float* __restrict__ bias,
                                                                 int T, int d, int E,
                                                                 float* __restrict__ logits, const Guard g) {
  if (guard_skip(g)) return;
  __shared__ float xs[RT_K][RT_T + 4];  // transposed: xs[k][token]
  __shared__ float wsm[RT_K][RT_E + 4];
  const int tid = threadIdx.x;
  const int e0 = blockIdx.x * RT_E, t0 = blockIdx.y * RT_T;
  const int tx = tid & 15, ty = tid >> 4;  // experts tx*4.., tokens ty*2..
  float acc[2][4] = {};

  for (int k0 = 0; k0 < d; k0 += RT_K) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int lin = i * 256 + tid;
      const int tt = lin >> 5, kk = lin & 31;
      const int t = min(t0 + tt, T - 1), kg = min(k0 + kk, d - 1);
      float v;
      if constexpr (XBF16)
        v = bf16_to_f32(static_cast<const uint16_t*>(xv)[(size_t)t * d + kg]);
      else
        v = static_cast<const float*>(xv)[(size_t)t * d + kg];
      xs[kk][tt] = (k0 + kk < d) ? v : 0.f;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int lin = i * 256 + tid;
      const int kk = lin >> 6, ee = lin & 63;
      const int kg = min(k0 + kk, d - 1), e = min(e0 + ee, E - 1);
      const float v = w_r[(size_t)kg * E + e];
      wsm[kk][ee] = (k0 + kk < d) ? v : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < RT_K; ++kk) {
      const float2 a = *reinterpret_cast<const float2*>(&xs[kk][ty * 2]);
      const float4 b = *reinterpret_cast<const float4*>(&wsm[kk][tx * 4]);
      acc[0][0] = fmaf(a.x, b.x, acc[0][0]);
      acc[0][1] = fmaf(a.x, b.y, acc[0][1]);
      acc[0][2] = fmaf(a.x, b.z, acc[0][2]);
      acc[0][3] = fmaf(a.x, b.w, acc[0][3]);
      acc[1][0] = fmaf(a.y, b.x, acc[1][0]);
      acc[1][1] = fmaf(a.y, b.y, acc[1][1]);
      acc[1][2] = fmaf(a.y, b.z, acc[1][2]);
      acc[1][3] = fmaf(a.y, b.w, acc[1][3]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int t = t0 + ty * 2 + i;
    if (t >= T) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = e0 + tx * 4 + j;
      if (e < E) logits[(size_t)t * E + e] = acc[i][j] + (bias ? bias[e] : 0.f);
    }
  }
}

// ---------------------------------------------------------------------------
// Top-k over the first K logits of each token, one wavefront per token.
// Each lane holds experts lane, lane+64, ...; k rounds of a wavefront
// arg-max (value descending, index ascending on ties) pick the slots in
// order.  Weights are the softmax of the k selected logits.
// ---------------------------------------------------------------------------
constexpr int TK_MAXC = 16;  // E <= 1024 = 16 values per lane (MAXC: per instantiation)
constexpr int TK_SPLITS = 8;  // d-range splits whose loads are all issued together

// With `part` (split-K router), the logits are first formed here as
// (part[0] + part[1] + ... + part[S-1]) + b, written to `logits`, and used.
template <int MAXC>  // values per lane: E <= 64 MAXC
__global__ __launch_bounds__(256) void topk_kernel(float* __restrict__ logits, int T, int E,
                                                   int k, const int32_t* __restrict__ seg_offsets,
                                                   int n_seg, const int32_t* __restrict__ K_dev,
                                                   const float* __restrict__ part, int S,
                                                   const float* __restrict__ bias,
                                                   int32_t* __restrict__ idx, float* __restrict__ w, int* __restrict__ ctr_zero, const Guard g) {
  if (guard_skip(g)) return;
  if (ctr_zero && blockIdx.x == 0 && threadIdx.x == 0) *ctr_zero = 0;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;  // whole wavefront leaves together; no block barrier below
  int Klim = E;
  if (K_dev) {
    int s = seg_offsets ? find_segment(seg_offsets, n_seg, t) : 0;
    Klim = clampi(K_dev[s], k, E);
  }
  float* row = logits + (size_t)t * E;
  if (part) {
    // the logits are selected from registers (no reload of the stored row):
    // (part[0] + part[1] + ... + part[S-1]) + b per expert
    float v[MAXC];
    if (MAXC <= 2 && S <= TK_SPLITS) {
      // every partial's load in flight before the first addition
      float pv[TK_SPLITS][MAXC];
#pragma unroll
      for (int sp = 0; sp < TK_SPLITS; ++sp)
#pragma unroll
        for (int c = 0; c < MAXC; ++c) {
          const int e = lane + c * 64;
          pv[sp][c] = sp < S && e < E ? part[((size_t)sp * T + t) * E + e] : 0.f;
        }
#pragma unroll
      for (int c = 0; c < MAXC; ++c) {
        float a = pv[0][c];
#pragma unroll
        for (int sp = 1; sp < TK_SPLITS; ++sp)
          if (sp < S) a += pv[sp][c];
        v[c] = a;
      }
    } else {
#pragma unroll
      for (int c = 0; c < MAXC; ++c) {
        const int e = lane + c * 64;
        float a = e < E ? part[(size_t)t * E + e] : 0.f;
        // partials in order sp = 1..S-1; loads issued four at a time
        for (int sp = 1; sp < S; sp += 4) {
          float pv[4];
#pragma unroll
          for (int u = 0; u < 4; ++u)
            pv[u] = sp + u < S && e < E ? part[((size_t)(sp + u) * T + t) * E + e] : 0.f;
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (sp + u < S) a += pv[u];
        }
        v[c] = a;
      }
    }
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      const int e = lane + c * 64;
      if (e < E) {
        v[c] += bias ? bias[e] : 0.f;
        row[e] = v[c];
      } else {
        v[c] = 0.f;
      }
    }
    topk_select_vals<MAXC>(v, E, k, Klim, lane, idx + (size_t)t * k, w + (size_t)t * k);
    return;
  }
  topk_select<MAXC>(row, E, k, Klim, lane, idx + (size_t)t * k, w + (size_t)t * k);
}

// ---------------------------------------------------------------------------
// Top-k for E <= 16 MAXC (MAXC 8 or 16): four tokens per wavefront, one row
// of 16 lanes per token.  Lane j of a row holds experts j, j + 16, ...; a
// round's arg-max is a lane-local scan plus four DPP moves inside the row
// (quad swaps, half-row and row mirrors), so the 16 lanes end with the
// row's best pair and no value leaves the row.  Round r's winner is kept by
// lane r % 16 in slot r / 16 (k <= 32).  Same selection order, tie rule and
// weights as topk_kernel.
// ---------------------------------------------------------------------------

template <int MAXC>
__global__ __launch_bounds__(256) void topk_row_kernel(float* __restrict__ logits, int T, int E,
                                                       int k, const int32_t* __restrict__ seg_offsets,
                                                       int n_seg, const int32_t* __restrict__ K_dev,
                                                       const float* __restrict__ part, int S,
                                                       const float* __restrict__ bias,
                                                       int32_t* __restrict__ idx, float* __restrict__ w, int* __restrict__ ctr_zero, const Guard g) {
  if (guard_skip(g)) return;
  if (ctr_zero && blockIdx.x == 0 && threadIdx.x == 0) *ctr_zero = 0;
  const int j = threadIdx.x & 15;
  const int t = blockIdx.x * 16 + (threadIdx.x >> 4);
  if (t >= T) return;  // the whole row of 16 lanes leaves together
  int Klim = E;
  if (K_dev) {
    const int sg = seg_offsets ? find_segment(seg_offsets, n_seg, t) : 0;
    Klim = clampi(K_dev[sg], k, E);
  }
  float* row = logits + (size_t)t * E;
  float v[MAXC];
  if (part) {
    // partials in order sp = 0..S-1, then the bias; every load of a lane
    // is issued before the additions
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      const int e = j + 16 * c;
      v[c] = e < E ? part[(size_t)t * E + e] : 0.f;
    }
    for (int sp = 1; sp < S; sp += 4) {  // four partials' loads in flight together
      float pv[4][MAXC];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int c = 0; c < MAXC; ++c) {
          const int e = j + 16 * c;
          pv[u][c] = (sp + u < S && e < E) ? part[((size_t)(sp + u) * T + t) * E + e] : 0.f;
        }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (sp + u < S) {
#pragma unroll
          for (int c = 0; c < MAXC; ++c) v[c] += pv[u][c];
        }
    }
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      const int e = j + 16 * c;
      if (e < E) {
        v[c] += bias ? bias[e] : 0.f;
        row[e] = v[c];
      }
    }
  } else {
#pragma unroll
    for (int c = 0; c < MAXC; ++c) {
      const int e = j + 16 * c;
      v[c] = e < E ? row[e] : 0.f;
    }
  }
  row_topk_select<MAXC>(v, j, E, k, Klim, idx + (size_t)t * k, w + (size_t)t * k);
}
// ---------------------------------------------------------------------------
// Calibration and prefix re-route of one invocation in one launch (Eqs. 11,
// 12, then the re-route of Sec. 3.3).  Every workgroup forms the masses and
// K itself -- the same float64 sums as segment_mass_kernel (mass_sorted,
// prefix_K), over at most CAL_STAGE routing entries -- so no second launch
// waits for one workgroup's result; workgroup 0 writes mass and K.  Then
// workgroup b re-routes the tokens 16 b .. 16 b + 15 (stride 16 x grid)
// inside [0, K) with the selection of topk_kernel: for k <= 16 and E <= 16
// RMAXC one row of 16 lanes per token in wavefronts 0-3 (row_topk_select,
// bitwise the same slots and weights), else one wavefront per token
// (topk_select).
//
// With `ctr` (a counter that the Top-k launch before this one zeroed), the
// re-routed entries are also grouped by expert (Algorithm 2's dispatch,
// x = NULL): every workgroup publishes its entries and counts itself done;
// the last one to finish sorts all T k entries (sort_small), so no launch
// follows for the grouping.  It then also writes the n_zero ints at `zero`
// (0, and mark_val at index mark_at): the expert FFN's counter header in the
// same workspace, which the call that follows would otherwise clear with a
// launch of its own.
// ---------------------------------------------------------------------------
template <int MAXC, int RMAXC>
__global__ __launch_bounds__(CAL_THREADS) void calibrate_route_kernel(
    const float* __restrict__ logits, const int32_t* __restrict__ idx_full,
    const float* __restrict__ w_full, int T, int E, int k, int key_bits, double p,
    double* __restrict__ mass, int32_t* __restrict__ K_out, int32_t* __restrict__ idx,
    float* __restrict__ w, int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ src_of_row, int32_t* __restrict__ row_of_slot, int* __restrict__ ctr,
    int* __restrict__ zero, int n_zero, int mark_at, int mark_val, const Guard g) {
  static_assert(CAL_THREADS == DS_THREADS && CAL_WAVES == DS_WAVES, "the grouping runs on this workgroup");
  if (guard_skip(g)) return;
  __shared__ CalLds L;
  __shared__ int s_last;
  const double a = mass_sorted(idx_full, w_full, 0, T * k, E, key_bits, L);
  const int K = prefix_K(E, k, p, L);
  const int tid = threadIdx.x;
  if (blockIdx.x == 0) {
    if (tid < E) mass[tid] = a;
    if (tid == 0) K_out[0] = K;
  }
  const int Klim = clampi(K, k, E);
  constexpr int RM = RMAXC > 0 ? RMAXC : 1;
  if (RMAXC > 0 && k <= 16 && E <= 16 * RMAXC) {
    if (tid < 256) {
      const int j = tid & 15;
      for (int t = blockIdx.x * 16 + (tid >> 4); t < T; t += gridDim.x * 16) {
        const float* row = logits + (size_t)t * E;
        float v[RM];
#pragma unroll
        for (int c = 0; c < RM; ++c) {
          const int e = j + 16 * c;
          v[c] = e < Klim ? row[e] : 0.f;
        }
        row_topk_select<RM>(v, j, E, k, Klim, idx + (size_t)t * k, w + (size_t)t * k);
      }
    }
  } else {
    const int lane = tid & 63;
    for (int t = blockIdx.x * CAL_WAVES + (tid >> 6); t < T; t += gridDim.x * CAL_WAVES)
      topk_select<MAXC>(logits + (size_t)t * E, E, k, Klim, lane, idx + (size_t)t * k, w + (size_t)t * k);
  }
  if (!ctr) return;
  // every wavefront's entries have reached the cache (vmcnt 0) before the
  // barrier; then one thread per workgroup makes them visible device-wide
  // (release fence) and counts the workgroup done; the last one acquires
  // every workgroup's entries for the sort
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0) (gfx9 encoding; expcnt, lgkmcnt not waited)
  __syncthreads();
  if (tid == 0) {
    __threadfence();
    const bool last = __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                      (int)gridDim.x - 1;
    if (last) __threadfence();
    s_last = last;
  }
  __syncthreads();
  if (!s_last) return;
  sort_small(idx, T * k, E, key_bits, reinterpret_cast<int*>(L.table), E, L.part, counts, offsets, src_of_row,
             row_of_slot);
  // every other workgroup is done with the workspace
  for (int i = tid; i < n_zero; i += CAL_THREADS) zero[i] = i == mark_at ? mark_val : 0;
}

}  // namespace

bool calibrate_route_fused(int T, int E, int k) {
  return T >= 1 && (size_t)T * k <= (size_t)CAL_STAGE && E <= CAL_SORT_E;
}

hipError_t launch_calibrate_route(const float* logits, const int32_t* idx_full, const float* w_full,
                                  int T, int E, int k, double p, double* mass, int32_t* K_out,
                                  int32_t* idx, float* w, hipStream_t s, Guard g, const SortOut* sort) {
  if (!calibrate_route_fused(T, E, k)) {
    if (sort) return hipErrorInvalidValue;  // the grouping needs the one-launch path
    hipError_t err = launch_calibrate(idx_full, w_full, T, E, k, nullptr, 1, p, mass, K_out, nullptr,
                                      nullptr, s, g);
    if (err != hipSuccess || T == 0) return err;
    // logits are only read when the router is not run (x = NULL)
    return launch_route(nullptr, false, nullptr, nullptr, nullptr, T, 0, E, k, nullptr, 1, K_out,
                        const_cast<float*>(logits), idx, w, nullptr, s, g);
  }
  int key_bits = 0;
  while ((1 << key_bits) < E) ++key_bits;
  const unsigned grid = (unsigned)((T + 15) / 16);
  const SortOut so = sort ? *sort : SortOut{};
#define CAL_ROUTE_ARGS                                                                                      \
  logits, idx_full, w_full, T, E, k, key_bits, p, mass, K_out, idx, w, so.counts, so.offsets, so.src_of_row, \
      so.row_of_slot, so.ctr, so.zero, so.n_zero, so.mark_at, so.mark_val, g
  if (E <= 128)
    calibrate_route_kernel<2, 8><<<grid, CAL_THREADS, 0, s>>>(CAL_ROUTE_ARGS);
  else if (E <= 256)
    calibrate_route_kernel<4, 16><<<grid, CAL_THREADS, 0, s>>>(CAL_ROUTE_ARGS);
  else
    calibrate_route_kernel<8, 0><<<grid, CAL_THREADS, 0, s>>>(CAL_ROUTE_ARGS);
#undef CAL_ROUTE_ARGS
  return hipGetLastError();
}

bool route_rcep_fused(int T, int E, int k) {
  return calibrate_route_fused(T, E, k) && (size_t)T * k <= (size_t)DS_MAX && E <= DS_THREADS;
}

size_t route_rcep_ws_bytes(int T, int d, int E, int k) {
  if (!route_rcep_fused(T, E, k)) {
    const size_t a = route_x3_ws_bytes(T, d, E), b = dispatch_ws_bytes(T, k, E);
    return a > b ? a : b;
  }
  return (route_x3_ws_bytes(T, d, E) + 255) / 256 * 256 + 256;  // + the completion counter
}

hipError_t launch_route_rcep(const void* x, const void* w_r_packed, const float* bias, int T, int d, int E,
                             int k, double p, float* logits, int32_t* idx_full, float* w_full, double* mass,
                             int32_t* K_out, int32_t* idx, float* w, int32_t* counts, int32_t* offsets,
                             int32_t* src_of_row, int32_t* row_of_slot, void* ws, hipStream_t s, Guard g,
                             const ZeroAfter& za) {
  if (!route_rcep_fused(T, E, k)) {
    if (za.n) return hipErrorInvalidValue;  // only the one-launch grouping writes it
    hipError_t err = launch_route(x, true, nullptr, w_r_packed, bias, T, d, E, k, nullptr, 1, nullptr, logits,
                                  idx_full, w_full, ws, s, g);
    if (err == hipSuccess)
      err = launch_calibrate_route(logits, idx_full, w_full, T, E, k, p, mass, K_out, idx, w, s, g);
    if (err == hipSuccess)
      err = launch_dispatch(idx, T, k, E, nullptr, 2, 0, counts, offsets, src_of_row, row_of_slot, nullptr, ws,
                            s, g);
    return err;
  }
  // the counter sits past the router's partial sums (which the Top-k launch
  // reads while its first workgroup zeroes the counter)
  int* ctr = reinterpret_cast<int*>(static_cast<char*>(ws) + (route_x3_ws_bytes(T, d, E) + 255) / 256 * 256);
  hipError_t err = launch_route(x, true, nullptr, w_r_packed, bias, T, d, E, k, nullptr, 1, nullptr, logits,
                                idx_full, w_full, ws, s, g, ctr);
  if (err != hipSuccess) return err;
  const SortOut so{counts, offsets, src_of_row, row_of_slot, ctr, za.p, za.n, za.mark_at, za.mark_val};
  return launch_calibrate_route(logits, idx_full, w_full, T, E, k, p, mass, K_out, idx, w, s, g, &so);
}

hipError_t launch_route_rcep_chained(const void* y_prev, const int32_t* row_prev, const float* w_prev, void* h,
                                     const void* w_r_packed, const float* bias, int T, int d, int E, int k,
                                     double p, float* logits, int32_t* idx_full, float* w_full, double* mass,
                                     int32_t* K_out, int32_t* idx, float* w, int32_t* counts, int32_t* offsets,
                                     int32_t* src_of_row, int32_t* row_of_slot, void* ws, hipStream_t s, Guard g,
                                     const ZeroAfter& za) {
  if (y_prev && combine_router_fits(T, d, E, k) && route_rcep_fused(T, E, k)) {
    // the previous combine inside the router launch, then the Top-k (which
    // zeroes the grouping's counter) and the one-launch calibration
    int* ctr = reinterpret_cast<int*>(static_cast<char*>(ws) + (route_x3_ws_bytes(T, d, E) + 255) / 256 * 256);
    float* part = nullptr;
    int S = 1;
    hipError_t err = launch_combine_router_x3(y_prev, row_prev, w_prev, k, h, w_r_packed, bias, T, d, E, logits, ws,
                                              part, S, s, g);
    if (err == hipSuccess)
      err = launch_topk(logits, T, E, k, nullptr, 1, nullptr, part, S, bias, idx_full, w_full, s, g, ctr);
    if (err != hipSuccess) return err;
    const SortOut so{counts, offsets, src_of_row, row_of_slot, ctr, za.p, za.n, za.mark_at, za.mark_val};
    return launch_calibrate_route(logits, idx_full, w_full, T, E, k, p, mass, K_out, idx, w, s, g, &so);
  }
  if (y_prev) {  // the combine on its own, then the routing of the new rows
    hipError_t err = launch_combine(y_prev, true, row_prev, w_prev, T, k, d, h, h, s, g);
    if (err != hipSuccess) return err;
  }
  return launch_route_rcep(h, w_r_packed, bias, T, d, E, k, p, logits, idx_full, w_full, mass, K_out, idx, w,
                           counts, offsets, src_of_row, row_of_slot, ws, s, g, za);
}

// Split factor of the router's d-range: enough workgroups to cover the chip
// (about 512), in whole 128-wide quarters of d.  1 = no split.
int router_splits(int T, int d, int E) {
  if (d % 128 != 0) return 1;
  const int tiles = ((E + RM_E - 1) / RM_E) * ((T + RM_T - 1) / RM_T);
  int S = 1;
  while (tiles * S < 512 && d % (128 * 2 * S) == 0) S *= 2;
  return S;
}

size_t route_ws_bytes(int T, int d, int E) {
  const int S = router_splits(T, d, E);
  return S > 1 ? (size_t)S * T * E * sizeof(float) : 0;
}

hipError_t launch_route(const void* x, bool x_bf16, const float* w_r, const void* w_r_packed,
                        const float* bias, int T, int d, int E, int k, const int32_t* seg_offsets,
                        int n_seg, const int32_t* K_dev, float* logits, int32_t* idx, float* w,
                        void* ws, hipStream_t s, Guard g, int* ctr_zero) {
  float* part = nullptr;
  int S = 1;
  if (x && w_r_packed) {
    hipError_t err = launch_router_x3(x, w_r_packed, bias, T, d, E, logits, ws, part, S, s, g);
    if (err != hipSuccess) return err;
  } else if (x) {
    if (d % 128 == 0) {
      S = router_splits(T, d, E);
      if (S > 1) part = static_cast<float*>(ws);
      dim3 grid((E + RM_E - 1) / RM_E, (T + RM_T - 1) / RM_T, S);
      if (x_bf16)
        router_logits_mfma_kernel<true><<<grid, 256, 0, s>>>(x, w_r, bias, T, d, E, logits, part, g);
      else
        router_logits_mfma_kernel<false><<<grid, 256, 0, s>>>(x, w_r, bias, T, d, E, logits, part, g);
    } else {
      dim3 grid((E + RT_E - 1) / RT_E, (T + RT_T - 1) / RT_T);
      if (x_bf16)
        router_logits_simt_kernel<true><<<grid, 256, 0, s>>>(x, w_r, bias, T, d, E, logits, g);
      else
        router_logits_simt_kernel<false><<<grid, 256, 0, s>>>(x, w_r, bias, T, d, E, logits, g);
    }
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  return launch_topk(logits, T, E, k, seg_offsets, n_seg, K_dev, part, S, bias, idx, w, s, g, ctr_zero);
}

hipError_t launch_topk(float* logits, int T, int E, int k, const int32_t* seg_offsets, int n_seg,
                       const int32_t* K_dev, const float* part, int S, const float* bias, int32_t* idx, float* w,
                       hipStream_t s, Guard g, int* ctr_zero) {
  // many tokens: four per wavefront (fewer instructions per token); few
  // tokens: one per wavefront (more independent wavefronts, shorter chains).
  // Router + Top-k, measured (E 128, k 8): four per wavefront from 4096
  // tokens on (21.5 against 22.1 us; 8192: 29.2 against 33.1), one below
  // (512: 14.2 against 14.5; 64: 14.4 against 15.2)
  const int blocks = (T + 3) / 4, rblocks = (T + 15) / 16;
  const bool rows = T >= 4096;
  if (E <= 128 && rows)
    topk_row_kernel<8><<<rblocks, 256, 0, s>>>(logits, T, E, k, seg_offsets, n_seg, K_dev, part, S, bias, idx, w, ctr_zero, g);
  else if (E <= 128)
    topk_kernel<2><<<blocks, 256, 0, s>>>(logits, T, E, k, seg_offsets, n_seg, K_dev, part, S, bias, idx, w, ctr_zero, g);
  else if (E <= 256 && rows)
    topk_row_kernel<16><<<rblocks, 256, 0, s>>>(logits, T, E, k, seg_offsets, n_seg, K_dev, part, S, bias, idx, w, ctr_zero, g);
  else if (E <= 256)
    topk_kernel<4><<<blocks, 256, 0, s>>>(logits, T, E, k, seg_offsets, n_seg, K_dev, part, S, bias, idx, w, ctr_zero, g);
  else
    topk_kernel<TK_MAXC><<<blocks, 256, 0, s>>>(logits, T, E, k, seg_offsets, n_seg, K_dev, part, S, bias,
                                                idx, w, ctr_zero, g);
  return hipGetLastError();
}

}  // namespace decomoe
