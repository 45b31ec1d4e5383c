// Router logits and wavefront Top-k (Eq. 1; Eq. 10; prefix re-route of
// Sec. 3.3 and Algorithm 2).
#include "common.hpp"

#include <float.h>

namespace decomoe {

// ---------------------------------------------------------------------------
// logits[T, E] = x[T, d] W_r[d, E] + b, float32 accumulation.
// Block tile: 32 tokens x 64 experts, k-step 32; 256 threads, each thread
// owns 2 tokens x 4 experts.  x (bf16 or f32) is widened to f32 in LDS.
// ---------------------------------------------------------------------------
namespace {
constexpr int RT_T = 32, RT_E = 64, RT_K = 32;

template <bool XBF16>
__global__ __launch_bounds__(256) void router_logits_kernel(const void* __restrict__ xv,
                                                            const float* __restrict__ w_r,
                                                            const float* __restrict__ bias,
                                                            int T, int d, int E,
                                                            float* __restrict__ logits) {
  __shared__ float xs[RT_K][RT_T + 4];  // transposed: xs[k][token]
  __shared__ float wsm[RT_K][RT_E + 4];
  const int tid = threadIdx.x;
  const int e0 = blockIdx.x * RT_E, t0 = blockIdx.y * RT_T;
  const int tx = tid & 15, ty = tid >> 4;  // experts tx*4.., tokens ty*2..
  float acc[2][4] = {};

  for (int k0 = 0; k0 < d; k0 += RT_K) {
    // x tile: 32 tokens x 32 k = 1024 values, 4 per thread
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int lin = i * 256 + tid;
      int tt = lin >> 5, kk = lin & 31;
      int t = t0 + tt, kg = k0 + kk;
      float v = 0.f;
      if (t < T && kg < d) {
        if constexpr (XBF16)
          v = bf16_to_f32(static_cast<const uint16_t*>(xv)[(size_t)t * d + kg]);
        else
          v = static_cast<const float*>(xv)[(size_t)t * d + kg];
      }
      xs[kk][tt] = v;
    }
    // W tile: 32 k x 64 experts = 2048 values, 8 per thread, coalesced rows
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      int lin = i * 256 + tid;
      int kk = lin >> 6, ee = lin & 63;
      int kg = k0 + kk, e = e0 + ee;
      wsm[kk][ee] = (kg < d && e < E) ? w_r[(size_t)kg * E + e] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < RT_K; ++kk) {
      float2 a = *reinterpret_cast<const float2*>(&xs[kk][ty * 2]);
      float4 b = *reinterpret_cast<const float4*>(&wsm[kk][tx * 4]);
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
    int t = t0 + ty * 2 + i;
    if (t >= T) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int e = e0 + tx * 4 + j;
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
constexpr int TK_MAXC = 16;  // E <= 1024 = 16 values per lane

__device__ __forceinline__ void better(float& v, int& i, float ov, int oi) {
  if (ov > v || (ov == v && oi < i)) { v = ov; i = oi; }
}

__global__ __launch_bounds__(256) void topk_kernel(const float* __restrict__ logits, int T, int E,
                                                   int k, const int32_t* __restrict__ seg_offsets,
                                                   int n_seg, const int32_t* __restrict__ K_dev,
                                                   int32_t* __restrict__ idx, float* __restrict__ w) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;  // whole wavefront leaves together; no block barrier below
  int Klim = E;
  if (K_dev) {
    int s = seg_offsets ? find_segment(seg_offsets, n_seg, t) : 0;
    Klim = clampi(K_dev[s], k, E);
  }
  const float* row = logits + (size_t)t * E;
  float v[TK_MAXC];
  uint32_t alive = 0;
#pragma unroll
  for (int c = 0; c < TK_MAXC; ++c) {
    int e = lane + c * 64;
    v[c] = -FLT_MAX;
    if (e < Klim) { v[c] = row[e]; alive |= 1u << c; }
  }
  float my_v = 0.f;
  int my_i = 0;
  for (int r = 0; r < k; ++r) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int c = 0; c < TK_MAXC; ++c)
      if (alive & (1u << c)) better(bv, bi, v[c], lane + c * 64);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      float ov = __shfl_xor(bv, off, 64);
      int oi = __shfl_xor(bi, off, 64);
      better(bv, bi, ov, oi);
    }
    if (bi < E && (bi & 63) == lane) alive &= ~(1u << (bi >> 6));
    if (lane == r) { my_v = bv; my_i = bi; }
  }
  const float v0 = __shfl(my_v, 0, 64);
  float ex = lane < k ? expf(my_v - v0) : 0.f;
  float sum = ex;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, 64);
  if (lane < k) {
    idx[(size_t)t * k + lane] = my_i;
    w[(size_t)t * k + lane] = ex / sum;
  }
}
}  // namespace

hipError_t launch_router_logits(const void* x, bool x_bf16, const float* w_r, const float* bias,
                                int T, int d, int E, float* logits, hipStream_t s) {
  dim3 grid((E + RT_E - 1) / RT_E, (T + RT_T - 1) / RT_T);
  if (x_bf16)
    router_logits_kernel<true><<<grid, 256, 0, s>>>(x, w_r, bias, T, d, E, logits);
  else
    router_logits_kernel<false><<<grid, 256, 0, s>>>(x, w_r, bias, T, d, E, logits);
  return hipGetLastError();
}

hipError_t launch_topk(const float* logits, int T, int E, int k, const int32_t* seg_offsets,
                       int n_seg, const int32_t* K_dev, int32_t* idx, float* w, hipStream_t s) {
  topk_kernel<<<(T + 3) / 4, 256, 0, s>>>(logits, T, E, k, seg_offsets, n_seg, K_dev, idx, w);
  return hipGetLastError();
}

}  // namespace decomoe
