// SAVB exit gate (Sec. 3.2, Eqs. 2 and 3) and the flag-driven visual-block
// removal.
//
//   pool     the n - 1 preceding text rows are summed per column in float32,
//            rows split over blockIdx.y (each split sums its rows in order)
//   feature  x = [sum / (n - 1); row n - 1] (the splits added in order,
//            then one scaling), one column per thread
//   hidden   every workgroup loads x into LDS and each wavefront forms one
//            hidden unit relu(W1[u] . x + b1[u])
//   decide   one workgroup: the two class logits, p_exit = softmax(z)_1 and
//            the exit flag p_exit >= theta (compared in float64)
// Every sum has a fixed order, so the gate is deterministic.
#include "common.hpp"

namespace decomoe {
namespace {

constexpr int SG_ROWS = 32;  // rows per pooling split until there are 16 splits

int savb_splits(int n) {
  const int rows = n - 1;
  if (rows <= 0) return 0;
  int s = (rows + SG_ROWS - 1) / SG_ROWS;
  return s > 16 ? 16 : s;
}

// partial[s][c] = sum of rows [s*per, (s+1)*per) of column c (rows < n - 1)
template <bool BF16>
__global__ __launch_bounds__(256) void savb_pool_kernel(const void* __restrict__ rows, int n, int d,
                                                        int per, float* __restrict__ partial, const Guard g) {
  if (guard_skip(g)) return;
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= d) return;
  const int r0 = blockIdx.y * per, r1 = min(n - 1, r0 + per);
  float acc = 0.f;
  int r = r0;
  for (; r + 8 <= r1; r += 8) {  // eight loads in flight, added in row order
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      v[u] = BF16 ? bf16_to_f32(static_cast<const uint16_t*>(rows)[(size_t)(r + u) * d + c])
                  : static_cast<const float*>(rows)[(size_t)(r + u) * d + c];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
  }
  for (; r < r1; ++r)
    acc += BF16 ? bf16_to_f32(static_cast<const uint16_t*>(rows)[(size_t)r * d + c])
                : static_cast<const float*>(rows)[(size_t)r * d + c];
  partial[(size_t)blockIdx.y * d + c] = acc;
}

// x[c] = (sum of the splits' partials, in split order) / (n - 1) and
// x[d + c] = text row n - 1, one column per thread; the partial loads of a
// column are all issued before the additions
template <bool BF16>
__global__ __launch_bounds__(256) void savb_feature_kernel(const void* __restrict__ rows, int n, int d,
                                                           int splits, const float* __restrict__ partial,
                                                           float* __restrict__ x, const Guard g) {
  if (guard_skip(g)) return;
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= d) return;
  float v[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) v[q] = q < splits ? partial[(size_t)q * d + c] : 0.f;
  float s = 0.f;
#pragma unroll
  for (int q = 0; q < 16; ++q)
    if (q < splits) s += v[q];
  x[c] = n > 1 ? s * (1.f / static_cast<float>(n - 1)) : 0.f;
  x[d + c] = BF16 ? bf16_to_f32(static_cast<const uint16_t*>(rows)[(size_t)(n - 1) * d + c])
                  : static_cast<const float*>(rows)[(size_t)(n - 1) * d + c];
}

// x into LDS, then wavefront w of block b computes hidden unit 4 b + w
__global__ __launch_bounds__(256) void savb_hidden_kernel(const float* __restrict__ x, int d,
                                                          const float* __restrict__ w1,
                                                          const float* __restrict__ b1, int hid,
                                                          float* __restrict__ hidden, const Guard g) {
  if (guard_skip(g)) return;
  extern __shared__ float xs[];  // [2d]
  for (int c = threadIdx.x; c < 2 * d; c += 256) xs[c] = x[c];
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int u = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (u >= hid) return;
  const float* wr = w1 + (size_t)u * 2 * d;
  float acc = 0.f;
  if ((d & 127) == 0 && (reinterpret_cast<uintptr_t>(wr) & 15) == 0) {
    // 16-byte loads, eight in flight per lane: lane l takes columns
    // 4 (l + 64 j) .. + 4 for j = 0, 1, ...
    const float4* w4 = reinterpret_cast<const float4*>(wr);
    const int n4 = (2 * d) >> 2;
    for (int j0 = lane; j0 < n4; j0 += 64 * 8) {
      float4 v[8];
#pragma unroll
      for (int u8 = 0; u8 < 8; ++u8) v[u8] = j0 + 64 * u8 < n4 ? w4[j0 + 64 * u8] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int u8 = 0; u8 < 8; ++u8) {
        const int c = 4 * (j0 + 64 * u8);
        if (j0 + 64 * u8 < n4) {
          acc = fmaf(v[u8].x, xs[c], acc);
          acc = fmaf(v[u8].y, xs[c + 1], acc);
          acc = fmaf(v[u8].z, xs[c + 2], acc);
          acc = fmaf(v[u8].w, xs[c + 3], acc);
        }
      }
    }
  } else {
    for (int c = lane; c < 2 * d; c += 64) acc = fmaf(wr[c], xs[c], acc);
  }
  // lanes in order: the sum of lane partials is formed by lane 0
  for (int off = 32; off >= 1; off >>= 1) acc += __shfl_down(acc, off, 64);
  if (lane == 0) hidden[u] = fmaxf(acc + (b1 ? b1[u] : 0.f), 0.f);
}

// two wavefronts: class c = wavefront c; then thread 0 decides
__global__ __launch_bounds__(128) void savb_decide_kernel(const float* __restrict__ hidden, int hid,
                                                          const float* __restrict__ w2,
                                                          const float* __restrict__ b2, double theta,
                                                          float* __restrict__ p_exit,
                                                          int32_t* __restrict__ exit_flag,
                                                          int32_t* __restrict__ exit_layer, int layer,
                                                          const Guard g) {
  if (guard_skip(g)) return;
  __shared__ float z[2];
  const int lane = threadIdx.x & 63, cls = threadIdx.x >> 6;
  float acc = 0.f;
  for (int u = lane; u < hid; u += 64) acc = fmaf(w2[(size_t)cls * hid + u], hidden[u], acc);
  for (int off = 32; off >= 1; off >>= 1) acc += __shfl_down(acc, off, 64);
  if (lane == 0) z[cls] = acc + (b2 ? b2[cls] : 0.f);
  __syncthreads();
  if (threadIdx.x == 0) {
    const float mx = fmaxf(z[0], z[1]);
    const float e0 = expf(z[0] - mx), e1 = expf(z[1] - mx);
    const float p = e1 / (e0 + e1);
    *p_exit = p;
    const bool fire = static_cast<double>(p) >= theta;
    *exit_flag = fire ? 1 : 0;
    if (fire && exit_layer) *exit_layer = layer;  // the exit layer of a predicated gate
  }
}

// the rows outside [v0, v1) when *flag != 0; nothing otherwise
template <typename VEC>
__global__ __launch_bounds__(256) void drop_rows_if_kernel(const VEC* __restrict__ h, int rows_out,
                                                           int chunks, int v0, int nv,
                                                           const int32_t* __restrict__ flag,
                                                           VEC* __restrict__ out) {
  if (*flag == 0) return;
  const size_t n = (size_t)rows_out * chunks;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) {
    const int r = (int)(i / chunks), c = (int)(i % chunks);
    const int src = r < v0 ? r : r + nv;
    out[i] = h[(size_t)src * chunks + c];
  }
}
template <typename VEC>
hipError_t drop_if_launch(const void* h, int rows_out, int chunks, int v0, int nv, const int32_t* flag,
                          void* out, hipStream_t s) {
  const size_t n = (size_t)rows_out * chunks;
  size_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  drop_rows_if_kernel<VEC><<<(unsigned)blocks, 256, 0, s>>>(static_cast<const VEC*>(h), rows_out, chunks,
                                                             v0, nv, flag, static_cast<VEC*>(out));
  return hipGetLastError();
}
}  // namespace

size_t savb_ws_bytes(int n, int d, int hid) {
  const int splits = savb_splits(n);
  return ((size_t)splits * d + (size_t)hid + (size_t)2 * d) * sizeof(float);
}

hipError_t launch_savb_gate(const void* rows, bool bf16, int n, int d, const float* w1,
                            const float* b1, int hid, const float* w2, const float* b2, double theta,
                            float* feature, float* p_exit, int32_t* exit_flag, void* ws,
                            hipStream_t s, Guard g, int32_t* exit_layer, int layer) {
  const int splits = savb_splits(n);
  float* partial = static_cast<float*>(ws);
  float* hidden = partial + (size_t)splits * d;
  if (splits > 0) {
    const dim3 grid((d + 255) / 256, splits);
    const int per = (n - 1 + splits - 1) / splits;  // rows per split (splits * per >= n - 1)
    if (bf16)
      savb_pool_kernel<true><<<grid, 256, 0, s>>>(rows, n, d, per, partial, g);
    else
      savb_pool_kernel<false><<<grid, 256, 0, s>>>(rows, n, d, per, partial, g);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  float* x = hidden + hid;  // the feature (also the caller's copy when given)
  if (feature) x = feature;
  const unsigned fb = (unsigned)((d + 255) / 256);
  if (bf16)
    savb_feature_kernel<true><<<fb, 256, 0, s>>>(rows, n, d, splits, partial, x, g);
  else
    savb_feature_kernel<false><<<fb, 256, 0, s>>>(rows, n, d, splits, partial, x, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned hb = (unsigned)((hid + 3) / 4);
  const size_t lds = (size_t)2 * d * sizeof(float);
  savb_hidden_kernel<<<hb, 256, lds, s>>>(x, d, w1, b1, hid, hidden, g);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  savb_decide_kernel<<<1, 128, 0, s>>>(hidden, hid, w2, b2, theta, p_exit, exit_flag, exit_layer, layer, g);
  return hipGetLastError();
}

hipError_t launch_drop_rows_if(const void* h, int elt, int S, int d, int v0, int v1,
                               const int32_t* flag, void* out, hipStream_t s) {
  const int rows_out = S - (v1 - v0), nv = v1 - v0;
  const size_t row_bytes = (size_t)d * elt;
  const uintptr_t al = reinterpret_cast<uintptr_t>(h) | reinterpret_cast<uintptr_t>(out);
  if (row_bytes % 16 == 0 && al % 16 == 0)
    return drop_if_launch<uint4>(h, rows_out, (int)(row_bytes / 16), v0, nv, flag, out, s);
  if (row_bytes % 4 == 0 && al % 4 == 0)
    return drop_if_launch<uint32_t>(h, rows_out, (int)(row_bytes / 4), v0, nv, flag, out, s);
  return drop_if_launch<uint16_t>(h, rows_out, (int)(row_bytes / 2), v0, nv, flag, out, s);
}

}  // namespace decomoe
