// Weighted combine back to token order (Algorithm 2) and the SAVB
// visual-block row compaction (Sec. 3.2; Algorithm 2).
#include "common.hpp"

namespace decomoe {
namespace {

// out[t] = sum_j w[t, j] * y[row_of_slot[t*k + j]], float32 accumulation in
// slot order.  Each thread owns one 16-byte vector of the row (8 bf16 or 4
// f32); a block covers one token row, or several when rows are short.
template <bool BF16>
__global__ __launch_bounds__(256) void combine_kernel(const uint4* __restrict__ y,
                                                      const int32_t* __restrict__ row_of_slot,
                                                      const float* __restrict__ w, int T, int k,
                                                      int chunks, int rpb, uint4* __restrict__ out) {
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
  const int A = T * k;
  for (int c = c0; c < chunks; c += cstep) {
    float acc[8] = {};
    for (int j = 0; j < k; ++j) {
      const int r = row_of_slot[(size_t)t * k + j];
      if (r < 0 || r >= A) continue;
      const float wj = w[(size_t)t * k + j];
      const uint4 v = y[(size_t)r * chunks + c];
      if constexpr (BF16) {
        const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[2 * q] = fmaf(wj, __uint_as_float(u[q] << 16), acc[2 * q]);
          acc[2 * q + 1] = fmaf(wj, __uint_as_float(u[q] & 0xffff0000u), acc[2 * q + 1]);
        }
      } else {
        acc[0] = fmaf(wj, __uint_as_float(v.x), acc[0]);
        acc[1] = fmaf(wj, __uint_as_float(v.y), acc[1]);
        acc[2] = fmaf(wj, __uint_as_float(v.z), acc[2]);
        acc[3] = fmaf(wj, __uint_as_float(v.w), acc[3]);
      }
    }
    uint4 o;
    if constexpr (BF16) {
      o = make_uint4(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
                     pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7]));
    } else {
      o = make_uint4(__float_as_uint(acc[0]), __float_as_uint(acc[1]), __float_as_uint(acc[2]),
                     __float_as_uint(acc[3]));
    }
    out[(size_t)t * chunks + c] = o;
  }
}

// element-wise fallback when rows are not whole 16-byte vectors
template <bool BF16>
__global__ __launch_bounds__(256) void combine_scalar_kernel(const void* __restrict__ yv,
                                                             const int32_t* __restrict__ row_of_slot,
                                                             const float* __restrict__ w, int T,
                                                             int k, int d, void* __restrict__ outv) {
  const size_t n = (size_t)T * d;
  const int A = T * k;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) {
    const int t = (int)(i / d), c = (int)(i % d);
    float acc = 0.f;
    for (int j = 0; j < k; ++j) {
      const int r = row_of_slot[(size_t)t * k + j];
      if (r < 0 || r >= A) continue;
      float yv_ = BF16 ? bf16_to_f32(static_cast<const uint16_t*>(yv)[(size_t)r * d + c])
                       : static_cast<const float*>(yv)[(size_t)r * d + c];
      acc = fmaf(w[(size_t)t * k + j], yv_, acc);
    }
    if (BF16)
      static_cast<uint16_t*>(outv)[i] = f32_to_bf16(acc);
    else
      static_cast<float*>(outv)[i] = acc;
  }
}

// out row r = h row (r < v0 ? r : r + (v1 - v0)), copied as VEC vectors
template <typename VEC>
__global__ __launch_bounds__(256) void drop_rows_kernel(const VEC* __restrict__ h, int rows_out,
                                                        int chunks, int v0, int nv,
                                                        VEC* __restrict__ out) {
  const size_t n = (size_t)rows_out * chunks;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) {
    const int r = (int)(i / chunks), c = (int)(i % chunks);
    const int src = r < v0 ? r : r + nv;
    out[i] = h[(size_t)src * chunks + c];
  }
}

template <typename VEC>
hipError_t drop_rows_launch(const void* h, int rows_out, int chunks, int v0, int nv, void* out,
                            hipStream_t s) {
  const size_t n = (size_t)rows_out * chunks;
  size_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  drop_rows_kernel<VEC><<<(unsigned)blocks, 256, 0, s>>>(static_cast<const VEC*>(h), rows_out,
                                                         chunks, v0, nv, static_cast<VEC*>(out));
  return hipGetLastError();
}
}  // namespace

hipError_t launch_combine(const void* y_perm, bool bf16, const int32_t* row_of_slot,
                          const float* w, int T, int k, int d, void* out, hipStream_t s) {
  const size_t row_bytes = (size_t)d * (bf16 ? 2 : 4);
  if (row_bytes % 16 == 0) {
    const int chunks = (int)(row_bytes / 16);
    const int rpb = chunks >= 256 ? 1 : 256 / chunks;
    const int grid = (T + rpb - 1) / rpb;
    if (bf16)
      combine_kernel<true><<<grid, 256, 0, s>>>(static_cast<const uint4*>(y_perm), row_of_slot, w,
                                                T, k, chunks, rpb, static_cast<uint4*>(out));
    else
      combine_kernel<false><<<grid, 256, 0, s>>>(static_cast<const uint4*>(y_perm), row_of_slot, w,
                                                 T, k, chunks, rpb, static_cast<uint4*>(out));
  } else {
    size_t blocks = ((size_t)T * d + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (bf16)
      combine_scalar_kernel<true><<<(unsigned)blocks, 256, 0, s>>>(y_perm, row_of_slot, w, T, k, d, out);
    else
      combine_scalar_kernel<false><<<(unsigned)blocks, 256, 0, s>>>(y_perm, row_of_slot, w, T, k, d, out);
  }
  return hipGetLastError();
}

hipError_t launch_drop_rows(const void* h, int elt, int S, int d, int v0, int v1, void* out,
                            hipStream_t s) {
  const int rows_out = S - (v1 - v0), nv = v1 - v0;
  const size_t row_bytes = (size_t)d * elt;
  const uintptr_t al = reinterpret_cast<uintptr_t>(h) | reinterpret_cast<uintptr_t>(out);
  if (row_bytes % 16 == 0 && al % 16 == 0)
    return drop_rows_launch<uint4>(h, rows_out, (int)(row_bytes / 16), v0, nv, out, s);
  if (row_bytes % 4 == 0 && al % 4 == 0)
    return drop_rows_launch<uint32_t>(h, rows_out, (int)(row_bytes / 4), v0, nv, out, s);
  return drop_rows_launch<uint16_t>(h, rows_out, (int)(row_bytes / 2), v0, nv, out, s);
}

}  // namespace decomoe
