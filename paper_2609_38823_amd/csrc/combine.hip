// Weighted combine back to token order (Algorithm 2) and the SAVB
// visual-block row compaction (Sec. 3.2; Algorithm 2).
#include "common.hpp"

namespace decomoe {
namespace {

// 16-byte store, non-temporal when NT (outputs larger than the memory-side
// cache: their dirty lines would otherwise have to be written back before
// the next kernel's reads can use that cache)
template <bool NT>
__device__ __forceinline__ void store_out(uint4* p, uint4 v) {
  if constexpr (NT) {
    const u32x4_nt q = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(q, reinterpret_cast<u32x4_nt*>(p));
  } else {
    *p = v;
  }
}

// out[t] = sum_j w[t, j] * y[row_of_slot[t*k + j]], float32 accumulation in
// slot order; with RES the residual row is added to the float32 sum before
// the one rounding (res may be out itself: each thread reads its vector of
// res before it writes the same vector of out).  Each thread owns one 16-byte
// vector of the row (8 bf16 or 4 f32); a block covers one token row, or
// several when rows are short.
template <bool BF16, bool RES, bool NTST>
__global__ __launch_bounds__(256) void combine_kernel(const uint4* __restrict__ y,
                                                      const int32_t* __restrict__ row_of_slot,
                                                      const float* __restrict__ w, int T, int k,
                                                      int chunks, int rpb, const uint4* res,
                                                      uint4* out, const Guard g) {
  if (guard_skip(g)) return;
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
    // slots in groups of 8: the group's row loads are all issued before the
    // accumulation (a slot outside [0, T*k) reads row 0 and adds nothing)
    for (int j0 = 0; j0 < k; j0 += 8) {
      uint4 v[8];
      float wj[8];
      bool ok[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + u;
        const int r = j < k ? row_of_slot[(size_t)t * k + j] : -1;
        ok[u] = r >= 0 && r < A;
        wj[u] = j < k ? w[(size_t)t * k + j] : 0.f;
        v[u] = load_stream(y + (size_t)(ok[u] ? r : 0) * chunks + c);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (!ok[u]) continue;
        if constexpr (BF16) {
          const uint32_t q4[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            acc[2 * q] = fmaf(wj[u], __uint_as_float(q4[q] << 16), acc[2 * q]);
            acc[2 * q + 1] = fmaf(wj[u], __uint_as_float(q4[q] & 0xffff0000u), acc[2 * q + 1]);
          }
        } else {
          acc[0] = fmaf(wj[u], __uint_as_float(v[u].x), acc[0]);
          acc[1] = fmaf(wj[u], __uint_as_float(v[u].y), acc[1]);
          acc[2] = fmaf(wj[u], __uint_as_float(v[u].z), acc[2]);
          acc[3] = fmaf(wj[u], __uint_as_float(v[u].w), acc[3]);
        }
      }
    }
    if constexpr (RES) {
      const uint4 v = res[(size_t)t * chunks + c];
      if constexpr (BF16) {
        const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[2 * q] += __uint_as_float(u[q] << 16);
          acc[2 * q + 1] += __uint_as_float(u[q] & 0xffff0000u);
        }
      } else {
        acc[0] += __uint_as_float(v.x);
        acc[1] += __uint_as_float(v.y);
        acc[2] += __uint_as_float(v.z);
        acc[3] += __uint_as_float(v.w);
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
    store_out<NTST>(out + (size_t)t * chunks + c, o);
  }
}

// element-wise fallback when rows are not whole 16-byte vectors
template <bool BF16, bool RES>
__global__ __launch_bounds__(256) void combine_scalar_kernel(const void* __restrict__ yv,
                                                             const int32_t* __restrict__ row_of_slot,
                                                             const float* __restrict__ w, int T,
                                                             int k, int d, const void* resv,
                                                             void* outv, const Guard g) {
  if (guard_skip(g)) return;
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
    if constexpr (RES)
      acc += BF16 ? bf16_to_f32(static_cast<const uint16_t*>(resv)[i]) : static_cast<const float*>(resv)[i];
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

namespace {
template <bool RES>
hipError_t combine_launch(const void* y_perm, bool bf16, const int32_t* row_of_slot,
                          const float* w, int T, int k, int d, const void* res, void* out,
                          hipStream_t s, Guard g) {
  const size_t row_bytes = (size_t)d * (bf16 ? 2 : 4);
  if (row_bytes % 16 == 0) {
    const int chunks = (int)(row_bytes / 16);
    const int rpb = chunks >= 256 ? 1 : 256 / chunks;
    const int grid = (T + rpb - 1) / rpb;
    auto y = static_cast<const uint4*>(y_perm);
    auto r = static_cast<const uint4*>(res);
    auto o = static_cast<uint4*>(out);
    // outputs beyond 64 MiB are written past the caches (see store_out)
    const bool nt = (size_t)T * row_bytes > ((size_t)64 << 20);
    if (bf16 && nt)
      combine_kernel<true, RES, true><<<grid, 256, 0, s>>>(y, row_of_slot, w, T, k, chunks, rpb, r, o, g);
    else if (bf16)
      combine_kernel<true, RES, false><<<grid, 256, 0, s>>>(y, row_of_slot, w, T, k, chunks, rpb, r, o, g);
    else if (nt)
      combine_kernel<false, RES, true><<<grid, 256, 0, s>>>(y, row_of_slot, w, T, k, chunks, rpb, r, o, g);
    else
      combine_kernel<false, RES, false><<<grid, 256, 0, s>>>(y, row_of_slot, w, T, k, chunks, rpb, r, o, g);
  } else {
    size_t blocks = ((size_t)T * d + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (bf16)
      combine_scalar_kernel<true, RES><<<(unsigned)blocks, 256, 0, s>>>(y_perm, row_of_slot, w, T,
                                                                        k, d, res, out, g);
    else
      combine_scalar_kernel<false, RES><<<(unsigned)blocks, 256, 0, s>>>(y_perm, row_of_slot, w,
                                                                         T, k, d, res, out, g);
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_combine(const void* y_perm, bool bf16, const int32_t* row_of_slot,
                          const float* w, int T, int k, int d, const void* residual, void* out,
                          hipStream_t s, Guard g) {
  if (residual)
    return combine_launch<true>(y_perm, bf16, row_of_slot, w, T, k, d, residual, out, s, g);
  return combine_launch<false>(y_perm, bf16, row_of_slot, w, T, k, d, nullptr, out, s, g);
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
