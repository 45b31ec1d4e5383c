// Physical expert reorder by the Mean-Mass order pi (Sec. 3.3 after Eq. 9;
// Algorithm 1): new expert j takes native expert pi[j]'s router column,
// bias and expert weight blocks.  It moves storage and computes nothing; it
// runs once when a layer is loaded.
#include "common.hpp"

namespace decomoe {
namespace {

// one expert block per blockIdx.y, VEC-sized vectors grid-strided over x
template <typename VEC>
__global__ __launch_bounds__(256) void permute_blocks_kernel(const VEC* __restrict__ in,
                                                             const int32_t* __restrict__ order,
                                                             int E, size_t n_vec,
                                                             VEC* __restrict__ out) {
  const int j = blockIdx.y;
  const int src = order[j];
  const bool ok = src >= 0 && src < E;
  VEC* o = out + (size_t)j * n_vec;
  const VEC* i0 = in + (size_t)(ok ? src : 0) * n_vec;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n_vec; i += (size_t)gridDim.x * 256)
    o[i] = ok ? i0[i] : VEC{};
}

template <typename VEC>
hipError_t permute_blocks_launch(const void* in, const int32_t* order, int E, size_t n_vec,
                                 void* out, hipStream_t s) {
  size_t gx = (n_vec + 255) / 256;
  if (gx > 1024) gx = 1024;
  permute_blocks_kernel<VEC><<<dim3((unsigned)gx, (unsigned)E), 256, 0, s>>>(
      static_cast<const VEC*>(in), order, E, n_vec, static_cast<VEC*>(out));
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void permute_columns_kernel(const float* __restrict__ in,
                                                              const int32_t* __restrict__ order,
                                                              int rows, int E,
                                                              float* __restrict__ out) {
  const size_t n = (size_t)rows * E;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) {
    const size_t r = i / E;
    const int j = (int)(i % E);
    const int src = order[j];
    out[i] = (src >= 0 && src < E) ? in[r * E + src] : 0.f;
  }
}
}  // namespace

hipError_t launch_permute_blocks(const void* in, const int32_t* order, int E, size_t block_bytes,
                                 void* out, hipStream_t s) {
  const uintptr_t al = reinterpret_cast<uintptr_t>(in) | reinterpret_cast<uintptr_t>(out);
  if (block_bytes % 16 == 0 && al % 16 == 0)
    return permute_blocks_launch<uint4>(in, order, E, block_bytes / 16, out, s);
  if (block_bytes % 4 == 0 && al % 4 == 0)
    return permute_blocks_launch<uint32_t>(in, order, E, block_bytes / 4, out, s);
  return permute_blocks_launch<uint16_t>(in, order, E, block_bytes / 2, out, s);
}

hipError_t launch_permute_columns(const float* in, const int32_t* order, int rows, int E,
                                  float* out, hipStream_t s) {
  size_t blocks = ((size_t)rows * E + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks == 0) return hipSuccess;
  permute_columns_kernel<<<(unsigned)blocks, 256, 0, s>>>(in, order, rows, E, out);
  return hipGetLastError();
}

}  // namespace decomoe
