// Router logits of Eq. 1 on bf16 MFMA with the float32 router weights split
// into three bf16 terms.
//
// Split (done once, when the layer is loaded): W = W1 + W2 + W3 with
// W1 = bf16(W), W2 = bf16(W - W1), W3 = bf16(W - W1 - W2) (round to nearest
// even; both differences are exact in float32).  Together the three terms
// carry 24 significand bits, so |W - (W1 + W2 + W3)| <= 2^-24 |W| up to
// underflow.  The token rows x are bf16, so every product x W_p is exact in
// float32 and the MFMA accumulates x W1 + x W2 + x W3 in float32: the float32
// logits to within a small multiple of float32 rounding (splitting float32
// operands into bf16 terms: Henry, Tang and Heinecke, "Leveraging the
// bfloat16 Artificial Intelligence Datatype For Higher-Precision
// Computations", 2019).
//
// Packed layout: for expert block eb (32 experts), 16-wide k block kb and
// term p, the 1 KB fragment ((eb * (d / 16) + kb) * 3 + p) holds in lane l
// experts 32 eb + l % 32, k-values 16 kb + 8 (l / 32) .. + 8 -- the first
// operand of v_mfma_f32_32x32x16_bf16.
//
// Kernel: a workgroup computes 32 MI tokens (MI = 1, 2, 4) x 128 experts
// (wavefront w: the expert block 4 blockIdx.x + w) over the d-range of split
// blockIdx.z.  The token rows go global -> LDS in whole 128-byte row segments
// (stages of 64 k-values, ring of four, three stages ahead, chunk c of row r
// stored at c ^ ((r >> 1) & 7)); each wavefront reads its weight fragments
// straight from the packed array into a ring of NR register stages, NR - 1
// stages ahead (the split weights are shared by every token tile and come
// from L2).  Per 16-wide k block: 3 MI MFMAs (terms 1, 2, 3 of each token
// block in that order).
#include "common.hpp"

#include <type_traits>

namespace decomoe {
namespace {
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int XS_K = 64;                 // k-values per token-row stage
constexpr int XS_BYTES_ROW = XS_K * 2;   // 128 bytes

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, 0x00020000);
}
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, void* lds, int voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds, 16, voff, soff, 0, 0);
}
// wait until at most N vector-memory operations of this wavefront are
// outstanding (gfx9 encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] |
// vmcnt_hi[15:14])
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// one thread per (expert block, k block, lane): 8 weights, three fragments
__global__ __launch_bounds__(256) void pack_router_kernel(const float* __restrict__ w_r, int d, int E,
                                                          uint4* __restrict__ out) {
  const int KB = d / 16;
  const size_t n = (size_t)(E / 32) * KB * 64;
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int l = (int)(i & 63);
  const size_t f = i >> 6;  // eb * KB + kb
  const int kb = (int)(f % KB), eb = (int)(f / KB);
  const int e = 32 * eb + (l & 31), k0 = 16 * kb + 8 * (l >> 5);
  uint32_t t[3][4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float r[2][3];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float w = w_r[(size_t)(k0 + 2 * j + h) * E + e];
      const uint16_t b1 = f32_to_bf16(w);
      const float r1 = w - bf16_to_f32(b1);
      const uint16_t b2 = f32_to_bf16(r1);
      const float r2 = r1 - bf16_to_f32(b2);
      r[h][0] = bf16_to_f32(b1);
      r[h][1] = bf16_to_f32(b2);
      r[h][2] = bf16_to_f32(f32_to_bf16(r2));
    }
#pragma unroll
    for (int p = 0; p < 3; ++p) t[p][j] = pack_bf16x2(r[0][p], r[1][p]);
  }
#pragma unroll
  for (int p = 0; p < 3; ++p) out[(f * 3 + p) * 64 + l] = make_uint4(t[p][0], t[p][1], t[p][2], t[p][3]);
}

// MI: 32-token blocks per workgroup; NR: weight stages in registers (2 or 4);
// WPC: workgroups per compute unit.
template <int MI, int NR, int WPC>
__global__ __launch_bounds__(256, WPC) void router_x3_kernel(const uint16_t* __restrict__ x,
                                                             const uint16_t* __restrict__ wp,
                                                             const float* __restrict__ bias, int T,
                                                             int d, int E, float* __restrict__ logits,
                                                             float* __restrict__ split_part, const Guard g) {
  if (guard_skip(g)) return;
  static_assert(NR == 2 || NR == 4, "weight ring of 2 or 4 stages");
  constexpr int ROWS = 32 * MI;
  constexpr int SLOT = ROWS * XS_BYTES_ROW;
  __shared__ __attribute__((aligned(1024))) char ring[4 * SLOT];
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int KB = d / 16;
  const int eb_raw = blockIdx.x * 4 + wv;
  const int n_eb = E / 32;
  const int eb = eb_raw < n_eb ? eb_raw : n_eb - 1;  // idle wavefronts recompute the last block
  const int t0 = blockIdx.y * ROWS;
  const int rows = min(ROWS, T - t0);
  const int dch = d / gridDim.z;
  const int k_begin = blockIdx.z * dch;
  const int n_st = dch / XS_K;

  // token rows: transfer q of wavefront wv covers rows 8 (wv + 4 q) .. + 7;
  // lane l fills row 8 (wv + 4 q) + l / 8, physical chunk l % 8 with logical
  // chunk (l % 8) ^ ((row >> 1) & 7); rows past T re-read the tile's row 0
  const __amdgpu_buffer_rsrc_t x_rs = rsrc(x + (size_t)t0 * d, (uint32_t)rows * d * 2);
  int x_voff[MI];
#pragma unroll
  for (int q = 0; q < MI; ++q) {
    const int row = 8 * (wv + 4 * q) + (lane >> 3);
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    x_voff[q] = ((row < rows ? row : 0) * d + k_begin + c * 8) * 2;
  }
  auto issue_x = [&](int st) {
    char* slot = ring + (st & 3) * SLOT;
#pragma unroll
    for (int q = 0; q < MI; ++q) dma16(x_rs, slot + (wv + 4 * q) * 1024, x_voff[q], st * XS_K * 2);
  };
  const int r32 = lane & 31, kh = lane >> 5;
  int x_lane[4];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) x_lane[s4] = r32 * 128 + (((2 * s4 + kh) ^ ((r32 >> 1) & 7)) << 4);

  // weights: the 12 fragments (4 k blocks x 3 terms) of one stage
  const __amdgpu_buffer_rsrc_t w_rs = rsrc(wp + (size_t)eb * KB * 3 * 512, (uint32_t)KB * 3 * 1024);
  const int kb0 = k_begin / 16;
  auto load_w = [&](u32x4 (&wf)[4][3], int st) {
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
      for (int p = 0; p < 3; ++p)
        wf[s4][p] = __builtin_amdgcn_raw_buffer_load_b128(w_rs, lane * 16, ((kb0 + 4 * st + s4) * 3 + p) * 1024, 0);
  };

  f32x16 acc[MI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[i][e] = 0.f;

  // Stage st: wait until this wavefront's token-row transfers of stage st
  // have landed (WAIT = the loads issued after them), barrier (every
  // wavefront's have; every read of the slot refilled next is done), refill
  // the slot of stage st - 1 with stage st + 3 and the weight registers of
  // stage st - 1 with stage st + NR - 1, then 4 x 3 MI MFMAs.  Every stage
  // issues its loads, also past the d-range's end (there they stay inside
  // the buffers or read zeros, into slots and registers no stage uses), so
  // the counts are the same in every stage: after the transfers of stage st
  // come the weights of stage st + NR - 4 and the loads of two stages,
  // 12 + 2 (MI + 12).  The prologue issues x0, w0, x1, w1, x2, w2 (NR = 4)
  // or x0, x1, x2, w0 (NR = 2, whose stages 0 and 1 wait for fewer).
  u32x4 wr[NR][4][3];
  auto stage = [&](auto U, auto WAIT, int st) {
    constexpr int u = decltype(U)::value;
    wait_vm<decltype(WAIT)::value>();
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's reads of the previous stage
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    issue_x(st + 3);
    load_w(wr[(u + NR - 1) % NR], st + NR - 1);
    __builtin_amdgcn_sched_barrier(0);
    const char* slot = ring + (st & 3) * SLOT;
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
      bf16x8 xf[MI];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) xf[mi] = *reinterpret_cast<const bf16x8*>(slot + mi * 32 * 128 + x_lane[s4]);
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int p = 0; p < 3; ++p)
          acc[mi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wr[u][s4][p]), xf[mi],
                                                            acc[mi], 0, 0, 0);
    }
  };
  using WS = std::integral_constant<int, 36 + 2 * MI>;
  if constexpr (NR == 4) {
    issue_x(0);
    load_w(wr[0], 0);
    issue_x(1);
    load_w(wr[1], 1);
    issue_x(2);
    load_w(wr[2], 2);
    for (int st = 0; st < n_st; st += 4) {
      stage(std::integral_constant<int, 0>{}, WS{}, st);
      if (st + 1 < n_st) stage(std::integral_constant<int, 1>{}, WS{}, st + 1);
      if (st + 2 < n_st) stage(std::integral_constant<int, 2>{}, WS{}, st + 2);
      if (st + 3 < n_st) stage(std::integral_constant<int, 3>{}, WS{}, st + 3);
    }
  } else {
    issue_x(0);
    issue_x(1);
    issue_x(2);
    load_w(wr[0], 0);
    stage(std::integral_constant<int, 0>{}, std::integral_constant<int, 2 * MI + 12>{}, 0);
    if (1 < n_st) stage(std::integral_constant<int, 1>{}, std::integral_constant<int, 2 * MI + 24>{}, 1);
    for (int st = 2; st < n_st; st += 2) {
      stage(std::integral_constant<int, 0>{}, WS{}, st);
      if (st + 1 < n_st) stage(std::integral_constant<int, 1>{}, WS{}, st + 1);
    }
  }

  wait_vm<0>();  // transfers of stages past the d-range's end
  if (eb_raw >= n_eb) return;  // no barrier follows
  // lane l: token t0 + l % 32 (+ 32 mi), experts 32 eb + 8 g + 4 (l / 32) + 0..3
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    const int t = t0 + 32 * mi + r32;
    if (t >= T) continue;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int e = 32 * eb + 8 * g + 4 * kh;
      float4 v = make_float4(acc[mi][4 * g], acc[mi][4 * g + 1], acc[mi][4 * g + 2], acc[mi][4 * g + 3]);
      if (split_part) {
        *reinterpret_cast<float4*>(split_part + ((size_t)blockIdx.z * T + t) * E + e) = v;
      } else {
        if (bias) {
          const float4 b = *reinterpret_cast<const float4*>(bias + e);
          v.x += b.x;
          v.y += b.y;
          v.z += b.z;
          v.w += b.w;
        }
        *reinterpret_cast<float4*>(logits + (size_t)t * E + e) = v;
      }
    }
  }
}

// The previous layer's combine with the residual, fused into this layer's
// router: h[t] <- h[t] + sum_j w_prev[t, j] y_prev[row_prev[t, j]]
// (Algorithm 2's combine, float32 accumulation in slot order and one
// rounding, as combine_kernel), then the logits of the new rows as
// router_x3_kernel.  The router's workgroups own disjoint blocks of (token
// tile) x (d-range of the split), so each workgroup forms exactly the rows
// and columns it multiplies: it writes them to h and keeps them in LDS as its
// whole token tile (all stages of its d-range resident, no ring), after the
// tile's slot rows and weights (32 MI k_prev of each).  One expert group
// (E <= 128).  Rows past T are zeros in LDS and are not stored.
template <int MI>
__global__ __launch_bounds__(256, 2) void combine_router_x3_kernel(
    const uint16_t* __restrict__ y_prev, const int32_t* __restrict__ row_prev,
    const float* __restrict__ w_prev, int k_prev, const uint16_t* res, uint16_t* out,
    const uint16_t* __restrict__ wp, const float* __restrict__ bias, int T, int d, int E,
    float* __restrict__ logits, float* __restrict__ split_part, const Guard g) {
  if (guard_skip(g)) return;
  constexpr int ROWS = 32 * MI;
  constexpr int SLOT = ROWS * XS_BYTES_ROW;
  extern __shared__ __attribute__((aligned(1024))) char tile[];  // n_st slots of SLOT bytes
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int KB = d / 16;
  const int eb_raw = blockIdx.x * 4 + wv;
  const int n_eb = E / 32;
  const int eb = eb_raw < n_eb ? eb_raw : n_eb - 1;
  const int t0 = blockIdx.y * ROWS;
  const int dch = d / gridDim.z;
  const int k_begin = blockIdx.z * dch;
  const int n_st = dch / XS_K;
  const int A = T * k_prev;

  // the first weight stage does not depend on the combine
  const int r32 = lane & 31, kh = lane >> 5;
  const __amdgpu_buffer_rsrc_t w_rs = rsrc(wp + (size_t)eb * KB * 3 * 512, (uint32_t)KB * 3 * 1024);
  const int kb0 = k_begin / 16;
  auto load_w = [&](u32x4 (&wf)[4][3], int st) {
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
      for (int p = 0; p < 3; ++p)
        wf[s4][p] = __builtin_amdgcn_raw_buffer_load_b128(w_rs, lane * 16, ((kb0 + 4 * st + s4) * 3 + p) * 1024, 0);
  };
  u32x4 wr[2][4][3];
  load_w(wr[0], 0);

  // ---- combine.  The tile's slot rows and weights go to LDS once (a slot
  // outside [0, T k_prev) as -1: it adds nothing); then each thread takes
  // CB 16-byte chunks at a time and issues all their row loads before the
  // accumulation.  Chunk q is columns k_begin + 8 (q % cpr) of tile row
  // q / cpr; the columns of stage c / 8 sit at the router's swizzled place.
  int* s_row = reinterpret_cast<int*>(tile + n_st * SLOT);
  float* s_w = reinterpret_cast<float*>(s_row + ROWS * k_prev);
  for (int i = threadIdx.x; i < ROWS * k_prev; i += 256) {
    const int t = t0 + i / k_prev;
    int rr = -1;
    float wj = 0.f;
    if (t < T) {
      rr = row_prev[(size_t)t0 * k_prev + i];
      wj = w_prev[(size_t)t0 * k_prev + i];
      if (rr < 0 || rr >= A) rr = -1;
    }
    s_row[i] = rr;
    s_w[i] = wj;
  }
  __syncthreads();
  const int cpr = dch / 8;  // chunks per row
  const int nq = ROWS * cpr;
  constexpr int CB = 2;
  for (int q0 = threadIdx.x; q0 < nq; q0 += 256 * CB) {
    int r[CB], c[CB];
    bool live[CB];
#pragma unroll
    for (int b = 0; b < CB; ++b) {
      const int q = q0 + 256 * b;
      r[b] = q / cpr;
      c[b] = q % cpr;
      live[b] = q < nq && t0 + r[b] < T;
    }
    float acc[CB][8] = {};
    uint4 hv[CB];
#pragma unroll
    for (int b = 0; b < CB; ++b)
      hv[b] = live[b] ? *reinterpret_cast<const uint4*>(res + (size_t)(t0 + r[b]) * d + k_begin + 8 * c[b])
                      : make_uint4(0u, 0u, 0u, 0u);
    for (int j0 = 0; j0 < k_prev; j0 += 8) {
      uint4 v[CB][8];
      int rj[CB][8];
#pragma unroll
      for (int b = 0; b < CB; ++b)
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = j0 + u;
          rj[b][u] = live[b] && j < k_prev ? s_row[r[b] * k_prev + j] : -1;
          const size_t row = rj[b][u] >= 0 ? (size_t)rj[b][u] : 0;
          v[b][u] = load_stream(reinterpret_cast<const uint4*>(y_prev + row * d + k_begin + 8 * c[b]));
        }
#pragma unroll
      for (int b = 0; b < CB; ++b)
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (rj[b][u] < 0) continue;
          const float wj = s_w[r[b] * k_prev + j0 + u];
          const uint32_t q4[4] = {v[b][u].x, v[b][u].y, v[b][u].z, v[b][u].w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[b][2 * e] = fmaf(wj, __uint_as_float(q4[e] << 16), acc[b][2 * e]);
            acc[b][2 * e + 1] = fmaf(wj, __uint_as_float(q4[e] & 0xffff0000u), acc[b][2 * e + 1]);
          }
        }
    }
#pragma unroll
    for (int b = 0; b < CB; ++b) {
      if (q0 + 256 * b >= nq) continue;
      uint4 o = make_uint4(0u, 0u, 0u, 0u);
      if (live[b]) {
        const uint32_t u4[4] = {hv[b].x, hv[b].y, hv[b].z, hv[b].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[b][2 * e] += __uint_as_float(u4[e] << 16);
          acc[b][2 * e + 1] += __uint_as_float(u4[e] & 0xffff0000u);
        }
        o = make_uint4(pack_bf16x2(acc[b][0], acc[b][1]), pack_bf16x2(acc[b][2], acc[b][3]),
                       pack_bf16x2(acc[b][4], acc[b][5]), pack_bf16x2(acc[b][6], acc[b][7]));
        *reinterpret_cast<uint4*>(out + (size_t)(t0 + r[b]) * d + k_begin + 8 * c[b]) = o;
      }
      const int cc = c[b] & 7;
      *reinterpret_cast<uint4*>(tile + (c[b] >> 3) * SLOT + r[b] * XS_BYTES_ROW + ((cc ^ ((r[b] >> 1) & 7)) << 4)) = o;
    }
  }
  __syncthreads();

  // ---- logits of the tile over this d-range (the MFMA order of
  // router_x3_kernel, so the partial sums are bitwise the same)
  int x_lane[4];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) x_lane[s4] = r32 * 128 + (((2 * s4 + kh) ^ ((r32 >> 1) & 7)) << 4);
  f32x16 acc[MI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[i][e] = 0.f;
  auto stage = [&](auto U, int st) {
    constexpr int u = decltype(U)::value;
    if (st + 1 < n_st) load_w(wr[u ^ 1], st + 1);
    const char* slot = tile + st * SLOT;
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
      bf16x8 xf[MI];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) xf[mi] = *reinterpret_cast<const bf16x8*>(slot + mi * 32 * 128 + x_lane[s4]);
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int p = 0; p < 3; ++p)
          acc[mi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wr[u][s4][p]), xf[mi],
                                                            acc[mi], 0, 0, 0);
    }
  };
  for (int st = 0; st < n_st; st += 2) {
    stage(std::integral_constant<int, 0>{}, st);
    if (st + 1 < n_st) stage(std::integral_constant<int, 1>{}, st + 1);
  }

  if (eb_raw >= n_eb) return;
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    const int t = t0 + 32 * mi + r32;
    if (t >= T) continue;
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int e = 32 * eb + 8 * gq + 4 * kh;
      float4 v = make_float4(acc[mi][4 * gq], acc[mi][4 * gq + 1], acc[mi][4 * gq + 2], acc[mi][4 * gq + 3]);
      if (split_part) {
        *reinterpret_cast<float4*>(split_part + ((size_t)blockIdx.z * T + t) * E + e) = v;
      } else {
        if (bias) {
          const float4 b = *reinterpret_cast<const float4*>(bias + e);
          v.x += b.x;
          v.y += b.y;
          v.z += b.z;
          v.w += b.w;
        }
        *reinterpret_cast<float4*>(logits + (size_t)t * E + e) = v;
      }
    }
  }
}
}  // namespace

// Launch plan: 128-token tiles over the whole d-range once they give every
// compute unit two workgroups (the split weights then stream from L2 once
// per 128 tokens); else 64-token tiles when their grid, with at most 4
// d-splits, has about 256 workgroups, else 32-token tiles with up to 8
// splits (whole 64-wide stages per split; the Top-k kernel adds the split
// partials, so more splits lengthen it).
struct RouterPlan {
  int MI, S;
};
RouterPlan router_x3_plan(int T, int d, int E) {
  const int groups = (E / 32 + 3) / 4;
  if (groups * ((T + 127) / 128) >= 512) return RouterPlan{4, 1};
  for (int mi = 2; mi >= 1; mi /= 2) {
    const int tiles = groups * ((T + 32 * mi - 1) / (32 * mi));
    int s = 1;
    while (tiles * s < 256 && s < 4 && d % (XS_K * 2 * s) == 0) s *= 2;
    if (tiles * s >= 256 || mi == 1) {
      while (mi == 1 && tiles * s < 256 && s < 8 && d % (XS_K * 2 * s) == 0) s *= 2;
      return RouterPlan{mi, s};
    }
  }
  return RouterPlan{1, 1};
}

size_t route_x3_ws_bytes(int T, int d, int E) {
  const RouterPlan pl = router_x3_plan(T, d, E);
  return pl.S > 1 ? (size_t)pl.S * T * E * sizeof(float) : 0;
}

hipError_t launch_pack_router(const float* w_r, int d, int E, void* out, hipStream_t s) {
  const size_t n = (size_t)(E / 32) * (d / 16) * 64;
  if (n == 0) return hipSuccess;
  pack_router_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(w_r, d, E, static_cast<uint4*>(out));
  return hipGetLastError();
}

hipError_t launch_router_x3(const void* x, const void* w_packed, const float* bias, int T, int d,
                            int E, float* logits, void* ws, float*& part, int& S, hipStream_t s,
                            Guard g) {
  const RouterPlan pl = router_x3_plan(T, d, E);
  S = pl.S;
  part = S > 1 ? static_cast<float*>(ws) : nullptr;
  const dim3 grid((E / 32 + 3) / 4, (T + 32 * pl.MI - 1) / (32 * pl.MI), S);
  auto xp = static_cast<const uint16_t*>(x);
  auto wp = static_cast<const uint16_t*>(w_packed);
  if (pl.MI == 4)
    router_x3_kernel<4, 2, 2><<<grid, 256, 0, s>>>(xp, wp, bias, T, d, E, logits, part, g);
  else if (pl.MI == 2)
    router_x3_kernel<2, 2, 2><<<grid, 256, 0, s>>>(xp, wp, bias, T, d, E, logits, part, g);
  else
    router_x3_kernel<1, 2, 2><<<grid, 256, 0, s>>>(xp, wp, bias, T, d, E, logits, part, g);
  return hipGetLastError();
}

// The previous layer's combine fused into the router (one expert group, a
// token tile of at most 32 KB in LDS): false when the plan does not allow it
// LDS of the fused launch: the token tile of its d-range, then the slot
// rows and weights of the tile's rows
static size_t combine_router_lds(const RouterPlan& pl, int d, int k) {
  return (size_t)32 * pl.MI * (d / pl.S) * 2 + (size_t)32 * pl.MI * k * 8;
}

bool combine_router_fits(int T, int d, int E, int k) {
  if (T < 1 || E > 128 || E % 32 != 0 || d % 256 != 0) return false;
  const RouterPlan pl = router_x3_plan(T, d, E);
  return (size_t)32 * pl.MI * (d / pl.S) * 2 <= 32768 && combine_router_lds(pl, d, k) <= 49152;
}

hipError_t launch_combine_router_x3(const void* y_prev, const int32_t* row_prev, const float* w_prev, int k_prev,
                                    void* h, const void* w_packed, const float* bias, int T, int d, int E,
                                    float* logits, void* ws, float*& part, int& S, hipStream_t s, Guard g) {
  const RouterPlan pl = router_x3_plan(T, d, E);
  S = pl.S;
  part = S > 1 ? static_cast<float*>(ws) : nullptr;
  const dim3 grid((E / 32 + 3) / 4, (T + 32 * pl.MI - 1) / (32 * pl.MI), S);
  const size_t lds = combine_router_lds(pl, d, k_prev);
  auto yp = static_cast<const uint16_t*>(y_prev);
  auto hp = static_cast<uint16_t*>(h);
  auto wp = static_cast<const uint16_t*>(w_packed);
  if (pl.MI == 4)
    combine_router_x3_kernel<4><<<grid, 256, lds, s>>>(yp, row_prev, w_prev, k_prev, hp, hp, wp, bias, T, d, E, logits,
                                                       part, g);
  else if (pl.MI == 2)
    combine_router_x3_kernel<2><<<grid, 256, lds, s>>>(yp, row_prev, w_prev, k_prev, hp, hp, wp, bias, T, d, E, logits,
                                                       part, g);
  else
    combine_router_x3_kernel<1><<<grid, 256, lds, s>>>(yp, row_prev, w_prev, k_prev, hp, hp, wp, bias, T, d, E, logits,
                                                       part, g);
  return hipGetLastError();
}

}  // namespace decomoe
