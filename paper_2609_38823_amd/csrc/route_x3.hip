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
// Kernel: a workgroup computes 32 MI tokens (MI = 1, 2) x 128 experts (wavefront w: the
// expert block 4 blockIdx.x + w) over the d-range of split blockIdx.z.  The
// token rows go global -> LDS in whole 128-byte row segments (stages of 64
// k-values, ring of four, three stages ahead, chunk c of row r stored at
// c ^ ((r >> 1) & 7)); each wavefront reads its weight fragments straight
// from the packed array into registers, one stage ahead.  Per 16-wide
// k block: 3 MI MFMAs (terms 1, 2, 3 of each token block in that order).
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

template <int MI>
__global__ __launch_bounds__(256, 2) void router_x3_kernel(const uint16_t* __restrict__ x,
                                                           const uint16_t* __restrict__ wp,
                                                           const float* __restrict__ bias, int T,
                                                           int d, int E, float* __restrict__ logits,
                                                           float* __restrict__ split_part) {
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

  // stage st: barrier (every wavefront's token rows of the stage are in
  // LDS), refill the slot freed by stage st - 1 with stage st + 3
  // (ISSUE_X), load the weights of stage st + 1 (LOAD_W), then 4 x 3 MI
  // MFMAs.  The flags are compile-time so that the compiler's waits count
  // exactly.  The compiler waits for the weight registers, not for global ->
  // LDS transfers; the vector-memory counter completes in issue order, and
  // stage st's transfers precede the weights of stage st - 1, which the
  // MFMAs of stage st - 1 waited for before this barrier.  Stage 0 waits
  // explicitly (below).
  auto stage = [&](auto ISSUE_X, auto LOAD_W, int st, const u32x4 (&wc)[4][3], u32x4 (&wn)[4][3]) {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's reads of the previous stage
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (decltype(ISSUE_X)::value) issue_x(st + 3);
    if constexpr (decltype(LOAD_W)::value) load_w(wn, st + 1);
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
          acc[mi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wc[s4][p]), xf[mi],
                                                            acc[mi], 0, 0, 0);
    }
  };
  using F = std::integral_constant<bool, false>;
  using Tr = std::integral_constant<bool, true>;

  u32x4 wA[4][3], wB[4][3];
  // three stages always (past the split's end the loads stay inside the
  // buffer or read zeros at its end, into slots no stage reads), so that the
  // wait for stage 0 counts exactly: 2 MI transfers and 12 weight loads
  // follow it
  issue_x(0);
  issue_x(1);
  issue_x(2);
  load_w(wA, 0);
  wait_vm<2 * MI + 12>();
  int st = 0;
  for (; st + 4 < n_st; st += 2) {  // every refill and load in range
    stage(Tr{}, Tr{}, st, wA, wB);
    stage(Tr{}, Tr{}, st + 1, wB, wA);
  }
  switch (n_st - st) {  // the last 1..4 stages (st is even: stage st uses wA)
    case 4:
      stage(Tr{}, Tr{}, st, wA, wB);
      stage(F{}, Tr{}, st + 1, wB, wA);
      stage(F{}, Tr{}, st + 2, wA, wB);
      stage(F{}, F{}, st + 3, wB, wA);
      break;
    case 3:
      stage(F{}, Tr{}, st, wA, wB);
      stage(F{}, Tr{}, st + 1, wB, wA);
      stage(F{}, F{}, st + 2, wA, wB);
      break;
    case 2:
      stage(F{}, Tr{}, st, wA, wB);
      stage(F{}, F{}, st + 1, wB, wA);
      break;
    default:
      stage(F{}, F{}, st, wA, wB);
      break;
  }

  wait_vm<0>();                // transfers of stages past the split's end
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
}  // namespace

// Token rows per workgroup (32 MI, MI = 2 or 1) and d-splits S: 64-row
// tiles when their grid, with at most 4 splits, has about 256 workgroups;
// else 32-row tiles with up to 8 splits (whole 64-wide stages per split;
// more splits only lengthen the Top-k kernel's partial sums).
void router_x3_plan(int T, int d, int E, int& MI, int& S) {
  const int groups = (E / 32 + 3) / 4;
  for (int mi = 2; mi >= 1; mi /= 2) {
    const int tiles = groups * ((T + 32 * mi - 1) / (32 * mi));
    int s = 1;
    while (tiles * s < 256 && s < 4 && d % (XS_K * 2 * s) == 0) s *= 2;
    if (tiles * s >= 256 || mi == 1) {
      while (mi == 1 && tiles * s < 256 && s < 8 && d % (XS_K * 2 * s) == 0) s *= 2;
      MI = mi;
      S = s;
      return;
    }
  }
}

size_t route_x3_ws_bytes(int T, int d, int E) {
  int MI, S;
  router_x3_plan(T, d, E, MI, S);
  return S > 1 ? (size_t)S * T * E * sizeof(float) : 0;
}

hipError_t launch_pack_router(const float* w_r, int d, int E, void* out, hipStream_t s) {
  const size_t n = (size_t)(E / 32) * (d / 16) * 64;
  if (n == 0) return hipSuccess;
  pack_router_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(w_r, d, E, static_cast<uint4*>(out));
  return hipGetLastError();
}

hipError_t launch_router_x3(const void* x, const void* w_packed, const float* bias, int T, int d,
                            int E, float* logits, void* ws, float*& part, int& S, hipStream_t s) {
  int MI;
  router_x3_plan(T, d, E, MI, S);
  part = S > 1 ? static_cast<float*>(ws) : nullptr;
  const dim3 grid((E / 32 + 3) / 4, (T + 32 * MI - 1) / (32 * MI), S);
  auto xp = static_cast<const uint16_t*>(x);
  auto wp = static_cast<const uint16_t*>(w_packed);
  if (MI == 2)
    router_x3_kernel<2><<<grid, 256, 0, s>>>(xp, wp, bias, T, d, E, logits, part);
  else
    router_x3_kernel<1><<<grid, 256, 0, s>>>(xp, wp, bias, T, d, E, logits, part);
  return hipGetLastError();
}

}  // namespace decomoe
