// Grouped SwiGLU expert FFN over the dispatched rows (Algorithm 2: evaluate
// only the first K physically contiguous expert MLPs; gate, up and down
// projections as in App. A.3, Eq. 15).
//
//   tiles     a one-workgroup kernel turns the per-expert row ranges into a
//             list of (expert, first row, rows, n-tile) work items on the
//             device, so no host synchronisation is needed on K or on the
//             counts
//   gate_up   H[r, :] = SiLU(X W_gate^T) * (X W_up^T) for the rows of one
//             M-tile; the gate and up weight rows of the same h columns are
//             owned by the same wavefront, so SwiGLU is applied in registers
//   down      Y = H W_down^T
//
// bf16: v_mfma_f32_32x32x16_bf16 with float32 accumulation; 4 wavefronts per
// workgroup, each owning BM token rows x (BN/4) weight rows.  Two variants:
//   row-major weights  both operands stream global -> LDS (buffer_load ...
//                      lds) through a 4-stage ring; BN = 512 or 256; one
//                      launch per GEMM
//   packed weights     the weight operand streams from the fragment layout
//                      of moe_pack_expert_weights straight into registers;
//                      only the token rows use LDS; BN = 256 at two
//                      workgroups per CU; both GEMMs in one persistent launch
//                      with per-XCD work queues (the down GEMM of a token
//                      tile starts as soon as its h is complete), or one
//                      launch per GEMM where the XCD count is unknown
// float32: a plain LDS-tiled SIMT kernel (correctness path for small layers).
#include <cstdlib>
#include <type_traits>

#include "common.hpp"

namespace decomoe {
// Kernels live in a named namespace: device stubs of templated kernels with
// internal linkage are not emitted when instantiated from a template launcher.
namespace kern {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));


// ---------------------------------------------------------------------------
// Work items.  Experts e < Klim (Klim = max K_dev clamped to [kmin, E], or
// E) with rows
// [offsets[e], offsets[e+1]) (clamped to [0, rows_max]) become ceil(rows/bm)
// M-tiles; with nn n-tiles per GEMM the work list is ordered expert-major,
// then n-tile, then m-tile, and holds at most max_tiles * nn items.  Every
// workgroup derives its own item from the offsets (a block-wide scan over
// the experts), so no host synchronisation on K or on the counts is needed
// and no separate launch builds the list.
// ---------------------------------------------------------------------------
struct Work {
  int expert, row0, rows, nt;
};

struct Tiles {
  const int32_t* offsets;
  const int32_t* K_dev;
  int E, n_K, rows_max, bm, max_tiles, nn;
  int kmin;  // lower clamp of K (the routing's k where known, so that every
             // expert the prefix re-route can select is evaluated)
};

constexpr int NTHR = 256;  // threads per GEMM workgroup (4 wavefronts)

// Fills `out` with work item L and returns true, or returns false (for the
// whole workgroup) when L is past the end of the list.  With `xcd`, L follows
// the XCD-aware order: workgroup b runs on XCD b % 8, so XCD x is given the
// contiguous range [x n/8, (x+1) n/8) of the n-item list -- the m-tiles that
// share a weight tile, and the n-tiles that share an expert's rows, run
// together and meet in one L2, and every XCD gets an equal share.
// Otherwise L = blockIdx.x.  Supports E <= 4 * NTHR.  `lds` is 64 bytes of
// LDS that the caller may reuse as soon as this returns.
__device__ __forceinline__ bool find_work(const Tiles& tl, bool xcd, Work& out, char* lds) {
  int* s_part = reinterpret_cast<int*>(lds);           // [NTHR / 64]
  int& s_klim = reinterpret_cast<int*>(lds)[NTHR / 64];
  Work& s_wk = *reinterpret_cast<Work*>(lds + 32);
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (tid == 0) s_klim = 0;
  __syncthreads();
  int Klim = tl.E;
  if (tl.K_dev) {
    int mx = 0;
    for (int i = tid; i < tl.n_K; i += NTHR) mx = max(mx, tl.K_dev[i]);
    if (mx > 0) atomicMax(&s_klim, mx);
  }
  int lo[4], hi[4], cnt[4], local = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = 4 * tid + q;
    lo[q] = hi[q] = 0;
    if (e < tl.E) {
      lo[q] = clampi(tl.offsets[e], 0, tl.rows_max);
      hi[q] = clampi(tl.offsets[e + 1], lo[q], tl.rows_max);
    }
  }
  __syncthreads();
  if (tl.K_dev) Klim = clampi(s_klim, tl.kmin, tl.E);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    cnt[q] = 4 * tid + q < Klim ? (hi[q] - lo[q] + tl.bm - 1) / tl.bm : 0;
    local += cnt[q];
  }
  int incl = local;  // inclusive scan over the wavefront
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  if (lane == 63) s_part[wv] = incl;
  __syncthreads();
  int base = 0, total = 0;
#pragma unroll
  for (int i = 0; i < NTHR / 64; ++i) {
    if (i < wv) base += s_part[i];
    total += s_part[i];
  }
  total = min(total, tl.max_tiles);
  const int n_items = total * tl.nn;
  int L = blockIdx.x;
  if (xcd) {
    const int per_xcd = (n_items + 7) >> 3;
    const int slot = blockIdx.x >> 3;
    if (slot >= per_xcd) return false;
    L = (blockIdx.x & 7) * per_xcd + slot;
  }
  if (L >= n_items) return false;
  int start = base + incl - local;  // first tile of this thread's first expert
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = min(cnt[q], max(0, total - start));  // tiles kept
    if (c > 0 && L >= tl.nn * start && L < tl.nn * (start + c)) {
      const int o = L - tl.nn * start;
      const int r0 = lo[q] + (o % c) * tl.bm;
      s_wk = Work{4 * tid + q, r0, min(tl.bm, hi[q] - r0), o / c};
    }
    start += cnt[q];
  }
  __syncthreads();
  // uniform across the workgroup: keep the fields in scalar registers (they
  // form buffer descriptors and offsets)
  out.expert = __builtin_amdgcn_readfirstlane(s_wk.expert);
  out.row0 = __builtin_amdgcn_readfirstlane(s_wk.row0);
  out.rows = __builtin_amdgcn_readfirstlane(s_wk.rows);
  out.nt = __builtin_amdgcn_readfirstlane(s_wk.nt);
  __syncthreads();  // every thread holds its copy before the caller reuses `lds`
  return true;
}

// ---------------------------------------------------------------------------
// bf16 MFMA grouped GEMM
//
// Block tile BM token rows x BN weight rows, k-step 32; the 4 wavefronts
// split the weight rows, so each owns BM x (BN/4) outputs as 32x32 fragments
// of v_mfma_f32_32x32x16_bf16 (float32 accumulation; BM = 128, BN = 512
// gives 128x128 per wavefront, 256 accumulator registers, and 64 bytes of
// LDS reads per 32 MFMA cycles -- half the LDS bandwidth of a 64x64 tile).
// Operand tiles stream from global memory straight into LDS with
// buffer_load_dwordx4 ... lds through a 4-stage ring of separate LDS arrays
// (the compiler's wait tracking then keeps the three younger stages in flight
// while the oldest is consumed; with about 3 us of loaded memory latency,
// stages in flight rather than bandwidth set the pace).  Each 64-byte LDS row holds one tile row's 32
// k-values as four 16-byte chunks, chunk c stored at position
// c ^ ((row >> 2) & 3): the 16 rows read by one quarter-wavefront hit 16
// distinct bank groups.  The two 16-wide k-substeps of a stage are
// software-pipelined in registers.
// ---------------------------------------------------------------------------
constexpr int BK = 32;
constexpr int LDS_STAGE_MAX = (128 + 512) * BK * 2;  // bytes, largest tile pair

__shared__ __attribute__((aligned(1024))) char ring0[LDS_STAGE_MAX];
__shared__ __attribute__((aligned(1024))) char ring1[LDS_STAGE_MAX];
__shared__ __attribute__((aligned(1024))) char ring2[LDS_STAGE_MAX];
__shared__ __attribute__((aligned(1024))) char ring3[LDS_STAGE_MAX];

typedef float f32x16 __attribute__((ext_vector_type(16)));

// SiLU(g) * u with the hardware exp2 and reciprocal (about 1 ulp each; the
// result is rounded to bf16 afterwards)
__device__ __forceinline__ float swiglu_f(float g, float u) {
  const float e = __builtin_amdgcn_exp2f(-g * 1.4426950408889634f);
  return g * __builtin_amdgcn_rcpf(1.f + e) * u;
}

// 16-byte buffer -> LDS copy per lane (buffer_load_dwordx4 ... lds): lane l
// writes lds + 16 l, reading rsrc.base + voff + soff.  A non-template wrapper:
// the host compilation pass rejects this builtin inside a kernel template.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, void* lds_wave_base, int voff,
                                      int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds_wave_base, 16, voff, soff, 0, 0);
}

// raw buffer resource over [base, base + bytes); dword3 is the CDNA raw-buffer
// format (32-bit data, no swizzle)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14])
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Epilogue of the bf16 GEMM kernels.  The weight fragment is the MFMA's first
// operand, so acc[mi][ni] = W_frag X_frag^T: lane l holds token row
// mi*32 + l%32 and, for e = 4g + t, output column 8g + 4(l/32) + t of the
// fragment -- four consecutive columns per g.  MODE 0 pairs gate fragment f
// with up fragment f + NI/2 and writes SiLU(g) * u.  Each wavefront stages
// its 32-row slices through its own LDS region `reg` with 8-byte writes,
// reads them back as row-major 16-byte chunks and writes them with buffer
// stores, which drop the rows past the tile's last valid row (no branches,
// so all reads of a slice are in flight together).
template <int MODE, int MI, int NI>
__device__ __forceinline__ void store_tile(const f32x16 (&acc)[MI][NI], char* reg, uint16_t* C,
                                           int ldc, const Work& wk, int colbase, int lane) {
  constexpr int FO = MODE == 0 ? NI / 2 : NI;  // output fragments per wavefront
  constexpr int CWV = FO * 32;                 // output columns per wavefront
  constexpr int RS = CWV * 2 + 16;             // padded LDS row stride (bytes)
  constexpr int CPR = CWV / 8;                 // 16-byte chunks per row
  constexpr int NST = 32 * CPR / 64;           // chunks per lane per 32-row slice
  const int r32 = lane & 31, kh = lane >> 5;
  const __amdgpu_buffer_rsrc_t c_rs =
      make_rsrc(C + (size_t)wk.row0 * ldc, (uint32_t)wk.rows * (uint32_t)ldc * 2);
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
    for (int f = 0; f < FO; ++f)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
          v[t] = MODE == 0 ? swiglu_f(acc[mi][f][4 * g + t], acc[mi][f + NI / 2][4 * g + t])
                           : acc[mi][f][4 * g + t];
        const uint2 pk = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
        *reinterpret_cast<uint2*>(reg + r32 * RS + (f * 32 + 8 * g + 4 * kh) * 2) = pk;
      }
    // same wavefront: LDS order makes the writes visible to these reads
    u32x4 val[NST];
#pragma unroll
    for (int i = 0; i < NST; ++i) {
      const int lin = i * 64 + lane;
      val[i] = *reinterpret_cast<const u32x4*>(reg + (lin / CPR) * RS + (lin % CPR) * 16);
    }
#pragma unroll
    for (int i = 0; i < NST; ++i) {
      const int lin = i * 64 + lane;
      const int row = mi * 32 + lin / CPR;
      __builtin_amdgcn_raw_buffer_store_b128(val[i], c_rs, (row * ldc + colbase + (lin % CPR) * 8) * 2, 0, 0);
    }
  }
}

// MODE 0: A = x_perm [rows, d], W = w_gate_up [E, 2m, d], C = h [rows, m];
//         the B tile's first BN/2 rows are gate rows nt*BN/2.., the rest the
//         matching up rows m + nt*BN/2..; C gets BN/2 columns.  Wavefront w
//         owns h columns [w BN/8, (w+1) BN/8) of the tile: its gate and up
//         fragments hold the same (row, column) in the same registers.
// MODE 1: A = h [rows, m], W = w_down [E, d, m], C = y_perm [rows, d];
//         B rows nt*BN.., C gets BN columns; wavefront w owns [w BN/4, ..).
template <int MODE, int BM, int BN>
__global__ __launch_bounds__(NTHR, 1) void ffn_gemm_bf16_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ W, uint16_t* __restrict__ C,
    const Tiles tl, int d, int m, const Guard g) {
  if (guard_skip(g)) return;
  constexpr int MI = BM / 32;             // 32-row fragments per wave (all tile rows)
  constexpr int NI = BN / 128;            // 32-col fragments per wave
  constexpr int AG = BM / 16;             // 1 KB DMA groups (16 rows) of the A tile
  constexpr int BG = BN / 16;
  constexpr int GPW = (AG + BG) / 4;      // DMA instructions per wave per stage
  static_assert(AG % 4 == 0 && BG % 8 == 0, "groups split over 4 waves");
  static_assert(MODE == 1 || NI % 2 == 0, "gate/up fragments come in pairs");
  static_assert((BM + BN) * BK * 2 <= LDS_STAGE_MAX, "stage too large");

  Work wk;
  if (!find_work(tl, true, wk, ring3)) return;
  const int nt = wk.nt;
  const int Kdim = MODE == 0 ? d : m;
  const int ldc = MODE == 0 ? m : d;
  const uint16_t* Wexp = W + (size_t)wk.expert * (size_t)(MODE == 0 ? 2 * m : d) * Kdim;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);

  // ---- DMA: group g = 16 rows x 64 bytes; wave wv issues groups wv, wv+4, ...
  // of the A tile and of the B tile; lane -> row 16 g + lane/4, LDS chunk
  // lane%4, global chunk (lane%4) ^ ((row >> 2) & 3) -- the same for every
  // group of a lane since groups start at multiples of 16 rows.  Per-lane
  // byte offsets go in VGPRs; k and the group's row offset in the scalar
  // offset.
  const int lrow = lane >> 2;
  const int swz_c = (lane & 3) ^ ((lrow >> 2) & 3);
  // A: rows of this tile; padding rows (past wk.rows) re-read row 0
  const __amdgpu_buffer_rsrc_t a_rs = make_rsrc(A + (size_t)wk.row0 * Kdim, (uint32_t)wk.rows * Kdim * 2);
  int a_voff[AG / 4];
#pragma unroll
  for (int q = 0; q < AG / 4; ++q) {
    const int r = wv * 16 + lrow + 64 * q;
    a_voff[q] = ((r < wk.rows ? r : 0) * Kdim + swz_c * 8) * 2;
  }
  // B: the expert's weight matrix; for MODE 0 the up half (groups
  // q >= BG/8) lives m - BN/2 rows further down
  const int ncolsW = MODE == 0 ? 2 * m : d;
  const __amdgpu_buffer_rsrc_t b_rs = make_rsrc(Wexp, (uint32_t)ncolsW * Kdim * 2);
  const int b_voff = (((MODE == 0 ? nt * (BN / 2) : nt * BN) + wv * 16 + lrow) * Kdim + swz_c * 8) * 2;
  const int b_step = 64 * Kdim * 2;
  const int b_jump = MODE == 0 ? (m - BN / 2) * Kdim * 2 : 0;

  auto issue = [&](char* stage, int k0) {
#pragma unroll
    for (int q = 0; q < AG / 4; ++q) dma16(a_rs, stage + (wv + 4 * q) * 1024, a_voff[q], k0 * 2);
#pragma unroll
    for (int q = 0; q < BG / 4; ++q)
      dma16(b_rs, stage + BM * 64 + (wv + 4 * q) * 1024, b_voff,
            q * b_step + (q >= BG / 8 ? b_jump : 0) + k0 * 2);
  };

  f32x16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // ---- fragments.  32x32x16: lane l supplies row (l % 32), k = 8 (l / 32)
  // .. +8 of its substep, i.e. chunk 2 s + l/32 of the stage.  Fragment row
  // groups start at multiples of 32 rows, so the swizzle term is
  // ((l % 32) >> 2) & 3 for all of them: one per-lane base per substep.
  const int r32 = lane & 31, kh = lane >> 5;
  const int sw = (r32 >> 2) & 3;
  const int lane_off0 = r32 * 64 + ((kh ^ sw) << 4);
  const int lane_off1 = r32 * 64 + (((2 + kh) ^ sw) << 4);
  auto brow0 = [&](int ni) {
    int b;
    if (MODE == 0)  // half gate, half up, same h columns
      b = ni < NI / 2 ? wv * (BN / 8) + ni * 32 : BN / 2 + wv * (BN / 8) + (ni - NI / 2) * 32;
    else
      b = wv * (BN / 4) + ni * 32;
    return (BM + b) * 64;
  };
  auto load_frags = [&](const char* stage, int s, bf16x8 (&af)[MI], bf16x8 (&bfr)[NI]) {
    const char* base = stage + (s ? lane_off1 : lane_off0);
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) af[mi] = *reinterpret_cast<const bf16x8*>(base + mi * 32 * 64);
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) bfr[ni] = *reinterpret_cast<const bf16x8*>(base + brow0(ni));
  };
  auto mma = [&](const bf16x8 (&af)[MI], const bf16x8 (&bfr)[NI]) {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
        acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[ni], af[mi], acc[mi][ni], 0, 0, 0);
  };
  // Interleave the fragment reads of the next substep with the MFMAs of the
  // current one (one wavefront per SIMD: nothing else hides LDS latency).
  // The scheduling group pattern is MFMA x R, ds_read x 1, repeated.
  constexpr int NMF = MI * NI, NRD = MI + NI;
  constexpr int RPER = NMF / NRD > 0 ? NMF / NRD : 1;
  auto interleave = [&]() {
#pragma unroll
    for (int i = 0; i < NRD; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, RPER, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);     // DS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, NMF - RPER * NRD, 0);
  };

  // Pipeline: four LDS stages of BK = 32 k-values; stages it+1..it+3 are in
  // flight while stage it is consumed.  Each stage is two 16-wide substeps
  // with register double buffering:
  //   MFMA(substep 0 of it)  || read substep 1 of it
  //   wait for stage it+1, lgkmcnt(0), barrier (every wave is done with the
  //   stage of it, and stage it+1 has landed for every wave)
  //   refill the stage of it with it+4
  //   MFMA(substep 1 of it)  || read substep 0 of it+1
  // LEFT = stages allowed in flight at the wait (2 in the steady state);
  // LEFT < 0 marks the last iteration.
  bf16x8 a0[MI], b0[NI], a1[MI], b1[NI];
  auto step = [&](auto ISSUE, auto LEFT, int it, char* cur, char* nxt) {
    load_frags(cur, 1, a1, b1);
    mma(a0, b0);
    interleave();
    if constexpr (decltype(LEFT)::value >= 0) {
      wait_vmcnt<decltype(LEFT)::value * GPW>();
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): reads of `cur` are complete
      __builtin_amdgcn_s_barrier();
      if constexpr (decltype(ISSUE)::value) issue(cur, (it + 4) * BK);
      load_frags(nxt, 0, a0, b0);
    }
    mma(a1, b1);
    if constexpr (decltype(LEFT)::value >= 0) interleave();
  };
  using T0 = std::integral_constant<int, 0>;
  using T1 = std::integral_constant<int, 1>;
  using L2 = std::integral_constant<int, 2>;
  using L1 = std::integral_constant<int, 1>;
  using L0 = std::integral_constant<int, 0>;
  using LE = std::integral_constant<int, -1>;

  // Kdim / BK is a multiple of 4 (the entry point requires d and m to be
  // multiples of 128), so the ring position of every step is static
  const int nk = Kdim / BK;
  issue(ring0, 0);
  issue(ring1, BK);
  issue(ring2, 2 * BK);
  issue(ring3, 3 * BK);
  wait_vmcnt<3 * GPW>();
  __builtin_amdgcn_s_barrier();
  load_frags(ring0, 0, a0, b0);
  for (int it = 0; it + 4 < nk; it += 4) {  // branch-free body: every step refills
    step(T1{}, L2{}, it, ring0, ring1);
    step(T1{}, L2{}, it + 1, ring1, ring2);
    step(T1{}, L2{}, it + 2, ring2, ring3);
    step(T1{}, L2{}, it + 3, ring3, ring0);
  }
  step(T0{}, L2{}, nk - 4, ring0, ring1);
  step(T0{}, L1{}, nk - 3, ring1, ring2);
  step(T0{}, L0{}, nk - 2, ring2, ring3);
  step(T0{}, LE{}, nk - 1, ring3, ring0);

  // ---- epilogue, staged through this wavefront's part of ring0
  __syncthreads();  // every wave is done with the ring
  constexpr int RS_MAX = (BN / 4) * 2 + 16;
  static_assert(4 * 32 * RS_MAX <= LDS_STAGE_MAX, "epilogue staging fits in one ring stage");
  const int colbase = MODE == 0 ? nt * (BN / 2) + wv * (BN / 8) : nt * BN + wv * (BN / 4);
  store_tile<MODE, MI, NI>(acc, ring0 + wv * 32 * RS_MAX, C, ldc, wk, colbase, lane);
}

// ---------------------------------------------------------------------------
// Packed expert weights.  A [R, K] bf16 weight matrix is stored as MFMA
// fragments: the 16 bytes at element offset ((kb * (R / 32)) + rb) * 512 + 8 l
// hold row 32 rb + l % 32, columns 16 kb + 8 (l / 32) .. +8 -- exactly what
// lane l supplies as the first operand of v_mfma_f32_32x32x16_bf16.  Every
// fragment is 1 KB contiguous and the fragments of one 16-wide k-slice
// follow each other in row order, so a wavefront loads its weight operand
// straight into registers with fully coalesced 1 KB loads, and the weight
// rows of one tile and k-step are a few contiguous runs in HBM.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void pack_weights_kernel(const uint4* __restrict__ w, int R, int K,
                                                           size_t n_chunks, uint4* __restrict__ out) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;  // output chunk
  if (i >= n_chunks) return;
  const int l = (int)(i & 63);
  size_t f = i >> 6;  // fragment index over (expert, kb, rb)
  const int RB = R / 32, KB = K / 16;
  const int rb = (int)(f % RB);
  f /= RB;
  const int kb = (int)(f % KB);
  const size_t e = f / KB;
  const int row = rb * 32 + (l & 31);
  const int col8 = kb * 2 + (l >> 5);  // 8-element column chunk
  out[i] = w[(e * R + row) * (size_t)(K / 8) + col8];
}

// ---------------------------------------------------------------------------
// bf16 MFMA grouped GEMM on packed weights
//
// Same MFMA tiles, work items and epilogue as the kernel above; the weight
// operand bypasses LDS.  Per k-step of 32, wavefront wv loads its 2 x NI
// weight fragments (NI 32-row blocks x two 16-wide substeps, 1 KB each,
// fully coalesced) into a ring of four register stages, three k-steps
// ahead (issued as soon as a stage's registers are free, at the top of the
// k-step after their last use).  Only the token-row tile A, which all four wavefronts share, goes
// through LDS: global -> LDS transfers of whole 128-byte row segments
// (A stages of 64 k-values, 8 rows per wave instruction) into a ring of
// four stages, three stages (192 k-values) ahead.  In LDS a 128-byte row
// holds 8 chunks of 16 bytes, chunk c stored at c ^ ((row >> 1) & 7): the
// 16 rows read by one quarter-wavefront hit 16 distinct bank groups.
//
// Waits: the compiler waits for the weight registers where the MFMAs use
// them, but not for global -> LDS transfers, so every read of an A stage
// must follow a wait that covers this wavefront's transfers of that stage,
// and then a barrier (covering every wavefront's part).  In the loop the
// weight wait does it: the vector-memory counter completes in issue order,
// and stage j's transfers (issued at the end of k-step 2j - 7) precede the
// weights of k-step 2j - 1 (issued at its top, three steps earlier), whose
// MFMAs wait for them before the barrier that ends k-step 2j - 1.  Before
// stage 0 nothing has waited yet: the prologue waits explicitly.
// ---------------------------------------------------------------------------
constexpr int AK = 64;  // k-values per A stage

// LDS bytes per A stage: BM rows of AK bf16, and at least one wavefront's
// epilogue staging (32 rows of BN / 4 values plus padding); 1 KB multiples
template <int BM, int BN>
constexpr int a_slot() {
  constexpr int a = BM * AK * 2, e = 32 * ((BN / 4) * 2 + 16);
  return ((a > e ? a : e) + 1023) & ~1023;
}
// weight-register ring depth: 4 stages (three k-steps ahead) for 128-row
// tiles; 64-row tiles (few rows per expert: weight streaming) run 8 stages,
// seven k-steps ahead, to keep more weight bytes in flight
template <int BM>
constexpr int packed_nb() { return BM >= 128 ? 4 : 8; }

// AUX: the load's cache policy; 2 sets the non-temporal hint (weight tiles
// that no other token tile of the call reads again)
template <int AUX>
__device__ __forceinline__ u32x4 load_frag(__amdgpu_buffer_rsrc_t rs, int voff, int soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, AUX);
}

// One work item: the BM x BN output tile `wk` of one GEMM.  `aring` is the
// workgroup's LDS: four A stages of a_slot<BM, BN>() bytes.  The caller
// synchronises the workgroup before the item reuses it.
// With gather.src_of_row (gate/up only), A is the token matrix x [gather.T,
// d] and tile row r is token src_of_row[row0 + r] / gather.k: the dispatch
// gather happens in the token-row transfers, which take a per-lane offset
// anyway, and x_perm is never formed.
template <int MODE, int BM, int BN, int AUX = 0, int NB = packed_nb<BM>()>
__device__ __forceinline__ void packed_item(const uint16_t* __restrict__ A, const uint16_t* __restrict__ Wp,
                                            uint16_t* __restrict__ C, const Work wk, int d, int m,
                                            const RowGather gather, char* aring) {
  constexpr int MI = BM / 32;   // 32-row token fragments (all tile rows)
  constexpr int NI = BN / 128;  // 32-row weight fragments per wavefront
  constexpr int AGW = BM / 32;  // A transfers (8 rows x 128 B) per wavefront per stage
  static_assert(MI >= 1 && AGW >= 1 && (MODE == 1 || NI % 2 == 0), "tile shape");

  constexpr int ASLOT = a_slot<BM, BN>();
  char* const aring0 = aring;
  char* const aring1 = aring + ASLOT;
  char* const aring2 = aring + 2 * ASLOT;
  char* const aring3 = aring + 3 * ASLOT;

  const int nt = wk.nt;
  const int Kdim = MODE == 0 ? d : m;
  const int R = MODE == 0 ? 2 * m : d;  // rows of the expert's weight matrix
  const int nk = Kdim / BK;             // k-steps of 32: a multiple of 8
  const int ldc = MODE == 0 ? m : d;

  // the lane offsets below are recomputed per item: an opaque copy of the
  // thread index keeps them from being hoisted out of a persistent kernel's
  // item loop (where they would stay live across items and spill)
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);

  // ---- A: transfer q of wave wv covers tile rows 8 g .. 8 g + 7, g = wv + 4 q;
  // lane l fills LDS row 8 g + l / 8, physical chunk l % 8, with logical
  // chunk (l % 8) ^ ((row >> 1) & 7).  Padding rows re-read the tile's row 0
  // (gathered: token 0); a gathered token index outside [0, T) reads token 0.
  const bool gat = MODE == 0 && gather.src_of_row != nullptr;
  const __amdgpu_buffer_rsrc_t a_rs =
      gat ? make_rsrc(A, (uint32_t)gather.T * Kdim * 2)
          : make_rsrc(A + (size_t)wk.row0 * Kdim, (uint32_t)wk.rows * Kdim * 2);
  int a_voff[AGW];
#pragma unroll
  for (int q = 0; q < AGW; ++q) {
    const int row = 8 * (wv + 4 * q) + (lane >> 3);
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    int src = 0;
    if (gat) {
      if (row < wk.rows) src = gather.src_of_row[wk.row0 + row] / gather.k;
      if ((unsigned)src >= (unsigned)gather.T) src = 0;
    } else {
      src = row < wk.rows ? row : 0;
    }
    a_voff[q] = (src * Kdim + c * 8) * 2;
  }
  auto issue_a = [&](char* stage, int js) {
#pragma unroll
    for (int q = 0; q < AGW; ++q) dma16(a_rs, stage + (wv + 4 * q) * 1024, a_voff[q], js * AK * 2);
  };

  // ---- B: this wavefront's NI 32-row blocks of the expert's packed matrix
  const __amdgpu_buffer_rsrc_t b_rs =
      make_rsrc(Wp + (size_t)wk.expert * R * Kdim, (uint32_t)R * Kdim * 2);
  const int RB = R / 32;
  int rb[NI];
#pragma unroll
  for (int ni = 0; ni < NI; ++ni) {
    if (MODE == 0)  // half gate, half up rows of the same h columns
      rb[ni] = ni < NI / 2 ? (nt * (BN / 2) + wv * (BN / 8)) / 32 + ni
                           : (m + nt * (BN / 2) + wv * (BN / 8)) / 32 + ni - NI / 2;
    else
      rb[ni] = (nt * BN + wv * (BN / 4)) / 32 + ni;
  }
  const int b_voff = lane * 16;
  auto load_b = [&](u32x4 (&b)[2][NI], int ks) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) b[h][ni] = load_frag<AUX>(b_rs, b_voff, ((2 * ks + h) * RB + rb[ni]) * 1024);
  };

  f32x16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // ---- A fragments: lane l supplies row l % 32 of each 32-row block and
  // logical chunk 2 s + l / 32 of substep s (0..3) of the stage
  const int r32 = lane & 31, kh = lane >> 5;
  int a_lane[4];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) a_lane[s4] = r32 * 128 + (((2 * s4 + kh) ^ ((r32 >> 1) & 7)) << 4);
  // The pipeline runs with MA = the item's 32-row token blocks that hold
  // rows (a tile's last item of an expert is often short): blocks past them
  // would only multiply padding, so their fragment reads and MFMAs are left
  // out (their accumulators stay zero and their rows are not stored).
  static_assert(NB == 4 || NB == 8, "weight ring of 4 or 8 stages");
  constexpr int LA = NB - 1;  // weight lookahead in k-steps
  u32x4 bq[NB][2][NI];
  auto pipeline = [&](auto MAC) {
    constexpr int MA = decltype(MAC)::value;
    auto load_a = [&](const char* stage, int s4, bf16x8 (&af)[MI]) {
  #pragma unroll
      for (int mi = 0; mi < MA; ++mi)
        af[mi] = *reinterpret_cast<const bf16x8*>(stage + mi * 32 * 128 + a_lane[s4]);
    };
    auto mma = [&](const bf16x8 (&af)[MI], const u32x4 (&bfr)[NI]) {
  #pragma unroll
      for (int mi = 0; mi < MA; ++mi)
  #pragma unroll
        for (int ni = 0; ni < NI; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, bfr[ni]), af[mi],
                                                                acc[mi][ni], 0, 0, 0);
    };
    auto interleave = [&]() {
  #pragma unroll
      for (int i = 0; i < MA; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, NI, 0);        // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);         // DS read
      }
    };

    // ---- k-step i (32 k-values): A stage i / 2, substeps 2 (i % 2) and +1;
    // weights in register stage i % 4.  At the end of an A stage (odd i) the
    // next stage is awaited and the finished one refilled with stage + 4.
    //   ODD          i is the second half of an A stage
    //   ISSUE_A      refill the finished A stage
    //   ISSUE_B      load the weights of k-step i + 3
    //   LAST         the final k-step (nothing follows)
    bf16x8 a0[MI], a1[MI];
    // WAIT (8-stage ring only): at the barrier of an odd k-step, at most WAIT
    // younger vector-memory operations may be outstanding -- exactly the
    // ones issued after the transfers of the stage read next (see below)
    auto step = [&](auto ODD, auto ISSUE_A, auto ISSUE_B, auto LAST, auto WAIT, int i, char* cur,
                    char* nxt, const u32x4 (&bc)[2][NI], u32x4 (&bn)[2][NI]) {
      constexpr bool odd = decltype(ODD)::value;
      // the weight registers of k-step i - 1 are free: refill them first
      if constexpr (decltype(ISSUE_B)::value) load_b(bn, i + LA);
      __builtin_amdgcn_sched_barrier(0);
      load_a(cur, odd ? 3 : 1, a1);
      mma(a0, bc[0]);
      interleave();
      if constexpr (!decltype(LAST)::value) {
        if constexpr (odd) {
          // nxt's transfers are complete (see the waits above): with 4
          // weight stages the weight wait of this k-step's first MFMAs
          // covered them; with 8 the weights of k-step i were issued before
          // them, so the wait is explicit
          if constexpr (NB == 8) wait_vmcnt<decltype(WAIT)::value>();
          __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): reads of `cur` are complete
          __builtin_amdgcn_s_barrier();
          __builtin_amdgcn_sched_barrier(0);
          if constexpr (decltype(ISSUE_A)::value) issue_a(cur, i / 2 + 4);
          __builtin_amdgcn_sched_barrier(0);
        }
        load_a(odd ? nxt : cur, odd ? 0 : 2, a0);
      }
      mma(a1, bc[1]);
      if constexpr (!decltype(LAST)::value) interleave();
    };
    using F = std::integral_constant<bool, false>;
    using Tr = std::integral_constant<bool, true>;

    // body of 8 k-steps = 4 A stages in slots 0..3; every issue active.
    // k-step i reads weight slot i % NB and refills slot (i - 1) % NB with
    // k-step i + LA.  Stage j's transfers leave at the end of k-step 2j - 7;
    // by the barrier of k-step 2j - 1 the loads issued after them are the
    // weights of six k-steps and the transfers of two stages.
    using WB = std::integral_constant<int, 12 * NI + 2 * AGW>;
    auto body = [&](int i) {
      step(F{}, F{}, Tr{}, F{}, WB{}, i + 0, aring0, aring0, bq[0 % NB], bq[(NB - 1) % NB]);
      step(Tr{}, Tr{}, Tr{}, F{}, WB{}, i + 1, aring0, aring1, bq[1 % NB], bq[0 % NB]);
      step(F{}, F{}, Tr{}, F{}, WB{}, i + 2, aring1, aring1, bq[2 % NB], bq[1 % NB]);
      step(Tr{}, Tr{}, Tr{}, F{}, WB{}, i + 3, aring1, aring2, bq[3 % NB], bq[2 % NB]);
      step(F{}, F{}, Tr{}, F{}, WB{}, i + 4, aring2, aring2, bq[4 % NB], bq[3 % NB]);
      step(Tr{}, Tr{}, Tr{}, F{}, WB{}, i + 5, aring2, aring3, bq[5 % NB], bq[4 % NB]);
      step(F{}, F{}, Tr{}, F{}, WB{}, i + 6, aring3, aring3, bq[6 % NB], bq[5 % NB]);
      step(Tr{}, Tr{}, Tr{}, F{}, WB{}, i + 7, aring3, aring0, bq[7 % NB], bq[6 % NB]);
    };

    issue_a(aring0, 0);
    issue_a(aring1, 1);
    issue_a(aring2, 2);
    issue_a(aring3, 3);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int q = 0; q < LA; ++q) load_b(bq[q], q);
    __builtin_amdgcn_sched_barrier(0);
    // stage 0 complete: its transfers precede the 3 AGW transfers of stages
    // 1..3 and the 2 NI LA weight loads of k-steps 0..LA-1
    wait_vmcnt<3 * AGW + 2 * NI * LA>();
    __builtin_amdgcn_s_barrier();
    load_a(aring0, 0, a0);
    int i = 0;
    for (; i + 8 < nk; i += 8) body(i);
    // last 8 k-steps: no A refills; weights up to k-step nk - 1 (tail step t
    // loads while t + LA <= 7).  With 8 weight stages only t = 0 loads, and
    // the odd tail barriers wait for stages issued in the body: after them
    // come 10 NI + 2 AGW, 6 NI + AGW and 2 NI operations (t = 1, 3, 5);
    // when the body did not run (nk = 8) more follow, so these bounds still
    // suffice
    constexpr bool B1 = 1 + LA <= 7, B2 = 2 + LA <= 7, B3 = 3 + LA <= 7, B4 = 4 + LA <= 7;
    using T1 = std::integral_constant<int, 10 * NI + 2 * AGW>;
    using T3 = std::integral_constant<int, 6 * NI + AGW>;
    using T5 = std::integral_constant<int, 2 * NI>;
    using BC1 = std::integral_constant<bool, B1>;
    using BC2 = std::integral_constant<bool, B2>;
    using BC3 = std::integral_constant<bool, B3>;
    using BC4 = std::integral_constant<bool, B4>;
    step(F{}, F{}, Tr{}, F{}, WB{}, i + 0, aring0, aring0, bq[0 % NB], bq[(NB - 1) % NB]);
    step(Tr{}, F{}, BC1{}, F{}, T1{}, i + 1, aring0, aring1, bq[1 % NB], bq[0 % NB]);
    step(F{}, F{}, BC2{}, F{}, WB{}, i + 2, aring1, aring1, bq[2 % NB], bq[1 % NB]);
    step(Tr{}, F{}, BC3{}, F{}, T3{}, i + 3, aring1, aring2, bq[3 % NB], bq[2 % NB]);
    step(F{}, F{}, BC4{}, F{}, WB{}, i + 4, aring2, aring2, bq[4 % NB], bq[3 % NB]);
    step(Tr{}, F{}, F{}, F{}, T5{}, i + 5, aring2, aring3, bq[5 % NB], bq[4 % NB]);
    step(F{}, F{}, F{}, F{}, WB{}, i + 6, aring3, aring3, bq[6 % NB], bq[5 % NB]);
    step(Tr{}, F{}, F{}, Tr{}, WB{}, i + 7, aring3, aring0, bq[7 % NB], bq[6 % NB]);
  };
  const int ma = (wk.rows + 31) >> 5;
  if constexpr (MI == 4) {
    if (ma >= 4)
      pipeline(std::integral_constant<int, 4>{});
    else if (ma == 3)
      pipeline(std::integral_constant<int, 3>{});
    else if (ma == 2)
      pipeline(std::integral_constant<int, 2>{});
    else
      pipeline(std::integral_constant<int, 1>{});
  } else if constexpr (MI == 2) {
    if (ma >= 2)
      pipeline(std::integral_constant<int, 2>{});
    else
      pipeline(std::integral_constant<int, 1>{});
  } else {
    pipeline(std::integral_constant<int, MI>{});
  }

  // ---- epilogue, wave w staged through A slot w
  __syncthreads();  // every wave is done with the A ring
  constexpr int RS = (BN / 4) * 2 + 16;
  static_assert(32 * RS <= ASLOT, "epilogue staging fits one wave per A slot");
  char* reg = wv == 0 ? aring0 : wv == 1 ? aring1 : wv == 2 ? aring2 : aring3;
  const int colbase = MODE == 0 ? nt * (BN / 2) + wv * (BN / 8) : nt * BN + wv * (BN / 4);
  store_tile<MODE, MI, NI>(acc, reg, C, ldc, wk, colbase, lane);
}

// Two launches on packed weights (one per GEMM): items from find_work.
template <int MODE, int BM>
__global__ __launch_bounds__(NTHR, 2) void ffn_gemm_packed_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ Wp, uint16_t* __restrict__ C,
    const Tiles tl, int d, int m, const RowGather gather, const Guard g) {
  if (guard_skip(g)) return;
  __shared__ __attribute__((aligned(1024))) char aring[4 * a_slot<BM, 256>()];
  Work wk;
  if (!find_work(tl, true, wk, aring)) return;
  packed_item<MODE, BM, 256>(A, Wp, C, wk, d, m, gather, aring);
}

// ---------------------------------------------------------------------------
// Persistent expert FFN: one launch runs both GEMMs, per XCD.
//
// The m-tiles (numbered expert-major, as in find_work) are split into n_xcc
// contiguous ranges of about equal estimated cost, one per XCD; a workgroup
// serves the range of the XCD it runs on (the XCC_ID hardware register),
// claiming items from that XCD's counter: first the nn0 gate/up items of
// every tile in the range (expert-major, then n-tile, then m-tile, so the
// m-tiles that share a weight tile run together), then its nn1 down items.
// A down item of tile t reads the h rows of t, written by the nn0 gate/up
// items of t, which ran on the same XCD and so behind the same L2: each of
// them waits for its stores (vmcnt 0), then bumps done[t]; the down item's
// workgroup polls done[t] until it reaches nn0 and only then loads h.  No
// vector L1 can hold a stale h line: h lines of a tile are first read after
// its count is complete, and different tiles and n-tiles never share a line
// (h rows are whole 128-byte lines, n-tile column blocks are 256 bytes).
// The wait always ends: within a queue items are claimed in order, so when a
// down item is claimed every gate/up item of its range has been claimed by a
// running workgroup, and gate/up items wait for nothing.  The poll is still
// bounded (FFN_SPIN_LIMIT) so that a broken invariant cannot hang the device;
// a wait that runs out is counted, so that moe_ffn_status reports it.
//   ctr[16 x]      claim counter of XCD x (the 64 bytes from 16 x are written
//   ctr[16 x + 1]  items completed on XCD x       only by workgroups of XCD x)
//   ctr[16 x + 2]  waits on XCD x that ran out of polls
//   ctr[16 x + 3]  items in the whole plan (every workgroup of XCD x stores it)
//   ctr[FFN_CTR_PATH]  launch path of the call (FFN_PATH_*; set by clear_kernel)
//   ctr[128 + t]   gate/up items of m-tile t completed
// ctr (128 + max_tiles ints) is zeroed by clear_kernel before each launch.
// A call ran every item of its plan exactly when no wait ran out and the
// completed counts add up to the plan: an XCD that received no workgroup
// leaves its items unclaimed and the sum short.
// Cost of a tile: 4 + its active 32-row blocks; the first tile of an expert
// costs more for the weight fetch that its later m-tiles find in L2: 2 with
// 128-row tiles, a whole tile's cost with 64-row tiles (few rows per
// expert, where an XCD's time follows the weight bytes it streams).  (Claiming
// the next item while the current one runs does not pay: the claim is older
// than the item's transfers, so the first counted wait of the pipeline waits
// for it too.)
// ---------------------------------------------------------------------------
constexpr int FFN_MAXE = 1024;
constexpr int FFN_SPIN_LIMIT = 1 << 22;
constexpr int FFN_CTR_TILES = 128;  // ctr index of done[0]
constexpr int FFN_CTR_PATH = 5;     // in XCD 0's block, written only by clear_kernel

struct XcdRange {
  int a0, a1;  // tiles [a0, a1) of this XCD
};

// tstart[e] = first m-tile of expert e (experts >= Klim have none),
// tstart[E] = the tile count; returns this XCD's tile range.  NT: threads of
// the workgroup (E <= 4 NT); part: 2 NT / 64 + 3 ints of LDS.
template <int NT>
__device__ XcdRange plan_tiles(const Tiles& tl, int xcc, int n_xcc, int* tstart, int* part) {
  constexpr int NW = NT / 64;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  int& s_klim = part[2 * NW];
  int& s_a0 = part[2 * NW + 1];
  int& s_a1 = part[2 * NW + 2];
  // the prefix lengths and the expert offsets are loaded together, before
  // the first barrier (their latencies overlap)
  int mx = 0;
  if (tl.K_dev)
    for (int i = tid; i < tl.n_K; i += NT) mx = max(mx, tl.K_dev[i]);
  // offsets[4 tid .. 4 tid + 4], indices clamped to E (E <= 4 NT): five
  // loads without a branch between them
  int ofs[5], rows[4];
#pragma unroll
  for (int q = 0; q < 5; ++q) ofs[q] = tl.offsets[min(4 * tid + q, tl.E)];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int lo = clampi(ofs[q], 0, tl.rows_max);
    rows[q] = 4 * tid + q < tl.E ? clampi(ofs[q + 1], lo, tl.rows_max) - lo : 0;
  }
  if (tid == 0) s_klim = 0;
  __syncthreads();
  if (tl.K_dev && mx > 0) atomicMax(&s_klim, mx);
  __syncthreads();
  const int Klim = tl.K_dev ? clampi(s_klim, tl.kmin, tl.E) : tl.E;
  constexpr int FULL = 4;  // + BM / 32 below
  const int full_cost = FULL + tl.bm / 32, bonus = tl.bm == 64 ? full_cost : 2;
  int cnt[4], cost[4], lc = 0, lw = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int c = 4 * tid + q < Klim ? (rows[q] + tl.bm - 1) / tl.bm : 0;
    cnt[q] = c;
    cost[q] = c == 0 ? 0 : bonus + (c - 1) * full_cost + FULL + (rows[q] - (c - 1) * tl.bm + 31) / 32;
    lc += c;
    lw += cost[q];
  }
  int ic = lc, iw = lw;  // inclusive scans over the wavefront
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int yc = __shfl_up(ic, off, 64), yw = __shfl_up(iw, off, 64);
    if (lane >= off) {
      ic += yc;
      iw += yw;
    }
  }
  if (lane == 63) {
    part[wv] = ic;
    part[NW + wv] = iw;
  }
  __syncthreads();
  int bc = 0, bw = 0, total = 0, W = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    if (i < wv) {
      bc += part[i];
      bw += part[NW + i];
    }
    total += part[i];
    W += part[NW + i];
  }
  total = min(total, tl.max_tiles);
  // cost boundaries of this XCD; A(C) = tiles whose cumulative cost is <= C
  const int C0 = (int)((long long)xcc * W / n_xcc), C1 = (int)((long long)(xcc + 1) * W / n_xcc);
  if (tid == 0) {
    s_a0 = xcc == 0 ? 0 : total;
    s_a1 = total;
  }
  __syncthreads();
  int start = bc + ic - lc, P = bw + iw - lw;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = 4 * tid + q;
    if (e < tl.E) tstart[e] = min(start, total);
    if (cnt[q] > 0) {
      // tiles of this expert counted by A(C) for P <= C < P + cost
      auto count = [&](int C) { return C - P - bonus < 0 ? 0 : min((C - P - bonus) / full_cost, cnt[q] - 1); };
      if (xcc > 0 && P <= C0 && C0 < P + cost[q]) s_a0 = min(start + count(C0), total);
      if (xcc + 1 < n_xcc && P <= C1 && C1 < P + cost[q]) s_a1 = min(start + count(C1), total);
    }
    start += cnt[q];
    P += cost[q];
  }
  if (tid == 0) tstart[tl.E] = total;
  __syncthreads();
  return XcdRange{s_a0, s_a1};
}

// zeroes the n counters and records the launch path of the call
__global__ void clear_kernel(int* __restrict__ p, int n, int path, const Guard g) {
  if (guard_skip(g)) return;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    p[i] = i == FFN_CTR_PATH ? path : 0;
}

// status[0] waits that ran out, [1] items completed, [2] items planned,
// [3] launch path, summed over the XCD blocks of the counter header
__global__ void ffn_status_kernel(const int* __restrict__ ctr, int32_t* __restrict__ status) {
  if (threadIdx.x != 0) return;
  int gave_up = 0, done = 0, planned = 0;
  for (int x = 0; x < 8; ++x) {
    done += ctr[16 * x + 1];
    gave_up += ctr[16 * x + 2];
    planned = max(planned, ctr[16 * x + 3]);
  }
  status[0] = gave_up;
  status[1] = done;
  status[2] = planned;
  status[3] = ctr[FFN_CTR_PATH];
}

// Item j of an XCD's queue (n_gu gate/up items first, then the down items;
// nn0 / nn1 n-tiles per GEMM): its work item, its m-tile t, and whether its
// expert's weights stream with the non-temporal hint -- an expert whose
// rows fit one m-tile has no other tile that reads its weights again (RCEP
// span, 512 rows over 85 experts: 169 -> 153 us); the weights of experts
// with several m-tiles keep the default policy, so that the m-tiles that run
// together share each fetch in L2.
struct Item {
  Work wk;
  int t;
  bool down, stream;
};
__device__ __forceinline__ Item decode_item(const Tiles& tl, const XcdRange& rg, const int* s_tstart, int j,
                                            int n_gu, int nn1, int bm) {
  Item it;
  it.down = j >= n_gu;
  const int nn = it.down ? nn1 : tl.nn;
  const int jm = it.down ? j - n_gu : j;
  // the expert holding tile a0 + jm / nn; its tiles in this range are
  // [t_lo, t_lo + c), items [nn (t_lo - a0), nn (t_lo - a0 + c))
  const int tq = rg.a0 + jm / nn;
  int a = 0, b = tl.E;  // tstart[a] <= tq < tstart[b]
  while (b - a > 1) {
    const int mid = (a + b) >> 1;
    if (s_tstart[mid] <= tq) a = mid; else b = mid;
  }
  const int t_lo = max(s_tstart[a], rg.a0);
  const int c = min(s_tstart[a + 1], rg.a1) - t_lo;
  const int o = jm - nn * (t_lo - rg.a0);
  it.t = t_lo + o % c;
  const int lo = clampi(tl.offsets[a], 0, tl.rows_max);
  const int hi = clampi(tl.offsets[a + 1], lo, tl.rows_max);
  const int r0 = lo + (it.t - s_tstart[a]) * bm;
  it.wk.expert = __builtin_amdgcn_readfirstlane(a);
  it.wk.row0 = __builtin_amdgcn_readfirstlane(r0);
  it.wk.rows = __builtin_amdgcn_readfirstlane(min(bm, hi - r0));
  it.wk.nt = __builtin_amdgcn_readfirstlane(o / c);
  it.stream = c == 1 && s_tstart[a + 1] - s_tstart[a] == 1;
  return it;
}

// gate/up item done: this wavefront's h stores have reached L2 (vmcnt 0),
// then, after the barrier, one thread counts the item for its tile
__device__ __forceinline__ void gate_up_done(int* done) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(done, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// down item: one thread polls its tile's gate/up count (bounded; a wait that
// runs out is counted in `gave_up`), then the workgroup may load h
__device__ __forceinline__ void wait_gate_up(const int* done, int nn0, int* gave_up) {
  if (threadIdx.x == 0) {
    bool ready = false;
    for (int n = 0; n < FFN_SPIN_LIMIT && !ready; ++n) {
      ready = __hip_atomic_load(done, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= nn0;
      if (!ready) __builtin_amdgcn_s_sleep(4);
    }
    if (!ready) __hip_atomic_fetch_add(gave_up, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
}

template <int BM, int AUX, int BN1>
__global__ __launch_bounds__(NTHR, 2) void ffn_fused_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ Wgu, const uint16_t* __restrict__ Wdn,
    uint16_t* __restrict__ H, uint16_t* __restrict__ Y, const Tiles tl, int nn1, int d, int m,
    const RowGather gather, int n_xcc, int* __restrict__ ctr, const Guard g) {
  if (guard_skip(g)) return;
  constexpr int BN = 256;
  constexpr int ASLOT = a_slot<BM, BN>();
  __shared__ __attribute__((aligned(1024))) char aring[4 * ASLOT];
  __shared__ int s_tstart[FFN_MAXE + 1];
  __shared__ int s_part[2 * (NTHR / 64) + 3];
  __shared__ int s_item;

  // the XCD this workgroup runs on (hardware register XCC_ID, bits 3:0)
  const int xcc = (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) % (unsigned)n_xcc);
  const XcdRange rg = plan_tiles<NTHR>(tl, xcc, n_xcc, s_tstart, s_part);
  const int ntile = rg.a1 - rg.a0;
  const int n_gu = ntile * tl.nn, n_all = n_gu + ntile * nn1;
  const int tid = threadIdx.x;
  int* const claim = ctr + 16 * xcc;
  if (tid == 0)  // every workgroup of this XCD stores the same value
    __hip_atomic_store(claim + 3, s_tstart[tl.E] * (tl.nn + nn1), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  for (;;) {
    __syncthreads();  // the previous item is done with LDS and s_item
    if (tid == 0) s_item = atomicAdd(claim, 1);
    __syncthreads();
    const int j = __builtin_amdgcn_readfirstlane(s_item);
    if (j >= n_all) break;
    const Item it = decode_item(tl, rg, s_tstart, j, n_gu, nn1, BM);
    int* const done = ctr + FFN_CTR_TILES + it.t;
    const bool stream = AUX == 2 || it.stream;
    if (!it.down) {
      if (stream)
        packed_item<0, BM, BN, 2>(X, Wgu, H, it.wk, d, m, gather, aring);
      else if constexpr (AUX != 2)
        packed_item<0, BM, BN, AUX>(X, Wgu, H, it.wk, d, m, gather, aring);
      gate_up_done(done);
    } else {
      wait_gate_up(done, tl.nn, claim + 2);
      if (stream)
        packed_item<1, BM, BN1, 2>(H, Wdn, Y, it.wk, d, m, RowGather{nullptr, 1, 0}, aring);
      else if constexpr (AUX != 2)
        packed_item<1, BM, BN1, AUX>(H, Wdn, Y, it.wk, d, m, RowGather{nullptr, 1, 0}, aring);
    }
    if (tid == 0) __hip_atomic_fetch_add(claim + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// ---------------------------------------------------------------------------
// Persistent expert FFN with alternating wavefronts (128-row token tiles when
// both weight matrices have a multiple of 512 rows).
//
// One workgroup of 8 wavefronts per compute unit computes a 128 x 512 tile
// (gate/up: 256 gate rows and their 256 up rows; down: 512 rows of w_down).
// Wavefront w owns all 128 token rows and weight rows [64 w, 64 w + 64) --
// the same 128 x 64 per wavefront, registers and fragment layout as the
// four-wavefront items above, so the results are bitwise the same -- and
// the token tile in LDS is shared by all eight.  Each SIMD holds two of the
// wavefronts (group 0 and group 1, from the hardware SIMD id).  Per k-step
// of 32 a wavefront runs a memory phase (refill of a token stage, the
// weights of k-step + 3, the LDS reads of its token fragments) and an MFMA
// phase, separated by workgroup barriers; group 1 starts one phase late, so
// while one wavefront of a SIMD runs its MFMAs the other issues its loads.
// (Dense Qwen3-VL layer, in-process against the two-workgroup kernel:
// 2048 rows 292 -> 287 us, 4096 rows 388 -> 377, 8192 rows 659 -> 629,
// 16384 rows 1220 -> 1153.)
// The four token stages are separate LDS arrays, so the compiler can tell
// that a refill does not write the stage being read, and does not wait for
// the refill's transfers before those reads.
// ---------------------------------------------------------------------------
constexpr int PP_THR = 512;
constexpr int PP_SLOT = 128 * AK * 2;  // one token stage: 128 rows x 64 k-values

template <int MODE, int AUX>
__device__ __forceinline__ void pingpong_item(const uint16_t* __restrict__ A, const uint16_t* __restrict__ Wp,
                                              uint16_t* __restrict__ C, const Work wk, int d, int m,
                                              const RowGather gather, char* st0, char* st1, char* st2,
                                              char* st3, int grp) {
  constexpr int MI = 4, NI = 2, AGW = 2, LA = 3;
  const int nt = wk.nt;
  const int Kdim = MODE == 0 ? d : m;
  const int R = MODE == 0 ? 2 * m : d;
  const int nk = Kdim / BK;  // a multiple of 8
  const int ldc = MODE == 0 ? m : d;
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));  // keep the per-item offsets out of the item loop
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);

  // ---- token rows: transfer q of wave wv covers tile rows 8 g .. 8 g + 7,
  // g = wv + 8 q; lane l fills row 8 g + l / 8, physical chunk l % 8, with
  // logical chunk (l % 8) ^ ((row >> 1) & 7) (as in packed_item)
  const bool gat = MODE == 0 && gather.src_of_row != nullptr;
  const __amdgpu_buffer_rsrc_t a_rs =
      gat ? make_rsrc(A, (uint32_t)gather.T * Kdim * 2)
          : make_rsrc(A + (size_t)wk.row0 * Kdim, (uint32_t)wk.rows * Kdim * 2);
  int a_voff[AGW];
#pragma unroll
  for (int q = 0; q < AGW; ++q) {
    const int row = 8 * (wv + 8 * q) + (lane >> 3);
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    int src = 0;
    if (gat) {
      if (row < wk.rows) src = gather.src_of_row[wk.row0 + row] / gather.k;
      if ((unsigned)src >= (unsigned)gather.T) src = 0;
    } else {
      src = row < wk.rows ? row : 0;
    }
    a_voff[q] = (src * Kdim + c * 8) * 2;
  }
  auto issue_a = [&](char* stage, int js) {
#pragma unroll
    for (int q = 0; q < AGW; ++q) dma16(a_rs, stage + (wv + 8 * q) * 1024, a_voff[q], js * AK * 2);
  };

  // ---- weights: gate/up, 32 gate rows and the matching 32 up rows; down,
  // 64 consecutive rows
  const __amdgpu_buffer_rsrc_t b_rs =
      make_rsrc(Wp + (size_t)wk.expert * R * Kdim, (uint32_t)R * Kdim * 2);
  const int RB = R / 32;
  const int rb0 = MODE == 0 ? nt * 8 + wv : nt * 16 + 2 * wv;
  const int rb1 = MODE == 0 ? m / 32 + nt * 8 + wv : rb0 + 1;
  const int b_voff = lane * 16;
  auto load_b = [&](u32x4 (&b)[2][NI], int ks) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      b[h][0] = load_frag<AUX>(b_rs, b_voff, ((2 * ks + h) * RB + rb0) * 1024);
      b[h][1] = load_frag<AUX>(b_rs, b_voff, ((2 * ks + h) * RB + rb1) * 1024);
    }
  };

  f32x16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int r32 = lane & 31, kh = lane >> 5;
  int a_lane[4];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) a_lane[s4] = r32 * 128 + (((2 * s4 + kh) ^ ((r32 >> 1) & 7)) << 4);

  u32x4 bq[4][2][NI];
  // The wait before reading the next token stage (at odd k-step i, for the
  // stage read from k-step i + 1) may leave the younger loads outstanding:
  // at least the weights of the last five k-steps (the fewest, at the end
  // of the loop; elsewhere also one or two stages' transfers, whose waits
  // then complete earlier than needed).
  constexpr int WAIT = 5 * 2 * NI;
  auto pipeline = [&](auto MAC) {
    constexpr int MA = decltype(MAC)::value;  // 32-row token blocks holding rows
    bf16x8 af[2][MI];
    // k-step i.  Memory phase: the refill of slot `rs` with stage i / 2 + 3
    // (even i), the weights of k-step i + 3 into `bn`, at odd i the wait for
    // the next stage, the token fragments of k-step i from stage `cur`.
    // Then a barrier, the MFMA phase with the weights `bc`, a barrier.
    auto step = [&](auto ODD, auto REFILL, auto LOADB, int i, char* cur, char* rs,
                    const u32x4 (&bc)[2][NI], u32x4 (&bn)[2][NI]) {
      if constexpr (decltype(REFILL)::value) issue_a(rs, i / 2 + 3);
      if constexpr (decltype(LOADB)::value) load_b(bn, i + LA);
      if constexpr (decltype(ODD)::value) wait_vmcnt<WAIT>();
      __builtin_amdgcn_sched_barrier(0);
      constexpr int so = decltype(ODD)::value ? 2 : 0;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int mi = 0; mi < MA; ++mi)
          af[h][mi] = *reinterpret_cast<const bf16x8*>(cur + mi * 32 * 128 + a_lane[so + h]);
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int mi = 0; mi < MA; ++mi)
#pragma unroll
          for (int ni = 0; ni < NI; ++ni)
            acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, bc[h][ni]),
                                                                  af[h][mi], acc[mi][ni], 0, 0, 0);
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
    };
    using F = std::integral_constant<bool, false>;
    using Tr = std::integral_constant<bool, true>;

    // stages 0..2 here; k-step i (even) refills slot (i / 2 + 3) % 4 with
    // stage i / 2 + 3 while that stage exists (at i = 0 slot 3 is empty)
    issue_a(st0, 0);
    issue_a(st1, 1);
    issue_a(st2, 2);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int q = 0; q < LA; ++q) load_b(bq[q], q);
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<2 * AGW + 2 * NI * LA>();  // stage 0 (younger: stages 1, 2, three k-steps of weights)
    __builtin_amdgcn_s_barrier();
    if (grp) __builtin_amdgcn_s_barrier();  // group 1 runs one phase behind
    __builtin_amdgcn_sched_barrier(0);
    int i = 0;
    for (; i + 8 < nk; i += 8) {
      step(F{}, Tr{}, Tr{}, i + 0, st0, st3, bq[0], bq[3]);
      step(Tr{}, F{}, Tr{}, i + 1, st0, st0, bq[1], bq[0]);
      step(F{}, Tr{}, Tr{}, i + 2, st1, st0, bq[2], bq[1]);
      step(Tr{}, F{}, Tr{}, i + 3, st1, st1, bq[3], bq[2]);
      step(F{}, Tr{}, Tr{}, i + 4, st2, st1, bq[0], bq[3]);
      step(Tr{}, F{}, Tr{}, i + 5, st2, st2, bq[1], bq[0]);
      step(F{}, Tr{}, Tr{}, i + 6, st3, st2, bq[2], bq[1]);
      step(Tr{}, F{}, Tr{}, i + 7, st3, st3, bq[3], bq[2]);
    }
    // last 8 k-steps: the last stage leaves at the first, weights up to nk - 1
    step(F{}, Tr{}, Tr{}, i + 0, st0, st3, bq[0], bq[3]);
    step(Tr{}, F{}, Tr{}, i + 1, st0, st0, bq[1], bq[0]);
    step(F{}, F{}, Tr{}, i + 2, st1, st0, bq[2], bq[1]);
    step(Tr{}, F{}, Tr{}, i + 3, st1, st1, bq[3], bq[2]);
    step(F{}, F{}, Tr{}, i + 4, st2, st1, bq[0], bq[3]);
    step(Tr{}, F{}, F{}, i + 5, st2, st2, bq[1], bq[0]);
    step(F{}, F{}, F{}, i + 6, st3, st2, bq[2], bq[1]);
    step(Tr{}, F{}, F{}, i + 7, st3, st3, bq[3], bq[2]);
    if (!grp) __builtin_amdgcn_s_barrier();  // group 0 catches up: equal barrier counts
  };
  const int ma = (wk.rows + 31) >> 5;
  if (ma >= 4)
    pipeline(std::integral_constant<int, 4>{});
  else if (ma == 3)
    pipeline(std::integral_constant<int, 3>{});
  else if (ma == 2)
    pipeline(std::integral_constant<int, 2>{});
  else
    pipeline(std::integral_constant<int, 1>{});

  // epilogue: every wavefront has passed the last barrier after its last LDS
  // read; wavefront w stages its slice through half w / 4 of stage slot w % 4
  char* reg = ((wv & 3) == 0 ? st0 : (wv & 3) == 1 ? st1 : (wv & 3) == 2 ? st2 : st3) + (wv >> 2) * (PP_SLOT / 2);
  const int colbase = MODE == 0 ? nt * 256 + 32 * wv : nt * 512 + 64 * wv;
  store_tile<MODE, MI, NI>(acc, reg, C, ldc, wk, colbase, lane);
}

// The persistent loop of ffn_fused_kernel with 128 x 512 tiles on
// pingpong_item: tl.nn = 2 m / 512 gate/up and nn1 = d / 512 down n-tiles.
__global__ __launch_bounds__(PP_THR, 1) void ffn_pingpong_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ Wgu, const uint16_t* __restrict__ Wdn,
    uint16_t* __restrict__ H, uint16_t* __restrict__ Y, const Tiles tl, int nn1, int d, int m,
    const RowGather gather, int n_xcc, int* __restrict__ ctr, const Guard g) {
  if (guard_skip(g)) return;
  constexpr int BM = 128;
  __shared__ __attribute__((aligned(1024))) char st0[PP_SLOT];
  __shared__ __attribute__((aligned(1024))) char st1[PP_SLOT];
  __shared__ __attribute__((aligned(1024))) char st2[PP_SLOT];
  __shared__ __attribute__((aligned(1024))) char st3[PP_SLOT];
  __shared__ int s_tstart[FFN_MAXE + 1];
  __shared__ int s_part[2 * (PP_THR / 64) + 3];
  __shared__ int s_item;
  __shared__ int s_simd[PP_THR / 64];

  const int tid = threadIdx.x;
  // the SIMD of each wavefront (hardware register HW_ID, bits 5:4)
  if ((tid & 63) == 0) s_simd[tid >> 6] = (int)(__builtin_amdgcn_s_getreg((1 << 11) | (4 << 6) | 4) & 3);
  const int xcc = (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) % (unsigned)n_xcc);
  const XcdRange rg = plan_tiles<PP_THR>(tl, xcc, n_xcc, s_tstart, s_part);  // its barriers publish s_simd
  // group 1: a lower-numbered wavefront shares this one's SIMD (the barrier
  // counts of pingpong_item do not depend on the groups)
  int grp = 0;
  for (int v = 0; v < (tid >> 6); ++v) grp |= s_simd[v] == s_simd[tid >> 6] ? 1 : 0;
  grp = __builtin_amdgcn_readfirstlane(grp);
  const int ntile = rg.a1 - rg.a0;
  const int n_gu = ntile * tl.nn, n_all = n_gu + ntile * nn1;
  int* const claim = ctr + 16 * xcc;
  if (tid == 0)
    __hip_atomic_store(claim + 3, s_tstart[tl.E] * (tl.nn + nn1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (;;) {
    __syncthreads();  // the previous item is done with LDS and s_item
    if (tid == 0) s_item = atomicAdd(claim, 1);
    __syncthreads();
    const int j = __builtin_amdgcn_readfirstlane(s_item);
    if (j >= n_all) break;
    const Item it = decode_item(tl, rg, s_tstart, j, n_gu, nn1, BM);
    int* const done = ctr + FFN_CTR_TILES + it.t;
    if (!it.down) {
      if (it.stream)
        pingpong_item<0, 2>(X, Wgu, H, it.wk, d, m, gather, st0, st1, st2, st3, grp);
      else
        pingpong_item<0, 0>(X, Wgu, H, it.wk, d, m, gather, st0, st1, st2, st3, grp);
      gate_up_done(done);
    } else {
      wait_gate_up(done, tl.nn, claim + 2);
      if (it.stream)
        pingpong_item<1, 2>(H, Wdn, Y, it.wk, d, m, RowGather{nullptr, 1, 0}, st0, st1, st2, st3, grp);
      else
        pingpong_item<1, 0>(H, Wdn, Y, it.wk, d, m, RowGather{nullptr, 1, 0}, st0, st1, st2, st3, grp);
    }
    if (tid == 0) __hip_atomic_fetch_add(claim + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

__device__ __forceinline__ float silu_f(float g) { return g / (1.f + expf(-g)); }

// ---------------------------------------------------------------------------
// float32 SIMT path: 32x32 output tiles, k-step 32, 256 threads x 2x2 outputs
// ---------------------------------------------------------------------------
constexpr int FBM = 32, FBN = 32, FBK = 32;

template <int MODE>
__global__ __launch_bounds__(256) void ffn_gemm_f32_kernel(const float* __restrict__ A,
                                                           const float* __restrict__ W,
                                                           float* __restrict__ C,
                                                           const Tiles tl, int d, int m, const Guard g) {
  if (guard_skip(g)) return;
  __shared__ float as[FBM][FBK + 1];
  __shared__ float bs[2][FBN][FBK + 1];  // MODE 0: gate, up; MODE 1: down only
  __shared__ __attribute__((aligned(16))) char wl[64];
  Work wk;
  if (!find_work(tl, false, wk, wl)) return;
  const int nt = wk.nt;
  struct { int row0, rows, expert; } tile{wk.row0, wk.rows, wk.expert};
  const int Kdim = MODE == 0 ? d : m;
  const int Ncols = MODE == 0 ? m : d;
  const float* Wexp = W + (size_t)tile.expert * (size_t)(MODE == 0 ? 2 * m : d) * Kdim;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  float acc[2][2][2] = {};  // [B part][row][col]
  for (int k0 = 0; k0 < Kdim; k0 += FBK) {
    for (int i = tid; i < FBM * FBK; i += 256) {
      int r = i / FBK, kk = i % FBK;
      int kg = k0 + kk;
      as[r][kk] = (r < tile.rows && kg < Kdim) ? A[(size_t)(tile.row0 + r) * Kdim + kg] : 0.f;
      int col = nt * FBN + r;
      bool ok = col < Ncols && kg < Kdim;
      bs[0][r][kk] = ok ? Wexp[(size_t)col * Kdim + kg] : 0.f;
      if (MODE == 0) bs[1][r][kk] = ok ? Wexp[(size_t)(m + col) * Kdim + kg] : 0.f;
    }
    __syncthreads();
    for (int kk = 0; kk < FBK; ++kk) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        float a = as[ty * 2 + i][kk];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[0][i][j] = fmaf(a, bs[0][tx * 2 + j][kk], acc[0][i][j]);
          if (MODE == 0) acc[1][i][j] = fmaf(a, bs[1][tx * 2 + j][kk], acc[1][i][j]);
        }
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      int r = ty * 2 + i, col = nt * FBN + tx * 2 + j;
      if (r < tile.rows && col < Ncols) {
        float v = MODE == 0 ? silu_f(acc[0][i][j]) * acc[1][i][j] : acc[0][i][j];
        C[(size_t)(tile.row0 + r) * Ncols + col] = v;
      }
    }
}

}  // namespace kern

namespace {
using kern::FBM;
using kern::FBN;
using kern::NTHR;
using kern::Tiles;
using kern::ffn_gemm_bf16_kernel;
using kern::ffn_gemm_f32_kernel;
using kern::FFN_CTR_TILES;
using kern::clear_kernel;
using kern::ffn_status_kernel;
using kern::ffn_fused_kernel;
using kern::ffn_pingpong_kernel;
using kern::ffn_gemm_packed_kernel;
using kern::pack_weights_kernel;

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }
int max_tiles_for(int rows_max, int E, int bm) { return (rows_max + bm - 1) / bm + E; }

// M-tile height: 128 rows when experts average enough rows, else 64
// (weight-streaming shapes with few rows per expert).  On packed weights an
// item skips the MFMAs of 32-row blocks with no rows, so a sparse 128-row
// tile costs little compute, and it reads its expert's weights once where
// 64-row tiles read them per tile: 128-row tiles from 48 rows per expert on
// average (Qwen3-VL layer, 128 experts, top-8: 1024 tokens 284 -> 254 us,
// 2048 tokens 369 -> 297 us; around 512 tokens either height can be ahead
// by a few percent, depending on the routing).  Row-major weights: from 160.
int pick_bm(int rows_max, int E, bool packed) { return rows_max >= (packed ? 48 : 160) * E ? 128 : 64; }

// n-tiles per GEMM.  bf16 weight-row tile: 512 when it divides the expert's
// rows (gate/up: 2m, down: d), else 256 -- `wide` selects 512; the packed
// kernel always runs 256-row tiles at two workgroups per CU.  float32: 32
// output columns.
void n_tiles_of(bool bf16, bool packed, int d, int m, int& nn0, int& nn1, bool& wide0, bool& wide1) {
  if (bf16) {
    wide0 = !packed && (2 * m) % 512 == 0;
    wide1 = !packed && d % 512 == 0;
    nn0 = 2 * m / (wide0 ? 512 : 256);
    nn1 = d / (wide1 ? 512 : 256);
  } else {
    wide0 = wide1 = false;
    nn0 = (m + FBN - 1) / FBN;
    nn1 = (d + FBN - 1) / FBN;
  }
}

// kernels are instantiated here, outside any function template (device stubs
// of kernels first instantiated inside a template launcher are not emitted)
#define FFN_GEMM(MODE, BM, BN)                                                   \
  ffn_gemm_bf16_kernel<MODE, BM, BN><<<grid, NTHR, 0, s>>>(A, W, C, tl, d, m, g)

// row-major bf16 weights: one launch per GEMM
hipError_t launch_gemm(int mode, int bm, bool wide, const Tiles& tl, const uint16_t* A,
                       const uint16_t* W, uint16_t* C, int d, int m, hipStream_t s, Guard g) {
  const int grid = (tl.max_tiles * tl.nn + 7) & ~7;  // whole XCD rounds
  if (mode == 0) {
    if (bm == 128) {
      if (wide) FFN_GEMM(0, 128, 512); else FFN_GEMM(0, 128, 256);
    } else {
      if (wide) FFN_GEMM(0, 64, 512); else FFN_GEMM(0, 64, 256);
    }
  } else {
    if (bm == 128) {
      if (wide) FFN_GEMM(1, 128, 512); else FFN_GEMM(1, 128, 256);
    } else {
      if (wide) FFN_GEMM(1, 64, 512); else FFN_GEMM(1, 64, 256);
    }
  }
  return hipGetLastError();
}
#undef FFN_GEMM

// Persistent launch geometry: two workgroups per compute unit and the XCD
// count (false when the runtime cannot report them, or when the environment
// variable DECOMOE_FFN_TWO_LAUNCH is "1", which selects the two-launch path)
bool persistent_shape(int& grid, int& n_xcc) {
  const char* two = std::getenv("DECOMOE_FFN_TWO_LAUNCH");
  if (two && two[0] == '1') return false;
  int dev = 0, cus = 0, nx = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    return false;
  if (hipDeviceGetAttribute(&nx, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess || nx < 1 || nx > 8)
    return false;
  grid = 2 * cus;
  n_xcc = nx;
  return true;
}

// zeroes the counter header and the first n_tiles tile counters, and records
// the launch path (a kernel rather than a memset, so that a captured graph
// replays it)
hipError_t clear_counters(int* ctr, int n_tiles, int path, hipStream_t s, Guard g) {
  const int n_ctr = FFN_CTR_TILES + n_tiles;
  const int blocks = (n_ctr + 255) / 256 < 64 ? (n_ctr + 255) / 256 : 64;
  clear_kernel<<<blocks, 256, 0, s>>>(ctr, n_ctr, path, g);
  return hipGetLastError();
}

#define FFN_PACKED(MODE, BM)                                                      \
  ffn_gemm_packed_kernel<MODE, BM><<<(t.max_tiles * t.nn + 7) & ~7, NTHR, 0, s>>>( \
      A, W, C, t, d, m, rg, g)

// packed bf16 weights: both GEMMs in one persistent launch per call (after
// zeroing its counters), or one launch per GEMM when the XCD layout is unknown
hipError_t launch_packed(int bm, const Tiles& t0, int nn1, const uint16_t* X, const uint16_t* Wgu,
                         const uint16_t* Wdn, uint16_t* H, uint16_t* Y, int d, int m,
                         const RowGather g0, int* ctr, hipStream_t s, Guard g, bool counters_ready) {
  int grid = 0, n_xcc = 0;
  if (persistent_shape(grid, n_xcc)) {
    if (!counters_ready) {
      hipError_t e = clear_counters(ctr, t0.max_tiles, FFN_PATH_PERSISTENT, s, g);
      if (e != hipSuccess) return e;
    }
    // few rows per expert (decode): one token tile per expert, so every
    // weight tile is read once and streams with the non-temporal hint
    // (measured at 64 tokens x top-8 over 93 experts: 166 -> 151 us)
    const bool stream_weights = bm == 64 && t0.rows_max <= 16 * t0.E;
    // 64-row tiles (few rows per expert, weight streaming): 128-row weight
    // tiles in the down GEMM, twice as many items of half the bytes, so that
    // the queues drain evenly at the end (64 tokens x top-8 through 48
    // layers: 8.26 -> 8.00 ms per step)
    // 128-row tiles: 128 x 512 tiles of eight alternating wavefronts, one
    // workgroup per compute unit, where 512 divides both weight matrices
    if (bm == 128 && (2 * m) % 512 == 0 && d % 512 == 0) {
      Tiles tp = t0;
      tp.nn = 2 * m / 512;
      ffn_pingpong_kernel<<<grid / 2, kern::PP_THR, 0, s>>>(X, Wgu, Wdn, H, Y, tp, d / 512, d, m, g0, n_xcc, ctr,
                                                            g);
    } else if (bm == 128)
      ffn_fused_kernel<128, 0, 256><<<grid, NTHR, 0, s>>>(X, Wgu, Wdn, H, Y, t0, nn1, d, m, g0, n_xcc, ctr, g);
    else if (stream_weights)
      ffn_fused_kernel<64, 2, 128><<<grid, NTHR, 0, s>>>(X, Wgu, Wdn, H, Y, t0, d / 128, d, m, g0, n_xcc, ctr, g);
    else
      ffn_fused_kernel<64, 0, 128><<<grid, NTHR, 0, s>>>(X, Wgu, Wdn, H, Y, t0, d / 128, d, m, g0, n_xcc, ctr, g);
    return hipGetLastError();
  }
  hipError_t e = clear_counters(ctr, 0, FFN_PATH_TWO_LAUNCH, s, g);
  if (e != hipSuccess) return e;
  {
    const Tiles& t = t0;
    const uint16_t* A = X;
    const uint16_t* W = Wgu;
    uint16_t* C = H;
    const RowGather rg = g0;
    if (bm == 128) FFN_PACKED(0, 128); else FFN_PACKED(0, 64);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    Tiles t = t0;
    t.nn = nn1;
    const uint16_t* A = H;
    const uint16_t* W = Wdn;
    uint16_t* C = Y;
    const RowGather rg{nullptr, 1, 0};
    if (bm == 128) FFN_PACKED(1, 128); else FFN_PACKED(1, 64);
  }
  return hipGetLastError();
}
#undef FFN_PACKED
}  // namespace

// Workspace, from ws rounded up to a 256-byte boundary: the counters of the
// persistent kernel (128 + max_tiles ints, sized for the smaller tile), then
// the intermediate h [rows_max, m].  The rounding keeps every h row block of
// a tile on whole 128-byte lines whatever the caller's alignment (a down item
// must never find a line of its tile's h in L1 from a neighbouring tile).
size_t ffn_ctr_bytes(int rows_max, int E) {
  return align256((size_t)(kern::FFN_CTR_TILES + max_tiles_for(rows_max, E, 64)) * 4);
}
size_t ffn_counter_span(int rows_max, int E) { return 256 + ffn_ctr_bytes(rows_max, E); }

size_t ffn_ws_bytes(bool bf16, int rows_max, int E, int d, int m) {
  (void)d;
  return 256 + ffn_ctr_bytes(rows_max, E) + align256((size_t)rows_max * m * (bf16 ? 2 : 4));
}

int* ffn_counters(void* ws) {
  return reinterpret_cast<int*>(align256(reinterpret_cast<uintptr_t>(ws)));
}

bool ffn_persistent_available() {
  int grid = 0, n_xcc = 0;
  return persistent_shape(grid, n_xcc);
}

ZeroAfter ffn_counters_zero(void* ws, int rows_max, int E) {
  // what clear_counters writes, for the largest tile count of either tile height
  return ZeroAfter{ffn_counters(ws), kern::FFN_CTR_TILES + max_tiles_for(rows_max, E, 64), kern::FFN_CTR_PATH,
                   FFN_PATH_PERSISTENT};
}

hipError_t launch_ffn_status(const void* ws, int32_t* status, hipStream_t s) {
  ffn_status_kernel<<<1, 64, 0, s>>>(ffn_counters(const_cast<void*>(ws)), status);
  return hipGetLastError();
}

hipError_t launch_expert_ffn(const void* x_perm, bool bf16, const int32_t* offsets, int E,
                             const int32_t* K_dev, int n_K, int rows_max, int d, int m,
                             const void* w_gate_up, const void* w_down, bool packed, void* y_perm,
                             void* ws, hipStream_t s, RowGather gather, int kmin, Guard g, bool counters_ready) {
  if (gather.src_of_row && !(bf16 && packed)) return hipErrorInvalidValue;
  const int bm = bf16 ? pick_bm(rows_max, E, packed) : FBM;
  int nn0, nn1;
  bool wide0, wide1;
  n_tiles_of(bf16, packed, d, m, nn0, nn1, wide0, wide1);
  Tiles t0{offsets, K_dev, E, K_dev ? n_K : 0, rows_max, bm, max_tiles_for(rows_max, E, bm), nn0,
           kmin};
  Tiles t1 = t0;
  t1.nn = nn1;
  int* const ctr = ffn_counters(ws);
  void* h = reinterpret_cast<char*>(ctr) + ffn_ctr_bytes(rows_max, E);
  hipError_t err;
  if (bf16 && packed) {
    return launch_packed(bm, t0, nn1, static_cast<const uint16_t*>(x_perm),
                        static_cast<const uint16_t*>(w_gate_up), static_cast<const uint16_t*>(w_down),
                        static_cast<uint16_t*>(h), static_cast<uint16_t*>(y_perm), d, m, gather, ctr, s, g,
                        counters_ready);
  }
  err = clear_counters(ctr, 0, bf16 ? FFN_PATH_ROW_MAJOR : FFN_PATH_F32, s, g);
  if (err != hipSuccess) return err;
  if (bf16) {
    err = launch_gemm(0, bm, wide0, t0, static_cast<const uint16_t*>(x_perm),
                      static_cast<const uint16_t*>(w_gate_up), static_cast<uint16_t*>(h), d, m, s, g);
    if (err != hipSuccess) return err;
    return launch_gemm(1, bm, wide1, t1, static_cast<const uint16_t*>(h),
                       static_cast<const uint16_t*>(w_down), static_cast<uint16_t*>(y_perm), d, m, s, g);
  }
  ffn_gemm_f32_kernel<0><<<t0.max_tiles * nn0, NTHR, 0, s>>>(
      static_cast<const float*>(x_perm), static_cast<const float*>(w_gate_up), static_cast<float*>(h),
      t0, d, m, g);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  ffn_gemm_f32_kernel<1><<<t1.max_tiles * nn1, NTHR, 0, s>>>(
      static_cast<const float*>(h), static_cast<const float*>(w_down), static_cast<float*>(y_perm),
      t1, d, m, g);
  return hipGetLastError();
}

hipError_t launch_pack_weights(const void* w, int E, int R, int K, void* out, hipStream_t s) {
  const size_t n_chunks = (size_t)E * R * (K / 8);
  if (n_chunks == 0) return hipSuccess;
  pack_weights_kernel<<<(unsigned)((n_chunks + 255) / 256), 256, 0, s>>>(
      static_cast<const uint4*>(w), R, K, n_chunks, static_cast<uint4*>(out));
  return hipGetLastError();
}

}  // namespace decomoe
