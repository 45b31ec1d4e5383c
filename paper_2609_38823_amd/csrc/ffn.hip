// Grouped SwiGLU expert FFN over the dispatched rows (Algorithm 2: evaluate
// only the first K physically contiguous expert MLPs; gate, up and down
// projections as in App. A.3, Eq. 15).
//
//   tiles     a one-workgroup kernel turns the per-expert row ranges into a
//             list of (expert, first row, rows) M-tiles on the device, so no
//             host synchronisation is needed on K or on the counts
//   gate_up   H[r, :] = SiLU(X W_gate^T) * (X W_up^T) for the rows of one
//             M-tile; the gate and up weight rows of the same h columns sit
//             in one B tile, so SwiGLU is applied in registers
//   down      Y = H W_down^T
//
// bf16: v_mfma_f32_16x16x32_bf16, 128x128x64 block tiles, 4 wavefronts of
// 64x64, LDS double buffered with an XOR swizzle of the 16-byte chunks
// (conflict-free ds_read_b128 of the MFMA fragments), float32 accumulation.
// float32: a plain LDS-tiled SIMT kernel (correctness path for small layers).
#include "common.hpp"

namespace decomoe {
// Kernels live in a named namespace: device stubs of templated kernels with
// internal linkage are not emitted when instantiated from a template launcher.
namespace kern {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct Tile {
  int expert, row0, rows, pad;
};

// ---------------------------------------------------------------------------
// M-tile list.  Experts e < Klim with rows [offsets[e], offsets[e+1]) (clamped
// to [0, rows_max]) become ceil(rows / bm) tiles, expert-major.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void ffn_tiles_kernel(const int32_t* __restrict__ offsets,
                                                         int E, const int32_t* __restrict__ K_dev,
                                                         int n_K, int rows_max, int bm,
                                                         Tile* __restrict__ tiles, int max_tiles,
                                                         int32_t* __restrict__ n_tiles) {
  __shared__ int sc[1024];
  const int e = threadIdx.x;
  int Klim = E;
  if (K_dev) {
    Klim = 0;
    for (int i = 0; i < n_K; ++i) Klim = max(Klim, K_dev[i]);
    Klim = clampi(Klim, 0, E);
  }
  int lo = 0, hi = 0, nt = 0;
  if (e < Klim) {
    lo = clampi(offsets[e], 0, rows_max);
    hi = clampi(offsets[e + 1], lo, rows_max);
    nt = (hi - lo + bm - 1) / bm;
  }
  sc[e] = nt;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    int v = e >= off ? sc[e - off] : 0;
    __syncthreads();
    sc[e] += v;
    __syncthreads();
  }
  const int start = sc[e] - nt;
  for (int i = 0; i < nt; ++i) {
    int ti = start + i;
    if (ti < max_tiles) {
      int r0 = lo + i * bm;
      tiles[ti] = Tile{e, r0, min(bm, hi - r0), 0};
    }
  }
  if (e == 1023) *n_tiles = min(sc[1023], max_tiles);
}

// ---------------------------------------------------------------------------
// bf16 MFMA grouped GEMM
//
// Block tile BM rows x BN weight rows, k-step 64; 4 wavefronts in 2 x 2, each
// owning (BM/2) x (BN/2) outputs as 16x16 fragments of
// v_mfma_f32_16x16x32_bf16.  Operand tiles stream from global memory straight
// into LDS with global_load_lds_dwordx4 through a 3-stage ring (three
// separate LDS arrays, so the compiler's wait tracking keeps the two younger
// stages in flight while the oldest is consumed).  Each 128-byte LDS row holds
// one tile row's 64 k-values as eight 16-byte chunks, chunk c stored at
// position c ^ ((row >> 1) & 7): the 16 rows read by one quarter-wavefront
// then hit 16 distinct bank groups.
// ---------------------------------------------------------------------------
constexpr int BK = 64, NTHR = 256, STAGES = 3;
constexpr int LDS_STAGE_MAX = (128 + 256) * BK * 2;  // bytes, largest tile pair

__shared__ __attribute__((aligned(1024))) char ring0[LDS_STAGE_MAX];
__shared__ __attribute__((aligned(1024))) char ring1[LDS_STAGE_MAX];
__shared__ __attribute__((aligned(1024))) char ring2[LDS_STAGE_MAX];

__device__ __forceinline__ int swz_off(int row, int chunk) {
  return row * 128 + ((chunk ^ ((row >> 1) & 7)) << 4);
}

__device__ __forceinline__ float silu_f(float g) { return g / (1.f + expf(-g)); }

// 16-byte global -> LDS copy per lane (global_load_lds_dwordx4): lane l writes
// lds + 16 l.  A non-template wrapper: the host compilation pass rejects this
// builtin inside a kernel template.
__device__ __forceinline__ void dma16(const void* gsrc, void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds(gsrc, lds_wave_base, 16, 0, 0);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14])
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

template <int MODE, int BM, int BN>
struct GemmCfg {
  static constexpr int MI = BM / 32;         // 16-row fragments per wave
  static constexpr int NI = BN / 32;         // 16-col fragments per wave
  static constexpr int ROWS = BM + BN;       // LDS rows per stage (A then B)
  static constexpr int GROUPS = ROWS / 8;    // 1 KB DMA groups per stage
  static constexpr int GPW = GROUPS / 4;     // DMA instructions per wave per stage
  static_assert(GROUPS % 4 == 0, "stage must split evenly over 4 waves");
  static_assert(ROWS * 128 <= LDS_STAGE_MAX, "stage too large");
};

// MODE 0: A = x_perm [rows, d], W = w_gate_up [E, 2m, d], C = h [rows, m];
//         the B tile's first BN/2 rows are gate rows nt*BN/2.., the rest the
//         matching up rows m + nt*BN/2..; C gets BN/2 columns
// MODE 1: A = h [rows, m], W = w_down [E, d, m], C = y_perm [rows, d];
//         B rows nt*BN.., C gets BN columns
template <int MODE, int BM, int BN>
__global__ __launch_bounds__(NTHR, 1) void ffn_gemm_bf16_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ W, uint16_t* __restrict__ C,
    const Tile* __restrict__ tiles, const int32_t* __restrict__ n_tiles, int d, int m,
    int n_tiles_n) {
  using Cfg = GemmCfg<MODE, BM, BN>;
  constexpr int MI = Cfg::MI, NI = Cfg::NI, GPW = Cfg::GPW;

  const int nt = blockIdx.x % n_tiles_n;
  const int mt = blockIdx.x / n_tiles_n;
  if (mt >= *n_tiles) return;
  const Tile tile = tiles[mt];
  const int Kdim = MODE == 0 ? d : m;
  const int ldc = MODE == 0 ? m : d;
  const uint16_t* Wexp = W + (size_t)tile.expert * (size_t)(MODE == 0 ? 2 * m : d) * Kdim;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wv = tid >> 6;
  const int wm = wv >> 1, wn = wv & 1;
  const int r16 = lane & 15, kq = lane >> 4;

  // ---- DMA source pointers: this lane's row and swizzled chunk per group --
  // group g (8 rows) of the stage: rows [8g, 8g+8); lane -> row 8g + lane/8,
  // LDS chunk lane%8, global chunk (lane%8) ^ ((row >> 1) & 7)
  const uint16_t* src[GPW];
#pragma unroll
  for (int q = 0; q < GPW; ++q) {
    const int g = wv * GPW + q;
    const int r = g * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((r >> 1) & 7);
    const uint16_t* rowp;
    if (r < BM) {
      const int rr = r < tile.rows ? r : 0;  // padding rows re-read row 0
      rowp = A + (size_t)(tile.row0 + rr) * Kdim;
    } else {
      const int b = r - BM;
      int wrow;
      if (MODE == 0)
        wrow = b < BN / 2 ? nt * (BN / 2) + b : m + nt * (BN / 2) + (b - BN / 2);
      else
        wrow = nt * BN + b;
      rowp = Wexp + (size_t)wrow * Kdim;
    }
    src[q] = rowp + c * 8;
  }

  auto issue = [&](char* stage, int k0) {
#pragma unroll
    for (int q = 0; q < GPW; ++q) {
      const int g = wv * GPW + q;
      dma16(src[q] + k0, stage + g * 1024);
    }
  };

  f32x4 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // LDS byte offsets of this lane's fragment rows (chunk applied per k-step)
  int arow[MI], brow[NI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) arow[mi] = wm * (BM / 2) + mi * 16 + r16;
#pragma unroll
  for (int ni = 0; ni < NI; ++ni) {
    int b;
    if (MODE == 0)  // half gate, half up, same h columns
      b = ni < NI / 2 ? wn * (BN / 4) + ni * 16 : BN / 2 + wn * (BN / 4) + (ni - NI / 2) * 16;
    else
      b = wn * (BN / 2) + ni * 16;
    brow[ni] = BM + b + r16;
  }

  // fragments of k-substep ks (32 k-values): 16 bytes per lane per fragment
  auto load_frags = [&](const char* stage, int ks, bf16x8 (&af)[MI], bf16x8 (&bfr)[NI]) {
    const int c = ks * 4 + kq;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
      af[mi] = *reinterpret_cast<const bf16x8*>(stage + swz_off(arow[mi], c));
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
      bfr[ni] = *reinterpret_cast<const bf16x8*>(stage + swz_off(brow[ni], c));
  };
  auto mma = [&](const bf16x8 (&af)[MI], const bf16x8 (&bfr)[NI]) {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
        acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[mi], bfr[ni], acc[mi][ni], 0, 0, 0);
  };
  // k-substep 0's fragments are read first; substep 1's twelve reads are
  // issued one after each of substep 0's first MFMAs, so at most 15 LDS reads
  // are outstanding (the counter limit) and they land under the MFMAs
  auto compute = [&](const char* stage) {
    bf16x8 a0[MI], b0[NI], a1[MI], b1[NI];
    load_frags(stage, 0, a0, b0);
    __builtin_amdgcn_sched_barrier(0);
    const int c1 = 4 + kq;
#pragma unroll
    for (int j = 0; j < MI * NI; ++j) {
      acc[j / NI][j % NI] =
          __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[j / NI], b0[j % NI], acc[j / NI][j % NI], 0, 0, 0);
      if (j < MI)
        a1[j] = *reinterpret_cast<const bf16x8*>(stage + swz_off(arow[j], c1));
      else if (j < MI + NI)
        b1[j - MI] = *reinterpret_cast<const bf16x8*>(stage + swz_off(brow[j - MI], c1));
      __builtin_amdgcn_sched_barrier(0);
    }
    mma(a1, b1);
  };

  const int nk = Kdim / BK;
  // steady-state step: wait until stage `cur` has landed (one younger stage
  // still in flight), barrier (every wave is also done with the stage read in
  // the previous step), refill that stage with iteration it+2, consume `cur`
  auto step_issue = [&](int it, char* cur, char* nxt) {
    wait_vmcnt<GPW>();
    __builtin_amdgcn_s_barrier();
    issue(nxt, (it + 2) * BK);
    compute(cur);
  };
  // drain steps: nothing left to issue
  auto step_tail = [&](char* cur, bool last) {
    if (last)
      wait_vmcnt<0>();
    else
      wait_vmcnt<GPW>();
    __builtin_amdgcn_s_barrier();
    compute(cur);
  };

  if (nk < 2) {  // a single k-step: no pipeline
    issue(ring0, 0);
    step_tail(ring0, true);
  } else {
  issue(ring0, 0);
  issue(ring1, BK);
  int it = 0;
  for (; it + 5 <= nk; it += 3) {  // branch-free body: every step issues
    step_issue(it, ring0, ring2);
    step_issue(it + 1, ring1, ring0);
    step_issue(it + 2, ring2, ring1);
  }
  // 1 to 4 iterations remain (it is a multiple of 3, so rings are static)
  const int rem = nk - it;
  if (rem >= 3) {
    step_issue(it, ring0, ring2);
    if (rem == 4) {
      step_issue(it + 1, ring1, ring0);
      step_tail(ring2, false);
      step_tail(ring0, true);
    } else {
      step_tail(ring1, false);
      step_tail(ring2, true);
    }
  } else if (rem == 2) {
    step_tail(ring0, false);
    step_tail(ring1, true);
  } else if (rem == 1) {
    step_tail(ring0, true);
  }
  }

  // ---- epilogue: bf16 tile staged in LDS, then 16-byte coalesced stores ----
  __syncthreads();  // every wave is done reading the ring
  uint16_t* ctile = reinterpret_cast<uint16_t*>(ring0);
  constexpr int CW = MODE == 0 ? BN / 2 : BN;  // output columns of the tile
  if (MODE == 0) {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int f = 0; f < NI / 2; ++f)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = wm * (BM / 2) + mi * 16 + kq * 4 + i;
          const int col = wn * (BN / 4) + f * 16 + r16;
          const float hv = silu_f(acc[mi][f][i]) * acc[mi][f + NI / 2][i];
          ctile[row * CW + col] = f32_to_bf16(hv);
        }
  } else {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = wm * (BM / 2) + mi * 16 + kq * 4 + i;
          const int col = wn * (BN / 2) + ni * 16 + r16;
          ctile[row * CW + col] = f32_to_bf16(acc[mi][ni][i]);
        }
  }
  __syncthreads();
  constexpr int CPR = CW / 8;  // 16-byte chunks per output row
#pragma unroll
  for (int i = 0; i < BM * CPR / NTHR; ++i) {
    const int lin = i * NTHR + tid;
    const int row = lin / CPR, ch = lin % CPR;
    if (row < tile.rows)
      *reinterpret_cast<uint4*>(C + (size_t)(tile.row0 + row) * ldc + nt * CW + ch * 8) =
          reinterpret_cast<const uint4*>(ctile)[row * CPR + ch];
  }
}

// ---------------------------------------------------------------------------
// float32 SIMT path: 32x32 output tiles, k-step 32, 256 threads x 2x2 outputs
// ---------------------------------------------------------------------------
constexpr int FBM = 32, FBN = 32, FBK = 32;

template <int MODE>
__global__ __launch_bounds__(256) void ffn_gemm_f32_kernel(const float* __restrict__ A,
                                                           const float* __restrict__ W,
                                                           float* __restrict__ C,
                                                           const Tile* __restrict__ tiles,
                                                           const int32_t* __restrict__ n_tiles,
                                                           int d, int m, int n_tiles_n) {
  __shared__ float as[FBM][FBK + 1];
  __shared__ float bs[2][FBN][FBK + 1];  // MODE 0: gate, up; MODE 1: down only
  const int nt = blockIdx.x % n_tiles_n;
  const int mt = blockIdx.x / n_tiles_n;
  if (mt >= *n_tiles) return;
  const Tile tile = tiles[mt];
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
using kern::Tile;
using kern::ffn_tiles_kernel;
using kern::FBM;
using kern::FBN;
using kern::NTHR;
using kern::ffn_gemm_bf16_kernel;
using kern::ffn_gemm_f32_kernel;

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }
int max_tiles_for(int rows_max, int E, int bm) { return (rows_max + bm - 1) / bm + E; }

// M-tile height: 128 rows when experts average enough rows to fill them,
// else 64 (weight-streaming shapes with few rows per expert)
int pick_bm(int rows_max, int E) { return rows_max >= 160 * E ? 128 : 64; }

// kernels are instantiated here, outside any function template (device stubs
// of kernels first instantiated inside a template launcher are not emitted)
#define FFN_GEMM(MODE, BM, BN) \
  ffn_gemm_bf16_kernel<MODE, BM, BN><<<max_tiles * nn, NTHR, 0, s>>>(A, W, C, tiles, n_tiles, d, m, nn)

hipError_t launch_gemm(int mode, int bm, const uint16_t* A, const uint16_t* W, uint16_t* C,
                       const Tile* tiles, const int32_t* n_tiles, int d, int m, int max_tiles,
                       hipStream_t s) {
  const int ncols = mode == 0 ? 2 * m : d;  // weight rows of one expert
  const bool wide = ncols % 256 == 0;
  const int nn = ncols / (wide ? 256 : 128);
  if (mode == 0) {
    if (bm == 128) {
      if (wide) FFN_GEMM(0, 128, 256); else FFN_GEMM(0, 128, 128);
    } else {
      if (wide) FFN_GEMM(0, 64, 256); else FFN_GEMM(0, 64, 128);
    }
  } else {
    if (bm == 128) {
      if (wide) FFN_GEMM(1, 128, 256); else FFN_GEMM(1, 128, 128);
    } else {
      if (wide) FFN_GEMM(1, 64, 256); else FFN_GEMM(1, 64, 128);
    }
  }
  return hipGetLastError();
}
#undef FFN_GEMM
}  // namespace

size_t ffn_ws_bytes(bool bf16, int rows_max, int E, int d, int m) {
  (void)d;
  const int bm = bf16 ? 64 : FBM;  // the smallest tile height gives the longest list
  size_t tiles = align256((size_t)max_tiles_for(rows_max, E, bm) * sizeof(Tile));
  size_t h = align256((size_t)rows_max * m * (bf16 ? 2 : 4));
  return 256 + tiles + h;
}

hipError_t launch_expert_ffn(const void* x_perm, bool bf16, const int32_t* offsets, int E,
                             const int32_t* K_dev, int n_K, int rows_max, int d, int m,
                             const void* w_gate_up, const void* w_down, void* y_perm, void* ws,
                             hipStream_t s) {
  const int bm = bf16 ? pick_bm(rows_max, E) : FBM;
  const int max_tiles = max_tiles_for(rows_max, E, bm);
  const int list_cap = max_tiles_for(rows_max, E, bf16 ? 64 : FBM);
  char* p = static_cast<char*>(ws);
  int32_t* n_tiles = reinterpret_cast<int32_t*>(p);
  Tile* tiles = reinterpret_cast<Tile*>(p + 256);
  void* h = p + 256 + align256((size_t)list_cap * sizeof(Tile));
  ffn_tiles_kernel<<<1, 1024, 0, s>>>(offsets, E, K_dev, n_K, rows_max, bm, tiles, max_tiles, n_tiles);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  if (bf16) {
    const auto* xp = static_cast<const uint16_t*>(x_perm);
    const auto* wgu = static_cast<const uint16_t*>(w_gate_up);
    const auto* wd = static_cast<const uint16_t*>(w_down);
    auto* hh = static_cast<uint16_t*>(h);
    auto* y = static_cast<uint16_t*>(y_perm);
    err = launch_gemm(0, bm, xp, wgu, hh, tiles, n_tiles, d, m, max_tiles, s);
    if (err == hipSuccess) err = launch_gemm(1, bm, hh, wd, y, tiles, n_tiles, d, m, max_tiles, s);
    return err;
  }
  const int n0 = (m + FBN - 1) / FBN, n1 = (d + FBN - 1) / FBN;
  ffn_gemm_f32_kernel<0><<<max_tiles * n0, 256, 0, s>>>(
      static_cast<const float*>(x_perm), static_cast<const float*>(w_gate_up),
      static_cast<float*>(h), tiles, n_tiles, d, m, n0);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  ffn_gemm_f32_kernel<1><<<max_tiles * n1, 256, 0, s>>>(
      static_cast<const float*>(h), static_cast<const float*>(w_down),
      static_cast<float*>(y_perm), tiles, n_tiles, d, m, n1);
  return hipGetLastError();
}

}  // namespace decomoe
