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
namespace {

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
// ---------------------------------------------------------------------------
constexpr int BM = 128, BN = 128, BK = 64, NTHR = 256;
constexpr int CHUNKS = BM * BK / 8;  // 16-byte chunks per operand tile (1024)

__device__ __forceinline__ int swz(int row, int chunk) { return row * 8 + (chunk ^ (row & 7)); }

__device__ __forceinline__ float silu_f(float g) { return g / (1.f + expf(-g)); }

// MODE 0: A = x_perm [rows, d], W = w_gate_up [E, 2m, d], C = h [rows, m]
//         block n-tile = 64 h columns (64 gate rows + 64 up rows of W)
// MODE 1: A = h [rows, m], W = w_down [E, d, m], C = y_perm [rows, d]
//         block n-tile = 128 output columns
template <int MODE>
__global__ __launch_bounds__(NTHR, 2) void ffn_gemm_bf16_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ W, uint16_t* __restrict__ C,
    const Tile* __restrict__ tiles, const int32_t* __restrict__ n_tiles, int d, int m,
    int n_tiles_n) {
  __shared__ uint4 lds[2][2][CHUNKS];  // [stage][A | B][chunk]  64 KB

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

  // global -> register staging: rows (tid >> 3) + 32 i, 16-byte chunk tid & 7
  const int gc = tid & 7;
  const int gr = tid >> 3;
  int a_ok = 0;  // bit i: staging row i lies inside the tile
#pragma unroll
  for (int i = 0; i < 4; ++i) a_ok |= (gr + 32 * i < tile.rows) << i;
  const uint16_t* a_base = A + (size_t)(tile.row0 + gr) * Kdim + gc * 8;
  // MODE 0: staging rows 0,1 are gate rows nt*64 + gr (+32), rows 2,3 the
  // matching up rows m + nt*64 + gr (+32); MODE 1: rows nt*128 + gr + 32 i
  const uint16_t* b_base0 = Wexp + (size_t)((MODE == 0 ? nt * 64 : nt * BN) + gr) * Kdim + gc * 8;
  const uint16_t* b_base1 =
      MODE == 0 ? Wexp + (size_t)(m + nt * 64 + gr) * Kdim + gc * 8 : b_base0 + (size_t)64 * Kdim;
  const size_t step32 = (size_t)32 * Kdim;
  uint4 ra[4], rb[4];
  auto load_global = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = (a_ok >> i) & 1 ? *reinterpret_cast<const uint4*>(a_base + i * step32 + k0)
                              : make_uint4(0, 0, 0, 0);
      const uint16_t* bp = (i < 2 ? b_base0 : b_base1) + (i & 1) * step32 + k0;
      rb[i] = *reinterpret_cast<const uint4*>(bp);
    }
  };
  auto store_lds = [&](int st) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int r = gr + 32 * i;
      lds[st][0][swz(r, gc)] = ra[i];
      lds[st][1][swz(r, gc)] = rb[i];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // B-tile rows of this wave's four 16-column fragments
  int brow[4];
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) {
    if (MODE == 0)
      brow[ni] = (ni < 2 ? wn * 32 + ni * 16 : 64 + wn * 32 + (ni - 2) * 16) + r16;
    else
      brow[ni] = wn * 64 + ni * 16 + r16;
  }

  const int nk = Kdim / BK;
  load_global(0);
  store_lds(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int st = kt & 1;
    if (kt + 1 < nk) load_global((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) {
        int row = wm * 64 + mi * 16 + r16;
        uint4 v = lds[st][0][swz(row, ks * 4 + kq)];
        af[mi] = __builtin_bit_cast(bf16x8, v);
      }
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        uint4 v = lds[st][1][swz(brow[ni], ks * 4 + kq)];
        bfr[ni] = __builtin_bit_cast(bf16x8, v);
      }
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[mi], bfr[ni], acc[mi][ni], 0, 0, 0);
    }
    if (kt + 1 < nk) store_lds(st ^ 1);
    __syncthreads();
  }

  // epilogue: stage the bf16 tile in LDS, then 16-byte coalesced stores
  uint16_t* ctile = reinterpret_cast<uint16_t*>(&lds[0][0][0]);
  if (MODE == 0) {
    // h tile [128 rows][64 cols]
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          int row = wm * 64 + mi * 16 + kq * 4 + i;
          int col = wn * 32 + f * 16 + r16;
          float hv = silu_f(acc[mi][f][i]) * acc[mi][f + 2][i];
          ctile[row * 64 + col] = f32_to_bf16(hv);
        }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int row = (tid >> 3) + 32 * i, ch = tid & 7;
      if (row < tile.rows)
        *reinterpret_cast<uint4*>(C + (size_t)(tile.row0 + row) * ldc + nt * 64 + ch * 8) =
            reinterpret_cast<const uint4*>(ctile)[row * 8 + ch];
    }
  } else {
    // y tile [128 rows][128 cols]
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < 4; ++ni)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          int row = wm * 64 + mi * 16 + kq * 4 + i;
          int col = wn * 64 + ni * 16 + r16;
          ctile[row * 128 + col] = f32_to_bf16(acc[mi][ni][i]);
        }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      int row = (tid >> 4) + 16 * i, ch = tid & 15;
      if (row < tile.rows)
        *reinterpret_cast<uint4*>(C + (size_t)(tile.row0 + row) * ldc + nt * BN + ch * 8) =
            reinterpret_cast<const uint4*>(ctile)[row * 16 + ch];
    }
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

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }
int max_tiles_for(int rows_max, int E, int bm) { return (rows_max + bm - 1) / bm + E; }
}  // namespace

size_t ffn_ws_bytes(bool bf16, int rows_max, int E, int d, int m) {
  (void)d;
  const int bm = bf16 ? BM : FBM;
  size_t tiles = align256((size_t)max_tiles_for(rows_max, E, bm) * sizeof(Tile));
  size_t h = align256((size_t)rows_max * m * (bf16 ? 2 : 4));
  return 256 + tiles + h;
}

hipError_t launch_expert_ffn(const void* x_perm, bool bf16, const int32_t* offsets, int E,
                             const int32_t* K_dev, int n_K, int rows_max, int d, int m,
                             const void* w_gate_up, const void* w_down, void* y_perm, void* ws,
                             hipStream_t s) {
  const int bm = bf16 ? BM : FBM;
  const int max_tiles = max_tiles_for(rows_max, E, bm);
  char* p = static_cast<char*>(ws);
  int32_t* n_tiles = reinterpret_cast<int32_t*>(p);
  Tile* tiles = reinterpret_cast<Tile*>(p + 256);
  void* h = p + 256 + align256((size_t)max_tiles * sizeof(Tile));
  ffn_tiles_kernel<<<1, 1024, 0, s>>>(offsets, E, K_dev, n_K, rows_max, bm, tiles, max_tiles, n_tiles);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  if (bf16) {
    const int n0 = m / 64, n1 = d / BN;
    ffn_gemm_bf16_kernel<0><<<max_tiles * n0, NTHR, 0, s>>>(
        static_cast<const uint16_t*>(x_perm), static_cast<const uint16_t*>(w_gate_up),
        static_cast<uint16_t*>(h), tiles, n_tiles, d, m, n0);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    ffn_gemm_bf16_kernel<1><<<max_tiles * n1, NTHR, 0, s>>>(
        static_cast<const uint16_t*>(h), static_cast<const uint16_t*>(w_down),
        static_cast<uint16_t*>(y_perm), tiles, n_tiles, d, m, n1);
  } else {
    const int n0 = (m + FBN - 1) / FBN, n1 = (d + FBN - 1) / FBN;
    ffn_gemm_f32_kernel<0><<<max_tiles * n0, 256, 0, s>>>(
        static_cast<const float*>(x_perm), static_cast<const float*>(w_gate_up),
        static_cast<float*>(h), tiles, n_tiles, d, m, n0);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    ffn_gemm_f32_kernel<1><<<max_tiles * n1, 256, 0, s>>>(
        static_cast<const float*>(h), static_cast<const float*>(w_down),
        static_cast<float*>(y_perm), tiles, n_tiles, d, m, n1);
  }
  return hipGetLastError();
}

}  // namespace decomoe
