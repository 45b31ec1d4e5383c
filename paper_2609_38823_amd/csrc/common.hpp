// Shared device helpers and launcher declarations of the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace decomoe {

constexpr int kWave = 64;  // CDNA wavefront width

// ---- bf16 <-> f32 (bf16 is the upper half of an IEEE binary32) ----------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}
// round to nearest, ties to even (gfx950 converts in hardware:
// v_cvt_pk_bf16_f32); NaN stays NaN
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

// 16-byte load with the non-temporal hint: every expert output row is read
// once, so it should not displace reused lines from the caches (measured at
// 65 536 rows x top-8, d 2048: 5.1 -> 5.8 TB/s in the combine)
typedef unsigned int u32x4_nt __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
  const u32x4_nt q = __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(p));
  return make_uint4(q.x, q.y, q.z, q.w);
}
__device__ __forceinline__ int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// segment containing token t: the last s with seg_offsets[s] <= t
__device__ __forceinline__ int find_segment(const int32_t* seg_offsets, int n_seg, int t) {
  int lo = 0, hi = n_seg - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (seg_offsets[mid] <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// ---- launch predicate ----------------------------------------------------
// A launch runs only when *flag lies in [lo, hi) at the time its kernels
// execute (read on the device: a predicate that a captured graph keeps); a
// NULL flag always runs.  A skipped kernel returns at once and writes
// nothing.
struct Guard {
  const int32_t* flag = nullptr;
  int lo = 0, hi = 0;
};
__device__ __forceinline__ bool guard_skip(const Guard& g) {
  if (!g.flag) return false;
  const int v = *g.flag;
  return v < g.lo || v >= g.hi;
}

// ---- launchers (host side; return hipError_t of the launch) -------------
size_t route_ws_bytes(int T, int d, int E);
// logits (x != NULL; from w_r_packed when given, else w_r) and Top-k in one
// call; x == NULL reads `logits`
hipError_t launch_route(const void* x, bool x_bf16, const float* w_r, const void* w_r_packed,
                        const float* bias, int T, int d, int E, int k, const int32_t* seg_offsets,
                        int n_seg, const int32_t* K_dev, float* logits, int32_t* idx, float* w,
                        void* ws, hipStream_t s, Guard g = Guard{}, int* ctr_zero = nullptr);
// (ctr_zero: an int the Top-k launch sets to 0, for a launch that follows)
// the Top-k of launch_route on given logits or split partials (part, S)
hipError_t launch_topk(float* logits, int T, int E, int k, const int32_t* seg_offsets, int n_seg,
                       const int32_t* K_dev, const float* part, int S, const float* bias, int32_t* idx, float* w,
                       hipStream_t s, Guard g = Guard{}, int* ctr_zero = nullptr);
// bf16 x (three-term split router weights): packing and the logits kernel;
// `part`/`S` receive the split partials the Top-k kernel has to add
size_t route_x3_ws_bytes(int T, int d, int E);
hipError_t launch_pack_router(const float* w_r, int d, int E, void* out, hipStream_t s);
hipError_t launch_router_x3(const void* x, const void* w_packed, const float* bias, int T, int d,
                            int E, float* logits, void* ws, float*& part, int& S, hipStream_t s,
                            Guard g = Guard{});
// the previous layer's combine with the residual (h updated in place) fused
// into the router over the new h; combine_router_fits says when it applies
bool combine_router_fits(int T, int d, int E, int k);
hipError_t launch_combine_router_x3(const void* y_prev, const int32_t* row_prev, const float* w_prev, int k_prev,
                                    void* h, const void* w_packed, const float* bias, int T, int d, int E,
                                    float* logits, void* ws, float*& part, int& S, hipStream_t s,
                                    Guard g = Guard{});
size_t calibrate_ws_bytes(int T, int E);
hipError_t launch_calibrate(const int32_t* idx, const float* w, int T, int E, int k,
                            const int32_t* seg_offsets, int n_seg, double p, double* mass,
                            int32_t* K_out, int32_t* order, void* ws, hipStream_t s, Guard g = Guard{});
// calibration (one segment) and prefix re-route in one launch when
// calibrate_route_fused(T, E, k), else the two launches.  `sort` (one-launch
// path only): the same launch also groups the re-routed entries by expert;
// ctr must be 0 when it runs
struct SortOut {
  int32_t* counts = nullptr;
  int32_t* offsets = nullptr;
  int32_t* src_of_row = nullptr;
  int32_t* row_of_slot = nullptr;
  int* ctr = nullptr;
  int* zero = nullptr;  // then n_zero ints set to 0 (mark_val at mark_at)
  int n_zero = 0, mark_at = -1, mark_val = 0;
};
// ints a launch sets where it no longer uses, or never uses, that part of the
// workspace (0, and mark_val at mark_at): the counters of the call that
// follows, so that it needs no clearing launch
struct ZeroAfter {
  int* p = nullptr;
  int n = 0, mark_at = -1, mark_val = 0;
};
bool calibrate_route_fused(int T, int E, int k);
hipError_t launch_calibrate_route(const float* logits, const int32_t* idx_full, const float* w_full,
                                  int T, int E, int k, double p, double* mass, int32_t* K_out,
                                  int32_t* idx, float* w, hipStream_t s, Guard g = Guard{},
                                  const SortOut* sort = nullptr);
// RCEP routing of one invocation through the dispatch grouping: the split
// router and Top-k, then calibration, re-route and grouping in one launch
// when route_rcep_fused(T, E, k), else route, calibrate_route and dispatch
bool route_rcep_fused(int T, int E, int k);
size_t route_rcep_ws_bytes(int T, int d, int E, int k);
hipError_t launch_route_rcep(const void* x, const void* w_r_packed, const float* bias, int T, int d, int E,
                             int k, double p, float* logits, int32_t* idx_full, float* w_full, double* mass,
                             int32_t* K_out, int32_t* idx, float* w, int32_t* counts, int32_t* offsets,
                             int32_t* src_of_row, int32_t* row_of_slot, void* ws, hipStream_t s,
                             Guard g = Guard{}, const ZeroAfter& za = ZeroAfter{});
// launch_route_rcep on h after the previous layer's combine with the residual
// (h <- h + combine(y_prev, row_prev, w_prev), k slots per token), fused into
// the router launch where combine_router_fits; y_prev = NULL: no combine
hipError_t launch_route_rcep_chained(const void* y_prev, const int32_t* row_prev, const float* w_prev, void* h,
                                     const void* w_r_packed, const float* bias, int T, int d, int E, int k,
                                     double p, float* logits, int32_t* idx_full, float* w_full, double* mass,
                                     int32_t* K_out, int32_t* idx, float* w, int32_t* counts, int32_t* offsets,
                                     int32_t* src_of_row, int32_t* row_of_slot, void* ws, hipStream_t s,
                                     Guard g = Guard{}, const ZeroAfter& za = ZeroAfter{});
size_t dispatch_ws_bytes(int T, int k, int E);
hipError_t launch_dispatch(const int32_t* idx, int T, int k, int E, const void* x, int elt, int d,
                           int32_t* counts, int32_t* offsets, int32_t* src_of_row,
                           int32_t* row_of_slot, void* x_perm, void* ws, hipStream_t s,
                           Guard g = Guard{}, const ZeroAfter& za = ZeroAfter{});
hipError_t launch_expand_dense(const int32_t* idx, const float* w, int T, int k, int E,
                               const int32_t* K_dev, int32_t* idx_dense, float* w_dense, hipStream_t s);
size_t ffn_ws_bytes(bool bf16, int rows_max, int E, int d, int m);
// bytes of the expert FFN's counter header for rows_max rows and E experts
size_t ffn_ctr_bytes(int rows_max, int E);
// bytes from the start of the workspace past the expert FFN's counters (a
// multiple of 256): scratch of earlier launches placed there leaves the
// counters alone
size_t ffn_counter_span(int rows_max, int E);
// Token rows of the gate/up GEMM: x_perm [rows_max, d] when src_of_row is
// NULL; else x [T, d] with dispatched row r read from x[src_of_row[r] / k]
// (packed weights only)
struct RowGather {
  const int32_t* src_of_row;
  int k, T;
};
// K_dev values are clamped to [kmin, E] (kmin: the routing's k where the
// entry point knows it)
hipError_t launch_expert_ffn(const void* a_rows, bool bf16, const int32_t* offsets, int E,
                             const int32_t* K_dev, int n_K, int rows_max, int d, int m,
                             const void* w_gate_up, const void* w_down, bool packed, void* y_perm,
                             void* ws, hipStream_t s, RowGather gather = RowGather{nullptr, 1, 0},
                             int kmin = 1, Guard g = Guard{}, bool counters_ready = false);
// The persistent expert FFN (packed bf16 weights): whether the device runs
// it, and what a launch before it must write so that it runs with no
// clearing launch (counters_ready): the counter header of ws, zeroed, with
// the launch path recorded
bool ffn_persistent_available();
ZeroAfter ffn_counters_zero(void* ws, int rows_max, int E);
// launch path recorded in the expert FFN's counter header
constexpr int FFN_PATH_PERSISTENT = 1;  // both GEMMs in one persistent launch
constexpr int FFN_PATH_TWO_LAUNCH = 2;  // packed weights, one launch per GEMM
constexpr int FFN_PATH_ROW_MAJOR = 3;   // bf16 row-major weights
constexpr int FFN_PATH_F32 = 4;         // float32
// status of the last expert FFN call on a workspace (see ffn_status_kernel)
hipError_t launch_ffn_status(const void* ws, int32_t* status, hipStream_t s);
hipError_t launch_pack_weights(const void* w, int E, int R, int K, void* out, hipStream_t s);
hipError_t launch_combine(const void* y_perm, bool bf16, const int32_t* row_of_slot,
                          const float* w, int T, int k, int d, const void* residual, void* out,
                          hipStream_t s, Guard g = Guard{});
// out block j = in block order[j] for E blocks of `block_bytes` (zeros when
// order[j] lies outside [0, E))
hipError_t launch_permute_blocks(const void* in, const int32_t* order, int E, size_t block_bytes,
                                 void* out, hipStream_t s);
// out[r, j] = in[r, order[j]] for a [rows, E] float32 matrix (0 when out of range)
hipError_t launch_permute_columns(const float* in, const int32_t* order, int rows, int E,
                                  float* out, hipStream_t s);
hipError_t launch_drop_rows(const void* h, int elt, int S, int d, int v0, int v1, void* out,
                            hipStream_t s);
// SAVB gate (Eqs. 2, 3) over n contiguous text rows, and the flag-driven drop
size_t savb_ws_bytes(int n, int d, int hid);
hipError_t launch_savb_gate(const void* rows, bool bf16, int n, int d, const float* w1,
                            const float* b1, int hid, const float* w2, const float* b2, double theta,
                            float* feature, float* p_exit, int32_t* exit_flag, void* ws,
                            hipStream_t s, Guard g = Guard{}, int32_t* exit_layer = nullptr,
                            int layer = 0);
hipError_t launch_drop_rows_if(const void* h, int elt, int S, int d, int v0, int v1,
                               const int32_t* flag, void* out, hipStream_t s);

}  // namespace decomoe
