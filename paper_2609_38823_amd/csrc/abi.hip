// Exported C ABI: host-side validation, then the launches.  Nothing here
// allocates, frees or synchronises.
#include <mutex>

#include "common.hpp"

#include "../../include/decomoe.h"

namespace {

using decomoe::calibrate_ws_bytes;
using decomoe::dispatch_ws_bytes;
using decomoe::ffn_ws_bytes;
using decomoe::route_ws_bytes;

static_assert(MOE_FFN_PATH_PERSISTENT == decomoe::FFN_PATH_PERSISTENT &&
                  MOE_FFN_PATH_TWO_LAUNCH == decomoe::FFN_PATH_TWO_LAUNCH &&
                  MOE_FFN_PATH_ROW_MAJOR == decomoe::FFN_PATH_ROW_MAJOR &&
                  MOE_FFN_PATH_F32 == decomoe::FFN_PATH_F32,
              "launch path codes of the header and the kernels agree");

constexpr int kMaxE = 1024;
constexpr int kMaxK = 32;

struct Range {
  uintptr_t lo, hi;  // [lo, hi)
};
Range rng(const void* p, size_t bytes) {
  uintptr_t a = reinterpret_cast<uintptr_t>(p);
  return Range{a, a + bytes};
}
bool overlap(Range a, Range b) {
  if (a.lo == a.hi || b.lo == b.hi || !a.lo || !b.lo) return false;
  return a.lo < b.hi && b.lo < a.hi;
}
// true if any output overlaps any input or another output
bool any_alias(std::initializer_list<Range> outs, std::initializer_list<Range> ins) {
  for (auto o = outs.begin(); o != outs.end(); ++o) {
    for (const Range& i : ins)
      if (overlap(*o, i)) return true;
    for (auto o2 = o + 1; o2 != outs.end(); ++o2)
      if (overlap(*o, *o2)) return true;
  }
  return false;
}
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned_all(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (p && !aligned16(p)) return false;
  return true;
}
int elt_size(moe_dtype dt) { return dt == MOE_BF16 ? 2 : 4; }
// the predicate of the *_if entry points: a device int32 (4-byte aligned) or NULL
bool guard_ok(const int32_t* guard) { return (reinterpret_cast<uintptr_t>(guard) & 3u) == 0; }
bool valid_dtype(moe_dtype dt) { return dt == MOE_F32 || dt == MOE_BF16; }
int hip_status(hipError_t e) { return e == hipSuccess ? MOE_OK : MOE_EHIP; }
size_t a256(size_t b) { return (b + 255) & ~size_t(255); }
// shapes of the three-term bf16 router (32-expert blocks, 64-wide k stages)
bool router_packable(int d, int E) { return E % 32 == 0 && d % 64 == 0; }
size_t dense_layer_ws_bytes(int T, int d, int E, int k, int m);

// validation shared by the row-major and packed expert FFN entry points
int expert_ffn(const void* x_perm, moe_dtype dtype, const int32_t* offsets, int E,
               const int32_t* K_dev, int n_K, int rows_max, int d, int m,
               const void* w_gate_up, const void* w_down, bool packed, void* y_perm, void* ws,
               size_t ws_bytes, hipStream_t stream) {
  if (!valid_dtype(dtype) || E < 1 || E > kMaxE || rows_max < 0 || d < 1 || m < 1) return MOE_EINVAL;
  if (K_dev && n_K < 1) return MOE_EINVAL;
  if (!offsets || !w_gate_up || !w_down) return MOE_EINVAL;
  if (rows_max > 0 && (!x_perm || !y_perm)) return MOE_EINVAL;
  const bool bf16 = dtype == MOE_BF16;
  if (bf16 && (d % 256 != 0 || m % 128 != 0)) return MOE_EUNSUPPORTED;
  // the GEMM addresses one expert's weights with 32-bit buffer offsets
  if ((size_t)2 * m * d * elt_size(dtype) > (size_t)INT32_MAX) return MOE_EUNSUPPORTED;
  if (!aligned_all({x_perm, offsets, K_dev, w_gate_up, w_down, y_perm, ws})) return MOE_EINVAL;
  if (rows_max == 0) return MOE_OK;
  const size_t need = ffn_ws_bytes(bf16, rows_max, E, d, m);
  if (!ws || ws_bytes < need) return MOE_EWORKSPACE;
  const int es = elt_size(dtype);
  Range o_y = rng(y_perm, (size_t)rows_max * d * es);
  Range o_ws = rng(ws, need);
  Range in_k = K_dev ? rng(K_dev, (size_t)n_K * 4) : Range{0, 0};
  if (any_alias({o_y, o_ws},
                {rng(x_perm, (size_t)rows_max * d * es), rng(offsets, (size_t)(E + 1) * 4), in_k,
                 rng(w_gate_up, (size_t)E * 2 * m * d * es), rng(w_down, (size_t)E * d * m * es)}))
    return MOE_EALIAS;
  return hip_status(decomoe::launch_expert_ffn(x_perm, bf16, offsets, E, K_dev, n_K, rows_max, d,
                                               m, w_gate_up, w_down, packed, y_perm, ws,
                                               stream));
}

}  // namespace

extern "C" {

const char* moe_status_string(int status) {
  switch (status) {
    case MOE_OK: return "ok";
    case MOE_EINVAL: return "invalid argument (size, range or pointer)";
    case MOE_EALIAS: return "an output overlaps an input or another output";
    case MOE_EWORKSPACE: return "workspace missing or too small";
    case MOE_EHIP: return "HIP runtime reported a launch error";
    case MOE_EUNSUPPORTED: return "shape not supported by this library";
    default: return "unknown status";
  }
}

size_t moe_workspace_size(int T, int E, int k, int d, int m, int n_seg) {
  if (T < 0 || E < 1 || E > kMaxE || k < 1 || k > E || d < 1 || m < 1 || n_seg < 1) return 0;
  // every entry point indexes the T * k routing entries with 32-bit ints
  if ((size_t)T * k > (size_t)INT32_MAX) return 0;
  size_t rows = (size_t)T * k;
  size_t w = 256;
  for (size_t b : {a256(dispatch_ws_bytes(T, k, E)), ffn_ws_bytes(true, (int)rows, E, d, m),
                   ffn_ws_bytes(false, (int)rows, E, d, m), a256(route_ws_bytes(T, d, E)),
                   a256(router_packable(d, E) ? decomoe::route_x3_ws_bytes(T, d, E) : 0),
                   a256(router_packable(d, E) && T > 0 ? decomoe::route_rcep_ws_bytes(T, d, E, k) : 0),
                   a256(calibrate_ws_bytes(T, E)),
                   router_packable(d, E) && T > 0 ? dense_layer_ws_bytes(T, d, E, k, m) : 0})
    w = b > w ? b : w;
  return w;
}

}  // extern "C"

namespace {
// shared by moe_route (float32 router weights) and moe_route_packed
// (three-term bf16 split of them, from moe_pack_router)
int route(const void* x, moe_dtype dtype, const float* w_r, const void* w_r_packed,
          const float* bias, int T, int d, int E, int k, const int32_t* seg_offsets, int n_seg,
          const int32_t* K_dev, float* logits, int32_t* topk_idx, float* topk_w, void* ws,
          size_t ws_bytes, hipStream_t stream, decomoe::Guard g = decomoe::Guard{}) {
  if (T < 0 || E < 1 || E > kMaxE || k < 1 || k > E) return MOE_EINVAL;
  if (k > kMaxK) return MOE_EUNSUPPORTED;
  if (!seg_offsets) n_seg = 1;
  if (n_seg < 1) return MOE_EINVAL;
  if (!logits) return MOE_EINVAL;
  if (x) {
    if (!valid_dtype(dtype) || d < 1 || (!w_r && !w_r_packed)) return MOE_EINVAL;
    if (dtype == MOE_BF16 && d % 8 != 0) return MOE_EINVAL;
  }
  if (T == 0) return MOE_OK;
  if (!topk_idx || !topk_w) return MOE_EINVAL;
  if (!aligned_all({x, w_r, w_r_packed, bias, seg_offsets, K_dev, logits, topk_idx, topk_w, ws}))
    return MOE_EINVAL;
  const size_t need = !x ? 0 : w_r_packed ? decomoe::route_x3_ws_bytes(T, d, E) : route_ws_bytes(T, d, E);
  if (need && (!ws || ws_bytes < need)) return MOE_EWORKSPACE;
  const size_t nl = (size_t)T * E * 4, nk = (size_t)T * k * 4;
  Range o_ws = need ? rng(ws, need) : Range{0, 0};
  Range in_x = x ? rng(x, (size_t)T * d * elt_size(dtype)) : Range{0, 0};
  Range in_w = !x ? Range{0, 0} : w_r_packed ? rng(w_r_packed, (size_t)d * E * 6) : rng(w_r, (size_t)d * E * 4);
  Range in_b = (x && bias) ? rng(bias, (size_t)E * 4) : Range{0, 0};
  Range in_s = seg_offsets ? rng(seg_offsets, (size_t)(n_seg + 1) * 4) : Range{0, 0};
  Range in_k = K_dev ? rng(K_dev, (size_t)n_seg * 4) : Range{0, 0};
  if (x) {
    if (any_alias({rng(logits, nl), rng(topk_idx, nk), rng(topk_w, nk), o_ws},
                  {in_x, in_w, in_b, in_s, in_k}))
      return MOE_EALIAS;
  } else {
    if (any_alias({rng(topk_idx, nk), rng(topk_w, nk)}, {rng(logits, nl), in_s, in_k})) return MOE_EALIAS;
  }
  return hip_status(decomoe::launch_route(x, dtype == MOE_BF16, w_r, x ? w_r_packed : nullptr, bias,
                                          T, d, E, k, seg_offsets, n_seg, K_dev, logits, topk_idx,
                                          topk_w, ws, stream, g));
}

int route_packed(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T,
                 int d, int E, int k, const int32_t* seg_offsets, int n_seg, const int32_t* K_dev,
                 float* logits, int32_t* topk_idx, float* topk_w, void* ws, size_t ws_bytes,
                 hipStream_t stream, decomoe::Guard g) {
  if (!x || !w_r_packed) return MOE_EINVAL;
  if (!valid_dtype(dtype)) return MOE_EINVAL;
  if (dtype != MOE_BF16) return MOE_EUNSUPPORTED;
  if (E < 1 || d < 1) return MOE_EINVAL;
  if (!router_packable(d, E)) return MOE_EUNSUPPORTED;
  return route(x, dtype, nullptr, w_r_packed, bias, T, d, E, k, seg_offsets, n_seg, K_dev, logits,
               topk_idx, topk_w, ws, ws_bytes, stream, g);
}
}  // namespace

extern "C" {

int moe_route(const void* x, moe_dtype dtype, const float* w_r, const float* bias, int T, int d,
              int E, int k, const int32_t* seg_offsets, int n_seg, const int32_t* K_dev,
              float* logits, int32_t* topk_idx, float* topk_w, void* ws, size_t ws_bytes,
              hipStream_t stream) {
  if (x && !w_r) return MOE_EINVAL;
  return route(x, dtype, w_r, nullptr, bias, T, d, E, k, seg_offsets, n_seg, K_dev, logits,
               topk_idx, topk_w, ws, ws_bytes, stream);
}

int moe_route_packed(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias,
                     int T, int d, int E, int k, const int32_t* seg_offsets, int n_seg,
                     const int32_t* K_dev, float* logits, int32_t* topk_idx, float* topk_w,
                     void* ws, size_t ws_bytes, hipStream_t stream) {
  return route_packed(x, dtype, w_r_packed, bias, T, d, E, k, seg_offsets, n_seg, K_dev, logits,
                      topk_idx, topk_w, ws, ws_bytes, stream, decomoe::Guard{});
}

int moe_route_packed_if(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias,
                        int T, int d, int E, int k, const int32_t* seg_offsets, int n_seg,
                        const int32_t* K_dev, float* logits, int32_t* topk_idx, float* topk_w,
                        void* ws, size_t ws_bytes, const int32_t* guard, int guard_lo, int guard_hi,
                        hipStream_t stream) {
  if (!guard_ok(guard)) return MOE_EINVAL;
  return route_packed(x, dtype, w_r_packed, bias, T, d, E, k, seg_offsets, n_seg, K_dev, logits,
                      topk_idx, topk_w, ws, ws_bytes, stream, decomoe::Guard{guard, guard_lo, guard_hi});
}

int moe_pack_router(const float* w_r, int d, int E, void* w_r_packed, hipStream_t stream) {
  if (d < 1 || E < 1 || E > kMaxE || !w_r || !w_r_packed) return MOE_EINVAL;
  if (!router_packable(d, E)) return MOE_EUNSUPPORTED;
  if (!aligned_all({w_r, w_r_packed})) return MOE_EINVAL;
  if (overlap(rng(w_r, (size_t)d * E * 4), rng(w_r_packed, (size_t)d * E * 6))) return MOE_EALIAS;
  return hip_status(decomoe::launch_pack_router(w_r, d, E, w_r_packed, stream));
}

int moe_calibrate_prefix(const int32_t* topk_idx, const float* topk_w, int T, int E, int k,
                         const int32_t* seg_offsets, int n_seg, double p, double* mass,
                         int32_t* K_out, int32_t* order, void* ws, size_t ws_bytes,
                         hipStream_t stream) {
  if (T < 0 || E < 1 || E > kMaxE || k < 1 || k > E) return MOE_EINVAL;
  if (k > kMaxK) return MOE_EUNSUPPORTED;
  if (!seg_offsets) n_seg = 1;
  if (n_seg < 1) return MOE_EINVAL;
  if (!(p > 0.0 && p <= 1.0)) return MOE_EINVAL;
  if (!mass || (T > 0 && (!topk_idx || !topk_w))) return MOE_EINVAL;
  if (!aligned_all({topk_idx, topk_w, seg_offsets, mass, K_out, order, ws})) return MOE_EINVAL;
  const size_t need = calibrate_ws_bytes(T, E);
  if (need && (!ws || ws_bytes < need)) return MOE_EWORKSPACE;
  const size_t nk = (size_t)T * k * 4;
  Range in_i = T ? rng(topk_idx, nk) : Range{0, 0};
  Range in_w = T ? rng(topk_w, nk) : Range{0, 0};
  Range in_s = seg_offsets ? rng(seg_offsets, (size_t)(n_seg + 1) * 4) : Range{0, 0};
  Range o_k = K_out ? rng(K_out, (size_t)n_seg * 4) : Range{0, 0};
  Range o_o = order ? rng(order, (size_t)E * 4) : Range{0, 0};
  Range o_ws = need ? rng(ws, need) : Range{0, 0};
  if (any_alias({rng(mass, (size_t)n_seg * E * 8), o_k, o_o, o_ws}, {in_i, in_w, in_s}))
    return MOE_EALIAS;
  return hip_status(decomoe::launch_calibrate(topk_idx, topk_w, T, E, k, seg_offsets, n_seg, p,
                                              mass, K_out, order, ws, stream));
}

}  // extern "C"

namespace {
int calibrate_route_prefix(const float* logits, const int32_t* topk_idx_full,
                           const float* topk_w_full, int T, int E, int k, double p, double* mass,
                           int32_t* K_out, int32_t* topk_idx, float* topk_w, hipStream_t stream,
                           decomoe::Guard g) {
  if (T < 0 || E < 1 || E > kMaxE || k < 1 || k > E) return MOE_EINVAL;
  if (k > kMaxK) return MOE_EUNSUPPORTED;
  if (!(p > 0.0 && p <= 1.0)) return MOE_EINVAL;
  if (!mass || !K_out) return MOE_EINVAL;
  if (T > 0 && (!logits || !topk_idx_full || !topk_w_full || !topk_idx || !topk_w)) return MOE_EINVAL;
  if (!aligned_all({logits, topk_idx_full, topk_w_full, mass, K_out, topk_idx, topk_w})) return MOE_EINVAL;
  const size_t nl = (size_t)T * E * 4, nk = (size_t)T * k * 4;
  Range in_l = T ? rng(logits, nl) : Range{0, 0};
  Range in_i = T ? rng(topk_idx_full, nk) : Range{0, 0};
  Range in_w = T ? rng(topk_w_full, nk) : Range{0, 0};
  Range o_i = T ? rng(topk_idx, nk) : Range{0, 0};
  Range o_w = T ? rng(topk_w, nk) : Range{0, 0};
  if (any_alias({rng(mass, (size_t)E * 8), rng(K_out, 4), o_i, o_w}, {in_l, in_i, in_w})) return MOE_EALIAS;
  return hip_status(decomoe::launch_calibrate_route(logits, topk_idx_full, topk_w_full, T, E, k, p, mass,
                                                    K_out, topk_idx, topk_w, stream, g));
}
}  // namespace

extern "C" {

int moe_calibrate_route_prefix(const float* logits, const int32_t* topk_idx_full,
                               const float* topk_w_full, int T, int E, int k, double p, double* mass,
                               int32_t* K_out, int32_t* topk_idx, float* topk_w, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  (void)ws;
  (void)ws_bytes;
  return calibrate_route_prefix(logits, topk_idx_full, topk_w_full, T, E, k, p, mass, K_out, topk_idx,
                                topk_w, stream, decomoe::Guard{});
}

int moe_calibrate_route_prefix_if(const float* logits, const int32_t* topk_idx_full,
                                  const float* topk_w_full, int T, int E, int k, double p,
                                  double* mass, int32_t* K_out, int32_t* topk_idx, float* topk_w,
                                  void* ws, size_t ws_bytes, const int32_t* guard, int guard_lo,
                                  int guard_hi, hipStream_t stream) {
  (void)ws;
  (void)ws_bytes;
  if (!guard_ok(guard)) return MOE_EINVAL;
  return calibrate_route_prefix(logits, topk_idx_full, topk_w_full, T, E, k, p, mass, K_out, topk_idx,
                                topk_w, stream, decomoe::Guard{guard, guard_lo, guard_hi});
}

}  // extern "C"

namespace {
int dispatch(const int32_t* topk_idx, int T, int k, int E, const void* x, moe_dtype dtype, int d,
             int32_t* counts, int32_t* offsets, int32_t* src_of_row, int32_t* row_of_slot,
             void* x_perm, void* ws, size_t ws_bytes, hipStream_t stream, decomoe::Guard g) {
  if (T < 0 || E < 1 || E > kMaxE || k < 1 || k > E) return MOE_EINVAL;
  if ((size_t)T * k > (size_t)INT32_MAX) return MOE_EUNSUPPORTED;
  if (!counts || !offsets) return MOE_EINVAL;
  if (T > 0 && (!topk_idx || !src_of_row || !row_of_slot)) return MOE_EINVAL;
  if (x && (!valid_dtype(dtype) || d < 1 || (T > 0 && !x_perm))) return MOE_EINVAL;
  if (!aligned_all({topk_idx, x, counts, offsets, src_of_row, row_of_slot, x_perm, ws}))
    return MOE_EINVAL;
  const size_t need = dispatch_ws_bytes(T, k, E);
  if (need > 0 && (!ws || ws_bytes < need)) return MOE_EWORKSPACE;
  const size_t A = (size_t)T * k;
  Range in_i = rng(topk_idx, A * 4);
  Range in_x = x ? rng(x, (size_t)T * d * elt_size(dtype)) : Range{0, 0};
  Range o_xp = x ? rng(x_perm, A * d * elt_size(dtype)) : Range{0, 0};
  Range o_ws = rng(ws, need);
  if (any_alias({rng(counts, (size_t)E * 4), rng(offsets, (size_t)(E + 1) * 4), rng(src_of_row, A * 4),
                 rng(row_of_slot, A * 4), o_xp, o_ws},
                {in_i, in_x}))
    return MOE_EALIAS;
  return hip_status(decomoe::launch_dispatch(topk_idx, T, k, E, x, elt_size(dtype), d, counts,
                                             offsets, src_of_row, row_of_slot, x_perm, ws, stream, g));
}
}  // namespace

extern "C" {

}  // extern "C"

namespace {
// moe_route_packed (full pool) + moe_calibrate_route_prefix +
// moe_dispatch (x = NULL) of one invocation
int route_rcep(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d,
               int E, int k, double p, float* logits, int32_t* idx_full, float* w_full, double* mass,
               int32_t* K_out, int32_t* idx, float* w, int32_t* counts, int32_t* offsets,
               int32_t* src_of_row, int32_t* row_of_slot, void* ws, size_t ws_bytes, hipStream_t stream,
               decomoe::Guard g) {
  if (!valid_dtype(dtype) || T < 0 || d < 1 || E < 1 || E > kMaxE || k < 1 || k > E) return MOE_EINVAL;
  if (dtype != MOE_BF16 || !router_packable(d, E)) return MOE_EUNSUPPORTED;
  if (k > kMaxK) return MOE_EUNSUPPORTED;
  if ((size_t)T * k > (size_t)INT32_MAX) return MOE_EUNSUPPORTED;
  if (!(p > 0.0 && p <= 1.0)) return MOE_EINVAL;
  if (!mass || !K_out || !counts || !offsets) return MOE_EINVAL;
  if (T > 0 && (!x || !w_r_packed || !logits || !idx_full || !w_full || !idx || !w || !src_of_row ||
                !row_of_slot))
    return MOE_EINVAL;
  if (!aligned_all({x, w_r_packed, bias, logits, idx_full, w_full, mass, K_out, idx, w, counts, offsets,
                    src_of_row, row_of_slot, ws}))
    return MOE_EINVAL;
  const size_t need = T > 0 ? decomoe::route_rcep_ws_bytes(T, d, E, k) : 0;
  if (need && (!ws || ws_bytes < need)) return MOE_EWORKSPACE;
  const size_t A = (size_t)T * k, nl = (size_t)T * E * 4;
  if (any_alias({rng(logits, nl), rng(idx_full, A * 4), rng(w_full, A * 4), rng(mass, (size_t)E * 8),
                 rng(K_out, 4), rng(idx, A * 4), rng(w, A * 4), rng(counts, (size_t)E * 4),
                 rng(offsets, (size_t)(E + 1) * 4), rng(src_of_row, A * 4), rng(row_of_slot, A * 4),
                 need ? rng(ws, need) : Range{0, 0}},
                {rng(x, (size_t)T * d * 2), rng(w_r_packed, (size_t)d * E * 6),
                 bias ? rng(bias, (size_t)E * 4) : Range{0, 0}}))
    return MOE_EALIAS;
  if (T == 0) {  // an empty invocation: K = k, no rows
    hipError_t e = decomoe::launch_calibrate_route(logits, idx_full, w_full, 0, E, k, p, mass, K_out, idx,
                                                   w, stream, g);
    if (e == hipSuccess)
      e = decomoe::launch_dispatch(idx, 0, k, E, nullptr, 2, 0, counts, offsets, src_of_row, row_of_slot,
                                   nullptr, ws, stream, g);
    return hip_status(e);
  }
  return hip_status(decomoe::launch_route_rcep(x, w_r_packed, bias, T, d, E, k, p, logits, idx_full, w_full,
                                               mass, K_out, idx, w, counts, offsets, src_of_row, row_of_slot,
                                               ws, stream, g));
}
}  // namespace

extern "C" {

int moe_route_rcep(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d,
                   int E, int k, double p, float* logits, int32_t* topk_idx_full, float* topk_w_full,
                   double* mass, int32_t* K_out, int32_t* topk_idx, float* topk_w, int32_t* counts,
                   int32_t* offsets, int32_t* src_of_row, int32_t* row_of_slot, void* ws, size_t ws_bytes,
                   hipStream_t stream) {
  return route_rcep(x, dtype, w_r_packed, bias, T, d, E, k, p, logits, topk_idx_full, topk_w_full, mass,
                    K_out, topk_idx, topk_w, counts, offsets, src_of_row, row_of_slot, ws, ws_bytes, stream,
                    decomoe::Guard{});
}

int moe_route_rcep_if(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T,
                      int d, int E, int k, double p, float* logits, int32_t* topk_idx_full,
                      float* topk_w_full, double* mass, int32_t* K_out, int32_t* topk_idx, float* topk_w,
                      int32_t* counts, int32_t* offsets, int32_t* src_of_row, int32_t* row_of_slot,
                      void* ws, size_t ws_bytes, const int32_t* guard, int guard_lo, int guard_hi,
                      hipStream_t stream) {
  if (!guard_ok(guard)) return MOE_EINVAL;
  return route_rcep(x, dtype, w_r_packed, bias, T, d, E, k, p, logits, topk_idx_full, topk_w_full, mass,
                    K_out, topk_idx, topk_w, counts, offsets, src_of_row, row_of_slot, ws, ws_bytes, stream,
                    decomoe::Guard{guard, guard_lo, guard_hi});
}

int moe_dispatch(const int32_t* topk_idx, int T, int k, int E, const void* x, moe_dtype dtype,
                 int d, int32_t* counts, int32_t* offsets, int32_t* src_of_row,
                 int32_t* row_of_slot, void* x_perm, void* ws, size_t ws_bytes,
                 hipStream_t stream) {
  return dispatch(topk_idx, T, k, E, x, dtype, d, counts, offsets, src_of_row, row_of_slot, x_perm, ws,
                  ws_bytes, stream, decomoe::Guard{});
}

int moe_dispatch_if(const int32_t* topk_idx, int T, int k, int E, const void* x, moe_dtype dtype,
                    int d, int32_t* counts, int32_t* offsets, int32_t* src_of_row,
                    int32_t* row_of_slot, void* x_perm, void* ws, size_t ws_bytes,
                    const int32_t* guard, int guard_lo, int guard_hi, hipStream_t stream) {
  if (!guard_ok(guard)) return MOE_EINVAL;
  return dispatch(topk_idx, T, k, E, x, dtype, d, counts, offsets, src_of_row, row_of_slot, x_perm, ws,
                  ws_bytes, stream, decomoe::Guard{guard, guard_lo, guard_hi});
}

int moe_expert_ffn(const void* x_perm, moe_dtype dtype, const int32_t* offsets, int E,
                   const int32_t* K_dev, int n_K, int rows_max, int d, int m,
                   const void* w_gate_up, const void* w_down, void* y_perm, void* ws,
                   size_t ws_bytes, hipStream_t stream) {
  return expert_ffn(x_perm, dtype, offsets, E, K_dev, n_K, rows_max, d, m, w_gate_up, w_down,
                    false, y_perm, ws, ws_bytes, stream);
}

int moe_expert_ffn_packed(const void* x_perm, moe_dtype dtype, const int32_t* offsets, int E,
                          const int32_t* K_dev, int n_K, int rows_max, int d, int m,
                          const void* w_gate_up_packed, const void* w_down_packed, void* y_perm,
                          void* ws, size_t ws_bytes, hipStream_t stream) {
  if (dtype != MOE_BF16) return valid_dtype(dtype) ? MOE_EUNSUPPORTED : MOE_EINVAL;
  if (d % 256 != 0 || m % 256 != 0) return (d > 0 && m > 0) ? MOE_EUNSUPPORTED : MOE_EINVAL;
  return expert_ffn(x_perm, dtype, offsets, E, K_dev, n_K, rows_max, d, m, w_gate_up_packed,
                    w_down_packed, true, y_perm, ws, ws_bytes, stream);
}

}  // extern "C"

namespace {
// Host-side checks of moe_expert_ffn_packed_gather and its allocation-free
// variant, before the workspace: MOE_OK with *rows_max set, or the status.
int gather_ffn_args(const void* x, moe_dtype dtype, int T, int k, const int32_t* src_of_row,
                    const int32_t* offsets, int E, const int32_t* K_dev, int n_K, int d, int m,
                    const void* w_gate_up_packed, const void* w_down_packed, void* y_perm,
                    int* rows_max_out) {
  if (!valid_dtype(dtype) || T < 0 || k < 1 || E < 1 || E > kMaxE || k > E || d < 1 || m < 1)
    return MOE_EINVAL;
  if (dtype != MOE_BF16) return MOE_EUNSUPPORTED;
  if (d % 256 != 0 || m % 256 != 0) return MOE_EUNSUPPORTED;
  // token rows and dispatched rows are addressed with 32-bit offsets
  if ((size_t)T * k > (size_t)INT32_MAX || (size_t)T * d * 2 > (size_t)INT32_MAX)
    return MOE_EUNSUPPORTED;
  if ((size_t)2 * m * d * 2 > (size_t)INT32_MAX) return MOE_EUNSUPPORTED;
  if (K_dev && n_K < 1) return MOE_EINVAL;
  if (!offsets || !w_gate_up_packed || !w_down_packed) return MOE_EINVAL;
  const int rows_max = T * k;
  if (rows_max > 0 && (!x || !src_of_row || !y_perm)) return MOE_EINVAL;
  if (!aligned_all({x, src_of_row, offsets, K_dev, w_gate_up_packed, w_down_packed, y_perm}))
    return MOE_EINVAL;
  *rows_max_out = rows_max;
  return MOE_OK;
}

// Aliasing checks and the launch (ws: the caller's workspace, or the
// library's scratch array of the allocation-free variant).
int gather_ffn_launch(const void* x, int T, int k, const int32_t* src_of_row, const int32_t* offsets,
                      int E, const int32_t* K_dev, int n_K, int d, int m, const void* w_gate_up_packed,
                      const void* w_down_packed, void* y_perm, void* ws, size_t need,
                      hipStream_t stream, decomoe::Guard g = decomoe::Guard{}) {
  const int rows_max = T * k;
  Range o_y = rng(y_perm, (size_t)rows_max * d * 2);
  Range o_ws = rng(ws, need);
  Range in_k = K_dev ? rng(K_dev, (size_t)n_K * 4) : Range{0, 0};
  if (any_alias({o_y, o_ws},
                {rng(x, (size_t)T * d * 2), rng(src_of_row, (size_t)rows_max * 4),
                 rng(offsets, (size_t)(E + 1) * 4), in_k,
                 rng(w_gate_up_packed, (size_t)E * 2 * m * d * 2),
                 rng(w_down_packed, (size_t)E * d * m * 2)}))
    return MOE_EALIAS;
  return hip_status(decomoe::launch_expert_ffn(x, true, offsets, E, K_dev, n_K, rows_max, d, m,
                                               w_gate_up_packed, w_down_packed, true, y_perm, ws,
                                               stream, decomoe::RowGather{src_of_row, k, T}, k, g));
}
}  // namespace

extern "C" {

int moe_expert_ffn_packed_gather(const void* x, moe_dtype dtype, int T, int k,
                                 const int32_t* src_of_row, const int32_t* offsets, int E,
                                 const int32_t* K_dev, int n_K, int d, int m,
                                 const void* w_gate_up_packed, const void* w_down_packed,
                                 void* y_perm, void* ws, size_t ws_bytes, hipStream_t stream) {
  int rows_max = 0;
  const int st = gather_ffn_args(x, dtype, T, k, src_of_row, offsets, E, K_dev, n_K, d, m,
                                 w_gate_up_packed, w_down_packed, y_perm, &rows_max);
  if (st != MOE_OK) return st;
  if (!aligned_all({ws})) return MOE_EINVAL;
  if (rows_max == 0) return MOE_OK;
  const size_t need = ffn_ws_bytes(true, rows_max, E, d, m);
  if (!ws || ws_bytes < need) return MOE_EWORKSPACE;
  return gather_ffn_launch(x, T, k, src_of_row, offsets, E, K_dev, n_K, d, m, w_gate_up_packed,
                           w_down_packed, y_perm, ws, need, stream);
}

int moe_expert_ffn_packed_gather_if(const void* x, moe_dtype dtype, int T, int k,
                                    const int32_t* src_of_row, const int32_t* offsets, int E,
                                    const int32_t* K_dev, int n_K, int d, int m,
                                    const void* w_gate_up_packed, const void* w_down_packed,
                                    void* y_perm, void* ws, size_t ws_bytes, const int32_t* guard,
                                    int guard_lo, int guard_hi, hipStream_t stream) {
  if (!guard_ok(guard)) return MOE_EINVAL;
  int rows_max = 0;
  const int st = gather_ffn_args(x, dtype, T, k, src_of_row, offsets, E, K_dev, n_K, d, m,
                                 w_gate_up_packed, w_down_packed, y_perm, &rows_max);
  if (st != MOE_OK) return st;
  if (!aligned_all({ws})) return MOE_EINVAL;
  if (rows_max == 0) return MOE_OK;
  const size_t need = ffn_ws_bytes(true, rows_max, E, d, m);
  if (!ws || ws_bytes < need) return MOE_EWORKSPACE;
  return gather_ffn_launch(x, T, k, src_of_row, offsets, E, K_dev, n_K, d, m, w_gate_up_packed,
                           w_down_packed, y_perm, ws, need, stream,
                           decomoe::Guard{guard, guard_lo, guard_hi});
}

int moe_ffn_status(const void* ws, size_t ws_bytes, int32_t* status, hipStream_t stream) {
  if (!ws || !status || !aligned_all({ws, status})) return MOE_EINVAL;
  // the counter header starts at the first 256-byte boundary of ws
  if (ws_bytes < 256 + decomoe::ffn_ctr_bytes(0, 1)) return MOE_EWORKSPACE;
  if (overlap(rng(status, 16), rng(ws, ws_bytes))) return MOE_EALIAS;
  return hip_status(decomoe::launch_ffn_status(ws, status, stream));
}

int moe_pack_expert_weights(const void* w, moe_dtype dtype, int E, int rows, int cols,
                            void* w_packed, hipStream_t stream) {
  if (!valid_dtype(dtype) || E < 0 || rows < 0 || cols < 0) return MOE_EINVAL;
  if (dtype != MOE_BF16) return MOE_EUNSUPPORTED;
  if (rows % 32 != 0 || cols % 16 != 0) return MOE_EUNSUPPORTED;
  const size_t bytes = (size_t)E * rows * cols * 2;
  if (bytes == 0) return MOE_OK;
  if (!w || !w_packed || !aligned_all({w, w_packed})) return MOE_EINVAL;
  if (overlap(rng(w, bytes), rng(w_packed, bytes))) return MOE_EALIAS;
  return hip_status(decomoe::launch_pack_weights(w, E, rows, cols, w_packed, stream));
}

int moe_combine(const void* y_perm, moe_dtype dtype, const int32_t* row_of_slot,
                const float* topk_w, int T, int k, int d, void* out, hipStream_t stream) {
  if (!valid_dtype(dtype) || T < 0 || k < 1 || k > kMaxE || d < 1) return MOE_EINVAL;
  if ((size_t)T * k > (size_t)INT32_MAX) return MOE_EUNSUPPORTED;
  if (T == 0) return MOE_OK;
  if (!y_perm || !row_of_slot || !topk_w || !out) return MOE_EINVAL;
  if (!aligned_all({y_perm, row_of_slot, topk_w, out})) return MOE_EINVAL;
  const int es = elt_size(dtype);
  const size_t A = (size_t)T * k;
  if (any_alias({rng(out, (size_t)T * d * es)},
                {rng(y_perm, A * d * es), rng(row_of_slot, A * 4), rng(topk_w, A * 4)}))
    return MOE_EALIAS;
  return hip_status(decomoe::launch_combine(y_perm, dtype == MOE_BF16, row_of_slot, topk_w, T, k,
                                            d, nullptr, out, stream));
}

}  // extern "C"

namespace {
int combine_residual(const void* y_perm, moe_dtype dtype, const int32_t* row_of_slot,
                     const float* topk_w, int T, int k, int d, const void* residual, void* out,
                     hipStream_t stream, decomoe::Guard g) {
  if (!valid_dtype(dtype) || T < 0 || k < 1 || k > kMaxE || d < 1) return MOE_EINVAL;
  if ((size_t)T * k > (size_t)INT32_MAX) return MOE_EUNSUPPORTED;
  if (T == 0) return MOE_OK;
  if (!y_perm || !row_of_slot || !topk_w || !residual || !out) return MOE_EINVAL;
  if (!aligned_all({y_perm, row_of_slot, topk_w, residual, out})) return MOE_EINVAL;
  const int es = elt_size(dtype);
  const size_t A = (size_t)T * k;
  const Range o = rng(out, (size_t)T * d * es), r = rng(residual, (size_t)T * d * es);
  // out may be residual itself, but not a shifted view of it
  if (r.lo != o.lo && overlap(o, r)) return MOE_EALIAS;
  if (any_alias({o}, {rng(y_perm, A * d * es), rng(row_of_slot, A * 4), rng(topk_w, A * 4)}))
    return MOE_EALIAS;
  return hip_status(decomoe::launch_combine(y_perm, dtype == MOE_BF16, row_of_slot, topk_w, T, k,
                                            d, residual, out, stream, g));
}
}  // namespace

extern "C" {

int moe_combine_residual(const void* y_perm, moe_dtype dtype, const int32_t* row_of_slot,
                         const float* topk_w, int T, int k, int d, const void* residual,
                         void* out, hipStream_t stream) {
  return combine_residual(y_perm, dtype, row_of_slot, topk_w, T, k, d, residual, out, stream,
                          decomoe::Guard{});
}

int moe_combine_residual_if(const void* y_perm, moe_dtype dtype, const int32_t* row_of_slot,
                            const float* topk_w, int T, int k, int d, const void* residual,
                            void* out, const int32_t* guard, int guard_lo, int guard_hi,
                            hipStream_t stream) {
  if (!guard_ok(guard)) return MOE_EINVAL;
  return combine_residual(y_perm, dtype, row_of_slot, topk_w, T, k, d, residual, out, stream,
                          decomoe::Guard{guard, guard_lo, guard_hi});
}

}  // extern "C"

namespace {
// One RCEP layer of Algorithm 2 over one invocation: moe_route_rcep, then
// moe_expert_ffn_packed_gather over experts [0, K_out), then
// moe_combine_residual.  Every check runs before the first launch.
int rcep_layer(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d, int E,
               int k, double p, const void* w_gate_up_packed, const void* w_down_packed, int m,
               const void* residual, void* out, float* logits, int32_t* idx_full, float* w_full, double* mass,
               int32_t* K_out, int32_t* idx, float* w, int32_t* counts, int32_t* offsets, int32_t* src_of_row,
               int32_t* row_of_slot, void* y_perm, void* ws, size_t ws_bytes, hipStream_t stream,
               decomoe::Guard g) {
  if (!valid_dtype(dtype) || T < 0 || d < 1 || E < 1 || E > kMaxE || k < 1 || k > E || m < 1)
    return MOE_EINVAL;
  if (dtype != MOE_BF16 || !router_packable(d, E)) return MOE_EUNSUPPORTED;
  if (k > kMaxK) return MOE_EUNSUPPORTED;
  if (d % 256 != 0 || m % 256 != 0) return MOE_EUNSUPPORTED;
  if ((size_t)T * k > (size_t)INT32_MAX || (size_t)T * d * 2 > (size_t)INT32_MAX ||
      (size_t)2 * m * d * 2 > (size_t)INT32_MAX)
    return MOE_EUNSUPPORTED;
  if (!(p > 0.0 && p <= 1.0)) return MOE_EINVAL;
  if (!mass || !K_out || !counts || !offsets || !w_gate_up_packed || !w_down_packed) return MOE_EINVAL;
  if (T > 0 && (!x || !w_r_packed || !logits || !idx_full || !w_full || !idx || !w || !src_of_row ||
                !row_of_slot || !y_perm || !out))
    return MOE_EINVAL;
  if (!aligned_all({x, w_r_packed, bias, w_gate_up_packed, w_down_packed, residual, out, logits, idx_full,
                    w_full, mass, K_out, idx, w, counts, offsets, src_of_row, row_of_slot, y_perm, ws}))
    return MOE_EINVAL;
  const int rows = T * k;
  size_t need = 0;
  if (T > 0) {
    const size_t a = decomoe::route_rcep_ws_bytes(T, d, E, k), b = ffn_ws_bytes(true, rows, E, d, m);
    need = a > b ? a : b;
  }
  if (need && (!ws || ws_bytes < need)) return MOE_EWORKSPACE;
  const size_t A = (size_t)rows, nl = (size_t)T * E * 4, xb = (size_t)T * d * 2;
  // out may be the residual rows and x themselves (the hidden state updated
  // in place), but no shifted view of them
  const Range o = rng(out, xb), r = residual ? rng(residual, xb) : Range{0, 0}, xi = rng(x, xb);
  if ((residual && o.lo != r.lo && overlap(o, r)) || (o.lo != xi.lo && overlap(o, xi))) return MOE_EALIAS;
  const Range wr = rng(w_r_packed, (size_t)d * E * 6), bi = bias ? rng(bias, (size_t)E * 4) : Range{0, 0},
              wgu = rng(w_gate_up_packed, (size_t)E * 2 * m * d * 2),
              wdn = rng(w_down_packed, (size_t)E * d * m * 2);
  if (any_alias({o}, {wr, bi, wgu, wdn}) ||
      any_alias({rng(logits, nl), rng(idx_full, A * 4), rng(w_full, A * 4), rng(mass, (size_t)E * 8),
                 rng(K_out, 4), rng(idx, A * 4), rng(w, A * 4), rng(counts, (size_t)E * 4),
                 rng(offsets, (size_t)(E + 1) * 4), rng(src_of_row, A * 4), rng(row_of_slot, A * 4),
                 rng(y_perm, A * d * 2), need ? rng(ws, need) : Range{0, 0}},
                {xi, r, o, wr, bi, wgu, wdn}))
    return MOE_EALIAS;
  if (T == 0)  // K = k and empty counts; no rows to evaluate or combine
    return route_rcep(nullptr, dtype, nullptr, nullptr, 0, d, E, k, p, nullptr, nullptr, nullptr, mass, K_out,
                      nullptr, nullptr, counts, offsets, nullptr, nullptr, ws, ws_bytes, stream, g);
  // with the one-launch grouping the calibration launch also clears the
  // expert FFN's counters in the workspace, and the FFN runs with no
  // clearing launch of its own
  const bool fold = decomoe::route_rcep_fused(T, E, k) && decomoe::ffn_persistent_available();
  const decomoe::ZeroAfter za = fold ? decomoe::ffn_counters_zero(ws, rows, E) : decomoe::ZeroAfter{};
  hipError_t e = decomoe::launch_route_rcep(x, w_r_packed, bias, T, d, E, k, p, logits, idx_full, w_full, mass,
                                            K_out, idx, w, counts, offsets, src_of_row, row_of_slot, ws, stream,
                                            g, za);
  if (e == hipSuccess)
    e = decomoe::launch_expert_ffn(x, true, offsets, E, K_out, 1, rows, d, m, w_gate_up_packed, w_down_packed,
                                   true, y_perm, ws, stream, decomoe::RowGather{src_of_row, k, T}, k, g, fold);
  if (e == hipSuccess)
    e = decomoe::launch_combine(y_perm, true, row_of_slot, w, T, k, d, residual, out, stream, g);
  return hip_status(e);
}

// moe_dense_layer: see the header
size_t dense_layer_ws_bytes(int T, int d, int E, int k, int m) {
  const int rows = T * k;
  const size_t r = a256(decomoe::route_x3_ws_bytes(T, d, E)), q = a256(dispatch_ws_bytes(T, k, E));
  const size_t early = decomoe::ffn_counter_span(rows, E) + (r > q ? r : q);
  const size_t f = ffn_ws_bytes(true, rows, E, d, m);
  return early > f ? early : f;
}

int dense_layer(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d, int E,
                int k, const void* w_gate_up_packed, const void* w_down_packed, int m, const void* residual,
                void* out, float* logits, int32_t* idx, float* w, int32_t* counts, int32_t* offsets,
                int32_t* src_of_row, int32_t* row_of_slot, void* y_perm, void* ws, size_t ws_bytes,
                hipStream_t stream) {
  if (!valid_dtype(dtype) || T < 0 || d < 1 || E < 1 || E > kMaxE || k < 1 || k > E || m < 1)
    return MOE_EINVAL;
  if (dtype != MOE_BF16 || !router_packable(d, E)) return MOE_EUNSUPPORTED;
  if (k > kMaxK) return MOE_EUNSUPPORTED;
  if (d % 256 != 0 || m % 256 != 0) return MOE_EUNSUPPORTED;
  if ((size_t)T * k > (size_t)INT32_MAX || (size_t)T * d * 2 > (size_t)INT32_MAX ||
      (size_t)T * k * d * 2 > (size_t)INT32_MAX || (size_t)2 * m * d * 2 > (size_t)INT32_MAX)
    return MOE_EUNSUPPORTED;
  if (!counts || !offsets || !w_gate_up_packed || !w_down_packed) return MOE_EINVAL;
  if (T > 0 && (!x || !w_r_packed || !logits || !idx || !w || !src_of_row || !row_of_slot || !y_perm || !out))
    return MOE_EINVAL;
  if (!aligned_all({x, w_r_packed, bias, w_gate_up_packed, w_down_packed, residual, out, logits, idx, w, counts,
                    offsets, src_of_row, row_of_slot, y_perm, ws}))
    return MOE_EINVAL;
  const size_t need = T > 0 ? dense_layer_ws_bytes(T, d, E, k, m) : 0;
  if (need && (!ws || ws_bytes < need)) return MOE_EWORKSPACE;
  const size_t A = (size_t)T * k, xb = (size_t)T * d * 2;
  // out may be the residual rows and x themselves, but no shifted view of them
  const Range o = rng(out, xb), r = residual ? rng(residual, xb) : Range{0, 0}, xi = rng(x, xb);
  if ((residual && o.lo != r.lo && overlap(o, r)) || (o.lo != xi.lo && overlap(o, xi))) return MOE_EALIAS;
  const Range wr = rng(w_r_packed, (size_t)d * E * 6), bi = bias ? rng(bias, (size_t)E * 4) : Range{0, 0},
              wgu = rng(w_gate_up_packed, (size_t)E * 2 * m * d * 2),
              wdn = rng(w_down_packed, (size_t)E * d * m * 2);
  if (any_alias({o}, {wr, bi, wgu, wdn}) ||
      any_alias({rng(logits, (size_t)T * E * 4), rng(idx, A * 4), rng(w, A * 4), rng(counts, (size_t)E * 4),
                 rng(offsets, (size_t)(E + 1) * 4), rng(src_of_row, A * 4), rng(row_of_slot, A * 4),
                 rng(y_perm, A * d * 2), need ? rng(ws, need) : Range{0, 0}},
                {xi, r, o, wr, bi, wgu, wdn}))
    return MOE_EALIAS;
  if (T == 0)  // empty counts and offsets; nothing else to do
    return hip_status(decomoe::launch_dispatch(nullptr, 0, k, E, nullptr, 2, 0, counts, offsets, nullptr, nullptr,
                                               nullptr, nullptr, stream));
  // the router's partial logits and the dispatch's histograms sit past the
  // expert FFN's counters, which the dispatch's first launch then zeroes:
  // the FFN runs without a clearing launch of its own
  const int rows = T * k;
  void* early = static_cast<char*>(ws) + decomoe::ffn_counter_span(rows, E);
  const bool fold = decomoe::ffn_persistent_available();
  const decomoe::ZeroAfter za = fold ? decomoe::ffn_counters_zero(ws, rows, E) : decomoe::ZeroAfter{};
  hipError_t e = decomoe::launch_route(x, true, nullptr, w_r_packed, bias, T, d, E, k, nullptr, 1, nullptr, logits,
                                       idx, w, early, stream);
  if (e == hipSuccess)
    e = decomoe::launch_dispatch(idx, T, k, E, nullptr, 2, 0, counts, offsets, src_of_row, row_of_slot, nullptr,
                                 early, stream, decomoe::Guard{}, za);
  if (e == hipSuccess)
    e = decomoe::launch_expert_ffn(x, true, offsets, E, nullptr, 0, rows, d, m, w_gate_up_packed, w_down_packed,
                                   true, y_perm, ws, stream, decomoe::RowGather{src_of_row, k, T}, k,
                                   decomoe::Guard{}, fold);
  if (e == hipSuccess) e = decomoe::launch_combine(y_perm, true, row_of_slot, w, T, k, d, residual, out, stream,
                                                   decomoe::Guard{});
  return hip_status(e);
}

// moe_rcep_layer_chained: see the header
int rcep_layer_chained(const void* prev_y_perm, const int32_t* prev_row_of_slot, const float* prev_topk_w, void* h,
                       moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d, int E, int k,
                       double p, const void* w_gate_up_packed, const void* w_down_packed, int m, float* logits,
                       int32_t* idx_full, float* w_full, double* mass, int32_t* K_out, int32_t* idx, float* w,
                       int32_t* counts, int32_t* offsets, int32_t* src_of_row, int32_t* row_of_slot, void* y_perm,
                       void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!valid_dtype(dtype) || T < 0 || d < 1 || E < 1 || E > kMaxE || k < 1 || k > E || m < 1)
    return MOE_EINVAL;
  if (dtype != MOE_BF16 || !router_packable(d, E)) return MOE_EUNSUPPORTED;
  if (k > kMaxK) return MOE_EUNSUPPORTED;
  if (d % 256 != 0 || m % 256 != 0) return MOE_EUNSUPPORTED;
  if ((size_t)T * k > (size_t)INT32_MAX || (size_t)T * d * 2 > (size_t)INT32_MAX ||
      (size_t)T * k * d * 2 > (size_t)INT32_MAX || (size_t)2 * m * d * 2 > (size_t)INT32_MAX)
    return MOE_EUNSUPPORTED;
  if (!(p > 0.0 && p <= 1.0)) return MOE_EINVAL;
  const bool prev = prev_y_perm || prev_row_of_slot || prev_topk_w;
  if (prev && !(prev_y_perm && prev_row_of_slot && prev_topk_w)) return MOE_EINVAL;
  if (!mass || !K_out || !counts || !offsets || !w_gate_up_packed || !w_down_packed) return MOE_EINVAL;
  if (T > 0 && (!h || !w_r_packed || !logits || !idx_full || !w_full || !idx || !w || !src_of_row ||
                !row_of_slot || !y_perm))
    return MOE_EINVAL;
  if (!aligned_all({prev_y_perm, prev_row_of_slot, prev_topk_w, h, w_r_packed, bias, w_gate_up_packed,
                    w_down_packed, logits, idx_full, w_full, mass, K_out, idx, w, counts, offsets, src_of_row,
                    row_of_slot, y_perm, ws}))
    return MOE_EINVAL;
  const int rows = T * k;
  size_t need = 0;
  if (T > 0) {
    const size_t a = decomoe::route_rcep_ws_bytes(T, d, E, k), b = ffn_ws_bytes(true, rows, E, d, m);
    need = a > b ? a : b;
  }
  if (need && (!ws || ws_bytes < need)) return MOE_EWORKSPACE;
  const size_t A = (size_t)rows, nl = (size_t)T * E * 4, xb = (size_t)T * d * 2;
  const Range hr = rng(h, xb), wr = rng(w_r_packed, (size_t)d * E * 6),
              bi = bias ? rng(bias, (size_t)E * 4) : Range{0, 0},
              wgu = rng(w_gate_up_packed, (size_t)E * 2 * m * d * 2), wdn = rng(w_down_packed, (size_t)E * d * m * 2);
  const Range o_ws = need ? rng(ws, need) : Range{0, 0}, o_ros = rng(row_of_slot, A * 4), o_w = rng(w, A * 4),
              o_y = rng(y_perm, A * d * 2);
  const std::initializer_list<Range> outs_rest = {rng(logits, nl), rng(idx_full, A * 4), rng(w_full, A * 4),
                                                  rng(mass, (size_t)E * 8), rng(K_out, 4), rng(idx, A * 4),
                                                  rng(counts, (size_t)E * 4), rng(offsets, (size_t)(E + 1) * 4),
                                                  rng(src_of_row, A * 4), o_ws};
  if (any_alias({hr}, {wr, bi, wgu, wdn}) || any_alias(outs_rest, {hr, wr, bi, wgu, wdn}) ||
      any_alias({o_ros, o_w, o_y}, {hr, wr, bi, wgu, wdn}) || any_alias(outs_rest, {o_ros, o_w, o_y}))
    return MOE_EALIAS;
  if (prev && T > 0) {
    // each previous-layer array is this call's array of the same role or
    // overlaps nothing of the call (it is read by the first launch, before
    // any launch of the call writes those arrays)
    const Range q_y = rng(prev_y_perm, A * d * 2), q_r = rng(prev_row_of_slot, A * 4), q_w = rng(prev_topk_w, A * 4);
    const Range others[] = {hr, wr, bi, wgu, wdn};
    for (const Range& q : {q_y, q_r, q_w})
      for (const Range& o : others)
        if (overlap(q, o)) return MOE_EALIAS;
    if (any_alias({q_y, q_r, q_w}, outs_rest)) return MOE_EALIAS;
    if (overlap(q_y, q_r) || overlap(q_y, q_w) || overlap(q_r, q_w)) return MOE_EALIAS;
    if ((q_y.lo != o_y.lo && (overlap(q_y, o_y) || overlap(q_y, o_ros) || overlap(q_y, o_w))) ||
        (q_r.lo != o_ros.lo && (overlap(q_r, o_y) || overlap(q_r, o_ros) || overlap(q_r, o_w))) ||
        (q_w.lo != o_w.lo && (overlap(q_w, o_y) || overlap(q_w, o_ros) || overlap(q_w, o_w))))
      return MOE_EALIAS;
  }
  if (T == 0)
    return route_rcep(nullptr, dtype, nullptr, nullptr, 0, d, E, k, p, nullptr, nullptr, nullptr, mass, K_out,
                      nullptr, nullptr, counts, offsets, nullptr, nullptr, ws, ws_bytes, stream, decomoe::Guard{});
  const bool fold = decomoe::route_rcep_fused(T, E, k) && decomoe::ffn_persistent_available();
  const decomoe::ZeroAfter za = fold ? decomoe::ffn_counters_zero(ws, rows, E) : decomoe::ZeroAfter{};
  hipError_t e = decomoe::launch_route_rcep_chained(prev ? prev_y_perm : nullptr, prev_row_of_slot, prev_topk_w, h,
                                                    w_r_packed, bias, T, d, E, k, p, logits, idx_full, w_full,
                                                    mass, K_out, idx, w, counts, offsets, src_of_row, row_of_slot,
                                                    ws, stream, decomoe::Guard{}, za);
  if (e == hipSuccess)
    e = decomoe::launch_expert_ffn(h, true, offsets, E, K_out, 1, rows, d, m, w_gate_up_packed, w_down_packed, true,
                                   y_perm, ws, stream, decomoe::RowGather{src_of_row, k, T}, k, decomoe::Guard{},
                                   fold);
  return hip_status(e);
}
}  // namespace

extern "C" {

int moe_rcep_layer(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d, int E,
                   int k, double p, const void* w_gate_up_packed, const void* w_down_packed, int m,
                   const void* residual, void* out, float* logits, int32_t* topk_idx_full, float* topk_w_full,
                   double* mass, int32_t* K_out, int32_t* topk_idx, float* topk_w, int32_t* counts,
                   int32_t* offsets, int32_t* src_of_row, int32_t* row_of_slot, void* y_perm, void* ws,
                   size_t ws_bytes, hipStream_t stream) {
  return rcep_layer(x, dtype, w_r_packed, bias, T, d, E, k, p, w_gate_up_packed, w_down_packed, m, residual, out,
                    logits, topk_idx_full, topk_w_full, mass, K_out, topk_idx, topk_w, counts, offsets, src_of_row,
                    row_of_slot, y_perm, ws, ws_bytes, stream, decomoe::Guard{});
}

int moe_rcep_layer_if(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d,
                      int E, int k, double p, const void* w_gate_up_packed, const void* w_down_packed, int m,
                      const void* residual, void* out, float* logits, int32_t* topk_idx_full,
                      float* topk_w_full, double* mass, int32_t* K_out, int32_t* topk_idx, float* topk_w,
                      int32_t* counts, int32_t* offsets, int32_t* src_of_row, int32_t* row_of_slot,
                      void* y_perm, void* ws, size_t ws_bytes, const int32_t* guard, int guard_lo,
                      int guard_hi, hipStream_t stream) {
  if (!guard_ok(guard)) return MOE_EINVAL;
  return rcep_layer(x, dtype, w_r_packed, bias, T, d, E, k, p, w_gate_up_packed, w_down_packed, m, residual, out,
                    logits, topk_idx_full, topk_w_full, mass, K_out, topk_idx, topk_w, counts, offsets, src_of_row,
                    row_of_slot, y_perm, ws, ws_bytes, stream, decomoe::Guard{guard, guard_lo, guard_hi});
}

int moe_dense_layer(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d, int E,
                    int k, const void* w_gate_up_packed, const void* w_down_packed, int m, const void* residual,
                    void* out, float* logits, int32_t* topk_idx, float* topk_w, int32_t* counts, int32_t* offsets,
                    int32_t* src_of_row, int32_t* row_of_slot, void* y_perm, void* ws, size_t ws_bytes,
                    hipStream_t stream) {
  return dense_layer(x, dtype, w_r_packed, bias, T, d, E, k, w_gate_up_packed, w_down_packed, m, residual, out,
                     logits, topk_idx, topk_w, counts, offsets, src_of_row, row_of_slot, y_perm, ws, ws_bytes, stream);
}

int moe_rcep_layer_chained(const void* prev_y_perm, const int32_t* prev_row_of_slot, const float* prev_topk_w,
                           void* h, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d, int E,
                           int k, double p, const void* w_gate_up_packed, const void* w_down_packed, int m,
                           float* logits, int32_t* topk_idx_full, float* topk_w_full, double* mass, int32_t* K_out,
                           int32_t* topk_idx, float* topk_w, int32_t* counts, int32_t* offsets, int32_t* src_of_row,
                           int32_t* row_of_slot, void* y_perm, void* ws, size_t ws_bytes, hipStream_t stream) {
  return rcep_layer_chained(prev_y_perm, prev_row_of_slot, prev_topk_w, h, dtype, w_r_packed, bias, T, d, E, k, p,
                            w_gate_up_packed, w_down_packed, m, logits, topk_idx_full, topk_w_full, mass, K_out,
                            topk_idx, topk_w, counts, offsets, src_of_row, row_of_slot, y_perm, ws, ws_bytes,
                            stream);
}

int moe_permute_experts(const int32_t* order, int E, int d, int m, moe_dtype dtype,
                        const float* w_r, const float* bias, const void* w_gate_up,
                        const void* w_down, float* w_r_out, float* bias_out,
                        void* w_gate_up_out, void* w_down_out, hipStream_t stream) {
  if (!valid_dtype(dtype) || E < 1 || E > kMaxE || d < 1 || m < 1 || !order) return MOE_EINVAL;
  if (!w_r != !w_r_out || !bias != !bias_out || !w_gate_up != !w_gate_up_out ||
      !w_down != !w_down_out)
    return MOE_EINVAL;
  const int es = elt_size(dtype);
  const size_t b_gu = (size_t)2 * m * d * es, b_dn = (size_t)d * m * es;
  if ((reinterpret_cast<uintptr_t>(order) | reinterpret_cast<uintptr_t>(w_r) |
       reinterpret_cast<uintptr_t>(bias) | reinterpret_cast<uintptr_t>(w_r_out) |
       reinterpret_cast<uintptr_t>(bias_out)) % 4)
    return MOE_EINVAL;
  if ((reinterpret_cast<uintptr_t>(w_gate_up) | reinterpret_cast<uintptr_t>(w_down) |
       reinterpret_cast<uintptr_t>(w_gate_up_out) | reinterpret_cast<uintptr_t>(w_down_out)) % es)
    return MOE_EINVAL;
  const Range o_r = w_r ? rng(w_r_out, (size_t)d * E * 4) : Range{0, 0};
  const Range o_b = bias ? rng(bias_out, (size_t)E * 4) : Range{0, 0};
  const Range o_gu = w_gate_up ? rng(w_gate_up_out, E * b_gu) : Range{0, 0};
  const Range o_dn = w_down ? rng(w_down_out, E * b_dn) : Range{0, 0};
  if (any_alias({o_r, o_b, o_gu, o_dn},
                {rng(order, (size_t)E * 4), w_r ? rng(w_r, (size_t)d * E * 4) : Range{0, 0},
                 bias ? rng(bias, (size_t)E * 4) : Range{0, 0},
                 w_gate_up ? rng(w_gate_up, E * b_gu) : Range{0, 0},
                 w_down ? rng(w_down, E * b_dn) : Range{0, 0}}))
    return MOE_EALIAS;
  hipError_t e = hipSuccess;
  if (w_r) e = decomoe::launch_permute_columns(w_r, order, d, E, w_r_out, stream);
  if (e == hipSuccess && bias) e = decomoe::launch_permute_columns(bias, order, 1, E, bias_out, stream);
  if (e == hipSuccess && w_gate_up)
    e = decomoe::launch_permute_blocks(w_gate_up, order, E, b_gu, w_gate_up_out, stream);
  if (e == hipSuccess && w_down)
    e = decomoe::launch_permute_blocks(w_down, order, E, b_dn, w_down_out, stream);
  return hip_status(e);
}

int moe_expand_dense_routing(const int32_t* topk_idx, const float* topk_w, int T, int k, int E,
                             const int32_t* K_dev, int32_t* idx_dense, float* w_dense,
                             hipStream_t stream) {
  if (T < 0 || k < 1 || E < 1 || E > kMaxE) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!topk_idx || !topk_w || !idx_dense || !w_dense) return MOE_EINVAL;
  if (!aligned_all({topk_idx, topk_w, K_dev, idx_dense, w_dense})) return MOE_EINVAL;
  const size_t nk = (size_t)T * k * 4, ne = (size_t)T * E * 4;
  if (any_alias({rng(idx_dense, ne), rng(w_dense, ne)},
                {rng(topk_idx, nk), rng(topk_w, nk), K_dev ? rng(K_dev, 4) : Range{0, 0}}))
    return MOE_EALIAS;
  return hip_status(decomoe::launch_expand_dense(topk_idx, topk_w, T, k, E, K_dev, idx_dense, w_dense,
                                                 stream));
}

size_t moe_savb_workspace_size(int n, int d, int hid) {
  if (n < 1 || d < 1 || hid < 1) return 0;
  return a256(decomoe::savb_ws_bytes(n, d, hid));
}

}  // extern "C"

namespace {
int savb_gate(const void* text_rows, moe_dtype dtype, int n, int d, const float* w1, const float* b1,
              int hid, const float* w2, const float* b2, double theta, float* feature, float* p_exit,
              int32_t* exit_flag, void* ws, size_t ws_bytes, hipStream_t stream, decomoe::Guard g,
              int32_t* exit_layer, int layer) {
  if (!valid_dtype(dtype) || n < 1 || d < 1 || d > 8192 || hid < 1) return MOE_EINVAL;
  if (!(theta == theta)) return MOE_EINVAL;  // NaN
  if (!text_rows || !w1 || !w2 || !p_exit || !exit_flag || !ws) return MOE_EINVAL;
  if (!aligned_all({text_rows, w1, b1, w2, b2, feature, p_exit, exit_flag, ws})) return MOE_EINVAL;
  const size_t need = decomoe::savb_ws_bytes(n, d, hid);
  if (ws_bytes < need) return MOE_EWORKSPACE;
  const Range o_f = feature ? rng(feature, (size_t)2 * d * 4) : Range{0, 0};
  if (any_alias({o_f, rng(p_exit, 4), rng(exit_flag, 4), rng(ws, need)},
                {rng(text_rows, (size_t)n * d * elt_size(dtype)), rng(w1, (size_t)hid * 2 * d * 4),
                 b1 ? rng(b1, (size_t)hid * 4) : Range{0, 0}, rng(w2, (size_t)2 * hid * 4),
                 b2 ? rng(b2, 8) : Range{0, 0}}))
    return MOE_EALIAS;
  if (exit_layer && (overlap(rng(exit_layer, 4), rng(exit_flag, 4)) ||
                     overlap(rng(exit_layer, 4), rng(p_exit, 4))))
    return MOE_EALIAS;
  return hip_status(decomoe::launch_savb_gate(text_rows, dtype == MOE_BF16, n, d, w1, b1, hid, w2, b2,
                                              theta, feature, p_exit, exit_flag, ws, stream, g,
                                              exit_layer, layer));
}
}  // namespace

extern "C" {

int moe_savb_gate(const void* text_rows, moe_dtype dtype, int n, int d, const float* w1,
                  const float* b1, int hid, const float* w2, const float* b2, double theta,
                  float* feature, float* p_exit, int32_t* exit_flag, void* ws, size_t ws_bytes,
                  hipStream_t stream) {
  return savb_gate(text_rows, dtype, n, d, w1, b1, hid, w2, b2, theta, feature, p_exit, exit_flag, ws,
                   ws_bytes, stream, decomoe::Guard{}, nullptr, 0);
}

int moe_savb_gate_if(const void* text_rows, moe_dtype dtype, int n, int d, const float* w1,
                     const float* b1, int hid, const float* w2, const float* b2, double theta,
                     float* feature, float* p_exit, int32_t* exit_flag, void* ws, size_t ws_bytes,
                     const int32_t* guard, int guard_lo, int guard_hi, int32_t* exit_layer,
                     int layer, hipStream_t stream) {
  if (!guard_ok(guard) || !guard_ok(exit_layer)) return MOE_EINVAL;
  return savb_gate(text_rows, dtype, n, d, w1, b1, hid, w2, b2, theta, feature, p_exit, exit_flag, ws,
                   ws_bytes, stream, decomoe::Guard{guard, guard_lo, guard_hi}, exit_layer, layer);
}

int drop_visual_block_if(const void* h, moe_dtype dtype, int S, int d, int v0, int v1,
                         const int32_t* exit_flag, void* out, hipStream_t stream) {
  if (!valid_dtype(dtype) || S < 0 || d < 1) return MOE_EINVAL;
  if (!(0 <= v0 && v0 <= v1 && v1 <= S)) return MOE_EINVAL;
  if (!exit_flag || (reinterpret_cast<uintptr_t>(exit_flag) & 3)) return MOE_EINVAL;
  const int rows_out = S - (v1 - v0);
  if (rows_out == 0) return MOE_OK;
  if (!h || !out) return MOE_EINVAL;
  const int es = elt_size(dtype);
  if ((reinterpret_cast<uintptr_t>(h) | reinterpret_cast<uintptr_t>(out)) % es) return MOE_EINVAL;
  if (overlap(rng(out, (size_t)rows_out * d * es), rng(h, (size_t)S * d * es))) return MOE_EALIAS;
  if (overlap(rng(out, (size_t)rows_out * d * es), rng(exit_flag, 4))) return MOE_EALIAS;
  return hip_status(decomoe::launch_drop_rows_if(h, es, S, d, v0, v1, exit_flag, out, stream));
}

int drop_visual_block(const void* h, moe_dtype dtype, int S, int d, int v0, int v1, void* out,
                      hipStream_t stream) {
  if (!valid_dtype(dtype) || S < 0 || d < 1) return MOE_EINVAL;
  if (!(0 <= v0 && v0 <= v1 && v1 <= S)) return MOE_EINVAL;
  const int rows_out = S - (v1 - v0);
  if (rows_out == 0) return MOE_OK;
  if (!h || !out) return MOE_EINVAL;
  const int es = elt_size(dtype);
  if ((reinterpret_cast<uintptr_t>(h) | reinterpret_cast<uintptr_t>(out)) % es) return MOE_EINVAL;
  if (overlap(rng(out, (size_t)rows_out * d * es), rng(h, (size_t)S * d * es))) return MOE_EALIAS;
  return hip_status(decomoe::launch_drop_rows(h, es, S, d, v0, v1, out, stream));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Allocation-free expert FFN: the intermediate h and the persistent kernel's
// counters live in `scratch`, a file-scope device array of fixed size that
// every GPU the library runs on holds until the process ends.  Host code
// reaches it only through the address hipGetSymbolAddress returns on that
// device (the array's name on the host is a stand-in, not a device address).
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[MOE_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch`, per device

// the current device's address of `scratch`, looked up once per device
int scratch_on_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return MOE_EHIP;
  if (dev >= kMaxDevices) return MOE_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MOE_EHIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return MOE_OK;
}
}  // namespace

extern "C" int moe_expert_ffn_packed_gather_noalloc(const void* x, moe_dtype dtype, int T, int k,
                                                    const int32_t* src_of_row, const int32_t* offsets,
                                                    int E, const int32_t* K_dev, int n_K, int d, int m,
                                                    const void* w_gate_up_packed,
                                                    const void* w_down_packed, void* y_perm,
                                                    hipStream_t stream) {
  int rows_max = 0;
  const int st = gather_ffn_args(x, dtype, T, k, src_of_row, offsets, E, K_dev, n_K, d, m,
                                 w_gate_up_packed, w_down_packed, y_perm, &rows_max);
  if (st != MOE_OK) return st;
  if (rows_max == 0) return MOE_OK;
  const size_t need = ffn_ws_bytes(true, rows_max, E, d, m);
  if (need > (size_t)MOE_NOALLOC_SCRATCH_BYTES) return MOE_EWORKSPACE;
  void* ws = nullptr;
  const int sst = scratch_on_current_device(&ws);
  if (sst != MOE_OK) return sst;
  return gather_ffn_launch(x, T, k, src_of_row, offsets, E, K_dev, n_K, d, m, w_gate_up_packed,
                           w_down_packed, y_perm, ws, need, stream);
}
