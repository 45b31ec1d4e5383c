/*
 * decomoe.h - C ABI of the MI355X (gfx950) hot path of DecoMoE's RCEP MoE layer.
 *
 * The library computes one MoE invocation of a multimodal MoE decoder layer
 * in the paper's notation (Sec. 3.1 and Sec. 3.3; Algorithm 2):
 *
 *   logits  a = x W_r + b over all E (reordered) experts        moe_route
 *     (bf16 x: split router weights on bf16 MFMA)                 moe_route_packed,
 *                                                                 moe_pack_router
 *   full-pool Top-k R_i and renormalised weights (Eq. 10)         moe_route
 *   activated mass s (Eq. 11), prefix length K (Eq. 12),
 *   Mean-Mass calibration order pi (Eqs. 8, 9)                    moe_calibrate_prefix
 *   prefix-restricted re-route inside [0, K)                      moe_route
 *     (s, K and the re-route in one call)                         moe_calibrate_route_prefix
 *   grouping of the T*k assignments by expert                     moe_dispatch
 *   SwiGLU expert MLPs over the dispatched rows                   moe_expert_ffn
 *     (same, on weights re-laid out once at load time)            moe_expert_ffn_packed,
 *                                                                 moe_pack_expert_weights
 *     (same, the dispatch gather folded into the GEMM)            moe_expert_ffn_packed_gather
 *   weighted combine back to token order                          moe_combine
 *     (same, plus the residual of a stack of MoE blocks)          moe_combine_residual
 *   one whole dense layer (routing through combine and residual)  moe_dense_layer
 *   one whole RCEP layer (routing through combine and residual)   moe_rcep_layer
 *   the previous layer's combine + one RCEP layer up to its FFN    moe_rcep_layer_chained
 *   SAVB visual-block removal from the hidden state (Sec. 3.2)   drop_visual_block
 *   dense-equivalent routing of the paper's executor (App. A.3)   moe_expand_dense_routing
 *   SAVB exit gate (Eqs. 2, 3) and its device-decided removal     moe_savb_gate,
 *                                                                 drop_visual_block_if
 *   physical expert reorder by pi at load time (Algorithm 1)      moe_permute_experts
 *
 * Conventions shared by every entry point
 *   - Every array pointer is a DEVICE pointer owned by the caller; the
 *     library never allocates or frees device memory at run time and
 *     retains none of the caller's (its only device memory of its own is
 *     the fixed scratch array of moe_expert_ffn_packed_gather_noalloc,
 *     part of the loaded code object).  Arrays are
 *     row-major and contiguous.  Scratch memory comes from the caller as
 *     (ws, ws_bytes); moe_workspace_size() returns a sufficient size.  Its
 *     contents need no initialisation and are not preserved between calls
 *     (the expert FFN clears its own work counters on the stream first, or
 *     in moe_rcep_layer the routing launch before it does).
 *     Calls ordered on one stream may share a workspace; calls that can run
 *     concurrently (other streams) need workspaces of their own.
 *   - Activations and expert weights are MOE_F32 or MOE_BF16 (the `dtype`
 *     argument); router weights, bias, logits and routing weights are
 *     float32; masses are float64; indices, counts and lengths are int32.
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL is the
 *     null stream) and never synchronises with the host.  Calls launch on
 *     the current HIP device (whose CU and XCD counts shape the expert
 *     FFN's persistent launch); the stream and every array must belong to
 *     that device.  Data-dependent
 *     sizes (K, per-expert counts) stay on the device; grids are sized from
 *     the host-side upper bounds passed in.
 *   - Errors: arguments are validated on the host before anything is
 *     launched; on error nothing is launched and a negative MOE_E* code is
 *     returned.  A launch failure reported by the HIP runtime returns
 *     MOE_EHIP.  Contents of device arrays (indices, K values) are not
 *     validated on the host; the kernels clamp or skip out-of-range entries
 *     as documented per function so that no access leaves its array.
 *   - Outputs must not overlap inputs or each other (MOE_EALIAS), except
 *     where stated.
 *   - Array pointers must be 16-byte aligned (MOE_EINVAL otherwise);
 *     drop_visual_block and moe_permute_experts only need element alignment.
 *   - All results are deterministic: repeated calls on the same inputs give
 *     bitwise-identical outputs (no floating-point atomics anywhere).
 */
#ifndef DECOMOE_H
#define DECOMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* hipStream_t;

typedef enum moe_dtype { MOE_F32 = 0, MOE_BF16 = 1 } moe_dtype;

enum {
  MOE_OK = 0,
  MOE_EINVAL = -1,       /* a size or value argument is out of range        */
  MOE_EALIAS = -2,       /* an output overlaps an input or another output   */
  MOE_EWORKSPACE = -3,   /* ws is NULL or ws_bytes is too small             */
  MOE_EHIP = -4,         /* the HIP runtime reported a launch error         */
  MOE_EUNSUPPORTED = -5  /* valid per the method but not supported here     */
};

/* Launch paths of the expert FFN, as reported by moe_ffn_status. */
enum {
  MOE_FFN_PATH_PERSISTENT = 1, /* packed bf16: both GEMMs in one persistent launch */
  MOE_FFN_PATH_TWO_LAUNCH = 2, /* packed bf16: one launch per GEMM                */
  MOE_FFN_PATH_ROW_MAJOR = 3,  /* bf16 row-major weights                          */
  MOE_FFN_PATH_F32 = 4         /* float32                                         */
};

/* Human-readable text of a status code (static storage, never NULL). */
const char* moe_status_string(int status);

/* Bytes of scratch sufficient for every entry point called with sizes up to
 * T tokens, E experts, k slots, hidden size d, expert width m and n_seg
 * segments.  Returns 0 for invalid sizes, including T * k above INT32_MAX
 * (every entry point indexes the routing entries with 32-bit integers). */
size_t moe_workspace_size(int T, int E, int k, int d, int m, int n_seg);

/*
 * moe_route - router logits and Top-k routing (Eq. 1; Eq. 10; the
 * prefix-restricted re-route after Eq. 12 and Algorithm 2).
 *
 *   x          [T, d] token rows (dtype) or NULL.  If x != NULL the logits
 *              a = x W_r + b are computed in float32 and written to
 *              `logits`.  If x == NULL, `logits` is an INPUT (e.g. the
 *              logits of a previous full-pool call) and w_r, bias are unused.
 *   w_r        [d, E] float32 router weights (reordered expert order).
 *   bias       [E] float32 or NULL (no bias).
 *   seg_offsets[n_seg + 1] int32 token offsets of the invocations
 *              (segments), non-decreasing from 0 to T; NULL means one
 *              segment [0, T) and n_seg is then ignored.
 *   K_dev      [n_seg] int32 prefix length per segment, or NULL for K = E
 *              (full-pool routing).  Each K is clamped to [k, E].
 *   logits     [T, E] float32 (output if x != NULL, input otherwise).
 *   topk_idx   [T, k] int32: per token the k experts with the largest
 *              logits among experts [0, K), in descending logit order,
 *              equal logits to the lower expert index.  Softmax is strictly
 *              increasing, so this is the Top-k of the probabilities.
 *   topk_w     [T, k] float32: the softmax over [0, K) restricted to the
 *              selected experts and renormalised, i.e. the softmax of the
 *              k selected logits; each row sums to 1.
 *   ws         scratch (moe_workspace_size): when x != NULL and T is small
 *              the logits are computed in d-range splits whose partial sums
 *              are added in a fixed order (deterministic); NULL is allowed
 *              when no split is needed, else MOE_EWORKSPACE.
 * Limits: 1 <= k <= min(E, 32); 1 <= E <= 1024; T >= 0; d >= 1; for bf16 x,
 * d % 8 == 0.  Logits must be finite.  x == NULL with logits == NULL is
 * MOE_EINVAL.
 */
int moe_route(const void* x, moe_dtype dtype, const float* w_r, const float* bias,
              int T, int d, int E, int k,
              const int32_t* seg_offsets, int n_seg, const int32_t* K_dev,
              float* logits, int32_t* topk_idx, float* topk_w,
              void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_pack_router - one-time split of the float32 router weights into three
 * bf16 terms for moe_route_packed, done when a layer is loaded (like the
 * reorder of Algorithm 1 it is a property of the stored parameters).
 *
 *   w_r         [d, E] float32 router weights.
 *   w_r_packed  d * E * 3 bf16 (6 d E bytes), caller-owned, must not
 *               overlap w_r.  With W1 = bf16(W), W2 = bf16(W - W1),
 *               W3 = bf16(W - W1 - W2) (round to nearest even), the 1 KB
 *               block ((eb * (d / 16) + kb) * 3 + p) holds term p + 1 for
 *               experts 32 eb .. + 32 and k-values 16 kb .. + 16: element
 *               8 l + j is expert 32 eb + l % 32, k = 16 kb + 8 (l / 32) + j.
 * Needs E % 32 == 0 and d % 64 == 0 (else MOE_EUNSUPPORTED).  No workspace.
 */
int moe_pack_router(const float* w_r, int d, int E, void* w_r_packed, hipStream_t stream);

/*
 * moe_route_packed - moe_route for bf16 token rows with the router weights
 * given as moe_pack_router's three-term split: the logits are
 * x W1 + x W2 + x W3 on bf16 MFMA with float32 accumulation.  Each product
 * is exact in float32 and W1 + W2 + W3 equals W to within 2^-24 |W|, so the
 * float32 logits of Eq. 1 are reproduced to within a small multiple of
 * float32 rounding: |a - a_exact| <= (gamma_{3d} + 2^-23) sum_j |x_j W_je|.
 * The Top-k, the weights and every other argument are those of moe_route.
 * x must be non-NULL and bf16 (float32 x: MOE_EUNSUPPORTED; a prefix
 * re-route with x == NULL goes through moe_route).  Needs E % 32 == 0 and
 * d % 64 == 0 (else MOE_EUNSUPPORTED).  ws as for moe_route (its split
 * partials, moe_workspace_size covers both).
 */
int moe_route_packed(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias,
                     int T, int d, int E, int k, const int32_t* seg_offsets, int n_seg,
                     const int32_t* K_dev, float* logits, int32_t* topk_idx, float* topk_w,
                     void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_calibrate_prefix - activated mass, prefix length and Mean-Mass order
 * (Eqs. 8, 9, 11 and 12).
 *
 *   topk_idx, topk_w  [T, k] full-pool routing (moe_route with K_dev = NULL).
 *   seg_offsets       [n_seg + 1] segment offsets or NULL (one segment).
 *   p                 routed-mass fraction, 0 < p <= 1.
 *   mass              [n_seg, E] float64 output: s_e of each segment (Eq. 11).
 *   K_out             [n_seg] int32 output or NULL: K = max(k, K_hat) with
 *                     K_hat the shortest prefix whose running fp64 sum c_K
 *                     satisfies c_K >= p * c_E (Eq. 12).  A segment with no
 *                     tokens gets K = k.
 *   order             [E] int32 output or NULL: the Mean-Mass order pi
 *                     (Eq. 9) with the segments taken as calibration cases:
 *                     each non-empty segment contributes its routed mass
 *                     s_e / len (Eq. 8), the case masses are averaged in
 *                     segment order, and experts are sorted by descending
 *                     mean, equal means keeping the lower index first.
 *                     order[j] is the expert placed at position j.  With no
 *                     non-empty segment the order is the identity.
 * A token's experts are distinct in moe_route output.  An expert repeated
 * within a token: in segments of up to 8192 entries (with E <= 512) its
 * weights are added one by one in slot order, like distinct experts; in
 * larger segments they are first summed within the token (in unspecified
 * order when it repeats three times or more).
 * Each segment's masses are one float64 running sum per expert in ascending
 * token order, and c_K one running sum in expert order, so K depends on the
 * inputs only (no reduction-order effects).  Index entries outside [0, E)
 * are skipped.  Limits: 1 <= k <= min(E, 32).  ws / ws_bytes: scratch per
 * moe_workspace_size; the current implementation needs none (NULL, 0 are accepted).
 */
int moe_calibrate_prefix(const int32_t* topk_idx, const float* topk_w,
                         int T, int E, int k,
                         const int32_t* seg_offsets, int n_seg, double p,
                         double* mass, int32_t* K_out, int32_t* order,
                         void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_calibrate_route_prefix - the RCEP routing of one invocation in one
 * call: the activated mass and prefix length K (Eqs. 11, 12), then the
 * prefix-restricted re-route of every token inside [0, K) (Sec. 3.3 after
 * Eq. 12; Algorithm 2).
 *
 *   logits            [T, E] float32 router logits (from the full-pool
 *                     moe_route / moe_route_packed call).
 *   topk_idx_full,
 *   topk_w_full       [T, k] full-pool routing of the same call.
 *   p                 routed-mass fraction, 0 < p <= 1.
 *   mass              [E] float64 output: s_e of the invocation.
 *   K_out             [1] int32 output: K.
 *   topk_idx, topk_w  [T, k] outputs: the re-routed experts (all < K) and
 *                     their renormalised weights.
 * Bitwise the same results as moe_calibrate_prefix (one segment, order =
 * NULL) followed by moe_route on the logits with K_dev = K_out.  When
 * T*k <= 8192 and E <= 512 it runs as one launch in which every workgroup
 * forms the masses and K itself (a few thousand routing entries) before
 * re-routing its share of the tokens; otherwise as those two launches.
 * Outputs must not overlap the inputs (MOE_EALIAS).  Limits: 1 <= k <=
 * min(E, 32), E <= 1024.  ws / ws_bytes: not needed (NULL, 0 accepted).
 */
int moe_calibrate_route_prefix(const float* logits, const int32_t* topk_idx_full,
                               const float* topk_w_full, int T, int E, int k, double p,
                               double* mass, int32_t* K_out, int32_t* topk_idx, float* topk_w,
                               void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_route_rcep - the RCEP routing of one invocation through the grouping
 * of its dispatch, in one call (Eq. 1, Eq. 10, Eqs. 11-12, the prefix
 * re-route after Eq. 12 and Algorithm 2's dispatch): bitwise the outputs of
 *   moe_route_packed(x, ..., K_dev = NULL)        -> logits, topk_idx_full, topk_w_full
 *   moe_calibrate_route_prefix(p)                  -> mass, K_out, topk_idx, topk_w
 *   moe_dispatch(topk_idx, x = NULL)               -> counts, offsets, src_of_row, row_of_slot
 * with the same arguments, layouts, limits and errors (bf16 x, packed
 * router weights; 1 <= k <= min(E, 32); p in (0, 1]).  When T*k <= 8192
 * and E <= 512, the masses, K, the re-route and the grouping run as one
 * launch after the router's (the last of its workgroups to finish groups
 * the entries); otherwise the three calls run.  T = 0 gives K = k and empty
 * counts.  Needs ws (moe_workspace_size).
 */
int moe_route_rcep(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d,
                   int E, int k, double p, float* logits, int32_t* topk_idx_full, float* topk_w_full,
                   double* mass, int32_t* K_out, int32_t* topk_idx, float* topk_w, int32_t* counts,
                   int32_t* offsets, int32_t* src_of_row, int32_t* row_of_slot, void* ws, size_t ws_bytes,
                   hipStream_t stream);

/*
 * moe_dense_layer - one MoE layer over the full expert pool (the layers
 * before the visual exit in Algorithm 2; Eqs. 1, 10 and App. A.3 Eq. 15),
 * optionally with the residual: bitwise the outputs of
 *   moe_route_packed(x, ..., K_dev = NULL)          -> logits, topk_idx, topk_w
 *   moe_dispatch(topk_idx, ..., x = NULL)           -> counts .. row_of_slot
 *   moe_expert_ffn_packed_gather(x, T, k, src_of_row, offsets, E,
 *                                K_dev = NULL, ...) -> y_perm
 *   moe_combine_residual(y_perm, row_of_slot, topk_w, residual) -> out
 *   (residual = NULL: moe_combine(y_perm, row_of_slot, topk_w) -> out)
 * with those calls' arguments, layouts, limits and errors (bf16 only, packed
 * router and expert weights, 1 <= k <= min(E, 32), d % 256 == 0,
 * m % 256 == 0).  Every argument is checked before anything is launched.
 * `out` [T, d] may be `residual`, `x`, or both; any other overlap of out with
 * an input, and any overlap among the other outputs and inputs, is
 * MOE_EALIAS.  The router's partial logits and the dispatch's histograms are
 * placed in ws past the expert FFN's work counters, so the dispatch's first
 * launch zeroes those counters and the FFN needs no clearing launch of its
 * own; moe_ffn_status afterwards reports the FFN as for
 * moe_expert_ffn_packed_gather.  T = 0 writes empty counts and offsets and
 * launches nothing else.  ws needs moe_workspace_size(T, E, k, d, m, 1)
 * bytes.
 */
int moe_dense_layer(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d, int E,
                    int k, const void* w_gate_up_packed, const void* w_down_packed, int m, const void* residual,
                    void* out, float* logits, int32_t* topk_idx, float* topk_w, int32_t* counts, int32_t* offsets,
                    int32_t* src_of_row, int32_t* row_of_slot, void* y_perm, void* ws, size_t ws_bytes,
                    hipStream_t stream);

/*
 * moe_rcep_layer - one RCEP MoE layer over one invocation (Algorithm 2 with
 * the prefix of Eq. 12), optionally with the residual: bitwise the outputs of
 *   moe_route_rcep(x, ..., p)                     -> logits .. row_of_slot
 *   moe_expert_ffn_packed_gather(x, T, k, src_of_row, offsets, E,
 *                                K_dev = K_out, n_K = 1, d, m, ...)
 *                                                  -> y_perm
 *   moe_combine_residual(y_perm, row_of_slot, topk_w, residual) -> out
 *   (residual = NULL: moe_combine(y_perm, row_of_slot, topk_w) -> out)
 * with those calls' arguments, layouts, limits and errors (bf16 only, packed
 * router and expert weights, 1 <= k <= min(E, 32), d % 256 == 0,
 * m % 256 == 0).  Every argument is checked before anything is launched.
 * `out` [T, d] may be `residual`, `x`, or both (the hidden state updated in
 * place: the combine is the last launch); any other overlap of out with an
 * input, and any overlap among the other outputs and inputs, is MOE_EALIAS.
 * When the routing groups its entries in one launch (T*k <= 8192,
 * E <= 512) and the expert FFN runs persistent, that launch also clears the
 * expert FFN's work counters, so the layer is four launches (router,
 * Top-k, calibration with re-route and grouping, expert FFN) plus the
 * combine; moe_ffn_status afterwards reports the FFN as for
 * moe_expert_ffn_packed_gather.  T = 0 gives K = k and empty counts and
 * launches nothing else.  ws needs max(moe_route_rcep's, the expert FFN's)
 * bytes (moe_workspace_size covers both).
 */
int moe_rcep_layer(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d,
                   int E, int k, double p, const void* w_gate_up_packed, const void* w_down_packed, int m,
                   const void* residual, void* out, float* logits, int32_t* topk_idx_full,
                   float* topk_w_full, double* mass, int32_t* K_out, int32_t* topk_idx, float* topk_w,
                   int32_t* counts, int32_t* offsets, int32_t* src_of_row, int32_t* row_of_slot,
                   void* y_perm, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_rcep_layer_chained - the next RCEP layer of a stack of MoE blocks,
 * starting from the previous layer's expert outputs (Algorithm 2's per-layer
 * loop: the combine with the residual of layer l, then the RCEP layer l + 1
 * up to its expert FFN).
 *
 *   prev_y_perm, prev_row_of_slot, prev_topk_w   the previous layer's y_perm
 *                [T*k, d] bf16, row_of_slot [T, k] and re-routed topk_w
 *                [T, k] (the same T and k), or all three NULL (no previous
 *                layer: the first layer of the stack).
 *   h            [T, d] bf16, in and out: the residual stream.  With the
 *                previous arrays, h <- h + sum_j prev_topk_w[t, j] *
 *                prev_y_perm[prev_row_of_slot[t, j]] (bitwise
 *                moe_combine_residual with residual = out = h); then h is
 *                this layer's input x.
 * The rest as moe_rcep_layer, which this call equals except for its last
 * step: bitwise the outputs of
 *   [moe_combine_residual(prev_y_perm, prev_row_of_slot, prev_topk_w, h, h)]
 *   moe_route_rcep(h, ..., p)                     -> logits .. row_of_slot
 *   moe_expert_ffn_packed_gather(h, ..., K_dev = K_out, n_K = 1)  -> y_perm
 * and this layer's combine is left to the next chained call (whose prev_*
 * are this call's y_perm, row_of_slot, topk_w) or to moe_combine_residual
 * after the last layer.  Each prev_* array may be this call's array of the
 * same role (prev_y_perm == y_perm, prev_row_of_slot == row_of_slot,
 * prev_topk_w == topk_w: the first launch reads them before any launch of
 * the call writes them); any other overlap of an argument with an output
 * is MOE_EALIAS.  When the router's plan keeps a token tile of at most
 * 32 KB per workgroup (one expert group: E <= 128) and the routing groups
 * its entries in one launch (T*k <= 8192), the combine runs inside the
 * router's launch: each router workgroup forms the rows and columns of h it
 * multiplies, writes them and keeps them in LDS; the layer is then four
 * launches (router with the previous combine, Top-k, calibration with
 * re-route and grouping, expert FFN).  Otherwise the combine is a launch of
 * its own.  Same limits, errors and workspace as moe_rcep_layer; T = 0
 * gives K = k and empty counts.
 */
int moe_rcep_layer_chained(const void* prev_y_perm, const int32_t* prev_row_of_slot, const float* prev_topk_w,
                           void* h, moe_dtype dtype, const void* w_r_packed, const float* bias, int T, int d, int E,
                           int k, double p, const void* w_gate_up_packed, const void* w_down_packed, int m,
                           float* logits, int32_t* topk_idx_full, float* topk_w_full, double* mass, int32_t* K_out,
                           int32_t* topk_idx, float* topk_w, int32_t* counts, int32_t* offsets, int32_t* src_of_row,
                           int32_t* row_of_slot, void* y_perm, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_dispatch - group the T*k (token, slot) assignments by expert
 * (Algorithm 2: only the selected experts are evaluated).
 *
 *   topk_idx     [T, k] int32 expert per slot.
 *   x            [T, d] token rows (dtype) or NULL (then x_perm is not written).
 *   counts       [E] int32: rows per expert.
 *   offsets      [E + 1] int32: exclusive prefix sum of counts.
 *   src_of_row   [T*k] int32: dispatched row r -> assignment t*k + j.
 *   row_of_slot  [T*k] int32: assignment t*k + j -> dispatched row r.
 *   x_perm       [T*k, d] (dtype): x_perm[r] = x[src_of_row[r] / k].
 * The grouping is a stable counting sort: within an expert rows ascend by
 * token.  Entries of topk_idx outside [0, E) are dropped (not counted, no
 * row), so offsets[E] < T*k flags them.  Needs ws.
 */
int moe_dispatch(const int32_t* topk_idx, int T, int k, int E,
                 const void* x, moe_dtype dtype, int d,
                 int32_t* counts, int32_t* offsets,
                 int32_t* src_of_row, int32_t* row_of_slot, void* x_perm,
                 void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_expert_ffn - SwiGLU expert MLPs over the dispatched rows, experts
 * [0, K) only (Algorithm 2; gate, up and down projections as counted in
 * App. A.3, Eq. 15).
 *
 *   x_perm     [rows_max, d] dispatched rows (dtype), grouped by `offsets`.
 *   offsets    [E + 1] int32 from moe_dispatch.
 *   K_dev      [n_K] int32 or NULL: experts e >= max(K_dev[0..n_K)), that
 *              maximum clamped to [1, E], are not evaluated (their rows, of
 *              which prefix routing leaves none, are left unwritten); NULL
 *              evaluates all E experts.  moe_route raises a K below its k to
 *              k, so K_dev must hold values >= that k (Eq. 12 gives
 *              K >= k); moe_expert_ffn_packed_gather, which knows k,
 *              clamps to [k, E] itself.
 *   rows_max   upper bound of offsets[E] (normally T*k).
 *   w_gate_up  [E, 2m, d] (dtype): rows [0, m) gate, [m, 2m) up projection.
 *   w_down     [E, d, m] (dtype).
 *   y_perm     [rows_max, d] (dtype) output: for row r of expert e,
 *              y = W_down[e] (SiLU(W_gate[e] x) * (W_up[e] x)),
 *              SiLU(z) = z / (1 + exp(-z)).
 * Arithmetic: bf16 inputs use bf16 MFMA with float32 accumulation; the
 * intermediate SiLU(g)*u is formed in float32 and rounded once to dtype
 * before the down projection; y is rounded once to dtype.  float32 inputs
 * use float32 arithmetic throughout.
 * Limits (bf16): d % 256 == 0 and m % 128 == 0, else MOE_EUNSUPPORTED.
 * Offsets are clamped to [0, rows_max].  Needs ws.
 */
int moe_expert_ffn(const void* x_perm, moe_dtype dtype, const int32_t* offsets, int E,
                   const int32_t* K_dev, int n_K, int rows_max, int d, int m,
                   const void* w_gate_up, const void* w_down, void* y_perm,
                   void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_pack_expert_weights - one-time re-layout of bf16 expert weights for
 * moe_expert_ffn_packed, done when a layer is loaded (like the physical
 * Mean-Mass reorder of the expert parameters, Sec. 3.3 and Algorithm 1, it
 * moves storage and computes nothing).
 *
 *   w         [E, rows, cols] bf16, row-major (w_gate_up: rows 2m, cols d;
 *             w_down: rows d, cols m).
 *   w_packed  E * rows * cols bf16 output, caller-owned, same size as w,
 *             must not overlap it.  For expert e, row r, column c it holds
 *             w[e, r, c] at element offset
 *               e*rows*cols + ((c/16) * (rows/32) + r/32) * 512
 *                 + 8 * ((r % 32) + 32 * ((c % 16) / 8)) + c % 8,
 *             i.e. 1 KB blocks that are the first operand of one
 *             32x32x16 bf16 MFMA (lane l: row 32 rb + l % 32, columns
 *             16 kb + 8 (l / 32) .. +8), blocks of one 16-wide column slice
 *             in row order.
 * bf16 only (MOE_EUNSUPPORTED for float32); rows % 32 == 0 and
 * cols % 16 == 0, else MOE_EUNSUPPORTED.  No workspace.
 */
int moe_pack_expert_weights(const void* w, moe_dtype dtype, int E, int rows, int cols,
                            void* w_packed, hipStream_t stream);

/*
 * moe_expert_ffn_packed - moe_expert_ffn on packed weights: the same
 * arguments, results and limits, with w_gate_up_packed and w_down_packed
 * produced by moe_pack_expert_weights from [E, 2m, d] and [E, d, m].  The
 * weight operand then streams from HBM in contiguous runs straight into
 * registers.  bf16 only (MOE_EUNSUPPORTED for float32); d % 256 == 0 and
 * m % 256 == 0, else MOE_EUNSUPPORTED.  Needs ws (moe_workspace_size).
 */
int moe_expert_ffn_packed(const void* x_perm, moe_dtype dtype, const int32_t* offsets, int E,
                          const int32_t* K_dev, int n_K, int rows_max, int d, int m,
                          const void* w_gate_up_packed, const void* w_down_packed,
                          void* y_perm, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_expert_ffn_packed_gather - moe_expert_ffn_packed with the row gather
 * of moe_dispatch folded into the expert GEMM (Algorithm 2: the selected
 * experts evaluate their tokens):
 *
 *   x           [T, d] bf16 token rows (not dispatched).
 *   k           slots per token (as given to moe_dispatch).
 *   src_of_row  [T*k] int32 from moe_dispatch: dispatched row r is token
 *               src_of_row[r] / k (an index outside [0, T) reads token 0).
 *   offsets, K_dev, n_K, weights, y_perm, ws: as moe_expert_ffn_packed,
 *               with rows_max = T*k.
 * y_perm is bitwise what moe_dispatch (with x) followed by
 * moe_expert_ffn_packed gives, but x_perm is never formed: call moe_dispatch
 * with x = NULL.  Each K_dev value is clamped to [k, E], the clamp moe_route
 * applies, so every expert the prefix re-route can select is evaluated.  bf16 only; d % 256 == 0 and m % 256 == 0, T*d*2 and T*k
 * below 2^31, else MOE_EUNSUPPORTED.  y_perm and ws must not overlap any
 * input (MOE_EALIAS).  Needs ws (moe_workspace_size).
 */
int moe_expert_ffn_packed_gather(const void* x, moe_dtype dtype, int T, int k,
                                 const int32_t* src_of_row, const int32_t* offsets, int E,
                                 const int32_t* K_dev, int n_K, int d, int m,
                                 const void* w_gate_up_packed, const void* w_down_packed,
                                 void* y_perm, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * moe_expert_ffn_packed_gather_noalloc - moe_expert_ffn_packed_gather for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops, harnesses that forbid hipMalloc): the same arguments
 * without (ws, ws_bytes), the same checks and bitwise the same y_perm.
 * Its scratch (the intermediate h and the persistent kernel's counters) is
 * a device array of MOE_NOALLOC_SCRATCH_BYTES inside the library, one per
 * GPU, held until the process ends; the call allocates nothing (no
 * hipMalloc, no hipFree) and on its first use on a device looks up that
 * device's copy of the array once.  Every call on a GPU shares that GPU's
 * array: calls that may overlap on one GPU (other streams, other threads)
 * race and must be serialised by the caller.  The counters are cleared by
 * each call; nothing else needs to start at zero.
 * Limit: the workspace moe_expert_ffn_packed_gather would need,
 * 256 + 4 * (128 + ceil(T*k / 64) + E) rounded up to 256
 *     + T * k * m * 2 rounded up to 256 bytes,
 * must fit MOE_NOALLOC_SCRATCH_BYTES, else MOE_EWORKSPACE (nothing is
 * launched).  With m = 768 that is up to 21 800 dispatched rows (T * k).
 */
#define MOE_NOALLOC_SCRATCH_BYTES (32u << 20)
int moe_expert_ffn_packed_gather_noalloc(const void* x, moe_dtype dtype, int T, int k,
                                         const int32_t* src_of_row, const int32_t* offsets, int E,
                                         const int32_t* K_dev, int n_K, int d, int m,
                                         const void* w_gate_up_packed, const void* w_down_packed,
                                         void* y_perm, hipStream_t stream);

/*
 * Predicated calls (for Algorithm 2's prefill as one captured HIP graph: the
 * SAVB exit, Sec. 3.2, is decided on the device, so both per-layer variants
 * are captured and the device state picks the one that runs).
 *
 * Each *_if call takes the arguments of the call it is named after, plus
 *   guard, guard_lo, guard_hi   a device int32 and a half-open range: the
 *       call's kernels run only if guard_lo <= *guard < guard_hi when they
 *       execute (the value is read on the device, so a captured graph
 *       replays the decision with the value of each replay); otherwise they
 *       return at once and every output, workspace contents included, is
 *       left as it was.  guard == NULL always runs.  guard must be 4-byte
 *       aligned (MOE_EINVAL otherwise).  Nothing else in the call may write
 *       *guard, except moe_savb_gate_if's exit_layer (below).
 * Host-side checks and errors are those of the plain call; they do not
 * depend on the predicate.  With guard == NULL the results are bitwise
 * those of the plain call.  moe_ffn_status after a skipped expert FFN call
 * reports the previous call.
 */
int moe_route_packed_if(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias,
                        int T, int d, int E, int k, const int32_t* seg_offsets, int n_seg,
                        const int32_t* K_dev, float* logits, int32_t* topk_idx, float* topk_w,
                        void* ws, size_t ws_bytes, const int32_t* guard, int guard_lo, int guard_hi,
                        hipStream_t stream);
int moe_route_rcep_if(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T,
                      int d, int E, int k, double p, float* logits, int32_t* topk_idx_full,
                      float* topk_w_full, double* mass, int32_t* K_out, int32_t* topk_idx, float* topk_w,
                      int32_t* counts, int32_t* offsets, int32_t* src_of_row, int32_t* row_of_slot,
                      void* ws, size_t ws_bytes, const int32_t* guard, int guard_lo, int guard_hi,
                      hipStream_t stream);
int moe_rcep_layer_if(const void* x, moe_dtype dtype, const void* w_r_packed, const float* bias, int T,
                      int d, int E, int k, double p, const void* w_gate_up_packed, const void* w_down_packed,
                      int m, const void* residual, void* out, float* logits, int32_t* topk_idx_full,
                      float* topk_w_full, double* mass, int32_t* K_out, int32_t* topk_idx, float* topk_w,
                      int32_t* counts, int32_t* offsets, int32_t* src_of_row, int32_t* row_of_slot,
                      void* y_perm, void* ws, size_t ws_bytes, const int32_t* guard, int guard_lo,
                      int guard_hi, hipStream_t stream);
int moe_calibrate_route_prefix_if(const float* logits, const int32_t* topk_idx_full,
                                  const float* topk_w_full, int T, int E, int k, double p,
                                  double* mass, int32_t* K_out, int32_t* topk_idx, float* topk_w,
                                  void* ws, size_t ws_bytes, const int32_t* guard, int guard_lo,
                                  int guard_hi, hipStream_t stream);
int moe_dispatch_if(const int32_t* topk_idx, int T, int k, int E, const void* x, moe_dtype dtype,
                    int d, int32_t* counts, int32_t* offsets, int32_t* src_of_row,
                    int32_t* row_of_slot, void* x_perm, void* ws, size_t ws_bytes,
                    const int32_t* guard, int guard_lo, int guard_hi, hipStream_t stream);
int moe_expert_ffn_packed_gather_if(const void* x, moe_dtype dtype, int T, int k,
                                    const int32_t* src_of_row, const int32_t* offsets, int E,
                                    const int32_t* K_dev, int n_K, int d, int m,
                                    const void* w_gate_up_packed, const void* w_down_packed,
                                    void* y_perm, void* ws, size_t ws_bytes, const int32_t* guard,
                                    int guard_lo, int guard_hi, hipStream_t stream);
int moe_combine_residual_if(const void* y_perm, moe_dtype dtype, const int32_t* row_of_slot,
                            const float* topk_w, int T, int k, int d, const void* residual,
                            void* out, const int32_t* guard, int guard_lo, int guard_hi,
                            hipStream_t stream);
/*
 * moe_savb_gate_if - moe_savb_gate (Eqs. 2, 3) under the predicate, and
 * when it runs and the gate fires (p_exit >= theta), also *exit_layer =
 * layer.  With guard == exit_layer and the range [L, L + 1) for a value L
 * that means "no exit yet", a chain of candidate layers records the first
 * layer whose gate fires and skips every later gate.  exit_layer must not
 * overlap p_exit or exit_flag (MOE_EALIAS) and be 4-byte aligned.
 */
int moe_savb_gate_if(const void* text_rows, moe_dtype dtype, int n, int d, const float* w1,
                     const float* b1, int hid, const float* w2, const float* b2, double theta,
                     float* feature, float* p_exit, int32_t* exit_flag, void* ws, size_t ws_bytes,
                     const int32_t* guard, int guard_lo, int guard_hi, int32_t* exit_layer,
                     int layer, hipStream_t stream);

/*
 * moe_ffn_status - how the last expert FFN call on a workspace ran
 * (Algorithm 2: the first K expert MLPs are all evaluated).
 *
 *   ws, ws_bytes  the workspace given to that call (any moe_expert_ffn*).
 *   status        [4] int32 device output, written on `stream` after the
 *                 call's kernels:
 *                   [0] waits of a down item for its h that ran out of polls
 *                       (the item then read h anyway: its y rows may be wrong)
 *                   [1] work items completed
 *                   [2] work items in the call's plan
 *                   [3] launch path (MOE_FFN_PATH_*)
 *                 Items are counted on the persistent path only (elsewhere
 *                 every item is a workgroup of its own and [0..2] are 0).
 *                 On the persistent path the call evaluated every planned
 *                 item exactly when [0] == 0 and [1] == [2].
 * Call it on the same stream after the FFN call and before anything else
 * reuses the workspace.  ws_bytes >= 1024, else MOE_EWORKSPACE.
 */
int moe_ffn_status(const void* ws, size_t ws_bytes, int32_t* status, hipStream_t stream);

/*
 * moe_combine - weighted combine back to token order (Algorithm 2).
 *
 *   y_perm       [T*k, d] expert outputs per dispatched row (dtype).
 *   row_of_slot  [T*k] int32 from moe_dispatch.
 *   topk_w       [T, k] float32 routing weights.
 *   out          [T, d] (dtype): out_t = sum_{j<k} w_{t,j} y_perm[row_of_slot[t*k+j]],
 *                accumulated in float32 in slot order, rounded once.
 * Slots whose row index lies outside [0, T*k) contribute nothing.
 */
int moe_combine(const void* y_perm, moe_dtype dtype, const int32_t* row_of_slot,
                const float* topk_w, int T, int k, int d, void* out,
                hipStream_t stream);

/*
 * moe_combine_residual - moe_combine followed by the residual connection of
 * a stack of MoE blocks (the hidden stream h <- h + MoE(h) between the
 * layers of Algorithm 2):
 *
 *   out_t = residual_t + sum_{j<k} w_{t,j} y_perm[row_of_slot[t*k+j]],
 *
 * the weighted sum accumulated in float32 in slot order, the residual added
 * in float32, then rounded once to dtype.  `residual` [T, d] (dtype) may be
 * `out` itself (in-place update of the hidden state); any other overlap of
 * out with an input is MOE_EALIAS.  Same arguments and limits otherwise.
 */
int moe_combine_residual(const void* y_perm, moe_dtype dtype, const int32_t* row_of_slot,
                         const float* topk_w, int T, int k, int d, const void* residual,
                         void* out, hipStream_t stream);

/*
 * moe_permute_experts - physical reorder of one layer's expert parameters by
 * the Mean-Mass order pi (Sec. 3.3 after Eq. 9; Algorithm 1): new expert j
 * is native expert order[j] in
 *   w_r        [d, E] float32 router weights (columns permuted),
 *   bias       [E] float32,
 *   w_gate_up  [E, 2m, d] (dtype) and w_down [E, d, m] (dtype) (blocks permuted).
 * `order` [E] int32 is a device array, e.g. moe_calibrate_prefix's order
 * output; it must be a permutation of [0, E).  An entry outside [0, E)
 * yields zeros for that new expert (no out-of-range read); duplicates are
 * not detected.  Each input/output pair may be NULL/NULL to skip that
 * tensor (one of a pair NULL without the other is MOE_EINVAL).  Outputs
 * must not overlap any input (MOE_EALIAS).  Runs once when a layer is
 * loaded; it moves storage and computes nothing.  No workspace.
 */
int moe_permute_experts(const int32_t* order, int E, int d, int m, moe_dtype dtype,
                        const float* w_r, const float* bias, const void* w_gate_up,
                        const void* w_down, float* w_r_out, float* bias_out,
                        void* w_gate_up_out, void* w_down_out, hipStream_t stream);

/*
 * drop_visual_block - SAVB visual-block removal from the hidden state
 * (Sec. 3.2: at the exit the complete visual block leaves the sequence;
 * Algorithm 2).
 *
 *   h    [S, d] hidden rows (dtype); the visual block is rows [v0, v1).
 *   out  [S - (v1 - v0), d]: rows [0, v0) then [v1, S) of h, order kept,
 *        copied bit for bit.  out must not overlap h (MOE_EALIAS).
 * Needs 0 <= v0 <= v1 <= S.  The exit decision itself is the caller's.
 */
int drop_visual_block(const void* h, moe_dtype dtype, int S, int d, int v0, int v1,
                      void* out, hipStream_t stream);

/*
 * moe_expand_dense_routing - the routing of the paper's dense-equivalent
 * executor (App. A.3: a dense batched product over every physically
 * retained expert, sparse routing weights applied afterwards), for
 * comparison with the sparse path.  With K = K_dev[0] (clamped to [0, E];
 * NULL: K = E):
 *   idx_dense [T, E] int32: slot j of token t is expert j if j < K, else -1
 *                            (moe_dispatch drops it);
 *   w_dense   [T, E] float32: the weight topk_w gave expert j for token t, or
 *                            0 when it was not among the token's k experts.
 * Then moe_dispatch (k = E) -> moe_expert_ffn -> moe_combine (k = E)
 * evaluates every token on experts [0, K): the same output as the sparse
 * path in exact arithmetic, at K/k times its expert FLOPs.  No workspace.
 */
int moe_expand_dense_routing(const int32_t* topk_idx, const float* topk_w, int T, int k, int E,
                             const int32_t* K_dev, int32_t* idx_dense, float* w_dense,
                             hipStream_t stream);

/*
 * moe_savb_gate - the SAVB visual-exit gate at one candidate layer
 * (Sec. 3.2, Eqs. 2 and 3).
 *
 *   text_rows  [n, d] (dtype): the incoming hidden states of the n text
 *              tokens, contiguous (e.g. h + t0 * d for text rows [t0, t0+n)).
 *   x          = [mean of text rows 0 .. n-2; text row n-1] (width 2d;
 *              n == 1: the mean part is zero), formed in float32.
 *   w1 [hid, 2d], b1 [hid] or NULL, w2 [2, hid], b2 [2] or NULL: float32
 *              weights of the two-class MLP g(x) = W2 relu(W1 x + b1) + b2
 *              (the hidden activation is a reading: the paper gives the
 *              layer sizes only).
 *   feature    [2d] float32 output x, or NULL.
 *   p_exit     [1] float32: softmax(g(x))_1, class 1 being the exit class.
 *   exit_flag  [1] int32: 1 if p_exit >= theta (compared in float64), else 0.
 * Every sum has a fixed order (deterministic).  Needs ws of
 * moe_savb_workspace_size(n, d, hid) bytes.  Limits: n >= 1, 1 <= d <= 8192,
 * hid >= 1, theta not NaN.  Device pointers; nothing is read back on the host.
 */
size_t moe_savb_workspace_size(int n, int d, int hid);
int moe_savb_gate(const void* text_rows, moe_dtype dtype, int n, int d, const float* w1,
                  const float* b1, int hid, const float* w2, const float* b2, double theta,
                  float* feature, float* p_exit, int32_t* exit_flag, void* ws, size_t ws_bytes,
                  hipStream_t stream);

/*
 * drop_visual_block_if - drop_visual_block decided on the device: the rows
 * outside [v0, v1) are written to `out` when *exit_flag != 0 (the gate
 * triggered); otherwise nothing is written.  exit_flag is a device int32
 * (moe_savb_gate's output), read by the kernel; the host never waits for it.
 * Same limits and errors as drop_visual_block; out must not overlap h or the
 * flag.
 */
int drop_visual_block_if(const void* h, moe_dtype dtype, int S, int d, int v0, int v1,
                         const int32_t* exit_flag, void* out, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DECOMOE_H */
