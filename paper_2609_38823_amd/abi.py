"""Thin ctypes binding of libdecomoe.so (C ABI in include/decomoe.h).

Argument marshalling only: every step of the path runs in the HIP kernels
of the library.  Functions carry the C names; array arguments are torch
tensors on the GPU (their ``data_ptr()`` is passed), sizes are taken from
the tensors, and the stream defaults to torch's current stream.  A non-zero
status raises ``MoeError``.  There is no fallback: without the built
library every call raises.
"""

from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdecomoe.so")

MOE_F32, MOE_BF16 = 0, 1
STATUS = {0: "MOE_OK", -1: "MOE_EINVAL", -2: "MOE_EALIAS", -3: "MOE_EWORKSPACE",
          -4: "MOE_EHIP", -5: "MOE_EUNSUPPORTED"}

EXPORTS = ("moe_status_string", "moe_workspace_size", "moe_route", "moe_route_packed",
           "moe_pack_router", "moe_calibrate_prefix", "moe_calibrate_route_prefix",
           "moe_dispatch", "moe_expert_ffn", "moe_expert_ffn_packed", "moe_expert_ffn_packed_gather",
           "moe_pack_expert_weights",
           "moe_combine", "moe_combine_residual", "drop_visual_block", "moe_permute_experts",
           "moe_savb_workspace_size", "moe_savb_gate", "drop_visual_block_if",
           "moe_expand_dense_routing", "moe_ffn_status", "moe_expert_ffn_packed_gather_noalloc",
           "moe_route_packed_if", "moe_calibrate_route_prefix_if", "moe_dispatch_if",
           "moe_expert_ffn_packed_gather_if", "moe_combine_residual_if", "moe_savb_gate_if",
           "moe_route_rcep", "moe_route_rcep_if", "moe_rcep_layer", "moe_rcep_layer_if",
           "moe_rcep_layer_chained", "moe_dense_layer")

# size of the library's own scratch array of the allocation-free expert FFN
NOALLOC_SCRATCH_BYTES = 32 << 20

# launch paths of the expert FFN (moe_ffn_status)
FFN_PATH_PERSISTENT, FFN_PATH_TWO_LAUNCH, FFN_PATH_ROW_MAJOR, FFN_PATH_F32 = 1, 2, 3, 4


class MoeError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} returned {STATUS.get(status, status)}: {_status_text(status)}")


_lib = None
_P, _I, _D, _S = ctypes.c_void_p, ctypes.c_int, ctypes.c_double, ctypes.c_size_t


def load() -> ctypes.CDLL:
    """Load the in-tree library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_38823_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    sig = {
        "moe_status_string": (ctypes.c_char_p, [_I]),
        "moe_workspace_size": (_S, [_I, _I, _I, _I, _I, _I]),
        "moe_route": (_I, [_P, _I, _P, _P, _I, _I, _I, _I, _P, _I, _P, _P, _P, _P, _P, _S, _P]),
        "moe_route_packed": (_I, [_P, _I, _P, _P, _I, _I, _I, _I, _P, _I, _P, _P, _P, _P, _P, _S, _P]),
        "moe_pack_router": (_I, [_P, _I, _I, _P, _P]),
        "moe_calibrate_prefix": (_I, [_P, _P, _I, _I, _I, _P, _I, _D, _P, _P, _P, _P, _S, _P]),
        "moe_calibrate_route_prefix": (_I, [_P, _P, _P, _I, _I, _I, _D, _P, _P, _P, _P, _P, _S, _P]),
        "moe_dispatch": (_I, [_P, _I, _I, _I, _P, _I, _I, _P, _P, _P, _P, _P, _P, _S, _P]),
        "moe_expert_ffn": (_I, [_P, _I, _P, _I, _P, _I, _I, _I, _I, _P, _P, _P, _P, _S, _P]),
        "moe_expert_ffn_packed": (_I, [_P, _I, _P, _I, _P, _I, _I, _I, _I, _P, _P, _P, _P, _S, _P]),
        "moe_expert_ffn_packed_gather": (_I, [_P, _I, _I, _I, _P, _P, _I, _P, _I, _I, _I, _P, _P, _P, _P,
                                              _S, _P]),
        "moe_pack_expert_weights": (_I, [_P, _I, _I, _I, _I, _P, _P]),
        "moe_combine": (_I, [_P, _I, _P, _P, _I, _I, _I, _P, _P]),
        "moe_combine_residual": (_I, [_P, _I, _P, _P, _I, _I, _I, _P, _P, _P]),
        "moe_permute_experts": (_I, [_P, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
        "drop_visual_block": (_I, [_P, _I, _I, _I, _I, _I, _P, _P]),
        "moe_savb_workspace_size": (_S, [_I, _I, _I]),
        "moe_savb_gate": (_I, [_P, _I, _I, _I, _P, _P, _I, _P, _P, _D, _P, _P, _P, _P, _S, _P]),
        "drop_visual_block_if": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P]),
        "moe_expand_dense_routing": (_I, [_P, _P, _I, _I, _I, _P, _P, _P, _P]),
        "moe_ffn_status": (_I, [_P, _S, _P, _P]),
        "moe_route_rcep": (_I, [_P, _I, _P, _P, _I, _I, _I, _I, _D, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                _P, _S, _P]),
        "moe_route_rcep_if": (_I, [_P, _I, _P, _P, _I, _I, _I, _I, _D, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                   _P, _P, _S, _P, _I, _I, _P]),
        "moe_rcep_layer": (_I, [_P, _I, _P, _P, _I, _I, _I, _I, _D, _P, _P, _I, _P, _P, _P, _P, _P, _P, _P,
                                _P, _P, _P, _P, _P, _P, _P, _P, _S, _P]),
        "moe_rcep_layer_chained": (_I, [_P, _P, _P, _P, _I, _P, _P, _I, _I, _I, _I, _D, _P, _P, _I, _P, _P,
                                        _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _S, _P]),
        "moe_dense_layer": (_I, [_P, _I, _P, _P, _I, _I, _I, _I, _P, _P, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                 _P, _P, _S, _P]),
        "moe_rcep_layer_if": (_I, [_P, _I, _P, _P, _I, _I, _I, _I, _D, _P, _P, _I, _P, _P, _P, _P, _P, _P,
                                   _P, _P, _P, _P, _P, _P, _P, _P, _P, _S, _P, _I, _I, _P]),
        "moe_route_packed_if": (_I, [_P, _I, _P, _P, _I, _I, _I, _I, _P, _I, _P, _P, _P, _P, _P, _S,
                                     _P, _I, _I, _P]),
        "moe_calibrate_route_prefix_if": (_I, [_P, _P, _P, _I, _I, _I, _D, _P, _P, _P, _P, _P, _S,
                                               _P, _I, _I, _P]),
        "moe_dispatch_if": (_I, [_P, _I, _I, _I, _P, _I, _I, _P, _P, _P, _P, _P, _P, _S, _P, _I, _I, _P]),
        "moe_expert_ffn_packed_gather_if": (_I, [_P, _I, _I, _I, _P, _P, _I, _P, _I, _I, _I, _P, _P, _P,
                                                 _P, _S, _P, _I, _I, _P]),
        "moe_combine_residual_if": (_I, [_P, _I, _P, _P, _I, _I, _I, _P, _P, _P, _I, _I, _P]),
        "moe_savb_gate_if": (_I, [_P, _I, _I, _I, _P, _P, _I, _P, _P, _D, _P, _P, _P, _P, _S, _P, _I, _I,
                                  _P, _I, _P]),
        "moe_expert_ffn_packed_gather_noalloc": (_I, [_P, _I, _I, _I, _P, _P, _I, _P, _I, _I, _I, _P, _P,
                                                      _P, _P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    _lib = lib
    return lib


def _status_text(status: int) -> str:
    try:
        return load().moe_status_string(status).decode()
    except Exception:
        return "?"


def _p(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("device arrays are passed as torch tensors")
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("arrays must be contiguous GPU tensors")
    return t.data_ptr()


def _typed(t, dtype):
    if t is not None and isinstance(t, torch.Tensor) and t.dtype != dtype:
        raise TypeError(f"expected a {dtype} tensor, got {t.dtype}")
    return _p(t)


def _i32(t):
    return _typed(t, torch.int32)


def _f32(t):
    return _typed(t, torch.float32)


def _f64(t):
    return _typed(t, torch.float64)


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def _dt(t) -> int:
    if t.dtype == torch.bfloat16:
        return MOE_BF16
    if t.dtype == torch.float32:
        return MOE_F32
    raise TypeError(f"unsupported activation dtype {t.dtype}")


def _check(fn: str, status: int):
    if status != 0:
        raise MoeError(fn, status)


def _nseg(seg_offsets):
    return 1 if seg_offsets is None else seg_offsets.numel() - 1


def moe_workspace_size(T: int, E: int, k: int, d: int, m: int, n_seg: int = 1) -> int:
    return int(load().moe_workspace_size(T, E, k, d, m, n_seg))


def _nbytes(ws):
    return ws.numel() * ws.element_size() if ws is not None else 0


def moe_route(x, w_r, bias, k, logits, topk_idx, topk_w, seg_offsets=None, K_dev=None, ws=None,
              stream=None):
    """x [T, d] or None (then `logits` [T, E] is an input)."""
    T, E = logits.shape
    d = x.shape[1] if x is not None else 0
    dt = _dt(x) if x is not None else MOE_F32
    _check("moe_route", load().moe_route(
        _p(x), dt, _f32(w_r) if x is not None else None, _f32(bias) if x is not None else None,
        T, d, E, k, _i32(seg_offsets), _nseg(seg_offsets), _i32(K_dev),
        _f32(logits), _i32(topk_idx), _f32(topk_w), _p(ws), _nbytes(ws), _stream(stream)))


def moe_route_packed(x, w_r_packed, bias, k, logits, topk_idx, topk_w, seg_offsets=None, K_dev=None,
                     ws=None, stream=None):
    """x [T, d] bf16; w_r_packed from moe_pack_router (d * E * 3 bf16)."""
    T, E = logits.shape
    d = x.shape[1]
    _check("moe_route_packed", load().moe_route_packed(
        _p(x), _dt(x), _p(w_r_packed), _f32(bias), T, d, E, k, _i32(seg_offsets), _nseg(seg_offsets),
        _i32(K_dev), _f32(logits), _i32(topk_idx), _f32(topk_w), _p(ws), _nbytes(ws), _stream(stream)))


def moe_pack_router(w_r, w_r_packed, stream=None):
    """w_r [d, E] float32 -> w_r_packed (3 d E bf16, any shape)."""
    d, E = w_r.shape
    if w_r_packed.numel() * w_r_packed.element_size() != 6 * d * E:
        raise ValueError("w_r_packed must hold 3 * d * E bf16 values")
    _check("moe_pack_router", load().moe_pack_router(_f32(w_r), d, E, _p(w_r_packed), _stream(stream)))


def moe_calibrate_prefix(topk_idx, topk_w, E, p, mass, ws, K_out=None, order=None,
                         seg_offsets=None, stream=None):
    T, k = topk_idx.shape
    _check("moe_calibrate_prefix", load().moe_calibrate_prefix(
        _i32(topk_idx), _f32(topk_w), T, E, k, _i32(seg_offsets), _nseg(seg_offsets), float(p),
        _f64(mass), _i32(K_out), _i32(order), _p(ws), _nbytes(ws), _stream(stream)))


def moe_calibrate_route_prefix(logits, idx_full, w_full, p, mass, K_out, idx, w, stream=None):
    """Eqs. 11-12 and the prefix re-route of one invocation in one call."""
    T, k = idx_full.shape
    E = logits.shape[1]
    _check("moe_calibrate_route_prefix", load().moe_calibrate_route_prefix(
        _f32(logits), _i32(idx_full), _f32(w_full), T, E, k, float(p), _f64(mass), _i32(K_out), _i32(idx), _f32(w),
        None, 0, _stream(stream)))


def moe_dispatch(topk_idx, E, x, counts, offsets, src_of_row, row_of_slot, x_perm, ws,
                 stream=None):
    T, k = topk_idx.shape
    d = x.shape[1] if x is not None else 0
    dt = _dt(x) if x is not None else MOE_F32
    _check("moe_dispatch", load().moe_dispatch(
        _i32(topk_idx), T, k, E, _p(x), dt, d, _i32(counts), _i32(offsets), _i32(src_of_row),
        _i32(row_of_slot), _p(x_perm), _p(ws), ws.numel() * ws.element_size() if ws is not None else 0,
        _stream(stream)))


def moe_expert_ffn(x_perm, offsets, w_gate_up, w_down, y_perm, ws, K_dev=None, stream=None):
    rows_max, d = x_perm.shape
    E, two_m, _ = w_gate_up.shape
    n_K = K_dev.numel() if K_dev is not None else 0
    _check("moe_expert_ffn", load().moe_expert_ffn(
        _p(x_perm), _dt(x_perm), _i32(offsets), E, _i32(K_dev), n_K, rows_max, d, two_m // 2,
        _p(w_gate_up), _p(w_down), _p(y_perm), _p(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def moe_expert_ffn_packed(x_perm, offsets, w_gate_up_packed, w_down_packed, y_perm, ws, K_dev=None,
                          stream=None):
    """Packed weights keep the shapes of the row-major tensors they came from."""
    rows_max, d = x_perm.shape
    E, two_m, _ = w_gate_up_packed.shape
    n_K = K_dev.numel() if K_dev is not None else 0
    _check("moe_expert_ffn_packed", load().moe_expert_ffn_packed(
        _p(x_perm), _dt(x_perm), _i32(offsets), E, _i32(K_dev), n_K, rows_max, d, two_m // 2,
        _p(w_gate_up_packed), _p(w_down_packed), _p(y_perm), _p(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def moe_expert_ffn_packed_gather(x, k, src_of_row, offsets, w_gate_up_packed, w_down_packed, y_perm,
                                 ws, K_dev=None, stream=None):
    """Token rows read from x through src_of_row (moe_dispatch with x=None)."""
    T, d = x.shape
    E, two_m, _ = w_gate_up_packed.shape
    n_K = K_dev.numel() if K_dev is not None else 0
    _check("moe_expert_ffn_packed_gather", load().moe_expert_ffn_packed_gather(
        _p(x), _dt(x), T, k, _i32(src_of_row), _i32(offsets), E, _i32(K_dev), n_K, d, two_m // 2,
        _p(w_gate_up_packed), _p(w_down_packed), _p(y_perm), _p(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def moe_expert_ffn_packed_gather_noalloc(x, k, src_of_row, offsets, w_gate_up_packed, w_down_packed,
                                         y_perm, K_dev=None, stream=None):
    """moe_expert_ffn_packed_gather on the library's own scratch array (no
    workspace; calls on one GPU must not overlap)."""
    T, d = x.shape
    E, two_m, _ = w_gate_up_packed.shape
    n_K = K_dev.numel() if K_dev is not None else 0
    _check("moe_expert_ffn_packed_gather_noalloc", load().moe_expert_ffn_packed_gather_noalloc(
        _p(x), _dt(x), T, k, _i32(src_of_row), _i32(offsets), E, _i32(K_dev), n_K, d, two_m // 2,
        _p(w_gate_up_packed), _p(w_down_packed), _p(y_perm), _stream(stream)))


def moe_pack_expert_weights(w, w_packed, stream=None):
    """w [E, rows, cols] -> w_packed (same shape and dtype, packed contents)."""
    E, rows, cols = w.shape
    if tuple(w_packed.shape) != (E, rows, cols) or w_packed.dtype != w.dtype:
        raise ValueError("w_packed must have the shape and dtype of w")
    _check("moe_pack_expert_weights", load().moe_pack_expert_weights(
        _p(w), _dt(w), E, rows, cols, _p(w_packed), _stream(stream)))


def moe_combine(y_perm, row_of_slot, topk_w, out, stream=None):
    T, k = topk_w.shape
    d = out.shape[1]
    _check("moe_combine", load().moe_combine(
        _p(y_perm), _dt(y_perm), _i32(row_of_slot), _f32(topk_w), T, k, d, _p(out), _stream(stream)))


def drop_visual_block(h, v0, v1, out, stream=None):
    S, d = h.shape
    _check("drop_visual_block", load().drop_visual_block(
        _p(h), _dt(h), S, d, v0, v1, _p(out), _stream(stream)))


def moe_combine_residual(y_perm, row_of_slot, topk_w, residual, out, stream=None):
    """out = residual + combine(...); `out` may be `residual` (in place)."""
    T, k = topk_w.shape
    d = out.shape[1]
    _check("moe_combine_residual", load().moe_combine_residual(
        _p(y_perm), _dt(y_perm), _i32(row_of_slot), _f32(topk_w), T, k, d, _p(residual), _p(out),
        _stream(stream)))


def moe_permute_experts(order, w_r=None, bias=None, w_gate_up=None, w_down=None, w_r_out=None,
                        bias_out=None, w_gate_up_out=None, w_down_out=None, d=None, m=None,
                        stream=None):
    """New expert j <- native expert order[j] (order: [E] int32 device
    tensor) for each given input/output pair."""
    E = order.numel()
    if w_r is not None:
        d = w_r.shape[0]
    if w_gate_up is not None:
        d, m = w_gate_up.shape[2], w_gate_up.shape[1] // 2
    elif w_down is not None:
        d, m = w_down.shape[1], w_down.shape[2]
    ref = w_gate_up if w_gate_up is not None else w_down
    dt = _dt(ref) if ref is not None else MOE_F32
    _check("moe_permute_experts", load().moe_permute_experts(
        _i32(order), E, d or 1, m or 1, dt, _f32(w_r), _f32(bias), _p(w_gate_up), _p(w_down),
        _f32(w_r_out), _f32(bias_out), _p(w_gate_up_out), _p(w_down_out), _stream(stream)))


def moe_savb_workspace_size(n: int, d: int, hid: int) -> int:
    return int(load().moe_savb_workspace_size(n, d, hid))


def moe_savb_gate(text_rows, w1, b1, w2, b2, theta, p_exit, exit_flag, ws, feature=None, stream=None):
    """text_rows [n, d] (bf16 or float32); w1 [hid, 2d]; w2 [2, hid]."""
    n, d = text_rows.shape
    hid = w1.shape[0]
    _check("moe_savb_gate", load().moe_savb_gate(
        _p(text_rows), _dt(text_rows), n, d, _f32(w1), _f32(b1), hid, _f32(w2), _f32(b2), float(theta),
        _f32(feature), _f32(p_exit), _i32(exit_flag), _p(ws), _nbytes(ws), _stream(stream)))


def drop_visual_block_if(h, v0, v1, exit_flag, out, stream=None):
    S, d = h.shape
    _check("drop_visual_block_if", load().drop_visual_block_if(
        _p(h), _dt(h), S, d, v0, v1, _i32(exit_flag), _p(out), _stream(stream)))


def moe_expand_dense_routing(topk_idx, topk_w, E, idx_dense, w_dense, K_dev=None, stream=None):
    T, k = topk_idx.shape
    _check("moe_expand_dense_routing", load().moe_expand_dense_routing(
        _i32(topk_idx), _f32(topk_w), T, k, E, _i32(K_dev), _i32(idx_dense), _f32(w_dense), _stream(stream)))


def moe_ffn_status(ws, status, stream=None):
    """status [4] int32 <- (waits that ran out, items completed, items
    planned, launch path) of the last expert FFN call on ws."""
    if status.numel() < 4:
        raise ValueError("status needs 4 int32 entries")
    _check("moe_ffn_status", load().moe_ffn_status(_p(ws), _nbytes(ws), _i32(status), _stream(stream)))


# --- predicated calls: the kernels run only while lo <= guard[0] < hi ------
def _guard(guard):
    """guard = (int32 device tensor, lo, hi) -> (pointer, lo, hi)."""
    if guard is None:
        return None, 0, 0
    g, lo, hi = guard
    return _i32(g), int(lo), int(hi)


def moe_route_packed_if(x, w_r_packed, bias, k, logits, topk_idx, topk_w, guard, seg_offsets=None,
                        K_dev=None, ws=None, stream=None):
    T, E = logits.shape
    d = x.shape[1]
    gp, lo, hi = _guard(guard)
    _check("moe_route_packed_if", load().moe_route_packed_if(
        _p(x), _dt(x), _p(w_r_packed), _f32(bias), T, d, E, k, _i32(seg_offsets), _nseg(seg_offsets),
        _i32(K_dev), _f32(logits), _i32(topk_idx), _f32(topk_w), _p(ws), _nbytes(ws), gp, lo, hi,
        _stream(stream)))


def moe_calibrate_route_prefix_if(logits, idx_full, w_full, p, mass, K_out, idx, w, guard, stream=None):
    T, k = idx_full.shape
    E = logits.shape[1]
    gp, lo, hi = _guard(guard)
    _check("moe_calibrate_route_prefix_if", load().moe_calibrate_route_prefix_if(
        _f32(logits), _i32(idx_full), _f32(w_full), T, E, k, float(p), _f64(mass), _i32(K_out), _i32(idx),
        _f32(w), None, 0, gp, lo, hi, _stream(stream)))


def moe_dispatch_if(topk_idx, E, x, counts, offsets, src_of_row, row_of_slot, x_perm, ws, guard,
                    stream=None):
    T, k = topk_idx.shape
    d = x.shape[1] if x is not None else 0
    dt = _dt(x) if x is not None else MOE_F32
    gp, lo, hi = _guard(guard)
    _check("moe_dispatch_if", load().moe_dispatch_if(
        _i32(topk_idx), T, k, E, _p(x), dt, d, _i32(counts), _i32(offsets), _i32(src_of_row),
        _i32(row_of_slot), _p(x_perm), _p(ws), _nbytes(ws), gp, lo, hi, _stream(stream)))


def moe_expert_ffn_packed_gather_if(x, k, src_of_row, offsets, w_gate_up_packed, w_down_packed, y_perm,
                                    ws, guard, K_dev=None, stream=None):
    T, d = x.shape
    E, two_m, _ = w_gate_up_packed.shape
    n_K = K_dev.numel() if K_dev is not None else 0
    gp, lo, hi = _guard(guard)
    _check("moe_expert_ffn_packed_gather_if", load().moe_expert_ffn_packed_gather_if(
        _p(x), _dt(x), T, k, _i32(src_of_row), _i32(offsets), E, _i32(K_dev), n_K, d, two_m // 2,
        _p(w_gate_up_packed), _p(w_down_packed), _p(y_perm), _p(ws), _nbytes(ws), gp, lo, hi,
        _stream(stream)))


def moe_combine_residual_if(y_perm, row_of_slot, topk_w, residual, out, guard, stream=None):
    T, k = topk_w.shape
    d = out.shape[1]
    gp, lo, hi = _guard(guard)
    _check("moe_combine_residual_if", load().moe_combine_residual_if(
        _p(y_perm), _dt(y_perm), _i32(row_of_slot), _f32(topk_w), T, k, d, _p(residual), _p(out), gp, lo,
        hi, _stream(stream)))


def moe_savb_gate_if(text_rows, w1, b1, w2, b2, theta, p_exit, exit_flag, ws, guard, exit_layer=None,
                     layer=0, feature=None, stream=None):
    """moe_savb_gate under the predicate; when it fires, exit_layer[0] = layer."""
    n, d = text_rows.shape
    hid = w1.shape[0]
    gp, lo, hi = _guard(guard)
    _check("moe_savb_gate_if", load().moe_savb_gate_if(
        _p(text_rows), _dt(text_rows), n, d, _f32(w1), _f32(b1), hid, _f32(w2), _f32(b2), float(theta),
        _f32(feature), _f32(p_exit), _i32(exit_flag), _p(ws), _nbytes(ws), gp, lo, hi, _i32(exit_layer),
        int(layer), _stream(stream)))


def moe_route_rcep(x, w_r_packed, bias, k, p, logits, idx_full, w_full, mass, K_out, idx, w, counts, offsets,
                   src_of_row, row_of_slot, ws, guard=None, stream=None):
    """The RCEP routing of one invocation through the dispatch grouping:
    moe_route_packed + moe_calibrate_route_prefix + moe_dispatch(x=None).
    With ``guard`` = (g, lo, hi) the predicated form (moe_route_rcep_if)."""
    T, d = x.shape
    E = logits.shape[1]
    args = (_p(x), _dt(x), _p(w_r_packed), _f32(bias), T, d, E, k, float(p), _f32(logits), _i32(idx_full),
            _f32(w_full), _f64(mass), _i32(K_out), _i32(idx), _f32(w), _i32(counts), _i32(offsets),
            _i32(src_of_row), _i32(row_of_slot), _p(ws), _nbytes(ws))
    if guard is None:
        _check("moe_route_rcep", load().moe_route_rcep(*args, _stream(stream)))
    else:
        gp, lo, hi = _guard(guard)
        _check("moe_route_rcep_if", load().moe_route_rcep_if(*args, gp, lo, hi, _stream(stream)))


def moe_rcep_layer(x, w_r_packed, bias, k, p, w_gate_up_packed, w_down_packed, residual, out, logits,
                   idx_full, w_full, mass, K_out, idx, w, counts, offsets, src_of_row, row_of_slot, y_perm, ws,
                   guard=None, stream=None):
    """One RCEP layer: moe_route_rcep + moe_expert_ffn_packed_gather (K_dev =
    K_out) + moe_combine_residual (residual = None: moe_combine).  `out` may
    be `residual` and/or `x`.
    With ``guard`` = (g, lo, hi) the predicated form (moe_rcep_layer_if)."""
    T, d = x.shape
    E, two_m, _ = w_gate_up_packed.shape
    args = (_p(x), _dt(x), _p(w_r_packed), _f32(bias), T, d, E, k, float(p), _p(w_gate_up_packed),
            _p(w_down_packed), two_m // 2, _p(residual), _p(out), _f32(logits), _i32(idx_full), _f32(w_full),
            _f64(mass), _i32(K_out), _i32(idx), _f32(w), _i32(counts), _i32(offsets), _i32(src_of_row),
            _i32(row_of_slot), _p(y_perm), _p(ws), _nbytes(ws))
    if guard is None:
        _check("moe_rcep_layer", load().moe_rcep_layer(*args, _stream(stream)))
    else:
        gp, lo, hi = _guard(guard)
        _check("moe_rcep_layer_if", load().moe_rcep_layer_if(*args, gp, lo, hi, _stream(stream)))


def moe_dense_layer(x, w_r_packed, bias, k, w_gate_up_packed, w_down_packed, residual, out, logits, idx, w,
                    counts, offsets, src_of_row, row_of_slot, y_perm, ws, stream=None):
    """One full-pool layer: moe_route_packed + moe_dispatch (x = None) +
    moe_expert_ffn_packed_gather + moe_combine_residual (residual = None:
    moe_combine).  `out` may be `residual` and/or `x`."""
    T, d = x.shape
    E, two_m, _ = w_gate_up_packed.shape
    _check("moe_dense_layer", load().moe_dense_layer(
        _p(x), _dt(x), _p(w_r_packed), _f32(bias), T, d, E, k, _p(w_gate_up_packed), _p(w_down_packed),
        two_m // 2, _p(residual), _p(out), _f32(logits), _i32(idx), _f32(w), _i32(counts), _i32(offsets),
        _i32(src_of_row), _i32(row_of_slot), _p(y_perm), _p(ws), _nbytes(ws), _stream(stream)))


def moe_rcep_layer_chained(prev, h, w_r_packed, bias, k, p, w_gate_up_packed, w_down_packed, logits, idx_full,
                           w_full, mass, K_out, idx, w, counts, offsets, src_of_row, row_of_slot, y_perm, ws,
                           stream=None):
    """The previous layer's combine with the residual (prev = (y_perm,
    row_of_slot, topk_w) of that layer, or None) into h, then this layer's
    RCEP routing and expert FFN over h; this layer's combine is left to the
    next chained call or to moe_combine_residual."""
    T, d = h.shape
    E, two_m, _ = w_gate_up_packed.shape
    py, pr, pw = prev if prev is not None else (None, None, None)
    _check("moe_rcep_layer_chained", load().moe_rcep_layer_chained(
        _p(py), _i32(pr), _f32(pw), _p(h), _dt(h), _p(w_r_packed), _f32(bias), T, d, E, k, float(p),
        _p(w_gate_up_packed), _p(w_down_packed), two_m // 2, _f32(logits), _i32(idx_full), _f32(w_full), _f64(mass),
        _i32(K_out), _i32(idx), _f32(w), _i32(counts), _i32(offsets), _i32(src_of_row), _i32(row_of_slot),
        _p(y_perm), _p(ws), _nbytes(ws), _stream(stream)))


def moe_rcep_layer_if(x, w_r_packed, bias, k, p, w_gate_up_packed, w_down_packed, residual, out, logits,
                      idx_full, w_full, mass, K_out, idx, w, counts, offsets, src_of_row, row_of_slot, y_perm, ws,
                      guard, stream=None):
    moe_rcep_layer(x, w_r_packed, bias, k, p, w_gate_up_packed, w_down_packed, residual, out, logits, idx_full,
                   w_full, mass, K_out, idx, w, counts, offsets, src_of_row, row_of_slot, y_perm, ws, guard=guard,
                   stream=stream)


def moe_route_rcep_if(x, w_r_packed, bias, k, p, logits, idx_full, w_full, mass, K_out, idx, w, counts,
                      offsets, src_of_row, row_of_slot, ws, guard, stream=None):
    moe_route_rcep(x, w_r_packed, bias, k, p, logits, idx_full, w_full, mass, K_out, idx, w, counts, offsets,
                   src_of_row, row_of_slot, ws, guard=guard, stream=stream)
