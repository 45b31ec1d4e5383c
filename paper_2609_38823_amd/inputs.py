"""Seeded synthetic inputs for the RCEP MoE layer.

This module only draws random numbers and rounds them to the storage
precision; it contains none of the method's arithmetic.  Both the HIP path
(through the tests and the bench) and the CPU oracle consume the arrays it
returns, so the two sides always see identical inputs.

Workload recipe (stand-in for the paper's benchmarks, which are not
available; see the design notes):
  * token rows x ~ N(0, 1); router weights W_r [d, E] and expert weights
    ~ N(0, 0.02^2), drawn in float32;
  * bf16 workloads round x and the expert weights to bf16 (round to nearest
    even); the router weights and bias stay float32;
  * skewed router bias: b[sigma(r)] = alpha * ln(r^-s / sum_r' r'^-s) for
    rank r = 1..E, sigma a seeded permutation (Zipf with exponent s);
  * visual rows come first, then text rows (a contiguous visual block).

Every stream comes from ``numpy.random.SeedSequence(seed, spawn_key=...)``
with a fixed key per role, so any array can be regenerated independently.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

# stream roles (first element of the spawn key)
_S_TOKENS, _S_PARAMS, _S_CALIB, _S_DECODE, _S_GATE = 0, 1, 2, 3, 4
# parameter sub-streams
_P_WR, _P_BIAS, _P_GU, _P_DOWN = 0, 1, 2, 3


@dataclass(frozen=True)
class LayerShape:
    """Shape and storage type of one MoE layer."""

    d: int
    E: int
    m: int
    k: int
    dtype: str  # "f32" or "bf16": token rows and expert weights
    zipf_alpha: float | None = None  # None: no router bias
    zipf_s: float = 1.1
    w_std: float = 0.02


@dataclass(frozen=True)
class Workload:
    """A named workload: layer shape, token counts and RCEP settings."""

    name: str
    shape: LayerShape
    T: int  # token rows of the invocation
    n_visual: int  # rows [0, n_visual) are the visual block
    p: float  # routed-mass fraction for the prefix
    layers: int = 1
    exit_layer: int | None = None  # first text-only layer of a stack
    seed: int = 0
    notes: dict = field(default_factory=dict)


QWEN3_VL_MOE = LayerShape(d=2048, E=128, m=768, k=8, dtype="bf16", zipf_alpha=0.35)
TINY = LayerShape(d=256, E=16, m=128, k=2, dtype="f32", zipf_alpha=None)
# the smallest shape the packed bf16 path takes (d, m multiples of 256, E of 32)
SMALL_BF16 = LayerShape(d=256, E=32, m=256, k=4, dtype="bf16", zipf_alpha=0.35)

WORKLOADS = {
    # tiny fp32 correctness layer: 384 visual + 128 text rows
    "tiny_f32": Workload("tiny_f32", TINY, T=512, n_visual=384, p=0.9),
    # Qwen3-VL-MoE-shaped layer over a 3584-visual + 512-text prefill (dense span)
    "qwen3vl_dense_4096": Workload("qwen3vl_dense_4096", QWEN3_VL_MOE, T=4096, n_visual=3584, p=0.9),
    # the same layer after the visual exit: 512 text rows (RCEP span)
    "qwen3vl_rcep_512": Workload("qwen3vl_rcep_512", QWEN3_VL_MOE, T=512, n_visual=0, p=0.9),
    # 48-layer stack over 7680 visual + 512 text rows, exit at layer 20
    "qwen3vl_stack48_8192": Workload("qwen3vl_stack48_8192", QWEN3_VL_MOE, T=8192, n_visual=7680,
                                     p=0.9, layers=48, exit_layer=20),
    # tiny fp32 stack: 6 layers over 384 visual + 128 text rows, exit at layer 3
    "tiny_stack_f32": Workload("tiny_stack_f32", TINY, T=512, n_visual=384, p=0.9, layers=6,
                               exit_layer=3),
    # small packed bf16 stack: 8 layers over 384 visual + 128 text rows, exit at layer 4
    "small_stack_bf16": Workload("small_stack_bf16", SMALL_BF16, T=512, n_visual=384, p=0.9, layers=8,
                                 exit_layer=4),
    # decode: 64 single text tokens through 48 layers
    "qwen3vl_decode64": Workload("qwen3vl_decode64", QWEN3_VL_MOE, T=64, n_visual=0, p=0.85,
                                 layers=48),
}


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=key)))


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); the result is
    float32 holding bf16-representable values (finite inputs only)."""
    a = np.ascontiguousarray(a, np.float32)
    bits = a.view(np.uint32)
    lsb = (bits >> np.uint32(16)) & np.uint32(1)
    r = (bits + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of float32 values that are bf16-representable."""
    a = np.ascontiguousarray(a, np.float32)
    return (a.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    out = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)
    return out


def _store(a: np.ndarray, dtype: str) -> np.ndarray:
    return round_to_bf16(a) if dtype == "bf16" else np.ascontiguousarray(a, np.float32)


def zipf_bias(E: int, s: float, alpha: float, rng: np.random.Generator) -> np.ndarray:
    """b[sigma(r)] = alpha * ln(pmf(r)), pmf(r) = r^-s / sum_r' r'^-s."""
    r = np.arange(1, E + 1, dtype=np.float64)
    pmf = r ** (-s)
    pmf /= pmf.sum()
    sigma = rng.permutation(E)
    b = np.empty(E, np.float64)
    b[sigma] = alpha * np.log(pmf)
    return b.astype(np.float32)


def layer_params(shape: LayerShape, seed: int = 0, layer: int = 0) -> dict:
    """Router and expert weights of one layer in native (unreordered) order.

    Returns float32 arrays: w_r [d, E], bias [E] or None, w_gate_up [E, 2m, d]
    (rows [0, m) gate, [m, 2m) up) and w_down [E, d, m]; for bf16 layers the
    expert weights hold bf16-representable values.
    """
    d, E, m = shape.d, shape.E, shape.m
    w_r = _normal(_rng(seed, _S_PARAMS, layer, _P_WR), (d, E), shape.w_std)
    bias = None
    if shape.zipf_alpha is not None:
        bias = zipf_bias(E, shape.zipf_s, shape.zipf_alpha, _rng(seed, _S_PARAMS, layer, _P_BIAS))
    w_gate_up = np.empty((E, 2 * m, d), np.float32)
    w_down = np.empty((E, d, m), np.float32)

    def fill(e):  # one independent stream per expert and tensor
        w_gate_up[e] = _store(_normal(_rng(seed, _S_PARAMS, layer, _P_GU, e), (2 * m, d), shape.w_std),
                              shape.dtype)
        w_down[e] = _store(_normal(_rng(seed, _S_PARAMS, layer, _P_DOWN, e), (d, m), shape.w_std),
                           shape.dtype)

    workers = max(1, min(16, len(os.sched_getaffinity(0))))
    with ThreadPoolExecutor(max_workers=workers) as ex:
        list(ex.map(fill, range(E)))
    return dict(w_r=w_r, bias=bias, w_gate_up=w_gate_up, w_down=w_down)


def device_expert_weights(shape: LayerShape, seed: int = 0, layer: int = 0, device="cuda"):
    """Expert weights of one layer of a deep stack, drawn on the device.

    A 48-layer stack holds 48 * E * 3 * d * m values (29 G at the
    Qwen3-VL-MoE shape), too many to draw on the host in the time of a test,
    so stacks draw them with torch's device generator: N(0, w_std^2) in
    float32 from a generator seeded per (seed, layer, tensor), then rounded
    to the storage precision (round to nearest even for bf16).  Returns
    (w_gate_up [E, 2m, d], w_down [E, d, m]) torch tensors in native expert
    order.  Checks on the CPU copy the same tensors to the host.
    """
    import torch

    dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    out = []
    for tensor, shp in ((_P_GU, (shape.E, 2 * shape.m, shape.d)), (_P_DOWN, (shape.E, shape.d, shape.m))):
        g = torch.Generator(device=device)
        g.manual_seed(int(np.random.SeedSequence(seed, spawn_key=(_S_PARAMS, layer, tensor, 7))
                          .generate_state(1, np.uint64)[0] >> np.uint64(1)))
        w = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
        w.mul_(shape.w_std)
        out.append(w.to(dt) if dt != torch.float32 else w)
        del w
    return tuple(out)


def gate_params(d: int, hid: int = 512, seed: int = 0, layer: int = 0, std: float = 0.02) -> dict:
    """Random SAVB gate weights of one candidate layer: the two-class MLP
    2d -> hid -> 2 with w1 [hid, 2d], b1 [hid], w2 [2, hid], b2 [2], all
    N(0, std^2) in float32."""
    rng = _rng(seed, _S_GATE, layer)
    return dict(w1=_normal(rng, (hid, 2 * d), std), b1=_normal(rng, (hid,), std),
                w2=_normal(rng, (2, hid), std), b2=_normal(rng, (2,), std))


def router_params(shape: LayerShape, seed: int = 0, layer: int = 0) -> dict:
    """Only the router weights and bias of a layer (same streams as
    ``layer_params``), for tests that need no expert weights."""
    w_r = _normal(_rng(seed, _S_PARAMS, layer, _P_WR), (shape.d, shape.E), shape.w_std)
    bias = None
    if shape.zipf_alpha is not None:
        bias = zipf_bias(shape.E, shape.zipf_s, shape.zipf_alpha,
                         _rng(seed, _S_PARAMS, layer, _P_BIAS))
    return dict(w_r=w_r, bias=bias)


def tokens(shape: LayerShape, T: int, seed: int = 0, stream: str = "prefill", layer: int = 0) -> np.ndarray:
    """T token rows ~ N(0, 1) in the layer's storage precision.

    ``stream`` selects independent draws: "prefill" (the invocation's rows),
    "calib" (per-layer calibration rows) or "decode".
    """
    role = {"prefill": _S_TOKENS, "calib": _S_CALIB, "decode": _S_DECODE}[stream]
    key = (role, layer) if stream == "calib" else (role,)
    return _store(_normal(_rng(seed, *key), (T, shape.d), 1.0), shape.dtype)


def logits_with_ties(T: int, E: int, seed: int = 0, levels: int = 4) -> np.ndarray:
    """Router-logit-shaped float32 test input drawn from a few discrete
    levels, so that exact ties between experts are common."""
    rng = _rng(seed, 9, T, E)
    return (rng.integers(0, levels, size=(T, E)).astype(np.float32) * np.float32(0.5))


# --------------------------------------------------------------------------
# Stage-level inputs: arrays shaped like the intermediate results of the
# layer, drawn directly, so that each stage can be fed identical inputs on
# both sides.
# --------------------------------------------------------------------------
def zipf_probs(E: int, s: float, rng: np.random.Generator) -> np.ndarray:
    """Zipf(s) popularity over E experts in a seeded random order."""
    r = np.arange(1, E + 1, dtype=np.float64) ** (-s)
    pr = np.empty(E)
    pr[rng.permutation(E)] = r / r.sum()
    return pr


def synthetic_routing(T: int, E: int, k: int, seed: int = 0, zipf_s: float = 1.1,
                      K: int | None = None):
    """Routing-shaped arrays: idx [T, k] int32 with k distinct experts per
    token drawn without replacement from [0, K) (K = E by default) with
    Zipf-skewed popularity, and weights w [T, k] float32 in (0, 1]."""
    K = E if K is None else K
    rng = _rng(seed, 10, T, E, k, K)
    pr = zipf_probs(K, zipf_s, rng)
    # sampling without replacement: the k largest of log(p) + Gumbel noise
    keys = np.log(pr)[None, :] + rng.gumbel(size=(T, K))
    idx = np.argsort(-keys, axis=1, kind="stable")[:, :k].astype(np.int32)
    w = (1.0 - rng.random((T, k), dtype=np.float32)).astype(np.float32)
    return idx, w


def synthetic_counts(E: int, rows: int, seed: int = 0, zipf_s: float = 1.1, K: int | None = None):
    """Rows per expert: a multinomial draw of `rows` rows over experts [0, K)
    with Zipf-skewed probabilities (experts >= K get none)."""
    K = E if K is None else K
    rng = _rng(seed, 11, E, rows, K)
    counts = np.zeros(E, np.int64)
    counts[:K] = rng.multinomial(rows, zipf_probs(K, zipf_s, rng))
    return counts


def synthetic_rows(n: int, d: int, dtype: str, seed: int = 0, std: float = 1.0) -> np.ndarray:
    """n rows ~ N(0, std^2) in the storage precision."""
    return _store(_normal(_rng(seed, 12, n, d), (n, d), std), dtype)


def synthetic_permutation(n: int, seed: int = 0) -> np.ndarray:
    return _rng(seed, 13, n).permutation(n).astype(np.int32)
