"""The paper's analytical decoder FLOPs accounting (App. A.3), as a report
beside the measured and algorithmic figures.

It counts what the paper's replay counts: per token the attention
projections, the router over all E experts and the retained experts under
the paper's dense-equivalent convention (every retained expert multiplies
every token: 6 K d m per token), plus the attention score and value
products, per layer; and the SAVB gate MLP per evaluation.  A
multiply-add is two FLOPs.  Nothing here runs on the device; the attention
terms are counted only (this library computes the MoE blocks).

Layer-index convention: ``exit_layer`` is the first text-only layer
(zero-based).  A trigger recorded after layer l* (the paper's one-based
sums run layers 1 .. l* + 1 on all S rows) is exit_layer = l* + 1.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Sequence


@dataclass(frozen=True)
class DecoderDims:
    """Sizes of the replay: d hidden, q attention output, kv the concatenated
    key/value projection, E experts, m expert width, h the gate's hidden
    width.  Defaults: the Qwen3-VL-MoE values the paper uses."""

    d: int = 2048
    q: int = 4096
    kv: int = 512
    E: int = 128
    m: int = 768
    h: int = 512


def c_proj(g: DecoderDims) -> int:
    """Linear projections per token (Eq. 13): 2 (d q + 2 d kv + q d)."""
    return 2 * (g.d * g.q + 2 * g.d * g.kv + g.q * g.d)


def c_router(g: DecoderDims) -> int:
    """Router over all E experts per token (Eq. 14): 2 d E."""
    return 2 * g.d * g.E


def c_expert(g: DecoderDims, K: int) -> int:
    """K retained experts per token, dense-equivalent (Eq. 15): 6 K d m
    (gate, up and down products)."""
    return 6 * int(K) * g.d * g.m


def prefill_layer(g: DecoderDims, S: int, K: int) -> int:
    """One decoder layer over a prefill of S rows (Eq. 16):
    S C_proj + 2 q S (S + 1) + S (C_router + C_expert(K))."""
    return S * c_proj(g) + 2 * g.q * S * (S + 1) + S * (c_router(g) + c_expert(g, K))


def decode_layer(g: DecoderDims, C: int, K: int) -> int:
    """One decoder layer of one decode forward with a KV cache of C entries
    (Eq. 17): C_proj + C_router + C_expert(K) + 4 q C."""
    return c_proj(g) + c_router(g) + c_expert(g, K) + 4 * g.q * C


def gate(g: DecoderDims, n_eval: int) -> int:
    """The SAVB gate MLP, 2d -> h -> 2, evaluated n_eval times (Eq. 20)."""
    return int(n_eval) * (2 * (2 * g.d) * g.h + 2 * g.h * 2)


def case_flops(g: DecoderDims, L: int, S: int, V: int, exit_layer: int | None,
               K_prefill: Sequence[int] = (), K_decode: Sequence[Sequence[int]] = (),
               n_gate: int = 0) -> dict:
    """One case (Eqs. 18-20): prefill of S rows of which V visual, and one
    decode forward per row of K_decode (K_decode[t][l]: the prefix length of
    layer l at step t; G - 1 steps for G generated tokens).

    DecoMoE: layers before exit_layer run (S, E) and the layers from it on
    (T, K_prefill[j]), T = S - V; decode step t (one-based) sees a KV cache
    of T + t - 1 entries.  exit_layer None: no trigger, every prefill layer
    at (S, E) and the cache keeps the visual rows.
    Baseline (READING: the same case without the method): every prefill
    layer at (S, E), decode at K = E with a cache of S + t - 1 entries.
    Returns the DecoMoE and baseline FLOPs and their parts.
    """
    T = S - V
    if exit_layer is None:
        pre = L * prefill_layer(g, S, g.E)
        C0 = S
    else:
        if len(K_prefill) != L - exit_layer:
            raise ValueError("K_prefill needs one prefix length per layer from the exit on")
        pre = exit_layer * prefill_layer(g, S, g.E) + sum(prefill_layer(g, T, K) for K in K_prefill)
        C0 = T
    dec = 0
    for t, Ks in enumerate(K_decode, start=1):
        if len(Ks) != L:
            raise ValueError("K_decode needs one prefix length per layer and step")
        dec += sum(decode_layer(g, C0 + t - 1, K) for K in Ks)
    base_pre = L * prefill_layer(g, S, g.E)
    base_dec = sum(L * decode_layer(g, S + t - 1, g.E) for t in range(1, len(K_decode) + 1))
    gt = gate(g, n_gate)
    return dict(method=pre + dec + gt, method_prefill=pre, method_decode=dec, method_gate=gt,
                baseline=base_pre + base_dec, baseline_prefill=base_pre, baseline_decode=base_dec)


def saving(cases: Sequence[dict]) -> float:
    """Total saving over matched cases (Eq. 21): 1 - sum F_method / sum
    F_baseline."""
    return 1.0 - sum(c["method"] for c in cases) / sum(c["baseline"] for c in cases)
