"""The paper's FLOPs replay (App. A.3, Eqs. 13-21) against a case worked by
hand, CPU only.

Sizes: d = 2, q = 2, kv = 1, E = 4, m = 3, gate hidden h = 4; L = 3 layers;
S = 5 prefill rows of which V = 3 visual (T = 2); the exit at layer 1 (a
trigger after layer 0); prefix lengths K = 2, 3 in layers 1, 2; two decode
steps (G = 3 generated tokens) with K = (3, 2, 2) and (4, 3, 2); one gate
evaluation.

  C_proj = 2 (2*2 + 2*2*1 + 2*2) = 24,  C_router = 2*2*4 = 16,
  C_expert(K) = 6*K*2*3 = 36 K
  F_pre(S, K) = 24 S + 2*2*S(S+1) + S (16 + 36 K)
    F_pre(5, 4) = 120 + 120 + 80 + 720 = 1040
    F_pre(2, 2) = 48 + 24 + 32 + 144 = 248
    F_pre(2, 3) = 48 + 24 + 32 + 216 = 320
  prefill: DecoMoE 1040 + 248 + 320 = 1608, baseline 3 * 1040 = 3120
  F_dec(C, K) = 24 + 16 + 36 K + 4*2*C
    step 1 (C = 2): 164 + 128 + 128 = 420
    step 2 (C = 3): 208 + 172 + 136 = 516
    baseline (K = 4, C = 5 and 6): 3 * (224 + 232) = 1368
  gate: 2*(2*2)*4 + 2*4*2 = 48
  totals: DecoMoE 1608 + 936 + 48 = 2592, baseline 3120 + 1368 = 4488
  saving 1 - 2592 / 4488
"""

import pytest

from _util import ROOT  # noqa: F401  (puts the repository on sys.path)
from paper_2609_38823_amd import flops as F

G = F.DecoderDims(d=2, q=2, kv=1, E=4, m=3, h=4)


def test_components():
    assert F.c_proj(G) == 24
    assert F.c_router(G) == 16
    assert F.c_expert(G, 1) == 36 and F.c_expert(G, 3) == 108


def test_layer_costs():
    assert F.prefill_layer(G, 5, 4) == 1040
    assert F.prefill_layer(G, 2, 2) == 248
    assert F.prefill_layer(G, 2, 3) == 320
    assert F.decode_layer(G, 2, 3) == 164
    assert F.decode_layer(G, 3, 4) == 208
    assert F.decode_layer(G, 5, 4) == 224
    assert F.gate(G, 1) == 48 and F.gate(G, 0) == 0


def test_hand_worked_case():
    c = F.case_flops(G, L=3, S=5, V=3, exit_layer=1, K_prefill=[2, 3], K_decode=[[3, 2, 2], [4, 3, 2]],
                     n_gate=1)
    assert c["method_prefill"] == 1608 and c["baseline_prefill"] == 3120
    assert c["method_decode"] == 936 and c["baseline_decode"] == 1368
    assert c["method_gate"] == 48
    assert c["method"] == 2592 and c["baseline"] == 4488
    assert F.saving([c]) == pytest.approx(1 - 2592 / 4488, rel=1e-15)


def test_no_trigger_and_full_prefix_cost_the_baseline():
    c = F.case_flops(G, L=3, S=5, V=3, exit_layer=None, K_decode=[[4, 4, 4]] * 2)
    assert c["method"] == c["baseline"]
    # an exit at layer 0 with every prefix full still saves the visual rows
    c0 = F.case_flops(G, L=3, S=5, V=3, exit_layer=0, K_prefill=[4, 4, 4])
    assert c0["method"] == 3 * F.prefill_layer(G, 2, 4) < c0["baseline"]


def test_saving_sums_cases_before_dividing():
    a = F.case_flops(G, L=3, S=5, V=3, exit_layer=1, K_prefill=[2, 3])
    b = F.case_flops(G, L=3, S=5, V=0, exit_layer=None)
    assert F.saving([a, b]) == pytest.approx(1 - (a["method"] + b["method"]) / (a["baseline"] + b["baseline"]))


def test_shape_errors():
    with pytest.raises(ValueError):
        F.case_flops(G, L=3, S=5, V=3, exit_layer=1, K_prefill=[2])
    with pytest.raises(ValueError):
        F.case_flops(G, L=3, S=5, V=3, exit_layer=1, K_prefill=[2, 3], K_decode=[[1, 2]])


def test_qwen_dims_are_the_papers():
    g = F.DecoderDims()
    assert (g.d, g.q, g.kv, g.E, g.m, g.h) == (2048, 4096, 512, 128, 768, 512)
    # router over all 128 experts and one retained expert per token
    assert F.c_router(g) == 524288 and F.c_expert(g, 1) == 6 * 2048 * 768
