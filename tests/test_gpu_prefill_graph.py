"""Algorithm 2's prefill as one captured HIP graph (GPU): the SAVB gate
decides the exit layer on the device and predicated calls pick each
layer's variant, so one graph serves every exit.

A small packed bf16 stack (8 layers, d 256, 32 experts x 256, top-4, 384
visual + 128 text rows) with gates at candidate layers 1, 3, 5, 7.  The
gate biases are rewritten in place between replays so that the exit falls
at each candidate in turn, and then at none; every replay is compared bit
for bit with the eager forward_gated (host-read flag per candidate) on the
same gates: final rows, exit layer, the evaluated p_exit values and the
prefix lengths of the RCEP layers.  Eager work and host synchronisations run
between the replays.
"""

import numpy as np
import pytest
import torch

from _util import ensure_built

pytestmark = pytest.mark.gpu

from paper_2609_38823_amd import inputs as I  # noqa: E402
from paper_2609_38823_amd.stack import MoEStack  # noqa: E402

CANDS = (1, 3, 5, 7)


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()
    torch.cuda.init()


@pytest.fixture(scope="module")
def stack():
    return MoEStack(I.WORKLOADS["small_stack_bf16"])


def host(t):
    torch.cuda.synchronize()
    return t.float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()


def set_exit(gates, target):
    """Gate biases that make candidate `target` the first to fire (None: no
    gate fires): class 1 (exit) strongly favoured there, class 0 elsewhere."""
    for l in CANDS:
        hi = 20.0 if l == target else -20.0
        gates[l]["b2"].copy_(torch.tensor([-hi, hi], dtype=torch.float32))


def test_captured_prefill_matches_eager_gated_prefill(stack):
    wl = stack.wl
    sh = wl.shape
    x = torch.from_numpy(I.tokens(sh, wl.T, seed=wl.seed)).cuda().to(torch.bfloat16)
    gates = {l: {k: torch.from_numpy(v).cuda() for k, v in I.gate_params(sh.d, seed=wl.seed, layer=l,
                                                                          std=0.05).items()}
             for l in CANDS}
    theta = 0.5
    set_exit(gates, None)
    pg = stack.capture_prefill(x, wl.n_visual, wl.p, gates, theta)
    other = torch.from_numpy(I.tokens(sh, wl.T, seed=wl.seed + 7)).cuda().to(torch.bfloat16)
    for rep, target in enumerate([3, None, 1, 5, 7, 3]):
        set_exit(gates, target)
        print(f"replay {rep}: exit at candidate {target}", flush=True)
        out_e, ex_e, trace_e = stack.forward_gated(x, wl.n_visual, wl.p, gates, theta)
        eager = host(out_e).copy()
        K_e = host(stack.K_trace)[:, 0].copy()
        assert ex_e == target
        stack.K_trace.fill_(-1)
        pg.replay()
        out_g, ex_g, trace_g = pg.result()
        assert ex_g == ex_e
        assert [l for l, _ in trace_g] == [l for l, _ in trace_e]
        assert [pv for _, pv in trace_g] == [pv for _, pv in trace_e]  # same kernels: equal floats
        assert out_g.shape == out_e.shape
        np.testing.assert_array_equal(host(out_g), eager)
        if ex_e is not None:
            np.testing.assert_array_equal(host(stack.K_trace)[ex_e:, 0], K_e[ex_e:])
            assert ((K_e[ex_e:] >= sh.k) & (K_e[ex_e:] <= sh.E)).all()
        # eager work on other rows between replays
        stack.forward(other, wl.n_visual, wl.p, wl.exit_layer)
        torch.cuda.synchronize()


def test_captured_prefill_needs_packed_layers():
    st = MoEStack(I.WORKLOADS["tiny_stack_f32"])
    x = torch.zeros((st.wl.T, st.sh.d), dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError):
        st.capture_prefill(x, st.wl.n_visual, st.wl.p, {}, 0.5)


def test_predicated_calls_run_or_leave_outputs(stack):
    """Each *_if call with the predicate in range gives bitwise the plain
    call's outputs; out of range it writes nothing (sentinels survive)."""
    from paper_2609_38823_amd import abi
    from paper_2609_38823_amd.layer import Buffers
    wl = stack.wl
    sh = wl.shape
    lay = stack.layers[2]
    T = 128
    x = torch.from_numpy(I.tokens(sh, T, seed=11)).cuda().to(torch.bfloat16)
    g = torch.full((4,), 5, dtype=torch.int32, device="cuda")[:1]

    def fresh():
        b = Buffers(T, sh.d, sh.E, sh.m, sh.k, torch.bfloat16, x_perm=False)
        for t in (b.logits, b.idx_full, b.w_full, b.mass, b.K, b.idx, b.w, b.counts, b.offsets, b.src_of_row,
                  b.row_of_slot, b.y_perm):
            t.fill_(-3)
        return b

    ref, res_ref = fresh(), x.clone()
    lay.forward_rcep(x, wl.p, b=ref, residual=x, out=res_ref)
    names = ["logits", "idx_full", "w_full", "mass", "K", "idx", "w", "counts", "offsets", "src_of_row",
             "row_of_slot", "y_perm"]
    # in range: bitwise the plain calls
    run, res_run = fresh(), x.clone()
    lay.forward_rcep(x, wl.p, b=run, residual=x, out=res_run, guard=(g, 5, 6))
    for n in names:
        assert torch.equal(getattr(run, n).view(torch.uint8), getattr(ref, n).view(torch.uint8)), n
    assert torch.equal(res_run.view(torch.int16), res_ref.view(torch.int16))
    # out of range (below and above): nothing written
    for lo, hi in ((6, 9), (0, 5), (5, 5)):
        skip, res_skip = fresh(), x.clone()
        lay.forward_rcep(x, wl.p, b=skip, residual=x, out=res_skip, guard=(g, lo, hi))
        for n in names:
            t = getattr(skip, n)
            assert torch.equal(t, torch.full_like(t, -3)), (n, lo, hi)
        assert torch.equal(res_skip.view(torch.int16), x.view(torch.int16))
    # the gate: skipped leaves p_exit, the flag and exit_layer; run writes them
    gp = {k: torch.from_numpy(v).cuda() for k, v in I.gate_params(sh.d, seed=1, layer=1).items()}
    gp["b2"].copy_(torch.tensor([-20.0, 20.0]))
    ws = torch.empty((abi.moe_savb_workspace_size(T, sh.d, gp["w1"].shape[0]),), dtype=torch.uint8,
                     device="cuda")
    pe = torch.full((4,), -1.0, device="cuda")[:1]
    fl = torch.full((4,), -1, dtype=torch.int32, device="cuda")[:1]
    el = torch.full((4,), 8, dtype=torch.int32, device="cuda")[:1]
    abi.moe_savb_gate_if(x, gp["w1"], gp["b1"], gp["w2"], gp["b2"], 0.5, pe, fl, ws, (el, 0, 8), exit_layer=el,
                         layer=3)
    assert float(pe.item()) == -1.0 and int(fl.item()) == -1 and int(el.item()) == 8
    abi.moe_savb_gate_if(x, gp["w1"], gp["b1"], gp["w2"], gp["b2"], 0.5, pe, fl, ws, (el, 8, 9), exit_layer=el,
                         layer=3)
    assert float(pe.item()) > 0.5 and int(fl.item()) == 1 and int(el.item()) == 3
    # once set, a later candidate's gate (same predicate) is skipped
    abi.moe_savb_gate_if(x, gp["w1"], gp["b1"], gp["w2"], gp["b2"], 0.5, pe, fl, ws, (el, 8, 9), exit_layer=el,
                         layer=5)
    assert int(el.item()) == 3
