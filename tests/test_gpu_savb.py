"""SAVB gate (Sec. 3.2, Eqs. 2 and 3) on the GPU against the oracle.

The feature x (mean of the preceding text rows, then the final row) compares
within 1e-5 of its max (float32 sums over up to a few hundred rows); the exit
probability is compared teacher-forced (the oracle's MLP on the GPU's
feature, widened) within 1e-5, and the exit flag exactly unless p_exit lies
within 1e-5 of theta.  drop_visual_block_if is checked bitwise for both flag
values.
"""

import numpy as np
import pytest
import torch

import oracle
from _util import ensure_built

pytestmark = pytest.mark.gpu

from paper_2609_38823_amd import abi  # noqa: E402
from paper_2609_38823_amd import inputs as I  # noqa: E402

TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()
    torch.cuda.init()


def dev(a, dt=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t.to(dt) if dt is not None else t


def host(t):
    torch.cuda.synchronize()
    return (t.float() if t.dtype == torch.bfloat16 else t).cpu().numpy()


def run_gate(rows_np, dt, gp, theta):
    n, d = rows_np.shape
    hid = gp["w1"].shape[0]
    rows = dev(rows_np, TDT[dt])
    p = torch.full((1,), -1.0, device="cuda")
    flag = torch.full((4,), -7, dtype=torch.int32, device="cuda")
    feat = torch.empty((2 * d,), device="cuda")
    ws = torch.empty((abi.moe_savb_workspace_size(n, d, hid),), dtype=torch.uint8, device="cuda")
    abi.moe_savb_gate(rows, dev(gp["w1"]), dev(gp["b1"]), dev(gp["w2"]), dev(gp["b2"]), theta, p, flag[:1],
                      ws, feature=feat)
    return host(feat), float(host(p)[0]), int(host(flag)[0])


# n = 512 text rows of the Qwen3-VL layer; 600 rows (16 splits of 38); a
# single text row (zero mean); small odd shapes in float32
@pytest.mark.parametrize("n,d,dt", [(512, 2048, "bf16"), (600, 2048, "bf16"), (1, 256, "f32"),
                                    (2, 64, "f32"), (33, 8, "f32"), (4096, 128, "bf16")])
def test_savb_gate(n, d, dt):
    rows = I.tokens(I.LayerShape(d=d, E=16, m=16, k=2, dtype=dt), n, seed=n + d)
    gp = I.gate_params(d, seed=d)
    feat, p, flag = run_gate(rows, dt, gp, 0.5)
    x_ref = oracle.savb_gate_feature(rows)
    assert np.abs(feat - x_ref).max() <= 1e-5 * max(np.abs(x_ref).max(), 1e-30)
    # teacher-forced MLP on the GPU's feature: the oracle's Eq. 3 on x
    hidden = np.maximum(gp["w1"].astype(np.float64) @ feat.astype(np.float64) + gp["b1"], 0.0)
    z = gp["w2"].astype(np.float64) @ hidden + gp["b2"]
    p_ref = float(oracle.softmax(z[None, :])[0, 1])
    assert abs(p - p_ref) <= 1e-5
    if abs(p_ref - 0.5) > 1e-5:
        assert flag == int(p_ref >= 0.5)
    # thresholds on either side of the probability decide the flag
    assert run_gate(rows, dt, gp, p_ref - 1e-3)[2] == 1
    assert run_gate(rows, dt, gp, p_ref + 1e-3)[2] == 0
    # the free-running oracle agrees within the same tolerance
    p_free, _, _, _ = oracle.savb_gate(rows, gp["w1"], gp["b1"], gp["w2"], gp["b2"], 0.5)
    assert abs(p - p_free) <= 1e-4


def test_savb_gate_deterministic():
    rows = I.tokens(I.QWEN3_VL_MOE, 512, seed=3)
    gp = I.gate_params(2048, seed=1)
    a = run_gate(rows, "bf16", gp, 0.5)
    b = run_gate(rows, "bf16", gp, 0.5)
    np.testing.assert_array_equal(a[0], b[0])
    assert a[1:] == b[1:]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("S,d,v0,v1", [(8192, 2048, 0, 7680), (37, 24, 5, 17), (10, 6, 0, 10)])
def test_drop_visual_block_if(dt, S, d, v0, v1):
    h_np = I.synthetic_rows(S, d, dt, seed=S + d)
    h = dev(h_np, TDT[dt])
    rows_out = S - (v1 - v0)
    for fl in (0, 1, 5):
        flag = torch.tensor([fl], dtype=torch.int32, device="cuda")
        out = torch.full((max(rows_out, 1), d), 3.0, dtype=TDT[dt], device="cuda")
        abi.drop_visual_block_if(h, v0, v1, flag, out[:rows_out] if rows_out else out[:0])
        got = host(out)[:rows_out]
        if fl == 0:
            assert (got == 3.0).all()  # untouched
        else:
            np.testing.assert_array_equal(got, oracle.drop_visual_block(h_np, v0, v1))
