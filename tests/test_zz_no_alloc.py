"""The allocation-free expert FFN (GPU): moe_expert_ffn_packed_gather_noalloc
against moe_expert_ffn_packed_gather on the same inputs, bitwise, on two
calls in a row whose second is smaller (the library's scratch array keeps
the first call's contents; its counters must be cleared by the second)."""

import numpy as np
import pytest
import torch

from _util import ensure_built

pytestmark = pytest.mark.gpu

from paper_2609_38823_amd import abi  # noqa: E402
from paper_2609_38823_amd import inputs as I  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()
    torch.cuda.init()


def _case(T, E, k, d, m, seed, K=None):
    sh = I.LayerShape(d=d, E=E, m=m, k=k, dtype="bf16")
    prm = I.layer_params(sh, seed=seed)
    idx, _ = I.synthetic_routing(T, E, k, seed=seed + 1, K=K)
    x = torch.from_numpy(I.synthetic_rows(T, d, "bf16", seed=seed + 2)).cuda().to(torch.bfloat16)
    A = T * k
    i32 = lambda n: torch.empty((n,), dtype=torch.int32, device="cuda")  # noqa: E731
    counts, offsets, src, ros = i32(E), i32(E + 1), i32(A), i32(A)
    ws = torch.empty(abi.moe_workspace_size(T, E, k, d, m, 1), dtype=torch.uint8, device="cuda")
    abi.moe_dispatch(torch.from_numpy(idx).cuda(), E, None, counts, offsets, src, ros, None, ws)
    wgu = torch.from_numpy(prm["w_gate_up"]).cuda().to(torch.bfloat16)
    wd = torch.from_numpy(prm["w_down"]).cuda().to(torch.bfloat16)
    wgu_p, wd_p = torch.empty_like(wgu), torch.empty_like(wd)
    abi.moe_pack_expert_weights(wgu, wgu_p)
    abi.moe_pack_expert_weights(wd, wd_p)
    K_dev = torch.full((4,), K, dtype=torch.int32, device="cuda")[:1] if K is not None else None
    return dict(x=x, k=k, src=src, offsets=offsets, wgu=wgu_p, wd=wd_p, ws=ws, K_dev=K_dev, A=A, d=d)


def _both(c):
    y_ref = torch.full((c["A"], c["d"]), 7.0, dtype=torch.bfloat16, device="cuda")
    y = torch.full((c["A"], c["d"]), 7.0, dtype=torch.bfloat16, device="cuda")
    abi.moe_expert_ffn_packed_gather(c["x"], c["k"], c["src"], c["offsets"], c["wgu"], c["wd"], y_ref,
                                     c["ws"], K_dev=c["K_dev"])
    abi.moe_expert_ffn_packed_gather_noalloc(c["x"], c["k"], c["src"], c["offsets"], c["wgu"], c["wd"], y,
                                             K_dev=c["K_dev"])
    torch.cuda.synchronize()
    return y, y_ref


@pytest.mark.parametrize("big,small", [
    ((512, 128, 8, 2048, 768, 1, None), (64, 128, 8, 2048, 768, 2, None)),    # RCEP span, then decode
    ((512, 128, 8, 2048, 768, 3, 85), (37, 6, 3, 512, 256, 4, None)),         # a prefix K, then ragged
    ((2000, 32, 4, 512, 256, 5, None), (300, 4, 2, 512, 256, 6, 3)),
])
def test_noalloc_matches_workspace_entry_point(big, small):
    for spec in (big, small):
        T, E, k, d, m, seed, K = spec
        print(f"noalloc case T={T} E={E} k={k} d={d} m={m} K={K}", flush=True)
        y, y_ref = _both(_case(T, E, k, d, m, seed, K))
        assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16))
        if K is None:
            assert not (y.float() == 7.0).all(dim=1).any()  # every row written


def test_noalloc_rejects_oversized_calls():
    c = _case(4096, 128, 8, 2048, 768, 7)  # 32 768 rows: h alone is 48 MiB
    y = torch.empty((c["A"], c["d"]), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(abi.MoeError) as e:
        abi.moe_expert_ffn_packed_gather_noalloc(c["x"], c["k"], c["src"], c["offsets"], c["wgu"], c["wd"], y)
    assert e.value.status == -3
    # the library's scratch still serves a valid call afterwards
    y2, y2_ref = _both(_case(100, 16, 2, 512, 256, 8))
    assert torch.equal(y2.view(torch.int16), y2_ref.view(torch.int16))
    np.testing.assert_array_equal(y2.float().cpu().numpy(), y2_ref.float().cpu().numpy())
