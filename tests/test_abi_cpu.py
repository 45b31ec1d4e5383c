"""C-ABI contract checks that need no GPU: the library loads, exports every
function that include/decomoe.h declares, and rejects invalid arguments on
the host before anything is launched (only rejected calls are made here)."""

import ctypes
import os
import re

import pytest

from _util import ROOT, ensure_built

HEADER = os.path.join(ROOT, "include", "decomoe.h")
EINVAL, EALIAS, EWORKSPACE, EUNSUPPORTED = -1, -2, -3, -5
F32, BF16 = 0, 1


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^[A-Za-z_][\w\s\*]*?\b([a-z_][a-z0-9_]*)\s*\(", src, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "while", "for")))


@pytest.fixture(scope="module")
def lib():
    return ensure_built()


def test_header_declares_the_boundary():
    assert declared_functions() == sorted([
        "drop_visual_block", "moe_calibrate_prefix", "moe_combine", "moe_combine_residual",
        "moe_dispatch", "moe_expert_ffn", "moe_expert_ffn_packed", "moe_pack_expert_weights",
        "moe_pack_router", "moe_permute_experts", "moe_route", "moe_route_packed", "moe_savb_gate",
        "moe_savb_workspace_size", "moe_status_string", "moe_workspace_size", "drop_visual_block_if",
        "moe_expand_dense_routing", "moe_expert_ffn_packed_gather", "moe_calibrate_route_prefix",
        "moe_ffn_status", "moe_expert_ffn_packed_gather_noalloc",
        "moe_route_packed_if", "moe_calibrate_route_prefix_if", "moe_dispatch_if",
        "moe_expert_ffn_packed_gather_if", "moe_combine_residual_if", "moe_savb_gate_if",
        "moe_route_rcep", "moe_route_rcep_if", "moe_rcep_layer", "moe_rcep_layer_if",
        "moe_rcep_layer_chained", "moe_dense_layer"])


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_exports_are_exactly_the_declared_functions(lib):
    """No helper leaks out of the library as a C symbol (read with nm)."""
    import shutil
    import subprocess
    from paper_2609_38823_amd import abi
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    out = subprocess.run([nm, "-D", "--defined-only", abi.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    c_syms = sorted({ln.split()[-1] for ln in out.splitlines()
                     if " T " in ln and not ln.split()[-1].startswith("_Z")})
    assert c_syms == declared_functions()


def test_binding_names_match_header():
    from paper_2609_38823_amd import abi
    assert sorted(abi.EXPORTS) == declared_functions()
    for name in declared_functions():
        if name != "moe_status_string":
            assert callable(getattr(abi, name))


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4, -5, 7):
        assert lib.moe_status_string(code)


def test_workspace_size(lib):
    assert lib.moe_workspace_size(4096, 128, 8, 2048, 768, 1) > 4096 * 8 * 768 * 2
    assert lib.moe_workspace_size(0, 128, 8, 2048, 768, 1) >= 256
    assert lib.moe_workspace_size(16, 128, 0, 2048, 768, 1) == 0  # k < 1
    assert lib.moe_workspace_size(16, 2000, 8, 2048, 768, 1) == 0  # E > 1024
    assert lib.moe_workspace_size(2**28, 128, 8, 2048, 768, 1) == 0  # T * k above INT32_MAX
    assert lib.moe_workspace_size(2**28 - 1, 128, 7, 2048, 768, 1) > 0


# fake, never dereferenced, 16-byte aligned addresses
P1, P2, P3, P4, P5, P6, P7 = (ctypes.c_void_p(0x10000 * i) for i in range(1, 8))
WS = ctypes.c_void_p(0x40000000)
NULL = None


def test_route_rejects(lib):
    # k > E, E > 1024, k > 32
    assert lib.moe_route(P1, BF16, P2, NULL, 8, 64, 4, 5, NULL, 1, NULL, P3, P4, P5, NULL, 0, NULL) == EINVAL
    assert lib.moe_route(P1, BF16, P2, NULL, 8, 64, 2000, 5, NULL, 1, NULL, P3, P4, P5, NULL, 0, NULL) == EINVAL
    assert lib.moe_route(P1, BF16, P2, NULL, 8, 64, 128, 33, NULL, 1, NULL, P3, P4, P5, NULL, 0, NULL) == EUNSUPPORTED
    # bf16 rows need d % 8 == 0; logits must be given; misaligned pointer
    assert lib.moe_route(P1, BF16, P2, NULL, 8, 60, 128, 8, NULL, 1, NULL, P3, P4, P5, NULL, 0, NULL) == EINVAL
    assert lib.moe_route(P1, BF16, P2, NULL, 8, 64, 128, 8, NULL, 1, NULL, NULL, P4, P5, NULL, 0, NULL) == EINVAL
    assert lib.moe_route(ctypes.c_void_p(0x10002), BF16, P2, NULL, 8, 64, 128, 8, NULL, 1, NULL,
                         P3, P4, P5, NULL, 0, NULL) == EINVAL
    # outputs overlapping inputs: logits on top of x
    assert lib.moe_route(P1, BF16, P2, NULL, 8, 64, 128, 8, NULL, 1, NULL, P1, P4, P5, NULL, 0, NULL) == EALIAS
    # logits-input mode: topk_w overlapping logits
    assert lib.moe_route(NULL, F32, NULL, NULL, 8, 0, 128, 8, NULL, 1, NULL, P3, P4, P3, NULL, 0, NULL) == EALIAS
    # T == 0 launches nothing
    assert lib.moe_route(P1, BF16, P2, NULL, 0, 64, 128, 8, NULL, 1, NULL, P3, P4, P5, NULL, 0, NULL) == 0


def test_route_and_calibrate_need_workspace(lib):
    # few tokens and d % 128 == 0: the router splits d and needs ws
    assert lib.moe_route(P1, BF16, P2, NULL, 8, 2048, 128, 8, NULL, 1, NULL, P3, P4, P5, NULL, 0,
                         NULL) == EWORKSPACE
    assert lib.moe_route(P1, BF16, P2, NULL, 8, 2048, 128, 8, NULL, 1, NULL, P3, P4, P5, WS, 64,
                         NULL) == EWORKSPACE
    assert lib.moe_route(P1, BF16, P2, NULL, 8, 2048, 128, 8, NULL, 1, NULL, P3, P4, P5, P2, 1 << 30,
                         NULL) == EALIAS  # ws over w_r
    assert lib.moe_calibrate_prefix(P1, P2, 8, 16, 2, NULL, 1, 0.9, P3, P1, NULL, NULL, 0,
                                    NULL) == EALIAS  # K_out over topk_idx; no scratch needed
    assert lib.moe_calibrate_prefix(P1, P2, 8, 16, 40, NULL, 1, 0.9, P3, P4, NULL, WS, 1 << 30,
                                    NULL) == EINVAL  # k > E
    assert lib.moe_calibrate_prefix(P1, P2, 8, 64, 40, NULL, 1, 0.9, P3, P4, NULL, WS, 1 << 30,
                                    NULL) == EUNSUPPORTED  # k > 32


def test_calibrate_rejects(lib):
    for p in (0.0, -1.0, 1.5, float("nan")):
        assert lib.moe_calibrate_prefix(P1, P2, 8, 16, 2, NULL, 1, p, P3, P4, NULL, WS, 1 << 30, NULL) == EINVAL
    assert lib.moe_calibrate_prefix(P1, P2, 8, 16, 20, NULL, 1, 0.9, P3, P4, NULL, WS, 1 << 30, NULL) == EINVAL
    assert lib.moe_calibrate_prefix(P1, P2, 8, 16, 2, P5, 0, 0.9, P3, P4, NULL, WS, 1 << 30, NULL) == EINVAL
    assert lib.moe_calibrate_prefix(P1, P2, 8, 16, 2, NULL, 1, 0.9, P1, P4, NULL, WS, 1 << 30, NULL) == EALIAS


def test_calibrate_route_prefix_rejects(lib):
    f = lib.moe_calibrate_route_prefix
    # (logits, idx_full, w_full, T, E, k, p, mass, K_out, idx, w, ws, ws_bytes, s)
    assert f(P1, P2, P3, 8, 16, 2, 0.0, P4, P5, P6, P7, NULL, 0, NULL) == EINVAL   # p outside (0, 1]
    assert f(P1, P2, P3, 8, 16, 2, 1.5, P4, P5, P6, P7, NULL, 0, NULL) == EINVAL
    assert f(P1, P2, P3, 8, 16, 17, 0.9, P4, P5, P6, P7, NULL, 0, NULL) == EINVAL  # k > E
    assert f(P1, P2, P3, 8, 128, 33, 0.9, P4, P5, P6, P7, NULL, 0, NULL) == EUNSUPPORTED
    assert f(P1, P2, P3, 8, 16, 2, 0.9, NULL, P5, P6, P7, NULL, 0, NULL) == EINVAL   # no mass
    assert f(P1, P2, P3, 8, 16, 2, 0.9, P4, NULL, P6, P7, NULL, 0, NULL) == EINVAL   # no K_out
    assert f(P1, P2, P3, 8, 16, 2, 0.9, P4, P5, P2, P7, NULL, 0, NULL) == EALIAS     # idx on idx_full
    assert f(P1, P2, P3, 8, 16, 2, 0.9, P1, P5, P6, P7, NULL, 0, NULL) == EALIAS     # mass on logits
    assert f(ctypes.c_void_p(0x10004), P2, P3, 8, 16, 2, 0.9, P4, P5, P6, P7, NULL, 0, NULL) == EINVAL


def test_dispatch_rejects(lib):
    assert lib.moe_dispatch(P1, 8, 2, 16, P2, F32, 32, P3, P4, P5, P6, P7, NULL, 0, NULL) == EWORKSPACE
    assert lib.moe_dispatch(P1, 8, 2, 16, P2, F32, 32, P3, P4, P5, P6, P7, ctypes.c_void_p(0x900000), 8,
                            NULL) == EWORKSPACE
    assert lib.moe_dispatch(P1, 8, 20, 16, P2, F32, 32, P3, P4, P5, P6, P7, NULL, 0, NULL) == EINVAL
    assert lib.moe_dispatch(P1, 8, 2, 16, P2, F32, 32, P3, P4, P5, P6, P2, ctypes.c_void_p(0x900000),
                            1 << 20, NULL) == EALIAS


def test_ffn_rejects(lib):
    ws = ctypes.c_void_p(0x1000000)
    assert lib.moe_expert_ffn(P1, BF16, P2, 16, NULL, 0, 64, 100, 64, P3, P4, P5, ws, 1 << 30, NULL) == EUNSUPPORTED
    assert lib.moe_expert_ffn(P1, BF16, P2, 16, NULL, 0, 64, 256, 64, P3, P4, P5, ws, 1 << 30, NULL) == EUNSUPPORTED
    assert lib.moe_expert_ffn(P1, BF16, P2, 16, NULL, 0, 64, 128, 128, P3, P4, P5, ws, 1 << 30, NULL) == EUNSUPPORTED
    assert lib.moe_expert_ffn(P1, BF16, P2, 16, P6, 0, 64, 256, 128, P3, P4, P5, ws, 1 << 30, NULL) == EINVAL
    assert lib.moe_expert_ffn(P1, BF16, P2, 16, NULL, 0, 64, 256, 128, P3, P4, P5, ws, 16, NULL) == EWORKSPACE
    assert lib.moe_expert_ffn(P1, 7, P2, 16, NULL, 0, 64, 256, 128, P3, P4, P5, ws, 1 << 30, NULL) == EINVAL


def test_packed_ffn_and_pack_reject(lib):
    ws = ctypes.c_void_p(0x1000000)
    # packed weights are bf16 only; same shape limits as the row-major call
    assert lib.moe_expert_ffn_packed(P1, F32, P2, 16, NULL, 0, 64, 256, 128, P3, P4, P5, ws, 1 << 30,
                                     NULL) == EUNSUPPORTED
    assert lib.moe_expert_ffn_packed(P1, 7, P2, 16, NULL, 0, 64, 256, 128, P3, P4, P5, ws, 1 << 30,
                                     NULL) == EINVAL
    assert lib.moe_expert_ffn_packed(P1, BF16, P2, 16, NULL, 0, 64, 256, 64, P3, P4, P5, ws, 1 << 30,
                                     NULL) == EUNSUPPORTED
    assert lib.moe_expert_ffn_packed(P1, BF16, P2, 16, NULL, 0, 64, 256, 128, P3, P4, P5, ws, 1 << 30,
                                     NULL) == EUNSUPPORTED  # m % 256 != 0
    assert lib.moe_expert_ffn_packed(P1, BF16, P2, 16, NULL, 0, 64, 256, 256, P3, P4, P5, ws, 16,
                                     NULL) == EWORKSPACE
    assert lib.moe_expert_ffn_packed(P1, BF16, P2, 16, NULL, 0, 64, 256, 256, P3, P4, P1, ws, 1 << 30,
                                     NULL) == EALIAS
    # pack: bf16 only, rows % 32 and cols % 16, no overlap, nothing to do for empty
    assert lib.moe_pack_expert_weights(P1, F32, 4, 64, 64, P2, NULL) == EUNSUPPORTED
    assert lib.moe_pack_expert_weights(P1, BF16, 4, 48, 64, P2, NULL) == EUNSUPPORTED
    assert lib.moe_pack_expert_weights(P1, BF16, 4, 64, 40, P2, NULL) == EUNSUPPORTED
    assert lib.moe_pack_expert_weights(P1, BF16, 4, 64, 64, P1, NULL) == EALIAS
    assert lib.moe_pack_expert_weights(P1, BF16, -1, 64, 64, P2, NULL) == EINVAL
    assert lib.moe_pack_expert_weights(P1, BF16, 0, 64, 64, P2, NULL) == 0


def test_gather_ffn_rejects(lib):
    ws = ctypes.c_void_p(0x1000000)
    f = lib.moe_expert_ffn_packed_gather
    # (x, dtype, T, k, src_of_row, offsets, E, K_dev, n_K, d, m, w_gu, w_dn, y_perm, ws, ws_bytes, s)
    ok = (P1, BF16, 16, 2, P2, P3, 16, NULL, 0, 256, 256, P4, P5, P6, ws, 1 << 30, NULL)

    def call(**kw):
        names = ["x", "dt", "T", "k", "src", "off", "E", "K", "nK", "d", "m", "wgu", "wdn", "y", "ws",
                 "wsb", "s"]
        a = dict(zip(names, ok))
        a.update(kw)
        return f(*[a[n] for n in names])

    assert call(dt=F32) == EUNSUPPORTED
    assert call(dt=7) == EINVAL
    assert call(m=128) == EUNSUPPORTED
    assert call(d=384) == EUNSUPPORTED
    assert call(k=0) == EINVAL and call(k=17) == EINVAL and call(T=-1) == EINVAL
    assert call(K=P7, nK=0) == EINVAL
    assert call(src=NULL) == EINVAL and call(x=NULL) == EINVAL and call(y=NULL) == EINVAL
    assert call(wsb=16) == EWORKSPACE
    assert call(y=P1) == EALIAS      # y_perm on top of x
    assert call(ws=P2) == EALIAS     # workspace on top of src_of_row
    assert call(T=1 << 20, d=2048) == EUNSUPPORTED  # T*d*2 >= 2^31
    assert call(T=0) == 0            # nothing to do
    assert call(x=ctypes.c_void_p(0x10002)) == EINVAL  # misaligned


def test_gather_ffn_noalloc_rejects(lib):
    """The allocation-free expert FFN checks its arguments like the gathering
    FFN, and rejects sizes whose scratch exceeds its fixed array, all on the
    host before any HIP call."""
    from paper_2609_38823_amd import abi
    f = lib.moe_expert_ffn_packed_gather_noalloc
    names = ["x", "dt", "T", "k", "src", "off", "E", "K", "nK", "d", "m", "wgu", "wdn", "y", "s"]
    ok = (P1, BF16, 16, 2, P2, P3, 16, NULL, 0, 256, 256, P4, P5, P6, NULL)

    def call(**kw):
        a = dict(zip(names, ok))
        a.update(kw)
        return f(*[a[n] for n in names])

    assert call(dt=F32) == EUNSUPPORTED
    assert call(m=128) == EUNSUPPORTED
    assert call(k=0) == EINVAL and call(T=-1) == EINVAL
    assert call(src=NULL) == EINVAL and call(y=NULL) == EINVAL
    assert call(x=ctypes.c_void_p(0x10002)) == EINVAL
    assert call(T=0) == 0
    # m = 768: 21 800 dispatched rows fit the scratch, 21 900 do not
    assert abi.NOALLOC_SCRATCH_BYTES == 32 << 20
    assert lib.moe_workspace_size(10900, 128, 2, 2048, 768, 1) >= 256 + 21800 * 768 * 2
    assert call(T=10950, k=2, E=128, d=2048, m=768) == EWORKSPACE
    assert call(T=4096, k=8, E=128, d=2048, m=768) == EWORKSPACE  # 32 768 rows
    assert call(T=1 << 20, d=2048) == EUNSUPPORTED  # T*d*2 >= 2^31


def test_predicated_calls_check_like_the_plain_calls(lib):
    """The *_if calls reject what the plain calls reject, plus a misaligned
    predicate, all on the host (only rejected calls are made here)."""
    bad = ctypes.c_void_p(0x10002)
    G = ctypes.c_void_p(0x70000)
    # moe_route_packed_if: float32 x, E not a multiple of 32, misaligned guard
    rp = lib.moe_route_packed_if
    base = [P1, BF16, P2, NULL, 16, 64, 32, 2, NULL, 1, NULL, P3, P4, P5, P6, 1 << 30]
    assert rp(*base[:1], F32, *base[2:], G, 0, 1, NULL) == EUNSUPPORTED
    a = list(base); a[6] = 48
    assert rp(*a, G, 0, 1, NULL) == EUNSUPPORTED
    assert rp(*base, bad, 0, 1, NULL) == EINVAL
    # moe_dispatch_if: k > E, misaligned guard
    di = lib.moe_dispatch_if
    assert di(P1, 16, 9, 8, NULL, F32, 0, P2, P3, P4, P5, NULL, P6, 1 << 20, G, 0, 1, NULL) == EINVAL
    assert di(P1, 16, 2, 8, NULL, F32, 0, P2, P3, P4, P5, NULL, P6, 1 << 20, bad, 0, 1, NULL) == EINVAL
    # moe_calibrate_route_prefix_if: p outside (0, 1]
    cr = lib.moe_calibrate_route_prefix_if
    assert cr(P1, P2, P3, 16, 32, 2, 0.0, P4, P5, P6, P7, NULL, 0, G, 0, 1, NULL) == EINVAL
    # moe_expert_ffn_packed_gather_if: m not a multiple of 256
    fi = lib.moe_expert_ffn_packed_gather_if
    assert fi(P1, BF16, 16, 2, P2, P3, 16, NULL, 0, 256, 128, P4, P5, P6, ctypes.c_void_p(0x1000000),
              1 << 30, G, 0, 1, NULL) == EUNSUPPORTED
    assert fi(P1, BF16, 16, 2, P2, P3, 16, NULL, 0, 256, 256, P4, P5, P6, ctypes.c_void_p(0x1000000),
              1 << 30, bad, 0, 1, NULL) == EINVAL
    # moe_combine_residual_if: out shifted onto the residual
    ci = lib.moe_combine_residual_if
    assert ci(P1, BF16, P2, P3, 8, 2, 64, P4, ctypes.c_void_p(0x40010), G, 0, 1, NULL) == EALIAS
    # moe_savb_gate_if: exit_layer on top of the flag, misaligned exit_layer
    gi = lib.moe_savb_gate_if
    ws = ctypes.c_void_p(0x1000000)
    args = [P1, F32, 4, 64, P2, NULL, 8, P3, NULL, 0.5, NULL, P4, P5, ws, 1 << 20, G, 0, 1]
    assert gi(*args, P5, 3, NULL) == EALIAS
    assert gi(*args, bad, 3, NULL) == EINVAL


def test_route_rcep_rejects(lib):
    f = lib.moe_route_rcep
    names = ["x", "dt", "wp", "b", "T", "d", "E", "k", "p", "lg", "if_", "wf", "ms", "K", "ix", "w", "cn", "of",
             "sr", "rs", "ws", "wsb", "s"]
    base = dict(zip(names, (P1, BF16, P2, NULL, 64, 256, 128, 8, 0.9, P3, P4, P5, P6, P7,
                            ctypes.c_void_p(0x80000), ctypes.c_void_p(0x90000), ctypes.c_void_p(0xA0000),
                            ctypes.c_void_p(0xB0000), ctypes.c_void_p(0xC0000), ctypes.c_void_p(0xD0000),
                            ctypes.c_void_p(0x1000000), 1 << 30, NULL)))

    def call(**kw):
        a = dict(base)
        a.update(kw)
        return f(*[a[n] for n in names])

    assert call(dt=F32) == EUNSUPPORTED
    assert call(E=100) == EUNSUPPORTED       # not a multiple of 32 (packed router)
    assert call(k=0) == EINVAL and call(k=129) == EINVAL
    assert call(p=0.0) == EINVAL and call(p=1.5) == EINVAL
    assert call(K=NULL) == EINVAL and call(ix=NULL) == EINVAL
    assert call(wsb=16) == EWORKSPACE
    assert call(ix=P4) == EALIAS              # re-routed indices on top of the full-pool ones
    assert call(lg=P1) == EALIAS              # logits on top of x
    assert call(sr=ctypes.c_void_p(0xC0002)) == EINVAL


def test_rcep_layer_rejects(lib):
    names = ["x", "dt", "wp", "b", "T", "d", "E", "k", "p", "wgu", "wd", "m", "res", "out", "lg", "if_", "wf",
             "ms", "K", "ix", "w", "cn", "of", "sr", "rs", "yp", "ws", "wsb"]
    # every array 16 MiB apart (T 64, d 256, E 32, m 256: the largest, w_gate_up, is 8 MiB)
    arrays = {n: ctypes.c_void_p((i + 1) << 24) for i, n in enumerate(
        ["x", "wp", "wgu", "wd", "res", "out", "lg", "if_", "wf", "ms", "K", "ix", "w", "cn", "of", "sr", "rs",
         "yp", "ws"])}
    base = dict(arrays, dt=BF16, b=NULL, T=64, d=256, E=32, k=8, p=0.9, m=256, wsb=1 << 30)

    def call(f=lib.moe_rcep_layer, extra=(), **kw):
        a = dict(base)
        a.update(kw)
        return f(*[a[n] for n in names], *extra, NULL)

    assert call(dt=F32) == EUNSUPPORTED
    assert call(m=128) == EUNSUPPORTED         # packed expert FFN: m % 256 == 0
    assert call(E=48) == EUNSUPPORTED          # packed router: E % 32 == 0
    assert call(k=0) == EINVAL and call(k=33) == EINVAL
    assert call(p=0.0) == EINVAL
    assert call(out=NULL) == EINVAL and call(yp=NULL) == EINVAL
    assert call(yp=ctypes.c_void_p(arrays["yp"].value + 8)) == EINVAL
    assert call(wsb=16) == EWORKSPACE
    # out one row past the residual: neither in place nor disjoint
    assert call(out=ctypes.c_void_p(arrays["res"].value + 512)) == EALIAS
    assert call(out=ctypes.c_void_p(arrays["x"].value + 512)) == EALIAS
    assert call(out=arrays["wgu"]) == EALIAS   # out on top of the expert weights
    assert call(yp=arrays["x"]) == EALIAS
    assert call(ws=arrays["res"]) == EALIAS
    assert call(ix=arrays["if_"]) == EALIAS
    fi = lib.moe_rcep_layer_if
    G = ctypes.c_void_p(0x7F000000)
    assert call(fi, (ctypes.c_void_p(0x7F000002), 0, 1)) == EINVAL   # misaligned guard
    assert call(fi, (G, 0, 1), wsb=16) == EWORKSPACE


def test_dense_layer_rejects(lib):
    names = ["x", "dt", "wp", "b", "T", "d", "E", "k", "wgu", "wd", "m", "res", "out", "lg", "ix", "w", "cn", "of",
             "sr", "rs", "yp", "ws", "wsb"]
    # every array 16 MiB apart (T 64, d 256, E 32, k 8, m 256)
    arrays = {n: ctypes.c_void_p((i + 1) << 24) for i, n in enumerate(
        ["x", "wp", "wgu", "wd", "res", "out", "lg", "ix", "w", "cn", "of", "sr", "rs", "yp", "ws"])}
    base = dict(arrays, dt=BF16, b=NULL, T=64, d=256, E=32, k=8, m=256, wsb=1 << 30)

    def call(**kw):
        a = dict(base)
        a.update(kw)
        return lib.moe_dense_layer(*[a[n] for n in names], NULL)

    assert call(dt=F32) == EUNSUPPORTED
    assert call(d=128) == EUNSUPPORTED and call(m=128) == EUNSUPPORTED
    assert call(E=48) == EUNSUPPORTED         # packed router: E % 32 == 0
    assert call(k=0) == EINVAL and call(k=33) == EINVAL
    assert call(out=NULL) == EINVAL and call(yp=NULL) == EINVAL and call(sr=NULL) == EINVAL
    assert call(yp=ctypes.c_void_p(arrays["yp"].value + 8)) == EINVAL
    assert call(wsb=16) == EWORKSPACE
    assert call(out=ctypes.c_void_p(arrays["res"].value + 512)) == EALIAS   # one row past the residual
    assert call(out=ctypes.c_void_p(arrays["x"].value + 512)) == EALIAS
    assert call(out=arrays["wgu"]) == EALIAS
    assert call(yp=arrays["x"]) == EALIAS
    assert call(ws=arrays["res"]) == EALIAS
    assert call(ix=arrays["w"]) == EALIAS
    assert call(lg=arrays["wp"]) == EALIAS


def test_rcep_layer_chained_rejects(lib):
    names = ["py", "pr", "pw", "h", "dt", "wp", "b", "T", "d", "E", "k", "p", "wgu", "wd", "m", "lg", "if_", "wf",
             "ms", "K", "ix", "w", "cn", "of", "sr", "rs", "yp", "ws", "wsb"]
    # every array 16 MiB apart (T 64, d 256, E 32, k 8, m 256)
    arrays = {n: ctypes.c_void_p((i + 1) << 24) for i, n in enumerate(
        ["py", "pr", "pw", "h", "wp", "wgu", "wd", "lg", "if_", "wf", "ms", "K", "ix", "w", "cn", "of", "sr", "rs",
         "yp", "ws"])}
    base = dict(arrays, dt=BF16, b=NULL, T=64, d=256, E=32, k=8, p=0.9, m=256, wsb=1 << 30)

    def call(**kw):
        a = dict(base)
        a.update(kw)
        return lib.moe_rcep_layer_chained(*[a[n] for n in names], NULL)

    def at(n, off):
        return ctypes.c_void_p(arrays[n].value + off)

    assert call(dt=F32) == EUNSUPPORTED
    assert call(d=128) == EUNSUPPORTED         # d % 256 == 0
    assert call(m=128) == EUNSUPPORTED
    assert call(E=48) == EUNSUPPORTED
    assert call(k=0) == EINVAL and call(k=33) == EINVAL
    assert call(p=0.0) == EINVAL and call(p=1.5) == EINVAL
    assert call(pr=NULL) == EINVAL             # the previous layer's arrays: all or none
    assert call(py=NULL, pw=NULL) == EINVAL
    assert call(h=NULL) == EINVAL and call(yp=NULL) == EINVAL
    assert call(h=at("h", 8)) == EINVAL        # misaligned
    assert call(wsb=16) == EWORKSPACE
    assert call(py=arrays["h"]) == EALIAS      # previous expert outputs on top of h
    assert call(py=arrays["lg"]) == EALIAS     # ... on top of this call's logits
    assert call(py=at("yp", 512)) == EALIAS    # ... one row into this call's expert outputs
    assert call(pr=at("rs", 16)) == EALIAS     # row_of_slot shifted by four slots
    assert call(pr=arrays["w"]) == EALIAS      # previous row_of_slot on this call's weights
    assert call(pw=arrays["pr"]) == EALIAS     # two previous arrays on one another
    assert call(yp=arrays["h"]) == EALIAS
    assert call(ws=arrays["wgu"]) == EALIAS


def test_ffn_status_rejects(lib):
    lib.moe_ffn_status.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]
    ws = ctypes.c_void_p(0x1000000)
    st = ctypes.c_void_p(0x2000000)
    assert lib.moe_ffn_status(NULL, 1 << 20, st, NULL) == EINVAL
    assert lib.moe_ffn_status(ws, 1 << 20, NULL, NULL) == EINVAL
    assert lib.moe_ffn_status(ws, 1023, st, NULL) == EWORKSPACE   # smaller than the counter header
    assert lib.moe_ffn_status(ws, 1 << 20, ctypes.c_void_p(0x1000100), NULL) == EALIAS
    assert lib.moe_ffn_status(ctypes.c_void_p(0x1000004), 1 << 20, st, NULL) == EINVAL  # misaligned


def test_combine_and_drop_reject(lib):
    assert lib.moe_combine(P1, BF16, P2, P3, 8, 2, 64, P1, NULL) == EALIAS
    assert lib.moe_combine(P1, BF16, P2, P3, 8, 0, 64, P4, NULL) == EINVAL
    assert lib.drop_visual_block(P1, BF16, 10, 64, 5, 4, P2, NULL) == EINVAL
    assert lib.drop_visual_block(P1, BF16, 10, 64, 0, 11, P2, NULL) == EINVAL
    assert lib.drop_visual_block(P1, BF16, 10, 64, 0, 4, P1, NULL) == EALIAS
    assert lib.drop_visual_block(P1, BF16, 10, 64, 0, 10, P2, NULL) == 0  # nothing left to copy


def test_combine_residual_rejects(lib):
    # residual shifted by one row inside out: neither in place nor disjoint
    assert lib.moe_combine_residual(P1, BF16, P2, P3, 8, 2, 64, ctypes.c_void_p(P4.value + 128), P4, NULL) == EALIAS
    assert lib.moe_combine_residual(P1, BF16, P2, P3, 8, 2, 64, P4, P1, NULL) == EALIAS
    assert lib.moe_combine_residual(P1, BF16, P2, P3, 8, 2, 64, None, P4, NULL) == EINVAL
    assert lib.moe_combine_residual(P1, BF16, P2, P3, 8, 0, 64, P4, P4, NULL) == EINVAL
    assert lib.moe_combine_residual(P1, BF16, P2, P3, 0, 2, 64, P4, P4, NULL) == 0  # T = 0


def test_permute_experts_rejects(lib):
    nul = None
    # a pair with only one side given
    assert lib.moe_permute_experts(P1, 4, 64, 32, BF16, P2, nul, nul, nul, nul, nul, nul, nul,
                                   NULL) == EINVAL
    # output overlapping its input
    assert lib.moe_permute_experts(P1, 4, 64, 32, BF16, nul, nul, P2, nul, nul, nul, P2, nul,
                                   NULL) == EALIAS
    # output overlapping the order array
    assert lib.moe_permute_experts(P1, 4, 64, 32, BF16, nul, nul, P2, nul, nul, nul, P1, nul,
                                   NULL) == EALIAS
    assert lib.moe_permute_experts(nul, 4, 64, 32, BF16, nul, nul, P2, nul, nul, nul, P3, nul,
                                   NULL) == EINVAL
    assert lib.moe_permute_experts(P1, 0, 64, 32, BF16, nul, nul, P2, nul, nul, nul, P3, nul,
                                   NULL) == EINVAL
    assert lib.moe_permute_experts(P1, 2000, 64, 32, BF16, nul, nul, P2, nul, nul, nul, P3, nul,
                                   NULL) == EINVAL
    # misaligned bf16 weights
    assert lib.moe_permute_experts(P1, 4, 64, 32, BF16, nul, nul, ctypes.c_void_p(P2.value + 1), nul, nul, nul, P3, nul,
                                   NULL) == EINVAL


def test_packed_router_rejects(lib):
    # float32 x, E % 32, d % 64, no x
    assert lib.moe_route_packed(P1, F32, P2, NULL, 8, 64, 32, 2, NULL, 1, NULL, P3, P4, P5, WS, 1 << 20,
                                NULL) == EUNSUPPORTED
    assert lib.moe_route_packed(P1, BF16, P2, NULL, 8, 64, 48, 2, NULL, 1, NULL, P3, P4, P5, WS, 1 << 20,
                                NULL) == EUNSUPPORTED
    assert lib.moe_route_packed(P1, BF16, P2, NULL, 8, 96, 32, 2, NULL, 1, NULL, P3, P4, P5, WS, 1 << 20,
                                NULL) == EUNSUPPORTED
    assert lib.moe_route_packed(NULL, BF16, P2, NULL, 8, 64, 32, 2, NULL, 1, NULL, P3, P4, P5, WS, 1 << 20,
                                NULL) == EINVAL
    # logits overlapping the packed weights
    assert lib.moe_route_packed(P1, BF16, P2, NULL, 8, 64, 32, 2, NULL, 1, NULL, P2, P4, P5, WS, 1 << 20,
                                NULL) == EALIAS
    # a split needs workspace (T = 8: 8 splits of the 2048-wide d-range)
    assert lib.moe_route_packed(P1, BF16, P2, NULL, 8, 2048, 128, 8, NULL, 1, NULL, P3, P4, P5, NULL, 0,
                                NULL) == EWORKSPACE
    assert lib.moe_pack_router(P1, 64, 48, P2, NULL) == EUNSUPPORTED
    assert lib.moe_pack_router(P1, 96, 32, P2, NULL) == EUNSUPPORTED
    assert lib.moe_pack_router(P1, 2048, 128, ctypes.c_void_p(P1.value + 1024), NULL) == EALIAS
    assert lib.moe_pack_router(NULL, 64, 32, P2, NULL) == EINVAL
    # the workspace covers the packed router's split partials
    assert lib.moe_workspace_size(64, 128, 8, 2048, 768, 1) >= 8 * 64 * 128 * 4


def test_savb_gate_rejects(lib):
    lib.moe_savb_workspace_size.restype = ctypes.c_size_t
    assert lib.moe_savb_workspace_size(512, 2048, 512) >= 16 * 2048 * 4 + 512 * 4
    assert lib.moe_savb_workspace_size(0, 2048, 512) == 0
    th = ctypes.c_double(0.5)
    nan = ctypes.c_double(float("nan"))
    big = ctypes.c_size_t(1 << 30)
    # n = 0, d > 8192, NaN theta, no workspace
    assert lib.moe_savb_gate(P1, BF16, 0, 64, P2, NULL, 16, P3, NULL, th, NULL, P4, P5, WS, big, NULL) == EINVAL
    assert lib.moe_savb_gate(P1, BF16, 4, 9000, P2, NULL, 16, P3, NULL, th, NULL, P4, P5, WS, big, NULL) == EINVAL
    assert lib.moe_savb_gate(P1, BF16, 4, 64, P2, NULL, 16, P3, NULL, nan, NULL, P4, P5, WS, big, NULL) == EINVAL
    assert lib.moe_savb_gate(P1, BF16, 40, 64, P2, NULL, 16, P3, NULL, th, NULL, P4, P5, WS,
                             ctypes.c_size_t(16), NULL) == EWORKSPACE
    # the flag written over the weights
    assert lib.moe_savb_gate(P1, BF16, 4, 64, P2, NULL, 16, P3, NULL, th, NULL, P4, P2, WS, big, NULL) == EALIAS
    # drop_visual_block_if: misaligned flag, output over the flag
    assert lib.drop_visual_block_if(P1, BF16, 10, 64, 0, 4, ctypes.c_void_p(P3.value + 2), P2, NULL) == EINVAL
    assert lib.drop_visual_block_if(P1, BF16, 10, 64, 0, 4, P2, P2, NULL) == EALIAS
    assert lib.drop_visual_block_if(P1, BF16, 10, 64, 5, 4, P3, P2, NULL) == EINVAL


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    from paper_2609_38823_amd import abi
    monkeypatch.setattr(abi, "_lib", None)
    monkeypatch.setattr(abi, "LIB_PATH", str(tmp_path / "absent.so"))
    with pytest.raises(RuntimeError, match="missing"):
        abi.load()


def test_binding_checks_array_dtypes():
    """Typed array arguments (indices, routing weights, masses) are checked
    before a pointer reaches the library."""
    import torch

    from paper_2609_38823_amd import abi
    with pytest.raises(TypeError):
        abi._i32(torch.zeros(3, dtype=torch.int64))
    with pytest.raises(TypeError):
        abi._f32(torch.zeros(3, dtype=torch.float64))
    with pytest.raises(TypeError):
        abi._f64(torch.zeros(3, dtype=torch.float32))
    with pytest.raises(ValueError):  # right dtype, but not on the GPU
        abi._i32(torch.zeros(3, dtype=torch.int32))
    assert abi._i32(None) is None
