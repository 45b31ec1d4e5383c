"""Build checks that need no GPU: the device code of every HIP source,
compiled with the library's own flags, contains no packed-fp32 VALU
instructions and no scratch (private memory) traffic in the kernels."""

import os
import re
import subprocess

import pytest

from paper_2609_38823_amd import build

SOURCES = build.sources()


@pytest.mark.parametrize("src", SOURCES, ids=[os.path.basename(s) for s in SOURCES])
def test_device_asm_has_no_packed_fp32(src, tmp_path):
    out = tmp_path / "dev.s"
    flags = [f for f in build.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    cmd = [build.hipcc(), *flags, "--cuda-device-only", "-S", "-I",
           os.path.join(build.ROOT, "include"), src, "-o", str(out)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    asm = out.read_text()
    assert not re.search(r"\bv_pk_(fma|mul|add)_f32\b", asm), "packed fp32 instruction emitted"
    assert not re.search(r"\bscratch_(load|store)", asm), "kernel spills to scratch"
