"""Properties of the generated gfx950 code that the kernels rely on (CPU only: hipcc
cross-compiles).  The direct global->LDS loads set m0 in inline asm; that is only safe while the
compiler itself never reads or writes m0 in the same kernels."""

import os
import re
import shutil
import subprocess

import pytest

from paper_2507_16697_amd import build as B

pytestmark = pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                                reason="hipcc not available")


def _asm(src, tmp_path):
    out = tmp_path / (os.path.basename(src) + ".s")
    cmd = [B.hipcc(), *B.HIPCC_FLAGS, "-I", B.INCLUDE, "-I", B.CSRC, "--cuda-device-only", "-S",
           os.path.join(B.CSRC, src), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return out.read_text()


@pytest.mark.parametrize("src", ["fwd_bf16.hip", "bwd_bf16.hip"])
def test_m0_only_feeds_direct_lds_loads(src, tmp_path):
    lines = [l.strip() for l in _asm(src, tmp_path).splitlines()]
    code = [l for l in lines if l and not l.startswith(";") and not l.startswith(".")]
    uses = [i for i, l in enumerate(code) if re.search(r"\bm0\b", l)]
    assert uses, "expected direct LDS loads"
    for i in uses:
        assert re.match(r"s_mov_b32 m0, s\d+$", code[i]), code[i]
        # one wait state between the scalar write of m0 and the LDS DMA that reads it
        assert code[i + 1] == "s_nop 0", code[i + 1]
        assert re.match(r"global_load_lds_dword(x4)? ", code[i + 2]), code[i + 2]


@pytest.mark.parametrize("src", ["fwd_bf16.hip", "bwd_bf16.hip", "merge.hip", "bwd_pre.hip"])
def test_no_packed_fp32_and_no_scalar_stores(src, tmp_path):
    text = _asm(src, tmp_path)
    assert not re.search(r"\bv_pk_(add|mul|fma)_f32\b", text)
    assert not re.search(r"\bs_(store|buffer_store|atomic|dcache_wb)", text)
