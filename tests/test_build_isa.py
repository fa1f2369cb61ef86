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


@pytest.mark.parametrize("src", ["fwd_bf16.hip", "bwd_bf16.hip", "bwd_bf16_d64.hip", "bwd_dq_bf16.hip",
                                 "bwd_dq_bf16_d64.hip", "bwd_dq_ds.hip"])
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


@pytest.mark.parametrize("src", ["fwd_bf16.hip", "bwd_bf16.hip", "bwd_bf16_d64.hip", "bwd_dq_bf16.hip",
                                 "bwd_dq_bf16_d64.hip", "bwd_dq_ds.hip", "merge.hip", "bwd_pre.hip"])
def test_no_packed_fp32_and_no_scalar_stores(src, tmp_path):
    text = _asm(src, tmp_path)
    assert not re.search(r"\bv_pk_(add|mul|fma)_f32\b", text)
    assert not re.search(r"\bs_(store|buffer_store|atomic|dcache_wb)", text)


# Memory instructions in the kernels are global (or LDS) ones: a flat access also counts against the
# LDS wait counter, so every wait for an LDS read would wait for it too (a pointer rebuilt from an
# integer loses its address space and turns a store into a flat store; the dS stores of the dK/dV
# kernel cost a third more time that way).
@pytest.mark.parametrize("src", ["fwd_bf16.hip", "bwd_bf16.hip", "bwd_bf16_d64.hip", "bwd_dq_bf16.hip",
                                 "bwd_dq_bf16_d64.hip", "bwd_dq_ds.hip", "merge.hip", "bwd_pre.hip",
                                 "tt_tokenize.hip"])
def test_no_flat_memory_instructions(src, tmp_path):
    text = _asm(src, tmp_path)
    assert not re.search(r"^\s*flat_(load|store|atomic)", text, re.M)


# The dK/dV kernel issues its matrix products as inline assembly (to choose the register file of
# every operand), so the compiler inserts no wait states for them.  Its schedule has to keep (1)
# every MFMA result away from any other instruction that reads or overwrites it for at least 20
# wait states (16-pass products need 19 on gfx940-class parts, 8-pass ones 12; only the next
# product of the same accumulation chain may follow at once), and (2) every vector-ALU write of an
# MFMA operand at least 2 wait states ahead of the product.  A wait state is one issued
# instruction, or n + 1 for s_nop n; the check walks each kernel's code in program order.
MFMA_RESULT_WAIT = 20
VALU_TO_MFMA_WAIT = 2


def _regs(tok):
    m = re.fullmatch(r"([va])\[(\d+):(\d+)\]", tok)
    if m:
        return {(m.group(1), r) for r in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.fullmatch(r"([va])(\d+)", tok)
    return {(m.group(1), int(m.group(2)))} if m else set()


def _split(inst):
    parts = inst.split(None, 1)
    ops = [t.strip() for t in parts[1].split(",")] if len(parts) > 1 else []
    return parts[0], ops


def _waits(inst):
    op, ops = _split(inst)
    return int(ops[0], 0) + 1 if op == "s_nop" else 1


def mfma_hazards(code, window=96):
    """(closest MFMA-result access, closest vector write before an MFMA read) in wait states,
    None where no such pair occurs within `window` instructions."""
    near_result, near_write = None, None
    for i, inst in enumerate(code):
        op, ops = _split(inst)
        if not op.startswith("v_mfma") or len(ops) < 4:
            continue
        dst = _regs(ops[0])
        w = 0
        for j in range(i + 1, min(len(code), i + window)):
            op2, ops2 = _split(code[j])
            touched = set().union(*(_regs(t) for t in ops2)) if ops2 else set()
            if touched & dst:
                same_chain = (op2.startswith("v_mfma") and _regs(ops2[0]) == dst and
                              _regs(ops2[3]) == dst and not (_regs(ops2[1]) | _regs(ops2[2])) & dst)
                if not same_chain:
                    near_result = w if near_result is None else min(near_result, w)
                break
            w += _waits(code[j])
        srcs = set().union(*(_regs(t) for t in ops[1:4]))
        w = 0
        for j in range(i - 1, max(-1, i - 16), -1):
            op2, ops2 = _split(code[j])
            if ops2 and not op2.startswith(("s_", "v_mfma")) and _regs(ops2[0]) & srcs:
                # the operand's last writer: a hazard only for the vector ALU (loads are waited on)
                if op2.startswith("v_"):
                    near_write = w if near_write is None else min(near_write, w)
                break
            w += _waits(code[j])
    return near_result, near_write


def _kernel_bodies(text):
    bodies, cur = [], None
    for line in text.splitlines():
        s = line.split(";")[0].strip()
        if re.match(r"^_Z\w+:$", s):
            cur = []
            bodies.append((s[:-1], cur))
        elif cur is not None:
            if s.startswith("s_endpgm"):
                cur = None
            elif s and not s.startswith(".") and not s.endswith(":"):
                cur.append(s)
    return bodies


def test_hazard_check_catches_close_accesses():
    mfma = "v_mfma_f32_32x32x16_bf16 v[0:15], v[16:19], a[0:3], v[0:15]"
    first = "v_mfma_f32_32x32x16_bf16 v[0:15], v[16:19], a[0:3], 0"
    # a result read by the vector ALU one instruction later; the same after 21 wait states
    assert mfma_hazards([first, mfma, "v_mov_b32 v40, v41", "v_add_f32 v20, v3, v4"])[0] == 1
    ok = [first, mfma, "s_nop 15", "v_mov_b32 v40, v41", "s_nop 3", "v_add_f32 v20, v3, v4"]
    assert mfma_hazards(ok)[0] == 21
    # the next product of the same chain may follow at once; a new chain over it may not
    assert mfma_hazards([first, mfma, mfma])[0] is None
    assert mfma_hazards([mfma, first])[0] == 0
    # an operand written by the vector ALU right before the product, and 2 wait states before it;
    # a load that overwrites the operand after the vector write ends the search
    assert mfma_hazards(["v_xor_b32 v17, v1, v2", mfma])[1] == 0
    assert mfma_hazards(["v_add_u32 v16, v1, v2", "ds_read_b128 v[16:19], v16", mfma])[1] is None
    assert mfma_hazards(["v_accvgpr_write_b32 a2, v9", "s_nop 1", mfma])[1] == 2
    assert mfma_hazards(["v_accvgpr_write_b32 a2, v9", "s_nop 0", mfma])[1] == 1


# bwd_bf16.hip holds two d = 128 instances of the dK/dV kernel (with and without the dS stores)
@pytest.mark.parametrize("src,kernel,products,count", [("bwd_bf16.hip", "bwd_dkdv_kernel", 80, 2),
                                                        ("bwd_dq_bf16.hip", "bwd_dq_kernel", 128, 1)])
def test_inline_mfma_spacing(src, kernel, products, count, tmp_path):
    text = _asm(src, tmp_path)
    # no register spills: these schedules keep every value in registers (a spill would add scratch
    # memory traffic the schedule does not account for)
    sizes = re.findall(r"\.amdhsa_private_segment_fixed_size (\d+)", text)
    assert sizes and all(int(x) == 0 for x in sizes), sizes
    bodies = _kernel_bodies(text)
    kernels = [(name, code) for name, code in bodies if kernel in name]
    assert len(kernels) == count, [n for n, _ in bodies]      # d = 128
    for name, code in kernels:
        assert sum(1 for c in code if c.startswith("v_mfma")) >= products, name
        near_result, near_write = mfma_hazards(code)
        assert near_result is not None and near_result >= MFMA_RESULT_WAIT, (name, near_result)
        assert near_write is None or near_write >= VALU_TO_MFMA_WAIT, (name, near_write)
