"""libringx on the host: it loads, exports every symbol include/ringx.h declares, and rejects bad
arguments before any HIP call (no GPU needed: every call here fails validation or is host-only)."""

import ctypes
import os
import re

import pytest

from oracle import attention_fp64 as oa
from paper_2507_16697_amd import ringx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ringx.h")

pytestmark = pytest.mark.skipif(not os.path.exists(ringx.LIB_PATH),
                                reason="libringx.so not built (run python -m paper_2507_16697_amd.build)")

OK, NULLPTR, SHAPE, CHUNKS, UNSUP, ALIGN, WORKSPACE, HIP, ALIAS, SCRATCH = range(10)
BF16, FP32 = ringx.RINGX_BF16, ringx.RINGX_FP32

# Fake, never dereferenced device addresses: validation rejects every call below before any HIP
# call, so these are only compared and aligned, never used.
GB = 1 << 30
QP, KP, VP, OP, LP = (0x10_0000_0000 + i * 64 * GB for i in range(5))


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:ringx_status|size_t|const char\*)\s+(ringx_\w+)\(", text, re.M)))


def test_header_declares_the_entry_points():
    assert declared_functions() == sorted(ringx.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(ringx.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings():
    for code in range(10):
        s = ringx.ringx_status_str(code)
        assert isinstance(s, str) and s
    assert ringx.ringx_status_str(OK) == "ok"
    assert ringx.ringx_status_str(1234) == "unknown status"


def test_chunk_bounds_equal_the_oracle_formula():
    for nk in list(range(1, 130)) + [1000, 4097, 262144, 524288]:
        for R in sorted({1, 2, 3, 7, 8, nk // 2 or 1, nk}):
            if R > nk:
                continue
            for r in range(R) if R <= 64 else (0, 1, R // 2, R - 1):
                assert ringx.ringx_chunk_bounds(nk, R, r) == oa.chunk_bounds(nk, R, r)


def test_chunk_bounds_huge_does_not_overflow():
    nk = (1 << 40) - 3
    R = 7
    prev = 0
    for r in range(R):
        lo, hi = ringx.ringx_chunk_bounds(nk, R, r)
        assert lo == prev and hi == ((r + 1) * nk) // R
        prev = hi


@pytest.mark.parametrize("args,code", [((5, 0, 0), CHUNKS), ((5, 6, 0), CHUNKS), ((5, 2, 2), CHUNKS),
                                       ((5, 2, -1), CHUNKS), ((0, 1, 0), SHAPE)])
def test_chunk_bounds_errors(args, code):
    with pytest.raises(ringx.RingxError) as e:
        ringx.ringx_chunk_bounds(*args)
    assert e.value.status == code


def fwd(q=QP, k=KP, v=VP, o=OP, l=LP, B=1, H=2, Nq=100, Nk=300, d=64, R=3, scale=0.125, dt=BF16):
    return ringx.lib().ringx_attn_fwd(q, k, v, o, l, B, H, Nq, Nk, d, R, scale, dt, None)


def part(q=QP, k=KP, v=VP, o=OP, l=LP, B=1, H=2, Nq=100, Nk=300, d=64, R=3, scale=0.125, dt=BF16):
    return ringx.lib().ringx_attn_fwd_partials(q, k, v, o, l, B, H, Nq, Nk, d, R, scale, dt, None)


@pytest.mark.parametrize("fn", [fwd, part])
def test_forward_validation(fn):
    assert fn(q=0) == NULLPTR and fn(l=0) == NULLPTR and fn(o=0) == NULLPTR
    assert fn(B=0) == SHAPE and fn(H=-1) == SHAPE and fn(Nq=0) == SHAPE and fn(Nk=0) == SHAPE
    assert fn(Nk=(1 << 31) + 1, R=1) == SHAPE
    assert fn(Nq=(1 << 31) - 127, B=1, H=1) == SHAPE               # queries per head above 2^31 - 128
    assert fn(scale=0.0) == SHAPE and fn(scale=float("nan")) == SHAPE and fn(scale=float("inf")) == SHAPE
    assert fn(scale=-1.0) == SHAPE
    assert fn(R=0) == CHUNKS and fn(R=301) == CHUNKS
    assert fn(d=96) == UNSUP and fn(d=32) == UNSUP and fn(d=256) == UNSUP
    assert fn(d=129, dt=FP32) == UNSUP and fn(d=0, dt=FP32) == UNSUP
    assert fn(dt=7) == UNSUP
    assert fn(q=QP + 8) == ALIGN and fn(o=OP + 2) == ALIGN and fn(l=LP + 4) == ALIGN
    assert fn(o=QP) == ALIAS and fn(l=KP + 1024) == ALIAS and fn(l=OP) == ALIAS
    assert fn(B=1 << 20, H=1 << 20, Nq=1 << 20) == SHAPE          # size overflow
    assert fn(B=70000, dt=FP32, H=1) == SHAPE                       # fp32 grid limit


def merge(po=QP, pl=KP, o=OP, l=LP, R=3, B=1, H=2, Nq=100, d=64, dt=BF16):
    return ringx.lib().ringx_lse_merge(po, pl, o, l, R, B, H, Nq, d, dt, None)


def test_merge_validation():
    assert merge(po=0) == NULLPTR and merge(l=0) == NULLPTR
    assert merge(R=0) == CHUNKS
    assert merge(B=0) == SHAPE and merge(Nq=0) == SHAPE
    assert merge(d=0) == UNSUP and merge(d=130) == UNSUP and merge(d=6) == UNSUP
    assert merge(dt=5) == UNSUP
    assert merge(po=QP + 4) == ALIGN
    assert merge(o=QP) == ALIAS and merge(l=KP) == ALIAS


def bwd(ws=VP + 32 * GB, wsb=1 << 20, dq=OP, dk=OP + 8 * GB, dv=OP + 16 * GB, acc=0, B=1, H=2,
        Nq=100, Nk=300, d=64, R=3, dt=BF16, q=QP, lse=LP):
    return ringx.lib().ringx_attn_bwd(q, KP, VP, QP + 8 * GB, QP + 16 * GB, lse, dq, dk, dv, B, H,
                                      Nq, Nk, d, R, 0.125, dt, acc, ws, wsb, None)


def test_backward_validation():
    need = ringx.ringx_bwd_workspace_bytes(1, 2, 100, 300, 64, 3, BF16)
    assert need >= 2 * 100 * 4 and need % 256 == 0
    assert ringx.ringx_bwd_workspace_bytes(1, 2, 100, 300, 96, 3, BF16) == 0
    assert bwd(q=0) == NULLPTR and bwd(dq=0) == NULLPTR and bwd(lse=0) == NULLPTR
    assert bwd(ws=0) == WORKSPACE and bwd(wsb=need - 1) == WORKSPACE
    assert bwd(R=301) == CHUNKS and bwd(d=80) == UNSUP and bwd(B=0) == SHAPE
    assert bwd(dq=OP + 4) == ALIGN and bwd(ws=VP + 32 * GB + 8) == ALIGN
    assert bwd(dq=QP) == ALIAS                      # dq over q
    assert bwd(dk=OP) == ALIAS                      # dk over dq
    assert bwd(ws=OP + 16 * GB) == ALIAS            # workspace over dv


def bwd_noalloc(q=QP, k=KP, v=VP, o=OP, do=OP + 4 * GB, lse=LP, dq=OP + 8 * GB,
                dk=OP + 12 * GB, dv=OP + 16 * GB, B=1, H=2, Nq=100, Nk=300, d=64, R=3,
                dt=BF16, acc=0):
    return ringx.lib().ringx_attn_bwd_noalloc(q, k, v, o, do, lse, dq, dk, dv, B, H, Nq, Nk, d,
                                              R, 0.125, dt, acc, None)


def test_backward_noalloc_validation():
    """Everything ringx_attn_bwd checks, plus the fixed scratch limit (B * H * Nq rows), before
    any HIP call."""
    rows = ringx.NOALLOC_MAX_ROWS
    assert bwd_noalloc(q=0) == NULLPTR and bwd_noalloc(dv=0) == NULLPTR
    assert bwd_noalloc(R=301) == CHUNKS and bwd_noalloc(d=80) == UNSUP
    assert bwd_noalloc(B=0) == SHAPE
    assert bwd_noalloc(B=1, H=1, Nq=rows + 1) == SCRATCH
    assert bwd_noalloc(B=2, H=16, Nq=rows // 32 + 1) == SCRATCH
    assert bwd_noalloc(B=3, H=5, Nq=1 << 20) == SCRATCH


def pre(o=QP, do=KP, l=VP, dl=LP, B=1, H=2, Nq=100, d=64, dt=BF16):
    return ringx.lib().ringx_bwd_preprocess(o, do, l, dl, B, H, Nq, d, dt, None)


def test_preprocess_validation():
    assert pre(o=0) == NULLPTR and pre(l=0) == NULLPTR and pre(dl=0) == NULLPTR
    assert pre(B=0) == SHAPE and pre(d=96) == UNSUP
    assert pre(dl=LP + 4) == ALIGN and pre(l=VP + 8) == ALIGN
    assert pre(dl=QP) == ALIAS and pre(dl=VP) == ALIAS
    # delta holds two rows of B*H*Nq floats (D, then nl): lse just past the first row overlaps it
    assert pre(l=LP + 800) == ALIAS


def dkdv(dk=OP, dv=OP + 8 * GB, lse=LP, delta=LP + 8 * GB, R=3, d=64, acc=0):
    return ringx.lib().ringx_attn_bwd_dkdv(QP, KP, VP, QP + 16 * GB, lse, delta, dk, dv, 1, 2, 100,
                                           300, d, R, 0.125, BF16, acc, None)


def dqs(dq=OP, lse=LP, delta=LP + 8 * GB, R=3, d=64):
    return ringx.lib().ringx_attn_bwd_dq(QP, KP, VP, QP + 16 * GB, lse, delta, dq, 1, 2, 100, 300,
                                         d, R, 0.125, BF16, None)


def test_gradient_stage_validation():
    assert dkdv(dk=0) == NULLPTR and dkdv(delta=0) == NULLPTR and dqs(dq=0) == NULLPTR
    assert dkdv(R=301) == CHUNKS and dqs(R=0) == CHUNKS
    assert dkdv(d=80) == UNSUP and dqs(d=80) == UNSUP
    assert dkdv(dv=OP + 8 * GB + 4) == ALIGN and dqs(dq=OP + 8) == ALIGN
    assert dkdv(dv=OP) == ALIAS and dkdv(dk=KP) == ALIAS and dqs(dq=LP) == ALIAS
    assert dqs(dq=LP + 8 * GB) == ALIAS    # dq over delta
    assert dqs(dq=LP + 8 * GB + 800) == ALIAS    # dq over delta's second row (nl)


def test_stored_ds_sizes():
    """Stored dS: 2 KiB per (query head, 32-query block, 32-key block) of the padded axes: the
    queries padded to 128 per head and every chunk's keys to whole 128-key tiles."""
    def pad(x, m):
        return -(-x // m) * m
    for H, Hkv, Nq, Nk, R, kv in [(1, 1, 128, 128, 1, 1), (2, 2, 200, 777, 3, 2), (4, 2, 130, 300, 5, 1),
                                   (16, 16, 32768, 262144, 8, 2), (4, 1, 64, 129, 1, 1)]:
        G = H // Hkv
        per_chunk = pad(-(-Nk // R), 128)
        want = kv * G * pad(Nq, 128) * R * per_chunk * 2
        assert ringx.ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, 128, R, kv) == want
    assert ringx.ringx_bwd_ds_bytes(16, 16, 32768, 262144, 128, 8, 1) == 16 << 30
    # invalid: head dim 64, Hkv not dividing H, no heads, R > Nk
    assert ringx.ringx_bwd_ds_bytes(2, 2, 100, 300, 64, 3, 1) == 0
    assert ringx.ringx_bwd_ds_bytes(4, 3, 100, 300, 128, 3, 1) == 0
    assert ringx.ringx_bwd_ds_bytes(2, 2, 100, 300, 128, 3, 0) == 0
    assert ringx.ringx_bwd_ds_bytes(2, 2, 100, 300, 128, 301, 1) == 0
    stats = ringx.ringx_bwd_workspace_bytes(2, 4, 100, 300, 128, 3, BF16)
    assert ringx.ringx_bwd_ds_workspace_bytes(2, 4, 2, 100, 300, 128, 3, 3) == \
        stats + ringx.ringx_bwd_ds_bytes(4, 2, 100, 300, 128, 3, 3)
    assert ringx.ringx_bwd_ds_workspace_bytes(2, 4, 2, 100, 300, 128, 3, 5) == 0   # > B * Hkv


DSP = OP + 32 * GB       # a fake stored-dS buffer


def dkdv_ds(ds=DSP, dsb=1 << 30, dk=OP, dv=OP + 8 * GB, delta=LP + 8 * GB, kv0=0, kvn=2, H=4,
            Hkv=2, B=1, d=128, dt=BF16, R=3, q=QP):
    return ringx.lib().ringx_attn_bwd_dkdv_ds(q, KP, VP, QP + 16 * GB, LP, delta, dk, dv, ds, dsb,
                                              B, H, Hkv, 100, 300, d, R, 0.125, dt, 0, kv0, kvn,
                                              None)


def dq_ds(ds=DSP, dsb=1 << 30, dq=OP, kv0=0, kvn=2, H=4, Hkv=2, B=1, d=128, dt=BF16, k=KP):
    return ringx.lib().ringx_attn_bwd_dq_ds(ds, dsb, k, dq, B, H, Hkv, 100, 300, d, 3, 0.125, dt,
                                            kv0, kvn, None)


def bwd_ds(ws=VP + 32 * GB, wsb=1 << 30, dq=OP, dk=OP + 8 * GB, dv=OP + 16 * GB, d=128, dt=BF16,
           Hkv=2):
    return ringx.lib().ringx_attn_bwd_ds(QP, KP, VP, QP + 8 * GB, QP + 16 * GB, LP, dq, dk, dv, 1,
                                         4, Hkv, 100, 300, d, 3, 0.125, dt, 0, ws, wsb, None)


def test_stored_ds_validation():
    need = ringx.ringx_bwd_ds_bytes(4, 2, 100, 300, 128, 3, 2)
    assert dkdv_ds(q=0) == NULLPTR and dkdv_ds(dk=0) == NULLPTR and dq_ds(dq=0) == NULLPTR
    assert dq_ds(k=0) == NULLPTR and bwd_ds(dq=0) == NULLPTR
    assert dkdv_ds(ds=0) == WORKSPACE and dq_ds(ds=0) == WORKSPACE
    assert dkdv_ds(dsb=need - 1) == WORKSPACE and dq_ds(dsb=need - 1) == WORKSPACE
    # the slab must lie inside the B * Hkv K/V heads
    assert dkdv_ds(kv0=-1) == SHAPE and dkdv_ds(kvn=0) == SHAPE and dkdv_ds(kv0=1, kvn=2) == SHAPE
    assert dq_ds(kv0=2, kvn=1) == SHAPE and dkdv_ds(B=2, kv0=3, kvn=2) == SHAPE
    assert dkdv_ds(Hkv=3) == SHAPE and dq_ds(Hkv=3) == SHAPE and bwd_ds(Hkv=3) == SHAPE
    # bf16 with d = 128 only
    for fn in (dkdv_ds, dq_ds, bwd_ds):
        assert fn(d=64) == UNSUP and fn(dt=FP32) == UNSUP
    assert dkdv_ds(R=301) == CHUNKS
    assert dkdv_ds(ds=DSP + 8) == ALIGN and dq_ds(dq=OP + 4) == ALIGN
    assert dkdv_ds(ds=QP) == ALIAS and dkdv_ds(ds=OP + 8 * GB - 64) == ALIAS   # ds over q, dv
    assert dq_ds(dq=DSP) == ALIAS and dq_ds(dq=KP) == ALIAS
    # the whole backward: the per-row statistics and one K/V head's dS at least
    one = ringx.ringx_bwd_ds_workspace_bytes(1, 4, 2, 100, 300, 128, 3, 1)
    assert bwd_ds(ws=0) == WORKSPACE and bwd_ds(wsb=one - 1) == WORKSPACE
    assert bwd_ds(ws=VP + 32 * GB + 8) == ALIGN
    assert bwd_ds(ws=OP + 16 * GB) == ALIAS and bwd_ds(dk=OP) == ALIAS


def fstep(q=QP, k=KP, v=VP, o=OP, l=LP, B=1, H=2, Nq=100, Nk=300, d=64, scale=0.125, dt=BF16,
          first=1):
    return ringx.lib().ringx_attn_fwd_step(q, k, v, o, l, B, H, Nq, Nk, d, scale, dt, first, None)


def test_fwd_step_validation():
    assert fstep(q=0) == NULLPTR and fstep(o=0) == NULLPTR and fstep(l=0) == NULLPTR
    assert fstep(Nk=0) == SHAPE and fstep(scale=0.0) == SHAPE and fstep(B=0) == SHAPE
    assert fstep(d=96) == UNSUP and fstep(dt=3) == UNSUP
    assert fstep(o=OP + 4) == ALIGN and fstep(l=LP + 8) == ALIGN
    assert fstep(o=QP) == ALIAS and fstep(l=VP) == ALIAS and fstep(l=OP) == ALIAS
    assert fstep(B=1 << 20, H=1 << 20, Nq=1 << 20) == SHAPE


def bstep(dq=OP, dk=OP + 8 * GB, dv=OP + 16 * GB, lse=LP, delta=LP + 8 * GB, d=64, Nk=300):
    return ringx.lib().ringx_attn_bwd_step(QP, KP, VP, QP + 16 * GB, lse, delta, dq, dk, dv, 1, 2,
                                           100, Nk, d, 0.125, BF16, 1, 0, None)


def test_bwd_step_validation():
    assert bstep(dq=0) == NULLPTR and bstep(dk=0) == NULLPTR and bstep(delta=0) == NULLPTR
    assert bstep(Nk=0) == SHAPE and bstep(d=80) == UNSUP
    assert bstep(dq=OP + 4) == ALIGN
    assert bstep(dq=QP) == ALIAS and bstep(dk=OP) == ALIAS and bstep(dv=LP) == ALIAS


def test_gqa_validation():
    L = ringx.lib()

    def fwd_gqa(H=4, Hkv=2, q=QP, o=OP):
        return L.ringx_attn_fwd_gqa(q, KP, VP, o, LP, 1, H, Hkv, 100, 300, 64, 3, 0.125, BF16,
                                    None)

    assert fwd_gqa(Hkv=3) == SHAPE and fwd_gqa(Hkv=0) == SHAPE and fwd_gqa(Hkv=8) == SHAPE
    assert fwd_gqa(q=0) == NULLPTR and fwd_gqa(o=KP) == ALIAS

    def bwd_gqa(Hkv=2, ws=VP + 32 * GB, wsb=1 << 20):
        return L.ringx_attn_bwd_gqa(QP, KP, VP, QP + 8 * GB, QP + 16 * GB, LP, OP, OP + 8 * GB,
                                    OP + 16 * GB, 1, 4, Hkv, 100, 300, 64, 3, 0.125, BF16, 0, ws,
                                    wsb, None)

    assert bwd_gqa(Hkv=3) == SHAPE and bwd_gqa(ws=0) == WORKSPACE


def test_tokenizer_validation():
    L = ringx.lib()
    FP, TP = QP, OP

    def tok(C=4, D=64, H=64, W=64, k=4, ratio=2, cz=0, cy=0, cx=0, p=1, sigma=2.0, dt=FP32,
            field=FP, tokens=TP):
        return L.ringx_tt_tokenize(field, tokens, C, D, H, W, k, ratio, cz, cy, cx, p, sigma, dt,
                                   None)

    assert tok(field=0) == NULLPTR and tok(tokens=0) == NULLPTR
    assert tok(C=0) == SHAPE and tok(k=0) == SHAPE and tok(ratio=0) == SHAPE and tok(p=0) == SHAPE
    assert tok(ratio=3) == SHAPE                    # 64 % 3
    assert tok(k=8, p=8) == SHAPE                   # k p does not divide 32
    assert tok(cz=64) == SHAPE and tok(cx=-1) == SHAPE
    assert tok(sigma=0.0) == SHAPE and tok(sigma=float("nan")) == SHAPE
    assert tok(k=33, D=66 * 32, H=66 * 32, W=66 * 32, ratio=1) == UNSUP
    assert tok(dt=9) == UNSUP
    assert tok(tokens=TP + 4) == ALIGN
    assert tok(tokens=FP + 1024) == ALIAS
