"""Every entry point writes inside its output buffers and all of them, and its results depend
neither on where the buffers sit nor on the run (needs an MI355X).

Each output is the middle of a larger allocation whose 4 KiB bands on both sides, and the output
itself, start out holding a NaN with a fixed payload.  After the call the bands must hold that
pattern bit for bit (nothing was written out of bounds) and no element of the output may still
hold it (nothing was left unwritten).  The results must equal, bit for bit, those of a second call
on plainly allocated buffers (no race, no dependence on placement).  Shapes are ragged: query and
key lengths that fill no tile, chunks of unequal length, several heads and batches, grouped query
heads, and the fp32 path at a head size the bf16 kernels do not take.
"""

import numpy as np
import pytest
import torch

from paper_2507_16697_amd import ringx

from parity_util import random_case, to_device

pytestmark = pytest.mark.gpu

PAD_BYTES = 4096
# NaN bit patterns no kernel produces: quiet NaNs with a payload
_SENTINEL = {torch.float32: (torch.int32, 0x7FC0DEAD), torch.bfloat16: (torch.int16, 0x7FDE)}


class Guarded:
    """A tensor of `shape` in the middle of a larger buffer; bands and tensor start as sentinel
    NaNs, or the tensor as `fill` (outputs that are added to)."""

    def __init__(self, shape, dtype, fill=None):
        itype, self.pattern = _SENTINEL[dtype]
        self.n = int(np.prod(shape))
        self.pad = PAD_BYTES // torch.empty((), dtype=dtype).element_size()
        self.raw = torch.full((self.n + 2 * self.pad,), self.pattern, dtype=itype, device="cuda")
        self.t = self.raw[self.pad:self.pad + self.n].view(dtype).view(shape)
        if fill is not None:
            self.t.fill_(fill)

    def check(self, name, written=True):
        torch.cuda.synchronize()
        lo, hi = self.raw[:self.pad], self.raw[self.pad + self.n:]
        assert bool((lo == self.pattern).all()), f"{name}: write below the buffer"
        assert bool((hi == self.pattern).all()), f"{name}: write past the buffer"
        if written:
            body = self.raw[self.pad:self.pad + self.n]
            missed = int((body == self.pattern).sum())
            assert missed == 0, f"{name}: {missed} elements not written"


def _same(name, got, ref):
    assert got.shape == ref.shape and got.dtype == ref.dtype, name
    assert torch.equal(got, ref), f"{name}: differs from the plainly allocated run"


CASES = [("bf16", 64), ("bf16", 128), ("fp32", 40)]


@pytest.mark.parametrize("store,d", CASES)
def test_forward_entry_points(store, d):
    B, H, Nq, Nk, R = 2, 3, 203, 517, 3
    t, _ = random_case(61, B, H, Nq, Nk, d, store=store)
    g = {k: to_device(v, store) for k, v in t.items()}
    q, k, v = g["q"], g["k"], g["v"]
    dt = q.dtype
    f32 = torch.float32

    ref_o, ref_l = ringx.ringx_attn_fwd(q, k, v, R)
    o, l = Guarded((B, H, Nq, d), dt), Guarded((B, H, Nq), f32)
    ringx.ringx_attn_fwd(q, k, v, R, out=o.t, lse=l.t)
    o.check("fwd out"), l.check("fwd lse")
    _same("fwd out", o.t, ref_o), _same("fwd lse", l.t, ref_l)

    ref_po, ref_pl = ringx.ringx_attn_fwd_partials(q, k, v, R)
    po, pl = Guarded((R, B, H, Nq, d), f32), Guarded((R, B, H, Nq), f32)
    ringx.ringx_attn_fwd_partials(q, k, v, R, part_out=po.t, part_lse=pl.t)
    po.check("partials out"), pl.check("partials lse")
    _same("partials out", po.t, ref_po), _same("partials lse", pl.t, ref_pl)

    for odt in (dt, f32):
        ref_mo, ref_ml = ringx.ringx_lse_merge(ref_po, ref_pl, out_dtype=odt)
        mo, ml = Guarded((B, H, Nq, d), odt), Guarded((B, H, Nq), f32)
        ringx.ringx_lse_merge(ref_po, ref_pl, out=mo.t, lse=ml.t)
        mo.check(f"merge out {odt}"), ml.check("merge lse")
        _same(f"merge out {odt}", mo.t, ref_mo), _same("merge lse", ml.t, ref_ml)

    # ring steps over chunks of unequal length: the first step overwrites, the others merge
    bounds = [(0, 100), (100, 101), (101, Nk)]
    ks = [k[:, :, a:b].contiguous() for a, b in bounds]
    vs = [v[:, :, a:b].contiguous() for a, b in bounds]
    ref_ao = torch.empty((B, H, Nq, d), dtype=f32, device="cuda")
    ref_al = torch.empty((B, H, Nq), dtype=f32, device="cuda")
    ao, al = Guarded((B, H, Nq, d), f32), Guarded((B, H, Nq), f32)
    for r in range(len(bounds)):
        ringx.ringx_attn_fwd_step(q, ks[r], vs[r], ref_ao, ref_al, first=(r == 0))
        ringx.ringx_attn_fwd_step(q, ks[r], vs[r], ao.t, al.t, first=(r == 0))
        ao.check(f"step {r} out_acc"), al.check(f"step {r} lse_acc")
    _same("step out_acc", ao.t, ref_ao), _same("step lse_acc", al.t, ref_al)

    # grouped query heads: 3 query heads share each K/V head
    kg, vg = k[:, :1].contiguous(), v[:, :1].contiguous()
    ref_go, ref_gl = ringx.ringx_attn_fwd_gqa(q, kg, vg, R)
    go, gl = Guarded((B, H, Nq, d), dt), Guarded((B, H, Nq), f32)
    ringx.ringx_attn_fwd_gqa(q, kg, vg, R, out=go.t, lse=gl.t)
    go.check("gqa out"), gl.check("gqa lse")
    _same("gqa out", go.t, ref_go), _same("gqa lse", gl.t, ref_gl)


@pytest.mark.parametrize("store,d", CASES)
def test_backward_entry_points(store, d):
    B, H, Nq, Nk, R = 2, 3, 203, 517, 3
    t, _ = random_case(62, B, H, Nq, Nk, d, store=store)
    g = {k: to_device(v, store) for k, v in t.items()}
    q, k, v, do = g["q"], g["k"], g["v"], g["do"]
    f32 = torch.float32
    out, lse = ringx.ringx_attn_fwd(q, k, v, R)

    ref_delta = ringx.ringx_bwd_preprocess(out, do, lse)
    delta = Guarded((2, B, H, Nq), f32)
    ringx.ringx_bwd_preprocess(out, do, lse, delta=delta.t)
    delta.check("delta")
    _same("delta", delta.t, ref_delta)

    ref_dk, ref_dv = ringx.ringx_attn_bwd_dkdv(q, k, v, do, lse, ref_delta, R)
    dk, dv = Guarded((B, H, Nk, d), f32), Guarded((B, H, Nk, d), f32)
    ringx.ringx_attn_bwd_dkdv(q, k, v, do, lse, ref_delta, R, dk=dk.t, dv=dv.t)
    dk.check("dkdv dk"), dv.check("dkdv dv")
    _same("dkdv dk", dk.t, ref_dk), _same("dkdv dv", dv.t, ref_dv)

    # accumulate_dkv adds into the caller's buffers: started at zero it gives the same values
    dka, dva = Guarded((B, H, Nk, d), f32, fill=0.0), Guarded((B, H, Nk, d), f32, fill=0.0)
    ringx.ringx_attn_bwd_dkdv(q, k, v, do, lse, ref_delta, R, dk=dka.t, dv=dva.t,
                              accumulate_dkv=True)
    dka.check("dkdv dk (accumulate)"), dva.check("dkdv dv (accumulate)")
    assert torch.equal(dka.t, ref_dk) and torch.equal(dva.t, ref_dv)

    ref_dq = ringx.ringx_attn_bwd_dq(q, k, v, do, lse, ref_delta, R)
    dq = Guarded((B, H, Nq, d), f32)
    ringx.ringx_attn_bwd_dq(q, k, v, do, lse, ref_delta, R, dq=dq.t)
    dq.check("dq")
    _same("dq", dq.t, ref_dq)

    # the one-call backward, with its workspace in the middle of a banded byte buffer
    need = ringx.ringx_bwd_workspace_bytes(B, H, Nq, Nk, d, R, ringx._dtype_code(q))
    wraw = torch.full((need + 2 * PAD_BYTES,), 0xA5, dtype=torch.uint8, device="cuda")
    ws = wraw[PAD_BYTES:PAD_BYTES + need]
    bq, bk, bv = (Guarded((B, H, Nq, d), f32), Guarded((B, H, Nk, d), f32),
                  Guarded((B, H, Nk, d), f32))
    ringx.ringx_attn_bwd(q, k, v, out, do, lse, R, dq=bq.t, dk=bk.t, dv=bv.t, workspace=ws)
    bq.check("bwd dq"), bk.check("bwd dk"), bv.check("bwd dv")
    torch.cuda.synchronize()
    assert bool((wraw[:PAD_BYTES] == 0xA5).all()) and bool((wraw[PAD_BYTES + need:] == 0xA5).all())
    _same("bwd dq", bq.t, ref_dq), _same("bwd dk", bk.t, ref_dk), _same("bwd dv", bv.t, ref_dv)

    # ring steps: the first overwrites dq, the others add to it; each chunk's dk, dv written
    bounds = [(0, 100), (100, 101), (101, Nk)]
    sq = Guarded((B, H, Nq, d), f32)
    ref_sq = torch.empty((B, H, Nq, d), dtype=f32, device="cuda")
    for r, (a, b) in enumerate(bounds):
        kr, vr = k[:, :, a:b].contiguous(), v[:, :, a:b].contiguous()
        sk, sv = Guarded((B, H, b - a, d), f32), Guarded((B, H, b - a, d), f32)
        rk = torch.empty((B, H, b - a, d), dtype=f32, device="cuda")
        rv = torch.empty_like(rk)
        ringx.ringx_attn_bwd_step(q, kr, vr, do, lse, ref_delta, ref_sq, rk, rv,
                                  accumulate_dq=(r > 0))
        ringx.ringx_attn_bwd_step(q, kr, vr, do, lse, ref_delta, sq.t, sk.t, sv.t,
                                  accumulate_dq=(r > 0))
        sq.check(f"step {r} dq"), sk.check(f"step {r} dk"), sv.check(f"step {r} dv")
        _same(f"step {r} dk", sk.t, rk), _same(f"step {r} dv", sv.t, rv)
    _same("step dq", sq.t, ref_sq)

    # grouped query heads: dk, dv are sums over the 3 query heads of each K/V head
    kg, vg = k[:, :1].contiguous(), v[:, :1].contiguous()
    go, gl = ringx.ringx_attn_fwd_gqa(q, kg, vg, R)
    ref_gq, ref_gk, ref_gv = ringx.ringx_attn_bwd_gqa(q, kg, vg, go, do, gl, R)
    gq, gk, gv = (Guarded((B, H, Nq, d), f32), Guarded((B, 1, Nk, d), f32),
                  Guarded((B, 1, Nk, d), f32))
    ringx.ringx_attn_bwd_gqa(q, kg, vg, go, do, gl, R, dq=gq.t, dk=gk.t, dv=gv.t)
    gq.check("gqa dq"), gk.check("gqa dk"), gv.check("gqa dv")
    _same("gqa dq", gq.t, ref_gq), _same("gqa dk", gk.t, ref_gk), _same("gqa dv", gv.t, ref_gv)


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_tokenizer_entry_point(out_dtype):
    C, k, ratio, p = 3, 4, 2, 2
    D, Hh, W = 2 * ratio * k * p, ratio * k * p, 3 * ratio * k * p
    f = torch.from_numpy(np.random.default_rng(63).standard_normal((C, D, Hh, W))
                         .astype(np.float32)).cuda()
    centre = (5, 0, 17)
    ref = ringx.ringx_tt_tokenize(f, k, ratio, centre, p, out_dtype=out_dtype)
    tok = Guarded(tuple(ref.shape), out_dtype)
    ringx.ringx_tt_tokenize(f, k, ratio, centre, p, tokens=tok.t)
    tok.check("tokens")
    _same("tokens", tok.t, ref)
