"""One GPU's side of a RingX ring, step by step (arXiv 2507.16697 Sec. III-A).

At ring step r the GPU holds one K/V chunk, computes its local result and merges it (Eq. (5));
meanwhile the next chunk arrives in a second buffer ("Communication and computation overlap":
ping-pong buffers).  Here the chunks that other ranks would send are device tensors, and their
arrival is a device-to-device copy on a second HIP stream into two ping-pong buffers, ordered
against the compute stream with events.  All attention arithmetic is the library's:
ringx_attn_fwd_step / ringx_attn_bwd_step / ringx_lse_merge (this module only moves buffers and
orders streams).  Streams keep the default priority.

    out, lse = ring_forward(q, k_chunks, v_chunks)
    dq, dk_chunks, dv_chunks = ring_backward(q, k_chunks, v_chunks, out, dout, lse)
"""

from __future__ import annotations

from . import ringx


class _PingPong:
    """Two flat device buffers per tensor; chunk r of any length up to the longest lands in
    buffer r % 2 as a contiguous [B, H, n, d] view."""

    def __init__(self, torch, like, nmax, copy_stream):
        B, H, _, d = like.shape
        self.shape = (B, H, d)
        self.k = [torch.empty(B * H * nmax * d, dtype=like.dtype, device=like.device)
                  for _ in range(2)]
        self.v = [torch.empty_like(self.k[0]) for _ in range(2)]
        for t in self.k + self.v:
            t.record_stream(copy_stream)
        self.ready = [torch.cuda.Event() for _ in range(2)]
        self.free = [torch.cuda.Event() for _ in range(2)]
        self.used = [False, False]

    def view(self, which, slot, n):
        B, H, d = self.shape
        buf = (self.k if which == "k" else self.v)[slot]
        return buf[: B * H * n * d].view(B, H, n, d)

    def fill(self, torch, copy_stream, slot, k, v):
        """Enqueue the arrival of (k, v) into `slot` on the copy stream."""
        with torch.cuda.stream(copy_stream):
            if self.used[slot]:
                copy_stream.wait_event(self.free[slot])   # the step that read it is done
            n = k.shape[2]
            self.view("k", slot, n).copy_(k, non_blocking=True)
            self.view("v", slot, n).copy_(v, non_blocking=True)
            self.ready[slot].record(copy_stream)
        # the sources are read on the copy stream: keep their memory from being reused before
        k.record_stream(copy_stream)
        v.record_stream(copy_stream)
        self.used[slot] = True


def _start(torch, compute, overlap, like, nmax):
    """The copy stream and the ping-pong buffers.  The copy stream first waits for everything
    enqueued on the compute stream so far: the chunks may have been produced there just before the
    call, and the buffers' memory may have been freed by work still running there."""
    copy = torch.cuda.Stream() if overlap else compute
    pp = _PingPong(torch, like, nmax, copy)
    if overlap:
        copy.wait_stream(compute)
    return copy, pp


def _check_chunks(q, k_chunks, v_chunks):
    if len(k_chunks) == 0 or len(k_chunks) != len(v_chunks):
        raise ValueError("need one V chunk per K chunk, at least one")
    for k, v in zip(k_chunks, v_chunks):
        if k.shape != v.shape or k.shape[:2] != q.shape[:2] or k.shape[3] != q.shape[3]:
            raise ValueError("chunk shapes must be [B, H, n, d] matching q")
        if k.dtype != q.dtype or v.dtype != q.dtype:
            raise ValueError("chunks must have q's dtype")


def ring_forward(q, k_chunks, v_chunks, scale=None, out_dtype=None, overlap=True):
    """Attention of q over the concatenated chunks, one ring step per chunk.

    Returns (out, lse): out in out_dtype (q's dtype by default), lse fp32 natural log."""
    import torch
    _check_chunks(q, k_chunks, v_chunks)
    B, H, Nq, d = q.shape
    compute = torch.cuda.current_stream()
    copy, pp = _start(torch, compute, overlap, k_chunks[0], max(k.shape[2] for k in k_chunks))
    out_acc = torch.empty((B, H, Nq, d), dtype=torch.float32, device=q.device)
    lse_acc = torch.empty((B, H, Nq), dtype=torch.float32, device=q.device)
    pp.fill(torch, copy, 0, k_chunks[0], v_chunks[0])
    for r in range(len(k_chunks)):
        slot = r % 2
        if r + 1 < len(k_chunks):
            pp.fill(torch, copy, 1 - slot, k_chunks[r + 1], v_chunks[r + 1])
        compute.wait_event(pp.ready[slot])
        n = k_chunks[r].shape[2]
        ringx.ringx_attn_fwd_step(q, pp.view("k", slot, n), pp.view("v", slot, n), out_acc,
                                  lse_acc, first=(r == 0), scale=scale, stream=compute)
        pp.free[slot].record(compute)
    return ringx.ringx_lse_merge(out_acc[None], lse_acc[None], out_dtype=out_dtype or q.dtype,
                                 stream=compute)


def ring_backward(q, k_chunks, v_chunks, out, dout, lse, scale=None, overlap=True):
    """Gradients with the merged lse, one ring step per chunk.

    Returns (dq, dk_chunks, dv_chunks), all fp32; dk_chunks[r], dv_chunks[r] are the gradients of
    chunk r (what a ring sends back to the chunk's owner)."""
    import torch
    _check_chunks(q, k_chunks, v_chunks)
    B, H, Nq, d = q.shape
    compute = torch.cuda.current_stream()
    copy, pp = _start(torch, compute, overlap, k_chunks[0], max(k.shape[2] for k in k_chunks))
    delta = ringx.ringx_bwd_preprocess(out, dout, lse, stream=compute)
    dq = torch.empty((B, H, Nq, d), dtype=torch.float32, device=q.device)
    dks = [torch.empty(k.shape, dtype=torch.float32, device=q.device) for k in k_chunks]
    dvs = [torch.empty_like(t) for t in dks]
    pp.fill(torch, copy, 0, k_chunks[0], v_chunks[0])
    for r in range(len(k_chunks)):
        slot = r % 2
        if r + 1 < len(k_chunks):
            pp.fill(torch, copy, 1 - slot, k_chunks[r + 1], v_chunks[r + 1])
        compute.wait_event(pp.ready[slot])
        n = k_chunks[r].shape[2]
        ringx.ringx_attn_bwd_step(q, pp.view("k", slot, n), pp.view("v", slot, n), dout, lse,
                                  delta, dq, dks[r], dvs[r], accumulate_dq=(r > 0), scale=scale,
                                  stream=compute)
        pp.free[slot].record(compute)
    return dq, dks, dvs
