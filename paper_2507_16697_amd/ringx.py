"""Thin Python binding of libringx (C ABI in include/ringx.h).

Argument marshalling only: every step of the attention runs in the library's HIP kernels.  torch
supplies device memory and the current HIP stream.  Function names follow the C entry points.

    out, lse = ringx_attn_fwd(q, k, v, R)                     # q,k,v: [B,H,N,d] cuda tensors
    part_out, part_lse = ringx_attn_fwd_partials(q, k, v, R)
    out, lse = ringx_lse_merge(part_out, part_lse, out_dtype=torch.bfloat16)
    dq, dk, dv = ringx_attn_bwd(q, k, v, out, dout, lse, R)
    ringx_attn_fwd_step(q, k_r, v_r, out_acc, lse_acc, first=(r == 0))   # one ring step
    ringx_attn_bwd_step(q, k_r, v_r, dout, lse, delta, dq_acc, dk_r, dv_r, accumulate_dq=(r > 0))

The library must be built (``python -m paper_2507_16697_amd.build``); loading fails loudly if it
is missing -- there is no fallback implementation.
"""

from __future__ import annotations

import ctypes
import math
import os

# RINGX_LIB names another build of the same library (e.g. the host-sanitizer build of the tests)
LIB_PATH = os.environ.get("RINGX_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                       "libringx.so")

RINGX_FP32 = 0
RINGX_BF16 = 1

STATUS_NAMES = {
    0: "RINGX_OK", 1: "RINGX_E_NULLPTR", 2: "RINGX_E_SHAPE", 3: "RINGX_E_CHUNKS",
    4: "RINGX_E_UNSUPPORTED", 5: "RINGX_E_ALIGN", 6: "RINGX_E_WORKSPACE", 7: "RINGX_E_HIP",
    8: "RINGX_E_ALIAS", 9: "RINGX_E_SCRATCH",
}

# rows (B * H * Nq) of the fixed device array behind ringx_attn_bwd_noalloc (RINGX_NOALLOC_MAX_ROWS)
NOALLOC_MAX_ROWS = 2097152

EXPORTED = ("ringx_attn_fwd", "ringx_attn_fwd_partials", "ringx_lse_merge", "ringx_attn_bwd",
            "ringx_bwd_preprocess", "ringx_attn_bwd_dkdv", "ringx_attn_bwd_dq",
            "ringx_attn_fwd_step", "ringx_attn_bwd_step", "ringx_attn_fwd_gqa",
            "ringx_attn_bwd_gqa", "ringx_tt_tokenize", "ringx_bwd_workspace_bytes",
            "ringx_chunk_bounds", "ringx_status_str", "ringx_attn_bwd_noalloc",
            "ringx_bwd_ds_bytes", "ringx_attn_bwd_dkdv_ds", "ringx_attn_bwd_dq_ds",
            "ringx_attn_bwd_ds", "ringx_bwd_ds_workspace_bytes")


class RingxError(RuntimeError):
    def __init__(self, fn: str, status: int, message: str):
        super().__init__(f"{fn}: {STATUS_NAMES.get(status, status)} ({message})")
        self.status = status


_lib = None

_P = ctypes.c_void_p
_I = ctypes.c_int64


def lib() -> ctypes.CDLL:
    """The loaded libringx.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libringx.so not found at {LIB_PATH}; build it with "
                               "`python -m paper_2507_16697_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.ringx_attn_fwd.argtypes = [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, ctypes.c_float,
                                     ctypes.c_int, _P]
        L.ringx_attn_fwd_partials.argtypes = L.ringx_attn_fwd.argtypes
        L.ringx_lse_merge.argtypes = [_P, _P, _P, _P, _I, _I, _I, _I, _I, ctypes.c_int, _P]
        L.ringx_attn_bwd.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I,
                                     ctypes.c_float, ctypes.c_int, ctypes.c_int, _P,
                                     ctypes.c_size_t, _P]
        L.ringx_attn_bwd_noalloc.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I,
                                             _I, _I, ctypes.c_float, ctypes.c_int, ctypes.c_int,
                                             _P]
        L.ringx_bwd_preprocess.argtypes = [_P, _P, _P, _P, _I, _I, _I, _I, ctypes.c_int, _P]
        L.ringx_attn_bwd_dkdv.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I,
                                          ctypes.c_float, ctypes.c_int, ctypes.c_int, _P]
        L.ringx_attn_bwd_dq.argtypes = [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I,
                                        ctypes.c_float, ctypes.c_int, _P]
        L.ringx_attn_fwd_step.argtypes = [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, ctypes.c_float,
                                          ctypes.c_int, ctypes.c_int, _P]
        L.ringx_attn_bwd_step.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I,
                                          ctypes.c_float, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_int, _P]
        L.ringx_attn_fwd_gqa.argtypes = [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I,
                                         ctypes.c_float, ctypes.c_int, _P]
        L.ringx_attn_bwd_gqa.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I,
                                         _I, _I, ctypes.c_float, ctypes.c_int, ctypes.c_int, _P,
                                         ctypes.c_size_t, _P]
        L.ringx_tt_tokenize.argtypes = [_P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _I,
                                        ctypes.c_float, ctypes.c_int, _P]
        L.ringx_bwd_workspace_bytes.argtypes = [_I, _I, _I, _I, _I, _I, ctypes.c_int]
        L.ringx_bwd_workspace_bytes.restype = ctypes.c_size_t
        L.ringx_bwd_ds_bytes.argtypes = [_I, _I, _I, _I, _I, _I, _I]
        L.ringx_bwd_ds_bytes.restype = ctypes.c_size_t
        L.ringx_bwd_ds_workspace_bytes.argtypes = [_I, _I, _I, _I, _I, _I, _I, _I]
        L.ringx_bwd_ds_workspace_bytes.restype = ctypes.c_size_t
        L.ringx_attn_bwd_dkdv_ds.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t,
                                             _I, _I, _I, _I, _I, _I, _I, ctypes.c_float,
                                             ctypes.c_int, ctypes.c_int, _I, _I, _P]
        L.ringx_attn_bwd_dq_ds.argtypes = [_P, ctypes.c_size_t, _P, _P, _I, _I, _I, _I, _I, _I,
                                           _I, ctypes.c_float, ctypes.c_int, _I, _I, _P]
        L.ringx_attn_bwd_ds.argtypes = L.ringx_attn_bwd_gqa.argtypes
        L.ringx_chunk_bounds.argtypes = [_I, _I, _I, ctypes.POINTER(_I), ctypes.POINTER(_I)]
        L.ringx_status_str.argtypes = [ctypes.c_int]
        L.ringx_status_str.restype = ctypes.c_char_p
        for name in ("ringx_attn_fwd", "ringx_attn_fwd_partials", "ringx_lse_merge",
                     "ringx_attn_bwd", "ringx_bwd_preprocess", "ringx_attn_bwd_dkdv",
                     "ringx_attn_bwd_dq", "ringx_attn_fwd_step", "ringx_attn_bwd_step",
                     "ringx_attn_fwd_gqa", "ringx_attn_bwd_gqa", "ringx_tt_tokenize",
                     "ringx_chunk_bounds", "ringx_attn_bwd_noalloc", "ringx_attn_bwd_dkdv_ds",
                     "ringx_attn_bwd_dq_ds", "ringx_attn_bwd_ds"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def ringx_status_str(status: int) -> str:
    return lib().ringx_status_str(int(status)).decode()


def _check(fn: str, status: int):
    if status != 0:
        raise RingxError(fn, status, ringx_status_str(status))


def ringx_chunk_bounds(Nk: int, R: int, r: int) -> tuple[int, int]:
    lo, hi = _I(), _I()
    _check("ringx_chunk_bounds", lib().ringx_chunk_bounds(Nk, R, r, ctypes.byref(lo), ctypes.byref(hi)))
    return lo.value, hi.value


def ringx_bwd_workspace_bytes(B, H, Nq, Nk, d, R, dtype) -> int:
    return int(lib().ringx_bwd_workspace_bytes(B, H, Nq, Nk, d, R, int(dtype)))


def ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, d, R, kv_count) -> int:
    return int(lib().ringx_bwd_ds_bytes(H, Hkv, Nq, Nk, d, R, kv_count))


def ringx_bwd_ds_workspace_bytes(B, H, Hkv, Nq, Nk, d, R, kv_per_slab) -> int:
    return int(lib().ringx_bwd_ds_workspace_bytes(B, H, Hkv, Nq, Nk, d, R, kv_per_slab))


# ---------------------------------------------------------------------------------------------
# torch tensor helpers


def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return RINGX_BF16
    if t.dtype == torch.float32:
        return RINGX_FP32
    raise TypeError(f"unsupported dtype {t.dtype}; expected bfloat16 or float32")


def _dev(*ts):
    for t in ts:
        if not t.is_cuda:
            raise ValueError("tensors must live on the GPU")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous [B, H, N, d]")


def _expect(name, t, shape, dtype, device):
    """The kernels size every buffer from q and k: a tensor of another shape, dtype or device
    would be read or written out of bounds, so it is refused here."""
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype != dtype:
        raise TypeError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if t.device != device:
        raise ValueError(f"{name}: on {t.device}, expected {device}")


def _qkv(q, k, v, heads_kv=None):
    """Shapes of q [B,H,Nq,d] and k, v [B,Hkv,Nk,d] (Hkv = H unless heads_kv is allowed to
    differ); returns (B, H, Hkv, Nq, Nk, d)."""
    if q.dim() != 4 or k.dim() != 4:
        raise ValueError("q, k and v must be 4-D [B, H, N, d]")
    _dtype_code(q)
    B, H, Nq, d = q.shape
    Hkv, Nk = k.shape[1], k.shape[2]
    if heads_kv is None and Hkv != H:
        raise ValueError(f"k has {Hkv} heads, q has {H}")
    _expect("k", k, (B, Hkv, Nk, d), q.dtype, q.device)
    _expect("v", v, (B, Hkv, Nk, d), q.dtype, q.device)
    return B, H, Hkv, Nq, Nk, d


def _check_grad_inputs(q, dout, lse, delta):
    torch = _torch()
    B, H, Nq, _ = q.shape
    _expect("dout", dout, q.shape, q.dtype, q.device)
    _expect("lse", lse, (B, H, Nq), torch.float32, q.device)
    _expect("delta", delta, (2, B, H, Nq), torch.float32, q.device)


def _stream(stream):
    torch = _torch()
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if hasattr(stream, "cuda_stream"):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _scale(scale, d):
    return float(1.0 / math.sqrt(d)) if scale is None else float(scale)


def ringx_attn_fwd(q, k, v, R: int, scale=None, out=None, lse=None, stream=None):
    """Merged ring-chunked forward.  Returns (out [B,H,Nq,d] in q's dtype, lse [B,H,Nq] fp32)."""
    torch = _torch()
    _dev(q, k, v)
    B, H, _, Nq, Nk, d = _qkv(q, k, v)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((B, H, Nq), dtype=torch.float32, device=q.device)
    _dev(out, lse)
    _expect("out", out, q.shape, q.dtype, q.device)
    _expect("lse", lse, (B, H, Nq), torch.float32, q.device)
    st = lib().ringx_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                              lse.data_ptr(), B, H, Nq, Nk, d, R, _scale(scale, d),
                              _dtype_code(q), _stream(stream))
    _check("ringx_attn_fwd", st)
    return out, lse


def ringx_attn_fwd_partials(q, k, v, R: int, scale=None, part_out=None, part_lse=None,
                            stream=None):
    """Per-chunk local results: (part_out [R,B,H,Nq,d] fp32, part_lse [R,B,H,Nq] fp32)."""
    torch = _torch()
    _dev(q, k, v)
    B, H, _, Nq, Nk, d = _qkv(q, k, v)
    if part_out is None:
        part_out = torch.empty((R, B, H, Nq, d), dtype=torch.float32, device=q.device)
    if part_lse is None:
        part_lse = torch.empty((R, B, H, Nq), dtype=torch.float32, device=q.device)
    _dev(part_out, part_lse)
    _expect("part_out", part_out, (R, B, H, Nq, d), torch.float32, q.device)
    _expect("part_lse", part_lse, (R, B, H, Nq), torch.float32, q.device)
    st = lib().ringx_attn_fwd_partials(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                       part_out.data_ptr(), part_lse.data_ptr(), B, H, Nq, Nk, d,
                                       R, _scale(scale, d), _dtype_code(q), _stream(stream))
    _check("ringx_attn_fwd_partials", st)
    return part_out, part_lse


def ringx_lse_merge(part_out, part_lse, out_dtype=None, out=None, lse=None, stream=None):
    """Eq. (5) merge of R partials.  Returns (out [B,H,Nq,d] in out_dtype, lse [B,H,Nq] fp32)."""
    torch = _torch()
    _dev(part_out, part_lse)
    if part_out.dim() != 5:
        raise ValueError("part_out must be 5-D [R, B, H, Nq, d]")
    R, B, H, Nq, d = part_out.shape
    dev = part_out.device
    _expect("part_out", part_out, (R, B, H, Nq, d), torch.float32, dev)
    _expect("part_lse", part_lse, (R, B, H, Nq), torch.float32, dev)
    if out is None:
        out = torch.empty((B, H, Nq, d), dtype=out_dtype or torch.float32, device=dev)
    if lse is None:
        lse = torch.empty((B, H, Nq), dtype=torch.float32, device=dev)
    _dev(out, lse)
    _dtype_code(out)
    _expect("out", out, (B, H, Nq, d), out.dtype, dev)
    _expect("lse", lse, (B, H, Nq), torch.float32, dev)
    st = lib().ringx_lse_merge(part_out.data_ptr(), part_lse.data_ptr(), out.data_ptr(),
                               lse.data_ptr(), R, B, H, Nq, d, _dtype_code(out), _stream(stream))
    _check("ringx_lse_merge", st)
    return out, lse


def ringx_attn_bwd(q, k, v, out, dout, lse, R: int, scale=None, dq=None, dk=None, dv=None,
                   accumulate_dkv=False, workspace=None, stream=None):
    """Recompute backward.  Returns fp32 (dq, dk, dv); dk/dv are added to when accumulate_dkv."""
    torch = _torch()
    _dev(q, k, v, out, dout, lse)
    B, H, _, Nq, Nk, d = _qkv(q, k, v)
    _expect("out", out, q.shape, q.dtype, q.device)
    _expect("dout", dout, q.shape, q.dtype, q.device)
    _expect("lse", lse, (B, H, Nq), torch.float32, q.device)
    f32 = dict(dtype=torch.float32, device=q.device)
    if dq is None:
        dq = torch.empty((B, H, Nq, d), **f32)
    if dk is None:
        dk = torch.zeros((B, H, Nk, d), **f32) if accumulate_dkv else torch.empty((B, H, Nk, d), **f32)
    if dv is None:
        dv = torch.zeros((B, H, Nk, d), **f32) if accumulate_dkv else torch.empty((B, H, Nk, d), **f32)
    code = _dtype_code(q)
    need = ringx_bwd_workspace_bytes(B, H, Nq, Nk, d, R, code)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    _dev(dq, dk, dv, workspace)
    _expect("dq", dq, (B, H, Nq, d), torch.float32, q.device)
    _expect("dk", dk, (B, H, Nk, d), torch.float32, q.device)
    _expect("dv", dv, (B, H, Nk, d), torch.float32, q.device)
    if workspace.device != q.device:
        raise ValueError(f"workspace: on {workspace.device}, expected {q.device}")
    st = lib().ringx_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                              dout.data_ptr(), lse.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                              dv.data_ptr(), B, H, Nq, Nk, d, R, _scale(scale, d), code,
                              1 if accumulate_dkv else 0, workspace.data_ptr(),
                              workspace.numel() * workspace.element_size(), _stream(stream))
    _check("ringx_attn_bwd", st)
    return dq, dk, dv


def ringx_attn_bwd_noalloc(q, k, v, out, dout, lse, R: int, dq, dk, dv, scale=None,
                           accumulate_dkv=False, stream=None):
    """ringx_attn_bwd for callers that cannot allocate: the caller passes the fp32 outputs dq, dk,
    dv, and D lives in the library's fixed device array (B * H * Nq <= NOALLOC_MAX_ROWS).  Calls
    that overlap in time on one GPU race on that array.  Returns (dq, dk, dv)."""
    torch = _torch()
    _dev(q, k, v, out, dout, lse, dq, dk, dv)
    B, H, _, Nq, Nk, d = _qkv(q, k, v)
    _expect("out", out, q.shape, q.dtype, q.device)
    _expect("dout", dout, q.shape, q.dtype, q.device)
    _expect("lse", lse, (B, H, Nq), torch.float32, q.device)
    _expect("dq", dq, (B, H, Nq, d), torch.float32, q.device)
    _expect("dk", dk, (B, H, Nk, d), torch.float32, q.device)
    _expect("dv", dv, (B, H, Nk, d), torch.float32, q.device)
    st = lib().ringx_attn_bwd_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                      dout.data_ptr(), lse.data_ptr(), dq.data_ptr(),
                                      dk.data_ptr(), dv.data_ptr(), B, H, Nq, Nk, d, R,
                                      _scale(scale, d), _dtype_code(q),
                                      1 if accumulate_dkv else 0, _stream(stream))
    _check("ringx_attn_bwd_noalloc", st)
    return dq, dk, dv


def ringx_bwd_preprocess(out, dout, lse, delta=None, stream=None):
    """Per-row statistics delta [2,B,H,Nq] fp32: delta[0] = rowsum(dout * out),
    delta[1] = -lse * log2(e)."""
    torch = _torch()
    _dev(out, dout, lse)
    if out.dim() != 4:
        raise ValueError("out must be 4-D [B, H, Nq, d]")
    _dtype_code(out)
    B, H, Nq, d = out.shape
    _expect("dout", dout, out.shape, out.dtype, out.device)
    _expect("lse", lse, (B, H, Nq), torch.float32, out.device)
    if delta is None:
        delta = torch.empty((2, B, H, Nq), dtype=torch.float32, device=out.device)
    _dev(delta)
    _expect("delta", delta, (2, B, H, Nq), torch.float32, out.device)
    st = lib().ringx_bwd_preprocess(out.data_ptr(), dout.data_ptr(), lse.data_ptr(),
                                    delta.data_ptr(), B, H, Nq, d, _dtype_code(out),
                                    _stream(stream))
    _check("ringx_bwd_preprocess", st)
    return delta


def ringx_attn_bwd_dkdv(q, k, v, dout, lse, delta, R: int, scale=None, dk=None, dv=None,
                        accumulate_dkv=False, stream=None):
    """Key/value gradients of every chunk.  Returns fp32 (dk, dv)."""
    torch = _torch()
    _dev(q, k, v, dout, lse, delta)
    B, H, _, Nq, Nk, d = _qkv(q, k, v)
    _check_grad_inputs(q, dout, lse, delta)
    f32 = dict(dtype=torch.float32, device=q.device)
    if dk is None:
        dk = torch.zeros((B, H, Nk, d), **f32)
    if dv is None:
        dv = torch.zeros((B, H, Nk, d), **f32)
    _dev(dk, dv)
    _expect("dk", dk, (B, H, Nk, d), torch.float32, q.device)
    _expect("dv", dv, (B, H, Nk, d), torch.float32, q.device)
    st = lib().ringx_attn_bwd_dkdv(q.data_ptr(), k.data_ptr(), v.data_ptr(), dout.data_ptr(),
                                   lse.data_ptr(), delta.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                   B, H, Nq, Nk, d, R, _scale(scale, d), _dtype_code(q),
                                   1 if accumulate_dkv else 0, _stream(stream))
    _check("ringx_attn_bwd_dkdv", st)
    return dk, dv


def ringx_attn_bwd_dq(q, k, v, dout, lse, delta, R: int, scale=None, dq=None, stream=None):
    """Query gradient accumulated over every chunk.  Returns fp32 dq."""
    torch = _torch()
    _dev(q, k, v, dout, lse, delta)
    B, H, _, Nq, Nk, d = _qkv(q, k, v)
    _check_grad_inputs(q, dout, lse, delta)
    if dq is None:
        dq = torch.empty((B, H, Nq, d), dtype=torch.float32, device=q.device)
    _dev(dq)
    _expect("dq", dq, (B, H, Nq, d), torch.float32, q.device)
    st = lib().ringx_attn_bwd_dq(q.data_ptr(), k.data_ptr(), v.data_ptr(), dout.data_ptr(),
                                 lse.data_ptr(), delta.data_ptr(), dq.data_ptr(), B, H, Nq, Nk, d,
                                 R, _scale(scale, d), _dtype_code(q), _stream(stream))
    _check("ringx_attn_bwd_dq", st)
    return dq


def ringx_attn_fwd_step(q, k, v, out_acc, lse_acc, first: bool, scale=None, stream=None):
    """One ring step: merge q's attention over the chunk k, v into the running fp32
    (out_acc [B,H,Nq,d], lse_acc [B,H,Nq]) in place (Eq. (5)); first=True starts it."""
    torch = _torch()
    _dev(q, k, v, out_acc, lse_acc)
    B, H, _, Nq, Nk, d = _qkv(q, k, v)
    _expect("out_acc", out_acc, (B, H, Nq, d), torch.float32, q.device)
    _expect("lse_acc", lse_acc, (B, H, Nq), torch.float32, q.device)
    st = lib().ringx_attn_fwd_step(q.data_ptr(), k.data_ptr(), v.data_ptr(), out_acc.data_ptr(),
                                   lse_acc.data_ptr(), B, H, Nq, Nk, d, _scale(scale, d),
                                   _dtype_code(q), 1 if first else 0, _stream(stream))
    _check("ringx_attn_fwd_step", st)
    return out_acc, lse_acc


def ringx_attn_bwd_step(q, k, v, dout, lse, delta, dq_acc, dk, dv, accumulate_dq: bool,
                        accumulate_dkv: bool = False, scale=None, stream=None):
    """One ring step of the backward for the chunk k, v: its dk, dv (fp32, written or added to)
    and its contribution to dq_acc (added to, or written when accumulate_dq is False)."""
    torch = _torch()
    _dev(q, k, v, dout, lse, delta, dq_acc, dk, dv)
    B, H, _, Nq, Nk, d = _qkv(q, k, v)
    _check_grad_inputs(q, dout, lse, delta)
    _expect("dq_acc", dq_acc, (B, H, Nq, d), torch.float32, q.device)
    _expect("dk", dk, (B, H, Nk, d), torch.float32, q.device)
    _expect("dv", dv, (B, H, Nk, d), torch.float32, q.device)
    st = lib().ringx_attn_bwd_step(q.data_ptr(), k.data_ptr(), v.data_ptr(), dout.data_ptr(),
                                   lse.data_ptr(), delta.data_ptr(), dq_acc.data_ptr(),
                                   dk.data_ptr(), dv.data_ptr(), B, H, Nq, Nk, d, _scale(scale, d),
                                   _dtype_code(q), 1 if accumulate_dq else 0,
                                   1 if accumulate_dkv else 0, _stream(stream))
    _check("ringx_attn_bwd_step", st)
    return dq_acc, dk, dv


def ringx_attn_fwd_gqa(q, k, v, R: int, scale=None, out=None, lse=None, stream=None):
    """Grouped-query attention: q [B,H,Nq,d], k, v [B,Hkv,Nk,d] with Hkv dividing H."""
    torch = _torch()
    _dev(q, k, v)
    B, H, Hkv, Nq, Nk, d = _qkv(q, k, v, heads_kv=True)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((B, H, Nq), dtype=torch.float32, device=q.device)
    _dev(out, lse)
    _expect("out", out, q.shape, q.dtype, q.device)
    _expect("lse", lse, (B, H, Nq), torch.float32, q.device)
    st = lib().ringx_attn_fwd_gqa(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                  lse.data_ptr(), B, H, Hkv, Nq, Nk, d, R, _scale(scale, d),
                                  _dtype_code(q), _stream(stream))
    _check("ringx_attn_fwd_gqa", st)
    return out, lse


def ringx_attn_bwd_gqa(q, k, v, out, dout, lse, R: int, scale=None, dq=None, dk=None, dv=None,
                       accumulate_dkv=False, stream=None):
    """Backward of ringx_attn_fwd_gqa: fp32 dq [B,H,Nq,d], dk, dv [B,Hkv,Nk,d] (group sums)."""
    torch = _torch()
    _dev(q, k, v, out, dout, lse)
    B, H, Hkv, Nq, Nk, d = _qkv(q, k, v, heads_kv=True)
    _expect("out", out, q.shape, q.dtype, q.device)
    _expect("dout", dout, q.shape, q.dtype, q.device)
    _expect("lse", lse, (B, H, Nq), torch.float32, q.device)
    f32 = dict(dtype=torch.float32, device=q.device)
    dq = torch.empty((B, H, Nq, d), **f32) if dq is None else dq
    dk = torch.zeros((B, Hkv, Nk, d), **f32) if dk is None else dk
    dv = torch.zeros((B, Hkv, Nk, d), **f32) if dv is None else dv
    _dev(dq, dk, dv)
    _expect("dq", dq, (B, H, Nq, d), torch.float32, q.device)
    _expect("dk", dk, (B, Hkv, Nk, d), torch.float32, q.device)
    _expect("dv", dv, (B, Hkv, Nk, d), torch.float32, q.device)
    nbytes = ringx_bwd_workspace_bytes(B, H, Nq, Nk, d, R, _dtype_code(q))
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=q.device)
    st = lib().ringx_attn_bwd_gqa(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                  dout.data_ptr(), lse.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                                  dv.data_ptr(), B, H, Hkv, Nq, Nk, d, R, _scale(scale, d),
                                  _dtype_code(q), 1 if accumulate_dkv else 0, ws.data_ptr(),
                                  ws.numel(), _stream(stream))
    _check("ringx_attn_bwd_gqa", st)
    return dq, dk, dv


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def ringx_attn_bwd_dkdv_ds(q, k, v, dout, lse, delta, R: int, ds, kv_begin: int, kv_count: int,
                           scale=None, dk=None, dv=None, accumulate_dkv=False, stream=None):
    """dK/dV of K/V heads [kv_begin, kv_begin + kv_count) (of B * Hkv), writing their query
    heads' dS into the uint8 device buffer ds (ringx_bwd_ds_bytes(...) bytes).  Returns fp32
    (dk, dv) [B,Hkv,Nk,d]; rows of other heads are not touched."""
    torch = _torch()
    _dev(q, k, v, dout, lse, delta, ds)
    B, H, Hkv, Nq, Nk, d = _qkv(q, k, v, heads_kv=True)
    _check_grad_inputs(q, dout, lse, delta)
    f32 = dict(dtype=torch.float32, device=q.device)
    dk = torch.zeros((B, Hkv, Nk, d), **f32) if dk is None else dk
    dv = torch.zeros((B, Hkv, Nk, d), **f32) if dv is None else dv
    _dev(dk, dv)
    _expect("dk", dk, (B, Hkv, Nk, d), torch.float32, q.device)
    _expect("dv", dv, (B, Hkv, Nk, d), torch.float32, q.device)
    if ds.device != q.device:
        raise ValueError(f"ds: on {ds.device}, expected {q.device}")
    st = lib().ringx_attn_bwd_dkdv_ds(q.data_ptr(), k.data_ptr(), v.data_ptr(), dout.data_ptr(),
                                      lse.data_ptr(), delta.data_ptr(), dk.data_ptr(),
                                      dv.data_ptr(), ds.data_ptr(), _nbytes(ds), B, H, Hkv, Nq,
                                      Nk, d, R, _scale(scale, d), _dtype_code(q),
                                      1 if accumulate_dkv else 0, kv_begin, kv_count,
                                      _stream(stream))
    _check("ringx_attn_bwd_dkdv_ds", st)
    return dk, dv


def ringx_attn_bwd_dq_ds(ds, k, q_shape, R: int, kv_begin: int, kv_count: int, scale=None,
                         dq=None, stream=None):
    """dQ of the query heads of K/V heads [kv_begin, kv_begin + kv_count) from ds as written by
    ringx_attn_bwd_dkdv_ds.  q_shape = (B, H, Nq, d).  Returns fp32 dq [B,H,Nq,d] (rows of other
    heads are not touched)."""
    torch = _torch()
    _dev(ds, k)
    B, H, Nq, d = (int(x) for x in q_shape)
    if k.dim() != 4 or k.shape[0] != B or k.shape[3] != d:
        raise ValueError(f"k: shape {tuple(k.shape)} does not match q_shape {tuple(q_shape)}")
    Hkv, Nk = int(k.shape[1]), int(k.shape[2])
    if dq is None:
        dq = torch.empty((B, H, Nq, d), dtype=torch.float32, device=k.device)
    _dev(dq)
    _expect("dq", dq, (B, H, Nq, d), torch.float32, k.device)
    if ds.device != k.device:
        raise ValueError(f"ds: on {ds.device}, expected {k.device}")
    st = lib().ringx_attn_bwd_dq_ds(ds.data_ptr(), _nbytes(ds), k.data_ptr(), dq.data_ptr(), B, H,
                                    Hkv, Nq, Nk, d, R, _scale(scale, d), _dtype_code(k),
                                    kv_begin, kv_count, _stream(stream))
    _check("ringx_attn_bwd_dq_ds", st)
    return dq


def ringx_attn_bwd_ds(q, k, v, out, dout, lse, R: int, scale=None, dq=None, dk=None, dv=None,
                      accumulate_dkv=False, workspace=None, kv_per_slab=2, stream=None):
    """The backward through stored dS (bf16, d = 128): fp32 (dq, dk, dv), dk/dv [B,Hkv,Nk,d].
    Without a workspace, one of ringx_bwd_ds_workspace_bytes(..., kv_per_slab) bytes is
    allocated (slabs of kv_per_slab K/V heads, fewer if B * Hkv is smaller)."""
    torch = _torch()
    _dev(q, k, v, out, dout, lse)
    B, H, Hkv, Nq, Nk, d = _qkv(q, k, v, heads_kv=True)
    _expect("out", out, q.shape, q.dtype, q.device)
    _expect("dout", dout, q.shape, q.dtype, q.device)
    _expect("lse", lse, (B, H, Nq), torch.float32, q.device)
    f32 = dict(dtype=torch.float32, device=q.device)
    dq = torch.empty((B, H, Nq, d), **f32) if dq is None else dq
    dk = torch.zeros((B, Hkv, Nk, d), **f32) if dk is None else dk
    dv = torch.zeros((B, Hkv, Nk, d), **f32) if dv is None else dv
    _dev(dq, dk, dv)
    _expect("dq", dq, (B, H, Nq, d), torch.float32, q.device)
    _expect("dk", dk, (B, Hkv, Nk, d), torch.float32, q.device)
    _expect("dv", dv, (B, Hkv, Nk, d), torch.float32, q.device)
    if workspace is None:
        nbytes = ringx_bwd_ds_workspace_bytes(B, H, Hkv, Nq, Nk, d, R,
                                              max(1, min(int(kv_per_slab), B * Hkv)))
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=q.device)
    _dev(workspace)
    if workspace.device != q.device:
        raise ValueError(f"workspace: on {workspace.device}, expected {q.device}")
    st = lib().ringx_attn_bwd_ds(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                 dout.data_ptr(), lse.data_ptr(), dq.data_ptr(), dk.data_ptr(),
                                 dv.data_ptr(), B, H, Hkv, Nq, Nk, d, R, _scale(scale, d),
                                 _dtype_code(q), 1 if accumulate_dkv else 0, workspace.data_ptr(),
                                 _nbytes(workspace), _stream(stream))
    _check("ringx_attn_bwd_ds", st)
    return dq, dk, dv


def ringx_tt_tokenize(field, k: int, ratio: int, centre, p: int, sigma=None, out_dtype=None,
                      tokens=None, stream=None):
    """One fidelity mode of the multi-fidelity tokenizer: field [C, D, H, W] fp32 on the GPU ->
    tokens [L, C p^3] (fp32 by default).  sigma defaults to k / 2."""
    torch = _torch()
    _dev(field)
    if field.dtype != torch.float32:
        raise ValueError("field must be fp32")
    C, D, H, W = field.shape
    out_dtype = out_dtype or torch.float32
    L = (D // (ratio * k * p)) * (H // (ratio * k * p)) * (W // (ratio * k * p))
    if tokens is None:
        tokens = torch.empty((L, C * p ** 3), dtype=out_dtype, device=field.device)
    _dev(tokens)
    _dtype_code(tokens)
    _expect("tokens", tokens, (L, C * p ** 3), tokens.dtype, field.device)
    sigma = float(k) / 2.0 if sigma is None else float(sigma)
    cz, cy, cx = (int(c) for c in centre)
    st = lib().ringx_tt_tokenize(field.data_ptr(), tokens.data_ptr(), C, D, H, W, k, ratio, cz,
                                 cy, cx, p, sigma, _dtype_code(tokens), _stream(stream))
    _check("ringx_tt_tokenize", st)
    return tokens
