"""The Python binding refuses tensors whose shape, dtype or device differ from what the kernels
will assume (they size every buffer from q and k, so such a tensor would be read or written out
of bounds).  CPU only: the shape checks are plain functions of the tensors' metadata."""

import pytest
import torch

from paper_2507_16697_amd import ringx


def _t(*shape, dtype=torch.bfloat16):
    return torch.empty(shape, dtype=dtype)


def test_qkv_shapes():
    q, k = _t(2, 4, 100, 64), _t(2, 4, 300, 64)
    assert ringx._qkv(q, k, _t(2, 4, 300, 64)) == (2, 4, 4, 100, 300, 64)
    with pytest.raises(ValueError, match="v: shape"):
        ringx._qkv(q, k, _t(2, 4, 299, 64))
    with pytest.raises(ValueError, match="k: shape"):
        ringx._qkv(q, _t(2, 4, 300, 128), _t(2, 4, 300, 128))
    with pytest.raises(TypeError, match="v: dtype"):
        ringx._qkv(q, k, _t(2, 4, 300, 64, dtype=torch.float32))
    with pytest.raises(ValueError, match="heads"):
        ringx._qkv(q, _t(2, 2, 300, 64), _t(2, 2, 300, 64))
    # grouped-query attention: fewer K/V heads are allowed there
    assert ringx._qkv(q, _t(2, 2, 300, 64), _t(2, 2, 300, 64), heads_kv=True) == \
        (2, 4, 2, 100, 300, 64)
    with pytest.raises(TypeError):
        ringx._qkv(_t(2, 4, 100, 64, dtype=torch.float16), _t(2, 4, 300, 64, dtype=torch.float16),
                   _t(2, 4, 300, 64, dtype=torch.float16))
    with pytest.raises(ValueError, match="4-D"):
        ringx._qkv(_t(4, 100, 64), k, k)


def test_expect():
    x = _t(3, 5, dtype=torch.float32)
    ringx._expect("x", x, (3, 5), torch.float32, x.device)
    with pytest.raises(ValueError, match=r"x: shape \(3, 5\), expected \(3, 6\)"):
        ringx._expect("x", x, (3, 6), torch.float32, x.device)
    with pytest.raises(TypeError, match="x: dtype"):
        ringx._expect("x", x, (3, 5), torch.bfloat16, x.device)
    with pytest.raises(ValueError, match="x: on"):
        ringx._expect("x", x, (3, 5), torch.float32, torch.device("meta"))


def test_gradient_inputs():
    q = _t(1, 2, 10, 64)
    lse = _t(1, 2, 10, dtype=torch.float32)
    delta = _t(2, 1, 2, 10, dtype=torch.float32)
    ringx._check_grad_inputs(q, _t(1, 2, 10, 64), lse, delta)
    with pytest.raises(ValueError, match="dout: shape"):
        ringx._check_grad_inputs(q, _t(1, 2, 11, 64), lse, delta)
    with pytest.raises(ValueError, match="delta: shape"):
        ringx._check_grad_inputs(q, _t(1, 2, 10, 64), lse, _t(2, 1, 2, 9, dtype=torch.float32))
    with pytest.raises(ValueError, match="delta: shape"):
        ringx._check_grad_inputs(q, _t(1, 2, 10, 64), lse, lse)
    with pytest.raises(TypeError, match="lse: dtype"):
        ringx._check_grad_inputs(q, _t(1, 2, 10, 64), _t(1, 2, 10), delta)


def test_wrappers_refuse_host_tensors():
    q = _t(1, 1, 8, 64)
    with pytest.raises(ValueError, match="GPU"):
        ringx.ringx_attn_fwd(q, q, q, 1)
