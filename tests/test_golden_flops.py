"""The FLOP convention used for throughput against the paper's Table II and Eq. (7)."""

import json
import os

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def _load():
    with open(os.path.join(HERE, "golden", "flop_model.json")) as f:
        return json.load(f)


def _eval(expr, **sym):
    return eval(expr, {"__builtins__": {}}, sym)  # fixture text written in this repository


@pytest.mark.parametrize("b,S,h", [(1, 1024, 192), (128, 2_097_152, 960), (3, 4096, 3072)])
def test_table_ii_rows_sum_to_eq7(b, S, h):
    g = _load()
    total = sum(_eval(r["flops"], b=b, S=S, h=h) for r in g["table_II_rows"])
    assert total == pytest.approx(_eval(g["eq_7_forward_total"], b=b, S=S, h=h), rel=1e-12)


@pytest.mark.parametrize("B,H,S,d", [(1, 16, 16384, 64), (2, 8, 4096, 128)])
def test_per_pair_convention_matches_attention_rows(B, H, S, d):
    """Forward attention flops 4*B*H*Nq*Nk*d with Nq = Nk = S and h = H*d equal Table II's two
    attention rows."""
    g = _load()
    rows = {r["module"]: r["flops"] for r in g["table_II_rows"]}
    attn = sum(_eval(rows[m], b=B, S=S, h=H * d) for m in g["attention_rows"])
    assert 4 * B * H * S * S * d == attn
