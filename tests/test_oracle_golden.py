"""The oracle against the numbers the paper prints for its own worked examples.

The values and their citations live in ``tests/golden/paper_printed_values.json``;
each entry gives the inputs as the paper states them and the printed result
with the rounding it was printed at.
"""
import json
import os

import pytest

from oracle import cost, pool

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "paper_printed_values.json")
with open(GOLDEN) as f:
    ENTRIES = json.load(f)["entries"]


def _n_seq_case(n_layers, n_kv_heads, head_dim, dtype_bytes, c_max, m_gpu, util, m_model):
    return pool.n_seq(m_gpu, util, m_model, pool.m_seq(n_layers, n_kv_heads, head_dim, dtype_bytes, c_max))


def _n_seq_ratio(n_layers, n_kv_heads, head_dim, dtype_bytes, c_short, c_long, m_gpu, util, m_model):
    short = _n_seq_case(n_layers, n_kv_heads, head_dim, dtype_bytes, c_short, m_gpu, util, m_model)
    return short // _n_seq_case(n_layers, n_kv_heads, head_dim, dtype_bytes, c_long, m_gpu, util, m_model)


def _kv_budget(m_gpu, util, m_model):
    # the numerator of Eq. 2, read off n_seq with one-byte sequences
    return pool.n_seq(m_gpu, util, m_model, 1)


def _last_block_waste(n_seqs, waste_tokens, n_layers, n_kv_heads, head_dim, dtype_bytes):
    return n_seqs * waste_tokens * pool.kv_bytes_per_token(n_layers, n_kv_heads, head_dim, dtype_bytes)


QUANTITIES = {
    "savings_formula": lambda alpha, rho: cost.savings_formula(alpha, rho),
    "rho": cost.rho,
    "g_homo": cost.g_homo,
    "kv_bytes_per_token": pool.kv_bytes_per_token,
    "kv_budget": _kv_budget,
    "n_seq_case": _n_seq_case,
    "n_seq_ratio": _n_seq_ratio,
    "last_block_waste": _last_block_waste,
}


def test_every_entry_is_cited_and_known():
    assert len(ENTRIES) >= 10
    for e in ENTRIES:
        assert e["cite"].startswith(("Sec.", "Table")), e["id"]
        assert e["quantity"] in QUANTITIES, e["id"]


@pytest.mark.parametrize("entry", ENTRIES, ids=[e["id"] for e in ENTRIES])
def test_printed_value(entry):
    got = QUANTITIES[entry["quantity"]](**entry["args"]) / entry["scale"]
    assert abs(got - entry["expect"]) <= entry["tol"], (entry["id"], got, entry["expect"], entry["cite"])
