"""Pins for the analytic accounting: every value the paper prints."""
import json
import os
from fractions import Fraction

import pytest

from oracle import accounting as A

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


@pytest.mark.parametrize("row", GOLD["effective_throughput"], ids=lambda r: r["label"])
def test_effective_throughput_matches_paper(row):
    got = A.effective_throughput([tuple(b) for b in row["branches"]])
    assert got == Fraction(*row["exact"])
    assert round(float(got), 1) == row["printed"]


@pytest.mark.parametrize("row", GOLD["mac_reduction_percent"], ids=lambda r: f'{r["n"]}:{r["m"]}')
def test_mac_reduction(row):
    # an N:M unit runs the dense product at cost n/m (Section 3.1)
    assert float((1 - A.branch_cost(row["n"], row["m"], 16)) * 100) == row["printed"]


@pytest.mark.parametrize("row", GOLD["quantized_speedup"], ids=lambda r: str(r["bits"]))
def test_quantized_speedup(row):
    assert A.effective_throughput([(1, 1, row["bits"])]) == row["printed"]


@pytest.mark.parametrize("row", GOLD["index_bits_per_vector"], ids=lambda r: f'{r["n"]}:{r["m"]}')
def test_index_metadata(row):
    assert A.index_bits_per_vector(row["n"], row["m"]) == row["printed"]


def test_scale_overhead_example():
    e = GOLD["scale_overhead_example"]
    assert A.avg_bits_per_element(e["value_bits"], e["scale_bits"], e["qv"]) == e["printed"]


def test_sparse_can_cost_more_bits_than_dense():
    s = GOLD["sparse_vs_dense_4bit"]["sparse"]
    sparse = Fraction(s["n"] * (s["bits"] + A.index_bits_per_vector(1, s["m"])), s["m"])
    assert sparse > GOLD["sparse_vs_dense_4bit"]["dense_bits"]


def test_sdq_bits_per_weight_configs():
    # 1:8 e4m3 (per-row fp32) + 3:8 int4 (fp16 per 16), K = 4096:
    # (8+3)/8 + 3*(4+3)/8 + 16/16 + 32/4096
    b = A.sdq_bits_per_weight(1, 8, 8, 3, 8, 4, 32, 0, 16, 16, 4096)
    assert b == Fraction(11, 8) + Fraction(21, 8) + 1 + Fraction(32, 4096)
    # MX: 1:8 e4m3 + 2:8 e2m1, both e8m0 per 32
    b = A.sdq_bits_per_weight(1, 8, 8, 2, 8, 4, 8, 32, 8, 32, 4096)
    assert b == Fraction(11, 8) + Fraction(14, 8) + Fraction(8, 32) * 2
