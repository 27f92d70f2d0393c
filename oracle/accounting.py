"""Analytic accounting of the paper: effective throughput and bits per weight.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

* Section 3.1: an N:M structured-sparse unit is assumed to give M/N times the
  dense throughput.
* Section 3.2: with both operands quantized to n bits, a unit gives 16/n times
  the fp16 throughput.
* Section 5.1: the decomposed product costs the sum of its branch costs,
  each branch (n/m) * (bits/16) of the fp16 dense product; the effective
  throughput is the reciprocal.
* Section 3.3: an ELLPACK-like index costs log2(M) bits per non-zero; a scale
  factor of b bits shared by a Q-Vector of v elements costs b/v bits per
  element.
"""
from __future__ import annotations

import math
from fractions import Fraction
from typing import Iterable, Tuple


def branch_cost(n: int, m: int, bits: int) -> Fraction:
    """Cost of one N:M, n-bit SpMM relative to the dense fp16 GEMM."""
    return Fraction(n, m) * Fraction(bits, 16)


def effective_throughput(branches: Iterable[Tuple[int, int, int]]) -> Fraction:
    """1 / sum of branch costs, for branches given as (n, m, compute_bits)."""
    total = sum((branch_cost(n, m, b) for n, m, b in branches), Fraction(0))
    return 1 / total


def index_bits_per_vector(n: int, m: int) -> int:
    """ELLPACK-like metadata: log2(m) bits per non-zero, n non-zeros."""
    return n * int(math.log2(m))


def scale_bits_per_element(scale_bits: int, qv: int) -> Fraction:
    return Fraction(scale_bits, qv)


def avg_bits_per_element(value_bits: int, scale_bits: int, qv: int) -> Fraction:
    """Dense quantized data plus its scale, per element (Section 3.3 example)."""
    return Fraction(value_bits * qv + scale_bits, qv)


def sdq_bits_per_weight(n_o: int, m_o: int, bits_o: int, n_i: int, m_i: int, bits_i: int,
                        scale_o_bits: int, qv_o: int, scale_i_bits: int, qv_i: int,
                        K: int) -> Fraction:
    """Logical bits per dense weight of the decomposed, packed layer.

    Each branch stores n values and n log2(m)-bit indices per m weights, and
    one scale per Q-Vector; ``qv_o == 0`` means one scale per row of K weights.
    """
    b = Fraction(0)
    if n_o:
        b += Fraction(n_o * (bits_o + int(math.log2(m_o))), m_o)
        b += Fraction(scale_o_bits, qv_o if qv_o else K)
    b += Fraction(n_i * (bits_i + int(math.log2(m_i))), m_i)
    b += Fraction(scale_i_bits, qv_i)
    return b
