"""CPU oracle for the SDQ decomposed GEMM.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call, link
or execute anything under ``oracle/``: only the tests, the entry point's smoke
check and the benchmark's CPU-baseline leg use it.

The oracle is a plain, slow, obviously correct implementation of what the
method computes, written from the paper (Jeong et al., "SDQ: Sparse Decomposed
Quantization for LLM Inference"):

* ``formats``    number formats from their definitions (int4/int8, OCP fp8
                 E4M3FN, fp4 E2M1, E8M0, fp16), with nearest-even encoders;
* ``sdq``        the three offline stages of Section 5 (sparsify/decompose by a
                 significance metric under N:M, then per-vector quantization)
                 and the decomposed product of Section 5.1 in fp64;
* ``accounting`` the analytic throughput and bits-per-weight counts of
                 Sections 3.1-3.3 and 5.1.

It shares no code with the HIP path.  It is pinned by ``tests/test_oracle_*``
against closed forms, format definitions, brute force and invariants.
"""
from . import accounting, formats, sdq  # noqa: F401
