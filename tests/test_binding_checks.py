"""The Python binding checks every caller-supplied tensor before its pointer
reaches the C ABI (which cannot see sizes): a wrong shape, dtype, length or
byte count raises ValueError instead of becoming an out-of-bounds access on
the GPU.  CPU only: the checks run before any device call."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2406_13868_amd as sdq  # noqa: E402

INT = sdq.Config.int_family()
MX = sdq.Config.mx_family()
DUAL = sdq.Config.dual_family()
M, N, K = 4, 256, 256


def _raises(fn, match):
    with pytest.raises(ValueError, match=match):
        fn()


def test_quantize_act_checks_outputs():
    X = torch.zeros((M, K))
    _raises(lambda: sdq.quantize_act(X, INT, out=torch.empty((M, K - 128), dtype=torch.uint8)), r"Xq must be \[4, 256\]")
    _raises(lambda: sdq.quantize_act(X, INT, out=torch.empty((M, K), dtype=torch.int32)), "Xq must be")
    _raises(lambda: sdq.quantize_act(X, INT, scales=torch.empty((M - 1,))), r"s_a must be \[4\]")
    _raises(lambda: sdq.quantize_act(X, INT, scales=torch.empty((M,), dtype=torch.float16)), "s_a must be")
    _raises(lambda: sdq.quantize_act(X.to(torch.float16), INT), "float32 or bfloat16")
    # correct shapes on the CPU: refused because they are not GPU tensors
    _raises(lambda: sdq.quantize_act(X, INT, out=torch.empty((M, K), dtype=torch.uint8),
                                     scales=torch.empty((M,))), "CUDA")


def test_quantize_act_dual_checks_every_output():
    X = torch.zeros((M, K))
    good = [torch.empty((M, K), dtype=torch.uint8), torch.empty((M,)),
            torch.empty((M, K // 2), dtype=torch.uint8), torch.empty((M, K // 32), dtype=torch.uint8)]
    for i, (bad, what) in enumerate([(torch.empty((M, K // 2), dtype=torch.uint8), "Xq_o"),
                                     (torch.empty((M + 1,)), "s_a_o"),
                                     (torch.empty((M, K), dtype=torch.uint8), "Xq_i"),
                                     (torch.empty((M, K // 16), dtype=torch.uint8), "e_a_i")]):
        out = list(good)
        out[i] = bad
        _raises(lambda: sdq.quantize_act_dual(X, DUAL, out=tuple(out)), f"{what} must be")


def test_gemm_checks_activations_scales_weights_and_output():
    Xq = torch.empty((M, K), dtype=torch.uint8)
    s_a = torch.empty((M,))
    blob = torch.empty(sdq.pack_size(INT, N, K), dtype=torch.uint8)
    _raises(lambda: sdq.gemm(torch.empty((M, K + 128), dtype=torch.uint8), s_a, blob, N, K, INT), "Xq must be")
    _raises(lambda: sdq.gemm(Xq, torch.empty((M - 1,)), blob, N, K, INT), "s_a must be")
    _raises(lambda: sdq.gemm(Xq, s_a, blob[:-16], N, K, INT), "packed holds")
    _raises(lambda: sdq.gemm(Xq, s_a, blob, N, K, INT, out=torch.empty((M, N + 1))), "out must be")
    _raises(lambda: sdq.gemm(Xq, s_a, blob, N, K, INT, out=torch.empty((M, N), dtype=torch.bfloat16)), "out must be")


def test_gemm_checks_the_workspace():
    Mw, Nw, Kw = 2048, 11008, 256
    ws = sdq.gemm_workspace_size(MX, Mw, Nw, Kw)
    assert ws > 0  # the two-pass path of many MX tokens takes one
    Xq = torch.empty((Mw, Kw), dtype=torch.uint8)
    s_a = torch.empty((Mw,))
    blob = torch.empty(sdq.pack_size(MX, Nw, Kw), dtype=torch.uint8)
    Y = torch.empty((Mw, Nw))
    _raises(lambda: sdq.gemm(Xq, s_a, blob, Nw, Kw, MX, out=Y, workspace=torch.empty(ws - 16, dtype=torch.uint8)),
            "workspace holds")


def test_gemm_dual_checks_the_token_count_of_every_tensor():
    Xo = torch.empty((M, K), dtype=torch.uint8)
    s_a = torch.empty((M,))
    Xi = torch.empty((M, K // 2), dtype=torch.uint8)
    Ea = torch.empty((M, K // 32), dtype=torch.uint8)
    blob = torch.empty(sdq.pack_size(DUAL, N, K), dtype=torch.uint8)
    _raises(lambda: sdq.gemm_dual(Xo, s_a, Xi[:2], Ea, blob, N, K, DUAL), "Xq_i must be")
    _raises(lambda: sdq.gemm_dual(Xo, s_a, Xi, Ea[:2], blob, N, K, DUAL), "e_a_i must be")
    _raises(lambda: sdq.gemm_dual(Xo, s_a[:2], Xi, Ea, blob, N, K, DUAL), "s_a_o must be")
    _raises(lambda: sdq.gemm_dual(Xo, s_a, Xi, Ea, blob[:100], N, K, DUAL), "packed holds")


def test_linear_checks_its_buffers():
    X = torch.zeros((M, K))
    blob = torch.empty(sdq.pack_size(INT, N, K), dtype=torch.uint8)
    _raises(lambda: sdq.linear(X, blob, N, K + 128, INT), "X must be")
    _raises(lambda: sdq.linear(X, blob, N, K, INT, xq=torch.empty((M + 1, K), dtype=torch.uint8)), "Xq must be")
    _raises(lambda: sdq.linear(X, blob, N, K, INT, scales=torch.empty((2 * M,))), "s_a must be")
    _raises(lambda: sdq.linear(X, blob[:8], N, K, INT), "packed holds")
