"""Pins for the dual family of the oracle (Section 5.1's worked configuration:
1:8 int8 outliers with int8 activations A_o, 6:8 fp4 inliers with fp4
activations A_i, O = SpMM(A_o, W_o) + SpMM(A_i, W_i)).

What pins it: hand-computed MXFP4 activation codes and exponents (the OCP MX
rule, saturation, round-half-to-even, an all-zero block); A_o equal to the
int8 per-token quantizer pinned elsewhere; the pure-Python loops over the
stored slots of both SpMMs against the dense fp64 product; the branch
structure of 7:8 = 1:8 + 6:8 and of 6:8 = 2:8 + 4:8 (the paper's other
evaluated configuration); a weight matrix with no outliers or no inliers
reducing the product to the other branch alone.
"""
import numpy as np
import pytest

import synth
from oracle import formats as F
from oracle import sdq as S

DUAL = S.Config("dual", 1, 8, "int8", 6, 8, "e2m1", "int8+e2m1")


def test_mxfp4_activation_hand_values():
    X = np.zeros((2, 64), np.float32)
    X[0, :6] = [6.0, 5.0, -3.0, 0.25, 1.25, 0.75]   # amax 6: E = 2 - 2 = 0
    X[0, 32:36] = [12.0, -7.0, 2.5, 1.0]           # amax 12: E = 3 - 2 = 1, values / 2
    X[1, :2] = [7.0, 1.0]                           # amax 7: E = 0, 7 saturates to 6
    # X[1, 32:] all zero: E = -127, zero codes
    Ao, s_ao, Ai, Ea = S.quantize_act_dual(X)
    assert list(Ea[0]) == [127, 128] and list(Ea[1]) == [127, 0]
    v = F.e2m1_decode(Ai)
    # 5 lies halfway between 4 (even mantissa) and 6; 0.25 halfway between 0 and 0.5 -> 0;
    # 1.25 between 1 and 1.5 -> 1; 0.75 between 0.5 and 1 -> 1 (even mantissa)
    assert list(v[0, :6]) == [6.0, 4.0, -3.0, 0.0, 1.0, 1.0]
    # block 1 of row 0 at E = 1: 12/2 = 6, -7/2 = -3.5 -> -4 (halfway, even), 2.5/2 = 1.25 -> 1, 0.5
    assert list(v[0, 32:36]) == [6.0, -4.0, 1.0, 0.5]
    assert list(v[1, :2]) == [6.0, 1.0]
    assert not Ai[1, 32:].any()


def test_mxfp4_error_bound():
    X = synth.make_x(2, 16, 512)
    _, _, Ai, Ea = S.quantize_act_dual(X)
    scale = np.repeat(F.e8m0_value(Ea), 32, axis=1)
    A_i = F.e2m1_decode(Ai) * scale
    # half the e2m1 spacing (0.5 up to 2, 1 up to 4, 2 up to 6), times 2^E; past 6
    # the value saturates, and the block amax stays below 8 * 2^E
    v = np.abs(X) / scale
    half = np.where(v <= 2, 0.25, np.where(v <= 4, 0.5, np.where(v <= 6, 1.0, v - 6)))
    assert (np.abs(X - A_i) <= half * scale).all()
    assert (v < 8).all()


def test_act_o_is_the_int8_quantizer():
    X = synth.make_x(2, 8, 256)
    Ao, s_ao, _, _ = S.quantize_act_dual(X)
    Xq, s_a = S.quantize_act(X, S.Config("int", 1, 8, "e4m3", 3, 8, "int4", "int8"))
    assert np.array_equal(Ao, Xq) and np.array_equal(s_ao, s_a)


@pytest.mark.parametrize("n_o,n_i", [(1, 6), (1, 3), (2, 4), (2, 6)])
def test_slot_loops_equal_dense_product(n_o, n_i):
    cfg = S.Config("dual", n_o, 8, "int8", n_i, 8, "e2m1", "int8+e2m1")
    W = synth.make_w(2, 0, 12, 128)
    X = synth.make_x(2, 3, 128)
    Ao, s_ao, Ai, Ea = S.quantize_act_dual(X)
    L = S.pack_logical(W, cfg)
    Y, Y_o, Y_i = S.gemm_fp64_dual(Ao, s_ao, Ai, Ea, L)
    assert np.allclose(S.sparse_gemm_loops_dual(Ao, s_ao, Ai, Ea, L), Y, rtol=1e-12, atol=1e-12)
    assert np.allclose(Y_o + Y_i, Y)


def test_seven_of_eight_structure():
    W = synth.make_w(2, 0, 16, 256)
    L = S.pack_logical(W, DUAL)
    mo, mi = L["mask_o"], L["mask_i"]
    assert (mo.reshape(16, -1, 8).sum(-1) == 1).all() and (mi.reshape(16, -1, 8).sum(-1) == 6).all()
    assert not (mo & mi).any()
    # the pruned position of every group is its smallest magnitude
    A = np.abs(W).reshape(16, -1, 8)
    kept = (mo | mi).reshape(16, -1, 8)
    assert (np.where(kept, -np.inf, A).max(-1) <= np.where(kept, A, np.inf).min(-1)).all()
    # int8 outliers with one fp32 scale per row: the row's largest outlier is code 127
    codes = L["code_o_dense"].view(np.int8)
    assert (np.abs(codes).max(axis=1) == 127).all()


def test_six_of_eight_structure():
    """The paper's 6:8 configuration with two int8 outliers and four fp4
    inliers per group of 8: exactly that many of each, disjoint, the outliers
    the two largest magnitudes of the group and the pruned two the smallest."""
    cfg = S.Config("dual", 2, 8, "int8", 4, 8, "e2m1", "int8+e2m1")
    W = synth.make_w(2, 1, 16, 256)
    L = S.pack_logical(W, cfg)
    mo, mi = L["mask_o"].reshape(16, -1, 8), L["mask_i"].reshape(16, -1, 8)
    assert (mo.sum(-1) == 2).all() and (mi.sum(-1) == 4).all()
    assert not (mo & mi).any()
    A = np.abs(W).reshape(16, -1, 8)
    pruned = ~(mo | mi)
    assert (np.where(mo, A, np.inf).min(-1) >= np.where(mi, A, -np.inf).max(-1)).all()
    assert (np.where(mi, A, np.inf).min(-1) >= np.where(pruned, A, -np.inf).max(-1)).all()
    codes = L["code_o_dense"].view(np.int8)
    assert (np.abs(codes).max(axis=1) == 127).all()
    assert (L["pos_o"][..., 0] < L["pos_o"][..., 1]).all()  # slots in ascending position


def test_branches_alone():
    X = synth.make_x(2, 4, 128)
    Ao, s_ao, Ai, Ea = S.quantize_act_dual(X)
    W = synth.make_w(2, 0, 8, 128)
    # no outlier branch: only A_i W_i
    c0 = S.Config("dual", 0, 8, "int8", 7, 8, "e2m1", "int8+e2m1")
    L0 = S.pack_logical(W, c0)
    Y0, Yo0, _ = S.gemm_fp64_dual(Ao, s_ao, Ai, Ea, L0)
    assert not Yo0.any()
    _, A_i = S.dequant_act_dual(Ao, s_ao, Ai, Ea)
    assert np.allclose(Y0, A_i @ S.dequant_inliers(L0).T)
    # outliers only where the inliers quantize to zero: a matrix of one large
    # value per group and zeros elsewhere
    W1 = np.zeros((8, 128), np.float32)
    W1[:, 3::8] = 1.0
    L1 = S.pack_logical(W1, DUAL)
    Y1, Yo1, Yi1 = S.gemm_fp64_dual(Ao, s_ao, Ai, Ea, L1)
    assert not Yi1.any()
    A_o, _ = S.dequant_act_dual(Ao, s_ao, Ai, Ea)
    assert np.allclose(Y1, A_o[:, 3::8].sum(1)[:, None] * np.ones((1, 8)))
