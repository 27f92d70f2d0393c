"""Pins for the quantized inlier scale formats of the oracle (Section 3.3:
scale factors are metadata and are themselves quantized, VS-Quant; Section
7's quantization study compares ufp8-e6m2 and fp8-e4m3 scale factors) and
for other Q-Vector sizes.

What pins them: the ufp8-e6m2 codec against its definition by brute force;
the power-of-two row scale of the two-level e4m3 scheme at hand-computed
boundaries; hand-computed two-level codes; the error bounds of each scale
format; the unit-scale integer grid, which must stay exact; integer partials
over other block sizes reassembling the branch.
"""
import numpy as np
import pytest

import synth
from oracle import formats as F
from oracle import sdq as S


def test_ue6m2_values_from_definition():
    # bias 31, two mantissa bits, no sign; subnormals m/4 * 2^-30
    assert F.ue6m2_value(0) == 0.0
    assert F.ue6m2_value(1) == 2.0 ** -32
    assert F.ue6m2_value(4) == 2.0 ** -30          # smallest normal
    assert F.ue6m2_value(31 << 2) == 1.0
    assert F.ue6m2_value((31 << 2) | 3) == 1.75
    assert F.UE6M2_MAX == 1.75 * 2.0 ** 32
    assert (np.diff(F.UE6M2_TABLE) > 0).all()


def test_ue6m2_encoder_brute_force():
    rng = np.random.default_rng(3)
    mids = (F.UE6M2_TABLE[1:] + F.UE6M2_TABLE[:-1]) / 2
    xs = np.concatenate([F.UE6M2_TABLE, mids, np.nextafter(mids, 0), np.nextafter(mids, np.inf),
                         np.exp(rng.uniform(-25, 25, 2000)), [1e12, F.UE6M2_MAX * 1.01]])
    got = F.ue6m2_encode(xs)
    for x, c in zip(xs, got):
        d = np.abs(F.UE6M2_TABLE - min(x, F.UE6M2_MAX))
        best = np.flatnonzero(d == d.min())
        want = best[0] if len(best) == 1 else [b for b in best if b % 2 == 0][0]
        assert c == want, (x, c, want)
    assert (F.ue6m2_encode(F.UE6M2_TABLE) == np.arange(256)).all()


@pytest.mark.parametrize("vmax,E", [(1.0, -8), (1.75, -8), (np.float32(1.75) * (1 + 2 ** -23), -7),
                                    (448.0, 0), (449.0, 1), (0.0, 0), (2.0 ** -120, -128),
                                    (3.5, -7)])
def test_row_scale_exponent_hand_values(vmax, E):
    # the smallest E with vmax <= 448 * 2^E
    assert S.row_scale_exponent(np.array([vmax], np.float32))[0] == E


def _int_cfg(sfmt="", qv=0, n_i=3):
    return S.Config("int", 1, 8, "e4m3", n_i, 8, "int4", "int8", sfmt_i=sfmt, qv=qv)


def test_two_level_e4m3_hand_values():
    # inliers only in the first group of each 16-block (the outlier takes position 0)
    W = np.zeros((1, 64), np.float32)
    W[0, 0:4] = [100.0, 7.0, 3.0, -2.0]      # block 0: inlier amax 7 -> v = 1
    W[0, 16:20] = [100.0, 3.5, 1.0, 0.5]     # block 1: amax 3.5 -> v = 0.5
    W[0, 32:36] = [100.0, 0.1, 0.05, 0.02]   # block 2: amax 0.1 -> v = fp32(0.1/7)
    # block 3 empty: v = 0
    L = S.pack_logical(W, _int_cfg("e4m3"))
    # vmax = 1 -> E = -8: the stored scales are e4m3(v * 256)
    assert L["scale_i_row"][0] == np.float32(2.0 ** -8)
    v2 = np.float32(np.float32(0.1) / np.float32(7.0))
    assert [F.e4m3_value(c) for c in L["scale_i"][0]] == [256.0, 128.0, F.e4m3_value(F.e4m3_encode(v2 * 256.0)), 0.0]
    # 0.0142857 * 256 = 3.657 lies between 3.5 and 3.75 -> 3.75
    assert F.e4m3_value(L["scale_i"][0, 2]) == 3.75
    s = S.inlier_scale_values(L)[0]
    assert list(s) == [1.0, 0.5, 3.75 / 256, 0.0]
    # codes: w / s, rounded half to even, clamped to +-7
    assert list(L["code_i_dense"][0, 1:4]) == [7, 3, -2]
    assert list(L["code_i_dense"][0, 17:20]) == [7, 2, 1]
    assert list(L["code_i_dense"][0, 33:36]) == [7, 3, 1]   # 0.1/0.0146 = 6.83; 3.41; 1.37


def test_two_level_single_block_row():
    # a row whose largest vector scale is 0.1/7 uses E with that scale near 448
    W = np.zeros((1, 16), np.float32)
    W[0, :4] = [1.0, 0.1, 0.05, 0.0]
    L = S.pack_logical(W, _int_cfg("e4m3"))
    v = np.float32(np.float32(0.1) / np.float32(7.0))
    E = S.row_scale_exponent(np.array([v]))[0]
    assert E == -14                           # 448 * 2^-15 < v <= 448 * 2^-14
    assert F.e4m3_value(L["scale_i"][0, 0]) == 240.0    # v * 2^14 = 234.06 -> 240
    assert L["scale_i_row"][0] == np.float32(2.0 ** -14)


@pytest.mark.parametrize("sfmt", ["", "e4m3", "ue6m2"])
@pytest.mark.parametrize("qv", [16, 32, 64])
def test_scale_error_bounds(sfmt, qv):
    W = synth.make_w(1, 0, 64, 512)
    L = S.pack_logical(W, _int_cfg(sfmt, qv))
    mi = L["mask_i"]
    s = np.repeat(S.inlier_scale_values(L), qv, axis=1)
    deq = S.dequant_inliers(L)
    a = np.where(mi, np.abs(W), 0).reshape(64, -1, qv).max(-1)
    v = np.repeat(a / 7.0, qv, axis=1)
    inside = mi & (np.abs(W) <= 7 * s)          # no clamping
    assert (np.abs(W - deq)[inside] <= s[inside] / 2 * (1 + 1e-6)).all()
    # the stored scale is within the format's relative precision of amax/7
    ok = mi & (v > 0)
    rel = np.abs(s - v)[ok] / v[ok]
    bound = {"": 2.0 ** -11, "e4m3": 2.0 ** -4, "ue6m2": 2.0 ** -3}[sfmt]
    assert rel.max() <= bound * (1 + 1e-6)


@pytest.mark.parametrize("sfmt", ["", "e4m3", "ue6m2"])
def test_unit_scale_grid_exact(sfmt):
    # every block's inlier amax is 7: the effective scale is exactly 1 in every format
    rng = np.random.default_rng(5)
    W = rng.integers(-6, 7, (8, 128)).astype(np.float32)
    W[:, ::8] = 50.0                             # outliers take position 0 of every group
    W[:, 1::16] = 7.0                            # inlier amax 7 in every 16-block
    L = S.pack_logical(W, _int_cfg(sfmt, n_i=7))
    assert (S.inlier_scale_values(L) == 1.0).all()
    assert np.array_equal(S.dequant_inliers(L)[L["mask_i"]], W[L["mask_i"]])


@pytest.mark.parametrize("sfmt", ["", "e4m3"])
@pytest.mark.parametrize("qv", [16, 64])
def test_int_partials_reassemble_with_block_size(sfmt, qv):
    cfg = _int_cfg(sfmt, qv)
    W = synth.make_w(1, 0, 16, 256)
    X = synth.make_x(1, 4, 256)
    Xq, s_a = S.quantize_act(X, cfg)
    L = S.pack_logical(W, cfg)
    P_i, _ = S.int_partials(Xq, L)
    Y_i = S.gemm_fp64(Xq, s_a, L)[2]
    Y_re = s_a[:, None].astype(np.float64) * (P_i * S.inlier_scale_values(L)[None]).sum(-1)
    assert np.allclose(Y_re, Y_i, rtol=1e-12, atol=1e-12)
    # and the slot loops of the two SpMMs agree with the dense product
    Y = S.gemm_fp64(Xq, s_a, L)[0]
    assert np.allclose(S.sparse_gemm_loops(Xq, s_a, L), Y, rtol=1e-12, atol=1e-12)


def test_scale_format_validation():
    with pytest.raises(AssertionError):
        S.Config("mx", 1, 8, "e4m3", 2, 8, "e2m1", "e4m3", sfmt_i="e4m3").check(128)
    with pytest.raises(AssertionError):
        _int_cfg("e4m3", 48).check(192)
