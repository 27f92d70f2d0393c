"""Pins for the decomposition-metric variants of the oracle (Section 5,
"Stage 2", and Section 6.4's decomposition study: magnitude, weight-activation
product and quantization-error metrics, taken "Large" or "Small").

What pins them (none re-types the oracle's formula):

* the staged procedure (sparsify, then extract) with the significance metric
  and "Large" order selects the same sets as the default procedure (outliers
  first, then inliers), a theorem about top-k selection, for every supported
  configuration including 1:16 outliers with 8-groups of inliers;
* brute force over every subset of every group for the kept set, and over
  the kept positions for the outlier, with exact rational keys;
* hand-computed quantization errors on grids where the inlier quantizer's
  scale is 1 (int4: amax 7; e2m1: amax 6), including round-half-to-even;
* structural invariants for every variant.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest

from oracle import sdq as S

INT = dict(family="int", fmt_o="e4m3", fmt_i="int4", fmt_a="int8")
MX = dict(family="mx", fmt_o="e4m3", fmt_i="e2m1", fmt_a="e4m3")
VARIANTS = [(d, o) for d in ("same", "magnitude", "product", "error", "output_error")
            for o in ("large", "small")]


def cfg_of(base, m_o=8, n_i=3, metric="magnitude", decomp="same", order="large"):
    return S.Config(base["family"], 1, m_o, base["fmt_o"], n_i, 8, base["fmt_i"], base["fmt_a"],
                    metric, decomp, order)


def _brute_top(vals, allowed, n, largest=True):
    """Subset of n allowed positions with the largest (or smallest) exact sum;
    among equal sums the lexicographically smallest tuple of positions."""
    cand = [k for k in range(len(vals)) if allowed[k]]
    best, best_key = None, None
    for sub in itertools.combinations(cand, n):
        tot = sum(Fraction(float(vals[k])) for k in sub)
        key = (-tot if largest else tot, sub)
        if best_key is None or key < best_key:
            best, best_key = sub, key
    return set(best)


def _weights(seed, N, K, ties):
    rng = np.random.default_rng(seed)
    if ties:
        return (rng.integers(0, 4, (N, K)) * rng.choice([-1, 1], (N, K))).astype(np.float32) * 0.25
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    W[rng.random((N, K)) < 0.02] *= 12
    return W


@pytest.mark.parametrize("base", [INT, MX], ids=["int", "mx"])
@pytest.mark.parametrize("m_o,n_i", [(8, 3), (8, 2), (16, 3), (16, 2), (8, 1)])
@pytest.mark.parametrize("metric", ["magnitude", "product"])
@pytest.mark.parametrize("ties", [False, True])
def test_staged_default_equals_outliers_first(base, m_o, n_i, metric, ties):
    W = _weights(3, 12, 128, ties)
    c = np.exp(np.random.default_rng(4).standard_normal(128)).astype(np.float32)
    cfg = cfg_of(base, m_o, n_i, metric)
    a = S.decompose(W, cfg, act_norm=c)          # default: outliers first, then inliers
    b = S.decompose_staged(W, cfg, act_norm=c)   # paper order: sparsify, then extract
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("decomp,order", VARIANTS)
@pytest.mark.parametrize("m_o", [8, 16])
def test_selection_brute_force(decomp, order, m_o):
    rng = np.random.default_rng(21)
    N, K = 4, 64
    W = _weights(22, N, K, ties=(order == "small"))
    c = np.exp(rng.standard_normal(K)).astype(np.float32)
    cfg = cfg_of(INT, m_o, 3, "magnitude", decomp, order)
    mask_o, _, mask_i, pos_i = S.decompose(W, cfg, act_norm=c)
    A = np.abs(W)
    keep = np.zeros_like(mask_o)
    for n in range(N):
        for g in range(K // 8):
            kept = _brute_top([A[n, 8 * g + j] for j in range(8)], [True] * 8, 4)
            for j in kept:
                keep[n, 8 * g + j] = True
    # the decomposition key, from the definitions (the error metric from the
    # oracle's own inlier quantizer is pinned separately by hand values)
    if decomp in ("same", "magnitude"):
        D = A
    elif decomp == "product":
        D = A * c[None, :]
    else:
        D = S.inlier_error(W, keep, cfg) * (c[None, :] if decomp == "output_error" else 1)
    for n in range(N):
        for g in range(K // m_o):
            ks = list(range(g * m_o, (g + 1) * m_o))
            want = _brute_top([D[n, k] for k in ks], [keep[n, k] for k in ks], 1, order == "large")
            assert {k - g * m_o for k in ks if mask_o[n, k]} == want
        for g in range(K // 8):
            ks = list(range(8 * g, 8 * g + 8))
            allowed = [keep[n, k] and not mask_o[n, k] for k in ks]
            want = _brute_top([A[n, k] for k in ks], allowed, 3)
            got = {k - 8 * g for k in ks if mask_i[n, k]}
            assert got == want and list(pos_i[n, g]) == sorted(got)


def test_error_metric_int4_hand_values():
    # one 16-K block, 1:8 + 3:8; group 0 keeps {7.0, 3.4, 2.5, 1.0} (top 4 by |w|),
    # the block amax over kept positions is 7 so s = fp16(7/7) = 1 and the codes
    # are rne(w): 7 -> 7 (error 0), 3.4 -> 3 (0.4), 2.5 -> 2 (0.5, ties to even),
    # 1.0 -> 1 (0)
    w = np.array([[7.0, 3.4, 2.5, 1.0, 0.1, 0.2, 0.3, 0.05,
                   0.6, 2.2, -1.6, 0.05, 0.01, 3.5, 0.02, 0.0]], np.float32)
    # group 1 keeps {0.6, 2.2, -1.6, 3.5}: 3.5 -> 4 (0.5, ties to even), 2.2 -> 2
    # (0.2), 1.6 -> 2 (0.4), 0.6 -> 1 (0.4)
    def out(decomp, order, c=None):
        m, _, _, _ = S.decompose(w, cfg_of(INT, 8, 3, "magnitude", decomp, order), act_norm=c)
        return [int(np.nonzero(m[0, 8 * g:8 * g + 8])[0][0]) for g in range(2)]
    assert out("error", "large") == [2, 5]
    assert out("error", "small") == [0, 1]        # group 0 errors (0, 0.4, 0.5, 0): ties go to lower k
    assert out("magnitude", "large") == [0, 5]
    assert out("magnitude", "small") == [3, 0]
    assert out("same", "small") == [3, 0]
    # output error: the 0.5 errors on channels of norm 0.1 drop below the 0.4
    # ones; in group 1, 1 - fp32(0.6) and 2 - fp32(1.6) are the same fp32
    # number (6710886 * 2^-24), so the lower k (position 0) wins the tie
    c = np.ones(16, np.float32)
    c[2] = 0.1
    c[13] = 0.1
    assert out("output_error", "large", c) == [1, 0]
    e = S.inlier_error(w, np.abs(w) >= np.float32(0.6), cfg_of(INT))
    assert e[0, 0] == 0 and e[0, 2] == np.float32(0.5) and e[0, 1] == np.float32(3.4) - np.float32(3.0)


def test_error_metric_scales_over_kept_positions_only():
    # product significance prunes the 20.0 on a channel of norm 0.001 (0.02 <
    # the others), so the block's provisional scale comes from 7.0 alone:
    # s = 1, errors (0, 0.4, 0.5, 0) and the outlier is the 2.5.  Were the
    # pruned 20.0 in the amax, s = fp16(20/7) = 2.857421875 and the errors
    # (1.285, 0.543, 0.357, 1.0) would pick the 7.0 instead.
    w = np.zeros((1, 16), np.float32)
    w[0, :8] = [20.0, 7.0, 3.4, 2.5, 1.0, 0.1, 0.2, 0.3]
    c = np.ones(16, np.float32)
    c[0] = 0.001
    m, _, mi, _ = S.decompose(w, cfg_of(INT, 8, 3, "product", "error", "large"), act_norm=c)
    assert np.nonzero(m[0, :8])[0].tolist() == [3]
    assert np.nonzero(mi[0, :8])[0].tolist() == [1, 2, 4]


def test_error_metric_e2m1_hand_values():
    # one 32-K block with amax 6 over the kept positions: E = floor(log2 6) - 2 = 0,
    # the e2m1 grid is {0, 0.5, 1, 1.5, 2, 3, 4, 6}; 5 lies halfway between 4
    # (code 0b110, even) and 6 (0b111) and rounds to 4 (error 1); 2.7 -> 3
    # (0.3); 1.2 -> 1 (0.2)
    w = np.zeros((1, 32), np.float32)
    w[0, :8] = [6.0, 5.0, 2.7, 1.2, 0.1, 0.0, 0.0, 0.0]
    w[0, 8:16] = [0.5, 1.5, 0.9, 0.0, 0.0, 0.0, 0.0, 0.0]  # 0.9 -> 1 (0.1); others exact
    cfg = cfg_of(MX, 8, 2, "magnitude", "error", "large")
    m, _, mi, _ = S.decompose(w, cfg)
    assert m[0, 1] and not m[0, 0]
    assert m[0, 10]
    cfg_s = cfg_of(MX, 8, 2, "magnitude", "error", "small")
    ms, _, _, _ = S.decompose(w, cfg_s)
    assert ms[0, 0]           # error 0, lowest k
    assert ms[0, 8]           # 0.5 exact, lowest k among the zero errors
    e = S.inlier_error(w, w != 0, cfg)
    assert e[0, 1] == 1.0 and e[0, 2] == abs(np.float32(2.7) - np.float32(3.0))


@pytest.mark.parametrize("base", [INT, MX], ids=["int", "mx"])
@pytest.mark.parametrize("decomp,order", VARIANTS)
def test_structure_invariants(base, decomp, order):
    W = _weights(31, 16, 256, ties=False)
    c = np.exp(np.random.default_rng(32).standard_normal(256)).astype(np.float32)
    for m_o in (8, 16):
        cfg = cfg_of(base, m_o, 2, "product", decomp, order)
        L = S.pack_logical(W, cfg, act_norm=c)
        mo, mi = L["mask_o"], L["mask_i"]
        assert not (mo & mi).any()
        assert (mo.reshape(16, -1, m_o).sum(-1) == 1).all()
        assert (mi.reshape(16, -1, 8).sum(-1) == 2).all()
        # every chosen position is among the 3 most significant of its 8-group
        sig = np.abs(W) * c[None, :]
        kept, _ = S.top_n_per_group(sig.astype(np.float32), np.ones_like(mo), 8, 3)
        assert not ((mo | mi) & ~kept).any()
        # the two branches reconstruct the quantized kept weights exactly where chosen
        Wo, Wi = S.dequant_outliers(L), S.dequant_inliers(L)
        assert ((Wo != 0) <= mo).all() and ((Wi != 0) <= mi).all()


def test_variants_need_outliers_and_valid_names():
    with pytest.raises(AssertionError):
        S.Config("int", 0, 8, "e4m3", 3, 8, "int4", "int8", decomp="error").check(128)
    with pytest.raises(AssertionError):
        S.Config("int", 1, 8, "e4m3", 3, 8, "int4", "int8", order="middle").check(128)
