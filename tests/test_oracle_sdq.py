"""Pins for the oracle's decomposition, quantization and product.

What pins each part (none of these re-types the oracle's own formula):

* selection: brute force over every subset of every group, with exact
  rational sums and a lexicographic tie-break; the outlier-capture property
  of local extraction (Section 4); the ordering property of magnitude
  selection; the equivalence with "sparsify to (n_o+n_i):m, then extract
  n_o:m" (Section 5, Stages 1-2);
* quantizers: error bounds of each format, exact special cases (amax on a
  grid point), the OCP shared-exponent rule at hand-computed powers of two;
* product: a pure-Python loop over the stored (position, code) slots (the
  SpMMs of Section 5.1) against the dense fp64 product; a dense, unit-scale,
  integer configuration that must reduce to the textbook int64 matmul.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle import formats as F
from oracle import sdq as S

INT18 = S.Config("int", 1, 8, "e4m3", 3, 8, "int4", "int8")
INT18_I8 = S.Config("int", 1, 8, "int8", 3, 8, "int4", "int8")
INT116 = S.Config("int", 1, 16, "e4m3", 2, 8, "int4", "int8")
MX18 = S.Config("mx", 1, 8, "e4m3", 2, 8, "e2m1", "e4m3")
MX116 = S.Config("mx", 1, 16, "e4m3", 3, 8, "e2m1", "e4m3")
ALL = [INT18, INT18_I8, INT116, MX18, MX116,
       S.Config("int", 1, 16, "e4m3", 3, 8, "int4", "int8"),
       S.Config("int", 1, 8, "e4m3", 2, 8, "int4", "int8"),
       S.Config("mx", 1, 8, "e4m3", 3, 8, "e2m1", "e4m3"),
       S.Config("mx", 1, 16, "e4m3", 2, 8, "e2m1", "e4m3")]


def _brute_top(S_group, allowed, n):
    """Subset of size n of the allowed positions with the largest exact sum;
    among equal sums the lexicographically smallest position tuple."""
    cand = [k for k in range(len(S_group)) if allowed[k]]
    best, best_key = None, None
    for sub in itertools.combinations(cand, n):
        tot = sum(Fraction(float(S_group[k])) for k in sub)
        key = (-tot, sub)
        if best_key is None or key < best_key:
            best, best_key = sub, key
    return set(best)


def _tied_weights(rng, N, K):
    # few distinct magnitudes and random signs: many ties inside a group
    return (rng.integers(0, 4, (N, K)) * rng.choice([-1, 1], (N, K))).astype(np.float32) * 0.25


@pytest.mark.parametrize("cfg", [INT18, INT116, MX18, MX116], ids=lambda c: f"{c.n_o}:{c.m_o}+{c.n_i}:{c.m_i}")
@pytest.mark.parametrize("ties", [False, True])
def test_selection_brute_force(cfg, ties):
    rng = np.random.default_rng(11)
    N, K = 6, 64
    W = _tied_weights(rng, N, K) if ties else rng.standard_normal((N, K)).astype(np.float32)
    mask_o, pos_o, mask_i, pos_i = S.decompose(W, cfg)
    A = np.abs(W)
    for n in range(N):
        for g in range(K // cfg.m_o):
            ks = range(g * cfg.m_o, (g + 1) * cfg.m_o)
            want = _brute_top([A[n, k] for k in ks], [True] * cfg.m_o, cfg.n_o)
            got = {k - g * cfg.m_o for k in ks if mask_o[n, k]}
            assert got == want
        for g in range(K // cfg.m_i):
            ks = list(range(g * cfg.m_i, (g + 1) * cfg.m_i))
            allowed = [not mask_o[n, k] for k in ks]
            want = _brute_top([A[n, k] for k in ks], allowed, cfg.n_i)
            got = {k - g * cfg.m_i for k in ks if mask_i[n, k]}
            assert got == want
            assert list(pos_i[n, g]) == sorted(got)


def test_selection_product_metric_brute_force():
    rng = np.random.default_rng(12)
    N, K = 4, 32
    W = rng.standard_normal((N, K)).astype(np.float32)
    c = np.exp(rng.standard_normal(K) * 2).astype(np.float32)
    cfg = S.Config("int", 1, 8, "e4m3", 3, 8, "int4", "int8", metric="product")
    mask_o, _, mask_i, _ = S.decompose(W, cfg, act_norm=c)
    prod = np.abs(W) * c[None, :]
    for n in range(N):
        for g in range(K // 8):
            ks = list(range(8 * g, 8 * g + 8))
            want_o = _brute_top([prod[n, k] for k in ks], [True] * 8, 1)
            want_i = _brute_top([prod[n, k] for k in ks], [j not in want_o for j in range(8)], 3)
            assert {j for j in range(8) if mask_o[n, ks[j]]} == want_o
            assert {j for j in range(8) if mask_i[n, ks[j]]} == want_i
    # a tiny weight on a huge channel must be preferred over its magnitude rank
    W2 = np.full((1, 16), 0.5, np.float32)
    W2[0, 3] = 0.01
    c2 = np.ones(16, np.float32)
    c2[3] = 1000.0
    mo, _, _, _ = S.decompose(W2, cfg, act_norm=c2)
    assert mo[0, 3]


def test_sparsify_then_extract_equivalence():
    """Kept set = top (n_o+n_i); outliers = top n_o of the kept (Section 5)."""
    rng = np.random.default_rng(13)
    W = _tied_weights(rng, 8, 64)
    mo, _, mi, _ = S.decompose(W, INT18)
    A = np.abs(W)
    for n in range(8):
        for g in range(8):
            ks = list(range(8 * g, 8 * g + 8))
            kept = _brute_top([A[n, k] for k in ks], [True] * 8, 4)
            out = _brute_top([A[n, k] for k in ks], [j in kept for j in range(8)], 1)
            assert {j for j in range(8) if mo[n, ks[j]] or mi[n, ks[j]]} == kept
            assert {j for j in range(8) if mo[n, ks[j]]} == out


@pytest.mark.parametrize("cfg", ALL, ids=lambda c: f"{c.family}-{c.n_o}:{c.m_o}{c.fmt_o}+{c.n_i}:{c.m_i}")
def test_structure_invariants(cfg):
    W = synth.make_w(1, 0, 64, 256)
    L = S.pack_logical(W, cfg)
    mo, mi = L["mask_o"], L["mask_i"]
    assert not (mo & mi).any()
    assert (mo.reshape(64, -1, cfg.m_o).sum(-1) == cfg.n_o).all()
    assert (mi.reshape(64, -1, cfg.m_i).sum(-1) == cfg.n_i).all()
    assert (L["code_o_dense"][~mo] == 0).all() and (L["code_i_dense"][~mi] == 0).all()
    Wo, Wi = S.dequant_outliers(L), S.dequant_inliers(L)
    assert (Wo[~mo] == 0).all() and (Wi[~mi] == 0).all()
    # magnitude selection orders |outlier| >= |inlier| >= |pruned| in each group
    if cfg.m_o == cfg.m_i:
        A = np.abs(W).reshape(64, -1, 8)
        o = np.where(mo.reshape(A.shape), A, -1).max(-1)
        i_min = np.where(mi.reshape(A.shape), A, np.inf).min(-1)
        i_max = np.where(mi.reshape(A.shape), A, -1).max(-1)
        p = np.where(~(mo | mi).reshape(A.shape), A, -1).max(-1)
        assert (o >= i_max).all() and (i_min >= p).all()


@pytest.mark.parametrize("cfg", ALL, ids=lambda c: f"{c.family}-{c.n_o}:{c.m_o}{c.fmt_o}+{c.n_i}:{c.m_i}")
def test_reconstruction_error_bounds(cfg):
    """deq(W_o) + deq(W_i) is the quantization of W on the kept support."""
    W = synth.make_w(2, 0, 64, 512)
    L = S.pack_logical(W, cfg)
    mo, mi = L["mask_o"], L["mask_i"]
    Wd = S.dequant_outliers(L) + S.dequant_inliers(L)
    W64 = W.astype(np.float64)
    assert (Wd[~(mo | mi)] == 0).all()
    err = np.abs(Wd - W64)
    if cfg.family == "int":
        s = np.repeat(L["scale_i"].astype(np.float64), 16, axis=1)
        assert (err[mi] <= s[mi] / 2 * (1 + 1e-3) + 1e-12).all()
        so = np.repeat(L["scale_o"].astype(np.float64)[:, None], W.shape[1], axis=1)
        if cfg.fmt_o == "int8":
            assert (err[mo] <= so[mo] / 2 * (1 + 1e-6)).all()
        else:  # e4m3: relative 2^-4 for normals, absolute 2^-10 * s below
            assert (err[mo] <= np.maximum(2.0 ** -4 * np.abs(W64[mo]), 2.0 ** -10 * so[mo]) * (1 + 1e-6)).all()
    else:
        Ei = np.repeat(F.e8m0_value(L["scale_i"]), 32, axis=1)
        Eo = np.repeat(F.e8m0_value(L["scale_o"]), 32, axis=1)
        # saturating OCP rule: the block max may clip, everything else is within
        # half a step (step <= the largest element's spacing: 2 for e2m1, 32 for e4m3)
        assert (err[mi] <= np.maximum(0.25 * np.abs(W64[mi]), 0.25 * Ei[mi]) + 2.0 * Ei[mi] * (np.abs(W64[mi]) / Ei[mi] > 6)).all()
        assert (err[mo] <= np.maximum(2.0 ** -4 * np.abs(W64[mo]), 2.0 ** -10 * Eo[mo]) + 64 * Eo[mo] * (np.abs(W64[mo]) / Eo[mo] > 448)).all()


@pytest.mark.parametrize("cfg", [INT18, INT18_I8, INT116], ids=["e4m3-1:8", "int8-1:8", "e4m3-1:16"])
def test_row_outlier_scale_maps_the_row_maximum_to_qmax(cfg):
    """INT family, one outlier scale per row (reading R5: s_o = amax/qmax).  The
    outlier of largest magnitude in each row must come out as +-qmax: 448, the
    largest finite OCP E4M3FN value (codes 0x7E / 0xFE), or 127 for int8; no
    other outlier exceeds it, and |code| decodes back to |w| / s_o within half
    a step.  A wrong qmax (240, the fnuz maximum, or 127 for e4m3) or a scale
    taken over the inliers instead of the outliers fails here."""
    W = synth.make_w(2, 0, 64, 512)
    L = S.pack_logical(W, cfg)
    mo, code = L["mask_o"], L["code_o_dense"]
    qmax = 127.0 if cfg.fmt_o == "int8" else 448.0
    if cfg.fmt_o == "int8":
        v = code.view(np.int8).astype(np.float64)
    else:
        v = F.e4m3_decode(code)
    absW = np.where(mo, np.abs(W), 0)
    for n in range(W.shape[0]):
        k = int(np.argmax(absW[n]))
        assert mo[n, k] and absW[n, k] > 0
        assert abs(v[n, k]) == qmax, (n, k, v[n, k])
        if cfg.fmt_o == "e4m3":
            assert code[n, k] in (0x7E, 0xFE)
        else:
            assert code[n, k] in (127, 129)  # +127 / -127 as int8 bits
        assert np.abs(v[n][mo[n]]).max() == qmax
        # the scale is the row amax over the outliers only, divided by qmax
        assert np.float32(L["scale_o"][n]) == np.float32(np.float32(absW[n, k]) / np.float32(qmax))


def test_int4_unit_scale_grid_is_exact():
    """Blocks whose inlier amax is 7 get s = 1 and integer codes equal to W."""
    rng = np.random.default_rng(5)
    W = rng.integers(-7, 8, (16, 128)).astype(np.float32)
    W[:, ::16] = 7.0  # every 16-block holds a 7 ...
    W[:, 1::8] = 9.0  # ... and every 8-group an outlier of 9 (taken as outlier)
    L = S.pack_logical(W, INT18)
    assert (L["scale_i"] == 1.0).all()
    mi = L["mask_i"]
    assert np.array_equal(L["code_i_dense"][mi].astype(np.float32), W[mi])
    assert L["mask_o"][:, 1::8].all()


def test_mx_shared_exponent_rule_hand_values():
    # e4m3 emax = 8, e2m1 emax = 2 (OCP MX): E = floor(log2 amax) - emax
    cfg = MX18
    for amax, Eo, Ei in [(1.0, -8, -2), (448.0, 0, 6), (6.0, -6, 0), (0.75, -9, -3), (2.0 ** -20, -28, -22)]:
        W = np.zeros((1, 32), np.float32)
        W[0, 0] = amax      # outlier of group 0
        W[0, 1] = amax      # inlier of group 0 (same magnitude, higher k)
        L = S.pack_logical(W, cfg)
        assert int(L["scale_o"][0, 0]) - 127 == Eo
        assert int(L["scale_i"][0, 0]) - 127 == Ei
    W = np.zeros((1, 32), np.float32)
    L = S.pack_logical(W, cfg)
    assert L["scale_o"][0, 0] == 0 and L["scale_i"][0, 0] == 0 and (L["code_o"] == 0).all()


def test_outlier_capture_property():
    """Section 4: one global outlier per S-vector is always extracted; of two
    in one S-vector only the larger is."""
    rng = np.random.default_rng(6)
    W = (rng.standard_normal((32, 256)) * 0.02).astype(np.float32)
    plant = rng.integers(0, 8, (32, 32))
    for n in range(32):
        for g in range(32):
            W[n, 8 * g + plant[n, g]] *= 0.0
            W[n, 8 * g + plant[n, g]] += 0.5 * (1 + g % 3)
    L = S.pack_logical(W, INT18)
    for n in range(32):
        for g in range(32):
            assert L["pos_o"][n, g, 0] == plant[n, g]
    # two planted in one group: the larger is the outlier, the other an inlier
    W2 = (rng.standard_normal((1, 8)) * 0.02).astype(np.float32)
    W2[0, 2], W2[0, 6] = -0.4, 0.3
    L2 = S.pack_logical(np.tile(W2, (1, 2)), INT18)
    assert L2["pos_o"][0, 0, 0] == 2 and 6 in L2["pos_i"][0, 0]


@pytest.mark.parametrize("cfg", ALL[:5], ids=lambda c: f"{c.family}-{c.n_o}:{c.m_o}{c.fmt_o}+{c.n_i}:{c.m_i}")
def test_product_slot_loops_equal_dense(cfg):
    X = synth.make_x(1, 3, 64)
    W = synth.make_w(1, 0, 5, 64)
    Y, Xq, s_a, L = S.reference(X, W, cfg)
    Yl = S.sparse_gemm_loops(Xq, s_a, L)
    assert np.abs(Y - Yl).max() <= 1e-12 * np.abs(Y).max()
    Yd, Yo, Yi = S.gemm_fp64(Xq, s_a, L)
    assert np.allclose(Yo + Yi, Yd, rtol=1e-13, atol=1e-13 * np.abs(Yd).max())


def test_dense_unit_scale_reduces_to_textbook_int_matmul():
    """n_o = 0, n_i = m_i (dense), integer data on the unit-scale grid."""
    rng = np.random.default_rng(9)
    M, N, K = 5, 7, 64
    cfg = S.Config("int", 0, 8, "e4m3", 8, 8, "int4", "int8")
    W = rng.integers(-7, 8, (N, K)).astype(np.float32)
    W[:, ::16] = -7.0
    X = rng.integers(-127, 128, (M, K)).astype(np.float32)
    X[:, 0] = 127.0
    Y, Xq, s_a, L = S.reference(X, W, cfg)
    assert (s_a == 1.0).all() and (L["scale_i"] == 1.0).all()
    want = X.astype(np.int64) @ W.astype(np.int64).T
    assert np.array_equal(Y, want.astype(np.float64))
    P_i, _ = S.int_partials(Xq, L)
    assert np.array_equal(P_i.sum(-1), want)


def test_int_partials_reassemble_inlier_branch():
    X = synth.make_x(1, 4, 256)
    W = synth.make_w(1, 0, 9, 256)
    Y, Xq, s_a, L = S.reference(X, W, INT18_I8)
    P_i, P_o = S.int_partials(Xq, L)
    _, Yo, Yi = S.gemm_fp64(Xq, s_a, L)
    Yi2 = s_a[:, None].astype(np.float64) * (P_i * L["scale_i"].astype(np.float64)[None]).sum(-1)
    Yo2 = s_a[:, None].astype(np.float64) * P_o * L["scale_o"].astype(np.float64)[None, :]
    assert np.allclose(Yi, Yi2, rtol=1e-12, atol=1e-12 * np.abs(Yi).max())
    assert np.allclose(Yo, Yo2, rtol=1e-12, atol=1e-12 * np.abs(Yo).max())


@pytest.mark.parametrize("fmt_a", ["int8", "e4m3"])
def test_activation_quantization(fmt_a):
    cfg = INT18 if fmt_a == "int8" else MX18
    X = synth.make_x(2, 8, 512)
    X[3] = 0.0
    Xq, s_a = S.quantize_act(X, cfg)
    assert s_a[3] == 0 and (Xq[3] == 0).all()
    deq = S.dequant_act(Xq, s_a, cfg)
    amax = np.abs(X).max(1)
    qmax = 127 if fmt_a == "int8" else 448
    rows = [r for r in range(8) if r != 3]
    for r in rows:
        # the row maximum lands on the top code
        k = np.argmax(np.abs(X[r]))
        v = Xq[r, k].view(np.int8) if fmt_a == "int8" else F.E4M3_TABLE[Xq[r, k]]
        assert abs(float(v)) == qmax
        e = np.abs(deq[r] - X[r].astype(np.float64))
        if fmt_a == "int8":
            assert (e <= s_a[r] * 0.5 * (1 + 1e-5)).all()
        else:
            assert (e <= np.maximum(2.0 ** -4 * np.abs(X[r]), 2.0 ** -10 * s_a[r]) * (1 + 1e-5)).all()
    assert np.allclose(s_a[rows], amax[rows] / qmax, rtol=1e-7)


def test_ragged_and_degenerate_shapes():
    cfg = INT18
    X = np.zeros((0, 128), np.float32)
    Xq, s_a = S.quantize_act(X, cfg)
    assert Xq.shape == (0, 128)
    W = np.zeros((3, 128), np.float32)
    Y, Xq, s_a, L = S.reference(synth.make_x(1, 2, 128), W, cfg)
    assert (Y == 0).all() and (L["scale_o"] == 0).all() and (L["scale_i"] == 0).all()
