"""GPU: what gfx950's scaled matrix instruction does with the MX family's
products, on designed inputs, and the exact decoding of every weight.

The paper fixes no accumulation precision (Section 5.1 counts operations
only); the MX kernels use v_mfma_scale_f32_32x32x64_f8f6f4, whose summation
is the hardware's.  These tests pin the properties the MX tolerance rests on
(tests/gpu_util.py, mx_term_tol):

* every weight of a full LLaMA-7B gate layer decodes exactly: with one-hot
  activations (448 at one k, so s_a = 1) each output is a single product and
  equals 448 * deq(W)[n, k] bit for bit, on both MX paths;
* products of similar magnitude sum exactly: twenty products of 0.75 fp32
  ulps of 448 add up exactly when no larger product shares the instruction;
* the instruction's partial sums enter the fp32 accumulator rounded to
  nearest even: with 448 already in the accumulator, the same twenty products
  (an exact sum of 15 ulps) arrive as 14 ulps, which is the nearest-even
  rounding of four partial sums of 16 K (4.5, 4.5, 3.75 and 2.25 ulps) added
  one after the other; a single product of half an ulp ties to even and is
  dropped, one ulp is kept;
* inside one 32-K scale block a dominant product costs the others low-order
  bits: the block of the LLaMA-7B MLP gate weights (row 1064, token 348 of
  the prefill activations, K 3232..3263) whose products are 72 and eleven
  between 0.03 and 0.22 comes out 3 * 2^-8 below the exact sum, 2^-12.58 of
  its largest product.  That is the largest loss relative to a block's
  largest product found on the workload data (the full-size tests); the MX
  tolerance allows 2^-12 of the sum of |terms| per output plus the rounding
  of the partial sums.

All inputs are in range and every kernel launch is an ordinary sdq_gemm call.
"""
import numpy as np
import pytest

import synth
from oracle import sdq as S
from tests.gpu_util import MX_BLOCK_LOSS, say, torch_cuda

import paper_2406_13868_amd as sdq

pytestmark = pytest.mark.gpu

FMT = synth.WORKLOADS[3].formats[0]  # MX 1:8 e4m3 + 2:8 e2m1, e4m3 activations
ULP448 = 2.0 ** -15                  # fp32 spacing at 448


def _cfgs():
    return sdq.Config.of(FMT), S.config_from(FMT)


def _gemm(X, W, path):
    torch = torch_cuda()
    cfg, _ = _cfgs()
    N, K = W.shape
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    Xq, s_a = sdq.quantize_act(torch.from_numpy(np.ascontiguousarray(X, np.float32)).cuda(), cfg)
    ws = sdq.gemm_workspace_size(cfg, X.shape[0], N, K, path)
    wsb = torch.empty(ws, dtype=torch.uint8, device="cuda") if ws else None
    Y = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=path, workspace=wsb)
    torch.cuda.synchronize()
    return Y.cpu().numpy().astype(np.float64), s_a.cpu().numpy()


@pytest.mark.parametrize("path", [sdq.PATH_DENSE, sdq.PATH_MFMA], ids=["two-pass", "one-pass"])
def test_every_weight_of_a_prefill_layer_decodes_exactly(path):
    """Both MX paths reproduce 448 * deq(W) for all 45 M weights of the
    LLaMA-7B gate projection (11008 x 4096) with one-hot activations."""
    _, cfg_o = _cfgs()
    N, K = 11008, 4096
    W = synth.make_w(3, 0, N, K)
    L = S.pack_logical(W, cfg_o)
    ref = 448.0 * (S.dequant_outliers(L) + S.dequant_inliers(L)).T
    X = np.zeros((K, K), np.float32)
    np.fill_diagonal(X, 448.0)
    say("one-hot decode", N, K, "path", path)
    Y, s_a = _gemm(X, W, path)
    assert np.all(s_a == 1.0)
    bad = np.argwhere(Y != ref)
    assert len(bad) == 0, f"{len(bad)} weights differ, first (k, n) = {bad[:4].tolist()}"


def _kept(b):
    """Kept positions (0, 1, 2 of each 8-group) of 32-K block b: with equal
    magnitudes there, position 0 is the outlier and 1, 2 the inliers, and the
    block merges (inlier exponent = outlier exponent + 6)."""
    return [k for k in range(32 * b, 32 * b + 32) if k % 8 in (0, 1, 2)]


def test_partial_sums_round_to_nearest_even_into_the_accumulator():
    K = 256
    ws = [2.0 ** -16, 2.0 ** -17]  # small products 0.75 and 0.375 ulps of 448
    W = np.zeros((len(ws), K), np.float32)
    for r, w in enumerate(ws):
        W[r, _kept(0)] = 1.0
        W[r, _kept(4)] = 1.0
        W[r, _kept(2) + _kept(3)] = w
    small = (_kept(2) + _kept(3))[:20]

    def tok(big, xs, n=20):
        x = np.zeros(K, np.float32)
        x[3] = 448.0        # sets s_a = 1 (W is zero at k = 3)
        x[0], x[128] = big, -big  # +big in the first instruction, -big in the third
        x[small[:n]] = xs
        return x

    X = np.stack([tok(448.0, 1.5), tok(0.0, 1.5), tok(448.0, 1.5, 1), tok(448.0, 1.0)])
    say("accumulator rounding probe")
    Y, s_a = _gemm(X, W, sdq.PATH_MFMA)
    assert np.all(s_a == 1.0)
    u = ULP448
    # exact sums: 20 x 1.5 w
    assert Y[1, 0] == 30 * ws[0] and Y[1, 1] == 30 * ws[1], "similar products must sum exactly"
    # accumulator at 448: four 16-K partial sums, each rounded to nearest even
    assert Y[0, 0] == 14 * u, Y[0, 0] / u      # 4.5, 4.5, 3.75, 2.25 ulps -> 4, 8, 12, 14
    assert Y[0, 1] == 7 * u, Y[0, 1] / u       # 2.25, 2.25, 1.875, 1.125 -> 2, 4, 6, 7
    assert Y[2, 0] == 1 * u and Y[2, 1] == 0.0  # one product of 0.75 ulp -> 1; 0.375 -> 0
    assert Y[3, 0] == 10 * u                    # 20 x 0.5 ulp, partial sums 3, 3, 2.5 ... exact in halves
    assert Y[3, 1] == 6 * u, Y[3, 1] / u        # 1.5, 1.5, 1.25, 0.75 -> 2, 4, 5, 6


def test_dominant_product_in_a_scale_block():
    """The measured worst case: a block of the gate weights in which an
    activation-outlier channel meets an outlier weight (product 72)."""
    _, cfg_o = _cfgs()
    K = 4096
    n, m, k0 = 1064, 348, 3200  # instruction 50: K 3200..3263; the block is 3232..3263
    Wrow = synth.make_w(3, 0, 11008, K)[n]
    x = synth.make_x(3, 2048, K)[m]
    W = np.zeros((2, K), np.float32)
    W[0, k0:k0 + 64] = Wrow[k0:k0 + 64]       # the whole instruction
    W[1, k0 + 32:k0 + 64] = Wrow[k0 + 32:k0 + 64]  # the lossy block alone
    Yref, Xq_ref, s_ref, L = S.reference(x[None], W, cfg_o)
    A = S.dequant_act(Xq_ref, s_ref, cfg_o)[0] / s_ref[0]
    Wd = S.dequant_outliers(L) + S.dequant_inliers(L)
    prods = A * Wd[1]
    assert np.abs(prods).max() == 72.0 and np.count_nonzero(prods) == 12
    say("dominant-product block", n, m, k0)
    Y, s_a = _gemm(x[None], W, sdq.PATH_MFMA)
    assert s_a[0].view(np.uint32) == s_ref[0].view(np.uint32)
    got = Y[0] / s_ref[0]
    exact = (A * Wd).sum(axis=1)
    loss = got - exact
    # deterministic: both rows lose exactly 3 * 2^-8 (up to the final fp32 scaling by s_a)
    assert np.all(np.abs(loss + 3.0 / 256) < 1e-6 * np.abs(exact)), loss
    # and that loss is within the per-block bound the tolerance uses
    assert np.all(np.abs(loss) <= MX_BLOCK_LOSS * 72.0)
