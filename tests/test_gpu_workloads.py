"""GPU parity at the workloads' real sizes, in the configuration bench.py times.

Each layer runs the whole product path on the GPU (sdq_linear: activation
quantization + decomposed GEMM, weights packed by sdq_pack).  The oracle
computes a sample of the outputs one by one: a seeded sample of output rows
(packing only those rows of W, which is exact because rows are independent)
against a sample of tokens.  The activation codes and scales of the sampled
tokens are compared bit for bit.
"""
import numpy as np
import pytest

import synth
from oracle import sdq as S
from tests.gpu_util import REL_TOL, MX_TERM_TOL, rel_errors, say, torch_cuda

import paper_2406_13868_amd as sdq

pytestmark = pytest.mark.gpu

N_ROWS, N_TOKENS = 24, 24


def _run_layer(wid, li, M, fmt, W=None, X=None):
    torch = torch_cuda()
    L = synth.WORKLOADS[wid].layers[li]
    if W is None:
        W = synth.make_w(wid, li, L.N, L.K)
    if X is None:
        X = synth.make_x(wid, M, L.K)
    cfg = sdq.Config.of(fmt)
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    Xd = torch.from_numpy(X).cuda()
    if synth.WORKLOADS[wid].x_dtype == "bf16":
        Xd = Xd.to(torch.bfloat16)
    Y, Xq, s_a = sdq.linear(Xd, blob, L.N, L.K, cfg)
    torch.cuda.synchronize()
    return W, X, Y, Xq, s_a


def _check_sampled(W, X, Y, Xq, s_a, fmt, seed, what):
    cfg_o = S.config_from(fmt)
    rng = np.random.default_rng(seed)
    M, N = Y.shape
    ms = np.sort(rng.choice(M, size=min(M, N_TOKENS), replace=False))
    ns = np.sort(rng.choice(N, size=min(N, N_ROWS), replace=False))
    Xq_ref, s_ref = S.quantize_act(X[ms], cfg_o)
    assert np.array_equal(Xq.cpu().numpy()[ms], Xq_ref), f"{what}: Xq"
    assert np.array_equal(s_a.cpu().numpy()[ms].view(np.uint32), s_ref.view(np.uint32)), f"{what}: s_a"
    Lg = S.pack_logical(W[ns], cfg_o)
    Yref, _, _ = S.gemm_fp64(Xq_ref, s_ref, Lg)
    Yg = Y.cpu().numpy()[np.ix_(ms, ns)].astype(np.float64)
    mr, nr = rel_errors(Yg, Yref)
    if cfg_o.family == "mx":
        A = np.abs(S.dequant_act(Xq_ref, s_ref, cfg_o))
        T = A @ (np.abs(S.dequant_outliers(Lg)) + np.abs(S.dequant_inliers(Lg))).T
        comp = float(np.max(np.abs(Yg - Yref) / np.maximum(T, 1e-30)))
        assert nr <= REL_TOL and comp <= MX_TERM_TOL, f"{what}: norm={nr:.2e} term={comp:.2e}"
    else:
        assert mr <= REL_TOL and nr <= REL_TOL, f"{what}: max_rel={mr:.2e} norm={nr:.2e}"


@pytest.mark.parametrize("wid,li", [(2, 0), (3, 0), (3, 2), (4, 0), (4, 1), (1, 0), (7, 0)],
                         ids=["llama-attn-decode", "llama-mlp-gate-prefill", "llama-mlp-down-prefill",
                              "opt-fc1-decode", "opt-fc2-decode", "tiny", "llama-qkv-decode"])
def test_workload_layer(wid, li):
    w = synth.WORKLOADS[wid]
    M, fmt = w.M[0], w.formats[0]
    say("workload", w.name, w.layers[li].name, M, fmt.label)
    W, X, Y, Xq, s_a = _run_layer(wid, li, M, fmt)
    _check_sampled(W, X, Y, Xq, s_a, fmt, seed=wid * 10 + li, what=f"{w.name}/{w.layers[li].name}")


@pytest.mark.parametrize("li", range(7), ids=[L.name for L in synth.LLAMA7B_LAYERS])
def test_block_sweep_layer(li):
    """Every format of the block sweep at every token count, for one layer."""
    w = synth.WORKLOADS[5]
    L = w.layers[li]
    W = synth.make_w(5, li, L.N, L.K)
    Xs = {M: synth.make_x(5, M, L.K) for M in w.M}
    for (pli, _, M, fmt) in synth.sweep_points(5):
        if pli != li:
            continue
        say("sweep", L.name, M, fmt.label)
        _, _, Y, Xq, s_a = _run_layer(5, li, M, fmt, W=W, X=Xs[M])
        _check_sampled(W, Xs[M], Y, Xq, s_a, fmt, seed=li * 100 + M, what=f"{L.name} M={M} {fmt.label}")
