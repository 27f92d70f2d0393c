"""GPU parity at the workloads' real sizes, in the configuration bench.py times.

Each layer runs the whole product path on the GPU (sdq_linear: activation
quantization + decomposed GEMM, weights packed by sdq_pack).  For the named
workloads every output is compared: the oracle decomposes, quantizes and
multiplies the whole layer itself (fp64), and every activation code and
scale is compared bit for bit.  The 112-point block sweep compares a seeded
sample of outputs (packing only the sampled rows of W, which is exact because
rows are independent) against a sample of tokens, plus one INT layer at 4096
tokens in full.
"""
import numpy as np
import pytest

import synth
from oracle import sdq as S
from tests.gpu_util import REL_TOL, dual_term_tol, mx_term_tol, rel_errors, say, torch_cuda

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


def _compare(Yg, Yref, Xq_ref, s_ref, Lg, cfg_o, what):
    mr, nr = rel_errors(Yg, Yref)
    if cfg_o.family == "mx":
        A = np.abs(S.dequant_act(Xq_ref, s_ref, cfg_o))
        T = A @ (np.abs(S.dequant_outliers(Lg)) + np.abs(S.dequant_inliers(Lg))).T
        comp = float(np.max(np.abs(Yg - Yref) / np.maximum(T, 1e-30)))
        say(f"{what}: max_rel={mr:.3e} norm={nr:.3e} term={comp:.3e} outputs={Yg.size}")
        assert nr <= REL_TOL and comp <= mx_term_tol(Lg["K"]), f"{what}: norm={nr:.2e} term={comp:.2e}"
    else:
        say(f"{what}: max_rel={mr:.3e} norm={nr:.3e} outputs={Yg.size}")
        assert mr <= REL_TOL and nr <= REL_TOL, f"{what}: max_rel={mr:.2e} norm={nr:.2e}"


def _check_full(W, X, Y, Xq, s_a, fmt, what):
    """Every output and every activation code against the oracle's own pack and product."""
    cfg_o = S.config_from(fmt)
    Xq_ref, s_ref = S.quantize_act(X, cfg_o)
    assert np.array_equal(Xq.cpu().numpy(), Xq_ref), f"{what}: Xq"
    assert np.array_equal(s_a.cpu().numpy().view(np.uint32), s_ref.view(np.uint32)), f"{what}: s_a"
    Lg = S.pack_logical(W, cfg_o)
    Yref, _, _ = S.gemm_fp64(Xq_ref, s_ref, Lg)
    _compare(Y.cpu().numpy().astype(np.float64), Yref, Xq_ref, s_ref, Lg, cfg_o, what)


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
    _compare(Y.cpu().numpy()[np.ix_(ms, ns)].astype(np.float64), Yref, Xq_ref, s_ref, Lg, cfg_o, what)


@pytest.mark.parametrize("wid,li", [(2, 0), (3, 0), (3, 2), (4, 0), (4, 1), (1, 0), (7, 0)],
                         ids=["llama-attn-decode", "llama-mlp-gate-prefill", "llama-mlp-down-prefill",
                              "opt-fc1-decode", "opt-fc2-decode", "tiny", "llama-qkv-decode"])
def test_workload_layer_every_output(wid, li):
    w = synth.WORKLOADS[wid]
    M, fmt = w.M[0], w.formats[0]
    say("workload", w.name, w.layers[li].name, M, fmt.label)
    W, X, Y, Xq, s_a = _run_layer(wid, li, M, fmt)
    _check_full(W, X, Y, Xq, s_a, fmt, f"{w.name}/{w.layers[li].name}")


def test_block_sweep_int_prefill_every_output():
    """The LLaMA-7B q_proj at 4096 tokens in the INT family (1:8 e4m3 + 3:8
    int4, the tiled matrix-core kernel), every one of its 16.8 M outputs."""
    w = synth.WORKLOADS[5]
    fmt = w.formats[1]
    assert (fmt.family, fmt.n_o, fmt.m_o, fmt.n_i) == ("int", 1, 8, 3)
    L = w.layers[0]
    say("sweep full", L.name, 4096, fmt.label)
    W, X, Y, Xq, s_a = _run_layer(5, 0, 4096, fmt)
    _check_full(W, X, Y, Xq, s_a, fmt, f"{L.name} M=4096 {fmt.label}")


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


@pytest.mark.parametrize("fi", [0, 1], ids=["1:8+6:8", "2:8+4:8"])
def test_dual_block_gate_prefill_every_output(fi):
    """The paper's own configurations (1:8 or 2:8 int8 outliers against int8
    activations, 6:8 or 4:8 fp4 inliers against MXFP4 activations) on the
    LLaMA-7B gate projection at 4096 tokens, every output."""
    torch = torch_cuda()
    w = synth.WORKLOADS[6]
    fmt, L = w.formats[fi], w.layers[4]
    cfg, cfg_o = sdq.Config.of(fmt), S.config_from(fmt)
    W = synth.make_w(6, 4, L.N, L.K)
    X = synth.make_x(6, 4096, L.K)
    say("dual full", L.name, 4096, fmt.label)
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    Xd = torch.from_numpy(X).cuda().to(torch.bfloat16)
    Xo, s_a, Xi, Ea = sdq.quantize_act_dual(Xd, cfg)
    Y = sdq.gemm_dual(Xo, s_a, Xi, Ea, blob, L.N, L.K, cfg)
    torch.cuda.synchronize()
    Yref, (Ao, Ai), (s_ao, Ea_ref), Lg = S.reference(X, W, cfg_o)
    assert np.array_equal(Xo.cpu().numpy(), Ao) and np.array_equal(Ea.cpu().numpy(), Ea_ref)
    assert np.array_equal(s_a.cpu().numpy().view(np.uint32), s_ao.view(np.uint32))
    A_o, A_i = S.dequant_act_dual(Ao, s_ao, Ai, Ea_ref)
    T = np.abs(A_o) @ np.abs(S.dequant_outliers(Lg)).T + np.abs(A_i) @ np.abs(S.dequant_inliers(Lg)).T
    Yg = Y.cpu().numpy().astype(np.float64)
    mr, nr = rel_errors(Yg, Yref)
    comp = float(np.max(np.abs(Yg - Yref) / np.maximum(T, 1e-30)))
    say(f"dual {L.name} M=4096: max_rel={mr:.3e} norm={nr:.3e} term={comp:.3e} outputs={Yg.size}")
    assert nr <= REL_TOL and comp <= dual_term_tol(L.K), f"norm={nr:.2e} term={comp:.2e}"
