"""GPU: the INT family's quantized inlier scales (Section 3.3 quantizes the
scale factors and sets their vector length; Section 6.4 compares 8-bit scale
formats): Q-Vectors of 16, 32 and 64 dense K with fp16, two-level e4m3 or
ufp8-e6m2 scales, on every INT kernel (the decode kernel and its fused form,
the split-K and tiled matrix-core kernels), against the fp64 oracle; the
integer grid (every scale exactly 1) must stay exact."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import sdq as S
from tests.gpu_util import assert_close, say, torch_cuda

import paper_2406_13868_amd as sdq

pytestmark = pytest.mark.gpu

# (scale format, Q-Vector); fp16 and e4m3 at 16 are covered by test_gpu_gemm.py
COMBOS = [("", 32), ("", 64), ("e4m3", 32), ("e4m3", 64), ("ue6m2", 16), ("ue6m2", 32), ("ue6m2", 64)]
ID = [f"{s or 'f16'}-qv{q}" for s, q in COMBOS]


def _cfgs(sfmt, qv, fmt_o="e4m3", n_o=1, m_o=8, n_i=3):
    cfg = sdq.Config("int", n_o, m_o, fmt_o, n_i, 8, "int4", "int8", sfmt_i=sfmt, qv_i=qv)
    cfg_o = S.Config("int", n_o, m_o, fmt_o, n_i, 8, "int4", "int8", sfmt_i=sfmt, qv=qv)
    return cfg, cfg_o


def _run(X, W, cfg, path):
    torch = torch_cuda()
    N, K = W.shape
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    Xq, s_a = sdq.quantize_act(torch.from_numpy(np.ascontiguousarray(X)).cuda(), cfg)
    Y = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=path)
    torch.cuda.synchronize()
    return Y.cpu().numpy()


def _paths(M):
    return ([sdq.PATH_DECODE] if M <= 8 else []) + [sdq.PATH_MFMA, sdq.PATH_SPLITK]


@pytest.mark.parametrize("combo", COMBOS, ids=ID)
@pytest.mark.parametrize("fmt_o", ["e4m3", "int8"])
@pytest.mark.parametrize("M,N,K", [(1, 256, 256), (2, 96, 4096), (5, 100, 512), (8, 64, 128),
                                   (16, 256, 256), (33, 160, 384), (64, 256, 2048),
                                   (400, 8192, 256)])
def test_scale_formats_match_oracle(combo, fmt_o, M, N, K):
    sfmt, qv = combo
    cfg, cfg_o = _cfgs(sfmt, qv, fmt_o)
    X = synth.make_x(1, M, K)
    W = synth.make_w(1, 0, N, K)
    W[min(3, N - 1), :] = 0.0            # a row without inliers
    W[min(5, N - 1), :64] = 0.0          # zero Q-Vectors inside a row
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    for path in _paths(M):
        say("scales", sfmt or "f16", qv, fmt_o, M, N, K, "path", path)
        Y = _run(X, W, cfg, path)
        assert_close(Y, Yref, f"{sfmt or 'f16'} qv={qv} {fmt_o} M={M} N={N} K={K} path={path}")


@pytest.mark.parametrize("combo", COMBOS, ids=ID)
@pytest.mark.parametrize("M,N,K", [(1, 64, 4096), (16, 96, 1024), (96, 64, 512)])
def test_scale_formats_integer_grid_is_exact(combo, M, N, K):
    """Integer activations with amax 127 and int4-grid inliers whose every
    Q-Vector holds a 7: every scale is exactly 1 (fp16 1.0, e4m3 code 0x38 under
    a row scale of 2^-8 times 256, e6m2 code 124), so Y must equal the int64
    product."""
    sfmt, qv = combo
    cfg, cfg_o = _cfgs(sfmt, qv, "int8")
    rng = np.random.default_rng(M + N + qv)
    X = rng.integers(-127, 128, (M, K)).astype(np.float32)
    X[:, 0] = 127.0
    W = np.zeros((N, K), np.float32)
    W[:, 0::8] = rng.integers(8, 17, (N, K // 8))   # outliers: the largest of each group
    W[:, 0] = 127.0                                  # int8 outlier scale 1
    inl = rng.integers(-7, 8, (N, K // 8, 3)).astype(np.float32)
    inl[inl == 0] = 1.0
    W.reshape(N, K // 8, 8)[:, :, 1:4] = inl
    W.reshape(N, K // qv, qv)[:, :, 1] = 7.0          # every Q-Vector's amax is 7
    Yref, _, s_ref, L = S.reference(X, W, cfg_o)
    assert (s_ref == 1).all() and (S.inlier_scale_values(L) == 1).all() and (L["scale_o"] == 1).all()
    for path in _paths(M):
        say("scales grid", sfmt or "f16", qv, M, N, K, "path", path)
        Y = _run(X, W, cfg, path)
        assert np.array_equal(Y.astype(np.float64), Yref), f"path {path}: not exact"


@pytest.mark.parametrize("combo", [("ue6m2", 64), ("", 64)], ids=["ue6m2-qv64", "f16-qv64"])
@pytest.mark.parametrize("M", [1, 2])
def test_scale_formats_fused_linear_full_layer(combo, M):
    """sdq_linear (activation quantization fused into the decode kernel) on the
    LLaMA-7B attention projection (4096 x 4096), every output."""
    torch = torch_cuda()
    sfmt, qv = combo
    cfg, cfg_o = _cfgs(sfmt, qv)
    X = synth.make_x(2, M, 4096)
    W = synth.make_w(2, 0, 4096, 4096)
    Yref, Xq_ref, s_ref, _ = S.reference(X, W, cfg_o)
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    say("scales linear", sfmt or "f16", qv, M)
    Y, Xq, s_a = sdq.linear(torch.from_numpy(X).cuda().to(torch.bfloat16), blob, 4096, 4096, cfg)
    torch.cuda.synchronize()
    assert np.array_equal(Xq.cpu().numpy(), Xq_ref)
    assert_close(Y.cpu().numpy(), Yref, f"linear {sfmt or 'f16'} qv={qv} M={M}")
