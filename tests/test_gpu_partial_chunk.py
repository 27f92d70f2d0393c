"""GPU: K a multiple of 32 but not of 128.  The blob pads the last 128-K chunk
with zero codes and scales, and every kernel reads its activations through
bounds past which they read 0 (or, inside the tensor, the next row's values,
which meet zero weights).  Every path against the oracle; integer grids
exact."""
import numpy as np
import pytest

import synth
from oracle import sdq as S
from tests.gpu_util import assert_close, say, torch_cuda
from tests.test_gpu_gemm import _cfgs, _ids, _kernel_for, check, run_gpu, INT_CFGS, MX_CFGS

import paper_2406_13868_amd as sdq

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("c", [INT_CFGS[0], INT_CFGS[1], INT_CFGS[2], INT_CFGS[5]], ids=_ids)
@pytest.mark.parametrize("M,N,K", [(1, 96, 160), (2, 300, 288), (5, 64, 1056), (40, 160, 4128),
                                   (100, 70, 160), (256, 129, 416)])
def test_int_paths(c, M, N, K):
    cfg, cfg_o = _cfgs(*c)
    X = synth.make_x(6, M, K)
    W = synth.make_w(6, 0, N, K)
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    paths = ([sdq.PATH_DECODE] if M <= 8 and sdq.gemm_path(cfg, M, N, K) == sdq.PATH_DECODE else []) + \
        [sdq.PATH_MFMA, sdq.PATH_SPLITK]
    for path in paths:
        say("partial chunk int", _ids(c), M, N, K, "path", path)
        Y, _, _, _ = run_gpu(X, W, cfg, path)
        check(Y, Yref, X, W, cfg_o, f"{_ids(c)} M={M} N={N} K={K} path={path}")


@pytest.mark.parametrize("fam,M,N,K,kernel", [("int", 400, 8192, 160, "tiled"), ("int", 700, 2048, 288, "split-K"),
                                              ("int", 1000, 8192, 160, "tiled"),
                                              ("mx", 100, 70, 160, "block32"), ("mx", 200, 8192, 288, "block64"),
                                              ("mx", 300, 8192, 160, "block128")])
def test_every_matrix_kernel(fam, M, N, K, kernel):
    assert _kernel_for(fam, M, N) == kernel
    cfg, cfg_o = _cfgs(fam, 1, 8, "e4m3", 3 if fam == "int" else 2)
    X = synth.make_x(6, M, K)
    W = synth.make_w(6, 1, N, K)
    say("partial chunk kernel", fam, kernel, M, N, K)
    Y, _, _, _ = run_gpu(X, W, cfg, path=sdq.PATH_MFMA)
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    check(Y, Yref, X, W, cfg_o, f"{fam} {kernel} M={M} N={N} K={K}")


@pytest.mark.parametrize("c", [MX_CFGS[0], MX_CFGS[1], MX_CFGS[4]], ids=_ids)
@pytest.mark.parametrize("M,N,K", [(1, 96, 160), (33, 300, 288), (600, 544, 288), (520, 2080, 4128)])
def test_mx_paths(c, M, N, K):
    cfg, cfg_o = _cfgs(*c)
    X = synth.make_x(6, M, K)
    W = synth.make_w(6, 2, N, K)
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    paths = [sdq.PATH_MFMA, sdq.PATH_SPLITK] + ([sdq.PATH_DENSE] if c[1] else [])
    for path in paths:
        say("partial chunk mx", _ids(c), M, N, K, "path", path)
        Y, _, _, _ = run_gpu(X, W, cfg, path)
        check(Y, Yref, X, W, cfg_o, f"{_ids(c)} M={M} N={N} K={K} path={path}")


@pytest.mark.parametrize("M,N,K", [(1, 256, 160), (2, 70, 1056), (33, 160, 288), (100, 256, 160),
                                   (300, 16384, 160)])
def test_dual(M, N, K):
    from tests.test_gpu_dual import _cfgs as dual_cfgs, _check, _run
    cfg, cfg_o = dual_cfgs(1, 6)
    X = synth.make_x(6, M, K)
    W = synth.make_w(6, 3, N, K)
    say("partial chunk dual", M, N, K)
    Y, _ = _run(X, W, cfg)
    _check(Y, X, W, cfg_o, f"dual M={M} N={N} K={K}")


@pytest.mark.parametrize("M", [1, 2])
def test_fused_linear(M):
    """sdq_linear (activation quantization inside the decode kernel) with a
    partial last chunk: the codes equal the oracle's, the product its tolerance."""
    torch = torch_cuda()
    cfg, cfg_o = _cfgs(*INT_CFGS[0])
    N, K = 200, 1184
    X = synth.make_x(6, M, K)
    W = synth.make_w(6, 4, N, K)
    Yref, Xq_ref, _, _ = S.reference(X, W, cfg_o)
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    say("partial chunk linear", M)
    Y, Xq, _ = sdq.linear(torch.from_numpy(X).cuda(), blob, N, K, cfg)
    torch.cuda.synchronize()
    assert np.array_equal(Xq.cpu().numpy(), Xq_ref)
    assert_close(Y.cpu().numpy(), Yref, f"linear M={M}")


def test_int_integer_grid_is_exact():
    """Every scale exactly 1 (as in the full-chunk grid test): Y equals the
    int64 product on every INT path with K = 288."""
    rng = np.random.default_rng(11)
    M, N, K = 20, 64, 288
    X = rng.integers(-127, 128, (M, K)).astype(np.float32)
    X[:, 0] = 127.0
    W = rng.integers(-7, 8, (N, K)).astype(np.float32)
    W[:, ::16] = 7.0
    vals = rng.integers(8, 17, (N, K // 8)).astype(np.float32) * rng.choice([-1, 1], (N, K // 8))
    vals[:, 0] = 127.0
    W[:, 3::8] = vals
    W[:, 0] = 7.0
    cfg, cfg_o = _cfgs(*INT_CFGS[1])
    Yref, _, s_ref, L = S.reference(X, W, cfg_o)
    assert (s_ref == 1).all() and (L["scale_o"] == 1).all()
    for path in (sdq.PATH_MFMA, sdq.PATH_SPLITK):
        say("partial chunk grid", path)
        Y, _, _, _ = run_gpu(X, W, cfg, path)
        assert np.array_equal(Y.astype(np.float64), Yref), f"path {path}"
    for Mx in (1, 2):
        Y, _, _, _ = run_gpu(X[:Mx], W, cfg, sdq.PATH_DECODE)
        assert np.array_equal(Y.astype(np.float64), Yref[:Mx]), "decode"
