"""GPU: the decomposed GEMM against the fp64 oracle.

The whole path runs on the library: X -> sdq_quantize_act (GPU), W ->
sdq_pack (host C++) -> sdq_gemm (GPU).  The expected values come from the
oracle alone (``oracle.sdq.reference`` on the same X and W).  Integer-grid
inputs, on which every scale is exactly 1, must come out exact.
"""
import numpy as np
import pytest

import synth
from oracle import sdq as S
from tests.gpu_util import assert_close, assert_close_terms, say, torch_cuda

import paper_2406_13868_amd as sdq

pytestmark = pytest.mark.gpu

INT_CFGS = [("int", 1, 8, "e4m3", 3), ("int", 1, 8, "int8", 3), ("int", 1, 16, "e4m3", 3),
            ("int", 1, 8, "e4m3", 2), ("int", 1, 16, "e4m3", 2), ("int", 0, 8, "e4m3", 3)]
MX_CFGS = [("mx", 1, 8, "e4m3", 2), ("mx", 1, 8, "e4m3", 3), ("mx", 1, 16, "e4m3", 2),
           ("mx", 1, 16, "e4m3", 3), ("mx", 0, 8, "e4m3", 2)]


def _cfgs(fam, n_o, m_o, fmt_o, n_i):
    if fam == "int":
        return (sdq.Config("int", n_o, m_o, fmt_o, n_i, 8, "int4", "int8"),
                S.Config("int", n_o, m_o, fmt_o, n_i, 8, "int4", "int8"))
    return (sdq.Config("mx", n_o, m_o, "e4m3", n_i, 8, "e2m1", "e4m3"),
            S.Config("mx", n_o, m_o, "e4m3", n_i, 8, "e2m1", "e4m3"))


def _ids(c):
    return f"{c[0]}-{c[1]}:{c[2]}{c[3]}+{c[4]}:8"


def run_gpu(X, W, cfg, path=sdq.PATH_AUTO, x_bf16=False):
    torch = torch_cuda()
    N, K = W.shape
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    t = torch.from_numpy(np.ascontiguousarray(X))
    Xd = (t.to(torch.bfloat16) if x_bf16 else t).cuda()
    Xq, s_a = sdq.quantize_act(Xd, cfg)
    Y = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=path)
    torch.cuda.synchronize()
    return Y.cpu().numpy(), Xq, s_a, blob


def abs_terms(X, W, cfg_o, act_norm=None):
    """sum_k |s_a x_k| |w_k| per output (the scale of a dot product's rounding)."""
    Xq, s_a = S.quantize_act(X, cfg_o)
    L = S.pack_logical(W, cfg_o, act_norm)
    A = np.abs(S.dequant_act(Xq, s_a, cfg_o))
    return A @ (np.abs(S.dequant_outliers(L)) + np.abs(S.dequant_inliers(L))).T


def check(Y, Yref, X, W, cfg_o, what="", act_norm=None):
    if cfg_o.family == "mx":
        return assert_close_terms(Y, Yref, abs_terms(X, W, cfg_o, act_norm), W.shape[1], what)
    return assert_close(Y, Yref, what)


def _paths(fam, M, n_o=1):
    if fam == "int":
        return ([sdq.PATH_DECODE] if M <= 8 else []) + [sdq.PATH_MFMA, sdq.PATH_SPLITK]
    if fam == "mx" and n_o:
        return [sdq.PATH_MFMA, sdq.PATH_DENSE, sdq.PATH_SPLITK]
    return [sdq.PATH_MFMA, sdq.PATH_SPLITK]


@pytest.mark.parametrize("c", INT_CFGS + MX_CFGS, ids=_ids)
@pytest.mark.parametrize("M,N,K", [(1, 256, 256), (2, 96, 384), (3, 50, 256), (5, 256, 512),
                                   (8, 64, 128), (16, 256, 256), (17, 100, 384), (33, 160, 256),
                                   (64, 256, 512), (100, 70, 256), (130, 129, 384)])
def test_gemm_matches_oracle(c, M, N, K):
    cfg, cfg_o = _cfgs(*c)
    X = synth.make_x(1, M, K)
    W = synth.make_w(1, 0, N, K)
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    for path in _paths(c[0], M, c[1]):
        say("gemm", _ids(c), M, N, K, "path", path)
        Y, _, _, _ = run_gpu(X, W, cfg, path)
        check(Y, Yref, X, W, cfg_o, f"{_ids(c)} M={M} N={N} K={K} path={path}")


@pytest.mark.parametrize("c", [MX_CFGS[0], MX_CFGS[1], MX_CFGS[3]], ids=_ids)
@pytest.mark.parametrize("M,N,K", [(512, 256, 256), (600, 100, 384), (777, 544, 128),
                                   (1030, 288, 640), (4100, 4128, 128)])
def test_mx_many_rows(c, M, N, K):
    """Row counts of large prefill batches: several token blocks, a ragged last
    block, column groups of 32-wide tiles with a ragged last group, and odd and
    single chunk counts along K, on both matrix-core paths."""
    cfg, cfg_o = _cfgs(*c)
    X = synth.make_x(3, M, K)
    W = synth.make_w(3, 1, N, K)
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    for path in (sdq.PATH_AUTO, sdq.PATH_MFMA):
        say("mx rows", _ids(c), M, N, K, "path", path)
        Y, _, _, _ = run_gpu(X, W, cfg, path)
        check(Y, Yref, X, W, cfg_o, f"{_ids(c)} M={M} N={N} K={K} path={path}")


@pytest.mark.parametrize("c", [MX_CFGS[0], MX_CFGS[1], MX_CFGS[2], MX_CFGS[3]], ids=_ids)
@pytest.mark.parametrize("M,N,K", [(1, 64, 256), (40, 100, 384), (256, 288, 640), (300, 544, 128),
                                   (4096, 4096, 256)])
def test_dense_equals_one_pass(c, M, N, K):
    """Where every block merges its inliers the two-pass path runs the same
    matrix instructions per accumulator in the same order as the one-pass
    kernel: the outputs agree bit for bit (one workgroup per CU below 512
    workgroups, two from there)."""
    cfg, cfg_o = _cfgs(*c)
    X = synth.make_x(3, M, K)
    W = synth.make_w(3, 2, N, K)
    L = S.pack_logical(W, cfg_o)
    d = L["scale_i"].astype(int) - L["scale_o"].astype(int)
    assert not np.any((d < -5) | (d > 6)), "the case holds an unmergeable block"
    torch = torch_cuda()
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    Xq, s_a = sdq.quantize_act(torch.from_numpy(X).cuda(), cfg)
    say("dense vs one pass", _ids(c), M, N, K)
    Y1 = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=sdq.PATH_MFMA)
    ws = torch.full((sdq.gemm_workspace_size(cfg, M, N, K, sdq.PATH_DENSE),), 0xAB,
                    dtype=torch.uint8, device="cuda")  # stale contents must not matter
    Y2 = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=sdq.PATH_DENSE, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(Y1.view(torch.int32), Y2.view(torch.int32))


def _int_grid(rng, M, N, K, outlier_fmt):
    """Inputs on which every scale is exactly 1 (act, inlier and outlier)."""
    X = rng.integers(-127, 128, (M, K)).astype(np.float32)
    X[:, 0] = 127.0
    W = rng.integers(-7, 8, (N, K)).astype(np.float32)
    W[:, ::16] = 7.0                              # every 16-block: inlier amax 7
    big = 127.0 if outlier_fmt == "int8" else 448.0
    vals = rng.integers(8, 17, (N, K // 8)).astype(np.float32)  # exact in e4m3 and int8
    vals *= rng.choice([-1, 1], (N, K // 8))
    vals[:, 0] = big                              # row amax of the outliers
    W[:, 3::8] = vals                             # the largest of each 8-group
    W[:, 0] = 7.0
    return X, W


@pytest.mark.parametrize("fmt_o", ["int8", "e4m3"])
@pytest.mark.parametrize("M,N,K", [(1, 64, 4096), (2, 32, 1024), (16, 96, 1024), (64, 64, 4096),
                                   (400, 8192, 128)])
def test_integer_grid_is_exact(fmt_o, M, N, K):
    cfg, cfg_o = _cfgs("int", 1, 8, fmt_o, 3)
    rng = np.random.default_rng(M * 7 + N)
    X, W = _int_grid(rng, M, N, K, fmt_o)
    Yref, Xq_ref, s_ref, L = S.reference(X, W, cfg_o)
    assert (s_ref == 1).all() and (L["scale_i"] == 1).all() and (L["scale_o"] == 1).all()
    P_i, P_o = S.int_partials(Xq_ref, L)
    if fmt_o == "int8":
        exact = P_i.sum(-1) + P_o
        assert np.array_equal(Yref, exact.astype(np.float64))
    for path in _paths("int", M):
        say("int grid", fmt_o, M, N, K, "path", path)
        Y, _, _, _ = run_gpu(X, W, cfg, path)
        assert np.array_equal(Y.astype(np.float64), Yref), f"path {path}: not exact"


@pytest.mark.parametrize("M,N,K", [(32, 64, 1024), (100, 96, 512)])
def test_mx_grid_is_exact(M, N, K):
    cfg, cfg_o = _cfgs("mx", 1, 8, "e4m3", 2)
    rng = np.random.default_rng(5)
    X = rng.integers(-16, 17, (M, K)).astype(np.float32)
    X[:, 0] = 448.0                                   # s_a = 1, inv = 1
    W = rng.choice([-3.0, -2.0, -1.0, 1.0, 2.0, 3.0], (N, K)).astype(np.float32)
    W[:, ::32] = 4.0                                  # inlier block amax in [4, 8): E = 0
    W[:, 5::8] = (256 + 32 * rng.integers(0, 7, (N, K // 8))).astype(np.float32)  # e4m3-exact outliers, E = 0
    Yref, _, s_ref, L = S.reference(X, W, cfg_o)
    assert (s_ref == 1).all() and (L["scale_i"] == 127).all() and (L["scale_o"] == 127).all()
    for path in (sdq.PATH_MFMA, sdq.PATH_DENSE):
        say("mx grid", M, N, K, "path", path)
        Y, _, _, _ = run_gpu(X, W, cfg, path)
        assert np.array_equal(Y.astype(np.float64), Yref), f"path {path}"


@pytest.mark.parametrize("c", [INT_CFGS[0], MX_CFGS[0]], ids=_ids)
def test_degenerate_inputs(c):
    torch = torch_cuda()
    cfg, cfg_o = _cfgs(*c)
    X = synth.make_x(1, 20, 256)
    X[3] = 0.0
    W = synth.make_w(1, 0, 64, 256)
    W[10] = 0.0
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    say("degenerate", _ids(c))
    for path in _paths(c[0], 1):
        Xs = X[:1] if path == sdq.PATH_DECODE else X
        Y, _, _, _ = run_gpu(Xs, W, cfg, path)
        check(Y, Yref[: len(Xs)], Xs, W, cfg_o)
        assert (Y[:, 10] == 0).all()
    Y, _, _, _ = run_gpu(X, W, cfg)
    assert (Y[3] == 0).all()
    # all-zero weights
    Y, _, _, _ = run_gpu(X, np.zeros_like(W), cfg)
    assert (Y == 0).all()
    # M = 0
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    Xq = torch.zeros((0, 256), dtype=torch.uint8, device="cuda")
    s_a = torch.zeros((0,), dtype=torch.float32, device="cuda")
    for path in _paths(c[0], 0, c[1]):
        Y = sdq.gemm(Xq, s_a, blob, 64, 256, cfg, path=path)
        torch.cuda.synchronize()
        assert Y.shape == (0, 64)


@pytest.mark.parametrize("c", [INT_CFGS[0], INT_CFGS[1], MX_CFGS[0]], ids=_ids)
def test_repeat_runs_are_bit_identical(c):
    cfg, _ = _cfgs(*c)
    X = synth.make_x(2, 64, 1024)
    W = synth.make_w(2, 0, 512, 1024)
    for path in _paths(c[0], 2):
        say("determinism", _ids(c), path)
        Xs = X[:2] if path == sdq.PATH_DECODE else X
        Y0, _, _, _ = run_gpu(Xs, W, cfg, path)
        for _ in range(3):
            Y1, _, _, _ = run_gpu(Xs, W, cfg, path)
            assert np.array_equal(Y0.view(np.uint32), Y1.view(np.uint32))


def test_quantized_activations_feed_gemm_like_oracle():
    """The oracle's own Xq/s_a fed to the GPU GEMM give the same Y as the GPU's."""
    torch = torch_cuda()
    cfg, cfg_o = _cfgs(*INT_CFGS[0])
    X = synth.make_x(1, 16, 256)
    W = synth.make_w(1, 0, 256, 256)
    Yref, Xq_ref, s_ref, _ = S.reference(X, W, cfg_o)
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    Y = sdq.gemm(torch.from_numpy(Xq_ref).cuda(), torch.from_numpy(s_ref).cuda(), blob, 256, 256, cfg)
    torch.cuda.synchronize()
    assert_close(Y.cpu().numpy(), Yref)
    Y2, _, _, _ = run_gpu(X, W, cfg)
    assert np.array_equal(Y.cpu().numpy(), Y2)


def _kernel_for(fam, M, N):
    """Which matrix-core kernel the launcher picks above 64 tokens (the cost
    model the kernels' launchers state): INT "tiled" (128-token blocks, two
    workgroups per CU) when its grid of w4 = ceil(N/128) x ceil(M/128)
    workgroups, at 1.7 units of time per full round of 512 plus 1.7 for a
    last round of more than 256, or for at most 256 1 unit alone and 0.65
    after a full round, is faster than the split-K form at w4/200 units, else
    "split-K"; MX token blocks of 32, 64 or 128 (the largest whose grid stays
    within one round of 256 workgroups)."""
    groups = -(-N // 128)
    if fam == "int":
        w4 = groups * -(-M // 128)
        full, rem = divmod(w4, 512)
        tail20 = 0 if rem == 0 else 34 if rem > 256 else 13 if full else 20
        return "split-K" if w4 < 10 * (34 * full + tail20) else "tiled"
    if groups * -(-M // 32) <= 256:
        return "block32"
    if groups * -(-M // 64) <= 256:
        return "block64"
    return "block128"


@pytest.mark.parametrize("fam,M,N,K,kernel", [("int", 100, 70, 256, "split-K"), ("int", 384, 8192, 256, "split-K"),
                                              ("int", 400, 8192, 128, "tiled"), ("int", 700, 2048, 128, "split-K"),
                                              ("int", 1000, 8192, 128, "tiled"), ("int", 770, 16384, 256, "tiled"),
                                              ("int", 1300, 8192, 128, "tiled"),
                                              ("mx", 100, 70, 256, "block32"), ("mx", 200, 8192, 256, "block64"),
                                              ("mx", 300, 8192, 128, "block128")])
def test_every_matrix_kernel_above_64_tokens(fam, M, N, K, kernel):
    """Shapes that take each matrix-core kernel and token block past 64 tokens, ragged M."""
    assert _kernel_for(fam, M, N) == kernel
    cfg, cfg_o = _cfgs(fam, 1, 8, "e4m3", 3 if fam == "int" else 2)
    X = synth.make_x(1, M, K)
    W = synth.make_w(1, 0, N, K)
    say("kernel", fam, kernel, M, N, K)
    Y, _, _, _ = run_gpu(X, W, cfg, path=sdq.PATH_MFMA)
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    check(Y, Yref, X, W, cfg_o, f"{fam} {kernel} M={M} N={N} K={K}")


@pytest.mark.parametrize("c", [INT_CFGS[0], INT_CFGS[1], MX_CFGS[0]], ids=_ids)
@pytest.mark.parametrize("M", [1, 4, 64])
def test_concatenated_projections_equal_separate(c, M):
    """q, k and v stacked along N in one launch give the three separate
    launches' outputs: bit for bit on the decode path (whose per-output
    arithmetic does not depend on N), to the oracle's tolerance otherwise."""
    torch = torch_cuda()
    cfg, cfg_o = _cfgs(*c)
    N, K = 160, 1024
    X = synth.make_x(2, M, K)
    Ws = [synth.make_w(2, j, N, K) for j in range(3)]
    say("qkv concat", _ids(c), M)
    Yc, Xq, s_a, _ = run_gpu(X, np.concatenate(Ws), cfg)
    for j, W in enumerate(Ws):
        blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
        Yj = sdq.gemm(Xq, s_a, blob, N, K, cfg).cpu().numpy()
        if c[0] == "int" and M <= 8:
            assert np.array_equal(Yc[:, j * N:(j + 1) * N].view(np.uint32), Yj.view(np.uint32))
        Yref, _, _, _ = S.reference(X, W, cfg_o)
        check(Yc[:, j * N:(j + 1) * N], Yref, X, W, cfg_o, f"projection {j}")


@pytest.mark.parametrize("M", [1, 2])
def test_stacked_gate_up_equals_separate_full_size(M):
    """The LLaMA-7B gate and up projections (11008 x 4096 each) stacked into
    one launch of 22016 rows: every output equals the two separate launches'
    bit for bit on the decode path, and the oracle's within the tolerance."""
    torch = torch_cuda()
    cfg, cfg_o = _cfgs(*INT_CFGS[0])
    N, K = 11008, 4096
    X = synth.make_x(8, M, K)
    Ws = [synth.make_w(8, j, N, K) for j in range(2)]
    say("gate/up stacked", M)
    Yc, Xq, s_a, _ = run_gpu(X, np.concatenate(Ws), cfg, path=sdq.PATH_DECODE, x_bf16=True)
    for j, W in enumerate(Ws):
        blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
        Yj = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=sdq.PATH_DECODE).cpu().numpy()
        assert np.array_equal(Yc[:, j * N:(j + 1) * N].view(np.uint32), Yj.view(np.uint32))
        Yref, _, _, _ = S.reference(X, W, cfg_o)  # X holds bf16 values already
        check(Yc[:, j * N:(j + 1) * N], Yref, X, W, cfg_o, f"gate/up projection {j}")


@pytest.mark.parametrize("c", [INT_CFGS[0], INT_CFGS[1], INT_CFGS[4], MX_CFGS[0]], ids=_ids)
@pytest.mark.parametrize("M,dt", [(1, "bf16"), (2, "f32"), (3, "bf16"), (4, "f32"), (16, "bf16")])
def test_linear_equals_quantize_then_gemm(c, M, dt):
    """sdq_linear (one fused kernel on the decode path) == the two-call path, bit for bit."""
    torch = torch_cuda()
    cfg, cfg_o = _cfgs(*c)
    N, K = 300, 1024
    X = synth.bf16_round(synth.make_x(2, M, K))
    W = synth.make_w(2, 0, N, K)
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    Xd = torch.from_numpy(X).cuda()
    if dt == "bf16":
        Xd = Xd.to(torch.bfloat16)
    say("linear", _ids(c), M, dt)
    Y1, Xq1, s1 = sdq.linear(Xd, blob, N, K, cfg)
    Xq2, s2 = sdq.quantize_act(Xd, cfg)
    Y2 = sdq.gemm(Xq2, s2, blob, N, K, cfg)
    torch.cuda.synchronize()
    assert torch.equal(Xq1, Xq2) and torch.equal(s1.view(torch.int32), s2.view(torch.int32))
    assert torch.equal(Y1.view(torch.int32), Y2.view(torch.int32))
    Yref, Xq_ref, _, _ = S.reference(X, W, cfg_o)
    assert np.array_equal(Xq1.cpu().numpy(), Xq_ref)
    check(Y1.cpu().numpy(), Yref, X, W, cfg_o)


@pytest.mark.parametrize("c", [INT_CFGS[0], MX_CFGS[0]], ids=_ids)
def test_hip_graph_replays_match_eager(c):
    """The step captured in a HIP graph gives the eager result on every replay."""
    torch = torch_cuda()
    cfg, _ = _cfgs(*c)
    N, K, M = 512, 1024, (1 if c[0] == "int" else 64)
    X = torch.from_numpy(synth.make_x(2, M, K)).cuda().to(torch.bfloat16)
    blob = torch.from_numpy(sdq.pack(synth.make_w(2, 0, N, K), cfg)).cuda()
    Y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    Xq = torch.empty((M, K), dtype=torch.uint8, device="cuda")
    s_a = torch.empty((M,), dtype=torch.float32, device="cuda")
    say("graph", _ids(c))
    sdq.linear(X, blob, N, K, cfg, out=Y, xq=Xq, scales=s_a)
    torch.cuda.synchronize()
    ref = Y.clone()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        sdq.linear(X, blob, N, K, cfg, out=Y, xq=Xq, scales=s_a)
    torch.cuda.current_stream().wait_stream(side)
    with torch.cuda.graph(g):
        sdq.linear(X, blob, N, K, cfg, out=Y, xq=Xq, scales=s_a)
    for rep in range(4):
        Y.fill_(float("nan"))
        Xq.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y.view(torch.int32), ref.view(torch.int32)), f"replay {rep}"
        # eager work in between
        sdq.gemm(Xq, s_a, blob, N, K, cfg, out=torch.empty_like(Y))
        torch.cuda.synchronize()


@pytest.mark.parametrize("which", ["mx-dense", "int-splitk", "mx-splitk"])
def test_hip_graph_replays_match_eager_two_pass(which):
    """The workspace paths (two-pass MX, INT and MX split-K; workspace
    allocated before capture) replay like eager, whatever the workspace held."""
    torch = torch_cuda()
    if which == "mx-dense":
        cfg, _ = _cfgs(*MX_CFGS[1])
        N, K, M, path = 544, 640, 600, sdq.PATH_DENSE
    elif which == "mx-splitk":
        cfg, _ = _cfgs(*MX_CFGS[1])
        N, K, M, path = 1000, 2304, 200, sdq.PATH_SPLITK
    else:
        cfg, _ = _cfgs(*INT_CFGS[1])
        N, K, M, path = 1000, 2304, 100, sdq.PATH_SPLITK
    X = torch.from_numpy(synth.make_x(2, M, K)).cuda()
    blob = torch.from_numpy(sdq.pack(synth.make_w(2, 0, N, K), cfg)).cuda()
    Xq, s_a = sdq.quantize_act(X, cfg)
    ws = torch.empty(sdq.gemm_workspace_size(cfg, M, N, K, path), dtype=torch.uint8, device="cuda")
    Y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    say("graph two-pass", which)
    sdq.gemm(Xq, s_a, blob, N, K, cfg, out=Y, path=path, workspace=ws)
    torch.cuda.synchronize()
    ref = Y.clone()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        sdq.gemm(Xq, s_a, blob, N, K, cfg, out=Y, path=path, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    with torch.cuda.graph(g):
        sdq.gemm(Xq, s_a, blob, N, K, cfg, out=Y, path=path, workspace=ws)
    for rep in range(4):
        Y.fill_(float("nan"))
        ws.fill_(0x5A)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y.view(torch.int32), ref.view(torch.int32)), f"replay {rep}"
        sdq.gemm(Xq, s_a, blob, N, K, cfg, out=torch.empty_like(Y), path=path, workspace=ws)
        torch.cuda.synchronize()


@pytest.mark.parametrize("c", [INT_CFGS[0], INT_CFGS[1], INT_CFGS[3], INT_CFGS[5]], ids=_ids)
@pytest.mark.parametrize("M,N,K", [(9, 4128, 512), (31, 300, 2560), (33, 97, 4096), (64, 1000, 16384),
                                   (100, 544, 1152), (129, 64, 8192), (200, 2080, 640), (256, 33, 128),
                                   (100, 8200, 384), (300, 544, 2560), (520, 200, 4160)])
def test_split_k_ragged_shapes(c, M, N, K):
    """The split-K path on token counts around its 32- and 64-token blocks,
    row counts that leave a part of a 128-row group, K ranges from one chunk
    to 128 (1 to 32 ranges), against the oracle; and its tiled form over K
    ranges (128-token blocks: 129 x 64 x 8192 in 16 ranges, 100 x 8200 x 384
    in one, 300 x 544 x 2560 in 5, 520 x 200 x 4160 in 7 with a partial last
    chunk)."""
    cfg, cfg_o = _cfgs(*c)
    X = synth.make_x(4, M, K)
    W = synth.make_w(4, 3, N, K)
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    say("split-K ragged", _ids(c), M, N, K)
    Y, _, _, _ = run_gpu(X, W, cfg, sdq.PATH_SPLITK)
    check(Y, Yref, X, W, cfg_o, f"{_ids(c)} M={M} N={N} K={K} split-K")


@pytest.mark.parametrize("c", [MX_CFGS[0], MX_CFGS[1], MX_CFGS[4]], ids=_ids)
@pytest.mark.parametrize("M,N,K", [(9, 4128, 512), (33, 97, 4096), (64, 1000, 16384), (100, 544, 1152),
                                   (129, 64, 8192), (256, 4096, 4096), (300, 2080, 640), (511, 33, 1024)])
def test_mx_split_k_ragged_shapes(c, M, N, K):
    """The MX family's split-K path on shapes that give 1 to 32 K ranges,
    every token block and ragged tiles, against the oracle."""
    cfg, cfg_o = _cfgs(*c)
    X = synth.make_x(4, M, K)
    W = synth.make_w(4, 4, N, K)
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    say("mx split-K ragged", _ids(c), M, N, K)
    Y, _, _, _ = run_gpu(X, W, cfg, sdq.PATH_SPLITK)
    check(Y, Yref, X, W, cfg_o, f"{_ids(c)} M={M} N={N} K={K} mx split-K")


def _split_case(kind, N, K, rng):
    """MX weights whose blocks cannot merge the inliers into the outliers' e4m3
    fragment (inlier/outlier exponent difference outside [-5, 6])."""
    W = synth.make_w(1, 0, N, K).copy()
    an = None
    if kind == "product":          # inliers may exceed the outliers
        an = np.abs(rng.standard_normal(K)).astype(np.float32) * 10.0
    elif kind == "zero_inliers":   # blocks holding only their outliers
        blk = rng.random((N, K // 32)) < 0.3
        keep = np.zeros((N, K), bool)
        for n, b in zip(*np.nonzero(blk)):
            seg = W[n, 32 * b:32 * b + 32]
            top = np.argsort(-np.abs(seg.reshape(4, 8)), axis=1, kind="stable")[:, 0] + np.arange(4) * 8
            mask = np.zeros(32, bool)
            mask[top] = True
            W[n, 32 * b:32 * b + 32] = np.where(mask, seg, 0.0)
    elif kind == "huge_outliers":  # outliers 2^13 times the block's inliers
        W[:, 5::8] = np.sign(W[:, 5::8] + 1e-9) * 8192.0 * np.abs(W).max()
    return W, an


@pytest.mark.parametrize("kind", ["product", "zero_inliers", "huge_outliers"])
@pytest.mark.parametrize("n_i", [2, 3])
@pytest.mark.parametrize("M,N,K", [(64, 96, 512), (256, 64, 1024), (520, 96, 384)])
@pytest.mark.parametrize("path", [sdq.PATH_MFMA, sdq.PATH_DENSE, sdq.PATH_SPLITK])
def test_mx_unmergeable_blocks(kind, n_i, M, N, K, path):
    """The matrix kernel's correction path for blocks that stay split."""
    rng = np.random.default_rng(7)
    metric = "product" if kind == "product" else "magnitude"
    cfg = sdq.Config("mx", 1, 8, "e4m3", n_i, 8, "e2m1", "e4m3", metric)
    cfg_o = S.Config("mx", 1, 8, "e4m3", n_i, 8, "e2m1", "e4m3", metric)
    W, an = _split_case(kind, N, K, rng)
    X = synth.make_x(1, M, K)
    # the case must contain unmergeable blocks, or it tests nothing
    L = S.pack_logical(W, cfg_o, an)
    d = L["scale_i"].astype(int) - L["scale_o"].astype(int)
    assert np.any((d < -5) | (d > 6)), "no unmergeable block in the case"
    say("mx split", kind, n_i, M, N, K, "path", path)
    torch = torch_cuda()
    blob = torch.from_numpy(sdq.pack(W, cfg, act_norm=an)).cuda()
    Xq, s_a = sdq.quantize_act(torch.from_numpy(X).cuda(), cfg)
    Y = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=path).cpu().numpy()
    Yref, _, _, _ = S.reference(X, W, cfg_o, an)
    A = np.abs(S.dequant_act(*S.quantize_act(X, cfg_o), cfg_o))
    T = A @ (np.abs(S.dequant_outliers(L)) + np.abs(S.dequant_inliers(L))).T
    assert_close_terms(Y, Yref, T, K, f"{kind} n_i={n_i} M={M}")


@pytest.mark.parametrize("fam,fmt_o,decomp,order", [("int", "e4m3", "output_error", "small"),
                                                    ("int", "int8", "error", "large"),
                                                    ("mx", "e4m3", "product", "small"),
                                                    ("mx", "e4m3", "error", "large")])
def test_decomposition_variants_end_to_end(fam, fmt_o, decomp, order):
    """Weights packed with another decomposition metric and order (Section 6.4's
    decomposition study) go through the same kernels: the GEMM matches the
    oracle's product of its own decomposition on every path."""
    import dataclasses
    torch = torch_cuda()
    cfg, cfg_o = _cfgs(fam, 1, 8, fmt_o, 3 if fam == "int" else 2)
    cfg = dataclasses.replace(cfg, metric="product", decomp=decomp, order=order)
    cfg_o = dataclasses.replace(cfg_o, metric="product", decomp=decomp, order=order)
    N, K = 96, 384
    W = synth.make_w(1, 0, N, K)
    an = S.activation_norm(synth.make_x(2, 64, K))  # calibration tokens
    blob = torch.from_numpy(sdq.pack(W, cfg, act_norm=an)).cuda()
    cases = [(M, path) for M in (4, 40) for path in _paths(fam, M, 1)]
    for M, path in cases:
        X = synth.make_x(1, M, K)
        Yref = S.reference(X, W, cfg_o, act_norm=an)[0]
        Xq, s_a = sdq.quantize_act(torch.from_numpy(X).cuda(), cfg)
        say("variant", fam, fmt_o, decomp, order, M, N, K, "path", path)
        ws = None
        if path == sdq.PATH_DENSE:
            ws = torch.empty(sdq.gemm_workspace_size(cfg, M, N, K, path), dtype=torch.uint8,
                             device="cuda")
        Y = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=path, workspace=ws)
        torch.cuda.synchronize()
        check(Y.cpu().numpy(), Yref, X, W, cfg_o, f"{fam} {decomp} {order} M={M} path={path}", an)


# ---- two-level e4m3 inlier scales (Section 3.3: quantized scale factors)
SC8_CFGS = [("int", 1, 8, "e4m3", 3), ("int", 1, 8, "int8", 3), ("int", 1, 16, "e4m3", 2),
            ("int", 0, 8, "e4m3", 3)]


def _sc8(c):
    import dataclasses
    cfg, cfg_o = _cfgs(*c)
    return dataclasses.replace(cfg, sfmt_i="e4m3"), dataclasses.replace(cfg_o, sfmt_i="e4m3")


@pytest.mark.parametrize("c", SC8_CFGS, ids=_ids)
@pytest.mark.parametrize("M,N,K", [(1, 256, 256), (2, 96, 384), (5, 256, 512), (8, 64, 128),
                                   (16, 256, 256), (33, 160, 256), (64, 256, 2048),
                                   (100, 70, 256), (130, 129, 384)])
def test_e4m3_scales_match_oracle(c, M, N, K):
    cfg, cfg_o = _sc8(c)
    X = synth.make_x(1, M, K)
    W = synth.make_w(1, 0, N, K)
    W[min(3, N - 1), :] = 0.0                     # a row without inliers: row scale 0
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    for path in _paths("int", M):
        say("e4m3 scales", _ids(c), M, N, K, "path", path)
        Y, _, _, _ = run_gpu(X, W, cfg, path)
        check(Y, Yref, X, W, cfg_o, f"e4m3 scales {_ids(c)} M={M} N={N} K={K} path={path}")


@pytest.mark.parametrize("fmt_o", ["int8", "e4m3"])
@pytest.mark.parametrize("M,N,K", [(1, 64, 4096), (16, 96, 1024), (64, 64, 4096), (96, 64, 512)])
def test_e4m3_scales_integer_grid_is_exact(fmt_o, M, N, K):
    """With every inlier block's amax 7 the two-level scale is e4m3(256) * 2^-8 = 1
    exactly, so the integer grid must still come out exact."""
    cfg, cfg_o = _sc8(("int", 1, 8, fmt_o, 3))
    rng = np.random.default_rng(M * 5 + N)
    X, W = _int_grid(rng, M, N, K, fmt_o)
    Yref, _, s_ref, L = S.reference(X, W, cfg_o)
    assert (s_ref == 1).all() and (S.inlier_scale_values(L) == 1).all()
    for path in _paths("int", M):
        say("e4m3 scales grid", fmt_o, M, N, K, "path", path)
        Y, _, _, _ = run_gpu(X, W, cfg, path)
        assert np.array_equal(Y.astype(np.float64), Yref), f"path {path}: not exact"


@pytest.mark.parametrize("M,layer", [(1, 0), (64, 0), (64, 1)])
def test_e4m3_scales_full_size_layers(M, layer):
    """OPT-6.7B FFN shapes (fc1 16384x4096, fc2 4096x16384) with e4m3 scales,
    every output against the oracle."""
    cfg, cfg_o = _sc8(("int", 1, 8, "int8", 3))
    L = synth.WORKLOADS[4].layers[layer]
    X = synth.make_x(4, M, L.K)
    W = synth.make_w(4, layer, L.N, L.K)
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    say("e4m3 scales full", M, L.N, L.K)
    Y, _, _, _ = run_gpu(X, W, cfg, sdq.PATH_AUTO, x_bf16=True)
    check(Y, Yref, X, W, cfg_o, f"e4m3 scales full M={M} {L.N}x{L.K}")


@pytest.mark.parametrize("M", [1, 2])
def test_e4m3_scales_fused_linear(M):
    """sdq_linear (quantize fused into the decode GEMM) with e4m3 scales."""
    torch = torch_cuda()
    cfg, cfg_o = _sc8(("int", 1, 8, "e4m3", 3))
    N, K = 256, 1024
    X = synth.make_x(2, M, K)
    W = synth.make_w(2, 0, N, K)
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    say("e4m3 scales linear", M, N, K)
    Y, _, _ = sdq.linear(torch.from_numpy(X).cuda(), blob, N, K, cfg)
    torch.cuda.synchronize()
    check(Y.cpu().numpy(), Yref, X, W, cfg_o, f"e4m3 scales linear M={M}")
