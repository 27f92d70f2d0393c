"""GPU: the dual family (Section 5.1's worked configuration: int8 outliers
against int8 activations A_o, fp4 inliers against fp4 activations A_i)
against the fp64 oracle.

X -> sdq_quantize_act_dual (GPU) -> A_o, A_i; W -> sdq_pack (host) ->
sdq_gemm_dual (GPU).  The expected values come from the oracle alone.

Tolerance: the outlier branch is exact in int32.  The inlier branch runs
gfx950's scaled fp4 x fp4 matrix instruction, which adds its products to the
fp32 accumulator as partial sums of 32 K, each rounded to nearest even; inside
a scale block every fp4 x fp4 product is exact in the instruction's window
(tests/gpu_util.py, dual_term_tol).  An output is therefore off by at most
(K/32 + 2) * 2^-24 of the sum of |terms|, and 1e-3 normwise.
"""
import numpy as np
import pytest

import synth
from oracle import sdq as S
from tests.gpu_util import REL_TOL, dual_term_tol, rel_errors, say, torch_cuda

import paper_2406_13868_amd as sdq

pytestmark = pytest.mark.gpu

def _cfgs(n_o=1, n_i=6, metric="magnitude"):
    return (sdq.Config("dual", n_o, 8, "int8", n_i, 8, "e2m1", "int8", metric),
            S.Config("dual", n_o, 8, "int8", n_i, 8, "e2m1", "int8+e2m1", metric))


def _run(X, W, cfg, x_bf16=False):
    torch = torch_cuda()
    N, K = W.shape
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    t = torch.from_numpy(np.ascontiguousarray(X))
    Xd = (t.to(torch.bfloat16) if x_bf16 else t).cuda()
    Xo, s_a, Xi, Ea = sdq.quantize_act_dual(Xd, cfg)
    Y = sdq.gemm_dual(Xo, s_a, Xi, Ea, blob, N, K, cfg)
    torch.cuda.synchronize()
    return Y.cpu().numpy(), (Xo.cpu().numpy(), s_a.cpu().numpy(), Xi.cpu().numpy(), Ea.cpu().numpy())


def _nibbles(Ai):
    """[M, K] codes -> [M, K/2] bytes, the even k in the low nibble."""
    return (Ai[:, 0::2] | (Ai[:, 1::2] << 4)).astype(np.uint8)


def _check(Y, X, W, cfg_o, what):
    Yref, (Ao, Ai), (s_ao, Ea), L = S.reference(X, W, cfg_o)
    A_o, A_i = S.dequant_act_dual(Ao, s_ao, Ai, Ea)
    T = np.abs(A_o) @ np.abs(S.dequant_outliers(L)).T + np.abs(A_i) @ np.abs(S.dequant_inliers(L)).T
    _, nr = rel_errors(Y, Yref)
    comp = float(np.max(np.abs(Y - Yref) / np.maximum(T, 1e-30))) if Y.size else 0.0
    say(f"{what}: norm_rel={nr:.3e} term_rel={comp:.3e}")
    assert nr <= REL_TOL and comp <= dual_term_tol(W.shape[1]), f"{what}: norm_rel={nr:.3e} term_rel={comp:.3e}"


@pytest.mark.parametrize("M,K", [(1, 128), (5, 256), (64, 4096), (33, 1024),
                                 (300, 512), (1, 4096), (2, 11008), (1, 16384)])
@pytest.mark.parametrize("bf16", [False, True])
def test_act_quant_dual_bit_exact(M, K, bf16):
    rng = np.random.default_rng(M + K)
    X = synth.make_x(2, M, K)
    # rounding boundaries of e2m1 at E = 0: block 0 of every row has amax 6
    if K >= 64:
        X[:, :32] = rng.choice([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, -0.25, -5.0, 0.0, -0.0, 6.0],
                               (M, 32)).astype(np.float32)
        X[:, 0] = 6.0
    if M > 2:
        X[1, :] = 0.0                              # an all-zero token
        X[2, 32:64] = 0.0                          # an all-zero block
    cfg, _ = _cfgs()
    torch = torch_cuda()
    if bf16:  # the oracle quantizes the values the GPU reads
        X = torch.from_numpy(X).to(torch.bfloat16).float().numpy()
    t = torch.from_numpy(X)
    say("act quant dual", M, K, "bf16" if bf16 else "f32")
    Xo, s_a, Xi, Ea = sdq.quantize_act_dual((t.to(torch.bfloat16) if bf16 else t).cuda(), cfg)
    torch.cuda.synchronize()
    Ao_r, s_r, Ai_r, Ea_r = S.quantize_act_dual(X)
    assert np.array_equal(Xo.cpu().numpy(), Ao_r)
    assert np.array_equal(s_a.cpu().numpy().view(np.uint32), s_r.view(np.uint32))
    assert np.array_equal(Xi.cpu().numpy(), _nibbles(Ai_r))
    assert np.array_equal(Ea.cpu().numpy(), Ea_r)


@pytest.mark.parametrize("n_o,n_i", [(1, 6), (1, 3), (0, 7), (1, 7), (2, 4), (2, 6), (2, 1)])
@pytest.mark.parametrize("M,N,K", [(1, 256, 256), (5, 96, 384), (33, 160, 256), (64, 256, 2048),
                                   (100, 70, 256), (130, 129, 384), (300, 544, 128)])
def test_gemm_dual_matches_oracle(n_o, n_i, M, N, K):
    cfg, cfg_o = _cfgs(n_o, n_i)
    X = synth.make_x(2, M, K)
    W = synth.make_w(2, 0, N, K)
    say("gemm dual", n_o, n_i, M, N, K)
    Y, _ = _run(X, W, cfg)
    _check(Y, X, W, cfg_o, f"dual {n_o}:8+{n_i}:8 M={M} N={N} K={K}")


@pytest.mark.parametrize("n_o,n_i", [(1, 6), (2, 4)])
@pytest.mark.parametrize("M", [1, 2])
@pytest.mark.parametrize("N,K", [(256, 128), (70, 256), (544, 1152), (96, 4096), (40, 11008), (96, 6144)])
def test_gemm_dual_decode_matches_oracle(M, N, K, n_o, n_i):
    """One and two tokens (the vector decode kernel; two tokens at K = 11008
    exceed its register budget and take the matrix kernel): one chunk of K
    (half the lanes idle), ragged N, parts of K from one to eight; 1:8 and
    2:8 outliers."""
    cfg, cfg_o = _cfgs(n_o, n_i)
    X = synth.make_x(2, M, K)
    W = synth.make_w(2, 0, N, K)
    say("gemm dual decode", M, N, K)
    Y, _ = _run(X, W, cfg)
    _check(Y, X, W, cfg_o, f"dual decode M={M} N={N} K={K}")


def test_gemm_dual_decode_grid_is_exact():
    """The integer grid of test_gemm_dual_integer_grid_is_exact at one and two tokens."""
    rng = np.random.default_rng(9)
    N, K = 64, 512
    for M in (1, 2):
        X = rng.choice([-6.0, -4.0, -2.0, -1.0, 0.0, 1.0, 2.0, 3.0, 4.0, 6.0], (M, K)).astype(np.float32)
        X[:, 0] = 127.0
        X[:, 1:32] = rng.choice([-64.0, -32.0, 0.0, 32.0, 64.0, 96.0], (M, 31))
        W = rng.choice([-6.0, -3.0, -1.0, 1.0, 2.0, 4.0, 6.0], (N, K)).astype(np.float32)
        W[:, ::8] = 127.0 * rng.choice([-1.0, 1.0], (N, K // 8))
        W[:, 1::32] = 6.0
        cfg, cfg_o = _cfgs(1, 6)
        Yref, _, (s_ao, Ea), L = S.reference(X, W, cfg_o)
        assert (s_ao == 1).all() and (L["scale_o"] == 1).all()
        say("gemm dual decode grid", M)
        Y, _ = _run(X, W, cfg)
        assert np.array_equal(Y.astype(np.float64), Yref)


def _tokens_per_block(M, N, K=128):
    """The matrix form for this shape (above two tokens): "split" (one tile and
    32 tokens per workgroup, K over its waves) while its grid stays within a
    round (two on rows of 8192 and more), else the tiled kernel's token block
    (32, 64 or 128): the smallest that keeps the GPU full, by workgroup count."""
    split_grid = -(-N // 32) * -(-M // 32)
    if M <= 32 or split_grid <= 256 or (K >= 8192 and split_grid <= 512):
        return "split"
    groups = -(-(-(-N // 32)) // 4)
    if groups * -(-M // 32) <= 256:
        return 32
    if groups * -(-M // 64) <= 1024 and groups * -(-M // 128) < 512:
        return 64
    return 128


@pytest.mark.parametrize("M,N,K,block", [(100, 4096, 512, 32), (300, 16384, 256, 64),
                                         (1100, 4096, 128, 64), (300, 32768, 128, 128),
                                         (2100, 4096, 128, 128), (64, 4096, 4096, "split"),
                                         (96, 4096, 11008, "split"), (100, 256, 512, "split")])
@pytest.mark.parametrize("n_o,n_i", [(1, 6), (2, 4)])
def test_gemm_dual_every_token_block(M, N, K, block, n_o, n_i):
    """Shapes that take each token block of the tiled kernel, and the split-K
    form beyond 32 tokens, with ragged M."""
    assert _tokens_per_block(M, N, K) == block
    cfg, cfg_o = _cfgs(n_o, n_i)
    X = synth.make_x(2, M, K)
    W = synth.make_w(2, 0, N, K)
    say("gemm dual block", block, M, N, K)
    Y, _ = _run(X, W, cfg)
    _check(Y, X, W, cfg_o, f"dual block={block} M={M} N={N} K={K}")


@pytest.mark.parametrize("M", [1, 2, 256])
def test_gemm_dual_llama_layer(M):
    """A LLaMA-7B 4096x4096 projection with the paper's 1:8 int8 + 6:8 fp4, bf16 input."""
    cfg, cfg_o = _cfgs(1, 6, "magnitude")
    X = synth.make_x(2, M, 4096)
    W = synth.make_w(2, 0, 4096, 4096)
    say("gemm dual llama", M)
    Y, _ = _run(X, W, cfg, x_bf16=True)
    _check(Y, X, W, cfg_o, f"dual llama M={M}")


@pytest.mark.parametrize("n_o,n_i", [(1, 6), (2, 4)])
@pytest.mark.parametrize("M", [1, 2, 20, 64])
def test_gemm_dual_integer_grid_is_exact(M, n_o, n_i):
    """Inputs on which every scale is 1 and every product and partial sum is
    representable: the output must equal the oracle exactly, on every form
    (decode, split-K, tiled) and with one or two outliers per group."""
    rng = np.random.default_rng(9)
    N, K = 64, 512
    # activations: amax 127 per token (s_a = 1 for A_o); every 32-K block's amax
    # 4 would give A_i codes of x itself, but a token has one amax: use blocks
    # whose values are e2m1 grid points times 2^E with E = floor(log2 amax) - 2
    X = rng.choice([-6.0, -4.0, -2.0, -1.0, 0.0, 1.0, 2.0, 3.0, 4.0, 6.0], (M, K)).astype(np.float32)
    X[:, 0] = 127.0                                  # s_a = 1: A_o = X on the grid
    X[:, 1:32] = rng.choice([-64.0, -32.0, 0.0, 32.0, 64.0, 96.0], (M, 31))  # block 0: E = 4, x/16 on the grid
    W = rng.choice([-6.0, -3.0, -1.0, 1.0, 2.0, 4.0, 6.0], (N, K)).astype(np.float32)
    W[:, ::8] = 127.0 * rng.choice([-1.0, 1.0], (N, K // 8))   # outliers: row amax 127, s_o = 1
    if n_o == 2:
        W[:, 5::8] = rng.choice([-100.0, -9.0, 8.0, 77.0], (N, K // 8))  # the second outlier of a group
    W[:, 1::32] = 6.0                                # every inlier block amax 6: E = 0
    cfg, cfg_o = _cfgs(n_o, n_i)
    Yref, _, (s_ao, Ea), L = S.reference(X, W, cfg_o)
    assert (s_ao == 1).all() and (L["scale_o"] == 1).all()
    assert (L["mask_o"].reshape(N, -1, 8).sum(-1) == n_o).all()
    say("gemm dual grid", M, n_o)
    Y, _ = _run(X, W, cfg)
    assert np.array_equal(Y.astype(np.float64), Yref)


def test_dual_entry_points_refuse_other_families():
    torch = torch_cuda()
    cfg, _ = _cfgs()
    X = torch.zeros((4, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(sdq.SDQError):
        sdq.quantize_act(X, cfg)                       # two activation tensors: the dual call
    with pytest.raises(sdq.SDQError):
        sdq.quantize_act_dual(X, sdq.Config.int_family())


@pytest.mark.parametrize("M", [1, 16, 130])
@pytest.mark.parametrize("y_dtype", ["f32", "bf16"])
def test_dual_hip_graph_replays_match_eager(M, y_dtype):
    """Both dual calls captured in a HIP graph (the decode, split-K and tiled
    forms by M) give the eager result on every replay, with eager work in
    between."""
    import dataclasses
    torch = torch_cuda()
    cfg = dataclasses.replace(_cfgs(1, 6)[0], y_dtype=y_dtype)
    N, K = 512, 1024
    X = torch.from_numpy(synth.make_x(2, M, K)).cuda().to(torch.bfloat16)
    blob = torch.from_numpy(sdq.pack(synth.make_w(2, 0, N, K), cfg)).cuda()
    Xo = torch.empty((M, K), dtype=torch.uint8, device="cuda")
    s_a = torch.empty((M,), dtype=torch.float32, device="cuda")
    Xi = torch.empty((M, K // 2), dtype=torch.uint8, device="cuda")
    Ea = torch.empty((M, K // 32), dtype=torch.uint8, device="cuda")
    Y = torch.empty((M, N), dtype=cfg.y_torch_dtype(), device="cuda")

    def step():
        sdq.quantize_act_dual(X, cfg, out=(Xo, s_a, Xi, Ea))
        sdq.gemm_dual(Xo, s_a, Xi, Ea, blob, N, K, cfg, out=Y)

    say("dual graph", M, y_dtype)
    step()
    torch.cuda.synchronize()
    ref = Y.clone()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        Y.fill_(float("nan"))
        Xo.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y.view(torch.int16), ref.view(torch.int16)), f"replay {rep}"
        sdq.gemm_dual(Xo, s_a, Xi, Ea, blob, N, K, cfg, out=torch.empty_like(Y))
        torch.cuda.synchronize()


@pytest.mark.parametrize("n_o,n_i", [(1, 6), (2, 4)])
def test_gemm_dual_decode_eight_steps_per_wave(n_o, n_i):
    """A wide layer whose K parts take eight steps per wave at one token
    (8192 x 14464: 1024 slices x 113 chunks), checked on a seeded sample of
    rows (rows are independent, so the oracle packs only those)."""
    torch = torch_cuda()
    cfg, cfg_o = _cfgs(n_o, n_i)
    N, K = 8192, 14464
    W = synth.make_w(2, 3, N, K)
    X = synth.make_x(2, 1, K)
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    say("dual decode S=8", N, K, n_o)
    Xo, s_a, Xi, Ea = sdq.quantize_act_dual(torch.from_numpy(X).cuda(), cfg)
    Y = sdq.gemm_dual(Xo, s_a, Xi, Ea, blob, N, K, cfg)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(8).choice(N, 48, replace=False))
    _check(Y.cpu().numpy()[:, rows], X, W[rows], cfg_o, "dual decode S=8")
