"""GPU: the GEMMs' bf16 output (sdq_config.y_dtype = SDQ_DTYPE_BF16).

Every output is the same fp32 result rounded to nearest even (Section 5.1's
product, then one rounding), so a bf16 call must give, bit for bit, the
rounding of the fp32 call on the same inputs.  The host rounds with torch's
CPU conversion, which rounds to nearest even.  The single documented
exception -- on the two-pass MX path, outputs whose wave met a block which
did not merge its inliers are rounded twice: the main sum to bf16, then that
value plus those inliers -- is checked against the oracle: the final
rounding (2^-9 of the output), the first one (2^-9 of the main sum, itself at
most the sum of |terms|) and the MX accumulation bound.
"""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import sdq as S
from tests.gpu_util import mx_term_tol, say, torch_cuda

import paper_2406_13868_amd as sdq

pytestmark = pytest.mark.gpu


def _int(fmt_o="e4m3"):
    return sdq.Config("int", 1, 8, fmt_o, 3, 8, "int4", "int8")


def _mx(n_i=2):
    return sdq.Config("mx", 1, 8, "e4m3", n_i, 8, "e2m1", "e4m3")


def _bf16(cfg):
    return dataclasses.replace(cfg, y_dtype="bf16")


def _rne_bits(Y32):
    torch = torch_cuda()
    return Y32.cpu().to(torch.bfloat16).view(torch.int16)


def _assert_rounded(Yb, Y32, what):
    torch = torch_cuda()
    assert Yb.dtype == torch.bfloat16 and Yb.shape == Y32.shape
    got, want = Yb.cpu().view(torch.int16), _rne_bits(Y32)
    bad = int((got != want).sum())
    assert bad == 0, f"{what}: {bad} of {got.numel()} outputs differ from RNE(fp32)"


@pytest.mark.parametrize("cfg", [_int("e4m3"), _int("int8"), _mx(2), _mx(3)],
                         ids=["int-e4m3", "int-int8", "mx-2:8", "mx-3:8"])
@pytest.mark.parametrize("M", [1, 4, 16, 64, 130])
def test_gemm_bf16_is_rounded_fp32(cfg, M):
    torch = torch_cuda()
    N, K = 160, 512
    X = torch.from_numpy(synth.make_x(2, M, K)).cuda()
    blob = torch.from_numpy(sdq.pack(synth.make_w(2, 0, N, K), cfg)).cuda()
    Xq, s_a = sdq.quantize_act(X, cfg)
    paths = [sdq.PATH_MFMA, sdq.PATH_SPLITK]
    if cfg.family == "int":
        paths = ([sdq.PATH_DECODE] if M <= 8 else []) + paths
    for path in paths:
        say("bf16 out", cfg.family, cfg.fmt_o, cfg.n_i, M, "path", path)
        Y32 = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=path)
        Yb = sdq.gemm(Xq, s_a, blob, N, K, _bf16(cfg), path=path)
        torch.cuda.synchronize()
        _assert_rounded(Yb, Y32, f"M={M} path={path}")


@pytest.mark.parametrize("M", [1, 2, 16])
def test_linear_bf16_is_rounded_fp32(M):
    """The fused decode kernel (activation quantization inside) and the two-call path."""
    torch = torch_cuda()
    cfg = _int("e4m3")
    N, K = 300, 1024
    X = torch.from_numpy(synth.make_x(2, M, K)).cuda().to(torch.bfloat16)
    blob = torch.from_numpy(sdq.pack(synth.make_w(2, 0, N, K), cfg)).cuda()
    say("bf16 linear", M)
    Y32, _, _ = sdq.linear(X, blob, N, K, cfg)
    Yb, _, _ = sdq.linear(X, blob, N, K, _bf16(cfg))
    torch.cuda.synchronize()
    _assert_rounded(Yb, Y32, f"linear M={M}")


def test_two_pass_bf16_is_rounded_fp32():
    """The two-pass MX path on weights whose blocks all merge (checked)."""
    torch = torch_cuda()
    cfg = _mx(3)
    N, K, M = 544, 640, 600
    W = synth.make_w(2, 0, N, K)
    L = S.pack_logical(W, S.Config("mx", 1, 8, "e4m3", 3, 8, "e2m1", "e4m3"))
    d = L["scale_i"].astype(int) - L["scale_o"].astype(int)
    assert not np.any((d < -5) | (d > 6)), "the case must merge every block"
    X = torch.from_numpy(synth.make_x(2, M, K)).cuda()
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    Xq, s_a = sdq.quantize_act(X, cfg)
    say("bf16 two-pass", M, N, K)
    Y32 = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=sdq.PATH_DENSE)
    Yb = sdq.gemm(Xq, s_a, blob, N, K, _bf16(cfg), path=sdq.PATH_DENSE)
    torch.cuda.synchronize()
    _assert_rounded(Yb, Y32, "two-pass")


@pytest.mark.parametrize("path", [sdq.PATH_MFMA, sdq.PATH_DENSE])
def test_bf16_with_unmerged_blocks_matches_oracle(path):
    """Outliers 2^13 times their blocks' inliers: no block merges."""
    torch = torch_cuda()
    cfg = _mx(2)
    cfg_o = S.Config("mx", 1, 8, "e4m3", 2, 8, "e2m1", "e4m3")
    N, K, M = 96, 384, 520
    W = synth.make_w(1, 0, N, K).copy()
    W[:, 5::8] = np.sign(W[:, 5::8] + 1e-9) * 8192.0 * np.abs(W).max()
    X = synth.make_x(1, M, K)
    L = S.pack_logical(W, cfg_o)
    d = L["scale_i"].astype(int) - L["scale_o"].astype(int)
    assert np.any((d < -5) | (d > 6))
    blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
    Xq, s_a = sdq.quantize_act(torch.from_numpy(X).cuda(), cfg)
    say("bf16 unmerged", path)
    Yb = sdq.gemm(Xq, s_a, blob, N, K, _bf16(cfg), path=path)
    torch.cuda.synchronize()
    Y = Yb.cpu().float().numpy().astype(np.float64)
    Yref, _, _, _ = S.reference(X, W, cfg_o)
    A = np.abs(S.dequant_act(*S.quantize_act(X, cfg_o), cfg_o))
    T = A @ (np.abs(S.dequant_outliers(L)) + np.abs(S.dequant_inliers(L))).T
    excess = np.abs(Y - Yref) - (2.0 ** -8 * np.abs(Yref) + (2.0 ** -9 + mx_term_tol(K)) * T)
    assert float(excess.max()) <= 0.0, f"worst excess {float(excess.max()):.3e}"


@pytest.mark.parametrize("M", [5, 130])
def test_dual_bf16_is_rounded_fp32(M):
    torch = torch_cuda()
    cfg = sdq.Config.dual_family(1, 6)
    N, K = 160, 512
    X = torch.from_numpy(synth.make_x(2, M, K)).cuda()
    blob = torch.from_numpy(sdq.pack(synth.make_w(2, 0, N, K), cfg)).cuda()
    Xo, s_a, Xi, Ea = sdq.quantize_act_dual(X, cfg)
    say("bf16 dual", M)
    Y32 = sdq.gemm_dual(Xo, s_a, Xi, Ea, blob, N, K, cfg)
    Yb = sdq.gemm_dual(Xo, s_a, Xi, Ea, blob, N, K, _bf16(cfg))
    torch.cuda.synchronize()
    _assert_rounded(Yb, Y32, f"dual M={M}")


def test_bf16_out_argument_is_checked():
    torch = torch_cuda()
    cfg = _bf16(_int())
    N, K, M = 64, 256, 2
    blob = torch.from_numpy(sdq.pack(synth.make_w(2, 0, N, K), cfg)).cuda()
    Xq, s_a = sdq.quantize_act(torch.from_numpy(synth.make_x(2, M, K)).cuda(), cfg)
    with pytest.raises(ValueError):
        sdq.gemm(Xq, s_a, blob, N, K, cfg, out=torch.empty((M, N), dtype=torch.float32, device="cuda"))
