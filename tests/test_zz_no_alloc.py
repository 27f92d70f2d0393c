"""GPU: sdq_gemm_static, the entry point that allocates nothing, against
sdq_gemm_ws (the same product with a caller-owned workspace), through the C
ABI.  Two calls in a row on each path that takes a workspace (the two-pass
MX path and the INT split-K path), the second with a smaller input, must each
equal the workspace entry point bit for bit; the static scratch array keeps
the first call's contents, which the second must not see.
A shape whose workspace exceeds the array is refused before any GPU work."""
import ctypes as C

import numpy as np
import pytest

import synth
from tests.gpu_util import say, torch_cuda

import paper_2406_13868_amd as sdq
from paper_2406_13868_amd import _lib

pytestmark = pytest.mark.gpu

CFG = sdq.Config.of(synth.WORKLOADS[3].formats[0])  # MX 1:8 e4m3 + 2:8 e2m1


def _case(M, N, K, seed):
    torch = torch_cuda()
    W = synth.make_w(3, 10 + seed, N, K)
    X = synth.make_x(3, M, K, seed=seed)
    blob = torch.from_numpy(sdq.pack(W, CFG)).cuda()
    Xq, s_a = sdq.quantize_act(torch.from_numpy(X).cuda(), CFG)
    return blob, Xq, s_a


def test_static_entry_equals_workspace_entry_twice():
    torch = torch_cuda()
    for (M, N, K, seed) in ((1100, 4128, 4096, 1), (520, 2080, 1152, 2)):
        assert sdq.gemm_workspace_size(CFG, M, N, K, sdq.PATH_DENSE) <= _lib.STATIC_SCRATCH_BYTES
        blob, Xq, s_a = _case(M, N, K, seed)
        ws = torch.empty(sdq.gemm_workspace_size(CFG, M, N, K, sdq.PATH_DENSE), dtype=torch.uint8,
                         device="cuda")
        say("static scratch", M, N, K)
        Y_ws = sdq.gemm(Xq, s_a, blob, N, K, CFG, path=sdq.PATH_DENSE, workspace=ws)
        Y_st = torch.full((M, N), float("nan"), device="cuda")
        st = _lib.lib().sdq_gemm_static(C.byref(CFG.c()), C.c_void_p(Xq.data_ptr()),
                                        C.c_void_p(s_a.data_ptr()), M, C.c_void_p(blob.data_ptr()), N, K,
                                        C.c_void_p(Y_st.data_ptr()),
                                        C.c_void_p(torch.cuda.current_stream().cuda_stream), sdq.PATH_DENSE)
        assert st == 0, _lib.STATUS.get(st, st)
        torch.cuda.synchronize()
        a, b = Y_ws.cpu().numpy(), Y_st.cpu().numpy()
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), \
            f"M={M} N={N} K={K}: {int(np.sum(a != b))} outputs differ"
        # the binding's form of the same call
        Y_b = sdq.gemm_static(Xq, s_a, blob, N, K, CFG, path=sdq.PATH_DENSE)
        torch.cuda.synchronize()
        assert np.array_equal(a.view(np.uint32), Y_b.cpu().numpy().view(np.uint32))


def test_static_entry_refuses_a_workspace_beyond_the_array():
    torch = torch_cuda()
    M, N, K = 600, 16384, 4096  # 64 MiB of merged fragments
    assert sdq.gemm_workspace_size(CFG, M, N, K, sdq.PATH_DENSE) > _lib.STATIC_SCRATCH_BYTES
    Xq = torch.zeros((M, K), dtype=torch.uint8, device="cuda")
    s_a = torch.zeros((M,), device="cuda")
    blob = torch.zeros(sdq.pack_size(CFG, N, K), dtype=torch.uint8, device="cuda")
    with pytest.raises(sdq.SDQError) as e:
        sdq.gemm_static(Xq, s_a, blob, N, K, CFG, path=sdq.PATH_DENSE)
    assert e.value.status == -8


@pytest.mark.parametrize("fam", ["int", "mx"])
def test_static_entry_equals_workspace_entry_split_k(fam):
    """The split-K paths of the INT and MX families (partial sums of K ranges
    in the scratch array): two calls in a row, the second smaller, each bit
    for bit equal to sdq_gemm_ws with a caller-owned workspace."""
    torch = torch_cuda()
    cfg = sdq.Config.int_family(1, 8, "int8", 3) if fam == "int" else CFG
    for (M, N, K, seed) in ((64, 4128, 16384, 1), (20, 1000, 2048, 2)):
        assert 0 < sdq.gemm_workspace_size(cfg, M, N, K, sdq.PATH_SPLITK) <= _lib.STATIC_SCRATCH_BYTES
        W = synth.make_w(4, 10 + seed, N, K)
        blob = torch.from_numpy(sdq.pack(W, cfg)).cuda()
        Xq, s_a = sdq.quantize_act(torch.from_numpy(synth.make_x(4, M, K, seed=seed)).cuda(), cfg)
        ws = torch.full((sdq.gemm_workspace_size(cfg, M, N, K, sdq.PATH_SPLITK),), 0x7F,
                        dtype=torch.uint8, device="cuda")  # stale contents must not matter
        say("static scratch split-K", fam, M, N, K)
        Y_ws = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=sdq.PATH_SPLITK, workspace=ws)
        Y_st = torch.full((M, N), float("nan"), device="cuda")
        st = _lib.lib().sdq_gemm_static(C.byref(cfg.c()), C.c_void_p(Xq.data_ptr()),
                                        C.c_void_p(s_a.data_ptr()), M, C.c_void_p(blob.data_ptr()), N, K,
                                        C.c_void_p(Y_st.data_ptr()),
                                        C.c_void_p(torch.cuda.current_stream().cuda_stream), sdq.PATH_SPLITK)
        assert st == 0, _lib.STATUS.get(st, st)
        torch.cuda.synchronize()
        a, b = Y_ws.cpu().numpy(), Y_st.cpu().numpy()
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), \
            f"M={M} N={N} K={K}: {int(np.sum(a != b))} outputs differ"
