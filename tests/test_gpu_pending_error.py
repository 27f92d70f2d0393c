"""GPU: an error that an earlier, unrelated HIP call on the calling thread left
pending is not reported as a library call's own launch failure.

The runtime keeps one pending error per thread until hipGetLastError reads
it; the launchers read it to detect a failed launch.  Each case leaves one
pending (hipSetDevice with an ordinal that does not exist, a host-side
argument error) on the HIP runtime the library is bound to, right before a
device entry point of the C ABI, with every buffer allocated beforehand
(torch's allocator reads the pending error too).  The call must return
SDQ_OK and write the same bits as the same call without it."""
import ctypes as C
import re

import numpy as np
import pytest

import synth
from tests.gpu_util import say, torch_cuda

import paper_2406_13868_amd as sdq
from paper_2406_13868_amd import _lib

pytestmark = pytest.mark.gpu

HIP_ERROR_INVALID_DEVICE = 101


def _runtime():
    """The HIP runtime libsdq.so resolved (torch may have loaded its own copy
    of libamdhip64 first; opening the same path returns that copy)."""
    _lib.lib()
    maps = open("/proc/self/maps").read()
    paths = sorted(set(re.findall(r"\S*/libamdhip64\.so[.\d]*", maps)))
    assert len(paths) == 1, paths
    return C.CDLL(paths[0])


def _p(t):
    return C.c_void_p(t.data_ptr())


def _twice(hip, call, outs):
    """call() clean, then with a pending error: both SDQ_OK, same output bits."""
    torch = torch_cuda()
    for o in outs:
        o.fill_(0x55 if o.dtype == torch.uint8 else float("nan"))
    torch.cuda.synchronize()
    assert call() == 0
    torch.cuda.synchronize()
    first = [o.cpu().numpy().copy() for o in outs]
    for o in outs:
        o.fill_(0x55 if o.dtype == torch.uint8 else float("nan"))
    torch.cuda.synchronize()
    hip.hipGetLastError()
    assert hip.hipSetDevice(C.c_int(1 << 20)) == HIP_ERROR_INVALID_DEVICE
    assert hip.hipPeekAtLastError() == HIP_ERROR_INVALID_DEVICE
    try:
        st = call()
    finally:
        hip.hipGetLastError()
    assert st == 0, _lib.STATUS.get(st, st)
    torch.cuda.synchronize()
    for a, o in zip(first, outs):
        assert np.array_equal(a.view(np.uint8), o.cpu().numpy().view(np.uint8))


@pytest.mark.parametrize("fam,M,N,K,path", [("int", 1, 256, 512, sdq.PATH_DECODE),
                                            ("int", 40, 256, 512, sdq.PATH_MFMA),
                                            ("int", 40, 256, 512, sdq.PATH_SPLITK),
                                            ("mx", 40, 256, 512, sdq.PATH_MFMA),
                                            ("mx", 600, 256, 512, sdq.PATH_DENSE)])
def test_quantize_and_gemm(fam, M, N, K, path):
    torch = torch_cuda()
    hip = _runtime()
    L = _lib.lib()
    cfg = sdq.Config.int_family(1, 8, "e4m3", 3) if fam == "int" else sdq.Config.of(synth.WORKLOADS[3].formats[0])
    c = cfg.c()
    X = torch.from_numpy(synth.make_x(1, M, K)).cuda()
    blob = torch.from_numpy(sdq.pack(synth.make_w(1, 0, N, K), cfg)).cuda()
    Xq = torch.empty((M, K), dtype=torch.uint8, device="cuda")
    s_a = torch.empty((M,), device="cuda")
    Y = torch.empty((M, N), device="cuda")
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    say("pending error", fam, M, N, K, path)
    _twice(hip, lambda: L.sdq_quantize_act(C.byref(c), _p(X), _lib.DTYPE_F32, M, K, _p(Xq), _p(s_a), stream),
           [Xq, s_a])
    if path in (sdq.PATH_DENSE, sdq.PATH_SPLITK):
        nb = sdq.gemm_workspace_size(cfg, M, N, K, path)
        ws = torch.empty((nb,), dtype=torch.uint8, device="cuda")
        _twice(hip, lambda: L.sdq_gemm_ws(C.byref(c), _p(Xq), _p(s_a), M, _p(blob), N, K, _p(Y), _p(ws), nb,
                                          stream, path), [Y])
        _twice(hip, lambda: L.sdq_gemm_static(C.byref(c), _p(Xq), _p(s_a), M, _p(blob), N, K, _p(Y), stream,
                                              path), [Y])
    else:
        _twice(hip, lambda: L.sdq_gemm_ex(C.byref(c), _p(Xq), _p(s_a), M, _p(blob), N, K, _p(Y), stream,
                                          path), [Y])


def test_linear_and_dual():
    torch = torch_cuda()
    hip = _runtime()
    L = _lib.lib()
    M, N, K = 2, 256, 512
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    X = torch.from_numpy(synth.make_x(1, M, K)).cuda()
    Y = torch.empty((M, N), device="cuda")
    say("pending error linear")
    cfg = sdq.Config.int_family(1, 8, "e4m3", 3)
    c = cfg.c()
    blob = torch.from_numpy(sdq.pack(synth.make_w(1, 0, N, K), cfg)).cuda()
    Xq = torch.empty((M, K), dtype=torch.uint8, device="cuda")
    s_a = torch.empty((M,), device="cuda")
    _twice(hip, lambda: L.sdq_linear(C.byref(c), _p(X), _lib.DTYPE_F32, M, _p(Xq), _p(s_a), _p(blob), N, K,
                                     _p(Y), stream), [Xq, s_a, Y])
    say("pending error dual")
    dcfg = sdq.Config.dual_family(1, 6)
    d = dcfg.c()
    dblob = torch.from_numpy(sdq.pack(synth.make_w(1, 1, N, K), dcfg)).cuda()
    Xo = torch.empty((M, K), dtype=torch.uint8, device="cuda")
    Xi = torch.empty((M, K // 2), dtype=torch.uint8, device="cuda")
    Ea = torch.empty((M, K // 32), dtype=torch.uint8, device="cuda")
    _twice(hip, lambda: L.sdq_quantize_act_dual(C.byref(d), _p(X), _lib.DTYPE_F32, M, K, _p(Xo), _p(s_a),
                                                _p(Xi), _p(Ea), stream), [Xo, s_a, Xi, Ea])
    _twice(hip, lambda: L.sdq_gemm_dual(C.byref(d), _p(Xo), _p(s_a), _p(Xi), _p(Ea), M, _p(dblob), N, K,
                                        _p(Y), stream), [Y])
