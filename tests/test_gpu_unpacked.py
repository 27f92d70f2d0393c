"""GPU: the two passes of the MX family's two-pass path as separate calls
(sdq_unpack_weights, then sdq_gemm_unpacked) against sdq_gemm_ws with
SDQ_PATH_DENSE, bit for bit: ragged shapes, a partial last 128-K chunk, blocks
whose inliers stay apart from the outliers, bf16 output, and the unpack on a
second stream ordered before the product by an event (the form that lets a
caller unpack the next layer while this one multiplies)."""
import dataclasses

import numpy as np
import pytest

import synth
from tests.gpu_util import say, torch_cuda
from tests.test_gpu_gemm import _split_case

import paper_2406_13868_amd as sdq

pytestmark = pytest.mark.gpu

MX = sdq.Config.of(synth.WORKLOADS[3].formats[0])  # MX 1:8 e4m3 + 2:8 e2m1


def _bits(t):
    torch = torch_cuda()
    return t.contiguous().view(torch.uint8).cpu().numpy()


@pytest.mark.parametrize("M,N,K", [(600, 544, 1152), (1100, 4128, 4096), (33, 300, 288), (1, 64, 128)])
@pytest.mark.parametrize("y_dtype", ["f32", "bf16"])
def test_unpacked_equals_two_pass(M, N, K, y_dtype):
    torch = torch_cuda()
    cfg = dataclasses.replace(MX, y_dtype=y_dtype)
    blob = torch.from_numpy(sdq.pack(synth.make_w(3, 5, N, K), cfg)).cuda()
    Xq, s_a = sdq.quantize_act(torch.from_numpy(synth.make_x(3, M, K)).cuda(), cfg)
    say("unpacked", M, N, K, y_dtype)
    Y_ws = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=sdq.PATH_DENSE)
    ws = torch.full((sdq.gemm_workspace_size(cfg, M, N, K, sdq.PATH_DENSE),), 0x7F, dtype=torch.uint8,
                    device="cuda")
    sdq.unpack_weights(blob, N, K, cfg, workspace=ws)
    Y = sdq.gemm_unpacked(Xq, s_a, blob, N, K, cfg, ws)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(Y), _bits(Y_ws))
    # the workspace serves any number of products of the same weights
    Xq2, s_a2 = sdq.quantize_act(torch.from_numpy(synth.make_x(3, M, K, seed=1)).cuda(), cfg)
    Y2 = sdq.gemm_unpacked(Xq2, s_a2, blob, N, K, cfg, ws)
    Y2_ws = sdq.gemm(Xq2, s_a2, blob, N, K, cfg, path=sdq.PATH_DENSE)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(Y2), _bits(Y2_ws))


@pytest.mark.parametrize("kind", ["product", "zero_inliers", "huge_outliers"])
def test_unpacked_unmergeable_blocks(kind):
    torch = torch_cuda()
    rng = np.random.default_rng(7)
    N, K, M = 96, 384, 520
    metric = "product" if kind == "product" else "magnitude"
    cfg = sdq.Config("mx", 1, 8, "e4m3", 3, 8, "e2m1", "e4m3", metric)
    W, an = _split_case(kind, N, K, rng)
    blob = torch.from_numpy(sdq.pack(W, cfg, act_norm=an)).cuda()
    Xq, s_a = sdq.quantize_act(torch.from_numpy(synth.make_x(1, M, K)).cuda(), cfg)
    say("unpacked unmergeable", kind)
    Y_ws = sdq.gemm(Xq, s_a, blob, N, K, cfg, path=sdq.PATH_DENSE)
    ws = sdq.unpack_weights(blob, N, K, cfg)
    Y = sdq.gemm_unpacked(Xq, s_a, blob, N, K, cfg, ws)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(Y), _bits(Y_ws))


def test_unpack_on_a_second_stream():
    """Three layers: each layer's unpack on a side stream, each product on the
    main stream after an event recorded behind its own unpack; the outputs
    equal the sequential two-pass calls."""
    torch = torch_cuda()
    shapes = [(11008, 4096), (11008, 4096), (4096, 11008)]
    M = 600
    blobs = [torch.from_numpy(sdq.pack(synth.make_w(3, j, N, K), MX)).cuda() for j, (N, K) in enumerate(shapes)]
    acts = [sdq.quantize_act(torch.from_numpy(synth.make_x(3, M, K)).cuda(), MX) for (_, K) in shapes]
    refs = [sdq.gemm(Xq, s_a, b, N, K, MX, path=sdq.PATH_DENSE) for (Xq, s_a), b, (N, K) in zip(acts, blobs, shapes)]
    wss = [torch.empty((sdq.gemm_workspace_size(MX, M, N, K, sdq.PATH_DENSE),), dtype=torch.uint8, device="cuda")
           for (N, K) in shapes]
    outs = [torch.full((M, N), float("nan"), device="cuda") for (N, _) in shapes]
    torch.cuda.synchronize()
    say("unpack side stream")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    done = []
    with torch.cuda.stream(side):
        for b, ws, (N, K) in zip(blobs, wss, shapes):
            sdq.unpack_weights(b, N, K, MX, workspace=ws)
            ev = torch.cuda.Event()
            ev.record(side)
            done.append(ev)
    for (Xq, s_a), b, ws, ev, Y, (N, K) in zip(acts, blobs, wss, done, outs, shapes):
        torch.cuda.current_stream().wait_event(ev)
        sdq.gemm_unpacked(Xq, s_a, b, N, K, MX, ws, out=Y)
    torch.cuda.synchronize()
    for Y, R in zip(outs, refs):
        assert np.array_equal(_bits(Y), _bits(R))
