"""Host packer and C ABI (no GPU): bit-exact against the oracle.

The packer (C++, in libsdq.so) and the oracle (numpy) are independent
implementations of the same definitions; their logical outputs (positions,
codes, scales) must agree exactly, and the kernel layout must decode back to
the oracle's dense codes.
"""
import ctypes as C
import dataclasses
import os
import re

import numpy as np
import pytest

import synth
from oracle import accounting as A
from oracle import sdq as S

sdq = pytest.importorskip("paper_2406_13868_amd")
from paper_2406_13868_amd import _lib  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
HEADER = os.path.join(os.path.dirname(HERE), "include", "sdq.h")

CONFIGS = [
    ("int", 1, 8, "e4m3", 3), ("int", 1, 8, "int8", 3), ("int", 1, 16, "e4m3", 3),
    ("int", 1, 8, "e4m3", 2), ("int", 1, 16, "e4m3", 2), ("int", 0, 8, "e4m3", 3),
    ("mx", 1, 8, "e4m3", 2), ("mx", 1, 8, "e4m3", 3), ("mx", 1, 16, "e4m3", 2),
    ("mx", 1, 16, "e4m3", 3), ("mx", 0, 8, "e4m3", 2),
]


def _cfgs(fam, n_o, m_o, fmt_o, n_i, metric="magnitude"):
    if fam == "int":
        lib = sdq.Config("int", n_o, m_o, fmt_o, n_i, 8, "int4", "int8", metric)
        ora = S.Config("int", n_o, m_o, fmt_o, n_i, 8, "int4", "int8", metric)
    else:
        lib = sdq.Config("mx", n_o, m_o, "e4m3", n_i, 8, "e2m1", "e4m3", metric)
        ora = S.Config("mx", n_o, m_o, "e4m3", n_i, 8, "e2m1", "e4m3", metric)
    return lib, ora


def _ids(c):
    return f"{c[0]}-{c[1]}:{c[2]}{c[3]}+{c[4]}:8"


def _compare_logical(Lg, Lo, cfg_o):
    if cfg_o.n_o:
        assert np.array_equal(Lg["pos_o"], Lo["pos_o"].astype(np.uint8))
        assert np.array_equal(Lg["code_o"], Lo["code_o"])
    assert np.array_equal(Lg["pos_i"], Lo["pos_i"].astype(np.uint8))
    if cfg_o.family == "int":
        assert np.array_equal(Lg["code_i"].view(np.int8), Lo["code_i"].astype(np.int8))
        assert np.array_equal(Lg["scale_i"], Lo["scale_i"].view(np.uint16))
        if cfg_o.n_o:
            assert np.array_equal(Lg["scale_o"].view(np.uint32), Lo["scale_o"].view(np.uint32))
    else:
        assert np.array_equal(Lg["code_i"], Lo["code_i"])
        assert np.array_equal(Lg["scale_i"], Lo["scale_i"])
        if cfg_o.n_o:
            assert np.array_equal(Lg["scale_o"], Lo["scale_o"])


@pytest.mark.parametrize("c", CONFIGS, ids=_ids)
@pytest.mark.parametrize("shape", [(256, 256), (50, 384), (33, 128), (40, 160), (33, 1056), (9, 32)])
def test_logical_pack_matches_oracle(c, shape):
    cfg, cfg_o = _cfgs(*c)
    N, K = shape
    W = synth.make_w(2, 0, N, K)
    Lg = sdq.pack_logical(W, cfg)
    Lo = S.pack_logical(W, cfg_o)
    _compare_logical(Lg, Lo, cfg_o)


@pytest.mark.parametrize("c", CONFIGS, ids=_ids)
@pytest.mark.parametrize("K", [512, 160, 288, 4128])
def test_kernel_layout_roundtrip(c, K):
    """Blob -> dense codes and scales, against the oracle's decisions: a ragged
    last tile of 32 rows, and K that leaves a last partial 128-K chunk (which
    the blob pads with zero codes and scales)."""
    cfg, cfg_o = _cfgs(*c)
    N = 70  # ragged last tile of 32 rows
    W = synth.make_w(5, 0, N, K)
    blob = sdq.pack(W, cfg)
    U = sdq.unpack_dense(blob, cfg, N, K)
    Lo = S.pack_logical(W, cfg_o)
    if cfg_o.family == "int":
        assert np.array_equal(U["code_i_dense"].view(np.int8), Lo["code_i_dense"].astype(np.int8))
        assert np.array_equal(U["scale_i"], Lo["scale_i"].view(np.uint16))
        if cfg_o.n_o:
            assert np.array_equal(U["scale_o"].view(np.uint32), Lo["scale_o"].view(np.uint32))
    else:
        assert np.array_equal(U["code_i_dense"], Lo["code_i_dense"])
        assert np.array_equal(U["scale_i"], Lo["scale_i"])
        if cfg_o.n_o:
            assert np.array_equal(U["scale_o"], Lo["scale_o"])
    assert np.array_equal(U["code_o_dense"], Lo["code_o_dense"])


def test_product_metric_matches_oracle():
    cfg, cfg_o = _cfgs("int", 1, 8, "e4m3", 3, metric="product")
    W = synth.make_w(1, 0, 64, 256)
    X_cal = synth.make_x(1, 32, 256)
    c = S.activation_norm(X_cal)
    _compare_logical(sdq.pack_logical(W, cfg, act_norm=c), S.pack_logical(W, cfg_o, act_norm=c), cfg_o)
    cfg, cfg_o = _cfgs("mx", 1, 8, "e4m3", 2, metric="product")
    _compare_logical(sdq.pack_logical(W, cfg, act_norm=c), S.pack_logical(W, cfg_o, act_norm=c), cfg_o)


def test_concatenated_rows_pack_like_separate_matrices():
    """Packing is row by row, so W_q, W_k and W_v stacked along N pack to
    the stacked logical arrays of the three (one launch then serves all three)."""
    cfg = sdq.Config("int", 1, 8, "e4m3", 3, 8, "int4", "int8")
    Ws = [synth.make_w(2, j, 64, 512) for j in range(3)]
    cat = sdq.pack_logical(np.concatenate(Ws), cfg)
    parts = [sdq.pack_logical(W, cfg) for W in Ws]
    for key, v in cat.items():
        if v is None:
            continue
        assert np.array_equal(v, np.concatenate([p[key] for p in parts])), key


@pytest.mark.parametrize("wid", [1, 2, 4])
def test_workload_first_layer_matches_oracle(wid):
    """A row slice of each workload's first layer at its real K."""
    w = synth.WORKLOADS[wid]
    L = w.layers[0]
    W = synth.make_w(wid, 0, L.N, L.K)[:96]
    cfg = sdq.Config.of(w.formats[0])
    cfg_o = S.config_from(w.formats[0])
    _compare_logical(sdq.pack_logical(W, cfg), S.pack_logical(W, cfg_o), cfg_o)


def test_tied_and_degenerate_weights():
    cfg, cfg_o = _cfgs("int", 1, 8, "e4m3", 3)
    rng = np.random.default_rng(3)
    W = (rng.integers(-2, 3, (40, 256)) * 0.125).astype(np.float32)  # many exact ties
    W[5] = 0.0                                                        # an all-zero row
    W[7, :16] = 0.0                                                   # an all-zero block
    W[9] = -0.0
    _compare_logical(sdq.pack_logical(W, cfg), S.pack_logical(W, cfg_o), cfg_o)
    cfgm, cfgm_o = _cfgs("mx", 1, 8, "e4m3", 3)
    _compare_logical(sdq.pack_logical(W, cfgm), S.pack_logical(W, cfgm_o), cfgm_o)


def test_pack_is_thread_count_independent():
    cfg, _ = _cfgs("int", 1, 8, "e4m3", 3)
    W = synth.make_w(2, 0, 333, 1024)
    a = sdq.pack(W, cfg, n_threads=1)
    b = sdq.pack(W, cfg, n_threads=7)
    c = sdq.pack(W, cfg, n_threads=0)
    assert np.array_equal(a, b) and np.array_equal(a, c)


@pytest.mark.parametrize("c", CONFIGS, ids=_ids)
def test_logical_bytes_match_accounting(c):
    cfg, cfg_o = _cfgs(*c)
    N, K = 4096, 4096
    if cfg_o.family == "int":
        b = A.sdq_bits_per_weight(cfg.n_o, cfg.m_o, 8, cfg.n_i, 8, 4, 32, 0, 16, 16, K)
    else:
        b = A.sdq_bits_per_weight(cfg.n_o, cfg.m_o, 8, cfg.n_i, 8, 4, 8, 32, 8, 32, K)
    want = int(np.ceil(float(b * N * K) / 8))
    assert sdq.logical_bytes(cfg, N, K) == want


def test_logical_bytes_llama_decode_layer():
    # 4096x4096, 1:8 e4m3 + 3:8 int4 with fp16 scales per 16: 5.008 bits per weight
    assert sdq.logical_bytes(sdq.Config.int_family(), 4096, 4096) == 10_502_144


def _raw(name):
    return getattr(_lib.lib(), name)


def test_error_paths():
    cfg = sdq.Config.int_family().c()
    L = _lib.lib()
    n = C.c_size_t()
    assert L.sdq_pack_size(None, 32, 128, C.byref(n)) == -1
    assert L.sdq_pack_size(C.byref(cfg), 32, 100, C.byref(n)) == -2       # K % 32
    assert L.sdq_pack_size(C.byref(cfg), 32, 48, C.byref(n)) == -2        # K % 32
    assert L.sdq_pack_size(C.byref(cfg), 32, 160, C.byref(n)) == 0        # a partial last 128-K chunk
    assert n.value == sdq.pack_size(sdq.Config.int_family(), 32, 256)     # padded to whole chunks
    cq = dataclasses.replace(sdq.Config.int_family(), qv_i=64)
    assert L.sdq_pack_size(C.byref(cq.c()), 32, 160, C.byref(n)) == -2   # K % qv
    assert L.sdq_pack_size(C.byref(cfg), 0, 128, C.byref(n)) == -2
    bad = sdq.Config("int", 1, 8, "e2m1", 3).c()
    assert L.sdq_pack_size(C.byref(bad), 32, 128, C.byref(n)) == -3
    unsup = sdq.Config("int", 2, 8, "e4m3", 3).c()
    assert L.sdq_pack_size(C.byref(unsup), 32, 128, C.byref(n)) == -6
    W = np.zeros((32, 128), np.float32)
    buf = np.zeros(16, np.uint8)
    assert L.sdq_pack(C.byref(cfg), C.c_void_p(W.ctypes.data), 32, 128, None,
                      C.c_void_p(buf.ctypes.data), buf.nbytes, 1) == -4
    W[3, 7] = np.nan
    with pytest.raises(sdq.SDQError) as e:
        sdq.pack(W, sdq.Config.int_family())
    assert e.value.status == -7
    # product metric needs act_norm
    with pytest.raises(sdq.SDQError) as e:
        sdq.pack(np.zeros((32, 128), np.float32), sdq.Config.int_family(metric="product"))
    assert e.value.status == -1
    # device entry points validate before touching the GPU
    assert L.sdq_gemm(C.byref(cfg), None, None, 4, None, 32, 128, None, None) == -1
    assert L.sdq_gemm(C.byref(cfg), None, None, 4, None, 32, 120, None, None) == -2
    assert L.sdq_gemm(C.byref(cfg), None, None, 0, None, 32, 128, None, None) == 0  # M = 0
    assert L.sdq_quantize_act(C.byref(cfg), None, 0, 4, 128, None, None, None) == -1
    assert L.sdq_quantize_act(C.byref(cfg), None, 5, 4, 128, None, None, None) == -3
    mxc = sdq.Config.mx_family().c()
    assert L.sdq_gemm_ex(C.byref(mxc), C.c_void_p(16), C.c_void_p(16), 1, C.c_void_p(16),
                         32, 128, C.c_void_p(16), None, 1) == -6   # no decode path for MX
    # the output type: fp32 or bf16 only; a misaligned Y is refused before any launch
    bad_y = sdq.Config.int_family().c()
    bad_y.y_dtype = 7
    assert L.sdq_check(C.byref(bad_y), 32, 128) == -3
    bf = sdq.Config("int", 1, 8, "e4m3", 3, 8, "int4", "int8", y_dtype="bf16").c()
    assert L.sdq_check(C.byref(bf), 32, 128) == 0
    assert L.sdq_gemm(C.byref(bf), C.c_void_p(16), C.c_void_p(16), 1, C.c_void_p(16), 32, 128,
                      C.c_void_p(18), None) == -2
    dual = sdq.Config.dual_family().c()
    p16 = C.c_void_p(16)
    assert L.sdq_gemm_dual(C.byref(dual), p16, p16, p16, p16, 1, p16, 32, 128, C.c_void_p(18), None) == -2
    assert L.sdq_gemm_dual(C.byref(dual), p16, p16, p16, p16, 1, p16, 32, 120, p16, None) == -2  # K % 32
    assert L.sdq_gemm_dual(C.byref(dual), None, p16, p16, p16, 1, p16, 32, 128, p16, None) == -1
    assert L.sdq_gemm_dual(C.byref(cfg), p16, p16, p16, p16, 1, p16, 32, 128, p16, None) == -3  # INT config
    for s in list(_lib.STATUS) + [123]:
        assert L.sdq_status_string(s)


def test_fp16_scale_overflow_is_an_error():
    W = np.zeros((32, 128), np.float32)
    W[0, 0] = 1e6  # inlier scale 1e6/7 > 65504 (it is an inlier: the outlier is the other 1e6)
    W[0, 1] = 1e6
    with pytest.raises(sdq.SDQError) as e:
        sdq.pack(W, sdq.Config.int_family())
    assert e.value.status == -7


def test_library_exports_every_header_symbol():
    text = open(HEADER).read()
    declared = set(re.findall(r"^\s*(?:sdq_status|const char\*)\s+(sdq_\w+)\s*\(", text, re.M))
    assert declared == set(_lib.EXPORTS)
    L = _lib.lib()
    for name in declared:
        assert hasattr(L, name), name


def test_library_shares_the_hip_runtime_torch_uses():
    """Loaded before torch is imported, the library must still end up on the
    same HIP runtime as torch: one libamdhip64 mapped in the process (two would
    leave the library's launches without a device)."""
    import subprocess
    import sys
    code = ("import sys; sys.path.insert(0, sys.argv[1]); from paper_2406_13868_amd import _lib; "
            "_lib.lib(); import torch; r = _lib._hip_runtimes(); assert len(r) == 1, r; print('ok')")
    p = subprocess.run([sys.executable, "-c", code, os.path.dirname(HERE)], capture_output=True, text=True,
                       timeout=300)
    assert p.returncode == 0 and p.stdout.strip() == "ok", p.stderr[-2000:]


def test_unpacked_entry_points_validate():
    """sdq_unpack_weights / sdq_gemm_unpacked: argument errors before any GPU work."""
    L = _lib.lib()
    mx = sdq.Config.mx_family().c()
    p16 = C.c_void_p(16)
    N, K = 64, 256
    need = 32 * 2 * K
    assert L.sdq_unpack_weights(C.byref(sdq.Config.int_family().c()), p16, N, K, p16, need, None) == -6
    assert L.sdq_unpack_weights(C.byref(sdq.Config.mx_family(n_o=0).c()), p16, N, K, p16, need, None) == -6
    assert L.sdq_unpack_weights(C.byref(mx), None, N, K, p16, need, None) == -1
    assert L.sdq_unpack_weights(C.byref(mx), p16, N, K, None, need, None) == -1
    assert L.sdq_unpack_weights(C.byref(mx), p16, N, K, p16, need - 1, None) == -4
    assert L.sdq_unpack_weights(C.byref(mx), C.c_void_p(8), N, K, p16, need, None) == -2
    assert L.sdq_unpack_weights(C.byref(mx), p16, N, 120, p16, need, None) == -2
    assert L.sdq_gemm_unpacked(C.byref(mx), p16, p16, 0, p16, N, K, p16, need, p16, None) == 0  # M = 0
    assert L.sdq_gemm_unpacked(C.byref(mx), p16, p16, 4, p16, N, K, p16, need - 16, p16, None) == -4
    assert L.sdq_gemm_unpacked(C.byref(mx), None, p16, 4, p16, N, K, p16, need, p16, None) == -1
    assert L.sdq_gemm_unpacked(C.byref(mx), p16, p16, 4, p16, N, K, p16, need, C.c_void_p(18), None) == -2
    assert L.sdq_gemm_unpacked(C.byref(sdq.Config.int_family().c()), p16, p16, 4, p16, N, K, p16, need, p16,
                               None) == -6
    n = C.c_size_t()
    assert L.sdq_gemm_workspace_size(C.byref(mx), 4, N, K, sdq.PATH_DENSE, C.byref(n)) == 0 and n.value == need


def test_gemm_path_choice():
    cfg = sdq.Config.int_family()
    assert sdq.gemm_path(cfg, 1, 4096, 4096) == sdq.PATH_DECODE
    assert sdq.gemm_path(cfg, 2048, 4096, 4096) == sdq.PATH_MFMA
    assert sdq.gemm_path(sdq.Config.mx_family(), 1, 4096, 4096) == sdq.PATH_MFMA
    # the decode kernel up to 8 tokens where its registers fit the row
    for M in range(1, 9):
        assert sdq.gemm_path(cfg, M, 4096, 4096) == sdq.PATH_DECODE, M
    assert sdq.gemm_path(cfg, 9, 4096, 4096) == sdq.PATH_MFMA
    assert sdq.gemm_path(cfg, 2, 4096, 11008) == sdq.PATH_DECODE
    assert sdq.gemm_path(cfg, 3, 4096, 11008) == sdq.PATH_MFMA
    # the two-pass MX path only on a grid of at least 160 workgroups
    mx = sdq.Config.mx_family()
    # the MX split-K path where the one-pass grid of 128 x 128 holds at most 128 workgroups
    for (M, N, K) in ((1, 4096, 4096), (64, 11008, 4096), (128, 11008, 4096), (256, 4096, 11008),
                      (512, 4096, 4096), (16, 4096, 1024)):
        assert sdq.gemm_path(mx, M, N, K, workspace=True) == sdq.PATH_SPLITK, (M, N, K)
        assert sdq.gemm_path(mx, M, N, K) == sdq.PATH_MFMA  # without a workspace: one pass
    for (M, N, K) in ((256, 11008, 4096), (768, 4096, 4096), (16, 4096, 896)):
        assert sdq.gemm_path(mx, M, N, K, workspace=True) == sdq.PATH_MFMA, (M, N, K)
    assert sdq.gemm_path(mx, 512, 11008, 4096, workspace=True) == sdq.PATH_DENSE
    assert sdq.gemm_path(mx, 1024, 4096, 4096, workspace=True) == sdq.PATH_MFMA
    assert sdq.gemm_path(mx, 2048, 4096, 4096, workspace=True) == sdq.PATH_DENSE
    # the INT split-K path where it measured faster than the matrix-core path
    for (M, N, K) in ((16, 4096, 16384), (64, 4096, 16384), (64, 11008, 4096), (64, 16384, 4096),
                      (256, 4096, 4096), (256, 11008, 4096),
                      (257, 4096, 4096), (1024, 4096, 4096), (512, 11008, 4096), (1024, 4096, 11008)):
        assert sdq.gemm_path(cfg, M, N, K, workspace=True) == sdq.PATH_SPLITK, (M, N, K)
        assert sdq.gemm_workspace_size(cfg, M, N, K) > 0
    # above 256 tokens only while the tiled grid of ceil(N/128) x ceil(M/128)
    # workgroups stays under 384, and with K for two ranges
    for (M, N, K) in ((16, 16384, 4096), (32, 16384, 4096), (64, 4096, 4096), (128, 4096, 4096),
                      (1536, 4096, 4096), (640, 11008, 4096), (512, 4096, 896),
                      (4096, 4096, 4096)):
        assert sdq.gemm_path(cfg, M, N, K, workspace=True) == sdq.PATH_MFMA, (M, N, K)
        assert sdq.gemm_workspace_size(cfg, M, N, K) == 0
    assert sdq.gemm_path(cfg, 4, 4096, 4096, workspace=True) == sdq.PATH_DECODE
    assert sdq.gemm_path(cfg, 4, 4096, 16384) == sdq.PATH_MFMA  # the decode kernel does not fit
    assert sdq.gemm_path(cfg, 4, 4096, 16384, workspace=True) == sdq.PATH_SPLITK
    # its workspace: 4 * S * M * N bytes with S K ranges of at least 4 chunks
    for (M, N, K) in ((64, 16384, 4096), (16, 4096, 16384), (0, 4096, 4096), (200, 100, 128)):
        b = sdq.gemm_workspace_size(cfg, M, N, K, sdq.PATH_SPLITK)
        S = b // max(4 * M * N, 1)
        assert b == 4 * S * M * N and 1 <= max(S, 1) <= max(1, K // 512), (M, N, K, S)
    # the tiled kernel over K ranges (long rows, wide layers, above 256 tokens):
    # about 512 workgroups of 128 outputs x 128 tokens
    assert sdq.gemm_workspace_size(cfg, 256, 4096, 11008, sdq.PATH_SPLITK) == 8 * 256 * 4096 * 4
    assert sdq.gemm_workspace_size(cfg, 512, 4096, 4096, sdq.PATH_SPLITK) == 4 * 512 * 4096 * 4
    assert sdq.gemm_workspace_size(cfg, 512, 11008, 4096, sdq.PATH_SPLITK) == 2 * 512 * 11008 * 4
    # the MX family's split-K path: S K ranges of at least 4 chunks, about 512 workgroups
    for (M, N, K) in ((256, 4096, 4096), (128, 11008, 4096), (256, 4096, 11008), (64, 64, 288)):
        b = sdq.gemm_workspace_size(mx, M, N, K, sdq.PATH_SPLITK)
        S = b // (4 * M * N)
        assert b == 4 * S * M * N and 1 <= S <= max(1, -(-K // 128) // 4), (M, N, K, S)
    with pytest.raises(sdq.SDQError):
        sdq.gemm_workspace_size(sdq.Config.dual_family(), 64, 4096, 4096, sdq.PATH_SPLITK)


def test_gemm_workspace_size_and_validation():
    """The two-pass MX path: its workspace is one byte per weight position of
    the 32-row tiles, its automatic choice, and the checks that run before any
    GPU work."""
    mx, mx_no = sdq.Config.mx_family(), sdq.Config("mx", 0, 8, "e4m3", 2, 8, "e2m1", "e4m3")
    it = sdq.Config.int_family()
    assert sdq.gemm_workspace_size(mx, 2048, 11008, 4096) == 11008 * 4096
    assert sdq.gemm_workspace_size(mx, 512, 11008, 4096) == 11008 * 4096  # 43 x 4 workgroups
    assert sdq.gemm_workspace_size(mx, 512, 100, 384) == 0               # one pass: K holds one range
    assert sdq.gemm_workspace_size(mx, 512, 100, 1024) == 2 * 4 * 512 * 100  # split-K: two ranges
    assert sdq.gemm_workspace_size(mx, 1024, 4096, 4096) == 0            # 16 x 8 workgroups
    assert sdq.gemm_workspace_size(mx, 511, 11008, 4096) == 0            # one pass below 512 tokens
    assert sdq.gemm_workspace_size(mx, 512, 100, 384, sdq.PATH_DENSE) == 128 * 384  # N padded to 32
    assert sdq.gemm_workspace_size(mx, 1, 100, 384, sdq.PATH_DENSE) == 128 * 384
    assert sdq.gemm_workspace_size(mx, 4096, 100, 384, sdq.PATH_MFMA) == 0
    assert sdq.gemm_workspace_size(mx_no, 4096, 100, 384) == 0           # no outlier branch
    assert sdq.gemm_workspace_size(it, 4096, 100, 384) == 0
    for cfg in (mx_no, it):
        with pytest.raises(sdq.SDQError) as e:
            sdq.gemm_workspace_size(cfg, 4096, 100, 384, sdq.PATH_DENSE)
        assert e.value.status == -6
    L = _lib.lib()
    c = mx.c()
    p = C.c_void_p(256)  # never dereferenced: every call below fails its checks first
    need = 128 * 384
    assert L.sdq_gemm_ws(C.byref(c), p, p, 300, p, 100, 384, p, p, need - 1, None, 3) == -4
    assert L.sdq_gemm_ws(C.byref(c), p, p, 300, p, 100, 384, p, None, need, None, 3) == -1
    assert L.sdq_gemm_ws(C.byref(c), p, p, 300, p, 100, 384, p, C.c_void_p(264), need, None, 3) == -2
    assert L.sdq_gemm_ws(C.byref(c), p, p, 300, p, 100, 384, p, p, need, None, 9) == -3
    assert L.sdq_gemm_ws(C.byref(c), p, p, 0, p, 100, 384, p, None, 0, None, 3) == 0   # M = 0
    assert L.sdq_gemm_ws(C.byref(it.c()), p, p, 300, p, 100, 384, p, p, need, None, 3) == -6
    # the entry point without a workspace refuses, on the host, what the static
    # scratch cannot hold, and otherwise validates like sdq_gemm_ws
    big_n = 16384
    assert L.sdq_gemm_static(C.byref(c), p, p, 600, p, big_n, 4096, p, None, 3) == -8
    assert L.sdq_gemm_static(C.byref(c), p, p, 300, p, 100, 384, p, None, 9) == -3
    assert L.sdq_gemm_static(C.byref(c), None, p, 300, p, 100, 384, p, None, 3) == -1
    assert L.sdq_gemm_static(C.byref(c), p, p, 0, p, 100, 384, p, None, 3) == 0   # M = 0
    assert L.sdq_gemm_static(C.byref(it.c()), p, p, 300, p, 100, 384, p, None, 3) == -6
    assert b"SDQ_ERR_TOO_LARGE" in L.sdq_status_string(-8)
    assert L.sdq_gemm_ex(C.byref(c), p, p, 300, p, 100, 384, p, None, 3) == -6  # needs a workspace


@pytest.mark.parametrize("c", [c for c in CONFIGS if c[1] == 0 or c[2] == 16], ids=_ids)
def test_absent_outlier_position_is_free(c):
    """A group word without an outlier (1:16 words, or no outlier branch) keeps
    its outlier position off every inlier position (kernels scatter all four
    slots of a word into one dense fragment)."""
    cfg, cfg_o = _cfgs(*c)
    N, K = 64, 512
    blob = sdq.pack(synth.make_w(5, 0, N, K), cfg)
    n_words = ((N + 31) // 32) * (K // 128) * 512
    w = np.frombuffer(blob[: n_words * 4].tobytes(), dtype=np.uint32).astype(np.int64)
    po = ((w >> 3) & 1) | ((w >> 10) & 2) | ((w >> 17) & 4)
    absent = (w >> 24) == 0
    for j in range(cfg_o.n_i):
        pj = (w >> (8 * j)) & 7
        assert not np.any(absent & (po == pj)), f"slot {j}"


# ---- decomposition-metric variants (Section 5, "Stage 2"; Section 6.4's study)
DECOMPS = [(d, o) for d in ("same", "magnitude", "product", "error", "output_error")
           for o in ("large", "small") if (d, o) != ("same", "large")]


@pytest.mark.parametrize("decomp,order", DECOMPS, ids=lambda v: str(v))
@pytest.mark.parametrize("c", [c for c in CONFIGS if c[1] == 1], ids=_ids)
def test_decomposition_variants_match_oracle(c, decomp, order):
    fam, n_o, m_o, fmt_o, n_i = c
    lib, ora = _cfgs(fam, n_o, m_o, fmt_o, n_i, "product")
    import dataclasses
    lib = dataclasses.replace(lib, decomp=decomp, order=order)
    ora = dataclasses.replace(ora, decomp=decomp, order=order)
    N, K = 40, 256
    W = synth.make_w(1, 0, N, K)
    W[3, 10:14] = W[3, 2]           # ties inside groups
    W[5, :8] = 0.0                  # an all-zero group
    an = np.exp(np.random.default_rng(7).standard_normal(K)).astype(np.float32)
    _compare_logical(sdq.pack_logical(W, lib, act_norm=an), S.pack_logical(W, ora, act_norm=an), ora)
    # and the kernel layout carries the same codes
    blob = sdq.pack(W, lib, act_norm=an)
    U = sdq.unpack_dense(blob, lib, N, K)
    Lo = S.pack_logical(W, ora, act_norm=an)
    assert np.array_equal(U["code_o_dense"], Lo["code_o_dense"])


def test_decomposition_variant_errors():
    W = np.zeros((32, 128), np.float32)
    with pytest.raises(sdq.SDQError) as e:   # a variant needs an outlier branch
        sdq.pack(W, sdq.Config("int", 0, 8, "e4m3", 3, decomp="error"))
    assert e.value.status == -3
    for d in ("product", "output_error"):     # these read the activation norms
        with pytest.raises(sdq.SDQError) as e:
            sdq.pack(W, sdq.Config("int", 1, 8, "e4m3", 3, decomp=d))
        assert e.value.status == -1
    cfg = sdq.Config("int", 1, 8, "e4m3", 3).c()
    cfg.decomp = 5
    n = C.c_size_t()
    assert _lib.lib().sdq_pack_size(C.byref(cfg), 32, 128, C.byref(n)) == -3
    cfg.decomp, cfg.order = 0, 2
    assert _lib.lib().sdq_pack_size(C.byref(cfg), 32, 128, C.byref(n)) == -3


# ---- two-level e4m3 inlier scales (Section 3.3: quantized scale factors)
@pytest.mark.parametrize("c", [c for c in CONFIGS if c[0] == "int"], ids=_ids)
def test_e4m3_scales_match_oracle(c):
    import dataclasses
    fam, n_o, m_o, fmt_o, n_i = c
    lib, ora = _cfgs(fam, n_o, m_o, fmt_o, n_i)
    lib = dataclasses.replace(lib, sfmt_i="e4m3")
    ora = dataclasses.replace(ora, sfmt_i="e4m3")
    N, K = 40, 384
    W = synth.make_w(1, 0, N, K)
    W[5, :] = 0.0                   # a row without inlier magnitude: row scale 0
    W[6, :32] *= np.float32(1e-6)   # blocks far below the row's largest: e4m3 subnormal scales
    Lg, Lo = sdq.pack_logical(W, lib), S.pack_logical(W, ora)
    assert np.array_equal(Lg["pos_i"], Lo["pos_i"].astype(np.uint8))
    assert np.array_equal(Lg["code_i"].view(np.int8), Lo["code_i"].astype(np.int8))
    assert np.array_equal(Lg["scale_i"], Lo["scale_i"])
    assert np.array_equal(Lg["scale_i_row"].view(np.uint32), Lo["scale_i_row"].view(np.uint32))
    if n_o:
        assert np.array_equal(Lg["code_o"], Lo["code_o"])
    U = sdq.unpack_dense(sdq.pack(W, lib), lib, N, K)
    assert np.array_equal(U["scale_i"], Lo["scale_i"])
    assert np.array_equal(U["scale_i_row"], Lo["scale_i_row"])
    assert np.array_equal(U["code_i_dense"].view(np.int8), Lo["code_i_dense"].astype(np.int8))


def test_e4m3_scales_sizes_and_validation():
    lib = sdq.Config("int", 1, 8, "e4m3", 3, sfmt_i="e4m3")
    N, K = 4096, 4096
    n16 = C.c_size_t()
    n8 = C.c_size_t()
    L = _lib.lib()
    assert L.sdq_logical_bytes(C.byref(sdq.Config("int", 1, 8, "e4m3", 3).c()), N, K, C.byref(n16)) == 0
    assert L.sdq_logical_bytes(C.byref(lib.c()), N, K, C.byref(n8)) == 0
    # 8 bits instead of 16 per 16-K block, plus 32 bits per row
    assert n16.value - n8.value == N * (K // 16) - N * 4
    ps16, ps8 = C.c_size_t(), C.c_size_t()
    L.sdq_pack_size(C.byref(sdq.Config("int", 1, 8, "e4m3", 3).c()), N, K, C.byref(ps16))
    L.sdq_pack_size(C.byref(lib.c()), N, K, C.byref(ps8))
    assert ps16.value - ps8.value == N * (K // 16) - N * 4
    mx = sdq.Config("mx", 1, 8, "e4m3", 2, 8, "e2m1", "e4m3", sfmt_i="e4m3").c()
    assert L.sdq_pack_size(C.byref(mx), 32, 128, C.byref(ps8)) == -3   # INT family only


# ---- the dual family (Section 5.1's int8 A_o / fp4 A_i configuration)
@pytest.mark.parametrize("n_o,n_i,metric,decomp", [(1, 6, "magnitude", "same"), (1, 6, "product", "error"),
                                                   (1, 7, "magnitude", "same"), (1, 3, "product", "same"),
                                                   (0, 8, "magnitude", "same"), (0, 5, "magnitude", "same"),
                                                   (2, 4, "magnitude", "same"), (2, 4, "product", "error"),
                                                   (2, 6, "magnitude", "same"), (2, 1, "product", "same")])
@pytest.mark.parametrize("K", [384, 160])
def test_dual_pack_matches_oracle(n_o, n_i, metric, decomp, K):
    N = 40
    W = synth.make_w(2, 0, N, K)
    W[4, :] = 0.0
    W[6, :40] *= np.float32(1e-6)
    an = np.exp(np.random.default_rng(1).standard_normal(K)).astype(np.float32)
    c = sdq.Config("dual", n_o, 8, "int8", n_i, 8, "e2m1", "int8", metric, decomp)
    co = S.Config("dual", n_o, 8, "int8", n_i, 8, "e2m1", "int8+e2m1", metric, decomp)
    Lg, Lo = sdq.pack_logical(W, c, act_norm=an), S.pack_logical(W, co, act_norm=an)
    assert np.array_equal(Lg["pos_i"], Lo["pos_i"].astype(np.uint8))
    assert np.array_equal(Lg["code_i"], Lo["code_i"])
    assert np.array_equal(Lg["scale_i"], Lo["scale_i"])
    if n_o:
        assert np.array_equal(Lg["pos_o"], Lo["pos_o"].astype(np.uint8))
        assert np.array_equal(Lg["code_o"], Lo["code_o"])
        assert np.array_equal(Lg["scale_o"].view(np.uint32), Lo["scale_o"].view(np.uint32))
    U = sdq.unpack_dense(sdq.pack(W, c, act_norm=an), c, N, K)
    assert np.array_equal(U["code_i_dense"], Lo["code_i_dense"])
    assert np.array_equal(U["code_o_dense"], Lo["code_o_dense"])
    assert np.array_equal(U["scale_i"], Lo["scale_i"])


def test_dual_sizes_and_validation():
    L = _lib.lib()
    n = C.c_size_t()
    dual = sdq.Config.dual_family()
    N, K = 4096, 4096
    assert L.sdq_pack_size(C.byref(dual.c()), N, K, C.byref(n)) == 0
    # dense fp4 nibbles (4 b/w), outlier half-words (2 b/w), e8m0 per 32 (0.25 b/w), fp32 per row
    assert n.value == N * K // 2 + N * K // 4 + N * K // 32 + N * 4
    assert L.sdq_logical_bytes(C.byref(dual.c()), N, K, C.byref(n)) == 0
    # 1:8 int8 (8+3 bits per 8) + 6:8 fp4 (6 x (4+3) per 8) + e8m0 per 32 + fp32 per row
    assert n.value == (N * (K // 8 * 11 + K // 8 * 42 + K // 32 * 8 + 32) + 7) // 8
    assert L.sdq_pack_size(C.byref(sdq.Config("dual", 1, 16, "int8", 6, 8, "e2m1", "int8").c()), 32, 128,
                           C.byref(n)) == -6      # 1:16 outliers not built for this family
    # 2:8 outliers: a second plane of half-words (2 more bits per weight)
    two = sdq.Config("dual", 2, 8, "int8", 4, 8, "e2m1", "int8")
    assert L.sdq_pack_size(C.byref(two.c()), N, K, C.byref(n)) == 0
    assert n.value == N * K // 2 + 2 * (N * K // 4) + N * K // 32 + N * 4
    assert L.sdq_logical_bytes(C.byref(two.c()), N, K, C.byref(n)) == 0
    assert n.value == (N * (K // 8 * 22 + K // 8 * 28 + K // 32 * 8 + 32) + 7) // 8
    for bad in (sdq.Config("dual", 3, 8, "int8", 4, 8, "e2m1", "int8"),
                sdq.Config("dual", 2, 8, "int8", 7, 8, "e2m1", "int8")):
        assert L.sdq_pack_size(C.byref(bad.c()), 32, 128, C.byref(n)) in (-3, -6)
    # int8 outliers sum exactly in int32 up to K = 2^19
    for c8 in (two, dual, sdq.Config.int_family(1, 8, "int8", 3)):
        assert L.sdq_check(C.byref(c8.c()), 32, 1 << 19) == 0
        assert L.sdq_check(C.byref(c8.c()), 32, (1 << 19) + 32) == -2
    assert L.sdq_check(C.byref(sdq.Config.int_family().c()), 32, (1 << 19) + 32) == 0  # e4m3 outliers
    assert L.sdq_pack_size(C.byref(sdq.Config("dual", 1, 8, "e4m3", 6, 8, "e2m1", "int8").c()), 32, 128,
                           C.byref(n)) == -3
    cfg = dual.c()
    assert L.sdq_gemm(C.byref(cfg), C.c_void_p(16), C.c_void_p(16), 1, C.c_void_p(16), 32, 128,
                      C.c_void_p(16), None) == -6
    assert L.sdq_gemm_dual(C.byref(sdq.Config.int_family().c()), None, None, None, None, 1, None, 32, 128,
                           None, None) == -3
    assert L.sdq_gemm_dual(C.byref(cfg), None, None, None, None, 1, None, 32, 128, None, None) == -1
    assert L.sdq_gemm_dual(C.byref(cfg), None, None, None, None, 0, None, 32, 128, None, None) == 0


# ---- Q-Vector 32 / 64 and ufp8-e6m2 inlier scales (Section 3.3: quantized
# scale factors and their vector length; Section 6.4's scale-format study)
@pytest.mark.parametrize("qv", [16, 32, 64])
@pytest.mark.parametrize("sfmt", ["", "e4m3", "ue6m2"])
@pytest.mark.parametrize("c", [c for c in CONFIGS if c[0] == "int"], ids=_ids)
def test_qvector_and_scale_formats_match_oracle(c, sfmt, qv):
    import dataclasses
    fam, n_o, m_o, fmt_o, n_i = c
    lib, ora = _cfgs(fam, n_o, m_o, fmt_o, n_i)
    lib = dataclasses.replace(lib, sfmt_i=sfmt, qv_i=qv)
    ora = dataclasses.replace(ora, sfmt_i=sfmt, qv=qv)
    N, K = 40, 384
    W = synth.make_w(1, 0, N, K)
    W[5, :] = 0.0                   # a row without inlier magnitude
    W[7, 64:128] = 0.0              # all-zero Q-Vectors inside a row
    Lg, Lo = sdq.pack_logical(W, lib), S.pack_logical(W, ora)
    def bits(a):  # stored scales: fp16 bits, or one byte per code
        return a.view(np.uint16) if a.dtype in (np.float16, np.uint16) else a.astype(np.uint8)
    assert Lg["scale_i"].shape == (N, K // qv)
    assert np.array_equal(Lg["pos_i"], Lo["pos_i"].astype(np.uint8))
    assert np.array_equal(Lg["code_i"].view(np.int8), Lo["code_i"].astype(np.int8))
    assert np.array_equal(bits(Lg["scale_i"]), bits(Lo["scale_i"]))
    if sfmt == "e4m3":
        assert np.array_equal(Lg["scale_i_row"].view(np.uint32), Lo["scale_i_row"].view(np.uint32))
    if n_o:
        assert np.array_equal(Lg["code_o"], Lo["code_o"])
    U = sdq.unpack_dense(sdq.pack(W, lib), lib, N, K)
    assert np.array_equal(bits(U["scale_i"]), bits(Lo["scale_i"]))
    assert np.array_equal(U["code_i_dense"].view(np.int8), Lo["code_i_dense"].astype(np.int8))


def test_qvector_sizes_follow_the_scale_bits():
    """Logical and physical bytes shrink by the scale bits the longer Q-Vector saves."""
    N, K = 4096, 4096
    L = _lib.lib()
    def sizes(**kw):
        c = sdq.Config("int", 1, 8, "e4m3", 3, **kw).c()
        lb, pb = C.c_size_t(), C.c_size_t()
        assert L.sdq_logical_bytes(C.byref(c), N, K, C.byref(lb)) == 0
        assert L.sdq_pack_size(C.byref(c), N, K, C.byref(pb)) == 0
        return lb.value, pb.value
    l16, p16 = sizes()
    for qv in (32, 64):
        l, p = sizes(qv_i=qv)
        saved = N * (K // 16 - K // qv) * 2        # fp16 scales no longer stored
        assert l16 - l == saved and p16 - p == saved
    l6, p6 = sizes(sfmt_i="ue6m2", qv_i=64)
    assert l16 - l6 == N * (K // 16) * 2 - N * (K // 64)  # one byte per 64 K
    # validation: INT takes 16/32/64, the MX and dual families only their 32
    c = sdq.Config("int", 1, 8, "e4m3", 3).c()
    pb = C.c_size_t()
    for bad in (8, 48, 128):
        c.qv_i = bad
        assert L.sdq_pack_size(C.byref(c), 32, 256, C.byref(pb)) == -3
    mx = sdq.Config("mx", 1, 8, "e4m3", 2, 8, "e2m1", "e4m3").c()
    mx.qv_i = 64
    assert L.sdq_pack_size(C.byref(mx), 32, 256, C.byref(pb)) == -3
    mx.qv_i, mx.sfmt_i = 32, 2
    assert L.sdq_pack_size(C.byref(mx), 32, 256, C.byref(pb)) == -3   # e6m2 is INT only


def test_e6m2_scales_outside_the_fp16_exact_range_are_refused():
    """A nonzero ufp8-e6m2 scale must lie in [2^-22, 7168] (exponent field
    9..43), where an int4 code times it is exact in fp16; the packer refuses
    weights whose Q-Vector scale falls outside, as it refuses an fp16 overflow."""
    lib = sdq.Config("int", 1, 8, "e4m3", 3, sfmt_i="ue6m2")
    W = synth.make_w(1, 0, 32, 256)
    sdq.pack(W, lib)                                   # workload-scale weights fit
    for scale in (1e-7, 1e7):
        with pytest.raises(sdq.SDQError) as e:
            sdq.pack(W * np.float32(scale), lib)
        assert e.value.status == -7
    Z = np.zeros((32, 256), np.float32)                # zero scales are fine
    sdq.pack(Z, lib)
