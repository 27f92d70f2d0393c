"""SDQ (Sparse Decomposed Quantization) decomposed GEMM for MI355X (gfx950).

Thin Python binding over ``libsdq.so`` (C ABI in ``include/sdq.h``): it only
marshals arguments.  Every step of the hot path (activation quantization and
the decomposed product) runs in the library's HIP kernels; PyTorch provides
device memory and the current stream, nothing else.  There is no CPU
fallback: if the library is missing every call raises.

    cfg = Config.int_family(n_o=1, m_o=8, fmt_o="e4m3", n_i=3)
    blob = pack(W, cfg)                      # host numpy, offline (Section 5)
    packed = torch.from_numpy(blob).cuda()
    Xq, s_a = quantize_act(X_cuda, cfg)      # per-token activation quantization
    Y = gemm(Xq, s_a, packed, N, K, cfg)     # Y = s_a * Xq (W_o + W_i)^T (Section 5.1)
"""
from __future__ import annotations

import ctypes as C
import dataclasses
from typing import Dict, Optional

import numpy as np

from . import _lib
from ._lib import (DTYPE_BF16, DTYPE_F32, FAMILY_DUAL, FAMILY_INT, FAMILY_MX, FMT_E2M1, FMT_E4M3, FMT_INT4,
                   FMT_INT8, METRIC_MAGNITUDE, METRIC_PRODUCT, PATH_AUTO, PATH_DECODE, PATH_MFMA,
                   PATH_DENSE, PATH_SPLITK,
                   SDQError)

__all__ = ["Config", "pack", "pack_logical", "unpack_dense", "pack_size", "logical_bytes",
           "quantize_act", "gemm", "linear", "gemm_path", "SDQError", "PATH_AUTO", "PATH_DECODE",
           "PATH_MFMA", "PATH_DENSE", "PATH_SPLITK", "gemm_workspace_size", "check", "quantize_act_dual", "gemm_dual",
           "gemm_static", "unpack_weights", "gemm_unpacked"]

_FMT = {"int8": FMT_INT8, "int4": FMT_INT4, "e4m3": FMT_E4M3, "e2m1": FMT_E2M1}


@dataclasses.dataclass(frozen=True)
class Config:
    family: str = "int"      # "int" | "mx" | "dual"
    n_o: int = 1
    m_o: int = 8
    fmt_o: str = "e4m3"      # "e4m3" | "int8"
    n_i: int = 3
    m_i: int = 8
    fmt_i: str = "int4"      # "int4" | "e2m1"
    fmt_a: str = "int8"      # "int8" | "e4m3"
    metric: str = "magnitude"  # significance: "magnitude" | "product"
    decomp: str = "same"       # outlier metric: "same" | "magnitude" | "product" | "error" | "output_error"
    order: str = "large"       # outliers by the largest ("large") or smallest ("small") decomp metric
    sfmt_i: str = ""           # inlier scales: "" (int fp16 / mx e8m0) | "e4m3" (int, two-level) | "ue6m2" (int)
    y_dtype: str = "f32"       # GEMM output: "f32" | "bf16" (the fp32 result rounded to nearest even)
    qv_i: int = 0              # dense K per inlier scale: 0 = the family's (int 16, mx/dual 32); int 16/32/64

    @staticmethod
    def int_family(n_o=1, m_o=8, fmt_o="e4m3", n_i=3, metric="magnitude") -> "Config":
        return Config("int", n_o, m_o, fmt_o, n_i, 8, "int4", "int8", metric)

    @staticmethod
    def mx_family(n_o=1, m_o=8, n_i=2, metric="magnitude") -> "Config":
        return Config("mx", n_o, m_o, "e4m3", n_i, 8, "e2m1", "e4m3", metric)

    @staticmethod
    def of(fmt, metric: str = "magnitude") -> "Config":
        """From any object with the same field names (e.g. a workload format)."""
        return Config(fmt.family, fmt.n_o, fmt.m_o, fmt.fmt_o, fmt.n_i, fmt.m_i, fmt.fmt_i,
                      fmt.fmt_a, metric)

    @staticmethod
    def dual_family(n_o=1, n_i=6, metric="magnitude") -> "Config":
        """Section 5.1's worked configuration: n_o:8 int8 outliers against int8
        activations, n_i:8 fp4 inliers against fp4 (MXFP4) activations."""
        return Config("dual", n_o, 8, "int8", n_i, 8, "e2m1", "int8", metric)

    @property
    def label(self) -> str:
        """The formats as '{family}-{n_o}:{m_o}{fmt_o}-{n_i}:{m_i}{fmt_i}-A{fmt_a}', the
        form Config.parse reads back (metric and the other options are not part of it)."""
        return (f"{self.family}-{self.n_o}:{self.m_o}{self.fmt_o}-{self.n_i}:{self.m_i}{self.fmt_i}"
                f"-A{self.fmt_a}")

    @staticmethod
    def parse(label: str) -> "Config":
        """A configuration from a label: this library's form (Config.label, e.g.
        'mx-1:8e4m3-2:8e2m1-Ae4m3'), or the paper's SDQ names (Section 6.2's
        tables, e.g. 'SDQ-W7:8-1:8int8-6:8fp4': W for Wanda sparsification,
        i.e. the weight-activation product metric; then the kept N:M, the
        outliers' n:m and format, the inliers' n:m and format).  int8
        outliers with fp4 inliers are the dual family, with int4 inliers the
        INT family; the kept N must equal n_o + n_i.  Raises ValueError for
        anything else (SparseGPT, 'SDQ-S...', is not built).  Whether the
        kernels implement the result is for check() to say."""
        import re
        m = re.fullmatch(r"(int|mx|dual)-(\d+):(\d+)(e4m3|int8)-(\d+):(\d+)(int4|e2m1)-A(int8|e4m3)", label)
        if m:
            fam, n_o, m_o, fo, n_i, m_i, fi, fa = m.groups()
            return Config(fam, int(n_o), int(m_o), fo, int(n_i), int(m_i), fi, fa)
        m = re.fullmatch(r"SDQ-([A-Z])(\d+):(\d+)-(\d+):(\d+)(int8|fp8)-(\d+):(\d+)(fp4|int4)", label)
        if not m:
            raise ValueError(f"not a configuration label: {label!r}")
        sp, kept, m_kept, n_o, m_o, fo, n_i, m_i, fi = m.groups()
        if sp != "W":
            raise ValueError(f"{label!r}: sparsifier {sp!r} is not built (W, the Wanda product metric, is)")
        if int(kept) != int(n_o) + int(n_i) or not (int(m_kept) == int(m_o) == int(m_i)):
            raise ValueError(f"{label!r}: kept {kept}:{m_kept} is not outliers {n_o}:{m_o} + inliers {n_i}:{m_i}")
        if fo != "int8":
            raise ValueError(f"{label!r}: {fo} outliers with {fi} inliers is not a configuration of this library")
        if fi == "fp4":
            return Config("dual", int(n_o), int(m_o), "int8", int(n_i), int(m_i), "e2m1", "int8", "product")
        return Config("int", int(n_o), int(m_o), "int8", int(n_i), int(m_i), "int4", "int8", "product")

    @property
    def mx(self) -> bool:
        return self.family == "mx"

    @property
    def qv(self) -> int:
        """Dense K positions per inlier scale."""
        return self.qv_i or (16 if self.family == "int" else 32)

    @property
    def byte_scales(self) -> bool:
        """INT-family inlier scales of one byte (e4m3, e6m2) rather than fp16."""
        return self.sfmt_i in ("e4m3", "ue6m2")

    @property
    def e8m0_inliers(self) -> bool:
        """Inlier scales are e8m0 per 32 K (mx and dual families)."""
        return self.family in ("mx", "dual")

    def c(self) -> _lib.sdq_config:
        fam = {"int": FAMILY_INT, "mx": FAMILY_MX, "dual": FAMILY_DUAL}[self.family]
        return _lib.sdq_config(fam, self.n_o, self.m_o,
                               _FMT[self.fmt_o], self.n_i, self.m_i, _FMT[self.fmt_i],
                               _FMT[self.fmt_a],
                               METRIC_PRODUCT if self.metric == "product" else METRIC_MAGNITUDE,
                               _lib.DECOMP[self.decomp], _lib.ORDER[self.order],
                               _lib.SCALE[self.sfmt_i],
                               {"f32": DTYPE_F32, "bf16": DTYPE_BF16}[self.y_dtype], self.qv_i)

    def y_torch_dtype(self):
        import torch
        return torch.bfloat16 if self.y_dtype == "bf16" else torch.float32


def _p(a) -> C.c_void_p:
    return C.c_void_p(a.ctypes.data) if a is not None else None


def check(cfg: Config, N: int, K: int) -> None:
    _lib.check(_lib.lib().sdq_check(C.byref(cfg.c()), N, K), "sdq_check")


def pack_size(cfg: Config, N: int, K: int) -> int:
    n = C.c_size_t()
    _lib.check(_lib.lib().sdq_pack_size(C.byref(cfg.c()), N, K, C.byref(n)), "sdq_pack_size")
    return n.value


def logical_bytes(cfg: Config, N: int, K: int) -> int:
    n = C.c_size_t()
    _lib.check(_lib.lib().sdq_logical_bytes(C.byref(cfg.c()), N, K, C.byref(n)),
               "sdq_logical_bytes")
    return n.value


def pack(W: np.ndarray, cfg: Config, act_norm: Optional[np.ndarray] = None,
         n_threads: int = 0) -> np.ndarray:
    """Offline decomposition + quantization into the kernel layout (host)."""
    W = np.ascontiguousarray(W, dtype=np.float32)
    N, K = W.shape
    an = None if act_norm is None else np.ascontiguousarray(act_norm, dtype=np.float32)
    out = np.empty(pack_size(cfg, N, K), dtype=np.uint8)
    _lib.check(_lib.lib().sdq_pack(C.byref(cfg.c()), _p(W), N, K, _p(an), _p(out), out.nbytes,
                                   n_threads), "sdq_pack")
    return out


def pack_logical(W: np.ndarray, cfg: Config, act_norm: Optional[np.ndarray] = None,
                 n_threads: int = 0) -> Dict[str, np.ndarray]:
    W = np.ascontiguousarray(W, dtype=np.float32)
    N, K = W.shape
    an = None if act_norm is None else np.ascontiguousarray(act_norm, dtype=np.float32)
    no = max(cfg.n_o, 0)
    pos_o = np.zeros((N, K // cfg.m_o, no), np.uint8)
    code_o = np.zeros((N, K // cfg.m_o, no), np.uint8)
    pos_i = np.zeros((N, K // cfg.m_i, cfg.n_i), np.uint8)
    code_i = np.zeros((N, K // cfg.m_i, cfg.n_i), np.uint8)
    if cfg.mx:
        scale_o = np.zeros((N, K // 32), np.uint8)
        scale_i = np.zeros((N, K // 32), np.uint8)
    elif cfg.family == "dual":
        scale_o = np.zeros(N, np.float32)
        scale_i = np.zeros((N, K // 32), np.uint8)
    else:
        scale_o = np.zeros(N, np.float32)
        scale_i = np.zeros((N, K // cfg.qv), np.uint8 if cfg.byte_scales else np.uint16)
    scale_i_row = np.zeros(N, np.float32)
    _lib.check(_lib.lib().sdq_pack_logical(
        C.byref(cfg.c()), _p(W), N, K, _p(an), _p(pos_o), _p(code_o), _p(scale_o), _p(pos_i),
        _p(code_i), _p(scale_i), _p(scale_i_row), n_threads), "sdq_pack_logical")
    return dict(pos_o=pos_o, code_o=code_o, scale_o=scale_o, pos_i=pos_i, code_i=code_i,
                scale_i=scale_i, scale_i_row=scale_i_row)


def unpack_dense(blob: np.ndarray, cfg: Config, N: int, K: int) -> Dict[str, np.ndarray]:
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    co = np.zeros((N, K), np.uint8)
    ci = np.zeros((N, K), np.uint8)
    if cfg.mx:
        so, si = np.zeros((N, K // 32), np.uint8), np.zeros((N, K // 32), np.uint8)
    elif cfg.family == "dual":
        so, si = np.zeros(N, np.float32), np.zeros((N, K // 32), np.uint8)
    else:
        so = np.zeros(N, np.float32)
        si = np.zeros((N, K // cfg.qv), np.uint8 if cfg.byte_scales else np.uint16)
    sr = np.zeros(N, np.float32)
    _lib.check(_lib.lib().sdq_unpack_dense(C.byref(cfg.c()), _p(blob), blob.nbytes, N, K, _p(co),
                                           _p(ci), _p(so), _p(si), _p(sr)), "sdq_unpack_dense")
    return dict(code_o_dense=co, code_i_dense=ci, scale_o=so, scale_i=si, scale_i_row=sr)


# ----------------------------------------------------------------- device side
def _stream(stream) -> C.c_void_p:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _dev(t, what: str):
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{what} must be a contiguous CUDA (HIP) tensor")
    return C.c_void_p(t.data_ptr())


def _need(t, shape, dtype, what: str):
    """Check a caller-supplied tensor before its pointer reaches the library,
    which cannot see sizes: exact shape and dtype (placement and contiguity are
    checked where the pointer is taken)."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{what} must be a torch tensor")
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype:
        raise ValueError(f"{what} must be {list(shape)} {dtype}, got {list(t.shape)} {t.dtype}")
    return t


def _need_bytes(t, nbytes: int, what: str):
    """A raw byte buffer (packed weights, workspace): at least nbytes."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{what} must be a torch tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{what} holds {have} bytes, needs {nbytes}")
    return t


def _x_dtype(X):
    import torch
    if X.dtype == torch.float32:
        return DTYPE_F32
    if X.dtype == torch.bfloat16:
        return DTYPE_BF16
    raise ValueError("X must be float32 or bfloat16")


def _same_device(*ts):
    devs = {t.device for t in ts if t is not None}
    if len(devs) > 1:
        raise ValueError(f"tensors are on different devices: {sorted(map(str, devs))}")


def _out(out, M: int, N: int, cfg: Config, device):
    """The GEMM output: `out` checked against [M, N] of cfg's output dtype, or a new tensor."""
    import torch
    dt = cfg.y_torch_dtype()
    if out is None:
        return torch.empty((M, N), dtype=dt, device=device)
    if tuple(out.shape) != (M, N) or out.dtype != dt:
        raise ValueError(f"out must be [{M}, {N}] {dt}, got {list(out.shape)} {out.dtype}")
    return out


def quantize_act(X, cfg: Config, out=None, scales=None, stream=None):
    """Per-token activation quantization on the GPU: returns (Xq uint8, s_a f32)."""
    import torch
    if X.dim() != 2:
        raise ValueError("X must be [M, K]")
    M, K = X.shape
    dt = _x_dtype(X)
    Xq = out if out is not None else torch.empty((M, K), dtype=torch.uint8, device=X.device)
    s_a = scales if scales is not None else torch.empty((M,), dtype=torch.float32, device=X.device)
    _need(Xq, (M, K), torch.uint8, "Xq")
    _need(s_a, (M,), torch.float32, "s_a")
    _same_device(X, Xq, s_a)
    _lib.check(_lib.lib().sdq_quantize_act(C.byref(cfg.c()), _dev(X, "X"), dt, M, K,
                                           _dev(Xq, "Xq"), _dev(s_a, "s_a"), _stream(stream)),
               "sdq_quantize_act")
    return Xq, s_a


def quantize_act_dual(X, cfg: Config, out=None, stream=None):
    """The dual family's activations on the GPU: returns (Xq_o uint8 [M, K],
    s_a_o f32 [M], Xq_i uint8 [M, K/2] fp4 nibbles, e_a_i uint8 [M, K/32] e8m0),
    written into `out` (a tuple of those four tensors) when given."""
    import torch
    if X.dim() != 2:
        raise ValueError("X must be [M, K]")
    M, K = X.shape
    dt = _x_dtype(X)
    dev = X.device
    if out is not None:
        Xo, s_a, Xi, Ea = out
    else:
        Xo = torch.empty((M, K), dtype=torch.uint8, device=dev)
        s_a = torch.empty((M,), dtype=torch.float32, device=dev)
        Xi = torch.empty((M, K // 2), dtype=torch.uint8, device=dev)
        Ea = torch.empty((M, K // 32), dtype=torch.uint8, device=dev)
    _need(Xo, (M, K), torch.uint8, "Xq_o")
    _need(s_a, (M,), torch.float32, "s_a_o")
    _need(Xi, (M, K // 2), torch.uint8, "Xq_i")
    _need(Ea, (M, K // 32), torch.uint8, "e_a_i")
    _same_device(X, Xo, s_a, Xi, Ea)
    _lib.check(_lib.lib().sdq_quantize_act_dual(C.byref(cfg.c()), _dev(X, "X"), dt, M, K, _dev(Xo, "Xq_o"),
                                                _dev(s_a, "s_a_o"), _dev(Xi, "Xq_i"), _dev(Ea, "e_a_i"),
                                                _stream(stream)), "sdq_quantize_act_dual")
    return Xo, s_a, Xi, Ea


def gemm_dual(Xo, s_a, Xi, Ea, packed, N: int, K: int, cfg: Config, out=None, stream=None):
    """The dual family's GEMM on the GPU (output [M, N], fp32 or bf16 by cfg.y_dtype)."""
    import torch
    if Xo.dim() != 2:
        raise ValueError("Xq_o must be [M, K]")
    M = Xo.shape[0]
    _need(Xo, (M, K), torch.uint8, "Xq_o")
    _need(s_a, (M,), torch.float32, "s_a_o")
    _need(Xi, (M, K // 2), torch.uint8, "Xq_i")
    _need(Ea, (M, K // 32), torch.uint8, "e_a_i")
    _need_bytes(packed, pack_size(cfg, N, K), "packed")
    Y = _out(out, M, N, cfg, Xo.device)
    _same_device(Xo, s_a, Xi, Ea, packed, Y)
    _lib.check(_lib.lib().sdq_gemm_dual(C.byref(cfg.c()), _dev(Xo, "Xq_o"), _dev(s_a, "s_a_o"),
                                        _dev(Xi, "Xq_i"), _dev(Ea, "e_a_i"), M, _dev(packed, "packed"),
                                        N, K, _dev(Y, "Y"), _stream(stream)), "sdq_gemm_dual")
    return Y


def gemm_workspace_size(cfg: Config, M: int, N: int, K: int, path: int = PATH_AUTO) -> int:
    """Device workspace bytes the GEMM takes for this shape and path (0: none)."""
    b = C.c_size_t()
    _lib.check(_lib.lib().sdq_gemm_workspace_size(C.byref(cfg.c()), M, N, K, path, C.byref(b)),
               "sdq_gemm_workspace_size")
    return b.value


def gemm(Xq, s_a, packed, N: int, K: int, cfg: Config, out=None, path: int = PATH_AUTO,
         stream=None, workspace=None):
    """Y[M, N] = s_a * (Xq @ (W_o + W_i)^T) on the GPU (fp32 or bf16 output by cfg.y_dtype).

    Paths that take a workspace (the two-pass MX path for many tokens, the
    INT family's split-K path for tens to hundreds of tokens) use
    `workspace` (a uint8 CUDA tensor of at least gemm_workspace_size bytes)
    or a fresh one."""
    import torch
    if Xq.dim() != 2:
        raise ValueError("Xq must be [M, K]")
    M = Xq.shape[0]
    _need(Xq, (M, K), torch.uint8, "Xq")
    _need(s_a, (M,), torch.float32, "s_a")
    _need_bytes(packed, pack_size(cfg, N, K), "packed")
    Y = _out(out, M, N, cfg, Xq.device)
    _same_device(Xq, s_a, packed, Y, workspace)
    ws_bytes = gemm_workspace_size(cfg, M, N, K, path)
    if ws_bytes == 0 and path not in (PATH_DENSE, PATH_SPLITK):
        _lib.check(_lib.lib().sdq_gemm_ex(C.byref(cfg.c()), _dev(Xq, "Xq"), _dev(s_a, "s_a"), M,
                                          _dev(packed, "packed"), N, K, _dev(Y, "Y"),
                                          _stream(stream), path), "sdq_gemm")
        return Y
    ws = workspace if workspace is not None else torch.empty(ws_bytes, dtype=torch.uint8,
                                                             device=Xq.device)
    _need_bytes(ws, ws_bytes, "workspace")
    _lib.check(_lib.lib().sdq_gemm_ws(C.byref(cfg.c()), _dev(Xq, "Xq"), _dev(s_a, "s_a"), M,
                                      _dev(packed, "packed"), N, K, _dev(Y, "Y"),
                                      _dev(ws, "workspace"), ws.numel() * ws.element_size(),
                                      _stream(stream), path), "sdq_gemm_ws")
    return Y


def unpack_weights(packed, N: int, K: int, cfg: Config, workspace=None, stream=None):
    """Pass 1 of the two-pass MX path on its own (sdq_unpack_weights): the blob's
    expanded B operands in `workspace` (a uint8 CUDA tensor of at least
    gemm_workspace_size(cfg, M, N, K, PATH_DENSE) bytes, or a fresh one),
    which is returned for gemm_unpacked."""
    import torch
    _need_bytes(packed, pack_size(cfg, N, K), "packed")
    nb = gemm_workspace_size(cfg, 0, N, K, PATH_DENSE)
    ws = workspace if workspace is not None else torch.empty(nb, dtype=torch.uint8, device=packed.device)
    _need_bytes(ws, nb, "workspace")
    _same_device(packed, ws)
    _lib.check(_lib.lib().sdq_unpack_weights(C.byref(cfg.c()), _dev(packed, "packed"), N, K,
                                             _dev(ws, "workspace"), ws.numel() * ws.element_size(),
                                             _stream(stream)), "sdq_unpack_weights")
    return ws


def gemm_unpacked(Xq, s_a, packed, N: int, K: int, cfg: Config, workspace, out=None, stream=None):
    """Pass 2 of the two-pass MX path (sdq_gemm_unpacked): Y from the operands
    unpack_weights wrote into `workspace` for the same packed, N and K; equal
    to gemm(..., path=PATH_DENSE) bit for bit."""
    import torch
    if Xq.dim() != 2:
        raise ValueError("Xq must be [M, K]")
    M = Xq.shape[0]
    _need(Xq, (M, K), torch.uint8, "Xq")
    _need(s_a, (M,), torch.float32, "s_a")
    _need_bytes(packed, pack_size(cfg, N, K), "packed")
    _need_bytes(workspace, gemm_workspace_size(cfg, M, N, K, PATH_DENSE), "workspace")
    Y = _out(out, M, N, cfg, Xq.device)
    _same_device(Xq, s_a, packed, Y, workspace)
    _lib.check(_lib.lib().sdq_gemm_unpacked(C.byref(cfg.c()), _dev(Xq, "Xq"), _dev(s_a, "s_a"), M,
                                            _dev(packed, "packed"), N, K, _dev(workspace, "workspace"),
                                            workspace.numel() * workspace.element_size(), _dev(Y, "Y"),
                                            _stream(stream)), "sdq_gemm_unpacked")
    return Y


def gemm_static(Xq, s_a, packed, N: int, K: int, cfg: Config, out=None, path: int = PATH_AUTO,
                stream=None):
    """gemm() without a workspace: sdq_gemm_static, whose two-pass path uses the
    library's static 48 MiB scratch array (nothing is allocated by the call)."""
    import torch
    if Xq.dim() != 2:
        raise ValueError("Xq must be [M, K]")
    M = Xq.shape[0]
    _need(Xq, (M, K), torch.uint8, "Xq")
    _need(s_a, (M,), torch.float32, "s_a")
    _need_bytes(packed, pack_size(cfg, N, K), "packed")
    Y = _out(out, M, N, cfg, Xq.device)
    _same_device(Xq, s_a, packed, Y)
    _lib.check(_lib.lib().sdq_gemm_static(C.byref(cfg.c()), _dev(Xq, "Xq"), _dev(s_a, "s_a"), M,
                                          _dev(packed, "packed"), N, K, _dev(Y, "Y"),
                                          _stream(stream), path), "sdq_gemm_static")
    return Y


def linear(X, packed, N: int, K: int, cfg: Config, out=None, xq=None, scales=None, stream=None,
           workspace=None):
    """Quantize X per token and multiply: returns (Y, Xq, s_a).  One fused
    kernel on the decode path (sdq_linear); sdq_quantize_act then
    sdq_gemm_ws where the GEMM takes a workspace; otherwise sdq_linear's two
    kernels back to back."""
    import torch
    if X.dim() != 2 or X.shape[1] != K:
        raise ValueError(f"X must be [M, {K}], got {list(X.shape)}")
    M = X.shape[0]
    dt = _x_dtype(X)
    Xq = xq if xq is not None else torch.empty((M, K), dtype=torch.uint8, device=X.device)
    s_a = scales if scales is not None else torch.empty((M,), dtype=torch.float32, device=X.device)
    _need(Xq, (M, K), torch.uint8, "Xq")
    _need(s_a, (M,), torch.float32, "s_a")
    _need_bytes(packed, pack_size(cfg, N, K), "packed")
    Y = _out(out, M, N, cfg, X.device)
    _same_device(X, Xq, s_a, packed, Y, workspace)
    if gemm_workspace_size(cfg, M, N, K) > 0:
        quantize_act(X, cfg, out=Xq, scales=s_a, stream=stream)
        gemm(Xq, s_a, packed, N, K, cfg, out=Y, stream=stream, workspace=workspace)
        return Y, Xq, s_a
    _lib.check(_lib.lib().sdq_linear(C.byref(cfg.c()), _dev(X, "X"), dt, M, _dev(Xq, "Xq"),
                                     _dev(s_a, "s_a"), _dev(packed, "packed"), N, K, _dev(Y, "Y"),
                                     _stream(stream)), "sdq_linear")
    return Y, Xq, s_a


def gemm_path(cfg: Config, M: int, N: int, K: int, workspace: bool = False) -> int:
    """The path sdq_gemm takes (or sdq_gemm_ws and sdq_gemm_static, with workspace=True)."""
    p = C.c_int32()
    if workspace:
        _lib.check(_lib.lib().sdq_gemm_path_ws(C.byref(cfg.c()), M, N, K, C.byref(p)), "sdq_gemm_path_ws")
    else:
        _lib.check(_lib.lib().sdq_gemm_path(C.byref(cfg.c()), M, N, K, C.byref(p)), "sdq_gemm_path")
    return p.value
