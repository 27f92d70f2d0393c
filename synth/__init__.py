"""Seeded synthetic inputs for the SDQ decomposed GEMM.

This module only draws random numbers and describes workloads.  It holds none
of the method's arithmetic (no selection, no quantization, no product), so that
both the CPU oracle (``oracle/``) and the HIP path can be fed the same inputs
without sharing any code with each other.

Workloads stand in for the paper's evaluation models (OPT-6.7B and LLaMA-7B
linear layers, Section 6 "Methodology"); no weights or datasets are used.  The
shapes are those of the real layers, and the value distributions are chosen to
carry the outliers the method targets (Section 4): a few activation channels
scaled up, and a small fraction of heavy-tailed weights.

Every tensor is drawn from ``numpy.random.default_rng(SeedSequence([workload,
layer, tensor, seed]))``, in fp32 on the host.  Activations that are stated as
bf16 are rounded to bf16 here (round-to-nearest-even of the fp32 bits), because
bf16 is the dtype the input *is*; both sides then read the same bf16 values.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Tuple

import numpy as np

__all__ = [
    "Formats",
    "Layer",
    "Workload",
    "WORKLOADS",
    "INT_1x8_E4M3_3x8",
    "dual_formats",
    "rng_for",
    "bf16_round",
    "make_x",
    "make_w",
    "sweep_points",
]

# Tensor ids inside a SeedSequence.
_T_X, _T_X_CH, _T_W, _T_W_POS, _T_W_VAL = 0, 1, 2, 3, 4


@dataclasses.dataclass(frozen=True)
class Formats:
    """Plain description of an SDQ configuration (no behaviour).

    family "int": int8 per-token activations, outliers fp8-e4m3 or int8 with a
    per-row fp32 scale, inliers int4 with one fp16 scale per 16 dense K.
    family "mx": fp8-e4m3 per-token activations, outliers fp8-e4m3 and inliers
    fp4-e2m1, each branch with one e8m0 scale per 32 dense K.
    family "dual": int8 outliers (per-row fp32 scale) against int8 per-token
    activations, fp4-e2m1 inliers (e8m0 per 32) against MXFP4 activations.
    """

    family: str  # "int" | "mx" | "dual"
    n_o: int
    m_o: int
    fmt_o: str  # "e4m3" | "int8"
    n_i: int
    m_i: int
    fmt_i: str  # "int4" | "e2m1"
    fmt_a: str  # "int8" | "e4m3"

    @property
    def label(self) -> str:
        return (f"{self.family}-{self.n_o}:{self.m_o}{self.fmt_o}-"
                f"{self.n_i}:{self.m_i}{self.fmt_i}-A{self.fmt_a}")


def int_formats(n_o=1, m_o=8, fmt_o="e4m3", n_i=3, m_i=8) -> Formats:
    return Formats("int", n_o, m_o, fmt_o, n_i, m_i, "int4", "int8")


def mx_formats(n_o=1, m_o=8, n_i=2, m_i=8) -> Formats:
    return Formats("mx", n_o, m_o, "e4m3", n_i, m_i, "e2m1", "e4m3")


def dual_formats(n_o=1, n_i=6) -> Formats:
    return Formats("dual", n_o, 8, "int8", n_i, 8, "e2m1", "int8")


INT_1x8_E4M3_3x8 = int_formats()


@dataclasses.dataclass(frozen=True)
class Layer:
    name: str
    N: int  # output features (rows of W)
    K: int  # input features (reduction)
    input_of: str = ""  # an earlier layer whose input tensor this layer reads too


@dataclasses.dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    layers: Tuple[Layer, ...]
    M: Tuple[int, ...]
    formats: Tuple[Formats, ...]
    x_dtype: str  # "f32" | "bf16"
    # activation recipe
    x_outlier_frac: float  # fraction of channels scaled (ignored if x_fixed_ch)
    x_fixed_ch: int  # number of channels scaled (0: use x_outlier_frac)
    x_outlier_scale: float
    # weight recipe
    w_std: float
    w_outlier_frac: float
    w_outlier_kind: str  # "scale10" (entry * 10) | "t3" (std * 10 * Student-t df=3)


LLAMA7B_LAYERS = (
    Layer("q_proj", 4096, 4096), Layer("k_proj", 4096, 4096, "q_proj"),
    Layer("v_proj", 4096, 4096, "q_proj"), Layer("o_proj", 4096, 4096),
    Layer("gate_proj", 11008, 4096), Layer("up_proj", 11008, 4096, "gate_proj"),
    Layer("down_proj", 4096, 11008),
)

WORKLOADS: Dict[int, Workload] = {
    # Tiny case: small enough for pure-Python checks.
    1: Workload(1, "tiny 16x256x256", (Layer("tiny", 256, 256),), (16,),
                (INT_1x8_E4M3_3x8,), "f32", 0.0, 2, 20.0, 0.02, 0.005, "scale10"),
    # LLaMA-7B attention projection, single-token decode.
    2: Workload(2, "llama7b attn-proj decode M=1 4096x4096", (Layer("attn_proj", 4096, 4096),),
                (1,), (INT_1x8_E4M3_3x8,), "bf16", 0.001, 0, 30.0, 0.02, 0.002, "t3"),
    # LLaMA-7B MLP prefill, 2048 tokens, MX formats.
    3: Workload(3, "llama7b mlp prefill M=2048", (Layer("gate_proj", 11008, 4096),
                Layer("up_proj", 11008, 4096, "gate_proj"), Layer("down_proj", 4096, 11008)),
                (2048,), (mx_formats(1, 8, 2, 8),), "bf16", 0.001, 0, 30.0, 0.02, 0.002, "t3"),
    # OPT-6.7B FFN, batched decode of 64 tokens, int8 outliers.
    4: Workload(4, "opt6.7b ffn batched decode M=64", (Layer("fc1", 16384, 4096),
                Layer("fc2", 4096, 16384)), (64,), (int_formats(1, 8, "int8", 3, 8),),
                "bf16", 0.0, 6, 60.0, 0.015, 0.003, "scale10"),
    # Full LLaMA-7B block sweep.
    5: Workload(5, "llama7b block sweep", LLAMA7B_LAYERS, (1, 16, 256, 4096),
                tuple(int_formats(1, mo, "e4m3", ni, 8) for mo in (8, 16) for ni in (2, 3))
                + tuple(mx_formats(1, mo, ni, 8) for mo in (8, 16) for ni in (2, 3)),
                "bf16", 0.001, 0, 30.0, 0.02, 0.002, "t3"),
    # The paper's headline SDQ-W7:8-1:8int8-6:8fp4 on the LLaMA-7B block shapes.
    # the paper's three evaluated dual configurations: 7:8 = 1:8 int8 + 6:8
    # fp4, 6:8 = 2:8 int8 + 4:8 fp4, 8:8 = 1:8 int8 + 7:8 fp4
    6: Workload(6, "llama7b block, dual int8 outliers + fp4 inliers", LLAMA7B_LAYERS, (1, 16, 256, 4096),
                (dual_formats(1, 6), dual_formats(2, 4), dual_formats(1, 7)), "bf16", 0.001, 0, 30.0, 0.02,
                0.002, "t3"),
    # LLaMA-7B q, k and v projections stacked along N (one weight of 12288 rows,
    # the attention recipe), single-token decode: one launch for three layers.
    7: Workload(7, "llama7b qkv-concatenated decode M=1 12288x4096", (Layer("qkv_proj", 12288, 4096),),
                (1,), (INT_1x8_E4M3_3x8,), "bf16", 0.001, 0, 30.0, 0.02, 0.002, "t3"),
    # LLaMA-7B gate and up projections stacked along N (one weight of 22016
    # rows, the MLP recipe), single-token decode: they share their input.
    8: Workload(8, "llama7b gate/up-concatenated decode M=1 22016x4096",
                (Layer("gate_up_proj", 22016, 4096),), (1,), (INT_1x8_E4M3_3x8,), "bf16", 0.001, 0,
                30.0, 0.02, 0.002, "t3"),
}


def rng_for(wid: int, layer: int, tensor: int, seed: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([wid, layer, tensor, seed]))


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); return fp32."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (b >> 16) & 1
    r = ((b + 0x7FFF + lsb) >> 16) << 16
    return r.astype(np.uint32).view(np.float32)


def _x_channels(w: Workload, K: int, seed: int) -> np.ndarray:
    # Channel choice depends only on (workload, K, seed): the same outlier
    # channels for every token and for every layer with the same K.
    r = rng_for(w.wid, 1000 + K, _T_X_CH, seed)
    n = w.x_fixed_ch if w.x_fixed_ch else int(round(w.x_outlier_frac * K))
    return r.choice(K, size=n, replace=False)


def make_x(wid: int, M: int, K: int, seed: int = 0) -> np.ndarray:
    """Activations [M, K] as fp32 values (bf16-representable when stated bf16)."""
    w = WORKLOADS[wid]
    r = rng_for(wid, K, _T_X, seed)
    x = r.standard_normal((M, K), dtype=np.float32)
    ch = _x_channels(w, K, seed)
    x[:, ch] *= np.float32(w.x_outlier_scale)
    if w.x_dtype == "bf16":
        x = bf16_round(x)
    return x


def make_w(wid: int, layer: int, N: int, K: int, seed: int = 0) -> np.ndarray:
    """Weights [N, K] (row n = output channel), fp32."""
    w = WORKLOADS[wid]
    r = rng_for(wid, layer, _T_W, seed)
    W = r.standard_normal((N, K), dtype=np.float32)
    W *= np.float32(w.w_std)
    n_out = int(round(w.w_outlier_frac * N * K))
    rp = rng_for(wid, layer, _T_W_POS, seed)
    pos = rp.choice(N * K, size=n_out, replace=False)
    flat = W.reshape(-1)
    if w.w_outlier_kind == "scale10":
        flat[pos] *= np.float32(10.0)
    else:
        rv = rng_for(wid, layer, _T_W_VAL, seed)
        flat[pos] = (np.float32(w.w_std * 10.0) *
                     rv.standard_t(3, size=n_out).astype(np.float32))
    return W


def sweep_points(wid: int) -> List[Tuple[int, Layer, int, Formats]]:
    """All (layer index, layer, M, formats) points of a workload.

    For the block sweep the MX formats are only swept at M >= 256, where the
    matrix cores, not HBM, bound the product.
    """
    w = WORKLOADS[wid]
    out = []
    for li, L in enumerate(w.layers):
        for M in w.M:
            for f in w.formats:
                if wid == 5 and f.family == "mx" and M < 256:
                    continue
                out.append((li, L, M, f))
    return out
