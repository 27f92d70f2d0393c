"""The SDQ decomposition, quantization and decomposed product, plainly.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Paper passages followed (Jeong et al., SDQ):

* N:M structured sparsity: at most N non-zeros in every M consecutive values
  (Section 3.1).  Groups run along the reduction dimension K inside one row
  of ``W[N, K]`` (PyTorch ``Linear`` layout).
* Stage 1 sparsification keeps the N most significant values of every M;
  significance is the magnitude or the weight-activation product of Wanda
  (Section 5, "Stage 1").
* Stage 2 decomposition extracts n_o:m local outliers per S-vector with a
  metric taken in descending order ("Large"); the kept values that remain are
  the inliers, themselves n_i:m structured (Section 4 and Section 5,
  "Stage 2").  Selecting the top n_o first and then the next n_i equals
  sparsifying to (n_o+n_i):m first and then extracting n_o:m outliers.
* The decomposition metric may differ from the significance metric and be
  taken in either order: magnitude, weight-activation product, or the error
  the inlier quantizer makes on the weight (alone or times the activation
  norm), "Large" or "Small" (Section 5, "Stage 2", and Section 6.4's
  decomposition study).  These run the two stages in the paper's order.
* Stage 3 quantizes each branch with per-vector (VS-Quant) scale factors,
  outliers at a higher precision than inliers; activations are quantized too
  (Section 3.3 and Section 5, "Stage 3").
* The dual family follows Section 5.1's worked configuration: int8
  outliers with int8 activations A_o and fp4 inliers with fp4 activations
  A_i, O = SpMM(A_o, W_o) + SpMM(A_i, W_i).
* Inference is O = SpMM(A, W_o) + SpMM(A, W_i) (Section 5.1); since both
  branches skip only zeros, it equals the dense product of the activations
  with the dequantized W_o + W_i, which is what ``gemm_fp64`` computes.

Where the paper leaves a choice open the oracle takes these readings:
groups along K; ties in the metric go to the lower k; int4 inliers are
symmetric in [-7, 7] with s = fp16(amax/7) and are quantized with the
stored fp16 scale; int-family outliers have one fp32 scale per row
(amax/qmax); MX-family scales are OCP MX v1.0 shared exponents
E = floor(log2 amax) - emax(element) with saturating element conversion;
activations use one scale per token for both branches.

All scale and quantization arithmetic is IEEE fp32 in the order written
here (numpy float32 operations round once per operation); the product is
fp64.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional, Tuple

import numpy as np

from . import formats as F


@dataclasses.dataclass(frozen=True)
class Config:
    family: str        # "int" | "mx" | "dual"
    n_o: int
    m_o: int
    fmt_o: str         # "e4m3" | "int8"
    n_i: int
    m_i: int
    fmt_i: str         # "int4" | "e2m1"
    fmt_a: str         # "int8" | "e4m3"
    metric: str = "magnitude"  # significance (Stage 1): "magnitude" | "product"
    decomp: str = "same"       # outlier metric (Stage 2): "same" | "magnitude" | "product"
    #                            | "error" | "output_error"
    order: str = "large"       # outliers have the largest ("large") or smallest ("small") metric
    sfmt_i: str = ""           # inlier scale format (int family): "" = fp16 | "e4m3" (two-level,
    #                            with a power-of-two scale per row) | "ue6m2"; mx family: e8m0
    qv: int = 0                # dense K positions per inlier scale; 0 = the family's (16 / 32)

    @property
    def staged(self) -> bool:
        """Whether Stage 2 uses its own metric or order (not the default)."""
        return self.decomp != "same" or self.order != "large"

    @property
    def qv_i(self) -> int:
        """Dense-K positions that share one inlier scale."""
        return self.qv or (16 if self.family == "int" else 32)

    @property
    def sfmt(self) -> str:
        """The inlier scale format: "f16", "e4m3", "ue6m2" or "e8m0"."""
        return self.sfmt_i or ("f16" if self.family == "int" else "e8m0")

    @property
    def qv_o(self) -> int:
        """Dense-K positions that share one outlier scale (0 = whole row)."""
        return 32 if self.family == "mx" else 0

    @property
    def row_outliers(self) -> bool:
        """Outliers with one fp32 scale per row (int and dual families)."""
        return self.family in ("int", "dual")

    def check(self, K: int) -> None:
        assert self.family in ("int", "mx", "dual")
        assert self.m_i in (4, 8, 16) and 1 <= self.n_i <= self.m_i
        assert self.n_o == 0 or (self.m_o in (4, 8, 16) and 1 <= self.n_o <= self.m_o)
        if self.family == "int":
            assert self.fmt_o in ("e4m3", "int8") and self.fmt_i == "int4"
            assert self.fmt_a == "int8"
        elif self.family == "dual":
            assert self.fmt_o == "int8" and self.fmt_i == "e2m1" and self.fmt_a == "int8+e2m1"
        else:
            assert self.fmt_o == "e4m3" and self.fmt_i == "e2m1" and self.fmt_a == "e4m3"
        # every m_i-group must still hold n_i candidates after outlier extraction
        if self.n_o == 0:
            most = 0
        elif self.m_o >= self.m_i:
            most = min(self.n_o, self.m_i)
        else:
            most = self.n_o * (self.m_i // self.m_o)
        assert self.n_i + most <= self.m_i, "infeasible n_i"
        m_o = self.m_o if self.n_o else self.m_i
        for d in (self.m_i, self.qv_i, m_o, 1 if self.family == "int" else 32):
            assert K % d == 0, f"K={K} not divisible by {d}"
        assert self.decomp in ("same", "magnitude", "product", "error", "output_error")
        if self.family == "int":
            assert self.sfmt in ("f16", "e4m3", "ue6m2") and self.qv_i in (16, 32, 64)
        else:
            assert self.sfmt == "e8m0" and self.qv_i == 32
        assert self.order in ("large", "small")
        if self.staged:
            # outliers are chosen among the positions kept by sparsification
            assert self.n_o > 0 and self.m_o % self.m_i == 0
            assert self.n_o * (self.m_o // self.m_i) <= self.m_o and self.n_o + self.n_i <= self.m_i


def config_from(fmt, metric: str = "magnitude", decomp: str = "same", order: str = "large",
                sfmt_i: str = "", qv: int = 0) -> Config:
    """Build an oracle Config from a plain format description (duck-typed)."""
    fmt_a = "int8+e2m1" if fmt.family == "dual" else fmt.fmt_a
    return Config(fmt.family, fmt.n_o, fmt.m_o, fmt.fmt_o, fmt.n_i, fmt.m_i,
                  fmt.fmt_i, fmt_a, metric, decomp, order, sfmt_i or getattr(fmt, "sfmt_i", ""),
                  qv or getattr(fmt, "qv_i", 0))


# ---------------------------------------------------------------------------
# Stage 1/2: significance, outliers, inliers
# ---------------------------------------------------------------------------
def significance(W: np.ndarray, act_norm: Optional[np.ndarray] = None) -> np.ndarray:
    """S = |W| (magnitude), or |W| * c with c[k] the activation norm (Wanda)."""
    S = np.abs(np.asarray(W, dtype=np.float32))
    if act_norm is not None:
        S = S * np.asarray(act_norm, dtype=np.float32)[None, :]
    return S.astype(np.float32)


def activation_norm(X_cal: np.ndarray) -> np.ndarray:
    """Wanda's per-input-channel activation norm ||X[:, k]||_2 (fp64, cast fp32)."""
    X = np.asarray(X_cal, dtype=np.float64)
    return np.sqrt((X * X).sum(axis=0)).astype(np.float32)


def top_n_per_group(S: np.ndarray, allowed: np.ndarray, m: int, n: int):
    """In every m-group along K pick the first n allowed positions by (-S, k).

    Returns (mask [N, K] bool, positions [N, K/m, n] ascending within group).
    """
    N, K = S.shape
    G = K // m
    key = np.where(allowed.reshape(N, G, m), -S.reshape(N, G, m).astype(np.float64), np.inf)
    order = np.argsort(key, axis=-1, kind="stable")  # stable: equal keys keep k order
    chosen = order[..., :n]
    ok = np.take_along_axis(allowed.reshape(N, G, m), chosen, axis=-1)
    assert ok.all(), "fewer candidates than slots in a group"
    mask = np.zeros((N, G, m), dtype=bool)
    np.put_along_axis(mask, chosen, True, axis=-1)
    return mask.reshape(N, K), np.sort(chosen, axis=-1).astype(np.int64)


def top_n_by_key(key: np.ndarray, allowed: np.ndarray, m: int, n: int):
    """In every m-group pick the first n allowed positions by (key, k), key
    ascending.  Returns (mask [N, K] bool, positions [N, K/m, n] ascending)."""
    N, K = key.shape
    G = K // m
    k = np.where(allowed.reshape(N, G, m), key.reshape(N, G, m).astype(np.float64), np.inf)
    order = np.argsort(k, axis=-1, kind="stable")
    chosen = order[..., :n]
    assert np.take_along_axis(allowed.reshape(N, G, m), chosen, axis=-1).all(), \
        "fewer candidates than slots in a group"
    mask = np.zeros((N, G, m), dtype=bool)
    np.put_along_axis(mask, chosen, True, axis=-1)
    return mask.reshape(N, K), np.sort(chosen, axis=-1).astype(np.int64)


def inlier_error(W: np.ndarray, keep: np.ndarray, cfg: Config) -> np.ndarray:
    """|W - deq Q_i(W)| on the kept positions (0 elsewhere), fp32: the error the
    inlier quantizer (scales over the kept positions of each block) makes on
    every kept weight -- the quantization error of Section 6.4's error-based
    decomposition metric."""
    W = np.asarray(W, dtype=np.float32)
    q, scale, row = quantize_inliers(W, keep, cfg)
    deq = dequant_inliers(dict(cfg=cfg, code_i_dense=q, scale_i=scale, scale_i_row=row)).astype(np.float32)
    return np.where(keep, np.abs(W - deq), np.float32(0)).astype(np.float32)


def decomposition_metric(W: np.ndarray, keep: np.ndarray, cfg: Config,
                         act_norm: Optional[np.ndarray]) -> np.ndarray:
    """Stage 2's metric D (fp32): the significance itself, |W|, |W| * c, the
    inlier quantization error, or that error times c (c = act_norm)."""
    W = np.asarray(W, dtype=np.float32)
    if cfg.decomp == "same":
        return significance(W, act_norm if cfg.metric == "product" else None)
    if cfg.decomp == "magnitude":
        return np.abs(W)
    if cfg.decomp in ("product", "output_error"):
        assert act_norm is not None, f"the {cfg.decomp} metric needs act_norm"
    c = None if act_norm is None else np.asarray(act_norm, dtype=np.float32)[None, :]
    if cfg.decomp == "product":
        return (np.abs(W) * c).astype(np.float32)
    e = inlier_error(W, keep, cfg)
    return e if cfg.decomp == "error" else (e * c).astype(np.float32)


def decompose_staged(W: np.ndarray, cfg: Config, act_norm: Optional[np.ndarray] = None):
    """Stages 1 and 2 in the paper's order (Section 5): sparsify, then extract
    the outliers from what was kept.  Returns (mask_o, pos_o, mask_i, pos_i)."""
    N, K = W.shape
    assert cfg.n_o > 0 and cfg.m_o % cfg.m_i == 0
    assert cfg.metric != "product" or act_norm is not None, "the product metric needs act_norm"
    S = significance(W, act_norm if cfg.metric == "product" else None)
    # Stage 1: sparsify every m_i-group to its n_o + n_i most significant positions
    keep, _ = top_n_per_group(S, np.ones((N, K), dtype=bool), cfg.m_i, cfg.n_o + cfg.n_i)
    # Stage 2: n_o outliers per m_o-group among the kept, by D largest or smallest first
    D = decomposition_metric(W, keep, cfg, act_norm).astype(np.float64)
    mask_o, pos_o = top_n_by_key(-D if cfg.order == "large" else D, keep, cfg.m_o, cfg.n_o)
    # the kept positions that are not outliers are the inliers; an m_i-group
    # left with more than n_i of them keeps its n_i most significant
    mask_i, pos_i = top_n_per_group(S, keep & ~mask_o, cfg.m_i, cfg.n_i)
    return mask_o, pos_o, mask_i, pos_i


def decompose(W: np.ndarray, cfg: Config, act_norm: Optional[np.ndarray] = None):
    """Outlier and inlier supports.  Returns (mask_o, pos_o, mask_i, pos_i).

    Default decomposition (the significance metric, largest first): the n_o
    most significant positions of every m_o-group are the outliers and the
    n_i most significant remaining positions of every m_i-group the inliers.
    Any other decomposition metric or order runs ``decompose_staged``."""
    N, K = W.shape
    cfg.check(K)
    if cfg.staged:
        return decompose_staged(W, cfg, act_norm)
    assert cfg.metric != "product" or act_norm is not None, "the product metric needs act_norm"
    S = significance(W, act_norm if cfg.metric == "product" else None)
    everything = np.ones((N, K), dtype=bool)
    if cfg.n_o:
        mask_o, pos_o = top_n_per_group(S, everything, cfg.m_o, cfg.n_o)
    else:
        mask_o, pos_o = np.zeros((N, K), bool), np.zeros((N, K // cfg.m_i, 0), np.int64)
    mask_i, pos_i = top_n_per_group(S, ~mask_o, cfg.m_i, cfg.n_i)
    return mask_o, pos_o, mask_i, pos_i


# ---------------------------------------------------------------------------
# Stage 3: per-vector quantization
# ---------------------------------------------------------------------------
def _block_amax(absW: np.ndarray, mask: np.ndarray, qv: int) -> np.ndarray:
    N, K = absW.shape
    return np.where(mask, absW, np.float32(0)).reshape(N, K // qv, qv).max(axis=-1)


def quantize_outliers(W: np.ndarray, mask_o: np.ndarray, cfg: Config):
    """Outlier codes (dense [N, K], zero off-support) and scales.

    int, dual: one fp32 scale per row, s_o = amax/qmax, q = enc(W / s_o).
    mx family: one e8m0 exponent per 32 K, E = floor(log2 amax) - 8.
    """
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    absW = np.abs(W)
    if cfg.row_outliers:
        qmax = np.float32(127.0 if cfg.fmt_o == "int8" else F.E4M3_MAX)
        a = np.where(mask_o, absW, np.float32(0)).max(axis=1) if K else np.zeros(N, np.float32)
        s = (a / qmax).astype(np.float32)                          # fp32 divide
        safe = np.where(s == 0, np.float32(1), s)
        v = (W / safe[:, None]).astype(np.float32)                  # fp32 divide
        if cfg.fmt_o == "int8":
            code = F.int_rne_clamp(v, 127).astype(np.int8).view(np.uint8)
        else:
            code = F.e4m3_encode(v)
        code = np.where(mask_o & (s != 0)[:, None], code, 0).astype(np.uint8)
        return code, s
    # mx family
    a = _block_amax(absW, mask_o, 32)
    E = np.clip(F.floor_log2(np.where(a > 0, a, 1.0)) - 8, -127, 127)
    E = np.where(a > 0, E, -127)
    scale = np.ldexp(1.0, np.repeat(E, 32, axis=1))                  # exact power of two
    code = F.e4m3_encode(W.astype(np.float64) / scale)
    code = np.where(mask_o & np.repeat(a > 0, 32, axis=1), code, 0).astype(np.uint8)
    return code, (E + 127).astype(np.uint8)


def row_scale_exponent(vmax: np.ndarray) -> np.ndarray:
    """Per row, the smallest E with vmax <= 448 * 2^E (vmax = the row's largest
    vector scale), so that every vector scale divided by 2^E fits e4m3; 0 for
    an all-zero row.  Exact comparisons, no rounding."""
    vmax = np.asarray(vmax, dtype=np.float64)
    fl = F.floor_log2(np.where(vmax > 0, vmax, 1.0))
    E = fl - 8                                         # 448 * 2^(fl-8) = 1.75 * 2^fl
    E = np.where(vmax > np.ldexp(F.E4M3_MAX, E), E + 1, E)
    return np.where(vmax > 0, E, 0).astype(np.int64)


def quantize_inliers(W: np.ndarray, mask_i: np.ndarray, cfg: Config):
    """Inlier codes (dense [N, K], zero off-support) and scales.

    int family: int4 in [-7, 7] with a scale per qv dense K (16 by default),
                q = clamp(rne(W / s), -7, 7) using the stored scale s:
                  fp16:  s = fp16(amax/7);
                  e4m3:  VS-Quant's two levels, s = e4m3(v / 2^E) * 2^E with
                         v = amax/7 (fp32) and 2^E the smallest power of two
                         that puts the row's largest v within e4m3's 448;
                  ue6m2: s = ue6m2(amax/7).
    mx family:  fp4 e2m1 with E = floor(log2 amax) - 2 per 32 dense K.
    Returns (codes, stored scales, row scales): codes as int8 values (int
    family) or e2m1 nibbles (mx family); the stored scale codes per block; the
    power-of-two second-level scale per row (fp32) for e4m3 scales, else None.
    """
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    absW = np.abs(W)
    qv = cfg.qv_i
    a = _block_amax(absW, mask_i, qv)
    if cfg.family == "int":
        v_blk = (a / np.float32(7.0)).astype(np.float32)               # fp32 divide
        row = None
        if cfg.sfmt == "f16":
            stored = F.f16_round(v_blk)                                  # fp16 RNE
            if not np.isfinite(stored).all():
                raise ValueError("inlier scale overflows fp16")
            s32 = stored.astype(np.float32)
        elif cfg.sfmt == "e4m3":
            E = row_scale_exponent(v_blk.max(axis=1) if v_blk.size else np.zeros(N, np.float32))
            stored = F.e4m3_encode(np.ldexp(v_blk.astype(np.float64), -E[:, None]))   # exact scaling
            s32 = np.ldexp(F.e4m3_decode(stored), E[:, None]).astype(np.float32)      # exact
            row = np.where(v_blk.max(axis=1) > 0, np.ldexp(1.0, E), 0.0).astype(np.float32) \
                if v_blk.size else np.zeros(N, np.float32)
        else:  # ue6m2
            stored = F.ue6m2_encode(v_blk)
            s32 = F.ue6m2_decode(stored).astype(np.float32)                            # exact
        safe = np.where(s32 == 0, np.float32(1), s32)
        v = (W / np.repeat(safe, qv, axis=1)).astype(np.float32)      # fp32 divide
        q = F.int_rne_clamp(v, 7)
        q = np.where(mask_i & np.repeat(s32 != 0, qv, axis=1), q, 0).astype(np.int8)
        return q, stored, (row if cfg.sfmt == "e4m3" else None)
    E = np.clip(F.floor_log2(np.where(a > 0, a, 1.0)) - 2, -127, 127)
    E = np.where(a > 0, E, -127)
    scale = np.ldexp(1.0, np.repeat(E, qv, axis=1))
    code = F.e2m1_encode(W.astype(np.float64) / scale)
    code = np.where(mask_i & np.repeat(a > 0, qv, axis=1), code, 0).astype(np.uint8)
    return code, (E + 127).astype(np.uint8), None


def _gather(dense: np.ndarray, pos: np.ndarray, m: int) -> np.ndarray:
    N, K = dense.shape
    return np.take_along_axis(dense.reshape(N, K // m, m), pos, axis=-1)


def pack_logical(W: np.ndarray, cfg: Config, act_norm: Optional[np.ndarray] = None) -> Dict:
    """The logical packed form: per branch, row and group, n (position, code)
    slots with ascending positions, plus the scale arrays.  A slot keeps its
    position even when its code is zero."""
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    mask_o, pos_o, mask_i, pos_i = decompose(W, cfg, act_norm)
    code_o_dense, scale_o = quantize_outliers(W, mask_o, cfg) if cfg.n_o else (
        np.zeros((N, K), np.uint8), np.zeros(N, np.float32))
    code_i_dense, scale_i, scale_i_row = quantize_inliers(W, mask_i, cfg)
    return dict(
        N=N, K=K, cfg=cfg,
        pos_o=pos_o, code_o=_gather(code_o_dense, pos_o, cfg.m_o) if cfg.n_o else pos_o.astype(np.uint8),
        scale_o=scale_o,
        pos_i=pos_i, code_i=_gather(code_i_dense, pos_i, cfg.m_i),
        scale_i=scale_i, scale_i_row=scale_i_row,
        mask_o=mask_o, mask_i=mask_i,
        code_o_dense=code_o_dense, code_i_dense=code_i_dense,
    )


# ---------------------------------------------------------------------------
# dequantization
# ---------------------------------------------------------------------------
def dequant_outliers(L: Dict) -> np.ndarray:
    cfg: Config = L["cfg"]
    N, K = L["N"], L["K"]
    c = L["code_o_dense"]
    if not cfg.n_o:
        return np.zeros((N, K))
    if cfg.row_outliers:
        v = c.view(np.int8).astype(np.float64) if cfg.fmt_o == "int8" else F.e4m3_decode(c)
        return v * L["scale_o"].astype(np.float64)[:, None]
    return F.e4m3_decode(c) * np.repeat(F.e8m0_value(L["scale_o"]), 32, axis=1)


def inlier_scale_values(L: Dict) -> np.ndarray:
    """The effective inlier scale of every block, [N, K/qv], fp64 (exact)."""
    cfg: Config = L["cfg"]
    sc = L["scale_i"]
    if cfg.sfmt == "f16":
        return sc.astype(np.float64)
    if cfg.sfmt == "e4m3":
        return F.e4m3_decode(sc) * L["scale_i_row"].astype(np.float64)[:, None]
    if cfg.sfmt == "ue6m2":
        return F.ue6m2_decode(sc)
    return F.e8m0_value(sc)


def dequant_inliers(L: Dict) -> np.ndarray:
    cfg: Config = L["cfg"]
    c = L["code_i_dense"]
    v = c.astype(np.float64) if cfg.family == "int" else F.e2m1_decode(c)
    return v * np.repeat(inlier_scale_values(L), cfg.qv_i, axis=1)


# ---------------------------------------------------------------------------
# activations (one scale per token)
# ---------------------------------------------------------------------------
def quantize_act(X: np.ndarray, cfg: Config):
    """Per token m: a = max|X[m,:]|, s_a = a/qmax, inv = qmax/a (fp32 divides),
    q = enc(X * inv) (fp32 multiply).  int8: clamp(rne, +-127); e4m3:
    nearest-even saturating to +-448.  A zero row gets s_a = 0 and zero codes."""
    X = np.asarray(X, dtype=np.float32)
    qmax = np.float32(127.0 if cfg.fmt_a == "int8" else F.E4M3_MAX)
    a = np.abs(X).max(axis=1) if X.shape[1] else np.zeros(X.shape[0], np.float32)
    s_a = (a / qmax).astype(np.float32)
    safe = np.where(a == 0, np.float32(1), a)
    inv = (qmax / safe).astype(np.float32)
    v = (X * inv[:, None]).astype(np.float32)
    if cfg.fmt_a == "int8":
        q = F.int_rne_clamp(v, 127).astype(np.int8).view(np.uint8)
    else:
        q = F.e4m3_encode(v)
    q = np.where((a == 0)[:, None], 0, q).astype(np.uint8)
    return q, s_a


def dequant_act(Xq: np.ndarray, s_a: np.ndarray, cfg: Config) -> np.ndarray:
    if cfg.fmt_a == "int8":
        v = Xq.view(np.int8).astype(np.float64)
    else:
        v = F.e4m3_decode(Xq)
    return v * s_a.astype(np.float64)[:, None]


# ---------------------------------------------------------------------------
# the decomposed product (Section 5.1), fp64
# ---------------------------------------------------------------------------
def gemm_fp64(Xq: np.ndarray, s_a: np.ndarray, L: Dict):
    """Y = (s_a * Xq) @ (deq W_o + deq W_i)^T in fp64; also Y_o and Y_i."""
    A = dequant_act(Xq, s_a, L["cfg"])
    Wo = dequant_outliers(L)
    Wi = dequant_inliers(L)
    Y_o = A @ Wo.T
    Y_i = A @ Wi.T
    return A @ (Wo + Wi).T, Y_o, Y_i


def int_partials(Xq: np.ndarray, L: Dict):
    """Exact integer partials of the int family.

    P_i[m, n, kb] = sum_{k in block kb} Xq[m,k] * q_i[n,k] over the qv-K scale blocks;
    P_o[m, n] = sum_k Xq[m,k] * q_o[n,k] when outliers are int8 (else None).
    """
    cfg: Config = L["cfg"]
    assert cfg.family in ("int", "dual")
    X = Xq.view(np.int8).astype(np.int64)
    Qi = L["code_i_dense"].astype(np.int64)
    M, K = X.shape
    N = Qi.shape[0]
    qv = cfg.qv_i
    P_i = None if cfg.family == "dual" else \
        np.einsum("mbk,nbk->mnb", X.reshape(M, K // qv, qv), Qi.reshape(N, K // qv, qv))
    P_o = None
    if cfg.n_o and cfg.fmt_o == "int8":
        P_o = X @ L["code_o_dense"].view(np.int8).astype(np.int64).T
    return P_i, P_o


def sparse_gemm_loops(Xq: np.ndarray, s_a: np.ndarray, L: Dict) -> np.ndarray:
    """The two SpMMs written as loops over the stored (position, code) slots.

    Pure Python; for tiny shapes only.  Independent of the dense form above:
    it never materialises W_o or W_i.
    """
    cfg: Config = L["cfg"]
    A = dequant_act(Xq, s_a, cfg)
    M = A.shape[0]
    N, K = L["N"], L["K"]
    sv = inlier_scale_values(L)
    Y = np.zeros((M, N))
    for n in range(N):
        for m in range(M):
            acc = 0.0
            if cfg.n_o:
                for g in range(K // cfg.m_o):
                    for j in range(cfg.n_o):
                        k = g * cfg.m_o + int(L["pos_o"][n, g, j])
                        c = int(L["code_o"][n, g, j])
                        if cfg.row_outliers:
                            w = (c - 256 if c > 127 else c) if cfg.fmt_o == "int8" else F.e4m3_value(c)
                            w *= float(L["scale_o"][n])
                        else:
                            w = F.e4m3_value(c) * 2.0 ** (int(L["scale_o"][n, k // 32]) - 127)
                        acc += A[m, k] * w
            for g in range(K // cfg.m_i):
                for j in range(cfg.n_i):
                    k = g * cfg.m_i + int(L["pos_i"][n, g, j])
                    c = int(L["code_i"][n, g, j])
                    if cfg.family == "int":
                        w = (c - 256 if c > 127 else c) * float(sv[n, k // cfg.qv_i])
                    else:
                        w = F.e2m1_value(c) * float(sv[n, k // 32])
                    acc += A[m, k] * w
            Y[m, n] = acc
    return Y


# ---------------------------------------------------------------------------
# the dual family (Section 5.1's worked configuration): int8 A_o, fp4 A_i
# ---------------------------------------------------------------------------
def quantize_act_dual(X: np.ndarray):
    """A_o: int8 per token, as ``quantize_act`` for an int8 configuration.
    A_i: MXFP4 per token, one e8m0 exponent per 32 K, E = floor(log2 amax) - 2
    (clamped to [-127, 127]; an all-zero block gets E = -127 and zero codes),
    codes e2m1(X / 2^E) nearest-even, saturating.
    Returns (Ao int8 codes as uint8 [M, K], s_ao fp32 [M],
             Ai e2m1 codes [M, K] (one nibble per byte), Ea e8m0 codes [M, K/32])."""
    X = np.asarray(X, dtype=np.float32)
    M, K = X.shape
    Ao, s_ao = quantize_act(X, Config("int", 0, 8, "e4m3", 1, 8, "int4", "int8"))
    a = np.abs(X).reshape(M, K // 32, 32).max(axis=-1)
    E = np.clip(F.floor_log2(np.where(a > 0, a, 1.0)) - 2, -127, 127)
    E = np.where(a > 0, E, -127)
    Ai = F.e2m1_encode(X.astype(np.float64) / np.ldexp(1.0, np.repeat(E, 32, axis=1)))
    Ai = np.where(np.repeat(a > 0, 32, axis=1), Ai, 0).astype(np.uint8)
    return Ao, s_ao, Ai, (E + 127).astype(np.uint8)


def dequant_act_dual(Ao, s_ao, Ai, Ea):
    """(A_o, A_i) dequantized, fp64."""
    A_o = Ao.view(np.int8).astype(np.float64) * s_ao.astype(np.float64)[:, None]
    A_i = F.e2m1_decode(Ai) * np.repeat(F.e8m0_value(Ea), 32, axis=1)
    return A_o, A_i


def gemm_fp64_dual(Ao, s_ao, Ai, Ea, L: Dict):
    """O = A_o W_o^T + A_i W_i^T in fp64; also O_o and O_i."""
    A_o, A_i = dequant_act_dual(Ao, s_ao, Ai, Ea)
    Y_o = A_o @ dequant_outliers(L).T
    Y_i = A_i @ dequant_inliers(L).T
    return Y_o + Y_i, Y_o, Y_i


def sparse_gemm_loops_dual(Ao, s_ao, Ai, Ea, L: Dict) -> np.ndarray:
    """The two SpMMs of the dual family as loops over the stored slots (tiny
    shapes only): outliers against A_o, inliers against A_i."""
    cfg: Config = L["cfg"]
    A_o, A_i = dequant_act_dual(Ao, s_ao, Ai, Ea)
    M = A_o.shape[0]
    N, K = L["N"], L["K"]
    Y = np.zeros((M, N))
    for n in range(N):
        for m in range(M):
            acc = 0.0
            for g in range(K // cfg.m_o if cfg.n_o else 0):
                for j in range(cfg.n_o):
                    k = g * cfg.m_o + int(L["pos_o"][n, g, j])
                    c = int(L["code_o"][n, g, j])
                    acc += A_o[m, k] * (c - 256 if c > 127 else c) * float(L["scale_o"][n])
            for g in range(K // cfg.m_i):
                for j in range(cfg.n_i):
                    k = g * cfg.m_i + int(L["pos_i"][n, g, j])
                    w = F.e2m1_value(int(L["code_i"][n, g, j])) * 2.0 ** (int(L["scale_i"][n, k // 32]) - 127)
                    acc += A_i[m, k] * w
            Y[m, n] = acc
    return Y


def reference(X: np.ndarray, W: np.ndarray, cfg: Config, act_norm=None):
    """Convenience: quantize activations, pack, and multiply.  For the dual
    family the activations come back as (Ao, Ai) and their scales as
    (s_ao, Ea)."""
    L = pack_logical(W, cfg, act_norm)
    if cfg.family == "dual":
        Ao, s_ao, Ai, Ea = quantize_act_dual(X)
        Y, _, _ = gemm_fp64_dual(Ao, s_ao, Ai, Ea, L)
        return Y, (Ao, Ai), (s_ao, Ea), L
    Xq, s_a = quantize_act(X, cfg)
    Y, _, _ = gemm_fp64(Xq, s_a, L)
    return Y, Xq, s_a, L
