"""Output-error report of the decomposition variants, on synthetic layers.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``): computed with the oracle
alone, in fp64, for the design notes.  No dataset is involved; the error of
the layer output against the unquantized product is the quality proxy.

For one weight matrix W and activations X it reports
    err = ||Y_q - X W^T||_F / ||X W^T||_F
where Y_q is the oracle's product of the quantized activations with the
decomposed and quantized weights (Section 5.1), for
  * the dense round-to-nearest baseline with the same quantizers and no
    sparsity (every position an inlier: int4 with fp16 scales per 16, or
    e2m1 with e8m0 per 32, activations int8 / e4m3 per token), and
  * SDQ with each decomposition metric (same, magnitude, product, error,
    output error) in each order (Large, Small) of Section 6.4's study, with
    the magnitude or the product significance metric for sparsification.

It also reports, for the int family, the inlier scale format (fp16, the
two-level e4m3 of VS-Quant, ufp8-e6m2; Section 6.4's quantization study) and
the Q-Vector size (16, 32, 64 dense positions per scale; Section 3.3) next to
the resulting logical bits per weight.

    python -m oracle.quality            # prints markdown tables
"""
from __future__ import annotations

import itertools
import sys

import numpy as np

from . import accounting as A
from . import sdq as S

DECOMPS = ("same", "magnitude", "product", "error", "output_error")
ORDERS = ("large", "small")


def rel_error(X: np.ndarray, W: np.ndarray, cfg: S.Config, act_norm=None) -> float:
    Y = S.reference(X, W, cfg, act_norm)[0]
    Y0 = np.asarray(X, np.float64) @ np.asarray(W, np.float64).T
    return float(np.linalg.norm(Y - Y0) / np.linalg.norm(Y0))


def dense_baseline(family: str) -> S.Config:
    """All positions inliers: the plain per-vector round-to-nearest format."""
    if family == "int":
        return S.Config("int", 0, 8, "e4m3", 8, 8, "int4", "int8")
    return S.Config("mx", 0, 8, "e4m3", 8, 8, "e2m1", "e4m3")


def sdq_config(family: str, n_i: int, metric: str, decomp: str, order: str,
               fmt_o: str = "e4m3") -> S.Config:
    if family == "int":
        return S.Config("int", 1, 8, fmt_o, n_i, 8, "int4", "int8", metric, decomp, order)
    return S.Config("mx", 1, 8, "e4m3", n_i, 8, "e2m1", "e4m3", metric, decomp, order)


def report(W: np.ndarray, X: np.ndarray, X_cal: np.ndarray, family: str, n_is=(3, 6)):
    """Rows (label, error) for one layer."""
    an = S.activation_norm(X_cal)
    rows = [(f"dense RTN W4A8 ({'int4/16 fp16' if family == 'int' else 'e2m1/32 e8m0'})",
             rel_error(X, W, dense_baseline(family)))]
    for n_i in n_is:
        for metric, decomp, order in itertools.product(("magnitude", "product"), DECOMPS, ORDERS):
            if decomp == "same" and order == "large":
                label = f"SDQ 1:8+{n_i}:8, {metric} significance, default decomposition"
            else:
                label = f"SDQ 1:8+{n_i}:8, {metric} significance, {decomp} {order}"
            rows.append((label, rel_error(X, W, sdq_config(family, n_i, metric, decomp, order), an)))
    return rows


SCALE_BITS = {"f16": 16, "e4m3": 8, "ue6m2": 8}


def bits_per_weight(cfg: S.Config, K: int) -> float:
    """Logical bits per dense weight (values, indices, scales), int family."""
    b = A.sdq_bits_per_weight(cfg.n_o, cfg.m_o, 8, cfg.n_i, cfg.m_i, 4, 32, 0,
                              SCALE_BITS[cfg.sfmt], cfg.qv_i, K)
    if cfg.sfmt == "e4m3":
        b += A.Fraction(32, K)  # the power-of-two row scale
    return float(b)


def scale_report(W: np.ndarray, X: np.ndarray, X_cal: np.ndarray, n_is=(3, 6)):
    """Rows (n_i, scale format, qv, bits per weight, error), int family with
    product significance and the default decomposition."""
    an = S.activation_norm(X_cal)
    K = W.shape[1]
    rows = []
    for n_i, sfmt, qv in itertools.product(n_is, ("f16", "e4m3", "ue6m2"), (16, 32, 64)):
        cfg = S.Config("int", 1, 8, "e4m3", n_i, 8, "int4", "int8", "product",
                       sfmt_i="" if sfmt == "f16" else sfmt, qv=qv)
        rows.append((n_i, sfmt, qv, bits_per_weight(cfg, K), rel_error(X, W, cfg, an)))
    return rows


def main(argv=None) -> None:
    import synth
    N = int(argv[0]) if argv else 512
    K = 4096
    W = synth.make_w(2, 0, N, K)           # LLaMA-7B-like rows: N(0, 0.02^2) with heavy-tailed outliers
    X = synth.make_x(2, 64, K)             # 64 tokens with scaled outlier channels
    X_cal = synth.make_x(2, 256, K)[64:]   # other tokens of the same generator: calibration
    for family in ("int", "mx"):
        print(f"\n{family} family, W {N}x{K}, X 64x{K}\n")
        print("| configuration | relative output error |")
        print("|---|---|")
        for label, e in report(W, X, X_cal, family):
            print(f"| {label} | {e:.4f} |")
    print(f"\nint family, inlier scale format and Q-Vector size, W {N}x{K}, X 64x{K}\n")
    print("| SDQ | scale format | Q-Vector | bits / weight | relative output error |")
    print("|---|---|---|---|---|")
    for n_i, sfmt, qv, bits, e in scale_report(W, X, X_cal):
        print(f"| 1:8 int8/e4m3 + {n_i}:8 int4 | {sfmt} | {qv} | {bits:.3f} | {e:.4f} |")


if __name__ == "__main__":
    main(sys.argv[1:])
