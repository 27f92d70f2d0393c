"""Shared helpers of the GPU parity tests (no method arithmetic here)."""
import sys

import numpy as np
import pytest

REL_TOL = 1e-3  # max relative error (1%-RMS floor) and normwise relative error vs the fp64 oracle
# MX family: gfx950's scaled fp8/fp4 matrix instruction sums its 64 products in a
# fixed-point window about 2^-17.5 below the largest product of the instruction
# (measured), so outputs that cancel lose relative accuracy.  The check there is
# normwise <= 1e-3 plus a componentwise bound against the sum of |terms|: at
# most 32 nonzero products per instruction (1 outlier + 3 inliers per 8), each
# off by less than one window unit, give at most 32 * 2^-17.5 = 2^-12.5 of the
# sum of |terms|; 2^-12 leaves room for the measured window.
MX_TERM_TOL = 2.0 ** -12


def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def say(*a):
    """Name the case before a GPU step (flushed, so a fault still shows it)."""
    print("[case]", *a, file=sys.stderr, flush=True)


def rel_errors(Y: np.ndarray, Yref: np.ndarray):
    Y = np.asarray(Y, np.float64)
    Yref = np.asarray(Yref, np.float64)
    if Yref.size == 0:
        return 0.0, 0.0
    rms = np.sqrt(np.mean(Yref * Yref))
    floor = max(1e-2 * rms, 1e-30)
    max_rel = float(np.max(np.abs(Y - Yref) / np.maximum(np.abs(Yref), floor)))
    nrm = float(np.linalg.norm(Y - Yref) / max(np.linalg.norm(Yref), 1e-30))
    return max_rel, nrm


def assert_close(Y, Yref, what=""):
    mr, nr = rel_errors(Y, Yref)
    assert mr <= REL_TOL and nr <= REL_TOL, f"{what}: max_rel={mr:.3e} norm_rel={nr:.3e}"
    return mr, nr


def assert_close_terms(Y, Yref, Tabs, what=""):
    """Normwise <= REL_TOL and |Y - Yref| <= MX_TERM_TOL * sum_k |a_k w_k| per output."""
    Y = np.asarray(Y, np.float64)
    _, nr = rel_errors(Y, Yref)
    comp = float(np.max(np.abs(Y - Yref) / np.maximum(Tabs, 1e-30))) if Y.size else 0.0
    assert nr <= REL_TOL and comp <= MX_TERM_TOL, f"{what}: norm_rel={nr:.3e} term_rel={comp:.3e}"
    return nr, comp
