"""The output-error report of the decomposition variants (oracle only)."""
import numpy as np

import synth
from oracle import quality as Q
from oracle import sdq as S


def test_report_rows_and_identities():
    W = synth.make_w(2, 0, 32, 512)
    X = synth.make_x(2, 8, 512)
    X_cal = synth.make_x(2, 40, 512)[8:]
    rows = dict(Q.report(W, X, X_cal, "int", n_is=(3,)))
    assert len(rows) == 1 + 2 * len(Q.DECOMPS) * len(Q.ORDERS)
    assert all(np.isfinite(e) and e > 0 for e in rows.values())
    # the default decomposition is the staged one with the significance metric, largest first
    assert rows["SDQ 1:8+3:8, product significance, default decomposition"] == \
        rows["SDQ 1:8+3:8, product significance, product large"]
    assert rows["SDQ 1:8+3:8, magnitude significance, default decomposition"] == \
        rows["SDQ 1:8+3:8, magnitude significance, magnitude large"]
    # the dense baseline keeps every weight: its only errors are the quantizers'
    L = S.pack_logical(W, Q.dense_baseline("int"))
    assert L["mask_i"].all() and not L["mask_o"].any()
    assert rows[next(k for k in rows if k.startswith("dense"))] == Q.rel_error(X, W, Q.dense_baseline("int"))


def test_scale_report_bits_and_identities():
    W = synth.make_w(2, 0, 16, 512)
    X = synth.make_x(2, 4, 512)
    X_cal = synth.make_x(2, 20, 512)[4:]
    rows = Q.scale_report(W, X, X_cal, n_is=(3,))
    assert len(rows) == 9
    bits = {(r[1], r[2]): r[3] for r in rows}
    # 1:8 8-bit outliers (1.375) + 3:8 int4 (2.625) + fp32 row scale (32/K) + scales
    assert bits[("f16", 16)] == 1.375 + 2.625 + 32 / 512 + 1.0
    assert bits[("e4m3", 16)] == 1.375 + 2.625 + 32 / 512 + 0.5 + 32 / 512
    assert bits[("ue6m2", 64)] == 1.375 + 2.625 + 32 / 512 + 0.125
    assert all(np.isfinite(r[4]) and r[4] > 0 for r in rows)
