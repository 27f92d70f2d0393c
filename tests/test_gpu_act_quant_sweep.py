"""GPU: the activation quantizer's conversion over every fp32 value in range.

Each row holds qmax (127 for int8, 448 for e4m3) in its first 128 elements,
so its scale is s_a = qmax/qmax = 1 and inv = 1 exactly; the other elements
then convert as enc(x).  Every fp32 bit pattern with |x| <= qmax (2.25e9 per
format, both signs) passes through sdq_quantize_act in chunks that the GPU
generates itself.  Every variant of the activation kernel converts through the
same routine; this sweep uses the two-pass variant (long rows).

Rather than evaluate the oracle on all 4.5e9 values, the test uses the shape
of the map: the oracle's encoders round to nearest even, so the code (as a
signed magnitude) is a non-decreasing step function of |x| on each sign.  On
the GPU the sweep checks that the produced codes are non-decreasing and
collects every point where the code changes; the oracle is then evaluated at
each such point and at the value one ulp below it.  Two non-decreasing step
functions that agree at both sides of every step of one of them, and at the
start, agree everywhere: the GPU equals the oracle on every value in range.
"""
import numpy as np
import pytest

from oracle import formats as F
from tests.gpu_util import say, torch_cuda

import paper_2406_13868_amd as sdq

pytestmark = pytest.mark.gpu

ROWS, PAY, PAD = 8192, 16384, 128          # a chunk: 2^27 values in rows of 16512
CASES = {"int8": (sdq.Config.int_family(), 127.0), "e4m3": (sdq.Config.mx_family(), 448.0)}


def _oracle_codes(fmt, bits):
    x = np.asarray(bits, np.uint32).view(np.float32)
    if fmt == "int8":
        return F.int_rne_clamp(x, 127).astype(np.int8).view(np.uint8)
    return F.e4m3_encode(x)


def _magnitude(fmt, codes):
    """Signed magnitude order of the codes: non-decreasing in |x| for one sign."""
    import torch
    c = codes.to(torch.int32)
    if fmt == "int8":
        c = torch.where(c >= 128, c - 256, c)  # two's complement value
        return c.abs()
    return c & 0x7F                            # e4m3 magnitude bits


@pytest.mark.parametrize("fmt", ["int8", "e4m3"])
def test_every_fp32_value_in_range_converts_like_the_oracle(fmt):
    torch = torch_cuda()
    cfg, qmax = CASES[fmt]
    top = int(np.float32(qmax).view(np.uint32))   # largest pattern of a value <= qmax
    n_chunk = ROWS * PAY
    checked = 0
    for sign in (0, 1):
        steps_idx, steps_new = [], []
        prev_code = None
        start = 0
        while start <= top:
            n = min(n_chunk, top + 1 - start)
            say("act sweep", fmt, "sign", sign, "patterns", start, n)
            bits = torch.arange(start, start + n, dtype=torch.int64, device="cuda")
            if sign:
                bits = bits | 0x80000000
            vals = bits.to(torch.int32).view(torch.float32) if not sign else \
                (bits - (1 << 32)).to(torch.int32).view(torch.float32)
            X = torch.full((ROWS, PAD + PAY), qmax, dtype=torch.float32, device="cuda")
            pay = torch.full((ROWS * PAY,), qmax, dtype=torch.float32, device="cuda")
            pay[:n] = vals
            X[:, PAD:] = pay.view(ROWS, PAY)  # a 2-D block assignment (a reshape of the view would copy)
            del pay
            Xq, s_a = sdq.quantize_act(X, cfg)
            assert bool((s_a == 1.0).all()), "a row's scale is not 1"
            codes = Xq[:, PAD:].contiguous().view(-1)[:n]
            mag = _magnitude(fmt, codes)
            # the sign bit: int8 codes of negative values are <= 0, e4m3 ones carry 0x80
            if fmt == "e4m3":
                assert bool(((codes & 0x80) == (0x80 if sign else 0)).all()), "sign bit"
            else:
                v = torch.where(codes.to(torch.int32) >= 128, codes.to(torch.int32) - 256, codes.to(torch.int32))
                assert bool((v <= 0).all() if sign else (v >= 0).all()), "sign"
            assert bool((mag[1:] >= mag[:-1]).all()), "codes are not monotone in |x|"
            ch = torch.nonzero(codes[1:] != codes[:-1]).flatten() + 1
            if prev_code is not None and int(codes[0]) != prev_code:
                steps_idx.append(start)
                steps_new.append(int(codes[0]))
            steps_idx += (ch + start).tolist()
            steps_new += codes[ch].tolist()
            if start == 0:  # the first value, 0 or -0
                first = int(codes[0])
                assert first == int(_oracle_codes(fmt, [0x80000000 if sign else 0])[0])
            prev_code = int(codes[-1])
            checked += n
            start += n
            del X, Xq, bits, vals, codes, mag
        # the oracle at both sides of every step the GPU took
        idx = np.asarray(steps_idx, np.int64)
        sb = np.uint32(0x80000000) if sign else np.uint32(0)
        after = _oracle_codes(fmt, idx.astype(np.uint32) | sb)
        before = _oracle_codes(fmt, (idx - 1).astype(np.uint32) | sb)
        new = np.asarray(steps_new, np.uint8)
        assert np.array_equal(after, new), "a step of the GPU lands on another code than the oracle's"
        assert np.all(before != after), "the oracle does not step where the GPU does"
        # the GPU codes before each step are the previous step's new code
        prev = np.concatenate([[int(_oracle_codes(fmt, [sb])[0])], new[:-1]]).astype(np.uint8)
        assert np.array_equal(before, prev), "the oracle steps where the GPU does not"
        n_codes = 128 if fmt == "int8" else 127
        assert len(idx) == n_codes - 1, f"{len(idx)} steps"
    assert checked == 2 * (top + 1)
