"""GPU: per-token activation quantization must equal the oracle bit for bit."""
import numpy as np
import pytest

import synth
from oracle import formats as F
from oracle import sdq as S
from tests.gpu_util import say, torch_cuda

import paper_2406_13868_amd as sdq

pytestmark = pytest.mark.gpu

INT = (sdq.Config.int_family(), S.Config("int", 1, 8, "e4m3", 3, 8, "int4", "int8"))
MX = (sdq.Config.mx_family(), S.Config("mx", 1, 8, "e4m3", 2, 8, "e2m1", "e4m3"))


def _run(X: np.ndarray, dtype: str, cfgs):
    torch = torch_cuda()
    cfg, cfg_o = cfgs
    t = torch.from_numpy(X)
    Xd = (t.to(torch.bfloat16) if dtype == "bf16" else t).cuda()
    Xq, s_a = sdq.quantize_act(Xd, cfg)
    torch.cuda.synchronize()
    Xq_ref, s_ref = S.quantize_act(X, cfg_o)
    return Xq.cpu().numpy(), s_a.cpu().numpy(), Xq_ref, s_ref


@pytest.mark.parametrize("fam", ["int", "mx"])
@pytest.mark.parametrize("case", [(1, 16, 256, "f32"), (2, 1, 4096, "bf16"), (4, 64, 4096, "bf16"),
                                  (4, 64, 16384, "bf16"), (3, 40, 11008, "bf16"),
                                  (2, 3, 32768, "bf16"), (1, 5, 128, "f32"), (2, 2, 65536, "bf16"),
                                  (1, 2, 131072, "f32"), (2, 8, 8192, "bf16"),
                                  (2, 256, 8192, "bf16"), (1, 300, 4224, "f32")],
                         ids=lambda c: f"w{c[0]}-{c[1]}x{c[2]}-{c[3]}")
def test_act_quant_bit_exact(fam, case):
    wid, M, K, dt = case
    say("act_quant", fam, case)
    X = synth.make_x(wid, M, K)
    if dt == "bf16":
        X = synth.bf16_round(X)
    Xq, s_a, Xq_ref, s_ref = _run(X, dt, INT if fam == "int" else MX)
    assert np.array_equal(s_a.view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(Xq, Xq_ref)


def test_zero_row_and_tiny_values():
    X = synth.make_x(1, 6, 256)
    X[2] = 0.0
    X[4] *= np.float32(1e-30)  # subnormal-range row: scales stay finite
    for cfgs in (INT, MX):
        say("act_quant zero/tiny rows", cfgs[0].family)
        Xq, s_a, Xq_ref, s_ref = _run(X, "f32", cfgs)
        assert np.array_equal(s_a.view(np.uint32), s_ref.view(np.uint32))
        assert np.array_equal(Xq, Xq_ref)


def _boundary_values(pos_values, vmax):
    mids = (pos_values[1:] + pos_values[:-1]) / 2
    v = []
    for m in mids:
        m32 = np.float32(m)
        v += [m32, np.nextafter(m32, np.float32(0)), np.nextafter(m32, np.float32(1e9))]
    v = np.array(v, np.float32)
    v = np.concatenate([v, -v, pos_values.astype(np.float32), -pos_values.astype(np.float32)])
    return v[np.abs(v) <= vmax]


@pytest.mark.parametrize("fam", ["int", "mx"])
def test_conversion_boundaries(fam):
    """Rows whose max is qmax have inv = 1 exactly: every value goes through the
    conversion unscaled, so rounding at every boundary is checked directly."""
    rng = np.random.default_rng(0)
    if fam == "int":
        qmax, vals = 127.0, np.concatenate([np.arange(-127, 127) + 0.5, np.arange(-127, 127) + 0.5 - 1e-5,
                                            rng.uniform(-127, 127, 20000)]).astype(np.float32)
    else:
        qmax = 448.0
        vals = np.concatenate([_boundary_values(F.E4M3_TABLE[:0x7F], 448.0),
                               rng.uniform(-448, 448, 20000).astype(np.float32),
                               (rng.standard_normal(20000) * 2.0 ** rng.integers(-14, 8, 20000)).astype(np.float32)])
        vals = vals[np.abs(vals) <= 448]
    K = 1024
    n = int(np.ceil(len(vals) / (K - 1)))
    X = np.zeros((n, K), np.float32)
    flat = np.zeros(n * (K - 1), np.float32)
    flat[: len(vals)] = vals
    X[:, 1:] = flat.reshape(n, K - 1)
    X[:, 0] = qmax
    say("conversion boundaries", fam, X.shape)
    Xq, s_a, Xq_ref, s_ref = _run(X, "f32", INT if fam == "int" else MX)
    assert (s_ref == np.float32(1.0)).all()
    assert np.array_equal(Xq, Xq_ref)


def test_m_zero_is_noop():
    torch = torch_cuda()
    X = torch.zeros((0, 256), dtype=torch.float32, device="cuda")
    Xq, s_a = sdq.quantize_act(X, INT[0])
    torch.cuda.synchronize()
    assert Xq.shape == (0, 256)
