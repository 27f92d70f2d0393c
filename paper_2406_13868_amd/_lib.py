"""ctypes view of libsdq.so (declarations in include/sdq.h)."""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsdq.so")

SDQ_OK = 0
STATUS = {
    0: "SDQ_OK", -1: "SDQ_ERR_NULL", -2: "SDQ_ERR_SHAPE", -3: "SDQ_ERR_CONFIG",
    -4: "SDQ_ERR_BUFFER_TOO_SMALL", -5: "SDQ_ERR_HIP", -6: "SDQ_ERR_UNSUPPORTED",
    -7: "SDQ_ERR_VALUE", -8: "SDQ_ERR_TOO_LARGE",
}
FAMILY_INT, FAMILY_MX, FAMILY_DUAL = 0, 1, 2
FMT_INT8, FMT_INT4, FMT_E4M3, FMT_E2M1 = 1, 2, 3, 4
METRIC_MAGNITUDE, METRIC_PRODUCT = 0, 1
DECOMP = {"same": 0, "magnitude": 1, "product": 2, "error": 3, "output_error": 4}
ORDER = {"large": 0, "small": 1}
SCALE = {"": 0, "e4m3": 1, "ue6m2": 2}
DTYPE_F32, DTYPE_BF16 = 0, 1
PATH_AUTO, PATH_DECODE, PATH_MFMA, PATH_DENSE, PATH_SPLITK = 0, 1, 2, 3, 4

# Every exported symbol, as declared in include/sdq.h.
EXPORTS = (
    "sdq_status_string", "sdq_check", "sdq_pack_size", "sdq_logical_bytes", "sdq_pack",
    "sdq_pack_logical", "sdq_unpack_dense", "sdq_quantize_act", "sdq_gemm", "sdq_gemm_ex",
    "sdq_gemm_path", "sdq_linear", "sdq_gemm_workspace_size", "sdq_gemm_ws",
    "sdq_quantize_act_dual", "sdq_gemm_dual", "sdq_gemm_static", "sdq_gemm_path_ws",
    "sdq_unpack_weights", "sdq_gemm_unpacked",
)
STATIC_SCRATCH_BYTES = 48 * 1024 * 1024


class sdq_config(C.Structure):
    _fields_ = [("family", C.c_int32), ("n_o", C.c_int32), ("m_o", C.c_int32),
                ("fmt_o", C.c_int32), ("n_i", C.c_int32), ("m_i", C.c_int32),
                ("fmt_i", C.c_int32), ("fmt_a", C.c_int32), ("metric", C.c_int32),
                ("decomp", C.c_int32), ("order", C.c_int32), ("sfmt_i", C.c_int32),
                ("y_dtype", C.c_int32), ("qv_i", C.c_int32)]


class SDQError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {STATUS.get(status, status)}")
        self.status = status


_lib = None


def _bind_to_torch_runtime() -> None:
    """libsdq.so asks for the HIP runtime by its soname, libamdhip64.so.7.
    torch's ROCm wheel carries its own copy of the runtime (same soname), which
    its libraries ask for as libamdhip64.so.  With torch imported first the
    loader hands libsdq.so torch's copy.  Loaded the other way round, the
    process would hold two HIP runtimes (and two HSA runtimes): the one torch
    initialises owns the GPU and the library's launches find no device."""
    try:
        import torch  # noqa: F401
    except ImportError:  # no torch: the library's own runtime is the only one
        pass


def _hip_runtimes() -> set:
    """Distinct files of the HIP runtime mapped into this process (Linux)."""
    try:
        with open("/proc/self/maps") as f:
            maps = f.read()
    except OSError:
        return set()
    return {os.path.realpath(line.split()[-1]) for line in maps.splitlines()
            if "/libamdhip64.so" in line}


def _check_one_runtime() -> None:
    rts = _hip_runtimes()
    if len(rts) > 1:
        raise RuntimeError("two HIP runtimes are loaded in this process (" + ", ".join(sorted(rts)) +
                           "): load libsdq.so after the runtime the rest of the process uses "
                           "(import torch first)")


def lib() -> C.CDLL:
    """Load libsdq.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2406_13868_amd.build` (no CPU fallback exists)")
        _bind_to_torch_runtime()
        L = C.CDLL(LIB_PATH)
        _check_one_runtime()
        P = C.POINTER
        cfgp = P(sdq_config)
        i64, vp, f32p, u8p = C.c_int64, C.c_void_p, P(C.c_float), P(C.c_uint8)
        sig = {
            "sdq_status_string": (C.c_char_p, [C.c_int]),
            "sdq_check": (C.c_int, [cfgp, i64, i64]),
            "sdq_pack_size": (C.c_int, [cfgp, i64, i64, P(C.c_size_t)]),
            "sdq_logical_bytes": (C.c_int, [cfgp, i64, i64, P(C.c_size_t)]),
            "sdq_pack": (C.c_int, [cfgp, vp, i64, i64, vp, vp, C.c_size_t, C.c_int]),
            "sdq_pack_logical": (C.c_int, [cfgp, vp, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, C.c_int]),
            "sdq_unpack_dense": (C.c_int, [cfgp, vp, C.c_size_t, i64, i64, vp, vp, vp, vp, vp]),
            "sdq_quantize_act": (C.c_int, [cfgp, vp, C.c_int32, i64, i64, vp, vp, vp]),
            "sdq_gemm": (C.c_int, [cfgp, vp, vp, i64, vp, i64, i64, vp, vp]),
            "sdq_gemm_ex": (C.c_int, [cfgp, vp, vp, i64, vp, i64, i64, vp, vp, C.c_int32]),
            "sdq_gemm_path": (C.c_int, [cfgp, i64, i64, i64, P(C.c_int32)]),
            "sdq_gemm_path_ws": (C.c_int, [cfgp, i64, i64, i64, P(C.c_int32)]),
            "sdq_gemm_workspace_size": (C.c_int, [cfgp, i64, i64, i64, C.c_int32, P(C.c_size_t)]),
            "sdq_gemm_ws": (C.c_int, [cfgp, vp, vp, i64, vp, i64, i64, vp, vp, C.c_size_t, vp,
                                      C.c_int32]),
            "sdq_linear": (C.c_int, [cfgp, vp, C.c_int32, i64, vp, vp, vp, i64, i64, vp, vp]),
            "sdq_quantize_act_dual": (C.c_int, [cfgp, vp, C.c_int32, i64, i64, vp, vp, vp, vp, vp]),
            "sdq_gemm_dual": (C.c_int, [cfgp, vp, vp, vp, vp, i64, vp, i64, i64, vp, vp]),
            "sdq_gemm_static": (C.c_int, [cfgp, vp, vp, i64, vp, i64, i64, vp, vp, C.c_int32]),
            "sdq_unpack_weights": (C.c_int, [cfgp, vp, i64, i64, vp, C.c_size_t, vp]),
            "sdq_gemm_unpacked": (C.c_int, [cfgp, vp, vp, i64, vp, i64, i64, vp, C.c_size_t, vp, vp]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        del u8p, f32p
        _lib = L
    return _lib


def check(status: int, what: str) -> None:
    if status != SDQ_OK:
        raise SDQError(status, what)
