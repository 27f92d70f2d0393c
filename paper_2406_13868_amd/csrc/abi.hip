// C ABI of libsdq: argument validation and kernel dispatch (see include/sdq.h).
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

#include "kernels.h"

using namespace sdq;

namespace {

bool log_enabled() {
  static const bool on = [] {
    const char* e = std::getenv("SDQ_LOG");
    return e && e[0] == '1';
  }();
  return on;
}

// The weight-streaming decode kernel wherever its registers fit the tokens
// (measured at M = 2..8: 4096x4096 takes 3.8-8.4 us there against 13.7 us
// on the matrix cores, 11008x4096 6.3-17.8 against 23.6).
int32_t auto_path(const Cfg& c, int64_t M, int64_t K) {
  if (!c.mx && M <= 8 && decode_fits(M, K)) return SDQ_PATH_DECODE;
  return SDQ_PATH_MFMA;
}

// The path of sdq_gemm_ws: the two-pass form where its one expansion per
// weight beats the one-pass kernel's per token block, which needs many tokens
// and a grid of at least 160 workgroups of 256 outputs x 128 tokens (measured:
// 4096x4096 at M = 1024, 128 workgroups, takes 42 us in one pass against 48
// in two; 11008x4096 at M = 512, 172 workgroups, 56 against 52).
//
// The INT family's split-K path where it measured faster than the matrix-core
// path without a workspace: long rows (4096x16384 at M = 16 and 64: 25.4 and
// 33.0 us against 36.0 and 41.3), 64 tokens and more on wide layers
// (11008x4096 at M = 64: 32.7 against 42.4; 16384x4096: 32.6 against 34.4)
// and 256 tokens (4096x4096: 31.5 against 32.3; 11008x4096: 73.3 against
// 89.8).  It loses on small grids, where its second pass over the partial
// sums costs more than the fuller GPU saves (4096x4096 at M = 64 and 128:
// 18.9 and 24.4 against 15.6 and 22.2; 16384x4096 at M = 16: 25.4 against
// 22.2).
//
// Above 256 tokens the split-K path runs the tiled kernel over K ranges. It
// wins over the matrix-core path where that kernel's own grid of ceil(N/128)
// x ceil(M/128) workgroups would leave the GPU under-filled (under 384):
// 4096x4096 at M = 512 / 768 / 1024: 47.8 / 78.5 / 80.8 us against 58.9 /
// 81.1 / 86.1; 4096x11008 at M = 512 / 1024: 108 / 192 against 138 / 218;
// 11008x4096 at M = 512 (344 workgroups): 118 against 135.  On fuller grids
// it loses (11008x4096 at M = 640 / 768: 147 / 208 against 140 / 200).
bool split_wins(int64_t M, int64_t N, int64_t K) {
  if (M > kSplitMaxM) return K >= 1024 && (N + 127) / 128 * ((M + 127) / 128) < 384;
  return K >= 8192 || (M >= 64 && N >= 8192) || M >= 256;
}

// The MX family's split-K path where the one-pass grid of 128 outputs x 128
// tokens per workgroup would hold at most 128 workgroups (half the CUs):
// measured on the LLaMA-7B shapes, 4096x4096 takes 9.1 / 14.3 / 20.8 us at M
// = 1 / 64 / 128 against 25.9 / 29.8 / 26.5 in one pass, and 28.6 against 30.8
// at 512; 4096x11008 14.1 / 19.7 / 34.8 / 51.4 at M = 1 / 64 / 256 / 512
// against 63.1 / 72.4 / 64.7 / 73.9.  It loses on fuller grids (11008x4096
// at M = 256: 40.5 against 39.6; 4096x4096 at M = 768: 41.5 against 38.6),
// and needs K for at least two ranges.
bool mx_split_wins(int64_t M, int64_t N, int64_t K) {
  return K >= 2 * kMxSplitMinChunks * kChunkK && (N + 127) / 128 * ((M + 127) / 128) <= 128;
}

int32_t auto_path_ws(const Cfg& c, int64_t M, int64_t N, int64_t K) {
  const int64_t wgs = (N + 255) / 256 * ((M + 127) / 128);
  if (c.mx && c.n_o > 0 && M >= kDenseMinM && wgs >= 160) return SDQ_PATH_DENSE;
  if (c.mx && mx_split_wins(M, N, K)) return SDQ_PATH_SPLITK;
  const int32_t p = auto_path(c, M, K);
  if (!c.mx && p == SDQ_PATH_MFMA && split_wins(M, N, K)) return SDQ_PATH_SPLITK;
  return p;
}

// Workspace bytes of a path that takes one (0 for the others).
size_t path_workspace_bytes(const Cfg& c, int32_t path, int64_t M, int64_t N, int64_t K) {
  if (path == SDQ_PATH_DENSE) return mx_dense_workspace_bytes(N, K);
  if (path == SDQ_PATH_SPLITK) return c.mx ? mx_split_workspace_bytes(M, N, K) : int_split_workspace_bytes(M, N, K);
  return 0;
}

// Whether a workspace path serves the configuration.
bool path_serves(const Cfg& c, int32_t path) {
  if (path == SDQ_PATH_DENSE) return c.mx && c.n_o > 0;
  return true;  // SDQ_PATH_SPLITK: the INT and the MX family
}

// The launchers report a failed launch through hipGetLastError, which also
// returns an error that an earlier, unrelated HIP call on this thread left
// pending (the runtime keeps one per thread until it is read).  Reading it
// here, before the launches, keeps such an error from being reported as this
// call's.  A sticky error (a faulted context) is not lost: every later launch
// fails again.
void drop_pending_error() { (void)hipGetLastError(); }

}  // namespace

extern "C" const char* sdq_status_string(sdq_status s) {
  switch (s) {
    case SDQ_OK: return "SDQ_OK: success";
    case SDQ_ERR_NULL: return "SDQ_ERR_NULL: a required pointer is NULL";
    case SDQ_ERR_SHAPE: return "SDQ_ERR_SHAPE: M, N or K out of range, or K not a multiple of 32 (or of a 64-K scale vector)";
    case SDQ_ERR_CONFIG: return "SDQ_ERR_CONFIG: malformed configuration";
    case SDQ_ERR_BUFFER_TOO_SMALL: return "SDQ_ERR_BUFFER_TOO_SMALL: output buffer too small";
    case SDQ_ERR_HIP: return "SDQ_ERR_HIP: a HIP call or kernel launch failed";
    case SDQ_ERR_UNSUPPORTED: return "SDQ_ERR_UNSUPPORTED: configuration or path not implemented";
    case SDQ_ERR_VALUE: return "SDQ_ERR_VALUE: input value out of range";
    case SDQ_ERR_TOO_LARGE:
      return "SDQ_ERR_TOO_LARGE: the path needs more scratch than sdq_gemm_static's static array holds";
  }
  return "unknown sdq_status";
}

extern "C" sdq_status sdq_check(const sdq_config* cfg, int64_t N, int64_t K) {
  return check_config(cfg, N, K, nullptr);
}

extern "C" sdq_status sdq_quantize_act(const sdq_config* cfg, const void* X, int32_t x_dtype,
                                       int64_t M, int64_t K, void* Xq, float* s_a, void* stream) {
  Cfg c;
  const sdq_status s = check_config(cfg, 1, K, &c);
  if (s != SDQ_OK) return s;
  if (c.dual) return SDQ_ERR_UNSUPPORTED;  // two activation tensors: sdq_quantize_act_dual
  if (M < 0 || M > (int64_t(1) << 31)) return SDQ_ERR_SHAPE;
  if (x_dtype != SDQ_DTYPE_F32 && x_dtype != SDQ_DTYPE_BF16) return SDQ_ERR_CONFIG;
  if (M == 0) return SDQ_OK;
  if (!X || !Xq || !s_a) return SDQ_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(X) % 16 || reinterpret_cast<uintptr_t>(Xq) % 16) return SDQ_ERR_SHAPE;
  drop_pending_error();
  const hipError_t e = launch_act_quant(c, X, x_dtype, M, K, static_cast<uint8_t*>(Xq), s_a,
                                        static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SDQ_OK : SDQ_ERR_HIP;
}

extern "C" sdq_status sdq_gemm_path(const sdq_config* cfg, int64_t M, int64_t N, int64_t K,
                                    int32_t* path) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (!path) return SDQ_ERR_NULL;
  if (M < 0) return SDQ_ERR_SHAPE;
  if (c.dual) return SDQ_ERR_UNSUPPORTED;  // sdq_gemm_dual has one kernel
  *path = auto_path(c, M, K);
  return SDQ_OK;
}

extern "C" sdq_status sdq_gemm_path_ws(const sdq_config* cfg, int64_t M, int64_t N, int64_t K,
                                       int32_t* path) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (!path) return SDQ_ERR_NULL;
  if (M < 0) return SDQ_ERR_SHAPE;
  if (c.dual) return SDQ_ERR_UNSUPPORTED;
  *path = auto_path_ws(c, M, N, K);
  return SDQ_OK;
}

extern "C" sdq_status sdq_gemm_ex(const sdq_config* cfg, const void* Xq, const float* s_a,
                                  int64_t M, const void* packed, int64_t N, int64_t K, void* Y,
                                  void* stream, int32_t path) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (M < 0 || M > (int64_t(1) << 31) || M * N > (int64_t(1) << 40)) return SDQ_ERR_SHAPE;
  if (path < SDQ_PATH_AUTO || path > SDQ_PATH_SPLITK) return SDQ_ERR_CONFIG;
  if (path == SDQ_PATH_DENSE || path == SDQ_PATH_SPLITK) return SDQ_ERR_UNSUPPORTED;  // sdq_gemm_ws
  if (c.dual) return SDQ_ERR_UNSUPPORTED;                  // two activation tensors: sdq_gemm_dual
  if (M == 0) return SDQ_OK;
  if (!Xq || !s_a || !packed || !Y) return SDQ_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(Xq) % 16 || reinterpret_cast<uintptr_t>(packed) % 16 ||
      reinterpret_cast<uintptr_t>(Y) % 4)
    return SDQ_ERR_SHAPE;
  if (path == SDQ_PATH_AUTO) path = auto_path(c, M, K);
  if (path == SDQ_PATH_DECODE && (c.mx || !decode_fits(M, K))) return SDQ_ERR_UNSUPPORTED;
  const auto* xq = static_cast<const uint8_t*>(Xq);
  const auto* blob = static_cast<const uint8_t*>(packed);
  const hipStream_t st = static_cast<hipStream_t>(stream);
  drop_pending_error();
  hipError_t e;
  const char* name;
  if (c.mx) {
    e = launch_mx_mfma(c, xq, s_a, M, blob, N, K, Y, st);
    name = "mx_mfma";
  } else if (path == SDQ_PATH_DECODE) {
    e = launch_int_decode(c, xq, s_a, M, blob, N, K, Y, st);
    name = "int_decode";
  } else {
    e = launch_int_mfma(c, xq, s_a, M, blob, N, K, Y, st);
    name = "int_mfma";
  }
  if (log_enabled())
    std::fprintf(stderr, "[sdq] gemm M=%lld N=%lld K=%lld -> %s\n", (long long)M, (long long)N,
                 (long long)K, name);
  return e == hipSuccess ? SDQ_OK : SDQ_ERR_HIP;
}

extern "C" sdq_status sdq_gemm_workspace_size(const sdq_config* cfg, int64_t M, int64_t N,
                                              int64_t K, int32_t path, size_t* bytes) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (!bytes) return SDQ_ERR_NULL;
  if (M < 0) return SDQ_ERR_SHAPE;
  if (path < SDQ_PATH_AUTO || path > SDQ_PATH_SPLITK) return SDQ_ERR_CONFIG;
  if (c.dual) return SDQ_ERR_UNSUPPORTED;
  if (path == SDQ_PATH_AUTO) path = auto_path_ws(c, M, N, K);
  if (!path_serves(c, path)) return SDQ_ERR_UNSUPPORTED;
  *bytes = path_workspace_bytes(c, path, M, N, K);
  return SDQ_OK;
}

extern "C" sdq_status sdq_gemm_ws(const sdq_config* cfg, const void* Xq, const float* s_a,
                                  int64_t M, const void* packed, int64_t N, int64_t K, void* Y,
                                  void* workspace, size_t ws_bytes, void* stream, int32_t path) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (M < 0 || M > (int64_t(1) << 31) || M * N > (int64_t(1) << 40)) return SDQ_ERR_SHAPE;
  if (path < SDQ_PATH_AUTO || path > SDQ_PATH_SPLITK) return SDQ_ERR_CONFIG;
  if (c.dual) return SDQ_ERR_UNSUPPORTED;
  if (path == SDQ_PATH_AUTO) path = auto_path_ws(c, M, N, K);
  if (path != SDQ_PATH_DENSE && path != SDQ_PATH_SPLITK)
    return sdq_gemm_ex(cfg, Xq, s_a, M, packed, N, K, Y, stream, path);
  if (!path_serves(c, path)) return SDQ_ERR_UNSUPPORTED;
  if (M == 0) return SDQ_OK;
  if (!Xq || !s_a || !packed || !Y || !workspace) return SDQ_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(Xq) % 16 || reinterpret_cast<uintptr_t>(packed) % 16 ||
      reinterpret_cast<uintptr_t>(workspace) % 16 || reinterpret_cast<uintptr_t>(Y) % 4)
    return SDQ_ERR_SHAPE;
  if (ws_bytes < path_workspace_bytes(c, path, M, N, K)) return SDQ_ERR_BUFFER_TOO_SMALL;
  const auto* xq = static_cast<const uint8_t*>(Xq);
  const auto* blob = static_cast<const uint8_t*>(packed);
  const hipStream_t st = static_cast<hipStream_t>(stream);
  drop_pending_error();
  const hipError_t e = path == SDQ_PATH_DENSE ? launch_mx_dense(c, xq, s_a, M, blob, N, K, Y, workspace, st)
                       : c.mx                  ? launch_mx_split(c, xq, s_a, M, blob, N, K, Y, workspace, st)
                                               : launch_int_split(c, xq, s_a, M, blob, N, K, Y, workspace, st);
  if (log_enabled())
    std::fprintf(stderr, "[sdq] gemm M=%lld N=%lld K=%lld -> %s\n", (long long)M, (long long)N,
                 (long long)K, path == SDQ_PATH_DENSE ? "mx_dense (two passes)" : c.mx ? "mx_split (K ranges)" : "int_split (K ranges)");
  return e == hipSuccess ? SDQ_OK : SDQ_ERR_HIP;
}

extern "C" sdq_status sdq_unpack_weights(const sdq_config* cfg, const void* packed, int64_t N, int64_t K,
                                         void* workspace, size_t ws_bytes, void* stream) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (!path_serves(c, SDQ_PATH_DENSE)) return SDQ_ERR_UNSUPPORTED;  // the MX family with outliers
  if (!packed || !workspace) return SDQ_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(packed) % 16 || reinterpret_cast<uintptr_t>(workspace) % 16)
    return SDQ_ERR_SHAPE;
  if (ws_bytes < mx_dense_workspace_bytes(N, K)) return SDQ_ERR_BUFFER_TOO_SMALL;
  drop_pending_error();
  const hipError_t e = launch_mx_densify(c, static_cast<const uint8_t*>(packed), N, K, workspace,
                                         static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SDQ_OK : SDQ_ERR_HIP;
}

extern "C" sdq_status sdq_gemm_unpacked(const sdq_config* cfg, const void* Xq, const float* s_a, int64_t M,
                                        const void* packed, int64_t N, int64_t K, const void* workspace,
                                        size_t ws_bytes, void* Y, void* stream) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (M < 0 || M > (int64_t(1) << 31) || M * N > (int64_t(1) << 40)) return SDQ_ERR_SHAPE;
  if (!path_serves(c, SDQ_PATH_DENSE)) return SDQ_ERR_UNSUPPORTED;
  if (M == 0) return SDQ_OK;
  if (!Xq || !s_a || !packed || !workspace || !Y) return SDQ_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(Xq) % 16 || reinterpret_cast<uintptr_t>(packed) % 16 ||
      reinterpret_cast<uintptr_t>(workspace) % 16 || reinterpret_cast<uintptr_t>(Y) % 4)
    return SDQ_ERR_SHAPE;
  if (ws_bytes < mx_dense_workspace_bytes(N, K)) return SDQ_ERR_BUFFER_TOO_SMALL;
  drop_pending_error();
  const hipError_t e = launch_mx_dense_pass(c, static_cast<const uint8_t*>(Xq), s_a, M,
                                            static_cast<const uint8_t*>(packed), N, K, Y, workspace,
                                            static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SDQ_OK : SDQ_ERR_HIP;
}

extern "C" sdq_status sdq_gemm_static(const sdq_config* cfg, const void* Xq, const float* s_a,
                                      int64_t M, const void* packed, int64_t N, int64_t K, void* Y,
                                      void* stream, int32_t path) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (M < 0 || M > (int64_t(1) << 31) || M * N > (int64_t(1) << 40)) return SDQ_ERR_SHAPE;
  if (path < SDQ_PATH_AUTO || path > SDQ_PATH_SPLITK) return SDQ_ERR_CONFIG;
  if (c.dual) return SDQ_ERR_UNSUPPORTED;
  if (path == SDQ_PATH_AUTO) path = auto_path_ws(c, M, N, K);
  if (path != SDQ_PATH_DENSE && path != SDQ_PATH_SPLITK)
    return sdq_gemm_ex(cfg, Xq, s_a, M, packed, N, K, Y, stream, path);
  if (!path_serves(c, path)) return SDQ_ERR_UNSUPPORTED;
  if (path_workspace_bytes(c, path, M, N, K) > kStaticScratchBytes) return SDQ_ERR_TOO_LARGE;
  if (M == 0) return SDQ_OK;
  if (!Xq || !s_a || !packed || !Y) return SDQ_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(Xq) % 16 || reinterpret_cast<uintptr_t>(packed) % 16 ||
      reinterpret_cast<uintptr_t>(Y) % 4)
    return SDQ_ERR_SHAPE;
  const auto* xq = static_cast<const uint8_t*>(Xq);
  const auto* blob = static_cast<const uint8_t*>(packed);
  const hipStream_t st = static_cast<hipStream_t>(stream);
  drop_pending_error();
  const hipError_t e = path == SDQ_PATH_DENSE ? launch_mx_dense_static(c, xq, s_a, M, blob, N, K, Y, st)
                                              : split_static(c, xq, s_a, M, blob, N, K, Y, st);
  if (log_enabled())
    std::fprintf(stderr, "[sdq] gemm M=%lld N=%lld K=%lld -> %s, static scratch\n", (long long)M,
                 (long long)N, (long long)K, path == SDQ_PATH_DENSE ? "mx_dense (two passes)" : "int_split");
  return e == hipSuccess ? SDQ_OK : SDQ_ERR_HIP;
}

extern "C" sdq_status sdq_gemm(const sdq_config* cfg, const void* Xq, const float* s_a, int64_t M,
                               const void* packed, int64_t N, int64_t K, void* Y, void* stream) {
  return sdq_gemm_ex(cfg, Xq, s_a, M, packed, N, K, Y, stream, SDQ_PATH_AUTO);
}

extern "C" sdq_status sdq_linear(const sdq_config* cfg, const void* X, int32_t x_dtype, int64_t M,
                                 void* Xq, float* s_a, const void* packed, int64_t N, int64_t K,
                                 void* Y, void* stream) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (M < 0 || M > (int64_t(1) << 31) || M * N > (int64_t(1) << 40)) return SDQ_ERR_SHAPE;
  if (x_dtype != SDQ_DTYPE_F32 && x_dtype != SDQ_DTYPE_BF16) return SDQ_ERR_CONFIG;
  if (c.dual) return SDQ_ERR_UNSUPPORTED;
  if (M == 0) return SDQ_OK;
  if (!X || !Xq || !s_a || !packed || !Y) return SDQ_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(X) % 16 || reinterpret_cast<uintptr_t>(Xq) % 16 ||
      reinterpret_cast<uintptr_t>(packed) % 16 || reinterpret_cast<uintptr_t>(Y) % 4)
    return SDQ_ERR_SHAPE;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (auto_path(c, M, K) == SDQ_PATH_DECODE && decode_fused_fits(M, K)) {
    drop_pending_error();
    const hipError_t e = launch_int_decode_fused(c, X, x_dtype, M, static_cast<uint8_t*>(Xq), s_a,
                                                 static_cast<const uint8_t*>(packed), N, K, Y, st);
    if (log_enabled())
      std::fprintf(stderr, "[sdq] linear M=%lld N=%lld K=%lld -> int_decode (fused act quant)\n",
                   (long long)M, (long long)N, (long long)K);
    return e == hipSuccess ? SDQ_OK : SDQ_ERR_HIP;
  }
  const sdq_status q = sdq_quantize_act(cfg, X, x_dtype, M, K, Xq, s_a, stream);
  if (q != SDQ_OK) return q;
  return sdq_gemm(cfg, Xq, s_a, M, packed, N, K, Y, stream);
}

extern "C" sdq_status sdq_quantize_act_dual(const sdq_config* cfg, const void* X, int32_t x_dtype,
                                            int64_t M, int64_t K, void* Xq_o, float* s_a_o,
                                            void* Xq_i, void* e_a_i, void* stream) {
  Cfg c;
  const sdq_status s = check_config(cfg, 1, K, &c);
  if (s != SDQ_OK) return s;
  if (!c.dual) return SDQ_ERR_CONFIG;
  if (M < 0 || M > (int64_t(1) << 31)) return SDQ_ERR_SHAPE;
  if (x_dtype != SDQ_DTYPE_F32 && x_dtype != SDQ_DTYPE_BF16) return SDQ_ERR_CONFIG;
  if (M == 0) return SDQ_OK;
  if (!X || !Xq_o || !s_a_o || !Xq_i || !e_a_i) return SDQ_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(X) % 16 || reinterpret_cast<uintptr_t>(Xq_o) % 16 ||
      reinterpret_cast<uintptr_t>(Xq_i) % 16)
    return SDQ_ERR_SHAPE;
  drop_pending_error();
  const hipError_t e = launch_act_quant_dual(X, x_dtype, M, K, static_cast<uint8_t*>(Xq_o), s_a_o,
                                             static_cast<uint8_t*>(Xq_i), static_cast<uint8_t*>(e_a_i),
                                             static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SDQ_OK : SDQ_ERR_HIP;
}

extern "C" sdq_status sdq_gemm_dual(const sdq_config* cfg, const void* Xq_o, const float* s_a_o,
                                    const void* Xq_i, const void* e_a_i, int64_t M, const void* packed,
                                    int64_t N, int64_t K, void* Y, void* stream) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (!c.dual) return SDQ_ERR_CONFIG;
  if (M < 0 || M > (int64_t(1) << 31) || M * N > (int64_t(1) << 40)) return SDQ_ERR_SHAPE;
  if (M == 0) return SDQ_OK;
  if (!Xq_o || !s_a_o || !Xq_i || !e_a_i || !packed || !Y) return SDQ_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(Xq_o) % 16 || reinterpret_cast<uintptr_t>(Xq_i) % 16 ||
      reinterpret_cast<uintptr_t>(packed) % 16 || reinterpret_cast<uintptr_t>(Y) % 4)
    return SDQ_ERR_SHAPE;
  drop_pending_error();
  const hipError_t e = launch_dual_mfma(c, static_cast<const uint8_t*>(Xq_o), s_a_o,
                                        static_cast<const uint8_t*>(Xq_i), static_cast<const uint8_t*>(e_a_i),
                                        M, static_cast<const uint8_t*>(packed), N, K, Y,
                                        static_cast<hipStream_t>(stream));
  if (log_enabled())
    std::fprintf(stderr, "[sdq] gemm M=%lld N=%lld K=%lld -> dual_mfma\n", (long long)M, (long long)N,
                 (long long)K);
  return e == hipSuccess ? SDQ_OK : SDQ_ERR_HIP;
}
