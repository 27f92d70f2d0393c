// Kernel launchers of libsdq (device side).  Shapes and configurations are
// validated by the C ABI before any of these is called.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

#include "layout.h"
#include "sdq_internal.h"

namespace sdq {

// Workgroups are dispatched round robin over the 8 XCDs (workgroup b runs on
// XCD b % 8, each with its own L2).  This maps b to a work index so that every
// XCD takes a contiguous range of the G indices: neighbouring work items,
// which share cache lines, meet in one L2.  It is a bijection on [0, G).
__host__ __device__ __forceinline__ int xcd_contiguous(int b, int G) {
  const int x = b & 7, i = b >> 3, q = G >> 3, rem = G & 7;
  return x * q + min(x, rem) + i;
}

// (tile group, token block) of workgroup b in a grid of G x MB.  The items go
// to the XCDs in contiguous ranges of the order (token half, group, token
// block): with 8 or more token blocks the first four XCDs serve the first
// half of the tokens and the other four the second, so each XCD's L2 holds the
// activations of half the tokens while the weights of a group are read by
// one XCD per half.  Below 8 token blocks it is plain (group, token block).
// A bijection on [0, G * MB).
__host__ __device__ __forceinline__ void tile_work(int b, int G, int MB, int& group, int& mblock) {
  const int L = xcd_contiguous(b, G * MB);
  const int h0 = MB >= 8 ? (MB + 1) / 2 : MB;  // token blocks of the first half
  if (L < G * h0) {
    group = L / h0;
    mblock = L - group * h0;
  } else {
    const int L1 = L - G * h0, h1 = MB - h0;
    group = L1 / h1;
    mblock = h0 + (L1 - group * h1);
  }
}

hipError_t launch_act_quant(const Cfg& c, const void* X, int x_dtype, int64_t M, int64_t K,
                            uint8_t* Xq, float* s_a, hipStream_t st);
// Dual family: int8 A_o (Xo, s_a) and MXFP4 A_i (Xi: [M][K/2] nibbles, Ea: [M][K/32] e8m0).
hipError_t launch_act_quant_dual(const void* X, int x_dtype, int64_t M, int64_t K, uint8_t* Xo,
                                 float* s_a, uint8_t* Xi, uint8_t* Ea, hipStream_t st);
// Dual family, one or two tokens: weight-streaming vector kernel (when
// dual_decode_fits; launch_dual_mfma dispatches to it).
bool dual_decode_fits(int64_t M, int64_t N, int64_t K);
hipError_t launch_dual_decode(const Cfg& c, const uint8_t* Xo, const float* s_a, const uint8_t* Xi,
                              const uint8_t* Ea, int64_t M, const uint8_t* blob, int64_t N, int64_t K,
                              void* Y, hipStream_t st);
// Dual family, matrix-core kernel (any M): fp4 x fp4 inliers and int8 x int8 outliers.
hipError_t launch_dual_mfma(const Cfg& c, const uint8_t* Xo, const float* s_a, const uint8_t* Xi,
                            const uint8_t* Ea, int64_t M, const uint8_t* blob, int64_t N, int64_t K,
                            void* Y, hipStream_t st);

// INT family, weight-streaming vector kernel (small M).
constexpr int kDecodeMaxM = 8;
hipError_t launch_int_decode(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                             const uint8_t* blob, int64_t N, int64_t K, void* Y, hipStream_t st);
// Same kernel with the per-token activation quantization fused in front: every
// workgroup quantizes X into LDS; workgroup 0 also writes Xq and s_a.
hipError_t launch_int_decode_fused(const Cfg& c, const void* X, int x_dtype, int64_t M,
                                   uint8_t* Xq_out, float* s_a_out, const uint8_t* blob, int64_t N,
                                   int64_t K, void* Y, hipStream_t st);
// Whether the decode kernel takes M tokens of width K (it keeps them in LDS),
// and whether its fused form does.
bool decode_fits(int64_t M, int64_t K);
bool decode_fused_fits(int64_t M, int64_t K);

// INT family, matrix-core kernel (any M).
hipError_t launch_int_mfma(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                           const uint8_t* blob, int64_t N, int64_t K, void* Y, hipStream_t st);

// INT family, matrix-core kernel with K split across workgroups (tens to a
// few hundred tokens): partial sums of the K ranges in `workspace` (at least
// int_split_workspace_bytes(M, N, K) bytes, 16-byte aligned), then a second
// kernel adds them in range order and scales by s_a.
constexpr int64_t kSplitMaxM = 256;
size_t int_split_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_int_split(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                            const uint8_t* blob, int64_t N, int64_t K, void* Y, void* workspace,
                            hipStream_t st);
// Whether the split-K path takes the tiled matrix-core kernel (128-token
// blocks) over K ranges instead: partial sums in `workspace` (at least
// int_tiled_split_workspace_bytes(M, N, K) bytes), the same second kernel.
bool int_split_tiled(int64_t M, int64_t N, int64_t K);
size_t int_tiled_split_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_int_tiled_split(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                                  const uint8_t* blob, int64_t N, int64_t K, void* Y, void* workspace,
                                  hipStream_t st);

// MX family, scaled matrix-core kernel (any M).
hipError_t launch_mx_mfma(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                          const uint8_t* blob, int64_t N, int64_t K, void* Y, hipStream_t st);
// The same kernel with K split across workgroups: raw partial sums of the K
// ranges in `workspace` (mx_split_workspace_bytes(M, N, K) bytes, 16-byte
// aligned), then the split-K reduction below.
constexpr int kMxSplitMinChunks = 4;  // 128-K chunks per K range, at least
size_t mx_split_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_mx_split(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                           const uint8_t* blob, int64_t N, int64_t K, void* Y, void* workspace,
                           hipStream_t st);

// Y[m, n] = s_a[m] * (part[0][m, n] + ... + part[S-1][m, n]), the ranges added
// in order (part: [S][M][N] fp32, 16-byte aligned); fp32 or bf16 Y.
hipError_t launch_split_reduce(const float* part, const float* s_a, void* Y, int64_t M, int64_t N, int S,
                               bool y_bf16, hipStream_t st);

// MX family with outliers, two passes for many tokens: the blob is expanded
// once into dense merged fp8 fragments in `workspace` (at least
// mx_dense_workspace_bytes(N, K) bytes, 16-byte aligned), then multiplied.
constexpr int64_t kDenseMinM = 512;
size_t mx_dense_workspace_bytes(int64_t N, int64_t K);
hipError_t launch_mx_dense(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                           const uint8_t* blob, int64_t N, int64_t K, void* Y, void* workspace,
                           hipStream_t st);
// The two passes one at a time: pass 1 writes the expanded weights of the
// blob into `workspace`; pass 2 multiplies them (with the blob's scale words)
// whenever the caller orders it after pass 1.
hipError_t launch_mx_densify(const Cfg& c, const uint8_t* blob, int64_t N, int64_t K, void* workspace,
                             hipStream_t st);
hipError_t launch_mx_dense_pass(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                                const uint8_t* blob, int64_t N, int64_t K, void* Y, const void* workspace,
                                hipStream_t st);
// The same two passes with the library's static scratch array as the
// workspace (at most kStaticScratchBytes; the caller checks the size).
constexpr size_t kStaticScratchBytes = size_t(48) << 20;
hipError_t launch_mx_dense_static(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                                  const uint8_t* blob, int64_t N, int64_t K, void* Y,
                                  hipStream_t st);
// launch_int_split (INT) or launch_mx_split (MX) with the same static array
// as the workspace (the caller checks the size).
hipError_t split_static(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                        const uint8_t* blob, int64_t N, int64_t K, void* Y, hipStream_t st);

}  // namespace sdq
