// Per-token activation quantization (Section 5, Stage 3: activations are
// quantized to match the low-precision weights; one scale per token).
//
// For each row m of X[M, K]:
//   a = max_k |X[m,k]|,  s_a[m] = a / qmax,  inv = qmax / a   (IEEE divides)
//   Xq[m,k] = rne(X[m,k] * inv)   clamped to [-127, 127] (int8)
//                                 or saturated to +-448 (fp8 e4m3)
// A zero row gives s_a = 0 and zero codes.
//
// One workgroup per row: 256 threads, or 512 / 1024 when there are few rows
// and they are 2K..8K / wider (so that the few compute units busy keep more
// loads in flight).  Rows up to 8 pieces of 8 elements per thread are read once
// into registers (16-byte loads), reduced by a DPP/permlane wave maximum and
// LDS, then quantized and written back with 8-byte stores; wider rows take a
// second pass over the (L2-resident) row.  The pass is HBM-bound: K*(in+1)
// bytes per row.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace sdq {
namespace {

constexpr int kThreads = 256;

// Maximum over the 64 lanes of a wave: DPP row rotations by 1, 2, 4 and 8
// inside each row of 16 lanes, then the permlane swaps across rows.
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x121, 0xF, 0xF, false)));
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x122, 0xF, 0xF, false)));
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x124, 0xF, 0xF, false)));
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x128, 0xF, 0xF, false)));
  const auto p16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(p16[0]), __uint_as_float(p16[1]));
  const auto p32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(p32[0]), __uint_as_float(p32[1]));
}

// Maximum over a workgroup of NT threads (red: NT / 64 floats of LDS).
template <int NT>
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < NT / 64; ++i) r = fmaxf(r, red[i]);
  return r;
}

// Eight consecutive elements, widened to fp32.
template <bool BF16>
__device__ __forceinline__ void load8(const void* X, int64_t idx, float (&v)[8]) {
  if constexpr (BF16) {
    const uint4 raw = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(X) + idx);
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  } else {
    const float4 a = *reinterpret_cast<const float4*>(static_cast<const float*>(X) + idx);
    const float4 b = *reinterpret_cast<const float4*>(static_cast<const float*>(X) + idx + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

// Quantizes eight values scaled by inv and stores them as eight bytes.
template <bool E4M3>
__device__ __forceinline__ void quant_store8(const float (&v)[8], float inv, uint8_t* dst) {
  uint32_t lo = 0, hi = 0;
  if constexpr (E4M3) {
    float t[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) t[i] = fminf(fmaxf(v[i] * inv, -448.f), 448.f);
    // v_cvt_pk_fp8_f32: OCP e4m3, round to nearest even
    lo = __builtin_amdgcn_cvt_pk_fp8_f32(t[0], t[1], 0, false);
    lo = __builtin_amdgcn_cvt_pk_fp8_f32(t[2], t[3], lo, true);
    hi = __builtin_amdgcn_cvt_pk_fp8_f32(t[4], t[5], 0, false);
    hi = __builtin_amdgcn_cvt_pk_fp8_f32(t[6], t[7], hi, true);
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float r = rintf(v[i] * inv);  // one fp32 multiply, then round half to even
      const int q = (int)fminf(fmaxf(r, -127.f), 127.f);
      const uint32_t b = uint32_t(q) & 0xFFu;
      if (i < 4) lo |= b << (8 * i);
      else hi |= b << (8 * (i - 4));
    }
  }
  *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
}

// Eight consecutive elements as loaded (16 bytes of bf16 or 32 of fp32); a
// bf16 row is kept in this form between its two uses, which halves the
// registers of the widest rows (more rows in flight per compute unit).
template <bool BF16>
struct Raw8 {
  uint4 q[BF16 ? 1 : 2];
};
template <bool BF16>
__device__ __forceinline__ void load_raw8(const void* X, int64_t idx, Raw8<BF16>& r) {
  if constexpr (BF16) {
    r.q[0] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(X) + idx);
  } else {
    r.q[0] = *reinterpret_cast<const uint4*>(static_cast<const float*>(X) + idx);
    r.q[1] = *reinterpret_cast<const uint4*>(static_cast<const float*>(X) + idx + 4);
  }
}
template <bool BF16>
__device__ __forceinline__ void widen8(const Raw8<BF16>& r, float (&v)[8]) {
  if constexpr (BF16) {
    const uint32_t w[4] = {r.q[0].x, r.q[0].y, r.q[0].z, r.q[0].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      v[4 * h] = __uint_as_float(r.q[h].x); v[4 * h + 1] = __uint_as_float(r.q[h].y);
      v[4 * h + 2] = __uint_as_float(r.q[h].z); v[4 * h + 3] = __uint_as_float(r.q[h].w);
    }
  }
}

template <bool BF16, bool E4M3, int CH, int NT>
__global__ __launch_bounds__(NT) void act_quant_regs(const void* __restrict__ X, int64_t K,
                                                     uint8_t* __restrict__ Xq,
                                                     float* __restrict__ s_a) {
  __shared__ float red[NT / 64];
  const int64_t m = blockIdx.x;
  const int64_t P = K >> 3;  // pieces of 8 elements
  Raw8<BF16> r[CH];
  float amax = 0.f;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int64_t p = threadIdx.x + c * NT;
    if (p < P) load_raw8<BF16>(X, m * K + p * 8, r[c]);
  }
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int64_t p = threadIdx.x + c * NT;
    if (p < P) {
      float v[8];
      widen8<BF16>(r[c], v);
#pragma unroll
      for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(v[i]));
    }
  }
  amax = block_max<NT>(amax, red);
  const float qmax = E4M3 ? 448.f : 127.f;
  const float inv = amax > 0.f ? qmax / amax : 0.f;
  if (threadIdx.x == 0) s_a[m] = amax / qmax;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int64_t p = threadIdx.x + c * NT;
    if (p < P) {
      float v[8];
      widen8<BF16>(r[c], v);
      quant_store8<E4M3>(v, inv, Xq + m * K + p * 8);
    }
  }
}

template <bool BF16, bool E4M3>
__global__ __launch_bounds__(kThreads) void act_quant_2pass(const void* __restrict__ X, int64_t K,
                                                            uint8_t* __restrict__ Xq,
                                                            float* __restrict__ s_a) {
  __shared__ float red[4];
  const int64_t m = blockIdx.x;
  const int64_t P = K >> 3;
  float amax = 0.f;
  for (int64_t p = threadIdx.x; p < P; p += kThreads) {
    float v[8];
    load8<BF16>(X, m * K + p * 8, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(v[i]));
  }
  amax = block_max<kThreads>(amax, red);
  const float qmax = E4M3 ? 448.f : 127.f;
  const float inv = amax > 0.f ? qmax / amax : 0.f;
  if (threadIdx.x == 0) s_a[m] = amax / qmax;
  for (int64_t p = threadIdx.x; p < P; p += kThreads) {
    float v[8];
    load8<BF16>(X, m * K + p * 8, v);
    quant_store8<E4M3>(v, inv, Xq + m * K + p * 8);
  }
}

template <bool BF16, bool E4M3>
hipError_t launch_typed(const void* X, int64_t M, int64_t K, uint8_t* Xq, float* s_a,
                        hipStream_t st) {
  const dim3 grid(static_cast<unsigned>(M)), block(kThreads);
  const int64_t pieces = K / 8;
  // few wide rows: 1024 threads per row
  if (M < 256 && pieces > 1024 && pieces <= 4096 * 2) {
    const dim3 big(1024);
    if (pieces <= 1024 * 2)
      hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 2, 1024>), grid, big, 0, st, X, K, Xq, s_a);
    else if (pieces <= 1024 * 4)
      hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 4, 1024>), grid, big, 0, st, X, K, Xq, s_a);
    else
      hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 8, 1024>), grid, big, 0, st, X, K, Xq, s_a);
    return hipGetLastError();
  }
  if (M < 256 && pieces > kThreads && pieces <= 1024) {  // few rows of 2K..8K elements: 512 threads per row
    const dim3 mid(512);
    if (pieces <= 512)
      hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 1, 512>), grid, mid, 0, st, X, K, Xq, s_a);
    else
      hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 2, 512>), grid, mid, 0, st, X, K, Xq, s_a);
    return hipGetLastError();
  }
  if (pieces <= 1 * kThreads)
    hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 1, kThreads>), grid, block, 0, st, X, K, Xq, s_a);
  else if (pieces <= 2 * kThreads)
    hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 2, kThreads>), grid, block, 0, st, X, K, Xq, s_a);
  else if (pieces <= 4 * kThreads)
    hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 4, kThreads>), grid, block, 0, st, X, K, Xq, s_a);
  else if (pieces <= 8 * kThreads)
    hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 8, kThreads>), grid, block, 0, st, X, K, Xq, s_a);
  else
    hipLaunchKernelGGL((act_quant_2pass<BF16, E4M3>), grid, block, 0, st, X, K, Xq, s_a);
  return hipGetLastError();
}

// ---- the dual family's two activation tensors (Section 5.1: int8 A_o for
//      the outliers, fp4 A_i for the inliers).  A_o as above (int8, one fp32
//      scale per token); A_i is MXFP4: per token and 32-K block, E =
//      floor(log2 amax) - 2 clamped to [-127, 127] (an all-zero block: E =
//      -127 and zero codes), codes e2m1(x * 2^-E) to nearest even, saturating
//      at 6, with the sign of x; two codes per byte, the even k in the low
//      nibble, and one e8m0 byte E + 127 per block.

// e2m1 code (sign in bit 3) of t, nearest even: the tie points 0.25, 1.25, 2.5
// and 5 stay on the lower (even) code, 0.75, 1.75 and 3.5 go to the upper one.
__device__ __forceinline__ uint32_t e2m1_rne(float t) {
  const float a = fabsf(t);
  const uint32_t mag = uint32_t(a > 0.25f) + uint32_t(a >= 0.75f) + uint32_t(a > 1.25f) +
                       uint32_t(a >= 1.75f) + uint32_t(a > 2.5f) + uint32_t(a >= 3.5f) + uint32_t(a > 5.f);
  return mag | ((__float_as_uint(t) >> 28) & 8u);
}

// One workgroup of NT threads per token, two passes over the row (the
// second from L2): the row amax, then per 8-element piece the int8 codes, the
// block amax of the four pieces of its 32-K block (lanes 4j..4j+3 of a wave),
// and the fp4 codes.
template <bool BF16, int NT>
__global__ __launch_bounds__(NT) void act_quant_dual(const void* __restrict__ X, int64_t K,
                                                     uint8_t* __restrict__ Xo, float* __restrict__ s_a,
                                                     uint8_t* __restrict__ Xi, uint8_t* __restrict__ Ea) {
  __shared__ float red[NT / 64];
  const int64_t m = blockIdx.x;
  const int64_t P = K >> 3;  // pieces of 8 elements, a multiple of 4 (K a multiple of 32)
  float amax = 0.f;
  for (int64_t p = threadIdx.x; p < P; p += NT) {
    float v[8];
    load8<BF16>(X, m * K + p * 8, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(v[i]));
  }
  amax = block_max<NT>(amax, red);
  const float inv = amax > 0.f ? 127.f / amax : 0.f;
  if (threadIdx.x == 0) s_a[m] = amax / 127.f;
  for (int64_t base = 0; base < P; base += NT) {  // the same trip count for every lane
    const int64_t p = base + threadIdx.x;
    const bool ok = p < P;
    float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (ok) load8<BF16>(X, m * K + p * 8, v);
    float bm = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) bm = fmaxf(bm, fabsf(v[i]));
    bm = fmaxf(bm, __shfl_xor(bm, 1, 64));
    bm = fmaxf(bm, __shfl_xor(bm, 2, 64));
    const int E = bm > 0.f ? min(max(__builtin_amdgcn_frexp_expf(bm) - 1 - 2, -127), 127) : -127;
    if (!ok) continue;
    quant_store8<false>(v, inv, Xo + m * K + p * 8);
    uint32_t q = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) q |= (bm > 0.f ? e2m1_rne(ldexpf(v[i], -E)) : 0u) << (4 * i);
    *reinterpret_cast<uint32_t*>(Xi + m * (K / 2) + p * 4) = q;
    if ((p & 3) == 0) Ea[m * (K / 32) + (p >> 2)] = uint8_t(E + 127);
  }
}

}  // namespace

hipError_t launch_act_quant_dual(const void* X, int x_dtype, int64_t M, int64_t K, uint8_t* Xo,
                                 float* s_a, uint8_t* Xi, uint8_t* Ea, hipStream_t st) {
  // few tokens: more threads per token (measured at M = 1: one 256-thread
  // workgroup takes about 5 us on a 4096..11008-wide row)
  const dim3 grid(static_cast<unsigned>(M));
  const int64_t P = K / 8;
  const bool bf16 = x_dtype == SDQ_DTYPE_BF16;
  if (M < 256 && P >= 1024) {
    if (bf16) hipLaunchKernelGGL((act_quant_dual<true, 1024>), grid, dim3(1024), 0, st, X, K, Xo, s_a, Xi, Ea);
    else hipLaunchKernelGGL((act_quant_dual<false, 1024>), grid, dim3(1024), 0, st, X, K, Xo, s_a, Xi, Ea);
  } else if (M < 256 && P >= 512) {
    if (bf16) hipLaunchKernelGGL((act_quant_dual<true, 512>), grid, dim3(512), 0, st, X, K, Xo, s_a, Xi, Ea);
    else hipLaunchKernelGGL((act_quant_dual<false, 512>), grid, dim3(512), 0, st, X, K, Xo, s_a, Xi, Ea);
  } else {
    if (bf16) hipLaunchKernelGGL((act_quant_dual<true, kThreads>), grid, dim3(kThreads), 0, st, X, K, Xo, s_a, Xi, Ea);
    else hipLaunchKernelGGL((act_quant_dual<false, kThreads>), grid, dim3(kThreads), 0, st, X, K, Xo, s_a, Xi, Ea);
  }
  return hipGetLastError();
}

hipError_t launch_act_quant(const Cfg& c, const void* X, int x_dtype, int64_t M, int64_t K,
                            uint8_t* Xq, float* s_a, hipStream_t st) {
  const bool bf16 = x_dtype == SDQ_DTYPE_BF16;
  const bool e4m3 = c.fmt_a == SDQ_FMT_E4M3;
  if (bf16 && e4m3) return launch_typed<true, true>(X, M, K, Xq, s_a, st);
  if (bf16) return launch_typed<true, false>(X, M, K, Xq, s_a, st);
  if (e4m3) return launch_typed<false, true>(X, M, K, Xq, s_a, st);
  return launch_typed<false, false>(X, M, K, Xq, s_a, st);
}

}  // namespace sdq
