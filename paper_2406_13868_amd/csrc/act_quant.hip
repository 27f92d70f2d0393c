// Per-token activation quantization (Section 5, Stage 3: activations are
// quantized to match the low-precision weights; one scale per token).
//
// For each row m of X[M, K]:
//   a = max_k |X[m,k]|,  s_a[m] = a / qmax,  inv = qmax / a   (IEEE divides)
//   Xq[m,k] = rne(X[m,k] * inv)   clamped to [-127, 127] (int8)
//                                 or saturated to +-448 (fp8 e4m3)
// A zero row gives s_a = 0 and zero codes.
//
// One workgroup of 256 threads per row.  Rows up to 16384 wide are read once
// into registers (16-byte loads), reduced through a wave butterfly and LDS,
// then quantized and written back with 8-byte stores; wider rows take a
// second pass over the (L2-resident) row.  The pass is HBM-bound: K*(in+1)
// bytes per row.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace sdq {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
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

template <bool BF16, bool E4M3, int CH>
__global__ __launch_bounds__(kThreads) void act_quant_regs(const void* __restrict__ X, int64_t K,
                                                           uint8_t* __restrict__ Xq,
                                                           float* __restrict__ s_a) {
  __shared__ float red[4];
  const int64_t m = blockIdx.x;
  const int64_t P = K >> 3;  // pieces of 8 elements
  float v[CH][8];
  float amax = 0.f;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int64_t p = threadIdx.x + c * kThreads;
    if (p < P) {
      load8<BF16>(X, m * K + p * 8, v[c]);
#pragma unroll
      for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(v[c][i]));
    }
  }
  amax = block_max(amax, red);
  const float qmax = E4M3 ? 448.f : 127.f;
  const float inv = amax > 0.f ? qmax / amax : 0.f;
  if (threadIdx.x == 0) s_a[m] = amax / qmax;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int64_t p = threadIdx.x + c * kThreads;
    if (p < P) quant_store8<E4M3>(v[c], inv, Xq + m * K + p * 8);
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
  amax = block_max(amax, red);
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
  if (pieces <= 1 * kThreads)
    hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 1>), grid, block, 0, st, X, K, Xq, s_a);
  else if (pieces <= 2 * kThreads)
    hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 2>), grid, block, 0, st, X, K, Xq, s_a);
  else if (pieces <= 4 * kThreads)
    hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 4>), grid, block, 0, st, X, K, Xq, s_a);
  else if (pieces <= 8 * kThreads)
    hipLaunchKernelGGL((act_quant_regs<BF16, E4M3, 8>), grid, block, 0, st, X, K, Xq, s_a);
  else
    hipLaunchKernelGGL((act_quant_2pass<BF16, E4M3>), grid, block, 0, st, X, K, Xq, s_a);
  return hipGetLastError();
}

}  // namespace

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
