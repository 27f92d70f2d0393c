// Microbenchmark: issue rate of the matrix instructions used by libsdq (no memory traffic in the loop).
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#define CK(x) do { hipError_t e = (x); if (e != hipSuccess) { printf("HIP error %s at %d\n", hipGetErrorString(e), __LINE__); exit(1);} } while (0)
typedef int i8v __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));

template <int FA, int FB, int NACC>
__global__ __launch_bounds__(256) void k_scale(float* out, int iters, int seed) {
  i8v a, b;
  for (int i = 0; i < 8; ++i) { a[i] = seed * (threadIdx.x + i); b[i] = seed ^ (threadIdx.x * 7 + i); }
  f16v acc[NACC];
  for (int j = 0; j < NACC; ++j) for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < NACC; ++j)
      acc[j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc[j], FA, FB, 0, 127, 0, 127);
  }
  float s = 0.f;
  for (int j = 0; j < NACC; ++j) for (int e = 0; e < 16; ++e) s += acc[j][e];
  if (s == 1234.5f) out[threadIdx.x] = s;
}
template <int NACC>
__global__ __launch_bounds__(256) void k_f16(float* out, int iters, int seed) {
  h8 a, b;
  for (int i = 0; i < 8; ++i) { a[i] = (_Float16)(seed * (threadIdx.x + i) & 7); b[i] = (_Float16)((seed ^ i) & 7); }
  f16v acc[NACC];
  for (int j = 0; j < NACC; ++j) for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < NACC; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[j], 0, 0, 0);
  }
  float s = 0.f;
  for (int j = 0; j < NACC; ++j) for (int e = 0; e < 16; ++e) s += acc[j][e];
  if (s == 1234.5f) out[threadIdx.x] = s;
}
typedef int i4v __attribute__((ext_vector_type(4)));
typedef int i16v __attribute__((ext_vector_type(16)));
template <int NACC>
__global__ __launch_bounds__(256) void k_i8(float* out, int iters, int seed) {
  i4v a, b;
  for (int i = 0; i < 4; ++i) { a[i] = seed * (threadIdx.x + i); b[i] = seed ^ (threadIdx.x * 7 + i); }
  i16v acc[NACC];
  for (int j = 0; j < NACC; ++j) for (int e = 0; e < 16; ++e) acc[j][e] = 0;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < NACC; ++j) acc[j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc[j], 0, 0, 0);
  }
  int s = 0;
  for (int j = 0; j < NACC; ++j) for (int e = 0; e < 16; ++e) s += acc[j][e];
  if (s == 12345) out[threadIdx.x] = float(s);
}
// the dual GEMM's mix per 64 K: one scaled fp4 x fp4 and two int8 32x32x32, on NACC
// accumulator pairs (counted as 3 instructions per pair and iteration)
template <int NACC>
__global__ __launch_bounds__(256) void k_dual(float* out, int iters, int seed) {
  i8v a, b;
  i4v c, d;
  for (int i = 0; i < 8; ++i) { a[i] = seed * (threadIdx.x + i); b[i] = seed ^ (threadIdx.x * 7 + i); }
  for (int i = 0; i < 4; ++i) { c[i] = a[i] + 1; d[i] = b[i] + 3; }
  f16v acc[NACC];
  i16v acco[NACC];
  for (int j = 0; j < NACC; ++j) for (int e = 0; e < 16; ++e) { acc[j][e] = 0.f; acco[j][e] = 0; }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < NACC; ++j) {
      acc[j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc[j], 4, 4, 0, 127, 0, 127);
      acco[j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(c, d, acco[j], 0, 0, 0);
      acco[j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(d, c, acco[j], 0, 0, 0);
    }
  }
  float s = 0.f;
  for (int j = 0; j < NACC; ++j) for (int e = 0; e < 16; ++e) s += acc[j][e] + float(acco[j][e]);
  if (s == 1234.5f) out[threadIdx.x] = s;
}
int main() {
  float* out; CK(hipMalloc(&out, 1024 * 4));
  hipEvent_t e0, e1; CK(hipEventCreate(&e0)); CK(hipEventCreate(&e1));
  const int iters = 2000;
  auto run = [&](const char* nm, auto kern, int blocks, int nacc) {
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), 0, 0, out, 10, 3);
    CK(hipDeviceSynchronize());
    CK(hipEventRecord(e0)); hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), 0, 0, out, iters, 3); CK(hipEventRecord(e1));
    CK(hipEventSynchronize(e1)); float ms; CK(hipEventElapsedTime(&ms, e0, e1));
    const double mfmas_per_simd = double(blocks) * 4 / 1024.0 * iters * nacc;  // 4 waves per block, 1024 SIMDs
    printf("%-34s blocks %5d  %8.3f ms  %6.1f cycles/MFMA/SIMD @2.4GHz\n", nm, blocks, ms, ms * 1e-3 * 2.4e9 / mfmas_per_simd);
    fflush(stdout);
  };
  for (int blocks : {256, 512}) {
    run("scale fp8 x fp8, 4 acc", k_scale<0, 0, 4>, blocks, 4);
    run("scale fp8 x fp4, 4 acc", k_scale<0, 4, 4>, blocks, 4);
    run("scale fp4 x fp4, 4 acc", k_scale<4, 4, 4>, blocks, 4);
    run("scale fp8 x fp8, 8 acc", k_scale<0, 0, 8>, blocks, 8);
    run("f16 32x32x16, 4 acc", k_f16<4>, blocks, 4);
    run("f16 32x32x16, 8 acc", k_f16<8>, blocks, 8);
    run("i8 32x32x32, 4 acc", k_i8<4>, blocks, 4);
    run("i8 32x32x32, 8 acc", k_i8<8>, blocks, 8);
    run("dual mix (fp4 + 2 i8), 4 pairs", k_dual<4>, blocks, 12);
  }
  printf("mb done\n");
  return 0;
}
