// LDS read throughput on gfx950: ds_read_b128, conflict-free (lane i reads 16 B at i*16 + k*1024).
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#define CK(x) do { hipError_t e = (x); if (e != hipSuccess) { printf("HIP error %s at %d\n", hipGetErrorString(e), __LINE__); exit(1);} } while (0)
template <int WAVES>
__global__ __launch_bounds__(WAVES * 64) void k(unsigned* out, int iters) {
  __shared__ __align__(16) uint4 buf[4096];  // 64 KB
  for (int i = threadIdx.x; i < 4096; i += blockDim.x) buf[i] = make_uint4(i, i * 3, i ^ 5, i + 7);
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint4 acc = make_uint4(0, 0, 0, 0);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint4 v = buf[((it * 8 + j + wave) & 63) * 64 + lane];
      acc.x ^= v.x; acc.y += v.y; acc.z ^= v.z; acc.w += v.w;
    }
  }
  if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x1234567u) out[threadIdx.x] = acc.x;
}
int main() {
  unsigned* out; CK(hipMalloc(&out, 4096 * 4));
  hipEvent_t e0, e1; CK(hipEventCreate(&e0)); CK(hipEventCreate(&e1));
  const int iters = 2000;
  auto run = [&](const char* nm, auto kern, int waves, int blocks_per_cu) {
    const int blocks = 256 * blocks_per_cu;
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(waves * 64), 0, 0, out, 10);
    CK(hipDeviceSynchronize());
    CK(hipEventRecord(e0)); hipLaunchKernelGGL(kern, dim3(blocks), dim3(waves * 64), 0, 0, out, iters); CK(hipEventRecord(e1));
    CK(hipEventSynchronize(e1)); float ms; CK(hipEventElapsedTime(&ms, e0, e1));
    const double bytes_per_cu = double(blocks_per_cu) * waves * 64 * 16.0 * 8 * iters;
    printf("%-30s %8.3f ms  %6.1f B/clk/CU @2.4GHz\n", nm, ms, bytes_per_cu / (ms * 1e-3 * 2.4e9));
    fflush(stdout);
  };
  run("4 waves x 1 block/CU", k<4>, 4, 1);
  run("8 waves x 1 block/CU", k<8>, 8, 1);
  run("4 waves x 2 blocks/CU", k<4>, 4, 2);
  run("16 waves x 1 block/CU", k<16>, 16, 1);
  printf("mb done\n");
  return 0;
}
