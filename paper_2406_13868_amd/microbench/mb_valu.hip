// Microbenchmark: throughput of single VALU instruction kinds (8 independent chains per wave, 4 waves per SIMD).
// 4 waves per SIMD).  Inline asm pins the instruction; operands are plain VGPRs.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#define CK(x) do { hipError_t e = (x); if (e != hipSuccess) { printf("HIP error %s at %d\n", hipGetErrorString(e), __LINE__); exit(1);} } while (0)
#define BODY(OP)                                                                          \
  __global__ __launch_bounds__(256) void k_##OP(unsigned* out, int iters, unsigned seed) { \
    unsigned r[8], b = seed ^ threadIdx.x, c = seed * 3 + threadIdx.x;                     \
    for (int i = 0; i < 8; ++i) r[i] = seed + i * threadIdx.x;                             \
    for (int it = 0; it < iters; ++it) {                                                   \
      _Pragma("unroll") for (int i = 0; i < 8; ++i) OPASM_##OP(r[i], b, c);                \
    }                                                                                      \
    unsigned s = 0;                                                                        \
    for (int i = 0; i < 8; ++i) s ^= r[i];                                                 \
    if (s == 0x12345u) out[threadIdx.x] = s;                                               \
  }
#define OPASM_perm(d, b, c) asm volatile("v_perm_b32 %0, %0, %1, %2" : "+v"(d) : "v"(b), "v"(c))
#define OPASM_and(d, b, c) asm volatile("v_and_b32 %0, %0, %1" : "+v"(d) : "v"(b))
#define OPASM_lshl(d, b, c) asm volatile("v_lshlrev_b32 %0, %1, %0" : "+v"(d) : "v"(b))
#define OPASM_lshlor(d, b, c) asm volatile("v_lshl_or_b32 %0, %0, %1, %2" : "+v"(d) : "v"(b), "v"(c))
#define OPASM_andor(d, b, c) asm volatile("v_and_or_b32 %0, %0, %1, %2" : "+v"(d) : "v"(b), "v"(c))
#define OPASM_bfi(d, b, c) asm volatile("v_bfi_b32 %0, %0, %1, %2" : "+v"(d) : "v"(b), "v"(c))
#define OPASM_bfe(d, b, c) asm volatile("v_bfe_u32 %0, %0, %1, %2" : "+v"(d) : "v"(b), "v"(c))
#define OPASM_mul24(d, b, c) asm volatile("v_mul_u32_u24 %0, %0, %1" : "+v"(d) : "v"(b))
#define OPASM_add(d, b, c) asm volatile("v_add_u32 %0, %0, %1" : "+v"(d) : "v"(b))
#define OPASM_cnd(d, b, c) asm volatile("v_cmp_gt_u32 vcc, %0, %1\n\tv_cndmask_b32 %0, %0, %2, vcc" : "+v"(d) : "v"(b), "v"(c) : "vcc")
#define OPASM_fma(d, b, c) asm volatile("v_fma_f32 %0, %0, %1, %2" : "+v"(d) : "v"(b), "v"(c))
#define OPASM_pkfma16(d, b, c) asm volatile("v_pk_fma_f16 %0, %0, %1, %2" : "+v"(d) : "v"(b), "v"(c))
#define OPASM_dot4(d, b, c) asm volatile("v_dot4c_i32_i8 %0, %1, %2" : "+v"(d) : "v"(b), "v"(c))
#define OPASM_cvtfp8(d, b, c) asm volatile("v_cvt_f32_fp8 %0, %0" : "+v"(d))
#define OPASM_bitop3(d, b, c) asm volatile("v_bitop3_b32 %0, %0, %1, %2 bitop3:0x96" : "+v"(d) : "v"(b), "v"(c))
#define OPASM_xor(d, b, c) asm volatile("v_xor_b32 %0, %0, %1" : "+v"(d) : "v"(b))
#define OPASM_mov(d, b, c) asm volatile("v_mov_b32 %0, %1" : "=v"(d) : "v"(b))
BODY(perm) BODY(and) BODY(lshl) BODY(lshlor) BODY(andor) BODY(bfi) BODY(bfe) BODY(mul24) BODY(add)
BODY(cnd) BODY(fma) BODY(pkfma16) BODY(dot4) BODY(cvtfp8) BODY(bitop3) BODY(xor) BODY(mov)
int main() {
  unsigned* out; CK(hipMalloc(&out, 1024 * 4));
  hipEvent_t e0, e1; CK(hipEventCreate(&e0)); CK(hipEventCreate(&e1));
  const int iters = 4000, blocks = 1024;  // 4 waves per SIMD
  auto run = [&](const char* nm, auto kern, int per) {
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), 0, 0, out, 10, 3u);
    CK(hipDeviceSynchronize());
    CK(hipEventRecord(e0)); hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), 0, 0, out, iters, 3u); CK(hipEventRecord(e1));
    CK(hipEventSynchronize(e1)); float ms; CK(hipEventElapsedTime(&ms, e0, e1));
    const double ops_per_simd = double(blocks) * 4 / 1024 * iters * 8 * per;
    printf("%-10s %8.3f ms  %5.2f cycles per wave-op @2.4GHz\n", nm, ms, ms * 1e-3 * 2.4e9 / ops_per_simd);
    fflush(stdout);
  };
  run("perm", k_perm, 1); run("and", k_and, 1); run("lshl", k_lshl, 1); run("lshl_or", k_lshlor, 1);
  run("and_or", k_andor, 1); run("bfi", k_bfi, 1); run("bfe", k_bfe, 1); run("mul24", k_mul24, 1);
  run("add", k_add, 1); run("cmp+cnd", k_cnd, 2); run("fma_f32", k_fma, 1); run("pk_fma_f16", k_pkfma16, 1);
  run("dot4c", k_dot4, 1); run("cvt_fp8", k_cvtfp8, 1); run("bitop3", k_bitop3, 1); run("xor", k_xor, 1); run("mov", k_mov, 1);
  printf("mb done\n");
  return 0;
}
