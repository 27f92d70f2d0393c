// Output of a wave's 32x32 fp32 accumulator tiles: Y[m, n] = s_a[m] * acc,
// Y row-major [M, N], stored as fp32 or rounded to bf16 (the last step of
// Section 5.1's product).
//
// The 32x32 matrix instructions leave element e of a tile in lane
// l = 32h + col at row 8*(e/4) + 4*h + e%4 and column col.
//
// Loads and stores go through buffer resources over the rows of the
// workgroup's token block that exist (rows past M read 0 and their stores are
// dropped), so that no output needs a branch of its own.  Every row scale is
// read before the first store: the compiler cannot tell that Y and s_a do not
// overlap, so a scale read after a store would stay behind it, and the memory
// counter that read waits on also counts the store -- each output would cost
// a full store round trip.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace sdq {

// Buffer resource over [p, p + bytes): a wave-uniform base in scalar
// registers and a 32-bit offset per lane; accesses past the end read 0 and
// write nothing.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), short(0), int(bytes), 0x00020000);
}

// Row r of element e of a 32x32 tile, for lane half h.
__device__ __forceinline__ int tile_row(int e, int h) { return 8 * (e >> 2) + 4 * h + (e & 3); }

template <int MS>
struct RowScales {
  float v[MS][16];
};

// s_a of the rows of MS tiles of 32 tokens from m0 (0 past M), lane half h.
template <int MS>
__device__ __forceinline__ RowScales<MS> load_row_scales(const float* s_a, int M, int m0, int h) {
  const __amdgpu_buffer_rsrc_t r = buffer_rsrc(s_a + m0, uint32_t(min(M - m0, 32 * MS)) * 4u);
  RowScales<MS> s;
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e)
      s.v[ms][e] = __uint_as_float(
          __builtin_amdgcn_raw_buffer_load_b32(r, uint32_t(ms * 32 + tile_row(e, h)) * 4u, 0, 0));
  return s;
}

// bf16 bits of v, rounded to nearest even (NaN stays NaN).
__device__ __forceinline__ unsigned short bf16_bits(float v) {
  return __builtin_bit_cast(unsigned short, static_cast<__bf16>(v));
}

// Rows [m0, m0 + rows) of Y that exist, with fp32 or bf16 elements (a
// wave-uniform choice).  N * rows * 4 < 2^32 (the shape checks bound N).
struct OutRows {
  __amdgpu_buffer_rsrc_t r;
  bool bf16;
};
__device__ __forceinline__ OutRows out_rows(void* Y, bool bf16, int M, int N, int m0, int rows) {
  const uint32_t es = bf16 ? 2u : 4u;
  return {buffer_rsrc(static_cast<uint8_t*>(Y) + size_t(m0) * size_t(N) * es,
                      uint32_t(min(M - m0, rows)) * uint32_t(N) * es),
          bf16};
}

// Y[m0 + ms*32 + row(e), n] = v through the resource of out_rows.
__device__ __forceinline__ void store_out(const OutRows& y, int N, int n, int ms, int e, int h, float v) {
  const uint32_t idx = uint32_t(ms * 32 + tile_row(e, h)) * uint32_t(N) + uint32_t(n);
  if (y.bf16)
    __builtin_amdgcn_raw_buffer_store_b16(bf16_bits(v), y.r, idx * 2u, 0, 0);
  else
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), y.r, idx * 4u, 0, 0);
}

// Y[i] = v for a plain element index (fp32 or bf16 elements).
__device__ __forceinline__ void store_y(void* Y, bool bf16, size_t i, float v) {
  if (bf16)
    static_cast<unsigned short*>(Y)[i] = bf16_bits(v);
  else
    static_cast<float*>(Y)[i] = v;
}

}  // namespace sdq
