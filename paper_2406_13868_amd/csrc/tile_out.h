// Output of a wave's 32x32 fp32 accumulator tiles: Y[m, n] = s_a[m] * acc,
// Y row-major [M, N] (the last step of Section 5.1's product).
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

// Rows [m0, m0 + rows) of Y that exist.  N * rows * 4 < 2^32 (the shape
// checks bound N).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t out_rows(float* Y, int M, int N, int m0, int rows) {
  return buffer_rsrc(Y + size_t(m0) * N, uint32_t(min(M - m0, rows)) * uint32_t(N) * 4u);
}

// Y[m0 + ms*32 + row(e), n] = v through the resource of out_rows.
__device__ __forceinline__ void store_out(__amdgpu_buffer_rsrc_t y, int N, int n, int ms, int e, int h,
                                          float v) {
  const uint32_t off = (uint32_t(ms * 32 + tile_row(e, h)) * uint32_t(N) + uint32_t(n)) * 4u;
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), y, off, 0, 0);
}

}  // namespace sdq
