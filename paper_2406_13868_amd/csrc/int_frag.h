// Weight and activation fragments of the INT-family matrix-core kernels
// (f16 and int8 matrix instructions), shared by the kernels of
// gemm_int_mfma.hip and gemm_int_split.hip.  Section 5.1: the inlier branch
// (int4 codes times an inlier scale per Q-Vector) and the outlier branch
// (int8 or e4m3 codes, one per group) of one group word become dense
// fragments of the dense product.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace sdq {
namespace intfrag {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

constexpr uint32_t kOutPosMagic = (1u << 21) | (1u << 14) | (1u << 7);

// Inlier scale formats of the INT family (template parameter SF).
enum ScaleFmt { kScaleF16 = 0, kScaleE4M3 = 1, kScaleE6M2 = 2 };

// The fp16 inlier scale of 16-K block kb (its scale kb >> qs) from a row's
// scale registers sv: fp16 pairs (two per dword), or one code per byte (four
// per dword): e4m3 (every value is an fp16 value) or ufp8-e6m2, whose values
// (4 + m) * 2^(e - 33) the packer keeps within [2^-22, 7168], where they and
// their products with an int4 code are exact in fp16.
template <int SF>
__device__ __forceinline__ _Float16 block_scale(const uint32_t* sv, int kb, int qs) {
  const int e = kb >> qs;
  if constexpr (SF == kScaleF16) {
    const uint32_t sw = sv[e >> 1];
    return __builtin_bit_cast(_Float16, (unsigned short)((e & 1) ? (sw >> 16) : (sw & 0xFFFFu)));
  } else {
    const uint32_t byte = (sv[e >> 2] >> (8 * (e & 3))) & 0xFFu;
    if constexpr (SF == kScaleE4M3) {
      return (_Float16)__builtin_amdgcn_cvt_f32_fp8(int(byte), 0);
    } else {
      const uint32_t ex = byte >> 2, m = byte & 3u;
      const float v = ex ? float(4u + m) * __uint_as_float((ex + 94u) << 23) : 0.f;  // code 0: scale 0
      return (_Float16)v;
    }
  }
}

// A row's inlier scales of one chunk (srow = 16, 8, 4 or 2 bytes, naturally
// aligned), into the low end of four dwords.
__device__ __forceinline__ uint4 load_row_scales_chunk(const uint8_t* p, int srow) {
  if (srow == 16) return *reinterpret_cast<const uint4*>(p);
  if (srow == 8) { const uint2 v = *reinterpret_cast<const uint2*>(p); return make_uint4(v.x, v.y, 0, 0); }
  if (srow == 4) return make_uint4(*reinterpret_cast<const uint32_t*>(p), 0, 0, 0);
  return make_uint4(*reinterpret_cast<const uint16_t*>(p), 0, 0, 0);
}

// Four int8 -> four f16 (two dwords), exact: f16(1024 + (b ^ 0x80)) - 1152 = b.
__device__ __forceinline__ void i8x4_to_f16x4(uint32_t x, uint32_t& lo, uint32_t& hi) {
  const uint32_t xb = x ^ 0x80808080u;
  const uint32_t a = __builtin_amdgcn_perm(0x64646464u, xb, 0x04010400u);
  const uint32_t b = __builtin_amdgcn_perm(0x64646464u, xb, 0x04030402u);
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  const h2 bias = {(_Float16)-1152.0f, (_Float16)-1152.0f};
  lo = __builtin_bit_cast(uint32_t, __builtin_bit_cast(h2, a) + bias);
  hi = __builtin_bit_cast(uint32_t, __builtin_bit_cast(h2, b) + bias);
}

// Dense fp16 inlier fragment of one group word: element p = int4 code at
// position p (0 where the group has no inlier).  The codes are first placed
// as nibbles of one dword at their positions: byte j of the word holds slot
// j's position in bits 0-2, so (w << 2) & 0x1C1C1C holds each slot's shift
// 4 * position in a byte of its own, and a shift takes only the low five bits
// of its amount.  The biased nibbles q + 8 then become fp16 1024 + q + 8
// (0x6400 | nibble) and one packed add of -1032 gives q, two elements at a time.
template <int NI>
__device__ __forceinline__ h8 inlier_f16(uint32_t w) {
  uint32_t p4 = (w << 2) & 0x001C1C1Cu;
  // opaque, so that the shifts below take p4's bytes as they are (a shift
  // reads the low five bits of its amount) instead of re-deriving them from w
  asm("" : "+v"(p4));
  uint32_t D = __builtin_amdgcn_ubfe(w, 4, 4) << p4;
  if constexpr (NI > 1) D |= __builtin_amdgcn_ubfe(w, 12, 4) << (p4 >> 8);
  if constexpr (NI > 2) D |= __builtin_amdgcn_ubfe(w, 20, 4) << (p4 >> 16);
  const uint32_t Db = D ^ 0x88888888u;  // biased nibbles q + 8
  const uint32_t Ds = Db >> 4;
  // the two constants of the and-or in registers: a three-operand
  // instruction takes no literal on this target, so with literals it would
  // be two instructions
  uint32_t lo_mask = 0x000F000Fu, f16_top = 0x64006400u;
  asm("" : "+s"(lo_mask), "+v"(f16_top));
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  const h2 bias = {(_Float16)-1032.0f, (_Float16)-1032.0f};
  u4v out;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const uint32_t sel = uint32_t(v) | 0x0C00u | (uint32_t(4 + v) << 16) | 0x0C000000u;
    const uint32_t t = (__builtin_amdgcn_perm(Ds, Db, sel) & lo_mask) | f16_top;
    out[v] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(h2, t) + bias);
  }
  return __builtin_bit_cast(h8, out);
}

// Exact split of the scaled inlier fragment q * s (q an int4 code, s the
// block's fp16 scale) into two fp16 fragments: hi = f16(q*s) and the residual
// lo = q*s - hi, which one fused multiply-add produces exactly (q*s has at
// most 14 significant bits and is a multiple of the lowest bit of s, so the
// residual is an fp16 number).  Two MFMAs on hi and lo then add q*s*a
// exactly into the fp32 accumulator, with no per-block scaling of partials.
__device__ __forceinline__ void scaled_hi_lo(h8 q, _Float16 s, h8& hi, h8& lo) {
  const h8 sv = {s, s, s, s, s, s, s, s};
  hi = q * sv;
  lo = __builtin_elementwise_fma(q, sv, -hi);
}

// Dense fp16 outlier fragment of one group word (one non-zero at most).  The
// position bits gather as in outlier_i8, here into 16 * position (bits 20-23
// of the product are zero too); one 64-bit shift places the fp16 value in
// its half of the fragment and the position's top bit picks the half.
template <bool OUT_INT8>
__device__ __forceinline__ h8 outlier_f16(uint32_t w) {
  float f;
  if constexpr (OUT_INT8) f = (float)(int(w) >> 24);
  else f = __builtin_amdgcn_cvt_f32_fp8(int(w), 3);
  const uint32_t hb = uint32_t(__builtin_bit_cast(unsigned short, (_Float16)f));
  const uint32_t p16 = __builtin_amdgcn_ubfe(__umul24(w & 0x00080808u, kOutPosMagic), 20, 7);
  const uint64_t v = uint64_t(hb) << (p16 & 63u);
  const bool upper = (p16 & 64u) != 0;
  const uint32_t vlo = uint32_t(v), vhi = uint32_t(v >> 32);
  const u4v out = {upper ? 0u : vlo, upper ? 0u : vhi, upper ? vlo : 0u, upper ? vhi : 0u};
  return __builtin_bit_cast(h8, out);
}

// Dense int8 outlier bytes of one group word (position p at byte p of lo:hi).
// The outlier's position bits (bit 3 of bytes 0-2) gather into bits 24-26 of
// one 24-bit product, whose bits 21-23 are zero, so one field extract gives
// 8 * position; a 64-bit shift then places the code byte.
__device__ __forceinline__ void outlier_i8(uint32_t w, uint32_t& lo, uint32_t& hi) {
  const uint32_t p8 = __builtin_amdgcn_ubfe(__umul24(w & 0x00080808u, kOutPosMagic), 21, 6);
  const uint64_t v = uint64_t(w >> 24) << p8;
  lo = uint32_t(v);
  hi = uint32_t(v >> 32);
}

}  // namespace intfrag
}  // namespace sdq
