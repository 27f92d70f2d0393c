// MX-family weight fragments for gfx950's scaled matrix instruction
// v_mfma_scale_f32_32x32x64_f8f6f4: the packed group words of one 32-column
// row tile (layout.h) expanded into the fp8 / fp4 B operands, shared by the
// one-pass kernel (expansion in registers) and the two-pass kernel (expansion
// into a dense workspace).
//
// Operand layouts (32x32x64, lane l, lane half h = l/32, column/row l%32):
//   fp8 operand: byte i of the 8 dwords holds K = 32*(i/16) + 16*h + i%16
//   fp4 operand: nibble i of the first 4 dwords holds K = 32*h + i
//   scale:       lane half h supplies the scale of K block [32h, 32h+32)
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace sdq {
namespace mx {

typedef int i8v __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));

// group word flag bits (bit 3 of bytes 0-2) -> outlier position in bits 22-24
constexpr uint32_t kOutPosMagic = (1u << 21) | (1u << 14) | (1u << 7);

// Physical 16-byte piece offset of row r of an LDS tile with 128-byte rows.
// A-fragment reads take one logical piece of consecutive rows; with this XOR
// the rows of any aligned group of 8 fall on 8 distinct pieces, and those of
// any aligned group of 16 on 16 distinct (row parity, piece) pairs, so that
// the reads are free of bank conflicts whether the LDS serves 8 or 16 lanes
// of a 16-byte read per cycle (32 or 64 banks of 4 bytes).
__device__ __forceinline__ int lds_swizzle(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Dense e2m1 nibbles (position p at nibble p) of one group word.
template <int NI>
__device__ __forceinline__ uint32_t inlier_fp4(uint32_t w) {
  uint32_t D = 0;
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const uint32_t q = (w >> (8 * j + 4)) & 0xFu;
    const uint32_t sh = ((w >> (8 * j)) & 7u) << 2;
    D |= q << sh;
  }
  return D;
}

// ---- merged branches -------------------------------------------------------
// Within one 32-K block an inlier e2m1 value times 2^Ei equals an e4m3 value
// times 2^Eo when d = Ei - Eo lies in [-5, 6]: e2m1 magnitudes are 2^e or
// 1.5 * 2^e with e in [-1, 2], and shifting them by d keeps the e4m3 exponent
// field in [1, 15] without reaching the NaN code.  Then the outlier and the
// inlier branch of the block form one dense e4m3 fragment under the outlier's
// scale and take a single fp8 x fp8 matrix instruction.  Blocks with d
// outside that range keep their inliers out of the merged fragment and add
// them with the fp8 x fp4 instruction as before (a rare, wave-uniform path).

// e4m3 codes of the e2m1 magnitudes 0..7 shifted by d, as a v_perm table
// (bytes 0-3 in lo, 4-7 in hi); zero tables when the block cannot merge.
struct ShiftTable { uint32_t lo, hi, sign; };
__device__ __forceinline__ ShiftTable shift_table(int d, bool ok) {
  const int t = d * 8;                              // d in the exponent field
  const int x8 = __mul24(t, 0x010101) << 8;         // t in bytes 1..3
  ShiftTable T;
  T.lo = ok ? uint32_t(0x3C383000 + x8) : 0u;       // 0, 0.5, 1, 1.5
  T.hi = ok ? uint32_t(0x4C484440 + x8 + t) : 0u;   // 2, 3, 4, 6
  T.sign = ok ? 0x00808080u : 0u;
  return T;
}

// Dense e4m3 fragment (positions 0-3 in lo, 4-7 in hi) of one group word:
// the NI inliers converted with T and the outlier code, scattered by v_perm.
// A nibble map holds, per position, the v_perm selector of its byte: 4 + j
// for inlier slot j (bytes of the converted inliers), 3 for the outlier
// (byte 3 of the outlier-only word), 0 for an empty position (a zero byte).
template <int NI>
__device__ __forceinline__ void merged_e4m3(uint32_t w, const ShiftTable& T, uint32_t& lo, uint32_t& hi) {
  const uint32_t conv = __builtin_amdgcn_perm(T.hi, T.lo, (w >> 4) & 0x00070707u) | (w & T.sign);
  const uint32_t ob = w & 0xFF000000u;
  uint32_t N = 4u << (w << 2);  // slot 0 at 4 * p0 (bits 2-4 of w << 2; its low bits are 0)
  if constexpr (NI > 1) N |= 5u << ((w >> 6) & 0x1Cu);
  if constexpr (NI > 2) N |= 6u << ((w >> 14) & 0x1Cu);
  N |= 3u << (__umul24(w & 0x00080808u, kOutPosMagic) >> 22);  // 4 * outlier position
  const uint32_t Nh = N >> 4;
  const uint32_t e_lo = __builtin_amdgcn_perm(Nh, N, 0x05010400u) & 0x0F0F0F0Fu;
  const uint32_t e_hi = __builtin_amdgcn_perm(Nh, N, 0x07030602u) & 0x0F0F0F0Fu;
  lo = __builtin_amdgcn_perm(conv, ob, e_lo);
  hi = __builtin_amdgcn_perm(conv, ob, e_hi);
}

// Merged e4m3 fragment of one 64-K step for the fp8 operand order (lane half
// h holds groups {2h, 2h+1, 4+2h, 5+2h}) from the step's four fp4-order
// words of this lane (groups 4h..4h+3) and the lane's scale word (Eo, Ei of
// blocks 2s+h for s = 0, 1).  e: the outlier scale of block 2s+h (the MFMA
// scale this lane supplies); split: some block of this lane's groups did not
// merge its inliers.
struct MergedFrag { i8v b; int e; bool split; };
template <int NI>
__device__ __forceinline__ MergedFrag expand_merged(uint4 wq, uint32_t sc, int s) {
  MergedFrag f;
  auto s02 = __builtin_amdgcn_permlane32_swap(wq.x, wq.z, false, false);
  auto s13 = __builtin_amdgcn_permlane32_swap(wq.y, wq.w, false, false);
  const uint32_t u[4] = {s02[0], s13[0], s02[1], s13[1]};
  // scale bytes of block 2s + b of this row, b = 0, 1 (lane halves 0, 1)
  auto ss = __builtin_amdgcn_permlane32_swap(sc, sc, false, false);
  ShiftTable T[2];
  bool ok[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const uint32_t sb = ss[b] >> (16 * s);
    const int d = int((sb >> 8) & 0xFFu) - int(sb & 0xFFu);
    ok[b] = d >= -5 && d <= 6;
    T[b] = shift_table(d, ok[b]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t lo, hi;
    merged_e4m3<NI>(u[i], T[i >> 1], lo, hi);
    f.b[2 * i] = int(lo);
    f.b[2 * i + 1] = int(hi);
  }
  f.e = int((sc >> (16 * s)) & 0xFFu);  // Eo of block 2s + h
  f.split = !(ok[0] && ok[1]);
  return f;
}

// The inliers of this lane's block (fp4 order: block 2s + h) when that block
// did not merge, else zeros, with their scale Ei.
template <int NI>
__device__ __forceinline__ void split_inliers_fp4(uint4 wq, uint32_t sc, int s, i8v& bi, int& ei) {
  const uint32_t w[4] = {wq.x, wq.y, wq.z, wq.w};
  const uint32_t sb = sc >> (16 * s);
  const int d = int((sb >> 8) & 0xFFu) - int(sb & 0xFFu);
  const bool ok = d >= -5 && d <= 6;
#pragma unroll
  for (int i = 0; i < 4; ++i) bi[i] = ok ? 0 : int(inlier_fp4<NI>(w[i]));
#pragma unroll
  for (int i = 4; i < 8; ++i) bi[i] = 0;
  ei = int((sb >> 8) & 0xFFu);
}

}  // namespace mx
}  // namespace sdq
