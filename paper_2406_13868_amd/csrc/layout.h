// Physical layout of a packed SDQ weight blob, shared by the host packer and
// the GPU kernels of this library.
//
// The blob is organised in tiles of 32 rows of W by chunks of 128 K.  For
// every (tile t, chunk c), in this order:
//
//   section A  group words     512 x 32-bit   [t][c] (2 KiB)
//   section B  block scales    INT: 32 rows x 128/qv scales (qv = 16, 32 or
//                              64 dense K per scale) of 2 B (fp16) or 1 B
//                              (e4m3, e6m2): 512 B for fp16 per 16 K;
//                              MX: 256 B   [t][c]
//   section C  row scales      INT only: fp32 [t][32] outlier scales, then
//                              with e4m3 block scales fp32 [t][32] inlier
//                              row scales (powers of two)
//
// One 32-bit *group word* describes one 8-wide group (m_i = 8) of one row:
//
//   byte j (j = 0,1,2)  bits 0-2  position (0..7) of inlier slot j
//                       bit  3    bit j of the position of the outlier
//                       bits 4-7  code of inlier slot j (int4 two's
//                                 complement, or an e2m1 code)
//   byte 3              code of the outlier (e4m3 or int8 bits)
//
// Inlier slots are in ascending position order; an unused slot (n_i < 3) has
// position 0 and code 0.  With 1:16 outliers the outlier lives in the word
// of the 8-group that holds it; the other word of its 16-group (and every
// word when there is no outlier branch) has outlier code 0 at the lowest
// position that holds no inlier.  A zero code contributes nothing; keeping
// the outlier position off the inlier positions lets a kernel scatter all
// four slots of a word into one dense fragment without collisions.
//
// This layout lets a lane turn one word into a v_perm_b32 byte selector
// (positions in bits 0-2 of bytes 0-2 and 3 bits for byte 3), and keep the
// inlier codes at the top of each byte, where an int8 view of the byte is
// 16x the int4 value.
//
// Word order inside a (tile, chunk), with r the row inside the tile:
//   INT family (16-K scale blocks):   g = 8*j + 2*q + h,  kb = 4*j + q
//       word = ((h*32 + r)*2 + j)*4 + q          j,h in {0,1}, q in 0..3
//     so the 16 bytes at ((h*32 + r)*2 + j)*16 are the groups
//     {2*kb + h : kb = 4j..4j+3} of row r, and the words of four consecutive
//     rows (both j) for one h form one 128-byte run.
//   MX family (32-K scale blocks):    g = 4*b + i,  b = 2*s + h
//       word = ((s*2 + h)*32 + r)*4 + i          s,h in {0,1}, i in 0..3
//     so lane l = h*32 + r reads the four groups of 32-K block 2s+h of row r.
//
// Block scales inside a (tile, chunk):
//   INT: fp16 scale of row r, 16-K block kb (0..7) at byte (r*8 + kb)*2;
//        with e4m3 scales, the code at byte r*8 + kb
//   MX:  e8m0 of row r, 32-K block b = 2s+h at byte ((h*32 + r)*2 + s)*2 + br
//        with br = 0 for the outlier branch and 1 for the inlier branch
//
// Rows beyond N in the last tile are all-zero (codes and scales).
//
// Dual family (int8 outliers against int8 activations, fp4 inliers against
// fp4 activations), per (tile t, chunk c), in this order:
//   section A  inlier e2m1 codes, dense   2048 B  [t][c]
//              piece ((s*2 + h)*32 + r) of 16 bytes holds K 64s + 32h .. +32
//              of row r (64-K step s), byte j = K 2j (low nibble), 2j + 1
//              (high nibble): the fp4 operand of lane h*32 + r as loaded
//   section B  outlier half-words, P = max(1, n_o) planes of 1024 B
//              [t][c][plane]: plane p holds each group's p-th outlier in
//              ascending position order; group g = 4u + 2h + i (32-K step
//              u, half h, i in {0,1}) of row r at half-word
//              ((u*2 + h)*32 + r)*2 + i of the plane: bits 0-2 the position,
//              bits 8-15 the int8 code (0: no such outlier)
//   section C  inlier e8m0 scales          128 B  [t][c]
//              32-K block b = 2s + h of row r at byte b*32 + r
//   section D  outlier row scales, fp32 [t][32]
#pragma once
#include <cstddef>
#include <cstdint>

namespace sdq {

constexpr int kTileN = 32;
constexpr int kChunkK = 128;
constexpr int kGroup = 8;
constexpr int kWordsPerTC = kTileN * kChunkK / kGroup;            // 512
constexpr int kWordBytesPerTC = kWordsPerTC * 4;                  // 2048
constexpr int kIntScaleBytesPerTC = kTileN * (kChunkK / 16) * 2;  // 512
constexpr int kInt8ScaleBytesPerTC = kTileN * (kChunkK / 16);     // 256 (e4m3 block scales)
constexpr int kMxScaleBytesPerTC = kTileN * (kChunkK / 32) * 2;   // 256

struct Layout {
  int64_t n_tiles = 0, n_chunks = 0;
  int64_t words_off = 0, scales_off = 0, rows_off = 0, irow_off = 0, total = 0;
  int scale_bytes_per_tc = 0;
};

// INT family: qv dense K per inlier scale (16, 32 or 64) of sb bytes (fp16 2,
// e4m3 and e6m2 1); sc8: two-level e4m3 scales (inlier row scales at irow_off)
inline Layout make_layout(bool mx, int64_t N, int64_t K, bool sc8 = false, int qv = 16, int sb = 2) {
  Layout L;
  L.n_tiles = (N + kTileN - 1) / kTileN;
  L.n_chunks = (K + kChunkK - 1) / kChunkK;  // a last, partial chunk holds zeros past K
  L.scale_bytes_per_tc = mx ? kMxScaleBytesPerTC : kTileN * (kChunkK / qv) * sb;
  L.words_off = 0;
  L.scales_off = L.n_tiles * L.n_chunks * kWordBytesPerTC;
  L.rows_off = L.scales_off + L.n_tiles * L.n_chunks * L.scale_bytes_per_tc;
  L.irow_off = L.rows_off + (mx ? 0 : L.n_tiles * kTileN * 4);
  L.total = L.irow_off + (sc8 ? L.n_tiles * kTileN * 4 : 0);
  return L;
}

constexpr int kDualNibBytesPerTC = kTileN * kChunkK / 2;     // 2048
constexpr int kDualOutBytesPerTC = kTileN * (kChunkK / 8) * 2;  // 1024
constexpr int kDualScaleBytesPerTC = kTileN * (kChunkK / 32);   // 128

struct DualLayout {
  int64_t n_tiles = 0, n_chunks = 0;
  int64_t nib_off = 0, out_off = 0, scale_off = 0, rows_off = 0, total = 0;
  int out_planes = 1;                          // outlier half-word planes: max(1, n_o)
  int64_t out_bytes_per_tc = kDualOutBytesPerTC;  // out_planes * 1024
};

inline DualLayout make_dual_layout(int64_t N, int64_t K, int n_o) {
  DualLayout L;
  L.n_tiles = (N + kTileN - 1) / kTileN;
  L.n_chunks = (K + kChunkK - 1) / kChunkK;
  L.out_planes = n_o > 1 ? n_o : 1;
  L.out_bytes_per_tc = int64_t(L.out_planes) * kDualOutBytesPerTC;
  const int64_t tc = L.n_tiles * L.n_chunks;
  L.nib_off = 0;
  L.out_off = tc * kDualNibBytesPerTC;
  L.scale_off = L.out_off + tc * L.out_bytes_per_tc;
  L.rows_off = L.scale_off + tc * kDualScaleBytesPerTC;
  L.total = L.rows_off + L.n_tiles * kTileN * 4;
  return L;
}
inline int dual_nib_byte(int k, int r) {  // k in 0..127 within the chunk
  const int s = k >> 6, h = (k >> 5) & 1;
  return ((s * 2 + h) * 32 + r) * 16 + ((k & 31) >> 1);
}
inline int dual_out_halfword(int g, int r) {
  const int u = g >> 2, h = (g >> 1) & 1, i = g & 1;
  return ((u * 2 + h) * 32 + r) * 2 + i;
}
inline int dual_scale_byte(int b, int r) { return b * 32 + r; }

// Word index of group g (0..15 within the chunk) of tile row r.
inline int int_word_index(int g, int r) {
  const int kb = g >> 1, h = g & 1, j = kb >> 2, q = kb & 3;
  return ((h * 32 + r) * 2 + j) * 4 + q;
}
inline int mx_word_index(int g, int r) {
  const int b = g >> 2, i = g & 3, s = b >> 1, h = b & 1;
  return ((s * 2 + h) * 32 + r) * 4 + i;
}
inline int int_scale_byte(int kb, int r) { return (r * 8 + kb) * 2; }
inline int int8_scale_byte(int kb, int r) { return r * 8 + kb; }
// INT family, general Q-Vector: byte offset of scale b (0 .. 128/qv - 1 within
// the chunk) of tile row r, scales of sb bytes.  A row's scales of one chunk
// are contiguous: (128/qv) * sb bytes at r * (128/qv) * sb.
inline int int_scale_off(int b, int r, int qv, int sb) { return (r * (kChunkK / qv) + b) * sb; }
inline int mx_scale_byte(int b, int r, int branch) {
  const int s = b >> 1, h = b & 1;
  return ((h * 32 + r) * 2 + s) * 2 + branch;
}

}  // namespace sdq
