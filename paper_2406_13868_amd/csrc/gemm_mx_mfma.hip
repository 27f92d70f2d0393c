// MX-family decomposed GEMM on the matrix cores (any M).  Section 5.1:
// Y = SpMM(A, W_o) + SpMM(A, W_i), both branches accumulated by the matrix
// core itself into one fp32 accumulator per output.
//
// gfx950's v_mfma_scale_f32_32x32x64_f8f6f4 multiplies fp8 activations by
// fp8 or fp4 weights and applies an e8m0 scale to every 32 K of each weight
// column inside the instruction, which is exactly the MX form of both
// branches:
//   acc += Xq(e4m3) * W_o(e4m3, 2^Eo per 32 K)      fp8 x fp8
//   acc += Xq(e4m3) * W_i(e2m1, 2^Ei per 32 K)      fp8 x fp4
//   Y = s_a * acc
// The products are exact and accumulate in fp32.
//
// Operand layouts (32x32x64, lane l, lane half h = l/32, column/row l%32):
//   fp8 operand: byte i of the 8 dwords holds K = 32*(i/16) + 16*h + i%16
//   fp4 operand: nibble i of the first 4 dwords holds K = 32*h + i
//   scale:       lane half h supplies the scale of K block [32h, 32h+32)
// A lane reads the four group words of one 32-K block (the fp4 order); the
// fp8 order needs two of them from the other lane half, exchanged with
// v_permlane32_swap.
//
// Tiling: a workgroup of 4 waves owns 4 row tiles of W (128 outputs) and BM
// = 32*MS tokens; fp8 activations are staged per 128-K chunk in LDS (double
// buffered, XOR-swizzled) and shared by the 4 waves; weights stream from HBM
// into registers and are expanded there into dense fp8 / fp4 fragments.
// Weights and activations are requested two chunks before they are used.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace sdq {
namespace {

typedef int i8v __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr uint32_t kOutPosMagic = (1u << 21) | (1u << 14) | (1u << 7);

struct MxArgs {
  const uint8_t* Xq;
  const float* s_a;
  const uint8_t* blob;
  float* Y;
  int M, N, K, n_chunks, n_tiles;
  int64_t scales_off;
  int m_blocks;  // workgroups along M; the grid is 1-D over (tile group, M block)
};

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

// Dense e4m3 bytes (position p at byte p of lo:hi) of one group word.
__device__ __forceinline__ void outlier_fp8(uint32_t w, uint32_t& lo, uint32_t& hi) {
  const uint32_t pos = (__umul24(w & 0x00080808u, kOutPosMagic) >> 24) & 7u;
  const uint32_t v = (w >> 24) << ((pos & 3u) << 3);
  lo = pos < 4u ? v : 0u;
  hi = pos < 4u ? 0u : v;
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

template <int MS, int NI, bool HAS_O>
__global__ __launch_bounds__(kThreads, MS >= 8 ? 1 : 2) void mx_mfma_kernel(MxArgs a) {
  constexpr int BM = 32 * MS;
  // fp8 activations of one 128-K chunk, BM rows of 128 bytes, each 16-byte
  // piece p of row r at piece p ^ lds_swizzle(r)
  __shared__ __align__(16) uint8_t xs[2][BM * kChunkK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, h = lane >> 5;
  // every XCD takes a contiguous range of tile groups and all their M blocks,
  // so a tile's weights are reused from that XCD's L2
  const int work = xcd_contiguous(blockIdx.x, gridDim.x);
  const int group = work / a.m_blocks;
  const int m0 = (work - group * a.m_blocks) * BM;
  const int tile = min(group * kWaves + wave, a.n_tiles - 1);  // spare waves recompute the last tile
  const bool tile_ok = group * kWaves + wave < a.n_tiles;
  const int KC = a.n_chunks;

  // ---- activation staging: every thread moves kPerThread 16-byte pieces
  constexpr int kPerThread = BM * 8 / kThreads;
  static_assert(kPerThread * kThreads == BM * 8, "whole pieces per thread");
  // thread tid moves pieces p = tid & 7 of rows (tid >> 3) + 32 i; the
  // swizzle of those rows does not depend on i, so their LDS offsets are one
  // register plus i * 32 rows
  const uint8_t* xsrc[kPerThread];
  const uint32_t xdst0 = uint32_t((tid >> 3) * kChunkK + (((tid & 7) ^ lds_swizzle(tid >> 3)) << 4));
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int rr = (tid >> 3) + i * 32;
    // rows past M re-read row M-1 (their outputs are never stored)
    xsrc[i] = a.Xq + size_t(min(m0 + rr, a.M - 1)) * a.K + (tid & 7) * 16;
  }
  // activations of one chunk on their way to LDS, as named registers (the
  // compiler keeps a local array of them in scratch across the products)
  static_assert(kPerThread == 1 || kPerThread == 2 || kPerThread == 4 || kPerThread == 8,
                "1, 2, 4 or 8 pieces per thread");
  uint4 xr0, xr1, xr2, xr3, xr4, xr5, xr6, xr7;
#define SDQ_XLD(i, c) *reinterpret_cast<const uint4*>(xsrc[i] + size_t(c) * kChunkK)
#define SDQ_LOAD_X(c)                                        \
  {                                                          \
    xr0 = SDQ_XLD(0, c);                                     \
    if constexpr (kPerThread > 1) xr1 = SDQ_XLD(1, c);       \
    if constexpr (kPerThread > 2) {                          \
      xr2 = SDQ_XLD(2, c);                                   \
      xr3 = SDQ_XLD(3, c);                                   \
    }                                                        \
    if constexpr (kPerThread > 4) {                          \
      xr4 = SDQ_XLD(4, c);                                   \
      xr5 = SDQ_XLD(5, c);                                   \
      xr6 = SDQ_XLD(6, c);                                   \
      xr7 = SDQ_XLD(7, c);                                   \
    }                                                        \
  }
#define SDQ_XST(b, i) *reinterpret_cast<uint4*>(&xs[b][xdst0 + (i) * 32 * kChunkK])
#define SDQ_STORE_X(buf)                                                            \
  {                                                                                 \
    SDQ_XST(buf, 0) = xr0;                                                               \
    if constexpr (kPerThread > 1) SDQ_XST(buf, 1) = xr1;                                 \
    if constexpr (kPerThread > 2) {                                                 \
      SDQ_XST(buf, 2) = xr2;                                                           \
      SDQ_XST(buf, 3) = xr3;                                                           \
    }                                                                               \
    if constexpr (kPerThread > 4) {                                                 \
      SDQ_XST(buf, 4) = xr4;                                                           \
      SDQ_XST(buf, 5) = xr5;                                                           \
      SDQ_XST(buf, 6) = xr6;                                                           \
      SDQ_XST(buf, 7) = xr7;                                                           \
    }                                                                               \
  }

  // ---- weight stream of this wave's tile
  const uint8_t* wbase = a.blob + size_t(tile) * KC * kWordBytesPerTC + size_t(lane) * 16;
  const uint8_t* sbase = a.blob + a.scales_off + size_t(tile) * KC * kMxScaleBytesPerTC + lane * 4;
  struct WRegs { uint4 w0, w1; uint32_t sc; };
  auto load_w = [&](int c, WRegs& r) __attribute__((always_inline)) {
    r.w0 = *reinterpret_cast<const uint4*>(wbase + size_t(c) * kWordBytesPerTC);
    r.w1 = *reinterpret_cast<const uint4*>(wbase + size_t(c) * kWordBytesPerTC + 1024);
    r.sc = *reinterpret_cast<const uint32_t*>(sbase + size_t(c) * kMxScaleBytesPerTC);
  };

  f16v acc[MS];
#pragma unroll
  for (int s = 0; s < MS; ++s)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[s][e] = 0.f;

  // A-fragment byte offsets of this lane in a chunk buffer: row ms*32 + col,
  // logical pieces 4s + h and 4s + h + 2 for step s; the swizzle of row
  // ms*32 + col is that of col, so sub-tile ms adds ms * 32 rows
  uint32_t aoff[2][2];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int u = 0; u < 2; ++u) aoff[s][u] = uint32_t(col * kChunkK + (((4 * s + h + 2 * u) ^ lds_swizzle(col)) << 4));

  // B fragments of one 64-K step.  With outliers: the merged e4m3 fragment
  // (lane half h holds groups {2h, 2h+1, 4+2h, 5+2h} of the step, the fp8
  // operand order) under the scale of block h, plus the flags of blocks that
  // cannot merge.  Without outliers: the fp4 inlier fragment (groups 4h..4h+3).
  // When any block of the wave's step did not merge (wave-uniform flag), the
  // expansion also builds the fp4 inlier fragment of those blocks (bi, ei), so
  // that the product loop issues no memory access of its own.
  struct BFrag { i8v b; int e; bool split; i8v bi; int ei; };
  auto expand = [&](const WRegs& wr, int s) __attribute__((always_inline)) {
    BFrag f;
    const uint4 wq = s ? wr.w1 : wr.w0;
    const uint32_t w[4] = {wq.x, wq.y, wq.z, wq.w};
    if constexpr (HAS_O) {
      const MergedFrag m = expand_merged<NI>(wq, wr.sc, s);
      f.b = m.b;
      f.e = m.e;
      f.split = __any(m.split);
      if (f.split) split_inliers_fp4<NI>(wq, wr.sc, s, f.bi, f.ei);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) f.b[i] = int(inlier_fp4<NI>(w[i]));
#pragma unroll
      for (int i = 4; i < 8; ++i) f.b[i] = 0;
      f.e = int((wr.sc >> (16 * s + 8)) & 0xFFu);  // Ei of block 2s + h
      f.split = false;
    }
    return f;
  };
  auto mfmas = [&](int buf, int s, const BFrag& f) __attribute__((always_inline)) {
    i8v av[MS];
#pragma unroll
    for (int ms = 0; ms < MS; ++ms) {
      const uint4 a0 = *reinterpret_cast<const uint4*>(&xs[buf][aoff[s][0] + ms * 32 * kChunkK]);
      const uint4 a1 = *reinterpret_cast<const uint4*>(&xs[buf][aoff[s][1] + ms * 32 * kChunkK]);
      av[ms] = i8v{int(a0.x), int(a0.y), int(a0.z), int(a0.w), int(a1.x), int(a1.y), int(a1.z), int(a1.w)};
    }
    if constexpr (HAS_O) {
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
        acc[ms] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av[ms], f.b, acc[ms], 0, 0, 0, 127, 0, f.e);
      if (f.split) {  // wave-uniform, rare: the inliers of blocks that did not merge
#pragma unroll
        for (int ms = 0; ms < MS; ++ms)
          acc[ms] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av[ms], f.bi, acc[ms], 0, 4, 0, 127, 0, f.ei);
      }
    } else {
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
        acc[ms] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av[ms], f.b, acc[ms], 0, 4, 0, 127, 0, f.e);
    }
  };

  // ---- pipeline.  Weights are requested two chunks ahead and expanded one
  //      step ahead of their products (the next chunk's first step while
  //      this chunk's second step runs), so that the expansion of one step
  //      overlaps the matrix instructions of the other; activations of chunk
  //      c+1 go from registers to LDS after the products of chunk c.  Loads
  //      past the last chunk re-read it (in bounds, never used), so that no
  //      load is conditional.  A register set is refilled right after its
  //      last expansion, never copied (a copy would wait for the load).
  const int last = KC - 1;
  WRegs wA, wB;     // weights of the even / odd chunks
  SDQ_LOAD_X(0)
  load_w(0, wA);
  load_w(min(1, last), wB);
  SDQ_STORE_X(0)
  SDQ_LOAD_X(min(1, last))
  BFrag fE = expand(wA, 0), fO;  // first step of the next even / odd chunk
  __syncthreads();
  for (int c = 0; c < KC; c += 2) {
    {
      const BFrag f1 = expand(wA, 1);
      load_w(min(c + 2, last), wA);
      mfmas(0, 0, fE);
      fO = expand(wB, 0);
      mfmas(0, 1, f1);
      SDQ_STORE_X(1)
      SDQ_LOAD_X(min(c + 2, last))
      __syncthreads();
    }
    if (c + 1 >= KC) break;
    {
      const BFrag f1 = expand(wB, 1);
      load_w(min(c + 3, last), wB);
      mfmas(1, 0, fO);
      fE = expand(wA, 0);
      mfmas(1, 1, f1);
      SDQ_STORE_X(0)
      SDQ_LOAD_X(min(c + 3, last))
      __syncthreads();
    }
  }

#undef SDQ_XLD
#undef SDQ_XST
#undef SDQ_LOAD_X
#undef SDQ_STORE_X
  if (!tile_ok) return;
  const int n = tile * kTileN + col;
  if (n >= a.N) return;
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int m = m0 + ms * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
      if (m < a.M) a.Y[size_t(m) * a.N + n] = a.s_a[m] * acc[ms][e];
    }
}

template <int MS, int NI>
hipError_t launch_ms_ni(const Cfg& c, const MxArgs& a, hipStream_t st) {
  MxArgs b = a;
  b.m_blocks = int((a.M + 32 * MS - 1) / (32 * MS));
  const dim3 grid(unsigned((a.n_tiles + kWaves - 1) / kWaves * b.m_blocks));
  const dim3 block(kThreads);
  if (c.n_o)
    hipLaunchKernelGGL((mx_mfma_kernel<MS, NI, true>), grid, block, 0, st, b);
  else
    hipLaunchKernelGGL((mx_mfma_kernel<MS, NI, false>), grid, block, 0, st, b);
  return hipGetLastError();
}

template <int MS>
hipError_t launch_ms(const Cfg& c, const MxArgs& a, hipStream_t st) {
  if (c.n_i == 1) return launch_ms_ni<MS, 1>(c, a, st);
  if (c.n_i == 2) return launch_ms_ni<MS, 2>(c, a, st);
  return launch_ms_ni<MS, 3>(c, a, st);
}

}  // namespace

hipError_t launch_mx_mfma(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                          const uint8_t* blob, int64_t N, int64_t K, float* Y, hipStream_t st) {
  const Layout L = make_layout(true, N, K);
  MxArgs a{Xq, s_a, blob, Y, int(M), int(N), int(K), int(L.n_chunks), int(L.n_tiles), L.scales_off};
  if (M <= 32) return launch_ms<1>(c, a, st);
  if (M <= 64) return launch_ms<2>(c, a, st);
  return launch_ms<4>(c, a, st);
}

}  // namespace sdq
