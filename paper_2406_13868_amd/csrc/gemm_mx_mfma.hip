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
// Operand layouts and the weight-fragment expansion are in mx_frag.h.
//
// Tiling: a workgroup of 4 waves owns 4 row tiles of W (128 outputs) and BM
// = 32*MS tokens; fp8 activations are staged per 128-K chunk in LDS (double
// buffered, XOR-swizzled) and shared by the 4 waves; weights stream from HBM
// into registers and are expanded there into dense fp8 / fp4 fragments.
// Weights and activations are requested two chunks before they are used.
//
// Split-K form (a caller-owned workspace): the grid also runs over ranges of
// the 128-K chunks; each workgroup writes the raw fp32 sums of its range to
// the workspace, and a second kernel adds the ranges in order and scales by
// s_a.  For tens to hundreds of tokens, where the one-pass grid alone leaves
// CUs idle or runs one workgroup per CU through every chunk.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "kernels.h"
#include "mx_frag.h"
#include "tile_out.h"

namespace sdq {
namespace {

using namespace mx;

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int64_t kCUs = 256;  // compute units of an MI355X
struct MxArgs {
  const uint8_t* Xq;
  const float* s_a;
  const uint8_t* blob;
  void* Y;
  int M, N, K, n_chunks, n_tiles;
  int64_t scales_off;
  int m_blocks = 1;  // workgroups along M; the grid is 1-D over (K range, tile group, M block)
  bool y_bf16 = false;  // Y as bf16
  int k_ranges = 1;     // ranges of chunks the grid splits K into
  int kc_range = 0;     // chunks per range (the last may hold fewer)
  float* part = nullptr;  // split-K: [k_ranges][M][N] raw sums; null: Y = s_a * acc
};

template <int MS, int NI, bool HAS_O>
__global__ __launch_bounds__(kThreads, MS >= 8 ? 1 : 2) void mx_mfma_kernel(MxArgs a) {
  constexpr int BM = 32 * MS;
  // fp8 activations of one 128-K chunk, BM rows of 128 bytes, each 16-byte
  // piece p of row r at piece p ^ lds_swizzle(r)
  __shared__ __align__(16) uint8_t xs[2][BM * kChunkK];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: chunk offsets stay scalar
  const int col = lane & 31, h = lane >> 5;
  int group, mblock;
  const int items = int(gridDim.x) / a.k_ranges;  // (tile group, M block) items per K range
  const int range = int(blockIdx.x) / items;
  tile_work(int(blockIdx.x) - range * items, items / a.m_blocks, a.m_blocks, group, mblock);
  const int m0 = mblock * BM;
  const int tile = min(group * kWaves + wave, a.n_tiles - 1);  // spare waves recompute the last tile
  const bool tile_ok = group * kWaves + wave < a.n_tiles;
  const int KC = a.n_chunks;
  const int cb = range * a.kc_range, ce = min(KC, cb + a.kc_range);  // this workgroup's chunks

  // ---- activation staging: every thread moves kPerThread 16-byte pieces
  constexpr int kPerThread = BM * 8 / kThreads;
  static_assert(kPerThread * kThreads == BM * 8, "whole pieces per thread");
  // thread tid moves pieces p = tid & 7 of rows (tid >> 3) + 32 i; the
  // swizzle of those rows does not depend on i, so their LDS offsets are one
  // register plus i * 32 rows
  // the block's rows through a buffer resource: rows past M (whose outputs
  // are never stored) and the bytes of a last partial chunk past the end of
  // the tensor read 0
  const __amdgpu_buffer_rsrc_t x_rsrc =
      buffer_rsrc(a.Xq + size_t(m0) * a.K, uint32_t(min(a.M - m0, BM)) * uint32_t(a.K));
  uint32_t xsrc[kPerThread];
  const uint32_t xdst0 = uint32_t((tid >> 3) * kChunkK + (((tid & 7) ^ lds_swizzle(tid >> 3)) << 4));
#pragma unroll
  for (int i = 0; i < kPerThread; ++i)
    xsrc[i] = uint32_t((tid >> 3) + i * 32) * uint32_t(a.K) + uint32_t(tid & 7) * 16u;
  auto ld_x = [&](uint32_t voff, int c) __attribute__((always_inline)) {
    typedef unsigned int u4_ __attribute__((ext_vector_type(4)));
    const u4_ q = __builtin_bit_cast(
        u4_, __builtin_amdgcn_raw_buffer_load_b128(x_rsrc, voff, uint32_t(c) * kChunkK, 0));
    return make_uint4(q[0], q[1], q[2], q[3]);
  };
  // activations of one chunk on their way to LDS, as named registers (the
  // compiler keeps a local array of them in scratch across the products)
  static_assert(kPerThread == 1 || kPerThread == 2 || kPerThread == 4 || kPerThread == 8,
                "1, 2, 4 or 8 pieces per thread");
  uint4 xr0, xr1, xr2, xr3, xr4, xr5, xr6, xr7;
#define SDQ_XLD(i, c) ld_x(xsrc[i], c)
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
  const int last = ce - 1;
  WRegs wA, wB;     // weights of the even / odd chunks (counted from cb)
  SDQ_LOAD_X(cb)
  load_w(cb, wA);
  load_w(min(cb + 1, last), wB);
  SDQ_STORE_X(0)
  SDQ_LOAD_X(min(cb + 1, last))
  BFrag fE = expand(wA, 0), fO;  // first step of the next even / odd chunk
  __syncthreads();
  for (int c = cb; c < ce; c += 2) {
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
    if (c + 1 >= ce) break;
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
  if (a.part) {  // split-K: this range's raw sums
    const OutRows pr = out_rows(a.part + size_t(range) * size_t(a.M) * size_t(a.N), false, a.M, a.N, m0, BM);
#pragma unroll
    for (int ms = 0; ms < MS; ++ms)
#pragma unroll
      for (int e = 0; e < 16; ++e) store_out(pr, a.N, n, ms, e, h, acc[ms][e]);
    return;
  }
  const RowScales<MS> rs = load_row_scales<MS>(a.s_a, a.M, m0, h);
  const OutRows yr = out_rows(a.Y, a.y_bf16, a.M, a.N, m0, BM);
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e) store_out(yr, a.N, n, ms, e, h, rs.v[ms][e] * acc[ms][e]);
}

template <int MS, int NI>
hipError_t launch_ms_ni(const Cfg& c, const MxArgs& a, hipStream_t st) {
  MxArgs b = a;
  b.m_blocks = int((a.M + 32 * MS - 1) / (32 * MS));
  const dim3 grid(unsigned((a.n_tiles + kWaves - 1) / kWaves * b.m_blocks * b.k_ranges));
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
                          const uint8_t* blob, int64_t N, int64_t K, void* Y, hipStream_t st) {
  const Layout L = make_layout(true, N, K);
  MxArgs a{Xq, s_a, blob, Y, int(M), int(N), int(K), int(L.n_chunks), int(L.n_tiles), L.scales_off};
  a.y_bf16 = c.y_bf16;
  a.kc_range = int(L.n_chunks);
  if (M <= 32) return launch_ms<1>(c, a, st);
  if (M <= 64) return launch_ms<2>(c, a, st);
  // More tokens: the largest token block that still gives a full round of
  // workgroups wins (each block re-expands every weight it reads).  Measured
  // at M = 128/256: 4096x4096 takes 26/27 us with 32-token blocks against
  // 36/37 us with 128; 11008x4096 at M = 128 takes 31 us with 64 against 38.
  const int64_t groups = (a.n_tiles + kWaves - 1) / kWaves;
  if (groups * ((M + 31) / 32) <= kCUs) return launch_ms<1>(c, a, st);
  if (groups * ((M + 63) / 64) <= kCUs) return launch_ms<2>(c, a, st);
  return launch_ms<4>(c, a, st);
}

// Split-K shape: token blocks of 32 tokens up to 32, 64 up to 64, else 128
// (the K split, not the token block, fills the GPU), then K ranges of at
// least kMxSplitMinChunks chunks until about kMxSplitTarget workgroups run
// (two per CU).
constexpr int kMxSplitTarget = 512;

struct MxSplitShape {
  int MS, S, kc_range;
};

MxSplitShape mx_split_shape(int64_t M, int64_t N, int64_t K) {
  MxSplitShape s;
  const int64_t tiles = (N + kTileN - 1) / kTileN, groups = (tiles + kWaves - 1) / kWaves;
  const int64_t kc = (K + kChunkK - 1) / kChunkK;
  s.MS = M <= 32 ? 1 : M <= 64 ? 2 : 4;
  const int64_t items = groups * std::max<int64_t>(1, (M + 32 * s.MS - 1) / (32 * s.MS));
  int64_t S = (kMxSplitTarget + items - 1) / items;
  S = std::max<int64_t>(1, std::min<int64_t>(S, kc / kMxSplitMinChunks));
  s.kc_range = int((kc + S - 1) / S);
  s.S = int((kc + s.kc_range - 1) / s.kc_range);  // no empty range
  return s;
}

size_t mx_split_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  return size_t(mx_split_shape(M, N, K).S) * size_t(M) * size_t(N) * sizeof(float);
}

hipError_t launch_mx_split(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                           const uint8_t* blob, int64_t N, int64_t K, void* Y, void* workspace,
                           hipStream_t st) {
  const Layout L = make_layout(true, N, K);
  const MxSplitShape sh = mx_split_shape(M, N, K);
  MxArgs a{Xq, s_a, blob, Y, int(M), int(N), int(K), int(L.n_chunks), int(L.n_tiles), L.scales_off};
  a.k_ranges = sh.S;
  a.kc_range = sh.kc_range;
  a.part = static_cast<float*>(workspace);
  const hipError_t e = sh.MS == 1 ? launch_ms<1>(c, a, st) : sh.MS == 2 ? launch_ms<2>(c, a, st)
                                                                        : launch_ms<4>(c, a, st);
  if (e != hipSuccess) return e;
  return launch_split_reduce(a.part, s_a, Y, M, N, sh.S, c.y_bf16, st);
}

}  // namespace sdq
