// INT-family decomposed GEMM on the matrix cores (any M).  Section 5.1:
// Y = SpMM(A, W_o) + SpMM(A, W_i) with one fp32 result per output.
//
// gfx950 has no matrix instruction that applies a scale every 16 K, which is
// what the fp16 inlier scales need, and none that multiplies int8 by fp8.
// Both branches therefore run on v_mfma_f32_32x32x16_f16, which is exact
// here: int8 activations, int4 inliers and int8/e4m3 outliers are all exact
// fp16 numbers, their products are exact in fp32, and a 16-K sum of int8 x
// int4 products stays below 2^24.
//   inlier:  P = Xq_blk * q_blk (one MFMA per 16-K block, K = 16 = one scale
//            block), acc += P * s_blk  (fp32, per column scale)
//   outlier: acc_o += Xq_blk * q_o_blk (MFMA accumulation), scaled by the
//            per-row s_o once at the end
//   Y = s_a * (acc + s_o * acc_o)
//
// Tiling: a workgroup of 4 waves owns 4 row tiles of W (128 outputs) and BM
// = 32*MS = 128 tokens, two workgroups per CU (the register budget of two
// waves per SIMD holds the eight 32x32 accumulators of a wave without
// spilling).  Each 128-K chunk of activations is converted from int8 to
// fp16 and staged in LDS (double buffered) for all 4 waves; each wave streams
// its own tile's group words (32 bytes per lane per chunk) and
// expands them in registers into dense fp16 B fragments: lane l holds column
// l%32 and the 8-group 2*kb + l/32 of every 16-K block kb.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "int_frag.h"
#include "kernels.h"
#include "tile_out.h"

namespace sdq {
namespace {

using namespace intfrag;

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int64_t kCUs = 256;                      // compute units of an MI355X
constexpr int kRowPad = 8;                        // f16 elements of padding per LDS row
constexpr int kLdsRow = kChunkK + kRowPad;        // 136 f16 = 272 bytes

struct MfmaArgs {
  const uint8_t* Xq;
  const float* s_a;
  const uint8_t* blob;
  void* Y;
  int M, N, K, n_chunks, n_tiles;
  int64_t scales_off, rows_off, irow_off;
  bool y_bf16 = false;  // Y as bf16
  int qs = 0;           // log2(qv / 16): 16-K blocks per inlier scale = 1 << qs
  int srow = 16;        // bytes of one row's inlier scales in a chunk: (128 / qv) * (2 or 1)
  // tiled kernel over K ranges (grid z): chunks [z * kc_range, (z + 1) *
  // kc_range) of every tile, raw partial sums to part[z][M][N]
  int k_ranges = 1, kc_range = 0;
  float* part = nullptr;
};

template <int MS, int NI, bool OUT_INT8, int SF>
__global__ __launch_bounds__(kThreads, 2) void int_mfma_kernel(MfmaArgs a) {
  constexpr bool SC8 = SF == kScaleE4M3;       // two-level: a power of two per row
  constexpr bool ONE = SF != kScaleF16;        // q * s exact in one fp16 fragment
  const int kSB = kTileN * a.srow;             // inlier scale bytes per (tile, chunk)
  constexpr int BM = 32 * MS;
  __shared__ __align__(16) _Float16 xs[2][BM * kLdsRow];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: chunk offsets stay scalar
  const int col = lane & 31, h = lane >> 5;
  const int m0 = blockIdx.y * BM;
  const int tile = blockIdx.x * kWaves + wave;
  const bool tile_ok = tile < a.n_tiles;
  const int KC = a.n_chunks;
  const int cb = int(blockIdx.z) * a.kc_range;                   // this workgroup's chunks [cb, ce)
  const int ce = a.k_ranges > 1 ? min(KC, cb + a.kc_range) : KC;

  // ---- activation staging: BM rows x 128 int8 -> fp16 in LDS
  // thread -> (row, 16-byte column piece): 8 pieces per row
  constexpr int kPieces = BM * 8;
  constexpr int kPerThread = (kPieces + kThreads - 1) / kThreads;
  uint4 xr[kPerThread];
  // the block's rows through a buffer resource: rows past M, and the bytes of
  // a last partial chunk past the end of the tensor, read 0
  const __amdgpu_buffer_rsrc_t x_rsrc =
      buffer_rsrc(a.Xq + size_t(m0) * a.K, uint32_t(min(a.M - m0, BM)) * uint32_t(a.K));
  auto load_x = [&](int c) {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int pc = tid + i * kThreads;
      const int rr = pc >> 3, cp = pc & 7;
      xr[i] = make_uint4(0, 0, 0, 0);
      if (pc < kPieces) {
        typedef unsigned int u4_ __attribute__((ext_vector_type(4)));
        const u4_ q = __builtin_bit_cast(u4_, __builtin_amdgcn_raw_buffer_load_b128(
            x_rsrc, uint32_t(rr) * uint32_t(a.K) + uint32_t(cp) * 16u, uint32_t(c) * kChunkK, 0));
        xr[i] = make_uint4(q[0], q[1], q[2], q[3]);
      }
    }
  };
  auto store_x = [&](int buf) {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int pc = tid + i * kThreads;
      if (pc >= kPieces) continue;
      const int rr = pc >> 3, cp = pc & 7;
      uint32_t o[8];
      i8x4_to_f16x4(xr[i].x, o[0], o[1]);
      i8x4_to_f16x4(xr[i].y, o[2], o[3]);
      i8x4_to_f16x4(xr[i].z, o[4], o[5]);
      i8x4_to_f16x4(xr[i].w, o[6], o[7]);
      uint4* dst = reinterpret_cast<uint4*>(&xs[buf][rr * kLdsRow + cp * 16]);
      dst[0] = make_uint4(o[0], o[1], o[2], o[3]);
      dst[1] = make_uint4(o[4], o[5], o[6], o[7]);
    }
  };

  // ---- weight stream of this wave's tile
  // lane (col, h): the 32 bytes at ((h*32 + col)*2 + j)*16, j = 0, 1
  const uint8_t* wbase = a.blob + size_t(tile_ok ? tile : 0) * KC * kWordBytesPerTC + size_t(lane) * 32;
  const uint8_t* sbase = a.blob + a.scales_off + size_t(tile_ok ? tile : 0) * KC * kSB + col * a.srow;
  uint4 wr0, wr1, sr;
  auto load_w = [&](int c) {
    if (tile_ok) {
      wr0 = *reinterpret_cast<const uint4*>(wbase + size_t(c) * kWordBytesPerTC);
      wr1 = *reinterpret_cast<const uint4*>(wbase + size_t(c) * kWordBytesPerTC + 16);
      sr = load_row_scales_chunk(sbase + size_t(c) * kSB, a.srow);
    } else {
      wr0 = wr1 = sr = make_uint4(0, 0, 0, 0);
    }
  };

  f16v acc[MS], acco[MS];
#pragma unroll
  for (int s = 0; s < MS; ++s)
#pragma unroll
    for (int e = 0; e < 16; ++e) { acc[s][e] = 0.f; acco[s][e] = 0.f; }

  load_x(cb);
  load_w(cb);
  store_x(0);
  __syncthreads();

  for (int c = cb; c < ce; ++c) {
    const int buf = (c - cb) & 1;
    const uint32_t wv[8] = {wr0.x, wr0.y, wr0.z, wr0.w, wr1.x, wr1.y, wr1.z, wr1.w};
    const uint32_t sv[4] = {sr.x, sr.y, sr.z, sr.w};
    if (c + 1 < ce) { load_x(c + 1); load_w(c + 1); }
#pragma unroll
    for (int kb = 0; kb < 8; ++kb) {
      const _Float16 s = block_scale<SF>(sv, kb, a.qs);
      h8 bh, bl;
      if constexpr (ONE) {
        // an int4 code times an e4m3 (e6m2) scale has at most 7 (6)
        // significant bits: exact in fp16, so one fragment carries it
        const h8 sv8 = {s, s, s, s, s, s, s, s};
        bh = inlier_f16<NI>(wv[kb]) * sv8;
      } else {
        scaled_hi_lo(inlier_f16<NI>(wv[kb]), s, bh, bl);
      }
      const h8 bo = outlier_f16<OUT_INT8>(wv[kb]);
      h8 av[MS];
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
        av[ms] = *reinterpret_cast<const h8*>(&xs[buf][(ms * 32 + col) * kLdsRow + kb * 16 + h * 8]);
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) acc[ms] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[ms], bh, acc[ms], 0, 0, 0);
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) acco[ms] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[ms], bo, acco[ms], 0, 0, 0);
      if constexpr (!ONE) {
#pragma unroll
        for (int ms = 0; ms < MS; ++ms) acc[ms] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[ms], bl, acc[ms], 0, 0, 0);
      }
    }
    if (c + 1 < ce) {
      store_x(buf ^ 1);
      __syncthreads();
    }
  }

  if (!tile_ok) return;
  const int n = tile * kTileN + col;
  if (n >= a.N) return;
  const float so = reinterpret_cast<const float*>(a.blob + a.rows_off)[n];
  // the inlier row scale of two-level e4m3 scales (a power of two: exact)
  const float gi = SC8 ? reinterpret_cast<const float*>(a.blob + a.irow_off)[n] : 1.f;
  if (a.part) {
    // this K range's partial sums; split_reduce adds the ranges in order and
    // scales by s_a
    const OutRows pr = out_rows(a.part + size_t(blockIdx.z) * size_t(a.M) * size_t(a.N), false, a.M, a.N, m0,
                                32 * MS);
#pragma unroll
    for (int ms = 0; ms < MS; ++ms)
#pragma unroll
      for (int e = 0; e < 16; ++e) store_out(pr, a.N, n, ms, e, h, fmaf(so, acco[ms][e], gi * acc[ms][e]));
    return;
  }
  const RowScales<MS> rs = load_row_scales<MS>(a.s_a, a.M, m0, h);
  const OutRows yr = out_rows(a.Y, a.y_bf16, a.M, a.N, m0, 32 * MS);
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e)
      store_out(yr, a.N, n, ms, e, h, rs.v[ms][e] * fmaf(so, acco[ms][e], gi * acc[ms][e]));
}

// Split-K form for few tokens (M <= 64): one 32-row tile of W per workgroup,
// its NW waves take interleaved 128-K chunks (two chunks in flight per wave)
// and read their activations straight from L2 into registers; the wave
// partials are summed through LDS with a fixed-order tree at the end.  This
// keeps NT*NW waves in flight where the tiled form above would run only NT/4
// workgroups.
//
// Because the inlier scales travel inside the hi/lo fragments, the K order of
// an MFMA need not follow the 16-K scale blocks: MFMA i (0..7) of a chunk
// takes group i on lane half 0 and group 8 + i on lane half 1, so that each
// lane's activations for a chunk are 64 contiguous bytes (four 16-byte loads
// per 32-token sub-tile) and its group words two 16-byte runs.
template <int MS, int NI, bool OUT_INT8, int NW, int SF>
__global__ __launch_bounds__(NW * 64, 2) void int_mfma_splitk_kernel(MfmaArgs a) {
  constexpr bool SC8 = SF == kScaleE4M3;       // two-level: a power of two per row
  constexpr bool ONE = SF != kScaleF16;        // q * s exact in one fp16 fragment
  const int kSB = kTileN * a.srow;             // inlier scale bytes per (tile, chunk)
  constexpr int BM = 32 * MS;
  __shared__ float red[NW / 2][16][64];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = tid >> 6;  // (a wave-uniform copy makes the compiler spill at two sub-tiles)
  const int col = lane & 31, h = lane >> 5;
  const int m0 = blockIdx.y * BM;
  const int tile = blockIdx.x;
  const int KC = a.n_chunks;

  // groups 8h + i of row col: word ((h'*32 + col)*2 + h)*4 + q with i = 2q + h'.
  // Buffer resources over the tile's words and scales and over the block's
  // activation rows (rows past M read 0): wave-uniform bases, 32-bit offsets.
  const __amdgpu_buffer_rsrc_t wr =
      buffer_rsrc(a.blob + size_t(tile) * KC * kWordBytesPerTC, uint32_t(KC) * kWordBytesPerTC);
  const __amdgpu_buffer_rsrc_t sr =
      buffer_rsrc(a.blob + a.scales_off + size_t(tile) * KC * kSB, uint32_t(KC) * kSB);
  const __amdgpu_buffer_rsrc_t xr =
      buffer_rsrc(a.Xq + size_t(m0) * a.K, uint32_t(min(a.M - m0, BM)) * uint32_t(a.K));
  const uint32_t woff = uint32_t(col * 2 + h) * 16, soff = uint32_t(col) * uint32_t(a.srow);
  const uint32_t xoff = uint32_t(col) * uint32_t(a.K) + uint32_t(h) * 64;

  struct Stage {
    uint4 w0, w1, sc;   // words of h' = 0 and h' = 1, the row's scales of the chunk (from the low end)
    uint4 x[MS][4];     // 64 activation bytes per sub-tile
  };
  auto ld16 = [](__amdgpu_buffer_rsrc_t r, uint32_t v, uint32_t so) __attribute__((always_inline)) {
    typedef unsigned int u4_ __attribute__((ext_vector_type(4)));
    const u4_ q = __builtin_bit_cast(u4_, __builtin_amdgcn_raw_buffer_load_b128(r, v, so, 0));
    return make_uint4(q[0], q[1], q[2], q[3]);
  };
  auto load = [&](int cv, Stage& st) __attribute__((always_inline)) {
    // The chunk index derives from the wave index, which the compiler does
    // not know to be wave-uniform; read it into a scalar register here so
    // that the loads take it as their scalar offset (otherwise every load is
    // wrapped in a loop over the distinct values of its lanes).
    const int c = __builtin_amdgcn_readfirstlane(cv);
    st.w0 = ld16(wr, woff, uint32_t(c) * kWordBytesPerTC);
    st.w1 = ld16(wr, woff + 1024, uint32_t(c) * kWordBytesPerTC);
    // the row's scales of the chunk: a.srow bytes, naturally aligned
    if (a.srow == 16) {
      st.sc = ld16(sr, soff, uint32_t(c) * kSB);
    } else if (a.srow == 8) {
      typedef unsigned int u2_ __attribute__((ext_vector_type(2)));
      const u2_ q = __builtin_bit_cast(u2_, __builtin_amdgcn_raw_buffer_load_b64(sr, soff, uint32_t(c) * kSB, 0));
      st.sc = make_uint4(q[0], q[1], 0, 0);
    } else if (a.srow == 4) {
      st.sc = make_uint4(__builtin_amdgcn_raw_buffer_load_b32(sr, soff, uint32_t(c) * kSB, 0), 0, 0, 0);
    } else {
      st.sc = make_uint4(__builtin_amdgcn_raw_buffer_load_b16(sr, soff, uint32_t(c) * kSB, 0), 0, 0, 0);
    }
#pragma unroll
    for (int ms = 0; ms < MS; ++ms)
#pragma unroll
      for (int u = 0; u < 4; ++u)
        st.x[ms][u] = ld16(xr, xoff + uint32_t(ms * 32) * uint32_t(a.K) + u * 16, uint32_t(c) * kChunkK);
  };

  // the outlier branch: int8 outliers accumulate exactly in int32 through
  // the int8 matrix instruction (activation bytes as they are); e4m3
  // outliers through the f16 one
  typedef int i4v_ __attribute__((ext_vector_type(4)));
  typedef int i16v_ __attribute__((ext_vector_type(16)));
  using OAcc = std::conditional_t<OUT_INT8, i16v_, f16v>;
  f16v acc[MS];
  OAcc acco[MS];
#pragma unroll
  for (int s = 0; s < MS; ++s)
#pragma unroll
    for (int e = 0; e < 16; ++e) { acc[s][e] = 0.f; acco[s][e] = 0; }

  auto compute = [&](const Stage& st) {
    const uint32_t wv[2][4] = {{st.w0.x, st.w0.y, st.w0.z, st.w0.w}, {st.w1.x, st.w1.y, st.w1.z, st.w1.w}};
    const uint32_t sv[4] = {st.sc.x, st.sc.y, st.sc.z, st.sc.w};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t w = wv[i & 1][i >> 1];
      // the scale of 16-K block kb = 4h + (i >> 1) of group 8h + i
      const _Float16 s = block_scale<SF>(sv, 4 * h + (i >> 1), a.qs);
      h8 bh, bl;
      if constexpr (ONE) {
        const h8 sv8 = {s, s, s, s, s, s, s, s};
        bh = inlier_f16<NI>(w) * sv8;  // exact in fp16 (at most 7 significant bits)
      } else {
        scaled_hi_lo(inlier_f16<NI>(w), s, bh, bl);
      }
      h8 av[MS];
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const uint4 xv = st.x[ms][i >> 1];
        uint32_t a0, a1, a2, a3;
        i8x4_to_f16x4((i & 1) ? xv.z : xv.x, a0, a1);
        i8x4_to_f16x4((i & 1) ? xv.w : xv.y, a2, a3);
        const u4v av4 = {a0, a1, a2, a3};
        av[ms] = __builtin_bit_cast(h8, av4);
      }
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) acc[ms] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[ms], bh, acc[ms], 0, 0, 0);
      if constexpr (OUT_INT8) {
        // steps i, i + 1 (i even) in one int8 instruction over 32 K: a lane's
        // 16 activation bytes of the two groups are the uint4 st.x[ms][i/2]
        // as loaded, and its outlier bytes follow the same order
        if ((i & 1) == 0) {
          uint32_t o0, o1, o2, o3;
          outlier_i8(w, o0, o1);
          outlier_i8(wv[1][i >> 1], o2, o3);
          const i4v_ bo = {int(o0), int(o1), int(o2), int(o3)};
#pragma unroll
          for (int ms = 0; ms < MS; ++ms) {
            const uint4 xv = st.x[ms][i >> 1];
            const i4v_ ax = {int(xv.x), int(xv.y), int(xv.z), int(xv.w)};
            acco[ms] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ax, bo, acco[ms], 0, 0, 0);
          }
        }
      } else {
        const h8 bo = outlier_f16<false>(w);
#pragma unroll
        for (int ms = 0; ms < MS; ++ms) acco[ms] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[ms], bo, acco[ms], 0, 0, 0);
      }
      if constexpr (!ONE) {
#pragma unroll
        for (int ms = 0; ms < MS; ++ms) acc[ms] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[ms], bl, acc[ms], 0, 0, 0);
      }
    }
  };

  // two stages in flight: wave w takes chunks w, w + NW, w + 2 NW, ...; stage
  // s0 holds its even-numbered chunks and s1 its odd ones, each refilled
  // right after its products (a copy would wait for the load).  Loads past
  // the last chunk re-read it (in bounds, never used), so none is conditional.
  const int last = KC - 1;
  Stage s0, s1;
  load(min(wave, last), s0);
  load(min(wave + NW, last), s1);
  int c = wave;
  for (; c + NW < KC; c += 2 * NW) {  // one exit, so the accumulators stay in place
    compute(s0);
    load(min(c + 2 * NW, last), s0);
    compute(s1);
    load(min(c + 3 * NW, last), s1);
  }
  if (c < KC) compute(s0);  // a last chunk of odd rank

  // ---- tree over the waves: in round r, wave w + 2^r hands its partial to w
  // (the int32 outlier partials travel through the same buffer as bits)
  // (elements are copied to scalars first: a bit cast of a vector element
  // in place reads element 0)
  auto tree = [&](auto& v) __attribute__((always_inline)) {
#pragma unroll
    for (int stride = NW / 2; stride >= 1; stride >>= 1) {
      const bool sender = wave >= stride && wave < 2 * stride;
      if (sender) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const auto x = v[e];
          red[wave - stride][e][lane] = __builtin_bit_cast(float, x);
        }
      }
      __syncthreads();
      if (wave < stride) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float r = red[wave][e][lane];
          v[e] += __builtin_bit_cast(decltype(v[e] + 0), r);
        }
      }
      __syncthreads();
    }
  };
#pragma unroll
  for (int ms = 0; ms < MS; ++ms) {
    tree(acc[ms]);
    tree(acco[ms]);
  }
  if (wave > 0) return;
  const int n = tile * kTileN + col;
  if (n >= a.N) return;
  const float so = reinterpret_cast<const float*>(a.blob + a.rows_off)[n];
  const float gi = SC8 ? reinterpret_cast<const float*>(a.blob + a.irow_off)[n] : 1.f;  // a power of two
  const RowScales<MS> rs = load_row_scales<MS>(a.s_a, a.M, m0, h);
  const OutRows yr = out_rows(a.Y, a.y_bf16, a.M, a.N, m0, 32 * MS);
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e)
      store_out(yr, a.N, n, ms, e, h, rs.v[ms][e] * fmaf(so, float(acco[ms][e]), gi * acc[ms][e]));
}

template <int MS, int NI, int NW, int SF>
hipError_t launch_splitk(const Cfg& c, const MfmaArgs& a, hipStream_t st) {
  const dim3 grid(unsigned(a.n_tiles), unsigned((a.M + 32 * MS - 1) / (32 * MS)));
  const dim3 block(NW * 64);
  if (c.fmt_o == SDQ_FMT_INT8)
    hipLaunchKernelGGL((int_mfma_splitk_kernel<MS, NI, true, NW, SF>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((int_mfma_splitk_kernel<MS, NI, false, NW, SF>), grid, block, 0, st, a);
  return hipGetLastError();
}

// MS <= 2 (32 or 64 tokens per block): the split-K form; MS = 4: the tiled
// kernel.
template <int MS, int NI, int SF>
hipError_t launch_ms_ni(const Cfg& c, const MfmaArgs& a, hipStream_t st) {
  if constexpr (MS <= 2) {
    // split K inside the workgroup so that about 2048+ waves run
    const int64_t waves4 = int64_t(a.n_tiles) * 4 * ((a.M + 32 * MS - 1) / (32 * MS));
    if (waves4 >= 2048 || a.n_chunks < 16) return launch_splitk<MS, NI, 4, SF>(c, a, st);
    return launch_splitk<MS, NI, 8, SF>(c, a, st);
  } else {
    const dim3 grid(unsigned((a.n_tiles + kWaves - 1) / kWaves), unsigned((a.M + 32 * MS - 1) / (32 * MS)),
                    unsigned(a.k_ranges));
    const dim3 block(kThreads);
    if (c.fmt_o == SDQ_FMT_INT8)
      hipLaunchKernelGGL((int_mfma_kernel<MS, NI, true, SF>), grid, block, 0, st, a);
    else
      hipLaunchKernelGGL((int_mfma_kernel<MS, NI, false, SF>), grid, block, 0, st, a);
    return hipGetLastError();
  }
}

template <int MS, int SF>
hipError_t launch_ms_sc(const Cfg& c, const MfmaArgs& a, hipStream_t st) {
  if (c.n_i == 1) return launch_ms_ni<MS, 1, SF>(c, a, st);
  if (c.n_i == 2) return launch_ms_ni<MS, 2, SF>(c, a, st);
  return launch_ms_ni<MS, 3, SF>(c, a, st);
}

template <int MS>
hipError_t launch_ms(const Cfg& c, const MfmaArgs& a, hipStream_t st) {
  if (c.sc8) return launch_ms_sc<MS, kScaleE4M3>(c, a, st);
  if (c.e6m2) return launch_ms_sc<MS, kScaleE6M2>(c, a, st);
  return launch_ms_sc<MS, kScaleF16>(c, a, st);
}

// The tiled kernel over K ranges: S ranges of at least kSplitMinChunksTiled
// chunks, S chosen for about 512 workgroups (two per CU).
struct TiledSplit {
  int64_t groups, m_blocks, S, kc_range;
};
constexpr int64_t kSplitMinChunksTiled = 4;

TiledSplit tiled_split_shape(int64_t M, int64_t N, int64_t K) {
  TiledSplit t;
  t.groups = ((N + kTileN - 1) / kTileN + kWaves - 1) / kWaves;
  t.m_blocks = (M + 127) / 128;
  const int64_t kc = (K + kChunkK - 1) / kChunkK;
  const int64_t items = t.groups * t.m_blocks;
  int64_t S = (2 * kCUs + items - 1) / items;
  S = std::max<int64_t>(1, std::min<int64_t>(S, kc / kSplitMinChunksTiled));
  t.kc_range = (kc + S - 1) / S;
  t.S = (kc + t.kc_range - 1) / t.kc_range;  // no empty range
  return t;
}

}  // namespace

size_t int_tiled_split_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  return size_t(tiled_split_shape(M, N, K).S) * size_t(M) * size_t(N) * sizeof(float);
}

hipError_t launch_int_tiled_split(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                                  const uint8_t* blob, int64_t N, int64_t K, void* Y, void* workspace,
                                  hipStream_t st) {
  const Layout L = layout_for(c, N, K);
  const TiledSplit t = tiled_split_shape(M, N, K);
  MfmaArgs a{Xq, s_a, blob, Y, int(M), int(N), int(K), int(L.n_chunks), int(L.n_tiles),
             L.scales_off, L.rows_off, L.irow_off};
  a.qs = c.qv == 64 ? 2 : c.qv == 32 ? 1 : 0;
  a.srow = (kChunkK / c.qv) * c.scale_bytes();
  a.k_ranges = int(t.S);
  a.kc_range = int(t.kc_range);
  a.part = static_cast<float*>(workspace);
  const hipError_t e = launch_ms<4>(c, a, st);
  if (e != hipSuccess) return e;
  return launch_split_reduce(a.part, s_a, Y, M, N, int(t.S), c.y_bf16, st);
}

hipError_t launch_int_mfma(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                           const uint8_t* blob, int64_t N, int64_t K, void* Y, hipStream_t st) {
  const Layout L = layout_for(c, N, K);
  MfmaArgs a{Xq, s_a, blob, Y, int(M), int(N), int(K), int(L.n_chunks), int(L.n_tiles),
             L.scales_off, L.rows_off, L.irow_off};
  a.y_bf16 = c.y_bf16;
  a.qs = c.qv == 64 ? 2 : c.qv == 32 ? 1 : 0;
  a.srow = (kChunkK / c.qv) * c.scale_bytes();
  if (M <= 32) return launch_ms<1>(c, a, st);
  // 33..64 tokens: one 64-token block expands every weight once; when that
  // leaves fewer workgroups than compute units, two 32-token blocks fill the
  // GPU instead (each weight is then expanded twice)
  if (M <= 64) return L.n_tiles < kCUs ? launch_ms<1>(c, a, st) : launch_ms<2>(c, a, st);
  // More tokens: the tiled kernel (four row tiles x 128 tokens per
  // workgroup, two workgroups per CU) or the split-K form over 64-token
  // blocks, whichever this cost model says is faster.  A tiled workgroup
  // alone on a CU takes one unit of time and two sharing a CU take 1.7 units
  // (4096x4096: 85 us at 256 workgroups, 144 at 512), so a grid of w4
  // workgroups takes 1.7 units per full round of two per CU, plus 1.7 for a
  // last round of more than one per CU, or for at most one per CU 1 unit
  // alone and 0.65 after a full round (its workgroups start as the CUs of
  // the full round drain: 11008x4096 at M = 768, 512 + 4 workgroups, 200
  // us).  The split-K form costs about 1/200 unit per workgroup's worth of
  // work, with no rounds (4096x4096 at M = 768 / 1024 / 1536: 83 / 109 /
  // 158 us; tiled 84 / 85 / 132).
  const int64_t groups = (L.n_tiles + kWaves - 1) / kWaves;
  const int64_t w4 = groups * ((M + 127) / 128);
  const int64_t full = w4 / (2 * kCUs), rem = w4 % (2 * kCUs);
  const int64_t tail20 = rem == 0 ? 0 : rem > kCUs ? 34 : full > 0 ? 13 : 20;
  const int64_t tiled20 = 34 * full + tail20;            // tiled time x 20
  if (w4 < 10 * tiled20) return launch_ms<2>(c, a, st);  // w4 / 200 units < tiled
  return launch_ms<4>(c, a, st);
}

}  // namespace sdq
