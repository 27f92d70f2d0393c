// INT-family decomposed GEMM for tens to a few hundred tokens, with K split
// across workgroups.  Section 5.1: Y = SpMM(A, W_o) + SpMM(A, W_i), one fp32
// result per output, here summed over K ranges in a fixed order.
//
// Both branches run on the f16 and int8 matrix instructions as in
// gemm_int_mfma.hip (exact products: the inlier scale rides inside two fp16
// fragments, hi and lo; int8 outliers accumulate in int32, e4m3 ones in
// fp32).  What differs is the sharing of the activations:
//   - a workgroup of 4 waves owns 4 row tiles of W (128 outputs), BM = 32*MS
//     tokens and one range of 128-K chunks;
//   - each chunk of activations is loaded once per workgroup, converted from
//     int8 to f16 once, and kept in LDS (both forms: the int8 outlier
//     instruction reads the bytes) for all four waves.  A wave of the
//     single-tile split-K kernel converts every chunk it uses by itself, a
//     quarter of its vector instructions at 64 tokens;
//   - the K ranges of one row group go to different workgroups, so that every
//     shape fills the GPU: 4096 outputs are 32 row groups, which alone would
//     occupy 32 of the 256 compute units.
// Each workgroup writes its partial sums s_o*acc_o + g*acc for its K range to
// the workspace; a second kernel adds the partials of every output in range
// order and scales by s_a.  The result does not depend on the scheduling.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "int_frag.h"
#include "kernels.h"
#include "tile_out.h"

namespace sdq {
namespace {

using namespace intfrag;

constexpr int kSplitWaves = 4;                    // row tiles per workgroup, one per wave
constexpr int kSplitThreads = kSplitWaves * 64;
constexpr int kI8Row = kChunkK + 16;              // LDS bytes per token row, int8 activations
constexpr int kF16Row = kChunkK + 8;              // LDS f16 elements per token row
constexpr int kSplitTargetWaves = 2048;           // two waves per SIMD
constexpr int kSplitMinChunks = 4;                // chunks per K range, at least

struct SplitArgs {
  const uint8_t* Xq;
  const uint8_t* blob;
  float* part;  // [S][M][N] fp32 partial sums
  int M, N, K, n_chunks, n_tiles;
  int G, S, MB;  // row groups, K ranges, token blocks
  int64_t scales_off, rows_off, irow_off;
  int qs, srow;
};

template <int MS, int NI, bool OUT_INT8, int SF>
__global__ __launch_bounds__(kSplitThreads) void int_split_kernel(SplitArgs a) {
  constexpr bool SC8 = SF == kScaleE4M3;  // two-level: a power of two per row
  constexpr bool ONE = SF != kScaleF16;   // q * s exact in one fp16 fragment
  constexpr int BM = 32 * MS;
  constexpr int kI8Bytes = OUT_INT8 ? BM * kI8Row : 16;
  __shared__ __align__(16) uint8_t xi8[2][kI8Bytes];
  __shared__ __align__(16) _Float16 xf16[2][BM * kF16Row];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, h = lane >> 5;
  // (row group, K range, token block); the workgroups of one K range and
  // token block are contiguous, so each XCD's L2 holds few activation slices
  const int L = xcd_contiguous(blockIdx.x, a.G * a.S * a.MB);
  const int g = L % a.G, rest = L / a.G, p = rest % a.S, mb = rest / a.S;
  const int m0 = mb * BM;
  const int c0 = int(int64_t(p) * a.n_chunks / a.S), c1 = int(int64_t(p + 1) * a.n_chunks / a.S);
  const int last = c1 - 1;
  const int tile = g * kSplitWaves + wave;
  const bool tile_ok = tile < a.n_tiles;
  const int kSB = kTileN * a.srow;

  auto ld16 = [](__amdgpu_buffer_rsrc_t r, uint32_t v, uint32_t so) __attribute__((always_inline)) {
    typedef unsigned int u4_ __attribute__((ext_vector_type(4)));
    const u4_ q = __builtin_bit_cast(u4_, __builtin_amdgcn_raw_buffer_load_b128(r, v, so, 0));
    return make_uint4(q[0], q[1], q[2], q[3]);
  };

  // ---- activations: BM token rows x 128 bytes per chunk, MS pieces of 16
  // bytes per thread (piece pc: token pc >> 3, bytes 16*(pc & 7)); rows past
  // M read 0 through the buffer resource
  const __amdgpu_buffer_rsrc_t xr =
      buffer_rsrc(a.Xq + size_t(m0) * a.K, uint32_t(min(a.M - m0, BM)) * uint32_t(a.K));
  uint4 xs[MS];
  auto load_x = [&](int c) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < MS; ++i) {
      const int pc = tid + i * kSplitThreads;
      xs[i] = ld16(xr, uint32_t(pc >> 3) * uint32_t(a.K) + uint32_t(pc & 7) * 16u, uint32_t(c) * kChunkK);
    }
  };
  auto store_x = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < MS; ++i) {
      const int pc = tid + i * kSplitThreads;
      const int r = pc >> 3, cp = pc & 7;
      if constexpr (OUT_INT8) *reinterpret_cast<uint4*>(&xi8[buf][r * kI8Row + cp * 16]) = xs[i];
      uint32_t o[8];
      i8x4_to_f16x4(xs[i].x, o[0], o[1]);
      i8x4_to_f16x4(xs[i].y, o[2], o[3]);
      i8x4_to_f16x4(xs[i].z, o[4], o[5]);
      i8x4_to_f16x4(xs[i].w, o[6], o[7]);
      uint4* dst = reinterpret_cast<uint4*>(&xf16[buf][r * kF16Row + cp * 16]);
      dst[0] = make_uint4(o[0], o[1], o[2], o[3]);
      dst[1] = make_uint4(o[4], o[5], o[6], o[7]);
    }
  };

  // ---- this wave's tile: lane (col, h) takes groups 8h .. 8h+7 of row col
  // of every chunk, as in the split-K kernel (two 16-byte runs of words and
  // the row's scales of the chunk)
  const int t_ld = tile_ok ? tile : 0;
  const __amdgpu_buffer_rsrc_t wr =
      buffer_rsrc(a.blob + size_t(t_ld) * a.n_chunks * kWordBytesPerTC, uint32_t(a.n_chunks) * kWordBytesPerTC);
  const __amdgpu_buffer_rsrc_t sr =
      buffer_rsrc(a.blob + a.scales_off + size_t(t_ld) * a.n_chunks * kSB, uint32_t(a.n_chunks) * kSB);
  const uint32_t woff = uint32_t(col * 2 + h) * 16, soff = uint32_t(col) * uint32_t(a.srow);
  struct Stage {
    uint4 w0, w1, sc;
  };
  auto load_w = [&](int c, Stage& st) __attribute__((always_inline)) {
    st.w0 = ld16(wr, woff, uint32_t(c) * kWordBytesPerTC);
    st.w1 = ld16(wr, woff + 1024, uint32_t(c) * kWordBytesPerTC);
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
  };

  typedef int i4v_ __attribute__((ext_vector_type(4)));
  typedef int i16v_ __attribute__((ext_vector_type(16)));
  using OAcc = std::conditional_t<OUT_INT8, i16v_, f16v>;
  f16v acc[MS];
  OAcc acco[MS];
#pragma unroll
  for (int s = 0; s < MS; ++s)
#pragma unroll
    for (int e = 0; e < 16; ++e) { acc[s][e] = 0.f; acco[s][e] = 0; }

  // MFMA i (0..7) of a chunk takes group 8h + i on lane half h: its
  // activations are the f16 row elements 64h + 8i .. +8 of token col
  auto compute = [&](const Stage& st, int buf) __attribute__((always_inline)) {
    const uint32_t wv[2][4] = {{st.w0.x, st.w0.y, st.w0.z, st.w0.w}, {st.w1.x, st.w1.y, st.w1.z, st.w1.w}};
    const uint32_t sv[4] = {st.sc.x, st.sc.y, st.sc.z, st.sc.w};
    _Float16 sb[4];  // the scales of blocks 4h .. 4h + 3, once per chunk
#pragma unroll
    for (int q = 0; q < 4; ++q) sb[q] = block_scale<SF>(sv, 4 * h + q, a.qs);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t w = wv[i & 1][i >> 1];
      const _Float16 s = sb[i >> 1];
      h8 bh, bl;
      if constexpr (ONE) {
        const h8 sv8 = {s, s, s, s, s, s, s, s};
        bh = inlier_f16<NI>(w) * sv8;  // exact in fp16 (at most 7 significant bits)
      } else {
        scaled_hi_lo(inlier_f16<NI>(w), s, bh, bl);
      }
      h8 av[MS];
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
        av[ms] = *reinterpret_cast<const h8*>(&xf16[buf][(ms * 32 + col) * kF16Row + 64 * h + 8 * i]);
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) acc[ms] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[ms], bh, acc[ms], 0, 0, 0);
      if constexpr (OUT_INT8) {
        // steps i, i + 1 (i even) in one int8 instruction over 32 K: the
        // lane's 16 activation bytes 64h + 8i .. +16 and its outlier bytes
        // of the two groups in the same order
        if ((i & 1) == 0) {
          uint32_t o0, o1, o2, o3;
          outlier_i8(w, o0, o1);
          outlier_i8(wv[1][i >> 1], o2, o3);
          const i4v_ bo = {int(o0), int(o1), int(o2), int(o3)};
#pragma unroll
          for (int ms = 0; ms < MS; ++ms) {
            const uint4 xv = *reinterpret_cast<const uint4*>(&xi8[buf][(ms * 32 + col) * kI8Row + 64 * h + 8 * i]);
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

  // Chunk c sits in LDS buffer (c - c0) & 1 and weight stage s0 or s1 by the
  // same parity.  Each step requests the activations of the next chunk and
  // the words two chunks ahead, multiplies, then converts the next chunk
  // into the other buffer (which every wave finished reading before the
  // previous barrier).  Requests past the range re-read its last chunk (in
  // bounds, never used), so none is conditional.
  Stage s0, s1;
  load_x(c0);
  load_w(c0, s0);
  load_w(min(c0 + 1, last), s1);
  store_x(0);
  __syncthreads();
  int c = c0;
  for (; c + 1 < c1; c += 2) {  // one exit, so the accumulators stay in place
    load_x(c + 1);
    if (tile_ok) compute(s0, 0);
    load_w(min(c + 2, last), s0);
    store_x(1);
    __syncthreads();
    load_x(min(c + 2, last));
    if (tile_ok) compute(s1, 1);
    load_w(min(c + 3, last), s1);
    store_x(0);
    __syncthreads();
  }
  if (c < c1 && tile_ok) compute(s0, 0);  // a last chunk of even rank

  if (!tile_ok) return;
  const int n = tile * kTileN + col;
  if (n >= a.N) return;
  const float so = reinterpret_cast<const float*>(a.blob + a.rows_off)[n];
  const float gi = SC8 ? reinterpret_cast<const float*>(a.blob + a.irow_off)[n] : 1.f;  // a power of two
  const OutRows yr = out_rows(a.part + size_t(p) * size_t(a.M) * size_t(a.N), false, a.M, a.N, m0, BM);
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e) store_out(yr, a.N, n, ms, e, h, fmaf(so, float(acco[ms][e]), gi * acc[ms][e]));
}

// Y[m, n] = s_a[m] * (part[0][m, n] + part[1][m, n] + ... ) in range order,
// four outputs per thread (V4: N a multiple of 4, so they share a row).  The
// partial sums of up to 16 ranges are requested together before any is
// added (one memory round trip instead of one per range).
template <bool V4>
__global__ __launch_bounds__(256) void split_reduce(const float* part, const float* s_a, void* Y, int M,
                                                        int N, int S, bool y_bf16) {
  const size_t MN = size_t(M) * size_t(N);
  const size_t i0 = (size_t(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (i0 >= MN) return;
  if constexpr (V4) {
    constexpr int kMaxS = 16;
    float4 u[kMaxS];
#pragma unroll
    for (int q = 0; q < kMaxS; ++q)
      if (q < S) u[q] = *reinterpret_cast<const float4*>(part + size_t(q) * MN + i0);
    float4 v = u[0];
#pragma unroll
    for (int q = 1; q < kMaxS; ++q)
      if (q < S) { v.x += u[q].x; v.y += u[q].y; v.z += u[q].z; v.w += u[q].w; }
    for (int q = kMaxS; q < S; ++q) {  // more ranges than the requests above hold
      const float4 w = *reinterpret_cast<const float4*>(part + size_t(q) * MN + i0);
      v.x += w.x; v.y += w.y; v.z += w.z; v.w += w.w;
    }
    const float sa = s_a[i0 / size_t(N)];
    if (y_bf16) {
      const uint32_t lo = uint32_t(bf16_bits(sa * v.x)) | (uint32_t(bf16_bits(sa * v.y)) << 16);
      const uint32_t hi = uint32_t(bf16_bits(sa * v.z)) | (uint32_t(bf16_bits(sa * v.w)) << 16);
      *reinterpret_cast<uint2*>(static_cast<unsigned short*>(Y) + i0) = make_uint2(lo, hi);
    } else {
      *reinterpret_cast<float4*>(static_cast<float*>(Y) + i0) = make_float4(sa * v.x, sa * v.y, sa * v.z, sa * v.w);
    }
  } else {
    for (size_t i = i0; i < min(i0 + 4, MN); ++i) {
      float v = part[i];
      for (int q = 1; q < S; ++q) v += part[size_t(q) * MN + i];
      store_y(Y, y_bf16, i, s_a[i / size_t(N)] * v);
    }
  }
}

struct SplitShape {
  int MS, MB, G, S;
};

SplitShape split_shape(int64_t M, int64_t N, int64_t K) {
  SplitShape s;
  s.MS = M <= 32 ? 1 : 2;
  s.MB = int((M + 32 * s.MS - 1) / (32 * s.MS));
  const int64_t tiles = (N + kTileN - 1) / kTileN;
  s.G = int((tiles + kSplitWaves - 1) / kSplitWaves);
  const int64_t kc = (K + kChunkK - 1) / kChunkK;
  const int64_t per_range = int64_t(kSplitWaves) * s.G * std::max(s.MB, 1);  // waves per K range
  int64_t S = (kSplitTargetWaves + per_range - 1) / per_range;
  S = std::min<int64_t>(S, std::max<int64_t>(1, kc / kSplitMinChunks));
  s.S = int(std::max<int64_t>(S, 1));
  return s;
}

template <int MS, int NI, int SF>
hipError_t launch_split_kernel(const Cfg& c, const SplitArgs& a, hipStream_t st) {
  const dim3 grid(unsigned(a.G * a.S * a.MB)), block(kSplitThreads);
  if (c.fmt_o == SDQ_FMT_INT8)
    hipLaunchKernelGGL((int_split_kernel<MS, NI, true, SF>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((int_split_kernel<MS, NI, false, SF>), grid, block, 0, st, a);
  return hipGetLastError();
}

template <int MS, int SF>
hipError_t launch_split_ni(const Cfg& c, const SplitArgs& a, hipStream_t st) {
  if (c.n_i == 1) return launch_split_kernel<MS, 1, SF>(c, a, st);
  if (c.n_i == 2) return launch_split_kernel<MS, 2, SF>(c, a, st);
  return launch_split_kernel<MS, 3, SF>(c, a, st);
}

template <int MS>
hipError_t launch_split_ms(const Cfg& c, const SplitArgs& a, hipStream_t st) {
  if (c.sc8) return launch_split_ni<MS, kScaleE4M3>(c, a, st);
  if (c.e6m2) return launch_split_ni<MS, kScaleE6M2>(c, a, st);
  return launch_split_ni<MS, kScaleF16>(c, a, st);
}

}  // namespace

// The tiled kernel's 128-token blocks expand every weight once per 128
// tokens where this kernel's 64-token blocks expand it twice, but give half
// as many workgroups per K range, so more ranges and partial sums.  Measured
// (tiled over K ranges against this kernel): it wins on long rows and wide
// layers (4096x11008 at M = 256: 64.7 against 71.5 us; 16384x4096 at M =
// 256: 86.5 against 94.2; 11008x4096 at M = 128: 43.0 against 50.7) and
// above 256 tokens (4096x4096 at M = 384 / 512: 42.5 / 47.8 against 46.9 /
// 51.9), and loses on 4096x4096 at M = 256 (35.4 against 31.2) and on
// 11008x4096 at M = 192 / 256 (76.6 / 78.7 against 69.6 / 75.2).
bool int_split_tiled(int64_t M, int64_t N, int64_t K) {
  if (M <= 64) return false;
  return M > kSplitMaxM || K >= 8192 || N >= 16384 || (M <= 128 && N >= 8192);
}

size_t int_split_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  if (int_split_tiled(M, N, K)) return int_tiled_split_workspace_bytes(M, N, K);
  const SplitShape s = split_shape(M, N, K);
  return size_t(s.S) * size_t(M) * size_t(N) * sizeof(float);
}

hipError_t launch_int_split(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                            const uint8_t* blob, int64_t N, int64_t K, void* Y, void* workspace,
                            hipStream_t st) {
  if (int_split_tiled(M, N, K)) return launch_int_tiled_split(c, Xq, s_a, M, blob, N, K, Y, workspace, st);
  const Layout L = layout_for(c, N, K);
  const SplitShape sh = split_shape(M, N, K);
  SplitArgs a{Xq, blob, static_cast<float*>(workspace), int(M), int(N), int(K), int(L.n_chunks),
              int(L.n_tiles), sh.G, sh.S, sh.MB, L.scales_off, L.rows_off, L.irow_off,
              c.qv == 64 ? 2 : c.qv == 32 ? 1 : 0, int((kChunkK / c.qv) * c.scale_bytes())};
  const hipError_t e = sh.MS == 1 ? launch_split_ms<1>(c, a, st) : launch_split_ms<2>(c, a, st);
  if (e != hipSuccess) return e;
  return launch_split_reduce(a.part, s_a, Y, M, N, sh.S, c.y_bf16, st);
}

hipError_t launch_split_reduce(const float* part, const float* s_a, void* Y, int64_t M, int64_t N, int S,
                               bool y_bf16, hipStream_t st) {
  const size_t MN = size_t(M) * size_t(N);
  const dim3 grid(unsigned((MN + 1023) / 1024)), block(256);
  if (N % 4 == 0)
    hipLaunchKernelGGL(split_reduce<true>, grid, block, 0, st, part, s_a, Y, int(M), int(N), S, y_bf16);
  else
    hipLaunchKernelGGL(split_reduce<false>, grid, block, 0, st, part, s_a, Y, int(M), int(N), S, y_bf16);
  return hipGetLastError();
}

}  // namespace sdq
