// Dual-family decomposed GEMM: Section 5.1's worked configuration, in which
// the outliers (int8) multiply int8 activations A_o and the inliers (fp4)
// multiply fp4 activations A_i:
//   Y[m,n] = s_a[m] * s_o[n] * sum_k A_o[m,k] q_o[n,k]
//          + sum_k A_i[m,k] 2^Ea[m,k/32] * q_i[n,k] 2^Ei[n,k/32].
//
// On gfx950 both branches are matrix-core contractions:
//   * inliers: v_mfma_scale_f32_32x32x64_f8f6f4 with fp4 on both sides and
//     the two e8m0 scales applied inside the instruction.  The packer stores
//     the n_i:8 inliers as dense nibbles (zeros at the other positions) in
//     exactly the operand order, so the B fragment is one 16-byte load per
//     lane and needs no expansion;
//   * outliers: v_mfma_i32_32x32x32_i8, exact in int32.  Each lane expands
//     its two groups' (position, code) half-words into 16 dense bytes; with
//     2:8 outliers the second plane's half-words scatter into the same bytes
//     (the two positions of a group differ).
//     Lane half h covers K [16h, 16h + 16) of the 32-K step for both
//     operands (the K order inside the instruction is free as long as A and B
//     agree).
// The branches accumulate apart (fp32 and int32) and meet in the epilogue.
//
// A workgroup of four waves covers four 32-row tiles of W and 32*MS tokens;
// each wave owns one tile and all MS token sub-tiles.  The workgroup stages
// each 128-K chunk of both activation tensors in LDS once (double-buffered,
// one barrier per chunk) for its four waves; each wave streams its tile's
// weights into registers one chunk ahead.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "tile_out.h"

namespace sdq {
namespace {

constexpr int kDWaves = 4;
constexpr int kDThreads = kDWaves * 64;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));

struct DualArgs {
  const uint8_t* Xo;  // [M][K] int8 codes of A_o
  const float* s_a;   // [M] fp32 scales of A_o
  const uint8_t* Xi;  // [M][K/2] e2m1 codes of A_i, the even k in the low nibble
  const uint8_t* Ea;  // [M][K/32] e8m0 scales of A_i
  const uint8_t* blob;
  void* Y;
  int M, N, K, n_chunks, n_tiles;
  int64_t out_off, scale_off, rows_off;
  bool y_bf16 = false;  // Y as bf16
};

__device__ __forceinline__ v4i ld16(__amdgpu_buffer_rsrc_t r, uint32_t v, uint32_t s) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, v, s, 0);
}
__device__ __forceinline__ int ld8(__amdgpu_buffer_rsrc_t r, uint32_t v, uint32_t s) {
  return int(__builtin_amdgcn_raw_buffer_load_b8(r, v, s, 0));
}

// The four e8m0 scales of chunk cs of the A_i row at byte v of ea, block j
// in byte j.  One dword when K is a multiple of 128.  Otherwise a row's K/32
// bytes do not fill whole dwords, and a dword reaching past the end of the
// buffer's range would read as 0 whole: four byte loads, and 127 (2^0) for
// the blocks past K, whose weight codes are zero and add nothing whatever
// their scale.
__device__ __forceinline__ uint32_t ld_ea4(__amdgpu_buffer_rsrc_t ea, uint32_t v, uint32_t cs, uint32_t K) {
  if ((K & 127u) == 0) return __builtin_amdgcn_raw_buffer_load_b32(ea, v, cs * 4, 0);
  uint32_t e = 0;
#pragma unroll
  for (uint32_t j = 0; j < 4; ++j)
    e |= (cs * 4 + j < K / 32 ? uint32_t(__builtin_amdgcn_raw_buffer_load_b8(ea, v + j, cs * 4, 0)) : 127u)
         << (8 * j);
  return e;
}

// Dense int8 bytes of two 8-groups from their half-words (bits 0-2 position,
// bits 8-15 code): group i fills dwords 2i, 2i + 1.
__device__ __forceinline__ v4i outlier_bytes(uint32_t hw2) {
  const uint32_t v0 = hw2 & 0xFFFFu, v1 = hw2 >> 16;
  const uint32_t b0 = (v0 >> 8) << ((v0 & 3u) << 3), b1 = (v1 >> 8) << ((v1 & 3u) << 3);
  const bool u0 = (v0 & 4u) != 0, u1 = (v1 & 4u) != 0;
  const v4i r = {int(u0 ? 0u : b0), int(u0 ? b0 : 0u), int(u1 ? 0u : b1), int(u1 ? b1 : 0u)};
  return r;
}

// Outlier bytes per (tile, chunk) with NP half-word planes.
template <int NP>
constexpr uint32_t out_bytes_tc() { return uint32_t(NP) * kDualOutBytesPerTC; }

// Dense int8 outlier bytes of two groups from NP planes of half-word pairs.
template <int NP>
__device__ __forceinline__ v4i outlier_bytes_np(const uint32_t (&hw)[NP]) {
  v4i b = outlier_bytes(hw[0]);
  if constexpr (NP == 2) b |= outlier_bytes(hw[1]);
  return b;
}

// LDS rows of one 128-K chunk of activations, padded so that the 16-byte
// fragment reads of 8 consecutive rows fall on distinct banks.
constexpr int kRowO = kChunkK + 16;      // int8 codes of A_o: 144 bytes
constexpr int kRowI = kChunkK / 2 + 16;  // fp4 codes of A_i: 80 bytes

template <int MS, int NP>
__global__ __launch_bounds__(kDThreads, MS >= 4 ? 1 : 2) void dual_mfma_kernel(DualArgs a) {
  constexpr int BM = 32 * MS;
  // one chunk of the workgroup's activations, two buffers
  __shared__ __align__(16) uint8_t xo_s[2][BM * kRowO];
  __shared__ __align__(16) uint8_t xi_s[2][BM * kRowI];
  __shared__ __align__(16) uint32_t ea_s[2][BM];  // the four e8m0 bytes of a row's chunk

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, h = lane >> 5;
  const int m0 = blockIdx.y * BM;
  const int t_raw = blockIdx.x * kDWaves + wave;
  const bool tile_ok = t_raw < a.n_tiles;
  const int tile = min(t_raw, a.n_tiles - 1);  // a spare wave recomputes the last tile, stores nothing
  const int KC = a.n_chunks, last = KC - 1;
  const uint32_t K = uint32_t(a.K);

  // activations of the workgroup's rows (rows past M read 0)
  const uint32_t rows = uint32_t(min(a.M - m0, BM));
  const __amdgpu_buffer_rsrc_t xo = buffer_rsrc(a.Xo + size_t(m0) * K, rows * K);
  const __amdgpu_buffer_rsrc_t xi = buffer_rsrc(a.Xi + size_t(m0) * (K / 2), rows * (K / 2));
  const __amdgpu_buffer_rsrc_t ea = buffer_rsrc(a.Ea + size_t(m0) * (K / 32), rows * (K / 32));
  // the wave's tile: dense inlier nibbles, outlier half-words, inlier scales
  const __amdgpu_buffer_rsrc_t wn =
      buffer_rsrc(a.blob + size_t(tile) * KC * kDualNibBytesPerTC, uint32_t(KC) * kDualNibBytesPerTC);
  const __amdgpu_buffer_rsrc_t wo = buffer_rsrc(a.blob + a.out_off + size_t(tile) * KC * out_bytes_tc<NP>(),
                                                uint32_t(KC) * out_bytes_tc<NP>());
  const __amdgpu_buffer_rsrc_t ws = buffer_rsrc(a.blob + a.scale_off + size_t(tile) * KC * kDualScaleBytesPerTC,
                                                uint32_t(KC) * kDualScaleBytesPerTC);

  // ---- activation staging: thread tid moves 16-byte pieces tid + 256 i of
  //      the chunk (8 per row of A_o, 4 per row of A_i) and, below BM, the
  //      four scale bytes of row tid
  constexpr int kPo = BM * 8 / kDThreads;                       // BM * 8 >= 256
  constexpr int kPi = (BM * 4 + kDThreads - 1) / kDThreads;      // 128 pieces at BM = 32
  struct XRegs { v4i o[kPo]; v4i i[kPi]; uint32_t e; };
  auto load_x = [&](int c, XRegs& x) __attribute__((always_inline)) {
    const uint32_t cs = uint32_t(c);
#pragma unroll
    for (int j = 0; j < kPo; ++j) {
      const int p = tid + j * kDThreads;
      x.o[j] = ld16(xo, uint32_t(p >> 3) * K + uint32_t(p & 7) * 16, cs * kChunkK);
    }
#pragma unroll
    for (int j = 0; j < kPi; ++j) {
      const int p = tid + j * kDThreads;
      if (BM * 4 % kDThreads == 0 || p < BM * 4)
        x.i[j] = ld16(xi, uint32_t(p >> 2) * (K / 2) + uint32_t(p & 3) * 16, cs * (kChunkK / 2));
    }
    if (tid < BM) x.e = ld_ea4(ea, uint32_t(tid) * (K / 32), cs, K);
  };
  auto store_x = [&](int buf, const XRegs& x) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < kPo; ++j) {
      const int p = tid + j * kDThreads;
      *reinterpret_cast<v4i*>(&xo_s[buf][(p >> 3) * kRowO + (p & 7) * 16]) = x.o[j];
    }
#pragma unroll
    for (int j = 0; j < kPi; ++j) {
      const int p = tid + j * kDThreads;
      if (BM * 4 % kDThreads == 0 || p < BM * 4)
        *reinterpret_cast<v4i*>(&xi_s[buf][(p >> 2) * kRowI + (p & 3) * 16]) = x.i[j];
    }
    if (tid < BM) ea_s[buf][tid] = x.e;
  };

  // ---- the wave's weight stream, one chunk per stage
  struct BRegs {
    v4i bi[2];       // fp4 inlier fragments of the two 64-K steps
    int sb[2];       // their e8m0 scales (block 2s + h of row col)
    uint32_t hw[4][NP];  // outlier half-word pairs of the four 32-K steps, per plane
  };
  auto load_b = [&](int c, BRegs& st) __attribute__((always_inline)) {
    const uint32_t cs = uint32_t(c);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      st.bi[s] = ld16(wn, uint32_t(s * 64 + lane) * 16u, cs * kDualNibBytesPerTC);
      st.sb[s] = ld8(ws, uint32_t(s * 64 + lane), cs * kDualScaleBytesPerTC);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int p = 0; p < NP; ++p)
        st.hw[u][p] = __builtin_amdgcn_raw_buffer_load_b32(
            wo, uint32_t(p * kDualOutBytesPerTC) + uint32_t(u * 64 + lane) * 4u, cs * out_bytes_tc<NP>(), 0);
  };

  v16f acc[MS];
  v16i acco[MS];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e) { acc[ms][e] = 0.f; acco[ms][e] = 0; }

  auto compute = [&](int buf, const BRegs& st) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const v8i b = {st.bi[s][0], st.bi[s][1], st.bi[s][2], st.bi[s][3], 0, 0, 0, 0};
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const int r = ms * 32 + col;
        const v4i a4 = *reinterpret_cast<const v4i*>(&xi_s[buf][r * kRowI + s * 32 + h * 16]);
        const int sa = int((ea_s[buf][r] >> (8 * (2 * s + h))) & 0xFFu);
        const v8i av = {a4[0], a4[1], a4[2], a4[3], 0, 0, 0, 0};
        // fp4 (format 4) on both sides, each lane half with its block's scale
        acc[ms] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, b, acc[ms], 4, 4, 0, sa, 0, st.sb[s]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const v4i bo = outlier_bytes_np<NP>(st.hw[u]);
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const v4i ao = *reinterpret_cast<const v4i*>(&xo_s[buf][(ms * 32 + col) * kRowO + u * 32 + h * 16]);
        acco[ms] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ao, bo, acco[ms], 0, 0, 0);
      }
    }
  };

  // ---- pipeline: chunk c in LDS buffer c & 1 and weight stage c & 1; the
  //      activations of chunk c + 1 wait in registers and are stored after
  //      the products of chunk c.  Loads past the last chunk re-read it.
  XRegs X;
  BRegs B0, B1;
  load_x(0, X);
  load_b(0, B0);
  store_x(0, X);
  load_x(min(1, last), X);
  load_b(min(1, last), B1);
  __syncthreads();
  int c = 0;
  for (; c + 1 < KC; c += 2) {  // one exit, so the accumulators stay in place
    compute(0, B0);
    load_b(min(c + 2, last), B0);
    store_x(1, X);  // chunk c + 1 (buffer 1 was last read before the previous barrier)
    load_x(min(c + 2, last), X);
    __syncthreads();
    compute(1, B1);
    load_b(min(c + 3, last), B1);
    store_x(0, X);  // chunk c + 2
    load_x(min(c + 3, last), X);
    __syncthreads();
  }
  if (c < KC) compute(0, B0);  // a last chunk of even rank

  if (!tile_ok) return;
  const int n = tile * kTileN + col;
  if (n >= a.N) return;
  const float so = reinterpret_cast<const float*>(a.blob + a.rows_off)[n];
  const RowScales<MS> rs = load_row_scales<MS>(a.s_a, a.M, m0, h);
  const OutRows yr = out_rows(a.Y, a.y_bf16, a.M, a.N, m0, BM);
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e)
      store_out(yr, a.N, n, ms, e, h, fmaf(rs.v[ms][e], so * float(acco[ms][e]), acc[ms][e]));
}

// Split-K form for few tokens (up to 32, more on narrow layers): one 32-row tile per workgroup, its
// NW waves take interleaved 128-K chunks (two in flight per wave) and read
// their activations straight into registers; the wave partials of both
// accumulators are summed through LDS in a fixed-order tree.  This keeps
// n_tiles * NW waves streaming weights where the tiled form above would run
// only n_tiles / 4 workgroups.
template <int NW, int NP>
__global__ __launch_bounds__(NW * 64, 2) void dual_splitk_kernel(DualArgs a) {
  __shared__ float red[NW / 2][2][16][64];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, h = lane >> 5;
  const int m0 = blockIdx.y * 32;
  const int tile = blockIdx.x;
  const int KC = a.n_chunks, last = KC - 1;
  const uint32_t K = uint32_t(a.K);

  const uint32_t rows = uint32_t(min(a.M - m0, 32));
  const __amdgpu_buffer_rsrc_t xo = buffer_rsrc(a.Xo + size_t(m0) * K, rows * K);
  const __amdgpu_buffer_rsrc_t xi = buffer_rsrc(a.Xi + size_t(m0) * (K / 2), rows * (K / 2));
  const __amdgpu_buffer_rsrc_t ea = buffer_rsrc(a.Ea + size_t(m0) * (K / 32), rows * (K / 32));
  const __amdgpu_buffer_rsrc_t wn =
      buffer_rsrc(a.blob + size_t(tile) * KC * kDualNibBytesPerTC, uint32_t(KC) * kDualNibBytesPerTC);
  const __amdgpu_buffer_rsrc_t wo = buffer_rsrc(a.blob + a.out_off + size_t(tile) * KC * out_bytes_tc<NP>(),
                                                uint32_t(KC) * out_bytes_tc<NP>());
  const __amdgpu_buffer_rsrc_t ws = buffer_rsrc(a.blob + a.scale_off + size_t(tile) * KC * kDualScaleBytesPerTC,
                                                uint32_t(KC) * kDualScaleBytesPerTC);

  struct Stage {
    v4i bi[2];
    int sb[2];
    uint32_t hw[4][NP];
    v4i ai[2];
    uint32_t sa;  // the chunk's four e8m0 bytes of token row col
    v4i ao[4];
  };
  auto load = [&](int c, Stage& st) __attribute__((always_inline)) {
    const uint32_t cs = uint32_t(c);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      st.bi[s] = ld16(wn, uint32_t(s * 64 + lane) * 16u, cs * kDualNibBytesPerTC);
      st.sb[s] = ld8(ws, uint32_t(s * 64 + lane), cs * kDualScaleBytesPerTC);
      st.ai[s] = ld16(xi, uint32_t(col) * (K / 2) + uint32_t(s * 32 + h * 16), cs * (kChunkK / 2));
    }
    st.sa = ld_ea4(ea, uint32_t(col) * (K / 32), cs, K);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
#pragma unroll
      for (int p = 0; p < NP; ++p)
        st.hw[u][p] = __builtin_amdgcn_raw_buffer_load_b32(
            wo, uint32_t(p * kDualOutBytesPerTC) + uint32_t(u * 64 + lane) * 4u, cs * out_bytes_tc<NP>(), 0);
      st.ao[u] = ld16(xo, uint32_t(col) * K + uint32_t(u * 32 + h * 16), cs * kChunkK);
    }
  };

  v16f acc;
  v16i acco;
#pragma unroll
  for (int e = 0; e < 16; ++e) { acc[e] = 0.f; acco[e] = 0; }

  auto compute = [&](const Stage& st) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const v8i b = {st.bi[s][0], st.bi[s][1], st.bi[s][2], st.bi[s][3], 0, 0, 0, 0};
      const v8i av = {st.ai[s][0], st.ai[s][1], st.ai[s][2], st.ai[s][3], 0, 0, 0, 0};
      const int sa = int((st.sa >> (8 * (2 * s + h))) & 0xFFu);
      acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, b, acc, 4, 4, 0, sa, 0, st.sb[s]);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      acco = __builtin_amdgcn_mfma_i32_32x32x32_i8(st.ao[u], outlier_bytes_np<NP>(st.hw[u]), acco, 0, 0, 0);
  };

  // wave w takes chunks w, w + NW, ...; stage s0 its even-numbered ones and s1
  // the odd ones, each refilled right after its products; loads past the last
  // chunk re-read it (never used)
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
  if (c < KC) compute(s0);

  // ---- tree over the waves: in round r, wave w + 2^r hands its partials to w
#pragma unroll
  for (int stride = NW / 2; stride >= 1; stride >>= 1) {
    if (wave >= stride && wave < 2 * stride) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float x = acc[e];
        const int y = acco[e];
        red[wave - stride][0][e][lane] = x;
        red[wave - stride][1][e][lane] = __int_as_float(y);
      }
    }
    __syncthreads();
    if (wave < stride) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        acc[e] += red[wave][0][e][lane];
        acco[e] += __float_as_int(red[wave][1][e][lane]);
      }
    }
    __syncthreads();
  }
  if (wave > 0) return;
  const int n = tile * kTileN + col;
  if (n >= a.N) return;
  const float so = reinterpret_cast<const float*>(a.blob + a.rows_off)[n];
  const RowScales<1> rs = load_row_scales<1>(a.s_a, a.M, m0, h);
  const OutRows yr = out_rows(a.Y, a.y_bf16, a.M, a.N, m0, 32);
#pragma unroll
  for (int e = 0; e < 16; ++e) store_out(yr, a.N, n, 0, e, h, fmaf(rs.v[0][e], so * float(acco[e]), acc[e]));
}

template <int MS, int NP>
hipError_t launch_ms(const DualArgs& a, hipStream_t st) {
  const dim3 grid(unsigned((a.n_tiles + kDWaves - 1) / kDWaves), unsigned((a.M + 32 * MS - 1) / (32 * MS)));
  hipLaunchKernelGGL((dual_mfma_kernel<MS, NP>), grid, dim3(kDThreads), 0, st, a);
  return hipGetLastError();
}

// The split-K form up to 32 tokens, and beyond while its grid (one tile x 32
// tokens per workgroup) stays within one round, or two on long rows
// (measured: 4096x4096 at M = 48 / 64 takes 11.9 / 12.0 us against 18.8 in
// tiles, at 96 21.1 against 19.0; 4096x11008 at M = 64 / 96 / 128 takes 23.1
// / 41.7 / 42.6 against 48.6 / 48.5 / 48.7; 11008x4096 at M = 48 27.4
// against 22.6); else the tiled form (NP outlier planes).
template <int NP>
hipError_t launch_np(const DualArgs& a, hipStream_t st) {
  const int64_t split_grid = int64_t(a.n_tiles) * ((a.M + 31) / 32);
  if (a.M <= 32 || split_grid <= 256 || (a.K >= 8192 && split_grid <= 512)) {
    const dim3 grid(unsigned(a.n_tiles), unsigned((a.M + 31) / 32));
    hipLaunchKernelGGL((dual_splitk_kernel<4, NP>), grid, dim3(4 * 64), 0, st, a);
    return hipGetLastError();
  }
  // Tokens per workgroup: 32, 64 or 128 (one, two or four sub-tiles per
  // wave).  Larger blocks reuse every weight fragment for more tokens but
  // give fewer workgroups; the smallest block that leaves the GPU full wins.
  // Measured on the LLaMA-7B shapes: 4096x4096 at M = 128/256 takes 19/21 us
  // with 32-token blocks against 31/32 us with 128; 11008x4096 at M = 512
  // takes 60 us with 64-token blocks against 73 us with 128.
  const int64_t groups = (a.n_tiles + kDWaves - 1) / kDWaves;
  const int64_t M = a.M;
  if (groups * ((M + 31) / 32) <= 256) return launch_ms<1, NP>(a, st);
  if (groups * ((M + 63) / 64) <= 1024 && groups * ((M + 127) / 128) < 512) return launch_ms<2, NP>(a, st);
  return launch_ms<4, NP>(a, st);
}

}  // namespace

hipError_t launch_dual_mfma(const Cfg& c, const uint8_t* Xo, const float* s_a, const uint8_t* Xi,
                            const uint8_t* Ea, int64_t M, const uint8_t* blob, int64_t N, int64_t K,
                            void* Y, hipStream_t st) {
  const DualLayout L = make_dual_layout(N, K, c.n_o);
  DualArgs a{Xo, s_a, Xi, Ea, blob, Y, int(M), int(N), int(K), int(L.n_chunks), int(L.n_tiles),
             L.out_off, L.scale_off, L.rows_off};
  a.y_bf16 = c.y_bf16;
  if (dual_decode_fits(M, N, K)) return launch_dual_decode(c, Xo, s_a, Xi, Ea, M, blob, N, K, Y, st);
  return L.out_planes == 2 ? launch_np<2>(a, st) : launch_np<1>(a, st);
}

}  // namespace sdq
