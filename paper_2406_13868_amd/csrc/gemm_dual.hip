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
//     its two groups' (position, code) half-words into 16 dense bytes.
//     Lane half h covers K [16h, 16h + 16) of the 32-K step for both
//     operands (the K order inside the instruction is free as long as A and B
//     agree).
// The branches accumulate apart (fp32 and int32) and meet in the epilogue.
//
// A workgroup of four waves covers four 32-row tiles of W and 32*MS tokens;
// each wave owns one tile and all MS token sub-tiles.  Activations are read
// straight from L2 into registers (the four waves of a workgroup read the
// same lines, so the L1 cache serves most of them); each wave keeps two
// 128-K chunks of loads in flight.
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
  float* Y;
  int M, N, K, n_chunks, n_tiles;
  int64_t out_off, scale_off, rows_off;
};

__device__ __forceinline__ v4i ld16(__amdgpu_buffer_rsrc_t r, uint32_t v, uint32_t s) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, v, s, 0);
}
__device__ __forceinline__ int ld8(__amdgpu_buffer_rsrc_t r, uint32_t v, uint32_t s) {
  return int(__builtin_amdgcn_raw_buffer_load_b8(r, v, s, 0));
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

template <int MS>
__global__ __launch_bounds__(kDThreads, 1) void dual_mfma_kernel(DualArgs a) {
  constexpr int BM = 32 * MS;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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
  const __amdgpu_buffer_rsrc_t wo = buffer_rsrc(a.blob + a.out_off + size_t(tile) * KC * kDualOutBytesPerTC,
                                                uint32_t(KC) * kDualOutBytesPerTC);
  const __amdgpu_buffer_rsrc_t ws = buffer_rsrc(a.blob + a.scale_off + size_t(tile) * KC * kDualScaleBytesPerTC,
                                                uint32_t(KC) * kDualScaleBytesPerTC);

  struct Stage {
    v4i bi[2];        // fp4 inlier fragments of the two 64-K steps
    int sb[2];        // their e8m0 scales (block 2s + h of row col)
    uint32_t hw[4];   // outlier half-word pairs of the four 32-K steps
    v4i ai[MS][2];    // fp4 activations
    int sa[MS][2];    // their e8m0 scales
    v4i ao[MS][4];    // int8 activations
  };
  auto load = [&](int c, Stage& st) __attribute__((always_inline)) {
    const uint32_t cs = uint32_t(c);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      st.bi[s] = ld16(wn, uint32_t(s * 64 + lane) * 16u, cs * kDualNibBytesPerTC);
      st.sb[s] = ld8(ws, uint32_t(s * 64 + lane), cs * kDualScaleBytesPerTC);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      st.hw[u] = __builtin_amdgcn_raw_buffer_load_b32(wo, uint32_t(u * 64 + lane) * 4u, cs * kDualOutBytesPerTC, 0);
#pragma unroll
    for (int ms = 0; ms < MS; ++ms) {
      const uint32_t row = uint32_t(ms * 32 + col);
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        st.ai[ms][s] = ld16(xi, row * (K / 2) + uint32_t(s * 32 + h * 16), cs * (kChunkK / 2));
        st.sa[ms][s] = ld8(ea, row * (K / 32) + uint32_t(2 * s + h), cs * (kChunkK / 32));
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) st.ao[ms][u] = ld16(xo, row * K + uint32_t(u * 32 + h * 16), cs * kChunkK);
    }
  };

  v16f acc[MS];
  v16i acco[MS];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e) { acc[ms][e] = 0.f; acco[ms][e] = 0; }

  auto compute = [&](const Stage& st) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const v8i b = {st.bi[s][0], st.bi[s][1], st.bi[s][2], st.bi[s][3], 0, 0, 0, 0};
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const v8i av = {st.ai[ms][s][0], st.ai[ms][s][1], st.ai[ms][s][2], st.ai[ms][s][3], 0, 0, 0, 0};
        // fp4 (format 4) on both sides, each lane half with its block's scale
        acc[ms] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, b, acc[ms], 4, 4, 0, st.sa[ms][s], 0,
                                                                   st.sb[s]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const v4i bo = outlier_bytes(st.hw[u]);
#pragma unroll
      for (int ms = 0; ms < MS; ++ms)
        acco[ms] = __builtin_amdgcn_mfma_i32_32x32x32_i8(st.ao[ms][u], bo, acco[ms], 0, 0, 0);
    }
  };

  // two chunks in flight; loads past the last chunk re-read it (never used)
  Stage s0, s1;
  load(0, s0);
  load(min(1, last), s1);
  int c = 0;
  for (; c + 1 < KC; c += 2) {  // one exit, so the accumulators stay in place
    compute(s0);
    load(min(c + 2, last), s0);
    compute(s1);
    load(min(c + 3, last), s1);
  }
  if (c < KC) compute(s0);  // a last chunk of even rank

  if (!tile_ok) return;
  const int n = tile * kTileN + col;
  if (n >= a.N) return;
  const float so = reinterpret_cast<const float*>(a.blob + a.rows_off)[n];
  const RowScales<MS> rs = load_row_scales<MS>(a.s_a, a.M, m0, h);
  const __amdgpu_buffer_rsrc_t yr = out_rows(a.Y, a.M, a.N, m0, BM);
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e)
      store_out(yr, a.N, n, ms, e, h, fmaf(rs.v[ms][e], so * float(acco[ms][e]), acc[ms][e]));
}

template <int MS>
hipError_t launch_ms(const DualArgs& a, hipStream_t st) {
  const dim3 grid(unsigned((a.n_tiles + kDWaves - 1) / kDWaves), unsigned((a.M + 32 * MS - 1) / (32 * MS)));
  hipLaunchKernelGGL((dual_mfma_kernel<MS>), grid, dim3(kDThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_dual_mfma(const Cfg& c, const uint8_t* Xo, const float* s_a, const uint8_t* Xi,
                            const uint8_t* Ea, int64_t M, const uint8_t* blob, int64_t N, int64_t K,
                            float* Y, hipStream_t st) {
  (void)c;
  const DualLayout L = make_dual_layout(N, K);
  const DualArgs a{Xo, s_a, Xi, Ea, blob, Y, int(M), int(N), int(K), int(L.n_chunks), int(L.n_tiles),
                   L.out_off, L.scale_off, L.rows_off};
  if (M <= 32) return launch_ms<1>(a, st);
  if (M <= 64) return launch_ms<2>(a, st);
  return launch_ms<4>(a, st);
}

}  // namespace sdq
