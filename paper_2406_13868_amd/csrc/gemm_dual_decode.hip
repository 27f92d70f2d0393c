// Dual-family decomposed GEMM for one or two tokens (decode): a
// weight-streaming vector kernel.  Section 5.1's worked configuration:
//   Y[m,n] = s_a[m] * s_o[n] * sum_k A_o[m,k] q_o[n,k]
//          + sum_k A_i[m,k] 2^Ea[m,k/32] * q_i[n,k] 2^Ei[n,k/32].
//
// At M <= 2 the product is bound by the stream of packed weights; the matrix
// kernels would leave 31 of every 32 operand rows empty.  Here:
//   * a wave covers an 8-row slice of W and a part of K; lane l takes row
//     l & 7 of the slice, 32-K block (l >> 3) & 3 of a 128-K chunk and chunk
//     l >> 5 of each two-chunk step, so that one 16-byte load per lane reads
//     the slice's inlier nibbles of eight chunk-blocks as full 128-byte lines;
//   * inliers: v_cvt_scalef32_pk_f16_fp4 turns two e2m1 codes into two f16
//     values on both sides, and v_dot2 sums a block's 32 products in fp32,
//     exactly (every product is a multiple of 1/4 below 37, every block sum
//     below 2^11); the block sum is then scaled by 2^(Ea + Ei) and added to
//     the fp32 accumulator;
//   * outliers: each (position, code) half-word becomes a v_perm selector that
//     picks the group's int8 activation, and v_dot4 multiplies it by the
//     code into an exact int32 accumulator (with 2:8 outliers, once for each
//     of the two half-word planes);
//   * the eight lanes of a row are summed by three fixed butterfly steps and
//     the K parts in a fixed order through LDS, so the result does not depend
//     on timing.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "tile_out.h"

namespace sdq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));

constexpr int kSliceRowsD = 8;     // rows of W per wave
constexpr int kDecTokensMax = 2;

// Waves (parts of K) a workgroup may hold: 16 where a wave's registers fit a
// quarter of a SIMD (128), else 8.
constexpr int max_parts(int MT, int S) { return MT * S <= 4 ? 16 : 8; }

struct DualDecArgs {
  const uint8_t* Xo;  // [M][K] int8 codes of A_o
  const float* s_a;   // [M] fp32 scales of A_o
  const uint8_t* Xi;  // [M][K/2] e2m1 codes of A_i, the even k in the low nibble
  const uint8_t* Ea;  // [M][K/32] e8m0 scales of A_i
  const uint8_t* blob;
  void* Y;
  int M, N, K, n_chunks, n_slices, parts;
  int64_t out_off, scale_off, rows_off;
  bool y_bf16;
};

__device__ __forceinline__ v4i ld16(__amdgpu_buffer_rsrc_t r, uint32_t v) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, v, 0, 0);
}
__device__ __forceinline__ uint32_t ld32(__amdgpu_buffer_rsrc_t r, uint32_t v) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, v, 0, 0);
}
__device__ __forceinline__ uint32_t ld8(__amdgpu_buffer_rsrc_t r, uint32_t v) {
  return uint32_t(__builtin_amdgcn_raw_buffer_load_b8(r, v, 0, 0));
}

// Sum over the 32 products of one block: 16 e2m1 bytes of weights against 16
// of activations, as f16 pairs; four chains keep the dot products apart.
__device__ __forceinline__ float block_dot(const v4i w, const v4i x) {
  float s[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const uint32_t wd = uint32_t(w[d]), xd = uint32_t(x[d]);
    s[0] = __builtin_amdgcn_fdot2(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(wd, 1.f, 0),
                                  __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(xd, 1.f, 0), s[0], false);
    s[1] = __builtin_amdgcn_fdot2(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(wd, 1.f, 1),
                                  __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(xd, 1.f, 1), s[1], false);
    s[2] = __builtin_amdgcn_fdot2(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(wd, 1.f, 2),
                                  __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(xd, 1.f, 2), s[2], false);
    s[3] = __builtin_amdgcn_fdot2(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(wd, 1.f, 3),
                                  __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(xd, 1.f, 3), s[3], false);
  }
  return (s[0] + s[1]) + (s[2] + s[3]);
}

// int8 product of one 8-group: the half-word's code times the activation at
// its position (bytes lo:hi of the group's eight activation bytes).
__device__ __forceinline__ int outlier_dot(uint32_t hw, uint32_t lo, uint32_t hi, int acc) {
  const uint32_t sel = (hw & 7u) | 0x0C0C0C00u;  // bytes 1-3 read as zero
  const uint32_t a = __builtin_amdgcn_perm(hi, lo, sel);
  return __builtin_amdgcn_sdot4(int(a), int((hw >> 8) & 0xFFu), acc, false);
}

// MT tokens, S two-chunk steps per wave, NP outlier half-word planes.
template <int MT, int S, int NP>
__global__ __launch_bounds__(max_parts(MT, S) * 64) void dual_decode_kernel(DualDecArgs a) {
  constexpr uint32_t kOutTC = uint32_t(NP) * kDualOutBytesPerTC;  // outlier bytes per (tile, chunk)
  __shared__ float part[max_parts(MT, S)][MT][kSliceRowsD][2];

  const int lane = threadIdx.x & 63;
  const int kq = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // part of K
  const int rr = lane & 7, b = (lane >> 3) & 3, cc = lane >> 5;
  const int slice = xcd_contiguous(blockIdx.x, gridDim.x);
  const int t = slice >> 2;                      // 32-row tile
  const int r = ((slice & 3) << 3) + rr;         // row inside the tile
  const int KC = a.n_chunks, K = a.K;

  const __amdgpu_buffer_rsrc_t wn = buffer_rsrc(a.blob + size_t(t) * KC * kDualNibBytesPerTC,
                                                uint32_t(KC) * kDualNibBytesPerTC);
  const __amdgpu_buffer_rsrc_t wo = buffer_rsrc(a.blob + a.out_off + size_t(t) * KC * kOutTC, uint32_t(KC) * kOutTC);
  const __amdgpu_buffer_rsrc_t ws = buffer_rsrc(a.blob + a.scale_off + size_t(t) * KC * kDualScaleBytesPerTC,
                                                uint32_t(KC) * kDualScaleBytesPerTC);
  const uint32_t rows = uint32_t(a.M);
  const __amdgpu_buffer_rsrc_t xo = buffer_rsrc(a.Xo, rows * uint32_t(K));
  const __amdgpu_buffer_rsrc_t xi = buffer_rsrc(a.Xi, rows * uint32_t(K / 2));
  const __amdgpu_buffer_rsrc_t ea = buffer_rsrc(a.Ea, rows * uint32_t(K / 32));

  // ---- every load of the wave first: weights, then activations (chunks
  //      past K re-read the last one and are multiplied by zero activations)
  struct W { v4i nib; uint32_t hw[NP][2]; uint32_t e; };
  struct X { v4i ai; v4i ao[2]; uint32_t e; };
  W w[S];
  X x[S][MT];
  bool live[S];
#pragma unroll
  for (int d = 0; d < S; ++d) {
    const int c = kq * 2 * S + 2 * d + cc;
    live[d] = c < KC;
    const uint32_t ce = uint32_t(min(c, KC - 1));
    w[d].nib = ld16(wn, ce * kDualNibBytesPerTC + uint32_t(b * 32 + r) * 16u);
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
        w[d].hw[p][hh] = ld32(wo, ce * kOutTC + uint32_t(p * kDualOutBytesPerTC) + uint32_t((b * 2 + hh) * 32 + r) * 4u);
    w[d].e = ld8(ws, ce * kDualScaleBytesPerTC + uint32_t(b * 32 + r));
  }
#pragma unroll
  for (int d = 0; d < S; ++d) {
    const uint32_t ce = uint32_t(min(kq * 2 * S + 2 * d + cc, KC - 1));
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      // rows past M read zeros (the buffer resource ends at row M)
      const uint32_t mo = uint32_t(m) * uint32_t(K);
      x[d][m].ai = ld16(xi, mo / 2 + ce * (kChunkK / 2) + uint32_t(b) * 16u);
      x[d][m].ao[0] = ld16(xo, mo + ce * kChunkK + uint32_t(b) * 32u);
      x[d][m].ao[1] = ld16(xo, mo + ce * kChunkK + uint32_t(b) * 32u + 16u);
      x[d][m].e = ld8(ea, mo / 32 + ce * (kChunkK / 32) + uint32_t(b));
    }
  }

  // ---- products
  float acc[MT];
  int acco[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) { acc[m] = 0.f; acco[m] = 0; }
#pragma unroll
  for (int d = 0; d < S; ++d) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const X& xv = x[d][m];
      const float p = live[d] ? block_dot(w[d].nib, xv.ai) : 0.f;
      acc[m] += __builtin_ldexpf(p, int(xv.e + w[d].e) - 254);
      if (live[d]) {
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const uint32_t h2w = w[d].hw[p][hh];
            acco[m] = outlier_dot(h2w & 0xFFFFu, uint32_t(xv.ao[hh][0]), uint32_t(xv.ao[hh][1]), acco[m]);
            acco[m] = outlier_dot(h2w >> 16, uint32_t(xv.ao[hh][2]), uint32_t(xv.ao[hh][3]), acco[m]);
          }
      }
    }
  }

  // ---- the eight lanes of a row (blocks and chunks), fixed butterfly order
#pragma unroll
  for (int m = 0; m < MT; ++m) {
#pragma unroll
    for (int o = 8; o <= 32; o <<= 1) {
      acc[m] += __shfl_xor(acc[m], o, 64);
      acco[m] += __shfl_xor(acco[m], o, 64);
    }
    if (lane < kSliceRowsD) {
      part[kq][m][lane][0] = acc[m];
      part[kq][m][lane][1] = __int_as_float(acco[m]);
    }
  }
  __syncthreads();
  if (kq != 0 || lane >= kSliceRowsD) return;
  const int n = t * kTileN + r;
  if (n >= a.N) return;
  const float so = reinterpret_cast<const float*>(a.blob + a.rows_off)[n];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    if (m >= a.M) break;
    float s = 0.f;
    int so_acc = 0;
    for (int q = 0; q < a.parts; ++q) {  // parts in a fixed order
      s += part[q][m][lane][0];
      so_acc += __float_as_int(part[q][m][lane][1]);
    }
    store_y(a.Y, a.y_bf16, size_t(m) * a.N + n, fmaf(a.s_a[m], so * float(so_acc), s));
  }
}

template <int MT, int S>
hipError_t launch_s(const DualDecArgs& a, int planes, hipStream_t st) {
  if (planes == 2)
    hipLaunchKernelGGL((dual_decode_kernel<MT, S, 2>), dim3(unsigned(a.n_slices)), dim3(unsigned(a.parts * 64)), 0, st, a);
  else
    hipLaunchKernelGGL((dual_decode_kernel<MT, S, 1>), dim3(unsigned(a.n_slices)), dim3(unsigned(a.parts * 64)), 0, st, a);
  return hipGetLastError();
}

// Steps per wave S (a power of two, up to 8 for one token, the register
// budget): the smallest whose parts of K fit one workgroup, raised towards
// about 8192 waves in all (measured: 11008x4096 at M = 1 takes 8.8 us at
// that count against 11.0 us at 4096 waves).  Two tokens take this kernel
// only where that needs at most 2 steps (4096x4096 at M = 2: 6.2 us against
// 7.1 with the matrix kernel; 11008x4096: 13.8 against 11.9).  0: no fit.
int steps_for_dual(int64_t M, int64_t N, int64_t KC) {
  const int mt = int(M), smax = M == 1 ? 8 : 2;
  const int64_t slices = (N + kSliceRowsD - 1) / kSliceRowsD;
  int pref = 1;
  while (pref < (slices * KC + 16383) / 16384) pref <<= 1;
  if (M == 2 && pref > smax) return 0;
  int first = 0;
  for (int s = 1; s <= smax; s <<= 1) {
    if ((KC + 2 * s - 1) / (2 * s) > max_parts(mt, s)) continue;
    if (!first) first = s;
    if (s >= pref) return s;
  }
  return first ? smax : 0;
}

}  // namespace

bool dual_decode_fits(int64_t M, int64_t N, int64_t K) {
  if (M < 1 || M > kDecTokensMax) return false;
  return steps_for_dual(M, N, (K + kChunkK - 1) / kChunkK) > 0;
}

hipError_t launch_dual_decode(const Cfg& c, const uint8_t* Xo, const float* s_a, const uint8_t* Xi,
                              const uint8_t* Ea, int64_t M, const uint8_t* blob, int64_t N, int64_t K,
                              void* Y, hipStream_t st) {
  const DualLayout L = make_dual_layout(N, K, c.n_o);
  const int S = steps_for_dual(M, N, L.n_chunks);
  const int np = L.out_planes;
  DualDecArgs a{Xo, s_a, Xi, Ea, blob, Y, int(M), int(N), int(K), int(L.n_chunks),
                int(L.n_tiles * (kTileN / kSliceRowsD)), int((L.n_chunks + 2 * S - 1) / (2 * S)),
                L.out_off, L.scale_off, L.rows_off, c.y_bf16};
  if (M == 1) {
    if (S == 1) return launch_s<1, 1>(a, np, st);
    if (S == 2) return launch_s<1, 2>(a, np, st);
    if (S == 4) return launch_s<1, 4>(a, np, st);
    return launch_s<1, 8>(a, np, st);
  }
  if (S == 1) return launch_s<2, 1>(a, np, st);
  return launch_s<2, 2>(a, np, st);
}

}  // namespace sdq
