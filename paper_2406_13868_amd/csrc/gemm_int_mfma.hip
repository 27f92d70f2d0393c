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
// = 32*MS tokens.  Each 128-K chunk of activations is converted from int8 to
// fp16 and staged in LDS (double buffered) for all 4 waves; each wave streams
// its own tile's group words (32 bytes per lane per chunk) and
// expands them in registers into dense fp16 B fragments: lane l holds column
// l%32 and the 8-group 2*kb + l/32 of every 16-K block kb.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace sdq {
namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kRowPad = 8;                        // f16 elements of padding per LDS row
constexpr int kLdsRow = kChunkK + kRowPad;        // 136 f16 = 272 bytes
constexpr uint32_t kOutPosMagic = (1u << 21) | (1u << 14) | (1u << 7);

struct MfmaArgs {
  const uint8_t* Xq;
  const float* s_a;
  const uint8_t* blob;
  float* Y;
  int M, N, K, n_chunks, n_tiles;
  int64_t scales_off, rows_off;
};

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
// position p (0 where the group has no inlier).
template <int NI>
__device__ __forceinline__ h8 inlier_f16(uint32_t w) {
  uint32_t D = 0;
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const uint32_t q = (w >> (8 * j + 4)) & 0xFu;
    const uint32_t sh = ((w >> (8 * j)) & 7u) << 2;
    D |= q << sh;
  }
  const uint32_t Db = D ^ 0x88888888u;  // biased nibbles q + 8
  const uint32_t Ds = Db >> 4;
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  const h2 bias = {(_Float16)-1032.0f, (_Float16)-1032.0f};
  u4v out;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const uint32_t sel = uint32_t(v) | 0x0C00u | (uint32_t(4 + v) << 16) | 0x0C000000u;
    const uint32_t t = (__builtin_amdgcn_perm(Ds, Db, sel) & 0x000F000Fu) | 0x64006400u;
    out[v] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(h2, t) + bias);
  }
  return __builtin_bit_cast(h8, out);
}

// Dense fp16 outlier fragment of one group word (one non-zero at most).
template <bool OUT_INT8>
__device__ __forceinline__ h8 outlier_f16(uint32_t w) {
  float f;
  if constexpr (OUT_INT8) f = (float)(int(w) >> 24);
  else f = __builtin_amdgcn_cvt_f32_fp8(int(w), 3);
  const uint32_t hb = uint32_t(__builtin_bit_cast(unsigned short, (_Float16)f));
  const uint32_t pos = (__umul24(w & 0x00080808u, kOutPosMagic) >> 24) & 7u;
  const uint32_t val = hb << ((pos & 1u) << 4);
  const uint32_t d = pos >> 1;
  u4v out;
#pragma unroll
  for (int v = 0; v < 4; ++v) out[v] = d == uint32_t(v) ? val : 0u;
  return __builtin_bit_cast(h8, out);
}

template <int MS, int NI, bool OUT_INT8>
__global__ __launch_bounds__(kThreads) void int_mfma_kernel(MfmaArgs a) {
  constexpr int BM = 32 * MS;
  __shared__ __align__(16) _Float16 xs[2][BM * kLdsRow];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, h = lane >> 5;
  const int m0 = blockIdx.y * BM;
  const int tile = blockIdx.x * kWaves + wave;
  const bool tile_ok = tile < a.n_tiles;
  const int KC = a.n_chunks;

  // ---- activation staging: BM rows x 128 int8 -> fp16 in LDS
  // thread -> (row, 16-byte column piece): 8 pieces per row
  constexpr int kPieces = BM * 8;
  constexpr int kPerThread = (kPieces + kThreads - 1) / kThreads;
  uint4 xr[kPerThread];
  auto load_x = [&](int c) {
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
      const int pc = tid + i * kThreads;
      const int rr = pc >> 3, cp = pc & 7;
      xr[i] = make_uint4(0, 0, 0, 0);
      if (pc < kPieces && m0 + rr < a.M)
        xr[i] = *reinterpret_cast<const uint4*>(a.Xq + size_t(m0 + rr) * a.K + c * kChunkK + cp * 16);
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
  const uint8_t* sbase = a.blob + a.scales_off + size_t(tile_ok ? tile : 0) * KC * kIntScaleBytesPerTC + col * 16;
  uint4 wr0, wr1, sr;
  auto load_w = [&](int c) {
    if (tile_ok) {
      wr0 = *reinterpret_cast<const uint4*>(wbase + size_t(c) * kWordBytesPerTC);
      wr1 = *reinterpret_cast<const uint4*>(wbase + size_t(c) * kWordBytesPerTC + 16);
      sr = *reinterpret_cast<const uint4*>(sbase + size_t(c) * kIntScaleBytesPerTC);
    } else {
      wr0 = wr1 = sr = make_uint4(0, 0, 0, 0);
    }
  };

  f16v acc[MS], acco[MS];
#pragma unroll
  for (int s = 0; s < MS; ++s)
#pragma unroll
    for (int e = 0; e < 16; ++e) { acc[s][e] = 0.f; acco[s][e] = 0.f; }

  load_x(0);
  load_w(0);
  store_x(0);
  __syncthreads();

  for (int c = 0; c < KC; ++c) {
    const int buf = c & 1;
    const uint32_t wv[8] = {wr0.x, wr0.y, wr0.z, wr0.w, wr1.x, wr1.y, wr1.z, wr1.w};
    const uint32_t sv[4] = {sr.x, sr.y, sr.z, sr.w};
    if (c + 1 < KC) { load_x(c + 1); load_w(c + 1); }
#pragma unroll 2
    for (int kb = 0; kb < 8; ++kb) {
      const h8 bi = inlier_f16<NI>(wv[kb]);
      const h8 bo = outlier_f16<OUT_INT8>(wv[kb]);
      const uint32_t sw = sv[kb >> 1];
      const float s = (float)__builtin_bit_cast(_Float16, (unsigned short)((kb & 1) ? (sw >> 16) : (sw & 0xFFFFu)));
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const h8 av = *reinterpret_cast<const h8*>(&xs[buf][(ms * 32 + col) * kLdsRow + kb * 16 + h * 8]);
        f16v zero;
#pragma unroll
        for (int e = 0; e < 16; ++e) zero[e] = 0.f;
        const f16v P = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, bi, zero, 0, 0, 0);
        acco[ms] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, bo, acco[ms], 0, 0, 0);
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[ms][e] = fmaf(P[e], s, acc[ms][e]);
      }
    }
    if (c + 1 < KC) {
      store_x(buf ^ 1);
      __syncthreads();
    }
  }

  if (!tile_ok) return;
  const int n = tile * kTileN + col;
  if (n >= a.N) return;
  const float so = reinterpret_cast<const float*>(a.blob + a.rows_off)[n];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int m = m0 + ms * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
      if (m < a.M) a.Y[size_t(m) * a.N + n] = a.s_a[m] * fmaf(so, acco[ms][e], acc[ms][e]);
    }
}

// Split-K form for few tokens (M <= 64): one 32-row tile of W per workgroup,
// its NW waves take interleaved 128-K chunks and each lane reads its 8-byte
// A-fragment pieces of Xq straight from L2 (no LDS staging), converting them
// to fp16 in registers; the wave partials are summed through LDS with a
// fixed-order tree at the end.  This keeps NT*NW waves in flight where the
// tiled form above would run only NT/4 workgroups.
template <int MS, int NI, bool OUT_INT8, int NW>
__global__ __launch_bounds__(NW * 64) void int_mfma_splitk_kernel(MfmaArgs a) {
  constexpr int BM = 32 * MS;
  __shared__ float red[NW / 2][16][64];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, h = lane >> 5;
  const int m0 = blockIdx.y * BM;
  const int tile = blockIdx.x;
  const int KC = a.n_chunks;

  const uint8_t* wbase = a.blob + size_t(tile) * KC * kWordBytesPerTC + size_t(lane) * 32;
  const uint8_t* sbase = a.blob + a.scales_off + size_t(tile) * KC * kIntScaleBytesPerTC + col * 16;

  // lane (col, h) of sub-tile ms reads row m0 + 32*ms + col, K bytes 16*kb + 8*h .. +8
  uint2 xr[MS][8];
  auto load_x = [&](int c) {
#pragma unroll
    for (int ms = 0; ms < MS; ++ms) {
      const int m = m0 + ms * 32 + col;
      const uint8_t* xp = a.Xq + size_t(m < a.M ? m : 0) * a.K + c * kChunkK + h * 8;
#pragma unroll
      for (int kb = 0; kb < 8; ++kb)
        xr[ms][kb] = m < a.M ? *reinterpret_cast<const uint2*>(xp + kb * 16) : make_uint2(0, 0);
    }
  };
  uint4 wr0, wr1, sr;
  auto load_w = [&](int c) {
    wr0 = *reinterpret_cast<const uint4*>(wbase + size_t(c) * kWordBytesPerTC);
    wr1 = *reinterpret_cast<const uint4*>(wbase + size_t(c) * kWordBytesPerTC + 16);
    sr = *reinterpret_cast<const uint4*>(sbase + size_t(c) * kIntScaleBytesPerTC);
  };

  f16v acc[MS], acco[MS];
#pragma unroll
  for (int s = 0; s < MS; ++s)
#pragma unroll
    for (int e = 0; e < 16; ++e) { acc[s][e] = 0.f; acco[s][e] = 0.f; }

  int c = wave;
  if (c < KC) { load_x(c); load_w(c); }
  for (; c < KC; c += NW) {
    uint2 xc[MS][8];
#pragma unroll
    for (int ms = 0; ms < MS; ++ms)
#pragma unroll
      for (int kb = 0; kb < 8; ++kb) xc[ms][kb] = xr[ms][kb];
    const uint32_t wv[8] = {wr0.x, wr0.y, wr0.z, wr0.w, wr1.x, wr1.y, wr1.z, wr1.w};
    const uint32_t sv[4] = {sr.x, sr.y, sr.z, sr.w};
    if (c + NW < KC) { load_x(c + NW); load_w(c + NW); }
#pragma unroll 2
    for (int kb = 0; kb < 8; ++kb) {
      const h8 bi = inlier_f16<NI>(wv[kb]);
      const h8 bo = outlier_f16<OUT_INT8>(wv[kb]);
      const uint32_t sw = sv[kb >> 1];
      const float s = (float)__builtin_bit_cast(_Float16, (unsigned short)((kb & 1) ? (sw >> 16) : (sw & 0xFFFFu)));
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        uint32_t a0, a1, a2, a3;
        i8x4_to_f16x4(xc[ms][kb].x, a0, a1);
        i8x4_to_f16x4(xc[ms][kb].y, a2, a3);
        const u4v av4 = {a0, a1, a2, a3};
        const h8 av = __builtin_bit_cast(h8, av4);
        f16v zero;
#pragma unroll
        for (int e = 0; e < 16; ++e) zero[e] = 0.f;
        const f16v P = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, bi, zero, 0, 0, 0);
        acco[ms] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, bo, acco[ms], 0, 0, 0);
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[ms][e] = fmaf(P[e], s, acc[ms][e]);
      }
    }
  }

  // ---- tree over the waves: in round r, wave w + 2^r hands its partial to w
#pragma unroll
  for (int ms = 0; ms < MS; ++ms) {
#pragma unroll
    for (int which = 0; which < 2; ++which) {
      f16v& v = which ? acco[ms] : acc[ms];
#pragma unroll
      for (int stride = NW / 2; stride >= 1; stride >>= 1) {
        const bool sender = wave >= stride && wave < 2 * stride;
        if (sender) {
#pragma unroll
          for (int e = 0; e < 16; ++e) red[wave - stride][e][lane] = v[e];
        }
        __syncthreads();
        if (wave < stride) {
#pragma unroll
          for (int e = 0; e < 16; ++e) v[e] += red[wave][e][lane];
        }
        __syncthreads();
      }
    }
  }
  if (wave > 0) return;
  const int n = tile * kTileN + col;
  if (n >= a.N) return;
  const float so = reinterpret_cast<const float*>(a.blob + a.rows_off)[n];
#pragma unroll
  for (int ms = 0; ms < MS; ++ms)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int m = m0 + ms * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
      if (m < a.M) a.Y[size_t(m) * a.N + n] = a.s_a[m] * fmaf(so, acco[ms][e], acc[ms][e]);
    }
}

template <int MS, int NI, int NW>
hipError_t launch_splitk(const Cfg& c, const MfmaArgs& a, hipStream_t st) {
  const dim3 grid(unsigned(a.n_tiles), unsigned((a.M + 32 * MS - 1) / (32 * MS)));
  const dim3 block(NW * 64);
  if (c.fmt_o == SDQ_FMT_INT8)
    hipLaunchKernelGGL((int_mfma_splitk_kernel<MS, NI, true, NW>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((int_mfma_splitk_kernel<MS, NI, false, NW>), grid, block, 0, st, a);
  return hipGetLastError();
}

template <int MS, int NI>
hipError_t launch_ms_ni(const Cfg& c, const MfmaArgs& a, hipStream_t st) {
  if constexpr (MS <= 2) {
    // few tokens: split K inside the workgroup so that about 2048+ waves run
    if (int64_t(a.n_tiles) * 4 >= 2048 || a.n_chunks < 8) return launch_splitk<MS, NI, 4>(c, a, st);
    return launch_splitk<MS, NI, 8>(c, a, st);
  }
  const dim3 grid(unsigned((a.n_tiles + kWaves - 1) / kWaves), unsigned((a.M + 32 * MS - 1) / (32 * MS)));
  const dim3 block(kThreads);
  if (c.fmt_o == SDQ_FMT_INT8)
    hipLaunchKernelGGL((int_mfma_kernel<MS, NI, true>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((int_mfma_kernel<MS, NI, false>), grid, block, 0, st, a);
  return hipGetLastError();
}

template <int MS>
hipError_t launch_ms(const Cfg& c, const MfmaArgs& a, hipStream_t st) {
  if (c.n_i == 1) return launch_ms_ni<MS, 1>(c, a, st);
  if (c.n_i == 2) return launch_ms_ni<MS, 2>(c, a, st);
  return launch_ms_ni<MS, 3>(c, a, st);
}

}  // namespace

hipError_t launch_int_mfma(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                           const uint8_t* blob, int64_t N, int64_t K, float* Y, hipStream_t st) {
  const Layout L = make_layout(false, N, K);
  MfmaArgs a{Xq, s_a, blob, Y, int(M), int(N), int(K), int(L.n_chunks), int(L.n_tiles),
             L.scales_off, L.rows_off};
  if (M <= 32) return launch_ms<1>(c, a, st);
  if (M <= 64) return launch_ms<2>(c, a, st);
  return launch_ms<4>(c, a, st);
}

}  // namespace sdq
