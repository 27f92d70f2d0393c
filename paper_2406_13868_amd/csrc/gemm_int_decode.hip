// INT-family decomposed GEMM for small M (decode): a weight-streaming vector
// kernel.  Section 5.1 of the paper: Y = SpMM(A, W_o) + SpMM(A, W_i), here
// with both branches read from one stream of 32-bit group words.
//
// At M <= 8 the product is bound by the HBM stream of packed weights (about
// 5 bits per weight) and by the fixed cost of a launch, so the kernel keeps
// every wave's dependency chain short:
//
//   * four waves per 4-row slice of a 32-row tile split K into parts; each
//     owns S consecutive "steps" of eight 128-K chunks (S = ceil(K / 4096)
//     for K <= 32768); two slices (eight waves) per workgroup, and the
//     workgroups of one XCD take a contiguous range of slices, so the
//     128-byte lines of block scales that two slices share are fetched once;
//   * lane l works on row (l & 3) of the slice, on half j = (l>>2)&1 of the
//     16-K scale blocks of a chunk, and on chunk cc = l>>3 of a step; one
//     load instruction reads eight 128-byte runs of group words;
//   * a wave requests its activations first and then all of its weight
//     stream (S steps, three loads each), so the load counter lets it compute
//     each step as soon as that step has landed;
//   * each wave keeps the int8 activations of its own part of K in a private
//     LDS region (chunk stride 144 bytes, plus one zero chunk that stands in
//     for the chunks past K); only the fused form, which first needs the amax
//     of the whole token, synchronises the workgroup before the products;
//   * each group word becomes a v_perm_b32 selector that gathers the four
//     activations its slots need (three inliers, one outlier); v_dot4_i32_i8
//     multiplies them with the inlier codes (kept at the top nibble of each
//     byte, i.e. 16x the int4 value) into an exact integer partial per 16-K
//     block, scaled by the block's fp16 scale into the fp32 accumulator; the
//     outlier products are summed in fp32 (e4m3) or exactly in int32 (int8)
//     and added with the row's outlier scale at the end;
//   * the 16 lanes of a row are summed with DPP rotations and permlane swaps
//     and the parts of K in a fixed order through LDS: the result does not
//     depend on timing.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.h"
#include "tile_out.h"

namespace sdq {
namespace {

constexpr int kKSplit = 4;                     // waves per 4-row slice (each owns a part of K)
constexpr int kSliceRows = 4;
constexpr int kWavesPerWG = 8;                 // slices x K parts per workgroup (LDS permitting)
constexpr int kMaxLdsBytes = 64 * 1024;
constexpr int kStepChunks = 8;                 // 128-K chunks per wave step
constexpr int kMaxSteps = 8;                   // steps per wave: K <= 4 * 8 * 8 * 128
constexpr int kXStride = 144;                  // LDS bytes per 128-K chunk of one token
constexpr int kFusedMaxM = 2;  // the fused form serves the decode sizes sdq_linear sends here
// v_mul_u32_u24 magic that moves bits 3, 11, 19 of a group word to 24, 25, 26
// (it also leaves copies at bits 10, 17, 18, inside the inlier position mask,
// which the bitfield insert replaces).
constexpr uint32_t kOutPosMagic = (1u << 21) | (1u << 14) | (1u << 7);
constexpr uint32_t kInPosMask = 0x00070707u;

struct DecodeArgs {
  const uint8_t* Xq;   // [M][K] int8 (unfused form)
  const float* s_a;    // [M]    (unfused form)
  const void* X;       // fused form: [M][K] fp32 or bf16
  float* s_a_out;      // fused form: written by workgroup 0
  uint8_t* Xq_out;     // fused form: written by workgroup 0
  const uint8_t* blob;
  void* Y;
  int M, N, K, n_chunks;
  int64_t scales_off, rows_off, irow_off;
  bool y_bf16 = false;  // Y as bf16
  int qs = 0;           // log2(qv / 16): 16-K blocks per inlier scale = 1 << qs
  int srow = 16;        // bytes of one row's inlier scales in a chunk: (128 / qv) * (2 or 1)
};

// Inlier scale formats of the INT family (template parameter SF).
enum ScaleFmt { kScaleF16 = 0, kScaleE4M3 = 1, kScaleE6M2 = 2 };

// Value of a ufp8-e6m2 code: (4 + m) * 2^(e - 33), or m * 2^-32 for e = 0
// (exact in fp32: a 3-bit integer times a power of two).
__device__ __forceinline__ float e6m2_to_f32(uint32_t code) {
  const uint32_t e = (code >> 2) & 63u, m = code & 3u;
  const float mant = float(e ? 4u + m : m);
  const uint32_t ee = e ? e : 1u;
  return mant * __uint_as_float((ee + 94u) << 23);  // 2^(ee - 33)
}

// LDS bytes of one wave's activation region: MT tokens x (8S chunks + the zero chunk).
__host__ __device__ constexpr int wave_lds_bytes(int MT, int S) {
  return MT * (S * kStepChunks + 1) * kXStride;
}

// Perm selector of a group word: positions of the three inlier slots in
// bytes 0-2, the outlier position (bits 3, 11, 19 gathered by one 24-bit
// multiply) in byte 3.  The bitfield insert is spelled out because the
// compiler otherwise splits it into two ops.
__device__ __forceinline__ uint32_t perm_selector(uint32_t w) {
  const uint32_t u = __umul24(w & 0x00080808u, kOutPosMagic);
  uint32_t sel;
  asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(sel) : "s"(kInPosMask), "v"(w), "v"(u));
  return sel;
}

// Sum over the 16 lanes l' of the wave with l' = l (mod 4): two DPP row
// rotations inside each row of 16 lanes, then the rows are exchanged with
// the permlane swaps.  Every lane ends with the sum of its residue class,
// in an order that does not depend on timing.
__device__ __forceinline__ float sum_lanes_mod4(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x124, 0xF, 0xF, false));  // row_ror:4
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x128, 0xF, 0xF, false));  // row_ror:8
  const auto p16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(p16[0]) + __uint_as_float(p16[1]);
  const auto p32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(p32[0]) + __uint_as_float(p32[1]);
}

// Maximum over the 64 lanes of the wave: DPP row rotations by 1, 2, 4 and 8
// inside each row of 16 lanes, then the permlane swaps across rows (no LDS
// round trips).  A maximum is exact in any order.
__device__ __forceinline__ float max_lanes(float v) {
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x121, 0xF, 0xF, false)));  // row_ror:1
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x122, 0xF, 0xF, false)));  // row_ror:2
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x124, 0xF, 0xF, false)));  // row_ror:4
  v = fmaxf(v, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x128, 0xF, 0xF, false)));  // row_ror:8
  const auto p16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(p16[0]), __uint_as_float(p16[1]));
  const auto p32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(p32[0]), __uint_as_float(p32[1]));
}

__device__ __forceinline__ _Float16 f16lo(uint32_t v) {
  return __builtin_bit_cast(_Float16, (unsigned short)(v & 0xFFFFu));
}
__device__ __forceinline__ _Float16 f16hi(uint32_t v) {
  return __builtin_bit_cast(_Float16, (unsigned short)(v >> 16));
}

// int8 codes of eight activations: clamp(rne(x * inv), +-127), one fp32 multiply each.
__device__ __forceinline__ uint2 quant8(const float* v, float inv) {
  uint32_t lo = 0, hi = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float rq = rintf(v[i] * inv);
    const uint32_t b = uint32_t((int)fminf(fmaxf(rq, -127.f), 127.f)) & 0xFFu;
    if (i < 4) lo |= b << (8 * i);
    else hi |= b << (8 * (i - 4));
  }
  return make_uint2(lo, hi);
}

struct StepBuf {
  uint4 w0, w1;  // group words of (row, j) for h = 0 and h = 1
  uint2 sc;      // the lane's inlier scales (K [64j, 64j + 64) of the chunk): 1, 2 or 4
                 // fp16 values, or 1, 2 or 4 bytes (e4m3, e6m2), from the low end
};

// FUSE: 0 = activations from Xq/s_a, 1 = quantize fp32 X, 2 = quantize bf16 X.
// SF: inlier scale format (ScaleFmt); kScaleE4M3 is VS-Quant's two levels (an
// e4m3 code per Q-Vector, a power of two per row).
template <int MT, bool OUT_INT8, int FUSE, int S, int KS, int SPW, int SF>
__global__ __launch_bounds__(SPW * KS * 64) void int_decode_kernel(DecodeArgs a) {
  constexpr bool SC8 = SF == kScaleE4M3;
  const int kSB = kTileN * a.srow;               // inlier scale bytes per (tile, chunk)
  constexpr int kWG = SPW * KS;                  // waves per workgroup
  extern __shared__ __align__(16) uint8_t xs[];  // [wave][MT][8S + 1][kXStride]
  __shared__ float red[kWG][kDecodeMaxM];
  __shared__ float s_scale[kDecodeMaxM];
  __shared__ float part[SPW][KS][kDecodeMaxM][kSliceRows];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: chunk offsets stay scalar
  const int ws = wave / KS, kq = wave % KS;  // slice in the workgroup, part of K
  const int K = a.K, M = a.M, KC = a.n_chunks;
  const int r = lane & 3, j = (lane >> 2) & 1, cc = lane >> 3;
  const int slice = xcd_contiguous(blockIdx.x, gridDim.x) * SPW + ws;  // 4-row slice of the layer
  const int t = slice >> 3;                 // 32-row tile
  const int row = ((slice & 7) << 2) + r;   // row inside the tile
  const int chunk0 = kq * S * kStepChunks;  // first chunk of this wave's part of K
  constexpr int kTokBytes = (S * kStepChunks + 1) * kXStride;
  uint8_t* xw = xs + wave * wave_lds_bytes(MT, S);

  // ---- 1. this part's activations, requested first (the load counter is
  //         in order: waiting for them never waits for the weight stream).
  //         Piece i of a lane covers 16 bytes (or elements) of token i / S.
  constexpr int kPieces = MT * S;
  constexpr int kU = FUSE == 1 ? 4 : FUSE == 2 ? 2 : 1;
  uint4 xr[kPieces][kU];
#pragma unroll
  for (int i = 0; i < kPieces; ++i) {
    const int m = i / S;
    const int off = ((i % S) * 64 + lane) * 16;  // byte (element) offset in the part
    const int k = chunk0 * kChunkK + off;
    if (m < M && k < K) {
      const size_t e = size_t(m) * K + k;
      if constexpr (FUSE == 0) {
        xr[i][0] = *reinterpret_cast<const uint4*>(a.Xq + e);
      } else if constexpr (FUSE == 1) {
#pragma unroll
        for (int u = 0; u < 4; ++u) xr[i][u] = *reinterpret_cast<const uint4*>(static_cast<const float*>(a.X) + e + 4 * u);
      } else {
#pragma unroll
        for (int u = 0; u < 2; ++u) xr[i][u] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(a.X) + e + 8 * u);
      }
    } else {
#pragma unroll
      for (int u = 0; u < kU; ++u) xr[i][u] = make_uint4(0, 0, 0, 0);
    }
  }

  // ---- 2. the whole weight stream of the wave.  Chunks past K re-read the
  //         last chunk of the tile (in bounds) and meet the zero chunk.
  const uint8_t* tbase = a.blob + size_t(t) * KC * kWordBytesPerTC;
  const uint8_t* sbase = a.blob + a.scales_off + size_t(t) * KC * kSB;
  const uint32_t woff = uint32_t(row * 2 + j) * 16;
  // the lane covers K [64j, 64j + 64) of a chunk: half of its row's scales
  const int lbytes = a.srow >> 1;  // 8, 4, 2 or 1 (wave-uniform)
  const uint32_t soff = uint32_t(row * a.srow + j * lbytes);
  StepBuf buf[S];
#pragma unroll
  for (int d = 0; d < S; ++d) {
    const int c = min(chunk0 + d * kStepChunks + cc, KC - 1);
    const uint8_t* wp = tbase + (uint32_t(c) * kWordBytesPerTC + woff);
    buf[d].w0 = *reinterpret_cast<const uint4*>(wp);
    buf[d].w1 = *reinterpret_cast<const uint4*>(wp + 1024);  // h = 1: 32 rows x 32 bytes further
    const uint8_t* sp = sbase + (uint32_t(c) * kSB + soff);
    if (lbytes == 8) buf[d].sc = *reinterpret_cast<const uint2*>(sp);
    else if (lbytes == 4) buf[d].sc = make_uint2(*reinterpret_cast<const uint32_t*>(sp), 0u);
    else if (lbytes == 2) buf[d].sc = make_uint2(*reinterpret_cast<const uint16_t*>(sp), 0u);
    else buf[d].sc = make_uint2(*sp, 0u);
  }
  // 16 * s_o: the inlier dot products carry a factor 16, folded out at the end.
  const float so16 = 16.f * reinterpret_cast<const float*>(a.blob + a.rows_off)[t * kTileN + row];
  // the inlier row scale of two-level scales (a power of two)
  const float gi = SC8 ? reinterpret_cast<const float*>(a.blob + a.irow_off)[t * kTileN + row] : 1.f;

  // LDS address of piece i of this lane inside the wave's region
  auto lds_piece = [&](int i) -> uint8_t* {
    const int m = i / S;
    const int off = ((i % S) * 64 + lane) * 16;
    return xw + m * kTokBytes + (off >> 7) * kXStride + (off & 127);
  };
  // the zero chunk of every token (9 pieces of 16 bytes, stride padding included)
  for (int z = lane; z < MT * 9; z += 64) {
    const int m = z / 9, u = z % 9;
    *reinterpret_cast<uint4*>(xw + m * kTokBytes + S * kStepChunks * kXStride + u * 16) = make_uint4(0, 0, 0, 0);
  }

  // ---- 3. activations into the wave's LDS region
  if constexpr (FUSE == 0) {
#pragma unroll
    for (int i = 0; i < kPieces; ++i) *reinterpret_cast<uint4*>(lds_piece(i)) = xr[i][0];
    if (tid < kDecodeMaxM) s_scale[tid] = tid < M ? a.s_a[tid] : 0.f;
    // the products below read only this wave's region (plus s_scale at the end)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  } else {
    // per-token quantization with the arithmetic of the activation kernel:
    // a = max|x|, s_a = a/127, inv = 127/a, q = clamp(rne(x*inv), +-127)
    float v[kPieces][16];
#pragma unroll
    for (int i = 0; i < kPieces; ++i) {
      if constexpr (FUSE == 1) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          v[i][4 * u] = __uint_as_float(xr[i][u].x); v[i][4 * u + 1] = __uint_as_float(xr[i][u].y);
          v[i][4 * u + 2] = __uint_as_float(xr[i][u].z); v[i][4 * u + 3] = __uint_as_float(xr[i][u].w);
        }
      } else {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const uint32_t w[4] = {xr[i][u].x, xr[i][u].y, xr[i][u].z, xr[i][u].w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            v[i][8 * u + 2 * q] = __uint_as_float(w[q] << 16);
            v[i][8 * u + 2 * q + 1] = __uint_as_float(w[q] & 0xFFFF0000u);
          }
        }
      }
    }
    float amax[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) amax[m] = 0.f;
#pragma unroll
    for (int i = 0; i < kPieces; ++i) {
      float pm = 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e) pm = fmaxf(pm, fabsf(v[i][e]));
      amax[i / S] = fmaxf(amax[i / S], pm);
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      amax[m] = max_lanes(amax[m]);
      if (lane == 0) red[wave][m] = amax[m];
    }
    __syncthreads();
    float inv[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float am = red[0][m];
#pragma unroll
      for (int w = 1; w < kWG; ++w) am = fmaxf(am, red[w][m]);  // each slice covers all of K
      inv[m] = am > 0.f ? 127.f / am : 0.f;
      if (tid == 0) {
        const float sc = am / 127.f;
        s_scale[m] = sc;
        if (blockIdx.x == 0 && m < M) a.s_a_out[m] = sc;
      }
    }
#pragma unroll
    for (int i = 0; i < kPieces; ++i) {
      const uint2 q0 = quant8(&v[i][0], inv[i / S]), q1 = quant8(&v[i][8], inv[i / S]);
      const uint4 q = make_uint4(q0.x, q0.y, q1.x, q1.y);
      *reinterpret_cast<uint4*>(lds_piece(i)) = q;
      const int m = i / S;
      const int k = chunk0 * kChunkK + ((i % S) * 64 + lane) * 16;
      if (blockIdx.x == 0 && m < M && k < K)
        *reinterpret_cast<uint4*>(a.Xq_out + size_t(m) * K + k) = q;
    }
    // the products read only this wave's region; s_scale, written by thread
    // 0 above, is read after the workgroup barrier of the K-part sum
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // ---- 4. the products, one step at a time as the stream lands
  float acc[MT], acco[MT];
  int po[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) { acc[m] = 0.f; acco[m] = 0.f; po[m] = 0; }

#pragma unroll
  for (int d = 0; d < S; ++d) {
    if (chunk0 + d * kStepChunks >= KC) break;  // wave-uniform: the part starts past K
    const int c = chunk0 + d * kStepChunks + cc;
    const int lc = c < KC ? d * kStepChunks + cc : S * kStepChunks;  // past K: the zero chunk
    const uint8_t* xbase = xw + lc * kXStride;
    const StepBuf& cur = buf[d];
    const uint32_t wa[4] = {cur.w0.x, cur.w0.y, cur.w0.z, cur.w0.w};
    const uint32_t wb[4] = {cur.w1.x, cur.w1.y, cur.w1.z, cur.w1.w};
    // the scale of 16-K block q of the lane is its scale q >> qs
    float scl[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = q >> a.qs;
      if constexpr (SF == kScaleF16) {
        const uint32_t wd = e < 2 ? cur.sc.x : cur.sc.y;
        scl[q] = float((e & 1) ? f16hi(wd) : f16lo(wd));
      } else {
        const uint32_t byte = (cur.sc.x >> (8 * e)) & 0xFFu;
        if constexpr (SF == kScaleE4M3) scl[q] = __builtin_amdgcn_cvt_f32_fp8(int(byte), 0);
        else scl[q] = e6m2_to_f32(byte);
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int kb = 4 * j + q;  // 16-K block inside the chunk
      uint32_t sel[2], wi[2], wo_i8[2];
      float wo_f[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint32_t w = h ? wb[q] : wa[q];
        sel[h] = perm_selector(w);
        wi[h] = w & 0x00F0F0F0u;
        if constexpr (OUT_INT8) wo_i8[h] = w & 0xFF000000u;
        else wo_f[h] = __builtin_amdgcn_cvt_f32_fp8(int(w), 3);
      }
      const uint8_t* xk = xbase + kb * 16;
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const uint4 xv = *reinterpret_cast<const uint4*>(xk + m * kTokBytes);
        const uint32_t g0 = __builtin_amdgcn_perm(xv.y, xv.x, sel[0]);
        const uint32_t g1 = __builtin_amdgcn_perm(xv.w, xv.z, sel[1]);
        int P = __builtin_amdgcn_sdot4(int(g0), int(wi[0]), 0, false);
        P = __builtin_amdgcn_sdot4(int(g1), int(wi[1]), P, false);
        if constexpr (OUT_INT8) {
          po[m] = __builtin_amdgcn_sdot4(int(g0), int(wo_i8[0]), po[m], false);
          po[m] = __builtin_amdgcn_sdot4(int(g1), int(wo_i8[1]), po[m], false);
        } else {
          acco[m] = fmaf((float)(int(g0) >> 24), wo_f[0], acco[m]);
          acco[m] = fmaf((float)(int(g1) >> 24), wo_f[1], acco[m]);
        }
        acc[m] = fmaf((float)P, scl[q], acc[m]);
      }
    }
  }

  // ---- 5. sum the 16 lanes of a row (j, cc), fold in the outlier branch,
  //         then the parts of K in order
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    if constexpr (OUT_INT8) acco[m] = (float)po[m];
    const float v = sum_lanes_mod4(fmaf(acco[m], so16, SC8 ? gi * acc[m] : acc[m]));
    if (lane < kSliceRows) part[ws][kq][m][lane] = v;
  }
  __syncthreads();
  const int n = t * kTileN + row;
  if (kq == 0 && lane < kSliceRows && n < a.N) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float v = part[ws][0][m][r];
#pragma unroll
      for (int p = 1; p < KS; ++p) v += part[ws][p][m][r];
      if (m < M) store_y(a.Y, a.y_bf16, size_t(m) * a.N + n, s_scale[m] * (v * 0.0625f));
    }
  }
}

// steps per wave for K (a partial last chunk counts whole) when KS waves share a slice
int steps_for(int64_t K, int KS) {
  const int64_t all_steps = ((K + kChunkK - 1) / kChunkK + kStepChunks - 1) / kStepChunks;
  return int((all_steps + KS - 1) / KS);
}

// K split of a slice: kKSplit waves, more (up to 4) where one wave's steps
// would not fit MT * S <= kMaxSteps (activation registers and LDS)
int ks_for(int64_t MT, int64_t K) {
  for (int ks = kKSplit; ks < 4; ks *= 2)
    if (MT * steps_for(K, ks) <= kMaxSteps) return ks;
  return 4;
}

// slices per workgroup: kWavesPerWG / KS, fewer where the activation regions
// would not fit the workgroup's LDS; it divides the 8 slices of a tile
constexpr int spw_for(int MT, int S, int KS) {
  int spw = kWavesPerWG / KS;
  while (spw > 1 && spw * KS * wave_lds_bytes(MT, S) > kMaxLdsBytes) spw /= 2;
  return spw;
}

template <int MT, int FUSE, int S, int KS>
hipError_t launch_s(const Cfg& c, const DecodeArgs& a, hipStream_t st) {
  constexpr int SPW = spw_for(MT, S, KS);
  static_assert((kTileN / kSliceRows) % SPW == 0, "slices per workgroup must divide a tile");
  const Layout L = layout_for(c, a.N, a.K);
  const dim3 grid(unsigned(L.n_tiles * (kTileN / kSliceRows) / SPW));
  const dim3 block(SPW * KS * 64);
  const size_t lds = size_t(SPW) * KS * wave_lds_bytes(MT, S);
  const int sf = c.sc8 ? kScaleE4M3 : c.e6m2 ? kScaleE6M2 : kScaleF16;
  auto go = [&](auto sfc) {
    constexpr int SF = decltype(sfc)::value;
    if (c.fmt_o == SDQ_FMT_INT8)
      hipLaunchKernelGGL((int_decode_kernel<MT, true, FUSE, S, KS, SPW, SF>), grid, block, lds, st, a);
    else
      hipLaunchKernelGGL((int_decode_kernel<MT, false, FUSE, S, KS, SPW, SF>), grid, block, lds, st, a);
  };
  if (sf == kScaleE4M3) go(std::integral_constant<int, kScaleE4M3>{});
  else if (sf == kScaleE6M2) go(std::integral_constant<int, kScaleE6M2>{});
  else go(std::integral_constant<int, kScaleF16>{});
  return hipGetLastError();
}

// MT * S <= 8 keeps the activation registers and LDS bounded (decode_fits).
template <int MT, int FUSE, int KS>
hipError_t launch_ks(const Cfg& c, const DecodeArgs& a, hipStream_t st) {
  switch (steps_for(a.K, KS)) {
    case 1: return launch_s<MT, FUSE, 1, KS>(c, a, st);
    case 2: if constexpr (MT <= 4) return launch_s<MT, FUSE, 2, KS>(c, a, st); break;
    case 3: if constexpr (MT <= 2) return launch_s<MT, FUSE, 3, KS>(c, a, st); break;
    case 4: if constexpr (MT <= 2) return launch_s<MT, FUSE, 4, KS>(c, a, st); break;
    case 5: if constexpr (MT <= 1) return launch_s<MT, FUSE, 5, KS>(c, a, st); break;
    case 6: if constexpr (MT <= 1) return launch_s<MT, FUSE, 6, KS>(c, a, st); break;
    case 7: if constexpr (MT <= 1) return launch_s<MT, FUSE, 7, KS>(c, a, st); break;
    case 8: if constexpr (MT <= 1) return launch_s<MT, FUSE, 8, KS>(c, a, st); break;
    default: break;
  }
  return hipErrorInvalidValue;  // excluded by decode_fits
}

template <int MT, int FUSE>
hipError_t launch_mt(const Cfg& c, const DecodeArgs& a, hipStream_t st) {
  const int ks = ks_for(MT, a.K);
  if constexpr (kKSplit <= 1)
    if (ks == 1) return launch_ks<MT, FUSE, 1>(c, a, st);
  if constexpr (kKSplit <= 2)
    if (ks == 2) return launch_ks<MT, FUSE, 2>(c, a, st);
  return launch_ks<MT, FUSE, 4>(c, a, st);
}

template <int FUSE>
hipError_t launch_fuse(const Cfg& c, const DecodeArgs& a, hipStream_t st) {
  if (a.M <= 1) return launch_mt<1, FUSE>(c, a, st);
  if (a.M <= 2) return launch_mt<2, FUSE>(c, a, st);
  if constexpr (FUSE == 0) {
    if (a.M <= 4) return launch_mt<4, FUSE>(c, a, st);
    return launch_mt<8, FUSE>(c, a, st);
  }
  return hipErrorInvalidValue;  // the fused form is never asked for more tokens
}

}  // namespace

// Q-Vector and scale width of the configuration into the kernel arguments.
void set_scale_args(const Cfg& c, DecodeArgs& a) {
  a.qs = c.qv == 64 ? 2 : c.qv == 32 ? 1 : 0;
  a.srow = (kChunkK / c.qv) * c.scale_bytes();
}

bool decode_fused_fits(int64_t M, int64_t K) { return M <= kFusedMaxM && decode_fits(M, K); }

bool decode_fits(int64_t M, int64_t K) {
  if (M < 1 || M > kDecodeMaxM || K < kChunkK) return false;
  const int64_t mt = M <= 1 ? 1 : M <= 2 ? 2 : M <= 4 ? 4 : 8;
  return mt * steps_for(K, 4) <= kMaxSteps;
}

hipError_t launch_int_decode(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                             const uint8_t* blob, int64_t N, int64_t K, void* Y, hipStream_t st) {
  const Layout L = layout_for(c, N, K);
  DecodeArgs a{Xq, s_a, nullptr, nullptr, nullptr, blob, Y, int(M), int(N), int(K),
               int(L.n_chunks), L.scales_off, L.rows_off, L.irow_off};
  a.y_bf16 = c.y_bf16;
  set_scale_args(c, a);
  return launch_fuse<0>(c, a, st);
}

hipError_t launch_int_decode_fused(const Cfg& c, const void* X, int x_dtype, int64_t M,
                                   uint8_t* Xq_out, float* s_a_out, const uint8_t* blob, int64_t N,
                                   int64_t K, void* Y, hipStream_t st) {
  const Layout L = layout_for(c, N, K);
  DecodeArgs a{nullptr, nullptr, X, s_a_out, Xq_out, blob, Y, int(M), int(N), int(K),
               int(L.n_chunks), L.scales_off, L.rows_off, L.irow_off};
  a.y_bf16 = c.y_bf16;
  set_scale_args(c, a);
  if (x_dtype == SDQ_DTYPE_BF16) return launch_fuse<2>(c, a, st);
  return launch_fuse<1>(c, a, st);
}

}  // namespace sdq
