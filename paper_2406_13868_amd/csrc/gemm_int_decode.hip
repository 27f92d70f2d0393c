// INT-family decomposed GEMM for small M (decode): a weight-streaming vector
// kernel.  Section 5.1 of the paper: Y = SpMM(A, W_o) + SpMM(A, W_i), here
// with both branches read from one stream of 32-bit group words.
//
// At M <= 8 the product is bound by the HBM stream of packed weights (about
// 5 bits per weight).  The kernel is shaped so that every wave owns complete
// outputs and can leave as soon as its own stream is consumed:
//
//   * one wave per 4-row slice of a 32-row tile, over the whole of K (a
//     4096-row layer runs 1024 waves, one per SIMD); four slices per
//     workgroup, which share nothing but the per-token activation scales;
//   * lane l works on row (l & 3) of the slice, on half j = (l>>2)&1 of the
//     16-K scale blocks of a chunk, and on chunk cc = l>>3 of an 8-chunk
//     step; one load instruction reads eight 128-byte runs of group words;
//   * the weight stream of the first four steps is requested before
//     anything else and every step requests the one four ahead;
//   * the activations of all tokens are requested before the weight stream
//     (the load counter is in order, so waiting for them never waits for the
//     weights) and stored in LDS behind the one barrier of the kernel, copied
//     from Xq or, in the fused form, quantized there with the arithmetic of
//     the stand-alone activation kernel after a workgroup-wide amax;
//   * each group word becomes a v_perm_b32 selector that gathers the four
//     activations its slots need (three inliers, one outlier); v_dot4_i32_i8
//     multiplies them with the inlier codes (kept at the top nibble of each
//     byte, i.e. 16x the int4 value) into an exact integer partial per 16-K
//     block, scaled by the block's fp16 scale into the fp32 accumulator; the
//     outlier products are summed in fp32 (e4m3) or exactly in int32 (int8)
//     and added with the row's outlier scale at the end;
//   * the 16 lanes of a row are summed with a fixed butterfly: the result
//     does not depend on timing.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace sdq {
namespace {

constexpr int kSlices = 4;                     // waves (4-row slices) per workgroup
constexpr int kThreads = kSlices * 64;
constexpr int kSliceRows = 4;
constexpr int kStepChunks = 8;                 // 128-K chunks per wave step
constexpr int kDepth = 4;                      // steps in flight per wave
// The activations of all M tokens sit in LDS, read in 16-element pieces:
// at most kMaxPieces pieces per thread, i.e. M*K <= 16*kThreads*kMaxPieces.
constexpr int kMaxPieces = 8;
constexpr int kFusedMaxM = 2;  // the fused form serves the decode sizes sdq_linear sends here
// v_mul_u32_u24 magic that moves bits 3, 11, 19 of a group word to 24, 25, 26.
constexpr uint32_t kOutPosMagic = (1u << 21) | (1u << 14) | (1u << 7);

struct DecodeArgs {
  const uint8_t* Xq;   // [M][K] int8 (unfused form)
  const float* s_a;    // [M]    (unfused form)
  const void* X;       // fused form: [M][K] fp32 or bf16
  float* s_a_out;      // fused form: written by workgroup 0
  uint8_t* Xq_out;     // fused form: written by workgroup 0
  const uint8_t* blob;
  float* Y;
  int M, N, K, n_chunks;
  int64_t scales_off, rows_off;
};

__device__ __forceinline__ float f16lo(uint32_t v) {
  return (float)__builtin_bit_cast(_Float16, (unsigned short)(v & 0xFFFFu));
}
__device__ __forceinline__ float f16hi(uint32_t v) {
  return (float)__builtin_bit_cast(_Float16, (unsigned short)(v >> 16));
}

// Eight consecutive activations widened to fp32.
template <bool BF16>
__device__ __forceinline__ void load_x8(const void* X, size_t idx, float (&v)[8]) {
  if constexpr (BF16) {
    const uint4 raw = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(X) + idx);
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  } else {
    const float4 a = *reinterpret_cast<const float4*>(static_cast<const float*>(X) + idx);
    const float4 b = *reinterpret_cast<const float4*>(static_cast<const float*>(X) + idx + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

// int8 codes of eight activations: clamp(rne(x * inv), +-127), one fp32 multiply each.
__device__ __forceinline__ uint2 quant8(const float (&v)[8], float inv) {
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
  uint2 sc;      // the four fp16 scales of blocks 4j..4j+3
};

// FUSE: 0 = activations from Xq/s_a, 1 = quantize fp32 X, 2 = quantize bf16 X.
template <int MT, bool OUT_INT8, int FUSE, int PPT, int KSPLIT>
__global__ __launch_bounds__(kThreads) void int_decode_kernel(DecodeArgs a) {
  extern __shared__ __align__(16) uint8_t xs[];  // [MT][K] int8 activations
  __shared__ float red[kSlices][kDecodeMaxM];
  __shared__ float s_scale[kDecodeMaxM];
  __shared__ float part[kSlices][kDecodeMaxM][kSliceRows];  // second K half of a slice

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int K = a.K, M = a.M;
  const int r = lane & 3, j = (lane >> 2) & 1, cc = lane >> 3;
  // KSPLIT = 2: two waves per slice, each over half of the steps
  const int slices_per_wg = kSlices / KSPLIT;
  const int wslice = wave % slices_per_wg, khalf = wave / slices_per_wg;
  const int slice = blockIdx.x * slices_per_wg + wslice;  // 4-row slice of the layer
  const int t = slice >> 3;                                // 32-row tile
  const int row = ((slice & 7) << 2) + r;                  // row inside the tile
  const int KC = a.n_chunks;
  const int all_steps = (KC + kStepChunks - 1) / kStepChunks;
  const int s_begin = KSPLIT == 1 ? 0 : (khalf == 0 ? 0 : (all_steps + 1) / 2);
  const int s_end = KSPLIT == 1 ? all_steps : (khalf == 0 ? (all_steps + 1) / 2 : all_steps);

  // ---- 1. the activations first: their wait must not drain the weight loads
  //         (the load counter is in order), so they are requested before them.
  //         16 bytes of Xq, or 16 elements of X, per thread and piece.
  const int pieces = (MT * K) >> 4;
  uint4 xr[PPT][FUSE == 1 ? 4 : FUSE == 2 ? 2 : 1];
#pragma unroll
  for (int i = 0; i < PPT; ++i) {
    const int pc = tid + i * kThreads;
    const int m = (pc << 4) / K;
    if (pc < pieces && m < M) {
      const size_t e = size_t(pc) << 4;  // element index in [M][K]
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
      for (int u = 0; u < (FUSE == 1 ? 4 : FUSE == 2 ? 2 : 1); ++u) xr[i][u] = make_uint4(0, 0, 0, 0);
    }
  }

  // ---- 2. the weight stream: the first kDepth steps of this wave.  Loads
  //         are unconditional (addresses clamped into the tile), so the
  //         prefetch ring needs no copies; the ragged last step is masked.
  const uint8_t* tbase = a.blob + size_t(t) * KC * kWordBytesPerTC;
  const uint8_t* sbase = a.blob + a.scales_off + size_t(t) * KC * kIntScaleBytesPerTC;
  const uint32_t woff = uint32_t(row * 2 + j) * 16, soff = uint32_t(row * 16 + j * 8);
  auto load_step = [&](int s, StepBuf& b) {
    // past the wave's own steps: re-read its last one (a cache hit), never
    // the other K half's
    const int c = min(min(s, s_end - 1) * kStepChunks + cc, KC - 1);
    const uint8_t* wp = tbase + (uint32_t(c) * kWordBytesPerTC + woff);
    b.w0 = *reinterpret_cast<const uint4*>(wp);
    b.w1 = *reinterpret_cast<const uint4*>(wp + 1024);  // h = 1: 32 rows x 32 bytes further
    b.sc = *reinterpret_cast<const uint2*>(sbase + (uint32_t(c) * kIntScaleBytesPerTC + soff));
  };
  StepBuf buf[kDepth];
#pragma unroll
  for (int d = 0; d < kDepth; ++d) load_step(s_begin + d, buf[d]);
  // 16 * s_o: the inlier dot products carry a factor 16, folded out at the end.
  const float so16 = 16.f * reinterpret_cast<const float*>(a.blob + a.rows_off)[t * kTileN + row];

  // ---- 3. activations into LDS
  if constexpr (FUSE == 0) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int pc = tid + i * kThreads;
      if (pc < pieces) *reinterpret_cast<uint4*>(xs + (size_t(pc) << 4)) = xr[i][0];
    }
    if (tid < kDecodeMaxM) s_scale[tid] = tid < M ? a.s_a[tid] : 0.f;
  } else {
    // per-token quantization with the arithmetic of the activation kernel:
    // a = max|x|, s_a = a/127, inv = 127/a, q = clamp(rne(x*inv), +-127)
    float v[PPT][16];
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
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
    // a piece never straddles two tokens (K is a multiple of 16)
    float amax[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) amax[m] = 0.f;
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int pc = tid + i * kThreads;
      const int m = (pc << 4) / K;
      float pm = 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e) pm = fmaxf(pm, fabsf(v[i][e]));
#pragma unroll
      for (int mm = 0; mm < MT; ++mm)
        if (mm == m) amax[mm] = fmaxf(amax[mm], pm);
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) {
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) amax[m] = fmaxf(amax[m], __shfl_xor(amax[m], o, 64));
      if (lane == 0) red[wave][m] = amax[m];
    }
    __syncthreads();
    float inv[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float am = red[0][m];
#pragma unroll
      for (int w = 1; w < kSlices; ++w) am = fmaxf(am, red[w][m]);
      inv[m] = am > 0.f ? 127.f / am : 0.f;
      if (tid == 0) {
        const float sc = am / 127.f;
        s_scale[m] = sc;
        if (blockIdx.x == 0 && m < M) a.s_a_out[m] = sc;
      }
    }
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int pc = tid + i * kThreads;
      if (pc >= pieces) continue;
      const int m = (pc << 4) / K;
      float iv = 0.f;
#pragma unroll
      for (int mm = 0; mm < MT; ++mm)
        if (mm == m) iv = inv[mm];
      float lo8[8], hi8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) { lo8[e] = v[i][e]; hi8[e] = v[i][8 + e]; }
      const uint2 q0 = quant8(lo8, iv), q1 = quant8(hi8, iv);
      const uint4 q = make_uint4(q0.x, q0.y, q1.x, q1.y);
      *reinterpret_cast<uint4*>(xs + (size_t(pc) << 4)) = q;
      if (blockIdx.x == 0 && m < M) *reinterpret_cast<uint4*>(a.Xq_out + (size_t(pc) << 4)) = q;
    }
  }
  __syncthreads();

  // ---- 4. the steps
  float acc[MT], acco[MT];
  int po[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) { acc[m] = 0.f; acco[m] = 0.f; po[m] = 0; }

  for (int s0 = s_begin; s0 < s_end; s0 += kDepth) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      const int s = s0 + d;
      if (s >= s_end) break;  // wave-uniform
      const StepBuf cur = buf[d];
      load_step(s + kDepth, buf[d]);
      const int c = s * kStepChunks + cc;
      const bool valid = c < KC;
      const uint32_t wa[4] = {valid ? cur.w0.x : 0u, valid ? cur.w0.y : 0u, valid ? cur.w0.z : 0u, valid ? cur.w0.w : 0u};
      const uint32_t wb[4] = {valid ? cur.w1.x : 0u, valid ? cur.w1.y : 0u, valid ? cur.w1.z : 0u, valid ? cur.w1.w : 0u};
      const float scl[4] = {f16lo(cur.sc.x), f16hi(cur.sc.x), f16lo(cur.sc.y), f16hi(cur.sc.y)};
      const uint8_t* xbase = xs + uint32_t(min(c, KC - 1)) * kChunkK;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int kb = 4 * j + q;  // 16-K block inside the chunk
        uint32_t sel[2], wi[2], wo_i8[2];
        float wo_f[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint32_t w = h ? wb[q] : wa[q];
          const uint32_t u = __umul24(w & 0x00080808u, kOutPosMagic);
          sel[h] = (u & 0x07000000u) | (w & 0x00070707u);
          wi[h] = w & 0x00F0F0F0u;
          if constexpr (OUT_INT8) wo_i8[h] = w & 0xFF000000u;
          else wo_f[h] = __builtin_amdgcn_cvt_f32_fp8(int(w), 3);
        }
        const uint8_t* xk = xbase + kb * 16;
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const uint4 xv = *reinterpret_cast<const uint4*>(xk + uint32_t(m) * K);
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
  }

  // ---- 5. sum the 16 lanes of a row (j, cc) and fold in the outlier branch
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    if constexpr (OUT_INT8) acco[m] = (float)po[m];
    float v = fmaf(acco[m], so16, acc[m]);
    v += __shfl_xor(v, 4, 64);
    v += __shfl_xor(v, 8, 64);
    v += __shfl_xor(v, 16, 64);
    v += __shfl_xor(v, 32, 64);
    acc[m] = v;
  }
  const int n = t * kTileN + row;
  if constexpr (KSPLIT == 2) {
    // the second half hands its sums to the first through LDS (fixed order)
    if (khalf == 1 && lane < kSliceRows) {
#pragma unroll
      for (int m = 0; m < MT; ++m) part[wslice][m][lane] = acc[m];
    }
    __syncthreads();
    if (khalf == 1) return;
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] += part[wslice][m][r];
  }
  if (lane < kSliceRows && n < a.N) {
#pragma unroll
    for (int m = 0; m < MT; ++m)
      if (m < M) a.Y[size_t(m) * a.N + n] = s_scale[m] * (acc[m] * 0.0625f);
  }
}

template <int MT, int FUSE, int PPT>
hipError_t launch_ppt(const Cfg& c, const DecodeArgs& a, hipStream_t st) {
  const Layout L = make_layout(false, a.N, a.K);
  // slices of 4 rows (the last tile may be padded); a workgroup of 4 waves
  // takes 4 slices, or 2 slices with two waves each when there are too few
  // slices to give every SIMD two waves
  const int64_t slices = L.n_tiles * (kTileN / kSliceRows);
  const size_t lds = size_t(MT) * a.K;
  const bool split = slices < 2048 && (a.K / kChunkK) >= 2 * kStepChunks;
  const dim3 block(kThreads);
  if (split) {
    const dim3 grid(unsigned(slices / (kSlices / 2)));
    if (c.fmt_o == SDQ_FMT_INT8)
      hipLaunchKernelGGL((int_decode_kernel<MT, true, FUSE, PPT, 2>), grid, block, lds, st, a);
    else
      hipLaunchKernelGGL((int_decode_kernel<MT, false, FUSE, PPT, 2>), grid, block, lds, st, a);
  } else {
    const dim3 grid(unsigned(slices / kSlices));
    if (c.fmt_o == SDQ_FMT_INT8)
      hipLaunchKernelGGL((int_decode_kernel<MT, true, FUSE, PPT, 1>), grid, block, lds, st, a);
    else
      hipLaunchKernelGGL((int_decode_kernel<MT, false, FUSE, PPT, 1>), grid, block, lds, st, a);
  }
  return hipGetLastError();
}

template <int MT, int FUSE>
hipError_t launch_mt(const Cfg& c, const DecodeArgs& a, hipStream_t st) {
  const int64_t per_thread = (int64_t(MT) * a.K / 16 + kThreads - 1) / kThreads;
  if (per_thread <= 1) return launch_ppt<MT, FUSE, 1>(c, a, st);
  if (per_thread <= 2) return launch_ppt<MT, FUSE, 2>(c, a, st);
  if (per_thread <= 4) return launch_ppt<MT, FUSE, 4>(c, a, st);
  return launch_ppt<MT, FUSE, 8>(c, a, st);
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

bool decode_fused_fits(int64_t M, int64_t K) { return M <= kFusedMaxM && decode_fits(M, K); }

bool decode_fits(int64_t M, int64_t K) {
  const int64_t mt = M <= 1 ? 1 : M <= 2 ? 2 : M <= 4 ? 4 : 8;
  return M <= kDecodeMaxM && mt * K <= int64_t(16) * kThreads * kMaxPieces;
}

hipError_t launch_int_decode(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                             const uint8_t* blob, int64_t N, int64_t K, float* Y, hipStream_t st) {
  const Layout L = make_layout(false, N, K);
  DecodeArgs a{Xq, s_a, nullptr, nullptr, nullptr, blob, Y, int(M), int(N), int(K),
               int(L.n_chunks), L.scales_off, L.rows_off};
  return launch_fuse<0>(c, a, st);
}

hipError_t launch_int_decode_fused(const Cfg& c, const void* X, int x_dtype, int64_t M,
                                   uint8_t* Xq_out, float* s_a_out, const uint8_t* blob, int64_t N,
                                   int64_t K, float* Y, hipStream_t st) {
  const Layout L = make_layout(false, N, K);
  DecodeArgs a{nullptr, nullptr, X, s_a_out, Xq_out, blob, Y, int(M), int(N), int(K),
               int(L.n_chunks), L.scales_off, L.rows_off};
  if (x_dtype == SDQ_DTYPE_BF16) return launch_fuse<2>(c, a, st);
  return launch_fuse<1>(c, a, st);
}

}  // namespace sdq
