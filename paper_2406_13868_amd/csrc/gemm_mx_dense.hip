// MX-family decomposed GEMM for many tokens, in two passes.  Section 5.1
// computes Y = s_a * Xq (W_o + W_i)^T with both branches accumulated into one
// fp32 accumulator per output.
//
// The one-pass kernel (gemm_mx_mfma.hip) expands every packed weight fragment
// into its merged e4m3 form once per block of tokens.  At prefill sizes that
// vector work, repeated for every 128 tokens, costs more issue cycles than the
// matrix instructions it feeds.  Here every weight is expanded once:
//   pass 1, mx_densify_kernel: every (32-row tile, 128-K chunk) unit of the
//     blob becomes its two merged e4m3 B fragments (mx_frag.h), written to a
//     workspace in the order the matrix instruction reads them;
//   pass 2, mx_dense2_kernel: an fp8 x fp8 scaled-MFMA GEMM over the
//     workspace, the outlier scales (Eo, the merged fragments' e8m0 scales)
//     read from the blob's scale words.
// Blocks whose inliers cannot merge (Ei - Eo outside [-5, 6]) carry only their
// outliers in the merged fragments; pass 2 adds their inliers after its main
// loop with the fp8 x fp4 instruction, when the scale words it read show one.
//
// Workspace layout, one 16-byte piece per lane:
//   uint4 frag[n_tiles][n_chunks][2 steps][2 halves][64 lanes]
// half 0 holds dwords 0-3 and half 1 dwords 4-7 of lane l's fp8 B operand for
// 64-K step s of the chunk, so that every load of a wave is 1 KB contiguous.
//
// Pass 2 tiling: a workgroup of 4 waves owns 128 tokens and 8 row tiles (256
// outputs); each wave owns 2 tiles x 4 sub-tiles of 32 tokens (8 accumulators
// of 32x32), so every A fragment read from LDS feeds two matrix instructions.
// Activations are staged per 128-K chunk in LDS (three buffers,
// XOR-swizzled); B fragments go from the workspace straight into registers.
// Two workgroups run per CU where the grid has them (two waves per SIMD hide
// each other's waits).
//
// What bounds pass 2 (counters on 2048 x 8192 x 4096): the vector memory
// data path, not the matrix cores.  Every wave loads its own B fragments
// (8 KB per chunk) and a quarter of the chunk's activations (4 KB): 750 bytes
// per matrix instruction through the texture data unit, which reads 49% busy
// while the matrix cores read 31%.
#include <hip/hip_runtime.h>

#include <mutex>

#include <type_traits>

#include "kernels.h"
#include "mx_frag.h"
#include "tile_out.h"

namespace sdq {
namespace {

using namespace mx;

constexpr int kUnitPieces = 256;  // uint4 pieces per (tile, chunk) in the workspace
constexpr int kDWaves = 4;
constexpr int kDThreads = kDWaves * 64;
constexpr int kDTiles = 2 * kDWaves;  // row tiles per workgroup
constexpr int kDMS = 4;               // 32-token sub-tiles per wave
constexpr int kDBM = 32 * kDMS;       // tokens per workgroup

// ---- pass 1 ----------------------------------------------------------------
// One wave per (tile, chunk) unit u = tile * n_chunks + chunk, the order of
// the blob's words and scale words, so reads and writes both stream.
template <int NI>
__global__ __launch_bounds__(256) void mx_densify_kernel(const uint8_t* __restrict__ blob,
                                                         int64_t scales_off, int n_units,
                                                         uint4* __restrict__ frag) {
  const int lane = threadIdx.x & 63;
  const int u = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (u >= n_units) return;  // whole waves
  const uint8_t* wp = blob + size_t(u) * kWordBytesPerTC + lane * 16;
  const uint4 w0 = *reinterpret_cast<const uint4*>(wp);
  const uint4 w1 = *reinterpret_cast<const uint4*>(wp + 1024);
  const uint32_t sc =
      *reinterpret_cast<const uint32_t*>(blob + scales_off + size_t(u) * kMxScaleBytesPerTC + lane * 4);
  uint4* out = frag + size_t(u) * kUnitPieces + lane;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const MergedFrag f = expand_merged<NI>(s ? w1 : w0, sc, s);
    out[s * 128] = make_uint4(f.b[0], f.b[1], f.b[2], f.b[3]);
    out[s * 128 + 64] = make_uint4(f.b[4], f.b[5], f.b[6], f.b[7]);
  }
}

// ---- pass 2 ----------------------------------------------------------------
struct DenseArgs {
  const uint8_t* Xq;
  const float* s_a;
  const uint8_t* blob;
  const uint4* frag;
  void* Y;
  int M, N, K, n_chunks, n_tiles;
  int64_t scales_off;
  int m_blocks;  // workgroups along M; the grid is 1-D over (tile group, M block)
};

typedef int i4v __attribute__((ext_vector_type(4)));

// 16 bytes per lane through a buffer resource (tile_out.h)
__device__ __forceinline__ i4v load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}

// whether a lane's scale word (Eo, Ei of its block in steps 0 and 1) holds a
// block that did not merge its inliers
__device__ __forceinline__ bool unmerged(uint32_t sc) {
  const int d0 = int((sc >> 8) & 0xFFu) - int(sc & 0xFFu);
  const int d1 = int((sc >> 24) & 0xFFu) - int((sc >> 16) & 0xFFu);
  return d0 < -5 || d0 > 6 || d1 < -5 || d1 > 6;
}

// Inliers of blocks that did not merge (rare; wave-uniform branches): their
// fp8 x fp4 products accumulate from zero, A read from global memory, and are
// added to the outputs this wave stored.  Called after the main stores, when
// the wave's accumulators are dead, so that no second set is live.
template <int NI, bool YB>
__device__ __forceinline__ void add_unmerged(const DenseArgs& a, const int (&tile)[2], const bool (&tok)[2],
                                             __amdgpu_buffer_rsrc_t xr_rsrc, const OutRows& yr, int m0,
                                             int col, int h, uint32_t boff, uint32_t soff_l,
                                             const __amdgpu_buffer_rsrc_t (&sr)[2]) {
  const int KC = a.n_chunks;
  f16v acc[2][kDMS];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int ms = 0; ms < kDMS; ++ms)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[j][ms][e] = 0.f;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const __amdgpu_buffer_rsrc_t wr =
        buffer_rsrc(a.blob + size_t(tile[j]) * KC * kWordBytesPerTC, uint32_t(KC) * kWordBytesPerTC);
    for (int c = 0; c < KC; ++c) {
      const uint32_t sc = __builtin_amdgcn_raw_buffer_load_b32(sr[j], soff_l, uint32_t(c) * kMxScaleBytesPerTC, 0);
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const uint32_t q = sc >> (16 * s);
        const int d = int((q >> 8) & 0xFFu) - int(q & 0xFFu);
        if (!__any(d < -5 || d > 6)) continue;
        const i4v wv = load16(wr, boff + s * 1024, uint32_t(c) * kWordBytesPerTC);
        i8v bi;
        int ei;
        split_inliers_fp4<NI>(make_uint4(wv[0], wv[1], wv[2], wv[3]), sc, s, bi, ei);
#pragma unroll
        for (int ms = 0; ms < kDMS; ++ms) {
          const uint32_t ao = uint32_t(ms * 32 + col) * uint32_t(a.K) + s * 64 + h * 16;
          const i4v a0 = load16(xr_rsrc, ao, uint32_t(c) * kChunkK);
          const i4v a1 = load16(xr_rsrc, ao + 32, uint32_t(c) * kChunkK);
          const i8v av = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
          acc[j][ms] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bi, acc[j][ms], 0, 4, 0, 127, 0, ei);
        }
      }
    }
  }
  // this wave's output stores complete (in L2) before they are read back
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  const RowScales<kDMS> rs = load_row_scales<kDMS>(a.s_a, a.M, m0, h);
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    if (!tok[j]) continue;
    const int n = tile[j] * kTileN + col;
    if (n >= a.N) continue;
#pragma unroll
    for (int ms = 0; ms < kDMS; ++ms)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        // the stored value, from L2 (glc); a bf16 one was rounded once already
        const uint32_t idx = uint32_t(ms * 32 + tile_row(e, h)) * uint32_t(a.N) + uint32_t(n);
        float y;
        if constexpr (YB)
          y = __uint_as_float(uint32_t(__builtin_amdgcn_raw_buffer_load_b16(yr.r, idx * 2u, 0, 1)) << 16);
        else
          y = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(yr.r, idx * 4u, 0, 1));
        store_out(yr, a.N, n, ms, e, h, y + rs.v[ms][e] * acc[j][ms][e]);
      }
  }
}

// Pass 2: 4 waves own 128 tokens x 256 outputs (each wave 2 row tiles x 4
// token sub-tiles), two workgroups per CU where the grid has them.  How the
// activations reach the matrix instructions:
//   - three LDS chunk buffers: the activations of chunk c + 2 are requested
//     when chunk c starts and written to their buffer when it ends, so the
//     next chunk's buffer is complete and visible before the barrier that
//     ends chunk c;
//   - each sub-tile's A fragment is read from LDS right after the products
//     that used its registers (step 1 of the chunk after step 0, and step 0
//     of the next chunk after step 1, before the barrier), so after a barrier
//     the matrix instructions start on fragments already in registers.
// B fragments go from the workspace straight into registers, each step's
// requested right after that step's products of the previous chunk.
template <int NI, bool YB>
__global__ __launch_bounds__(kDThreads, 2) void mx_dense2_kernel(DenseArgs a) {
  constexpr int kBuf = kDBM * kChunkK;  // 16 KB per chunk
  __shared__ __align__(16) uint8_t xs[3 * kBuf];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, h = lane >> 5;
  int group, mblock;
  tile_work(blockIdx.x, gridDim.x / a.m_blocks, a.m_blocks, group, mblock);
  const int m0 = mblock * kDBM;
  const int KC = a.n_chunks;
  const int last = KC - 1;

  int tile[2];
  bool tok[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int t = group * kDTiles + 2 * wave + j;
    tok[j] = t < a.n_tiles;
    tile[j] = min(t, a.n_tiles - 1);  // spare waves recompute the last tile
  }

  // ---- activations of this block's rows (rows past M read 0, never stored):
  //      thread tid moves piece tid & 7 of rows (tid >> 3) + 32 i, i < 4; rows
  //      r and r + 32 i share their swizzle
  const __amdgpu_buffer_rsrc_t xr_rsrc =
      buffer_rsrc(a.Xq + size_t(m0) * a.K, uint32_t(min(a.M - m0, kDBM)) * uint32_t(a.K));
  const uint32_t xoff = uint32_t(tid >> 3) * uint32_t(a.K) + (tid & 7) * 16;
  const uint32_t xrow32 = 32u * uint32_t(a.K);
  const uint32_t xdst0 = uint32_t((tid >> 3) * kChunkK + (((tid & 7) ^ lds_swizzle(tid >> 3)) << 4));
  struct XRegs { i4v r0, r1, r2, r3; };
  auto load_x = [&](int c, XRegs& x) __attribute__((always_inline)) {
    const uint32_t so = uint32_t(c) * kChunkK;
    x.r0 = load16(xr_rsrc, xoff, so);
    x.r1 = load16(xr_rsrc, xoff + xrow32, so);
    x.r2 = load16(xr_rsrc, xoff + 2 * xrow32, so);
    x.r3 = load16(xr_rsrc, xoff + 3 * xrow32, so);
  };
  auto store_x = [&](uint32_t base, const XRegs& x) __attribute__((always_inline)) {
    *reinterpret_cast<i4v*>(&xs[base + xdst0]) = x.r0;
    *reinterpret_cast<i4v*>(&xs[base + xdst0 + 32 * kChunkK]) = x.r1;
    *reinterpret_cast<i4v*>(&xs[base + xdst0 + 64 * kChunkK]) = x.r2;
    *reinterpret_cast<i4v*>(&xs[base + xdst0 + 96 * kChunkK]) = x.r3;
  };

  // ---- B fragments and scale words of the wave's two tiles
  __amdgpu_buffer_rsrc_t fr[2], sr[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    fr[j] = buffer_rsrc(a.frag + size_t(tile[j]) * KC * kUnitPieces, uint32_t(KC) * kUnitPieces * 16);
    sr[j] = buffer_rsrc(a.blob + a.scales_off + size_t(tile[j]) * KC * kMxScaleBytesPerTC,
                        uint32_t(KC) * kMxScaleBytesPerTC);
  }
  const uint32_t boff = uint32_t(lane) * 16, soff_l = uint32_t(lane) * 4;
  struct BStep { i8v b[2]; };
  auto load_b = [&](int c, int s, BStep& r) __attribute__((always_inline)) {
    const uint32_t so = (uint32_t(c) * 2 + s) * 2048;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const i4v q0 = load16(fr[j], boff, so);
      const i4v q1 = load16(fr[j], boff + 1024, so);
      r.b[j] = __builtin_shufflevector(q0, q1, 0, 1, 2, 3, 4, 5, 6, 7);
    }
  };
  struct Scales { uint32_t w[2]; };
  auto load_sc = [&](int c, Scales& r) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
      r.w[j] = __builtin_amdgcn_raw_buffer_load_b32(sr[j], soff_l, uint32_t(c) * kMxScaleBytesPerTC, 0);
  };

  f16v acc[2][kDMS];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int ms = 0; ms < kDMS; ++ms)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[j][ms][e] = 0.f;

  // A-fragment byte offsets of this lane in a chunk buffer: row ms*32 + col,
  // logical pieces 4s + h and 4s + h + 2 for step s
  uint32_t aoff[2][2];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int u = 0; u < 2; ++u)
      aoff[s][u] = uint32_t(col * kChunkK + (((4 * s + h + 2 * u) ^ lds_swizzle(col)) << 4));
  i8v A[kDMS];
  auto read_a = [&](uint32_t base, int s, int ms) __attribute__((always_inline)) {
    const i4v a0 = *reinterpret_cast<const i4v*>(&xs[base + aoff[s][0] + ms * 32 * kChunkK]);
    const i4v a1 = *reinterpret_cast<const i4v*>(&xs[base + aoff[s][1] + ms * 32 * kChunkK]);
    A[ms] = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  auto pin_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int ms = 0; ms < kDMS; ++ms) asm volatile("" : "+a"(acc[j][ms]));
  };

  bool bad = false;  // this lane saw a block whose inliers did not merge
  BStep B[2];
  Scales S;
  XRegs X;
  load_b(0, 0, B[0]);
  load_b(0, 1, B[1]);
  load_sc(0, S);
  load_x(0, X);
  store_x(0, X);
  load_x(min(1, last), X);
  store_x(kBuf, X);
  __syncthreads();
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the prologue's requests complete
#pragma unroll
  for (int ms = 0; ms < kDMS; ++ms) read_a(0, 0, ms);

  // buffer offsets of chunks c, c + 1 and c + 2 (chunk x in buffer x % 3)
  uint32_t bcur = 0, bnxt = kBuf, bfar = 2 * kBuf;
  for (int c = 0; c < KC; ++c) {  // one exit, so the accumulators stay in place
    load_x(min(c + 2, last), X);
    // keep the requests here: the scheduler would otherwise sink them to the
    // middle of the chunk, half a chunk before the stores that wait on them
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      int e[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) e[j] = int((S.w[j] >> (16 * s)) & 0xFFu);  // Eo of block 2s + h
#pragma unroll
      for (int ms = 0; ms < kDMS; ++ms) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[j][ms] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A[ms], B[s].b[j], acc[j][ms], 0, 0, 0,
                                                                      127, 0, e[j]);
        if (s == 0) read_a(bcur, 1, ms);
        else read_a(bnxt, 0, ms);
      }
      if (s == 1) {
        bad |= unmerged(S.w[0]) || unmerged(S.w[1]);
        load_sc(min(c + 1, last), S);
      }
      load_b(min(c + 1, last), s, B[s]);
    }
    store_x(bfar, X);  // chunk c + 2
    pin_acc();
    __syncthreads();
    const uint32_t t = bcur;
    bcur = bnxt;
    bnxt = bfar;
    bfar = t;
  }

  const OutRows yr = out_rows(a.Y, YB, a.M, a.N, m0, kDBM);
  {
    const RowScales<kDMS> rs = load_row_scales<kDMS>(a.s_a, a.M, m0, h);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (!tok[j]) continue;
      const int n = tile[j] * kTileN + col;
      if (n >= a.N) continue;
#pragma unroll
      for (int ms = 0; ms < kDMS; ++ms)
#pragma unroll
        for (int e = 0; e < 16; ++e) store_out(yr, a.N, n, ms, e, h, rs.v[ms][e] * acc[j][ms][e]);
    }
  }
  if (__any(bad)) add_unmerged<NI, YB>(a, tile, tok, xr_rsrc, yr, m0, col, h, boff, soff_l, sr);
}

template <int NI>
hipError_t densify_ni(const uint8_t* blob, const Layout& L, uint4* frag, hipStream_t st) {
  const int n_units = int(L.n_tiles * L.n_chunks);
  hipLaunchKernelGGL((mx_densify_kernel<NI>), dim3(unsigned((n_units + 3) / 4)), dim3(256), 0, st,
                     blob, L.scales_off, n_units, frag);
  return hipGetLastError();
}

template <int NI>
hipError_t dense_ni(const uint8_t* Xq, const float* s_a, int64_t M, const uint8_t* blob,
                    const Layout& L, int64_t N, int64_t K, void* Y, bool y_bf16, const uint4* frag,
                    hipStream_t st) {
  DenseArgs a{Xq, s_a, blob, frag, Y, int(M), int(N), int(K), int(L.n_chunks), int(L.n_tiles),
              L.scales_off, int((M + kDBM - 1) / kDBM)};
  const int groups = int((L.n_tiles + kDTiles - 1) / kDTiles);
  const unsigned wgs = unsigned(groups * a.m_blocks);
  if (y_bf16)
    hipLaunchKernelGGL((mx_dense2_kernel<NI, true>), dim3(wgs), dim3(kDThreads), 0, st, a);
  else
    hipLaunchKernelGGL((mx_dense2_kernel<NI, false>), dim3(wgs), dim3(kDThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace

size_t mx_dense_workspace_bytes(int64_t N, int64_t K) {
  const Layout L = make_layout(true, N, K);
  return size_t(L.n_tiles) * size_t(L.n_chunks) * kUnitPieces * sizeof(uint4);
}

hipError_t launch_mx_densify(const Cfg& c, const uint8_t* blob, int64_t N, int64_t K, void* workspace,
                             hipStream_t st) {
  const Layout L = make_layout(true, N, K);
  uint4* frag = static_cast<uint4*>(workspace);
  if (c.n_i == 1) return densify_ni<1>(blob, L, frag, st);
  if (c.n_i == 2) return densify_ni<2>(blob, L, frag, st);
  return densify_ni<3>(blob, L, frag, st);
}

hipError_t launch_mx_dense_pass(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                                const uint8_t* blob, int64_t N, int64_t K, void* Y, const void* workspace,
                                hipStream_t st) {
  const Layout L = make_layout(true, N, K);
  const uint4* frag = static_cast<const uint4*>(workspace);
  if (c.n_i == 1) return dense_ni<1>(Xq, s_a, M, blob, L, N, K, Y, c.y_bf16, frag, st);
  if (c.n_i == 2) return dense_ni<2>(Xq, s_a, M, blob, L, N, K, Y, c.y_bf16, frag, st);
  return dense_ni<3>(Xq, s_a, M, blob, L, N, K, Y, c.y_bf16, frag, st);
}

hipError_t launch_mx_dense(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                           const uint8_t* blob, int64_t N, int64_t K, void* Y, void* workspace,
                           hipStream_t st) {
  const hipError_t e = launch_mx_densify(c, blob, N, K, workspace, st);
  if (e != hipSuccess) return e;
  return launch_mx_dense_pass(c, Xq, s_a, M, blob, N, K, Y, workspace, st);
}

}  // namespace sdq

// ------------------------------------------------------------ static scratch
// The workspace of sdq_gemm_static, for callers that cannot allocate: one
// array per GPU, which that GPU holds until the process ends.  In host code
// the array's name stands for a host-side shadow, not a device address, so it
// is never passed to a kernel or a copy: the device address is looked up once
// per device with hipGetSymbolAddress and only that address is used.
static __device__ __align__(256) uint8_t scratch[sdq::kStaticScratchBytes];

namespace sdq {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The scratch array's address on the current device (looked up on the first
// call with that device current).
hipError_t static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

hipError_t split_static(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                        const uint8_t* blob, int64_t N, int64_t K, void* Y, hipStream_t st) {
  const size_t need = c.mx ? mx_split_workspace_bytes(M, N, K) : int_split_workspace_bytes(M, N, K);
  if (need > kStaticScratchBytes) return hipErrorInvalidValue;
  void* ws = nullptr;
  const hipError_t e = static_scratch(&ws);
  if (e != hipSuccess) return e;
  return c.mx ? launch_mx_split(c, Xq, s_a, M, blob, N, K, Y, ws, st)
              : launch_int_split(c, Xq, s_a, M, blob, N, K, Y, ws, st);
}

hipError_t launch_mx_dense_static(const Cfg& c, const uint8_t* Xq, const float* s_a, int64_t M,
                                  const uint8_t* blob, int64_t N, int64_t K, void* Y,
                                  hipStream_t st) {
  if (mx_dense_workspace_bytes(N, K) > kStaticScratchBytes) return hipErrorInvalidValue;
  void* ws = nullptr;
  const hipError_t e = static_scratch(&ws);
  if (e != hipSuccess) return e;
  return launch_mx_dense(c, Xq, s_a, M, blob, N, K, Y, ws, st);
}

}  // namespace sdq
