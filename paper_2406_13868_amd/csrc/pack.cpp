// Offline SDQ packer (host): Section 5, Stages 1-3 of the paper.
//
//   Stage 1+2  In every m_o-group of a row the n_o most significant positions
//              become the outliers (local outlier extraction, Section 4); in
//              every 8-group the n_i most significant remaining positions
//              become the inliers; everything else is pruned.  Significance
//              is |w| or |w| * act_norm[k] (Wanda's product metric); ties go
//              to the lower k.  With a separate decomposition metric (the
//              variants of Section 6.4's decomposition study) the stages run in
//              the paper's order instead: sparsify every 8-group to
//              n_o + n_i kept positions, then extract the outliers among the
//              kept ones by that metric, largest or smallest first.
//   Stage 3    Per-vector quantization of each branch (VS-Quant style), with
//              the formats of the configuration's family.
//
// Arithmetic is IEEE fp32 with round-to-nearest-even, in the order stated in
// sdq.h, so that the result is reproducible bit for bit.  The packer writes
// either the logical form (positions, codes, scales) or the kernel layout
// described in layout.h.  Rows are independent; worker threads take
// contiguous row ranges, so the output does not depend on the thread count.
#include <atomic>
#include <cmath>
#include <algorithm>
#include <cstring>
#include <thread>
#include <vector>

#include "layout.h"
#include "sdq_internal.h"

namespace sdq {
namespace {

// ---------------------------------------------------------------- encoders
// fp32 -> IEEE binary16 bits, round to nearest even.
uint16_t f32_to_f16_bits(float f) {
  uint32_t x;
  std::memcpy(&x, &f, 4);
  const uint32_t sign = (x >> 16) & 0x8000u;
  const uint32_t ax = x & 0x7FFFFFFFu;
  if (ax >= 0x7F800000u) return uint16_t(sign | 0x7C00u | (ax > 0x7F800000u ? 0x200u : 0u));
  const int e = int(ax >> 23) - 127;  // unbiased exponent of the fp32 value
  if (e > 15) return uint16_t(sign | 0x7C00u);  // overflow to infinity
  uint32_t mant = (ax & 0x7FFFFFu) | 0x800000u;  // 24-bit significand (normal input)
  if (ax < 0x00800000u) return uint16_t(sign);     // fp32 subnormal: far below fp16 range
  int shift;                                        // bits to drop from the 24-bit significand
  uint32_t exp_field;
  if (e >= -14) {                                   // fp16 normal
    shift = 13;
    exp_field = uint32_t(e + 15);
  } else {                                          // fp16 subnormal (or underflow)
    shift = 13 + (-14 - e);
    exp_field = 0;
    if (shift > 24) return uint16_t(sign);
  }
  uint32_t q = mant >> shift;
  const uint32_t rem = mant & ((1u << shift) - 1u);
  const uint32_t half = 1u << (shift - 1);
  if (rem > half || (rem == half && (q & 1u))) ++q;
  uint32_t bits;
  if (exp_field) {
    bits = (exp_field << 10) + (q - 0x400u);  // q in [0x400, 0x800]; carry bumps the exponent
  } else {
    bits = q;  // subnormal; q == 0x400 rounds up into the smallest normal
  }
  if (bits >= 0x7C00u) bits = 0x7C00u;
  return uint16_t(sign | bits);
}

float f16_bits_to_f32(uint16_t h) {
  const uint32_t sign = uint32_t(h & 0x8000u) << 16;
  const uint32_t e = (h >> 10) & 0x1F, m = h & 0x3FF;
  float v;
  if (e == 0) v = std::ldexp(float(m), -24);
  else if (e == 31) v = m ? NAN : INFINITY;
  else v = std::ldexp(float(m | 0x400u), int(e) - 25);
  uint32_t b;
  std::memcpy(&b, &v, 4);
  b |= sign;
  std::memcpy(&v, &b, 4);
  return v;
}

// Nearest-even OCP fp8 E4M3FN code of x, saturating at +-448; keeps the sign.
uint8_t enc_e4m3(double x) {
  const uint8_t s = std::signbit(x) ? 0x80 : 0x00;
  double a = std::fabs(x);
  if (a > 448.0) a = 448.0;
  if (a < 0.015625) {  // below 2^-6: subnormal spacing 2^-9
    const int q = int(std::nearbyint(a * 512.0));  // 8 becomes the first normal code
    return uint8_t(s | q);
  }
  int e;
  const double f = std::frexp(a, &e);  // a = f * 2^e, f in [0.5, 1)
  int E = e - 1;
  int mq = int(std::nearbyint((2.0 * f - 1.0) * 8.0));
  if (mq == 8) { ++E; mq = 0; }
  return uint8_t(s | ((E + 7) << 3) | mq);
}

// Value of a non-NaN OCP fp8 E4M3FN code.
float e4m3_value(uint8_t code) {
  const int e = (code >> 3) & 0xF, m = code & 7;
  const float a = e ? std::ldexp(float(8 + m), e - 10) : std::ldexp(float(m), -9);
  return (code & 0x80) ? -a : a;
}

// Nearest-even OCP fp4 E2M1 code (low nibble), saturating at +-6; keeps the sign.
uint8_t enc_e2m1(double x) {
  const uint8_t s = std::signbit(x) ? 0x8 : 0x0;
  double a = std::fabs(x);
  if (a > 6.0) a = 6.0;
  if (a < 1.0) return uint8_t(s | int(std::nearbyint(a * 2.0)));  // 0, 0.5, (1.0)
  int e;
  const double f = std::frexp(a, &e);
  int E = e - 1;
  int mq = int(std::nearbyint((2.0 * f - 1.0) * 2.0));
  if (mq == 2) { ++E; mq = 0; }
  return uint8_t(s | ((E + 1) << 1) | mq);
}

// Nearest-even ufp8 E6M2 code of a >= 0 (6 exponent bits with bias 31, 2
// mantissa bits, no sign; exponent field 0 holds m/4 * 2^-30), saturating at
// the largest code, 1.75 * 2^32.
uint8_t enc_ue6m2(double a) {
  const double kMax = 1.75 * 4294967296.0;
  if (a > kMax) a = kMax;
  if (a < std::ldexp(1.0, -30)) {  // subnormal spacing 2^-32
    const int q = int(std::nearbyint(std::ldexp(a, 32)));  // 4 becomes the first normal code
    return uint8_t(q);
  }
  int e;
  const double f = std::frexp(a, &e);  // a = f * 2^e, f in [0.5, 1)
  int E = e - 1;
  int mq = int(std::nearbyint((2.0 * f - 1.0) * 4.0));
  if (mq == 4) { ++E; mq = 0; }
  return uint8_t(((E + 31) << 2) | mq);
}

// Value of a ufp8 E6M2 code (exact in fp32).
float ue6m2_value(uint8_t code) {
  const int e = code >> 2, m = code & 3;
  return e ? std::ldexp(float(4 + m), e - 33) : std::ldexp(float(m), -32);
}

int floor_log2f(float a) {
  int e;
  std::frexp(a, &e);
  return e - 1;
}

int clamp_int(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// The first n allowed positions of a group by (-S, k); returns a position mask.
uint32_t top_n(const float* S, uint32_t allowed, int m, int n) {
  float bs[16];
  int bk[16];
  int cnt = 0;
  for (int p = 0; p < m; ++p) {
    if (!((allowed >> p) & 1u)) continue;
    const float s = S[p];
    int pos = cnt;
    while (pos > 0 && bs[pos - 1] < s) --pos;  // equal keys keep the earlier k
    if (pos >= n) continue;
    const int last = cnt < n ? cnt : n - 1;
    for (int q = last; q > pos; --q) { bs[q] = bs[q - 1]; bk[q] = bk[q - 1]; }
    bs[pos] = s;
    bk[pos] = p;
    if (cnt < n) ++cnt;
  }
  uint32_t mask = 0;
  for (int i = 0; i < cnt; ++i) mask |= 1u << bk[i];
  return mask;
}

// ---------------------------------------------------------------- selection
// Per-thread scratch of the row packer.
struct Scratch {
  std::vector<float> S, D;          // significance, decomposition key (K each)
  std::vector<uint8_t> om8, im8;    // outlier / inlier position masks per 8-group
  std::vector<float> V;             // INT: effective inlier scale per 16-K block
  std::vector<uint16_t> SC;         // INT: stored scale per block (fp16 bits or e4m3 code)
  explicit Scratch(int64_t K)
      : S(size_t(K)), D(size_t(K)), om8(size_t(K / 8)), im8(size_t(K / 8)),
        V(size_t(K / 16)), SC(size_t(K / 16)) {}
};

// INT-family inlier scales of one row over the positions `mask8`: per
// Q-Vector of c.qv dense K, v = amax / 7 (fp32), stored as fp16 (eff = that
// fp16 value); with two-level e4m3 scales as e4m3(v * 2^-E), E the smallest
// exponent that puts the row's largest v within 448 * 2^E (eff = value * 2^E,
// exact); or as ufp8-e6m2(v) (eff = its value, exact).  Writes eff to V and
// the stored scales to SC; returns the row scale 2^E (0 for a row without
// inlier magnitude, always 0 for fp16 and e6m2 scales).  A nonzero e6m2 scale
// must have exponent field 9..43 ([2^-22, 7168], where an int4 code times it is
// exact in fp16): SDQ_ERR_VALUE otherwise, as for an fp16 overflow.
sdq_status int_inlier_scales(const Cfg& c, const float* w, int64_t K, const uint8_t* mask8, float* V,
                             uint16_t* SC, float* row_scale) {
  const int qv = c.qv;
  const int64_t B = K / qv;
  float vmax = 0.f;
  for (int64_t b = 0; b < B; ++b) {
    float a = 0.f;
    for (int kk = 0; kk < qv; ++kk) {
      const int64_t k = b * qv + kk;
      if ((mask8[k / 8] >> (k % 8)) & 1u) a = std::fmax(a, std::fabs(w[k]));
    }
    V[b] = a / 7.0f;
    vmax = std::fmax(vmax, V[b]);
  }
  *row_scale = 0.f;
  if (c.e6m2) {
    for (int64_t b = 0; b < B; ++b) {
      const uint8_t code = enc_ue6m2(double(V[b]));
      const int e = code >> 2;
      if (code != 0 && (e < 9 || e > 43)) return SDQ_ERR_VALUE;  // beyond the exact fp16 range
      SC[b] = code;
      V[b] = ue6m2_value(code);
    }
    return SDQ_OK;
  }
  if (!c.sc8) {
    for (int64_t b = 0; b < B; ++b) {
      const uint16_t h = f32_to_f16_bits(V[b]);
      if ((h & 0x7C00u) == 0x7C00u) return SDQ_ERR_VALUE;  // scale overflows fp16
      SC[b] = h;
      V[b] = f16_bits_to_f32(h);
    }
    return SDQ_OK;
  }
  int E = 0;
  if (vmax > 0.f) {
    E = floor_log2f(vmax) - 8;                        // 448 * 2^(fl - 8) = 1.75 * 2^fl
    if (double(vmax) > std::ldexp(448.0, E)) ++E;
    *row_scale = std::ldexp(1.0f, E);
  }
  for (int64_t b = 0; b < B; ++b) {
    const uint8_t code = vmax > 0.f ? enc_e4m3(std::ldexp(double(V[b]), -E)) : uint8_t(0);
    SC[b] = code;
    V[b] = std::ldexp(e4m3_value(code), E);
  }
  return SDQ_OK;
}

// The inlier quantizer applied to the positions `keep8` of row w, and the
// error it makes on each of them: D[k] = |w[k] - deq[k]| (fp32), 0 off the
// kept positions.  Same scale rules as the final inlier quantization.
sdq_status inlier_error(const Cfg& c, const float* w, int64_t K, const uint8_t* keep8, float* D,
                        float* V, uint16_t* SC) {
  const bool mx_in = c.mx || c.dual;  // fp4 inliers with e8m0 scales per 32 K
  const int qv = mx_in ? 32 : c.qv;
  if (!mx_in) {
    float row;
    const sdq_status st = int_inlier_scales(c, w, K, keep8, V, SC, &row);
    if (st != SDQ_OK) return st;
  }
  for (int64_t k0 = 0; k0 < K; k0 += qv) {
    float a = 0.f;
    for (int kk = 0; kk < qv; ++kk) {
      const int64_t k = k0 + kk;
      if ((keep8[k / 8] >> (k % 8)) & 1u) a = std::fmax(a, std::fabs(w[k]));
    }
    for (int kk = 0; kk < qv; ++kk) {
      const int64_t k = k0 + kk;
      float deq = 0.f;
      if (mx_in) {
        if (a > 0.f) {
          const int E = clamp_int(floor_log2f(a) - 2, -127, 127);
          const uint8_t q = enc_e2m1(std::ldexp(double(w[k]), -E));
          static const float mag[8] = {0.f, 0.5f, 1.f, 1.5f, 2.f, 3.f, 4.f, 6.f};
          deq = std::ldexp((q & 8u) ? -mag[q & 7u] : mag[q & 7u], E);
        }
      } else {
        const float sc = V[k0 / qv];
        if (sc != 0.f) deq = float(clamp_int(int(std::nearbyint(w[k] / sc)), -7, 7)) * sc;
      }
      D[k] = ((keep8[k / 8] >> (k % 8)) & 1u) ? std::fabs(w[k] - deq) : 0.f;
    }
  }
  return SDQ_OK;
}

// Outlier and inlier masks of every 8-group of row w into sc.om8 / sc.im8.
sdq_status select_row(const Cfg& c, const float* w, const float* act_norm, int64_t K, Scratch& sc) {
  float* S = sc.S.data();
  float* D = sc.D.data();
  uint8_t* om8 = sc.om8.data();
  uint8_t* im8 = sc.im8.data();
  const int64_t G8 = K / 8, Go = K / c.m_o;
  for (int64_t k = 0; k < K; ++k) {
    if (!std::isfinite(w[k])) return SDQ_ERR_VALUE;
    S[k] = std::fabs(w[k]);
    if (c.metric == SDQ_METRIC_PRODUCT) S[k] = S[k] * act_norm[k];
  }
  auto set_outliers = [&](int64_t go, uint32_t mk) {
    if (c.m_o == 8) {
      om8[go] = uint8_t(mk);
    } else {  // m_o == 16
      om8[2 * go] = uint8_t(mk & 0xFFu);
      om8[2 * go + 1] = uint8_t(mk >> 8);
    }
  };
  const bool staged = c.decomp != SDQ_DECOMP_SAME || c.order != SDQ_ORDER_LARGE;
  if (!staged) {
    // outliers first over each whole m_o-group, then inliers among the rest
    for (int64_t g = 0; g < G8; ++g) om8[g] = 0;
    if (c.n_o)
      for (int64_t go = 0; go < Go; ++go) set_outliers(go, top_n(S + go * c.m_o, (1u << c.m_o) - 1u, c.m_o, c.n_o));
    for (int64_t g = 0; g < G8; ++g) im8[g] = uint8_t(top_n(S + g * 8, 0xFFu & ~uint32_t(om8[g]), 8, c.n_i));
  } else {
    // Stage 1: every 8-group keeps its n_o + n_i most significant positions
    // (held in im8 until the inliers are chosen)
    for (int64_t g = 0; g < G8; ++g) im8[g] = uint8_t(top_n(S + g * 8, 0xFFu, 8, c.n_o + c.n_i));
    // Stage 2: the decomposition key, negated for the smallest-first order
    switch (c.decomp) {
      case SDQ_DECOMP_SAME:
        for (int64_t k = 0; k < K; ++k) D[k] = S[k];
        break;
      case SDQ_DECOMP_MAGNITUDE:
        for (int64_t k = 0; k < K; ++k) D[k] = std::fabs(w[k]);
        break;
      case SDQ_DECOMP_PRODUCT:
        for (int64_t k = 0; k < K; ++k) D[k] = std::fabs(w[k]) * act_norm[k];
        break;
      default: {
        const sdq_status st = inlier_error(c, w, K, im8, D, sc.V.data(), sc.SC.data());
        if (st != SDQ_OK) return st;
        if (c.decomp == SDQ_DECOMP_OUTPUT_ERROR)
          for (int64_t k = 0; k < K; ++k) D[k] = D[k] * act_norm[k];
      }
    }
    if (c.order == SDQ_ORDER_SMALL)
      for (int64_t k = 0; k < K; ++k) D[k] = -D[k];
    for (int64_t go = 0; go < Go; ++go) {
      const uint32_t kept = c.m_o == 8 ? uint32_t(im8[go]) : (uint32_t(im8[2 * go]) | (uint32_t(im8[2 * go + 1]) << 8));
      set_outliers(go, top_n(D + go * c.m_o, kept, c.m_o, c.n_o));
    }
    for (int64_t g = 0; g < G8; ++g) im8[g] = uint8_t(top_n(S + g * 8, uint32_t(im8[g]) & ~uint32_t(om8[g]), 8, c.n_i));
  }
  for (int64_t g = 0; g < G8; ++g) {
    int cnt = 0;
    for (int p = 0; p < 8; ++p) cnt += (im8[g] >> p) & 1;
    if (cnt != c.n_i) return SDQ_ERR_CONFIG;  // fewer candidates than slots
  }
  return SDQ_OK;
}

// ---------------------------------------------------------------- one row
// Everything the packer decides for one row of W.
struct RowSink {
  // logical outputs (any may be null)
  uint8_t* pos_o; uint8_t* code_o; void* scale_o;
  uint8_t* pos_i; uint8_t* code_i; void* scale_i; float* scale_i_row;
  // kernel layout output (may be null)
  uint8_t* blob;
  const Layout* lay;        // int and mx families
  const DualLayout* dlay;   // dual family
};

// Packs row n with the per-thread scratch sc.
sdq_status pack_row(const Cfg& c, const float* w, const float* act_norm, int64_t K, int64_t n,
                    Scratch& sc, const RowSink& out) {
  {
    const sdq_status st = select_row(c, w, act_norm, K, sc);
    if (st != SDQ_OK) return st;
  }
  const uint8_t* om8 = sc.om8.data();
  const uint8_t* im8 = sc.im8.data();
  const int64_t G8 = K / 8, Go = K / c.m_o;

  // ---- outlier row scale (INT family) needs the row amax over the outliers
  float s_o = 0.f;
  if (!c.mx && c.n_o) {
    float a = 0.f;
    for (int64_t k = 0; k < K; ++k)
      if ((om8[k / 8] >> (k % 8)) & 1u) a = std::fmax(a, std::fabs(w[k]));
    s_o = a / (c.fmt_o == SDQ_FMT_INT8 ? 127.0f : 448.0f);
    if (out.scale_o) static_cast<float*>(out.scale_o)[n] = s_o;
  }

  // ---- inlier block scales of the row (INT family)
  float s_irow = 0.f;
  if (!c.mx && !c.dual) {
    const sdq_status st = int_inlier_scales(c, w, K, im8, sc.V.data(), sc.SC.data(), &s_irow);
    if (st != SDQ_OK) return st;
    if (out.scale_i_row) out.scale_i_row[n] = s_irow;
  }

  // ---- walk 32-K spans (one MX block, two INT blocks, four 8-groups)
  const int64_t r = n % kTileN, t = n / kTileN;
  for (int64_t k0 = 0; k0 < K; k0 += 32) {
    uint32_t om[4], im[4];  // per 8-group position masks
    for (int gg = 0; gg < 4; ++gg) {
      om[gg] = om8[k0 / 8 + gg];
      im[gg] = im8[k0 / 8 + gg];
    }

    // ---- scales and codes
    uint8_t ocode[32] = {0}, icode[32] = {0};  // per position of the span
    if (c.mx) {
      float ao = 0.f, ai = 0.f;
      for (int gg = 0; gg < 4; ++gg)
        for (int p = 0; p < 8; ++p) {
          const float v = std::fabs(w[k0 + 8 * gg + p]);
          if ((om[gg] >> p) & 1u) ao = std::fmax(ao, v);
          if ((im[gg] >> p) & 1u) ai = std::fmax(ai, v);
        }
      const int Eo = ao > 0.f ? clamp_int(floor_log2f(ao) - 8, -127, 127) : -127;
      const int Ei = ai > 0.f ? clamp_int(floor_log2f(ai) - 2, -127, 127) : -127;
      for (int gg = 0; gg < 4; ++gg)
        for (int p = 0; p < 8; ++p) {
          const int kk = 8 * gg + p;
          const double v = double(w[k0 + kk]);
          if (((om[gg] >> p) & 1u) && ao > 0.f) ocode[kk] = enc_e4m3(std::ldexp(v, -Eo));
          if (((im[gg] >> p) & 1u) && ai > 0.f) icode[kk] = enc_e2m1(std::ldexp(v, -Ei));
        }
      const int64_t b = k0 / 32;
      if (out.scale_o && c.n_o) static_cast<uint8_t*>(out.scale_o)[n * (K / 32) + b] = uint8_t(Eo + 127);
      if (out.scale_i) static_cast<uint8_t*>(out.scale_i)[n * (K / 32) + b] = uint8_t(Ei + 127);
      if (out.blob) {
        const int64_t ch = k0 / kChunkK;
        const int bb = int((k0 % kChunkK) / 32);
        uint8_t* sb = out.blob + out.lay->scales_off + (t * out.lay->n_chunks + ch) * kMxScaleBytesPerTC;
        sb[mx_scale_byte(bb, int(r), 0)] = c.n_o ? uint8_t(Eo + 127) : 0;
        sb[mx_scale_byte(bb, int(r), 1)] = uint8_t(Ei + 127);
      }
    } else if (c.dual) {
      // fp4 inliers with an e8m0 scale per 32 K (the MX rule)
      float ai = 0.f;
      for (int gg = 0; gg < 4; ++gg)
        for (int p = 0; p < 8; ++p)
          if ((im[gg] >> p) & 1u) ai = std::fmax(ai, std::fabs(w[k0 + 8 * gg + p]));
      const int Ei = ai > 0.f ? clamp_int(floor_log2f(ai) - 2, -127, 127) : -127;
      for (int gg = 0; gg < 4; ++gg)
        for (int p = 0; p < 8; ++p)
          if (((im[gg] >> p) & 1u) && ai > 0.f)
            icode[8 * gg + p] = enc_e2m1(std::ldexp(double(w[k0 + 8 * gg + p]), -Ei));
      const int64_t b = k0 / 32;
      if (out.scale_i) static_cast<uint8_t*>(out.scale_i)[n * (K / 32) + b] = uint8_t(Ei + 127);
      if (out.blob) {
        const int64_t ch = k0 / kChunkK;
        out.blob[out.dlay->scale_off + (t * out.dlay->n_chunks + ch) * kDualScaleBytesPerTC +
                 dual_scale_byte(int((k0 % kChunkK) / 32), int(r))] = uint8_t(Ei + 127);
      }
      // int8 outliers with the row scale
      if (c.n_o && s_o != 0.f)
        for (int gg = 0; gg < 4; ++gg)
          for (int p = 0; p < 8; ++p)
            if ((om[gg] >> p) & 1u)
              ocode[8 * gg + p] = uint8_t(int8_t(clamp_int(int(std::nearbyint(w[k0 + 8 * gg + p] / s_o)), -127, 127)));
    } else {
      const int qv = c.qv, sbytes = c.scale_bytes();
      for (int gg = 0; gg < 4; ++gg) {  // the four 8-groups of the span
        const int64_t kg = k0 + 8 * gg;
        const int64_t kb = kg / qv;      // its Q-Vector
        const float s = sc.V[kb];
        for (int p = 0; p < 8; ++p)
          if (((im[gg] >> p) & 1u) && s != 0.f) {
            const float v = w[kg + p] / s;
            icode[8 * gg + p] = uint8_t(int8_t(clamp_int(int(std::nearbyint(v)), -7, 7)));
          }
        if (kg % qv != 0) continue;  // the Q-Vector's scale is written at its first group
        const uint16_t h = sc.SC[kb];
        if (out.scale_i) {
          if (sbytes == 1) static_cast<uint8_t*>(out.scale_i)[n * (K / qv) + kb] = uint8_t(h);
          else static_cast<uint16_t*>(out.scale_i)[n * (K / qv) + kb] = h;
        }
        if (out.blob) {
          const int64_t ch = kg / kChunkK;
          const int kbl = int((kg % kChunkK) / qv);
          uint8_t* sb = out.blob + out.lay->scales_off + (t * out.lay->n_chunks + ch) * out.lay->scale_bytes_per_tc;
          if (sbytes == 1) sb[int_scale_off(kbl, int(r), qv, 1)] = uint8_t(h);
          else std::memcpy(sb + int_scale_off(kbl, int(r), qv, 2), &h, 2);
        }
      }
      if (c.n_o && s_o != 0.f) {
        for (int gg = 0; gg < 4; ++gg)
          for (int p = 0; p < 8; ++p)
            if ((om[gg] >> p) & 1u) {
              const float v = w[k0 + 8 * gg + p] / s_o;
              ocode[8 * gg + p] = c.fmt_o == SDQ_FMT_INT8
                                      ? uint8_t(int8_t(clamp_int(int(std::nearbyint(v)), -127, 127)))
                                      : enc_e4m3(double(v));
            }
      }
    }

    // ---- logical outputs
    for (int gg = 0; gg < 4; ++gg) {
      const int64_t g8 = k0 / 8 + gg;
      int j = 0;
      for (int p = 0; p < 8; ++p)
        if ((im[gg] >> p) & 1u) {
          if (out.pos_i) out.pos_i[(n * G8 + g8) * c.n_i + j] = uint8_t(p);
          if (out.code_i) out.code_i[(n * G8 + g8) * c.n_i + j] = icode[8 * gg + p];
          ++j;
        }
    }
    if (c.n_o) {
      const int per = 32 / c.m_o;  // outlier groups in this span
      for (int go = 0; go < per; ++go) {
        const int64_t gidx = k0 / c.m_o + go;
        int j = 0;
        for (int p = 0; p < c.m_o; ++p) {
          const int kk = go * c.m_o + p;
          if ((om[kk / 8] >> (kk % 8)) & 1u) {
            if (out.pos_o) out.pos_o[(n * Go + gidx) * c.n_o + j] = uint8_t(p);
            if (out.code_o) out.code_o[(n * Go + gidx) * c.n_o + j] = ocode[kk];
            ++j;
          }
        }
      }
    }

    // ---- kernel layout
    if (out.blob && c.dual) {
      const int64_t ch = k0 / kChunkK;
      const int64_t tc = t * out.dlay->n_chunks + ch;
      uint8_t* nib = out.blob + out.dlay->nib_off + tc * kDualNibBytesPerTC;
      uint16_t* hw = reinterpret_cast<uint16_t*>(out.blob + out.dlay->out_off + tc * out.dlay->out_bytes_per_tc);
      for (int kk = 0; kk < 32; ++kk) {
        const int k = int(k0 % kChunkK) + kk;
        nib[dual_nib_byte(k, int(r))] |= uint8_t((icode[kk] & 0xFu) << ((k & 1) * 4));
      }
      // the j-th outlier of a group (ascending position) in plane j; a plane
      // without one keeps the zero half-word
      for (int gg = 0; gg < 4; ++gg) {
        int j = 0;
        for (int p = 0; p < 8; ++p)
          if ((om[gg] >> p) & 1u) {
            hw[j * (kDualOutBytesPerTC / 2) + dual_out_halfword(int((k0 % kChunkK) / 8) + gg, int(r))] =
                uint16_t(p | (ocode[8 * gg + p] << 8));
            ++j;
          }
      }
    } else if (out.blob) {
      const int64_t ch = k0 / kChunkK;
      uint32_t* words = reinterpret_cast<uint32_t*>(out.blob + out.lay->words_off) +
                        (t * out.lay->n_chunks + ch) * kWordsPerTC;
      for (int gg = 0; gg < 4; ++gg) {
        uint32_t word = 0;
        int j = 0;
        for (int p = 0; p < 8; ++p)
          if ((im[gg] >> p) & 1u) {
            word |= uint32_t(p) << (8 * j);
            word |= uint32_t(icode[8 * gg + p] & 0xF) << (8 * j + 4);
            ++j;
          }
        // the outlier of the group, or (1:16 word without one, or no outlier
        // branch) code 0 at the lowest position no inlier occupies
        int po = 0;
        while ((im[gg] >> po) & 1u) ++po;
        uint32_t oc = 0;
        for (int p = 0; p < 8; ++p)
          if ((om[gg] >> p) & 1u) {
            po = p;
            oc = ocode[8 * gg + p];
          }
        for (int bit = 0; bit < 3; ++bit) word |= uint32_t((po >> bit) & 1) << (8 * bit + 3);
        word |= oc << 24;
        const int g = int((k0 % kChunkK) / 8) + gg;
        words[c.mx ? mx_word_index(g, int(r)) : int_word_index(g, int(r))] = word;
      }
    }
  }
  if (out.blob && c.dual) {
    reinterpret_cast<float*>(out.blob + out.dlay->rows_off)[n] = s_o;
  } else if (out.blob && !c.mx) {
    float* rows = reinterpret_cast<float*>(out.blob + out.lay->rows_off);
    rows[n] = s_o;
    if (c.sc8) reinterpret_cast<float*>(out.blob + out.lay->irow_off)[n] = s_irow;
  }
  return SDQ_OK;
}

int resolve_threads(int n_threads, int64_t N) {
  int T = n_threads > 0 ? n_threads : int(std::thread::hardware_concurrency());
  if (T < 1) T = 1;
  if (T > 256) T = 256;
  if (int64_t(T) > N) T = int(N);
  return T;
}

sdq_status run_rows(const Cfg& c, const float* W, int64_t N, int64_t K, const float* act_norm,
                    const RowSink& sink, int n_threads) {
  const int T = resolve_threads(n_threads, N);
  std::atomic<int> err{SDQ_OK};
  auto work = [&](int64_t r0, int64_t r1) {
    Scratch sc(K);
    for (int64_t n = r0; n < r1 && err.load(std::memory_order_relaxed) == SDQ_OK; ++n) {
      const sdq_status s = pack_row(c, W + n * K, act_norm, K, n, sc, sink);
      if (s != SDQ_OK) {
        int expect = SDQ_OK;
        err.compare_exchange_strong(expect, s);
      }
    }
  };
  if (T == 1) {
    work(0, N);
  } else {
    std::vector<std::thread> pool;
    pool.reserve(size_t(T));
    for (int i = 0; i < T; ++i) pool.emplace_back(work, N * i / T, N * (i + 1) / T);
    for (auto& th : pool) th.join();
  }
  return sdq_status(err.load());
}

sdq_status check_act_norm(const Cfg& c, const float* act_norm, int64_t K) {
  if (!needs_act_norm(c)) return SDQ_OK;
  if (!act_norm) return SDQ_ERR_NULL;
  for (int64_t k = 0; k < K; ++k)
    if (!std::isfinite(act_norm[k]) || act_norm[k] < 0.f) return SDQ_ERR_VALUE;
  return SDQ_OK;
}

}  // namespace
}  // namespace sdq

using namespace sdq;

extern "C" sdq_status sdq_pack_size(const sdq_config* cfg, int64_t N, int64_t K, size_t* bytes) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (!bytes) return SDQ_ERR_NULL;
  *bytes = size_t(c.dual ? make_dual_layout(N, K, c.n_o).total : layout_for(c, N, K).total);
  return SDQ_OK;
}

extern "C" sdq_status sdq_logical_bytes(const sdq_config* cfg, int64_t N, int64_t K, size_t* bytes) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (!bytes) return SDQ_ERR_NULL;
  auto lg2 = [](int m) { int b = 0; while ((1 << b) < m) ++b; return b; };
  // bits per row
  int64_t bits = 0;
  if (c.n_o) bits += (K / c.m_o) * c.n_o * (8 + lg2(c.m_o));
  bits += (K / c.m_i) * c.n_i * (4 + lg2(c.m_i));
  if (c.mx) {
    bits += (K / 32) * 8;               // inlier e8m0
    if (c.n_o) bits += (K / 32) * 8;    // outlier e8m0
  } else if (c.dual) {
    bits += (K / 32) * 8;               // inlier e8m0
    if (c.n_o) bits += 32;              // outlier fp32 per row
  } else {
    bits += (K / c.qv) * 8 * c.scale_bytes();  // inlier fp16, or e4m3 / e6m2 ...
    if (c.sc8) bits += 32;                     // ... e4m3 with an fp32 (power of two) per row
    if (c.n_o) bits += 32;                // outlier fp32 per row
  }
  *bytes = size_t((bits * N + 7) / 8);
  return SDQ_OK;
}

extern "C" sdq_status sdq_pack(const sdq_config* cfg, const float* W, int64_t N, int64_t K,
                               const float* act_norm, void* packed, size_t bytes, int n_threads) {
  Cfg c;
  sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (!W || !packed) return SDQ_ERR_NULL;
  const Layout lay = layout_for(c, N, K);
  const DualLayout dlay = make_dual_layout(N, K, c.n_o);
  const size_t total = size_t(c.dual ? dlay.total : lay.total);
  if (bytes < total) return SDQ_ERR_BUFFER_TOO_SMALL;
  if ((s = check_act_norm(c, act_norm, K)) != SDQ_OK) return s;
  std::memset(packed, 0, total);
  RowSink sink{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
               static_cast<uint8_t*>(packed), &lay, &dlay};
  return run_rows(c, W, N, K, act_norm, sink, n_threads);
}

extern "C" sdq_status sdq_pack_logical(const sdq_config* cfg, const float* W, int64_t N, int64_t K,
                                       const float* act_norm, uint8_t* pos_o, uint8_t* code_o,
                                       void* scale_o, uint8_t* pos_i, uint8_t* code_i,
                                       void* scale_i, float* scale_i_row, int n_threads) {
  Cfg c;
  sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (!W || !pos_i || !code_i || !scale_i) return SDQ_ERR_NULL;
  if (c.n_o && (!pos_o || !code_o || !scale_o)) return SDQ_ERR_NULL;
  if ((s = check_act_norm(c, act_norm, K)) != SDQ_OK) return s;
  if (!c.n_o && scale_o) {  // no outlier branch: report zero scales
    if (c.mx) std::memset(scale_o, 0, size_t(N * (K / 32)));
    else std::memset(scale_o, 0, size_t(N) * 4);
  }
  if (scale_i_row && !c.sc8) std::memset(scale_i_row, 0, size_t(N) * 4);
  RowSink sink{pos_o, code_o, scale_o, pos_i, code_i, scale_i, c.sc8 ? scale_i_row : nullptr,
               nullptr, nullptr, nullptr};
  return run_rows(c, W, N, K, act_norm, sink, n_threads);
}

extern "C" sdq_status sdq_unpack_dense(const sdq_config* cfg, const void* packed, size_t bytes,
                                       int64_t N, int64_t K, uint8_t* code_o_dense,
                                       uint8_t* code_i_dense, void* scale_o, void* scale_i,
                                       float* scale_i_row) {
  Cfg c;
  const sdq_status s = check_config(cfg, N, K, &c);
  if (s != SDQ_OK) return s;
  if (!packed || !code_o_dense || !code_i_dense || !scale_o || !scale_i) return SDQ_ERR_NULL;
  const Layout lay = layout_for(c, N, K);
  const uint8_t* blob = static_cast<const uint8_t*>(packed);
  if (c.dual) {
    const DualLayout dl = make_dual_layout(N, K, c.n_o);
    if (bytes < size_t(dl.total)) return SDQ_ERR_BUFFER_TOO_SMALL;
    for (int64_t n = 0; n < N; ++n) {
      const int64_t t = n / kTileN;
      const int r = int(n % kTileN);
      for (int64_t ch = 0; ch < dl.n_chunks; ++ch) {
        const int64_t tc = t * dl.n_chunks + ch;
        const uint8_t* nib = blob + dl.nib_off + tc * kDualNibBytesPerTC;
        const uint16_t* hw = reinterpret_cast<const uint16_t*>(blob + dl.out_off + tc * dl.out_bytes_per_tc);
        const int kend = int(std::min<int64_t>(kChunkK, K - ch * kChunkK));  // a last chunk may be partial
        for (int k = 0; k < kend; ++k) {
          const int64_t kk = n * K + ch * kChunkK + k;
          code_i_dense[kk] = uint8_t((nib[dual_nib_byte(k, r)] >> ((k & 1) * 4)) & 0xFu);
          code_o_dense[kk] = 0;
        }
        for (int pl = 0; pl < dl.out_planes; ++pl)
          for (int g = 0; g < kend / 8; ++g) {
            const uint16_t v = hw[pl * (kDualOutBytesPerTC / 2) + dual_out_halfword(g, r)];
            if (v >> 8) code_o_dense[n * K + ch * kChunkK + g * 8 + (v & 7)] = uint8_t(v >> 8);
          }
        for (int b = 0; b < kend / 32; ++b)
          static_cast<uint8_t*>(scale_i)[n * (K / 32) + ch * 4 + b] =
              blob[dl.scale_off + tc * kDualScaleBytesPerTC + dual_scale_byte(b, r)];
      }
      static_cast<float*>(scale_o)[n] = reinterpret_cast<const float*>(blob + dl.rows_off)[n];
      if (scale_i_row) scale_i_row[n] = 0.f;
    }
    return SDQ_OK;
  }
  if (bytes < size_t(lay.total)) return SDQ_ERR_BUFFER_TOO_SMALL;
  std::memset(code_o_dense, 0, size_t(N * K));
  std::memset(code_i_dense, 0, size_t(N * K));
  for (int64_t n = 0; n < N; ++n) {
    const int64_t t = n / kTileN;
    const int r = int(n % kTileN);
    for (int64_t ch = 0; ch < lay.n_chunks; ++ch) {
      const uint32_t* words = reinterpret_cast<const uint32_t*>(blob + lay.words_off) +
                              (t * lay.n_chunks + ch) * kWordsPerTC;
      const uint8_t* sc = blob + lay.scales_off + (t * lay.n_chunks + ch) * lay.scale_bytes_per_tc;
      const int kend = int(std::min<int64_t>(kChunkK, K - ch * kChunkK));  // a last chunk may be partial
      for (int g = 0; g < kend / 8; ++g) {
        const uint32_t word = words[c.mx ? mx_word_index(g, r) : int_word_index(g, r)];
        const int64_t kbase = n * K + ch * kChunkK + g * 8;
        for (int j = 0; j < 3; ++j) {
          const int p = int((word >> (8 * j)) & 7u);
          const uint8_t nib = uint8_t((word >> (8 * j + 4)) & 0xFu);
          if (!nib) continue;
          code_i_dense[kbase + p] = c.mx ? nib : uint8_t(int8_t(int8_t(nib << 4) >> 4));
        }
        const uint8_t oc = uint8_t(word >> 24);
        if (oc) {
          const int p = int(((word >> 3) & 1u) | ((word >> 10) & 2u) | ((word >> 17) & 4u));
          code_o_dense[kbase + p] = oc;
        }
      }
      if (c.mx) {
        for (int b = 0; b < kend / 32; ++b) {
          const int64_t bi = n * (K / 32) + ch * 4 + b;
          static_cast<uint8_t*>(scale_o)[bi] = sc[mx_scale_byte(b, r, 0)];
          static_cast<uint8_t*>(scale_i)[bi] = sc[mx_scale_byte(b, r, 1)];
        }
      } else {
        const int nb = kChunkK / c.qv;
        for (int kb = 0; kb < kend / c.qv; ++kb) {
          if (c.scale_bytes() == 1) {
            static_cast<uint8_t*>(scale_i)[n * (K / c.qv) + ch * nb + kb] = sc[int_scale_off(kb, r, c.qv, 1)];
          } else {
            uint16_t h;
            std::memcpy(&h, sc + int_scale_off(kb, r, c.qv, 2), 2);
            static_cast<uint16_t*>(scale_i)[n * (K / c.qv) + ch * nb + kb] = h;
          }
        }
      }
    }
    if (!c.mx) {
      const float* rows = reinterpret_cast<const float*>(blob + lay.rows_off);
      static_cast<float*>(scale_o)[n] = rows[n];
      if (scale_i_row) scale_i_row[n] = c.sc8 ? reinterpret_cast<const float*>(blob + lay.irow_off)[n] : 0.f;
    }
  }
  return SDQ_OK;
}
