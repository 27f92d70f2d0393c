// Internal helpers shared by the host-side translation units of libsdq.
#pragma once
#include <cstdint>

#include "layout.h"
#include "sdq.h"

namespace sdq {

struct Cfg {
  bool mx;    // MX family (fp8 outliers and fp4 inliers, e8m0 scales, fp8 activations)
  bool dual;  // dual family (int8 outliers, fp4 inliers, int8 + fp4 activations)
  int n_o, m_o, fmt_o, n_i, m_i, fmt_i, fmt_a, metric, decomp, order;
  bool sc8;     // INT family with two-level e4m3 inlier scales
  bool e6m2;    // INT family with ufp8-e6m2 inlier scales
  int qv;       // dense K per inlier scale (INT 16, 32 or 64; MX and dual 32)
  bool y_bf16;  // the GEMM writes Y as bf16 (nearest even of the fp32 result)
  // INT family: bytes per inlier scale (fp16 2, e4m3 and e6m2 1)
  int scale_bytes() const { return (sc8 || e6m2) ? 1 : 2; }
};

inline Layout layout_for(const Cfg& c, int64_t N, int64_t K) {
  return make_layout(c.mx, N, K, c.sc8, c.qv, c.scale_bytes());
}

// Whether packing this configuration reads act_norm.
inline bool needs_act_norm(const Cfg& c) {
  return c.metric == SDQ_METRIC_PRODUCT || c.decomp == SDQ_DECOMP_PRODUCT ||
         c.decomp == SDQ_DECOMP_OUTPUT_ERROR;
}

// Validates a configuration and shape; fills `out` on success.
inline sdq_status check_config(const sdq_config* c, int64_t N, int64_t K, Cfg* out) {
  if (!c) return SDQ_ERR_NULL;
  if (c->family != SDQ_FAMILY_INT && c->family != SDQ_FAMILY_MX && c->family != SDQ_FAMILY_DUAL)
    return SDQ_ERR_CONFIG;
  const bool mx = c->family == SDQ_FAMILY_MX, dual = c->family == SDQ_FAMILY_DUAL;
  if (c->n_o < 0 || c->n_i < 0 || c->m_o <= 0 || c->m_i <= 0) return SDQ_ERR_CONFIG;
  if (c->n_o > c->m_o || c->n_i > c->m_i || c->n_i == 0) return SDQ_ERR_CONFIG;
  if (c->metric != SDQ_METRIC_MAGNITUDE && c->metric != SDQ_METRIC_PRODUCT) return SDQ_ERR_CONFIG;
  if (c->decomp < SDQ_DECOMP_SAME || c->decomp > SDQ_DECOMP_OUTPUT_ERROR) return SDQ_ERR_CONFIG;
  if (c->order != SDQ_ORDER_LARGE && c->order != SDQ_ORDER_SMALL) return SDQ_ERR_CONFIG;
  // a decomposition other than the default chooses among outliers
  if ((c->decomp != SDQ_DECOMP_SAME || c->order != SDQ_ORDER_LARGE) && c->n_o == 0) return SDQ_ERR_CONFIG;
  if (c->sfmt_i != SDQ_SCALE_DEFAULT && c->sfmt_i != SDQ_SCALE_E4M3 && c->sfmt_i != SDQ_SCALE_UE6M2)
    return SDQ_ERR_CONFIG;
  if (c->sfmt_i != SDQ_SCALE_DEFAULT && c->family != SDQ_FAMILY_INT) return SDQ_ERR_CONFIG;
  if (c->family == SDQ_FAMILY_INT) {
    if (c->qv_i != 0 && c->qv_i != 16 && c->qv_i != 32 && c->qv_i != 64) return SDQ_ERR_CONFIG;
  } else if (c->qv_i != 0 && c->qv_i != 32) {
    return SDQ_ERR_CONFIG;
  }
  if (c->y_dtype != SDQ_DTYPE_F32 && c->y_dtype != SDQ_DTYPE_BF16) return SDQ_ERR_CONFIG;
  if (mx) {
    if (c->fmt_o != SDQ_FMT_E4M3 || c->fmt_i != SDQ_FMT_E2M1 || c->fmt_a != SDQ_FMT_E4M3)
      return SDQ_ERR_CONFIG;
  } else if (dual) {
    if (c->fmt_o != SDQ_FMT_INT8 || c->fmt_i != SDQ_FMT_E2M1 || c->fmt_a != SDQ_FMT_INT8)
      return SDQ_ERR_CONFIG;
  } else {
    if ((c->fmt_o != SDQ_FMT_E4M3 && c->fmt_o != SDQ_FMT_INT8) || c->fmt_i != SDQ_FMT_INT4 ||
        c->fmt_a != SDQ_FMT_INT8)
      return SDQ_ERR_CONFIG;
  }
  // What the kernels implement.
  if (c->m_i != 8) return SDQ_ERR_UNSUPPORTED;
  if (dual) {
    // dense fp4 inliers: any n_i with n_o + n_i <= 8; 1:8 or 2:8 outliers
    if (c->n_o > 2 || (c->n_o > 0 && c->m_o != 8) || c->n_o + c->n_i > 8) return SDQ_ERR_UNSUPPORTED;
  } else {
    if (c->n_i > 3) return SDQ_ERR_UNSUPPORTED;
    if (c->n_o > 1 || (c->n_o == 1 && c->m_o != 8 && c->m_o != 16)) return SDQ_ERR_UNSUPPORTED;
  }
  // upper bounds keep every per-block offset of the kernels in 32 bits
  // K: whole 32-K blocks (the e8m0 block of the MX and dual families, two
  // 16-K inlier blocks of the INT family) and whole Q-Vectors
  const int qv_eff = c->qv_i ? c->qv_i : 16;
  if (N <= 0 || K <= 0 || K % 32 != 0 || K % qv_eff != 0 || N > (int64_t(1) << 21) ||
      K > (int64_t(1) << 22))
    return SDQ_ERR_SHAPE;
  if (N > (int64_t(1) << 31) || K > (int64_t(1) << 24)) return SDQ_ERR_SHAPE;
  // int8 outliers against int8 activations accumulate in int32: K n_o / m_o
  // products of at most 127^2 each stay below 2^31 for K <= 2^19 (n_o / m_o
  // <= 1/4)
  if (c->fmt_o == SDQ_FMT_INT8 && c->n_o > 0 && K > (int64_t(1) << 19)) return SDQ_ERR_SHAPE;
  if (out) {
    out->mx = mx;
    out->dual = dual;
    out->n_o = c->n_o;
    out->m_o = c->n_o ? c->m_o : 8;
    out->fmt_o = c->fmt_o;
    out->n_i = c->n_i;
    out->m_i = c->m_i;
    out->fmt_i = c->fmt_i;
    out->fmt_a = c->fmt_a;
    out->metric = c->metric;
    out->decomp = c->decomp;
    out->order = c->order;
    out->sc8 = c->sfmt_i == SDQ_SCALE_E4M3;
    out->e6m2 = c->sfmt_i == SDQ_SCALE_UE6M2;
    out->qv = c->qv_i ? c->qv_i : (c->family == SDQ_FAMILY_INT ? 16 : 32);
    out->y_bf16 = c->y_dtype == SDQ_DTYPE_BF16;
  }
  return SDQ_OK;
}

}  // namespace sdq
