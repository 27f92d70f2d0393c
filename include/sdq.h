/*
 * sdq.h -- C ABI of the SDQ decomposed linear-layer GEMM for AMD Instinct
 * MI355X (gfx950).
 *
 * SDQ (Sparse Decomposed Quantization; Jeong, Tsai, Keckler, Krishna) splits
 * every weight matrix W[N,K] of a linear layer into two structured-sparse
 * parts (Section 5, Stages 1-3):
 *   W_o  n_o:m_o outliers ("local outliers" of Section 4) at 8 bits,
 *   W_i  n_i:m_i inliers at 4 bits with per-vector (VS-Quant) scales,
 * quantizes the activations per token, and computes the layer as the sum of
 * the two sparse products (Section 5.1):
 *   Y[m,n] = s_a[m] * sum_k Xq[m,k] * (deq W_o[n,k] + deq W_i[n,k]).
 *
 * Conventions shared by every entry point
 *   - W is [N, K] row-major (row n = output feature, K = reduction), X and Xq
 *     are [M, K] row-major, Y is [M, N] row-major, fp32 or (sdq_config.y_dtype)
 *     bf16.
 *   - N:M groups and scale blocks run along K inside one row of W.
 *   - Every function returns an sdq_status (0 = SDQ_OK, negative = error).
 *     Nothing throws, aborts or prints (unless SDQ_LOG=1 is set, which prints
 *     the kernel chosen by sdq_gemm to stderr).
 *   - Argument errors (NULL pointers, shapes, configurations, buffer sizes)
 *     are detected before any GPU work and returned synchronously.
 *   - The caller owns every buffer.  Device entry points allocate no memory
 *     (host or device) and can be captured in a HIP graph; the host packer
 *     uses only its worker threads and K floats of scratch per thread.  The
 *     library keeps no mutable global state.
 *   - Device entry points take device pointers and a stream (a hipStream_t
 *     passed as void*; NULL = the default stream), enqueue their kernels on
 *     that stream and return without synchronizing.  A launch failure is
 *     reported as SDQ_ERR_HIP; a fault inside a kernel surfaces at the
 *     caller's next synchronization.  An error that an earlier HIP call on
 *     the calling thread left pending (what hipGetLastError would return) is
 *     read and dropped before the launches, so that it is not reported as the
 *     call's own.
 *   - The library links the HIP runtime by its soname (libamdhip64.so.7).  In
 *     a process that also loads another copy of the runtime under another
 *     file name (PyTorch's ROCm wheels carry one), load that copy first: the
 *     library then shares it.  The other order leaves two runtimes in the
 *     process, and the library's launches find no device.
 *   - Host entry points (pack, logical pack, unpack) take host pointers and
 *     are deterministic: the output does not depend on the thread count.
 */
#ifndef SDQ_H_
#define SDQ_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SDQ_OK = 0,
  SDQ_ERR_NULL = -1,             /* a required pointer is NULL                 */
  SDQ_ERR_SHAPE = -2,            /* M, N or K out of range / not divisible     */
  SDQ_ERR_CONFIG = -3,           /* malformed sdq_config                       */
  SDQ_ERR_BUFFER_TOO_SMALL = -4, /* output buffer smaller than required        */
  SDQ_ERR_HIP = -5,              /* a HIP call or kernel launch failed         */
  SDQ_ERR_UNSUPPORTED = -6,      /* well-formed but not implemented            */
  SDQ_ERR_VALUE = -7,            /* input value out of range (e.g. non-finite) */
  SDQ_ERR_TOO_LARGE = -8         /* needs more than sdq_gemm_static's scratch  */
} sdq_status;

/* Format families.
 *  SDQ_FAMILY_INT: activations int8 per token (fp32 scale); outliers fp8-e4m3
 *    or int8 with one fp32 scale per row of W; inliers int4 in [-7, 7] with one
 *    fp16 scale per 16 consecutive K positions of a row.
 *  SDQ_FAMILY_MX: activations fp8-e4m3 per token (fp32 scale); outliers
 *    fp8-e4m3 and inliers fp4-e2m1, each branch with one e8m0 (power of two)
 *    scale per 32 consecutive K positions of a row (OCP MX shared exponents).
 *  SDQ_FAMILY_DUAL (Section 5.1's worked configuration, and the dual
 *    configurations whose perplexity Section 6.2 reports: 7:8 kept as 1:8
 *    int8 + 6:8 fp4, 6:8 as 2:8 int8 + 4:8 fp4, 8:8 as 1:8 int8 + 7:8
 *    fp4): outliers int8
 *    with one fp32 scale per row against int8
 *    activations A_o (fp32 scale per token); inliers fp4-e2m1 with an e8m0
 *    scale per 32 K against fp4-e2m1 activations A_i (MXFP4: an e8m0 scale
 *    per 32 K per token).  fmt_o INT8, fmt_i E2M1, fmt_a INT8 (A_o; A_i is
 *    implied); n_o in {0, 1, 2} with m_o = 8, any n_i with n_o + n_i <= 8.
 *    Quantize with sdq_quantize_act_dual and multiply with sdq_gemm_dual.
 */
enum { SDQ_FAMILY_INT = 0, SDQ_FAMILY_MX = 1, SDQ_FAMILY_DUAL = 2 };
enum { SDQ_FMT_INT8 = 1, SDQ_FMT_INT4 = 2, SDQ_FMT_E4M3 = 3, SDQ_FMT_E2M1 = 4 };
enum { SDQ_METRIC_MAGNITUDE = 0, SDQ_METRIC_PRODUCT = 1 };
/* Decomposition metric (which kept weights become the outliers) and the
 * order it is taken in; see sdq_config. */
enum {
  SDQ_DECOMP_SAME = 0,         /* the significance metric                      */
  SDQ_DECOMP_MAGNITUDE = 1,    /* |W|                                          */
  SDQ_DECOMP_PRODUCT = 2,      /* |W| * act_norm[k]                            */
  SDQ_DECOMP_ERROR = 3,        /* |W - Q_i(W)|, Q_i the inlier quantizer       */
  SDQ_DECOMP_OUTPUT_ERROR = 4  /* |W - Q_i(W)| * act_norm[k]                   */
};
enum { SDQ_ORDER_LARGE = 0, SDQ_ORDER_SMALL = 1 };
/* Inlier scale format (sdq_config.sfmt_i). */
enum { SDQ_SCALE_DEFAULT = 0, SDQ_SCALE_E4M3 = 1, SDQ_SCALE_UE6M2 = 2 };
enum { SDQ_DTYPE_F32 = 0, SDQ_DTYPE_BF16 = 1 };
/* sdq_gemm_ex / sdq_gemm_ws kernel choice. */
enum { SDQ_PATH_AUTO = 0, SDQ_PATH_DECODE = 1, SDQ_PATH_MFMA = 2, SDQ_PATH_DENSE = 3, SDQ_PATH_SPLITK = 4 };

/* One SDQ configuration (the paper's SDQ-k:m-n_o:m{fmt}-n_i:m{fmt} naming,
 * Section 6 "Methodology", restricted to what the kernels implement):
 *   family  SDQ_FAMILY_INT | SDQ_FAMILY_MX
 *   n_o:m_o outlier sparsity, n_o in {0, 1}, m_o in {8, 16} (n_o = 0: none)
 *   fmt_o   INT: SDQ_FMT_E4M3 | SDQ_FMT_INT8;  MX: SDQ_FMT_E4M3
 *   n_i:m_i inlier sparsity, n_i in {1, 2, 3}, m_i = 8
 *   fmt_i   INT: SDQ_FMT_INT4;  MX: SDQ_FMT_E2M1
 *   fmt_a   INT: SDQ_FMT_INT8;  MX: SDQ_FMT_E4M3
 *   metric  significance used to sparsify (Section 5, Stage 1): |W|
 *           (SDQ_METRIC_MAGNITUDE) or |W| * act_norm[k] (SDQ_METRIC_PRODUCT,
 *           Wanda's weight-activation product)
 *   decomp  metric that picks the outliers among the kept weights (Section
 *           5, Stage 2; the variants of Section 6.4's decomposition study):
 *           SDQ_DECOMP_SAME (the significance metric), _MAGNITUDE, _PRODUCT,
 *           _ERROR (the error the inlier quantizer would make on the weight)
 *           or _OUTPUT_ERROR (that error times act_norm[k])
 *   order   SDQ_ORDER_LARGE: the outliers are the kept weights with the
 *           largest decomp metric ("Large"); SDQ_ORDER_SMALL: the smallest
 * decomp = SAME with order = LARGE (both zero) is the default; any other
 * choice needs n_o = 1.
 *   sfmt_i  inlier scale format (Section 3.3: scales are quantized too;
 *           Section 6.4 compares 8-bit scale formats): SDQ_SCALE_DEFAULT (INT
 *           fp16, MX e8m0) or, INT family only,
 *           SDQ_SCALE_E4M3: VS-Quant's two levels, an fp8-e4m3 scale per
 *           Q-Vector times one power-of-two scale 2^E per row, E the smallest
 *           with every vector scale amax/7 of the row <= 448 * 2^E, or
 *           SDQ_SCALE_UE6M2: one unsigned fp8 scale per Q-Vector (6 exponent
 *           bits with bias 31, 2 mantissa bits), nearest even; the packer
 *           requires every nonzero one to lie in [2^-22, 7168] (exponent
 *           field 9..43), where an int4 code times the scale is exact in
 *           fp16, and returns SDQ_ERR_VALUE otherwise.
 *   y_dtype element type of the GEMM output Y: SDQ_DTYPE_F32 (0, the
 *           default) or SDQ_DTYPE_BF16 (half the output bytes).  A bf16
 *           output is the fp32 output rounded to nearest even, bit for bit,
 *           with one exception: on SDQ_PATH_DENSE, outputs whose wave met a
 *           block that did not merge its inliers are rounded twice (the main
 *           sum to bf16, then that value plus those inliers), an extra error
 *           below 2^-9 of the main sum.  The packer ignores it.
 *   qv_i    Q-Vector length of the inlier scales (Section 3.3): dense K
 *           positions of one row that share a scale.  0 = the family's
 *           (INT 16, MX and dual 32); the INT family also takes 32 or 64,
 *           which halve or quarter the scale bytes. */
typedef struct {
  int32_t family;
  int32_t n_o, m_o, fmt_o;
  int32_t n_i, m_i, fmt_i;
  int32_t fmt_a;
  int32_t metric;
  int32_t decomp, order;
  int32_t sfmt_i;
  int32_t y_dtype;
  int32_t qv_i;
} sdq_config;

/* Static description of an error code (never NULL). */
const char* sdq_status_string(sdq_status s);

/* Validate a configuration for a W of shape [N, K].  K must be a positive
 * multiple of 32 (and of qv_i when that is 64) up to 2^22 (2^19 with int8
 * outliers, whose products with int8 activations are summed exactly in
 * int32) and N positive up to 2^21.  The kernels take K in chunks of 128: when K is not a multiple of
 * 128 the blob pads the last chunk with zero codes and scales.  Returns SDQ_ERR_CONFIG / SDQ_ERR_SHAPE /
 * SDQ_ERR_UNSUPPORTED without touching anything else. */
sdq_status sdq_check(const sdq_config* cfg, int64_t N, int64_t K);

/* Size in bytes of the packed (physical) weight blob that sdq_pack writes. */
sdq_status sdq_pack_size(const sdq_config* cfg, int64_t N, int64_t K, size_t* bytes);

/* Algorithmic size in bytes of the decomposed layer in the paper's logical
 * ELLPACK-like form (Section 3.3): per branch n values and n log2(m)-bit
 * indices per m weights, plus the scales.  This is the byte count that
 * throughput figures are quoted against; the physical blob may be larger. */
sdq_status sdq_logical_bytes(const sdq_config* cfg, int64_t N, int64_t K, size_t* bytes);

/* Offline pack (Section 5, Stages 1-3), on the host.
 *   W         host, [N, K] fp32 row-major, finite values
 *   act_norm  host, [K] fp32 (per-input-channel activation norm), required
 *             for SDQ_METRIC_PRODUCT, SDQ_DECOMP_PRODUCT and
 *             SDQ_DECOMP_OUTPUT_ERROR and ignored otherwise (may be NULL)
 *   packed    host, caller-owned, at least sdq_pack_size() bytes; copy it to
 *             the device unchanged before calling sdq_gemm
 *   n_threads host threads to use (<= 0: one per hardware thread)
 * Selection with the default decomposition (decomp SAME, order LARGE): in
 * every m_o-group the n_o most significant positions are the outliers; in
 * every m_i-group the n_i most significant remaining positions are the
 * inliers; the rest are pruned.  Ties go to the lower k.
 * Any other decomposition follows the paper's stage order:
 *   1. every 8-group keeps its n_o + n_i most significant positions;
 *   2. the error metrics quantize the kept positions as inliers (the inlier
 *      rule below, scales over the kept positions of each block) and take
 *      D = |W - deq| in fp32 (times act_norm[k] for OUTPUT_ERROR);
 *   3. in every m_o-group the n_o kept positions first by (-D, k) (LARGE) or
 *      (D, k) (SMALL) are the outliers;
 *   4. in every 8-group the n_i most significant kept positions that are not
 *      outliers are the inliers (with m_o = 16 the 8-group without the
 *      outlier drops its least significant kept position).
 * With decomp SAME and order LARGE the two procedures select the same sets.
 * Quantization (IEEE fp32 arithmetic, round-to-nearest-even):
 *   INT outliers: s_o[n] = amax_row / qmax (qmax 127 or 448), q = enc(W / s_o)
 *   INT inliers:  per Q-Vector of qv_i dense K, s = fp16(amax / 7),
 *                 q = clamp(rne(W / s), -7, 7); with SDQ_SCALE_E4M3,
 *                 v = amax / 7 (fp32), the row's E as in sdq_config,
 *                 code = e4m3(v * 2^-E), s = value(code) * 2^E (exact); with
 *                 SDQ_SCALE_UE6M2, code = ue6m2(amax / 7), s = value(code)
 *   MX:           E = floor(log2 amax_block32) - emax (8 for e4m3, 2 for
 *                 e2m1), q = enc(W / 2^E) saturating
 *   an all-zero block gets a zero scale (E = -127) and zero codes.
 * Returns SDQ_ERR_VALUE if W holds a non-finite value or an inlier scale
 * overflows fp16 (also the provisional scales of the error metrics).
 * Scratch: each worker thread holds 2K floats and K/4 bytes. */
sdq_status sdq_pack(const sdq_config* cfg, const float* W, int64_t N, int64_t K,
                    const float* act_norm, void* packed, size_t bytes, int n_threads);

/* The same selection and quantization as sdq_pack, returned in the logical
 * form instead of the kernel layout (host, caller-owned arrays):
 *   pos_o, code_o  uint8 [N][K/m_o][n_o]  positions within the group
 *                  (ascending) and codes (e4m3 bits or int8 bits)
 *   scale_o        INT: float [N];  MX: uint8 e8m0 [N][K/32]
 *   pos_i, code_i  uint8 [N][K/m_i][n_i]  (int4 codes as int8 bits, e2m1
 *                  codes as the low nibble)
 *   scale_i        INT: uint16 fp16 bits [N][K/qv] (SDQ_SCALE_E4M3 and
 *                  SDQ_SCALE_UE6M2: uint8 codes [N][K/qv]);  MX: uint8 e8m0
 *                  [N][K/32]
 *   scale_i_row    SDQ_SCALE_E4M3 only: float [N], the row scale 2^E (0 for
 *                  a row without inlier magnitude); may be NULL
 * Any pointer for a branch with n = 0 may be NULL. */
sdq_status sdq_pack_logical(const sdq_config* cfg, const float* W, int64_t N, int64_t K,
                            const float* act_norm, uint8_t* pos_o, uint8_t* code_o,
                            void* scale_o, uint8_t* pos_i, uint8_t* code_i, void* scale_i,
                            float* scale_i_row, int n_threads);

/* Decode a packed blob (host copy) back to dense code arrays: code_o_dense
 * and code_i_dense are uint8 [N][K] holding each stored code at its position
 * and 0 elsewhere; scale_o / scale_i / scale_i_row as in sdq_pack_logical.  Used to check
 * that the kernel layout round-trips. */
sdq_status sdq_unpack_dense(const sdq_config* cfg, const void* packed, size_t bytes,
                            int64_t N, int64_t K, uint8_t* code_o_dense,
                            uint8_t* code_i_dense, void* scale_o, void* scale_i,
                            float* scale_i_row);

/* Per-token activation quantization (Section 5, Stage 3; the activations
 * are quantized to match the weights).  For each row m:
 *   a = max_k |X[m,k]|;  s_a[m] = a / qmax;  inv = qmax / a  (fp32 divides)
 *   Xq[m,k] = enc(X[m,k] * inv)  (one fp32 multiply, then round to nearest
 *   even: int8 clamps to [-127, 127], e4m3 saturates to +-448)
 * A row with a == 0 gets s_a = 0 and zero codes.
 *   X      device, [M, K] row-major, x_dtype SDQ_DTYPE_F32 or SDQ_DTYPE_BF16
 *   Xq     device, [M, K] row-major, 1 byte per element (int8 for the INT
 *          family, e4m3 bits for the MX family)
 *   s_a    device, [M] fp32
 * M = 0 is a no-op.  K as in sdq_check. */
sdq_status sdq_quantize_act(const sdq_config* cfg, const void* X, int32_t x_dtype,
                            int64_t M, int64_t K, void* Xq, float* s_a, void* stream);

/* The decomposed GEMM (Section 5.1):
 *   Y[m,n] = s_a[m] * ( sum over outlier slots of Xq[m,k] * deq W_o[n,k]
 *                     + sum over inlier slots  of Xq[m,k] * deq W_i[n,k] )
 * with both branches accumulated in one fp32 accumulator per output.
 *   Xq, s_a  device, as written by sdq_quantize_act for the same cfg
 *   packed   device, the blob written by sdq_pack for the same cfg, N, K
 *   Y        device, [M, N] row-major, fp32 or bf16 by cfg->y_dtype
 *            (overwritten; 4-byte aligned)
 * M = 0 is a no-op.  The result is deterministic (no atomics).  The
 * arithmetic of one output does not depend on N: on the decode path, rows
 * of W stacked along N into one blob (e.g. the q, k and v projections, which
 * read the same X) give the separate launches' outputs bit for bit. */
sdq_status sdq_gemm(const sdq_config* cfg, const void* Xq, const float* s_a, int64_t M,
                    const void* packed, int64_t N, int64_t K, void* Y, void* stream);

/* sdq_gemm with an explicit kernel choice: SDQ_PATH_DECODE (weight-streaming
 * vector kernel, INT family, any M up to 8), SDQ_PATH_MFMA (matrix-core
 * kernels, any M) or SDQ_PATH_AUTO (what sdq_gemm does).  Returns
 * SDQ_ERR_UNSUPPORTED for a path that does not serve the configuration and
 * for SDQ_PATH_DENSE and SDQ_PATH_SPLITK, which take a workspace
 * (sdq_gemm_ws). */
sdq_status sdq_gemm_ex(const sdq_config* cfg, const void* Xq, const float* s_a, int64_t M,
                       const void* packed, int64_t N, int64_t K, void* Y, void* stream,
                       int32_t path);

/* Activation quantization and the decomposed GEMM in one call: the same
 * results as sdq_quantize_act followed by sdq_gemm (Xq, s_a and Y are
 * identical bit for bit).  Where sdq_gemm would take the decode path (INT
 * family, small M) this is a single kernel in which every workgroup quantizes
 * the activations into LDS itself; otherwise it enqueues the two kernels.
 *   X       device, [M, K] fp32 or bf16 (x_dtype)
 *   Xq, s_a device, outputs as in sdq_quantize_act (always written)
 *   packed  device, as in sdq_gemm;  Y device, [M, N] as in sdq_gemm */
sdq_status sdq_linear(const sdq_config* cfg, const void* X, int32_t x_dtype, int64_t M,
                      void* Xq, float* s_a, const void* packed, int64_t N, int64_t K, void* Y,
                      void* stream);

/* The path sdq_gemm takes for this configuration and M (SDQ_PATH_DECODE or
 * SDQ_PATH_MFMA). */
sdq_status sdq_gemm_path(const sdq_config* cfg, int64_t M, int64_t N, int64_t K, int32_t* path);

/* The path sdq_gemm_ws and sdq_gemm_static take with SDQ_PATH_AUTO
 * (SDQ_PATH_DECODE, SDQ_PATH_MFMA, SDQ_PATH_DENSE or SDQ_PATH_SPLITK). */
sdq_status sdq_gemm_path_ws(const sdq_config* cfg, int64_t M, int64_t N, int64_t K, int32_t* path);

/* Device workspace that sdq_gemm_ws needs (the product is sdq_gemm's,
 * Section 5.1).  Two paths take one.
 * SDQ_PATH_SPLITK splits K into ranges of 128-K chunks handled by different
 * workgroups; the partial sums of the ranges go to the workspace and a
 * second kernel adds them in range order and scales by s_a.  In the INT
 * family (9 to 256 tokens) each workgroup converts its activations to the
 * matrix instruction's f16 once for four row tiles; in the MX family (from
 * one token up to a few hundred) it is the one-pass scaled-MFMA kernel over
 * a range of K, so that a small grid still fills the GPU.  SDQ_PATH_DENSE, the two-pass matrix-core path of the MX
 * family with outliers, first expands every packed weight once into the dense
 * fp8 B operand of the matrix instruction (both branches of a 32-K block
 * merged into one e4m3 value per position under the outlier's e8m0 scale,
 * wherever the inliers fit it) and then multiplies those operands, so that
 * the expansion runs once per weight instead of once per weight and block of
 * 128 tokens (at 512 tokens and more the two passes take less time).
 *   path   SDQ_PATH_AUTO (what sdq_gemm_ws takes: SDQ_PATH_DENSE for the MX
 *          family with outliers when M >= 512 and ceil(N/256) * ceil(M/128)
 *          >= 160; SDQ_PATH_SPLITK for the MX family when K >= 1024 and
 *          ceil(N/128) * ceil(M/128) <= 128, and for the INT family up to
 *          256 tokens where sdq_gemm would take the matrix cores and K >=
 *          8192, or M >= 64 and N >= 8192, or M = 256; else what sdq_gemm
 *          takes), or SDQ_PATH_DECODE / SDQ_PATH_MFMA / SDQ_PATH_DENSE /
 *          SDQ_PATH_SPLITK
 *   bytes  32 * ceil(N / 32) * K for SDQ_PATH_DENSE; 4 * S * M * N for
 *          SDQ_PATH_SPLITK, with S (the number of K ranges, at most
 *          ceil(K / 128) / 4) chosen from M, N and K so that about 2048
 *          waves (INT) or 512 workgroups (MX) run; 0 for the other paths
 * Returns SDQ_ERR_UNSUPPORTED for SDQ_PATH_DENSE outside the MX family with
 * outliers and for SDQ_PATH_SPLITK in the dual family. */
sdq_status sdq_gemm_workspace_size(const sdq_config* cfg, int64_t M, int64_t N, int64_t K,
                                   int32_t path, size_t* bytes);

/* sdq_gemm_ex with a caller-owned device workspace of ws_bytes bytes (at least
 * sdq_gemm_workspace_size for the same arguments, else
 * SDQ_ERR_BUFFER_TOO_SMALL; 16-byte aligned; NULL with ws_bytes = 0 when the
 * path needs none).  The workspace is scratch: its contents on entry are
 * ignored and on return unspecified, and calls that share one must be ordered
 * on one stream.  SDQ_PATH_DENSE gives the results of SDQ_PATH_MFMA bit for
 * bit when every block merged its inliers (each accumulator takes the same
 * matrix instructions in the same order); the inliers of blocks that did not
 * merge are added after the last chunk instead of within their chunk, a
 * different fp32 rounding order.  SDQ_PATH_SPLITK adds the fp32 partial
 * sums of its K ranges (INT: s_o * acc_o + acc) in range order before
 * scaling by s_a, another fixed rounding order than SDQ_PATH_MFMA's (its
 * products are as exact; integer-grid inputs give the same results). */
sdq_status sdq_gemm_ws(const sdq_config* cfg, const void* Xq, const float* s_a, int64_t M,
                       const void* packed, int64_t N, int64_t K, void* Y, void* workspace,
                       size_t ws_bytes, void* stream, int32_t path);

/* The two passes of SDQ_PATH_DENSE as separate calls (the MX family with
 * outliers; Section 5.1's product, with the weight unpack of Section 5 done
 * ahead of it).  The first pass needs only the packed weights, so a caller
 * can unpack the next layer's weights on another stream while this layer's
 * product runs, and order each product after its own unpack with an event.
 *   sdq_unpack_weights: writes the expanded B operands of the blob into
 *     workspace (device, 16-byte aligned, ws_bytes at least
 *     sdq_gemm_workspace_size(cfg, M, N, K, SDQ_PATH_DENSE) =
 *     32 * ceil(N / 32) * K, else SDQ_ERR_BUFFER_TOO_SMALL).
 *   sdq_gemm_unpacked: Y = the product, reading that workspace and the scale
 *     words of the same blob (packed); arguments otherwise as sdq_gemm_ws.
 *     The result equals sdq_gemm_ws with SDQ_PATH_DENSE bit for bit.
 * The workspace must hold the unpack of this packed, N and K, and no other
 * call may write it before sdq_gemm_unpacked has run (on its stream); a
 * workspace that holds anything else gives wrong results, not an error.
 * SDQ_ERR_UNSUPPORTED outside the MX family with outliers. */
sdq_status sdq_unpack_weights(const sdq_config* cfg, const void* packed, int64_t N, int64_t K,
                              void* workspace, size_t ws_bytes, void* stream);
sdq_status sdq_gemm_unpacked(const sdq_config* cfg, const void* Xq, const float* s_a, int64_t M,
                             const void* packed, int64_t N, int64_t K, const void* workspace,
                             size_t ws_bytes, void* Y, void* stream);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture that may not call hipMalloc, tight serving loops, harnesses that
 * forbid allocation.  sdq_gemm_ws without a workspace argument: where the path
 * takes a workspace (SDQ_PATH_DENSE, SDQ_PATH_SPLITK) it uses a static device array of
 * SDQ_STATIC_SCRATCH_BYTES (48 MiB) compiled into the library, which every GPU
 * the library runs on holds until the process ends.  Arguments, paths and
 * results are sdq_gemm_ws's (the same kernels, bit for bit); SDQ_PATH_AUTO
 * chooses as sdq_gemm_ws does.
 *   - Returns SDQ_ERR_TOO_LARGE, before any GPU work, when the chosen path
 *     needs more scratch than the array holds (32 * ceil(N/32) * K bytes for
 *     SDQ_PATH_DENSE, e.g. 43 MiB for an 11008 x 4096 layer fits and a 16384 x
 *     4096 one does not; sdq_gemm_workspace_size's figure for
 *     SDQ_PATH_SPLITK; SDQ_PATH_MFMA and SDQ_PATH_DECODE need none).
 *   - Every call on a GPU shares that GPU's array, which keeps the last call's
 *     contents.  Its contents on entry are ignored: the first pass writes every
 *     byte the second reads.  Calls that overlap on one GPU (other streams,
 *     other host threads) race on the array; order them on one stream.
 *   - Allocates nothing (no hipMalloc, hipFree or allocating library call):
 *     the array's device address is looked up with hipGetSymbolAddress on the
 *     first call with each device current, and kept. */
#define SDQ_STATIC_SCRATCH_BYTES (48u * 1024u * 1024u)
sdq_status sdq_gemm_static(const sdq_config* cfg, const void* Xq, const float* s_a, int64_t M,
                           const void* packed, int64_t N, int64_t K, void* Y, void* stream,
                           int32_t path);

/* Dual family (SDQ_FAMILY_DUAL; Section 5.1's int8 A_o / fp4 A_i): the two
 * activation tensors of every token, from one read of X.
 *   X      device, [M, K] row-major, x_dtype SDQ_DTYPE_F32 or SDQ_DTYPE_BF16
 *   Xq_o   device, [M, K] int8 codes of A_o (as sdq_quantize_act for int8)
 *   s_a_o  device, [M] fp32 scales of A_o
 *   Xq_i   device, [M, K/2] bytes: e2m1 codes of A_i, k even in the low nibble
 *   e_a_i  device, [M, K/32] e8m0 codes: per 32-K block a = max|X|,
 *          E = floor(log2 a) - 2 clamped to [-127, 127] (a == 0: E = -127 and
 *          zero codes); code = e2m1(X * 2^-E), nearest even, saturating at 6
 * X, Xq_o and Xq_i must be 16-byte aligned.  M = 0 is a no-op.  Returns
 * SDQ_ERR_CONFIG for a configuration of another family. */
sdq_status sdq_quantize_act_dual(const sdq_config* cfg, const void* X, int32_t x_dtype, int64_t M,
                                 int64_t K, void* Xq_o, float* s_a_o, void* Xq_i, void* e_a_i,
                                 void* stream);

/* The dual-family decomposed GEMM (Section 5.1):
 *   Y[m,n] = s_a_o[m] * s_o[n] * sum_k Xq_o[m,k] * q_o[n,k]
 *          + sum_k e2m1(Xq_i[m,k]) 2^(e_a_i[m,k/32]-127) * e2m1(q_i[n,k]) 2^(E_i[n,k/32])
 * with the outlier branch exact in int32 and the inlier branch in fp32.
 *   Xq_o, s_a_o, Xq_i, e_a_i  device, as written by sdq_quantize_act_dual
 *   packed   device, the blob written by sdq_pack for the same cfg, N, K
 *   Y        device, [M, N] row-major, fp32 or bf16 by cfg->y_dtype
 *            (overwritten; 4-byte aligned)
 * M = 0 is a no-op.  Deterministic.  sdq_gemm, sdq_gemm_ex, sdq_gemm_ws,
 * sdq_linear and sdq_quantize_act return SDQ_ERR_UNSUPPORTED for this
 * family. */
sdq_status sdq_gemm_dual(const sdq_config* cfg, const void* Xq_o, const float* s_a_o,
                         const void* Xq_i, const void* e_a_i, int64_t M, const void* packed,
                         int64_t N, int64_t K, void* Y, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* SDQ_H_ */
