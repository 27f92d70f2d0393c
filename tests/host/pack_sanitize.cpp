// The host packer built with AddressSanitizer and UndefinedBehaviorSanitizer
// (by tests/test_pack_sanitizers.py, with g++, no GPU code).  It runs every
// host entry point (size queries, sdq_pack, sdq_pack_logical,
// sdq_unpack_dense) over every configuration family on ragged shapes, with
// one and several threads, including all-zero rows, ties, the error paths
// (NaN, too small a buffer, NULL pointers) and tight, exactly sized output
// buffers, so that any read or write outside a buffer or any undefined
// operation aborts the run.  It also checks that the output does not depend on
// the thread count and that unpacking reproduces the logical codes.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <random>
#include <vector>

#include "sdq.h"

namespace {

int failures = 0;

void expect(bool ok, const char* what, const sdq_config& c, long N, long K) {
  if (!ok) {
    std::printf("FAIL %s: family %d n_o %d m_o %d fmt_o %d n_i %d sfmt %d decomp %d N %ld K %ld\n", what,
                c.family, c.n_o, c.m_o, c.fmt_o, c.n_i, c.sfmt_i, c.decomp, N, K);
    ++failures;
  }
}

sdq_config cfg(int family, int n_o, int m_o, int fmt_o, int n_i, int metric = SDQ_METRIC_MAGNITUDE,
               int decomp = SDQ_DECOMP_SAME, int order = SDQ_ORDER_LARGE, int sfmt = SDQ_SCALE_DEFAULT) {
  sdq_config c{};
  c.family = family;
  c.n_o = n_o;
  c.m_o = m_o;
  c.fmt_o = fmt_o;
  c.n_i = n_i;
  c.m_i = 8;
  c.fmt_i = family == SDQ_FAMILY_INT ? SDQ_FMT_INT4 : SDQ_FMT_E2M1;
  c.fmt_a = family == SDQ_FAMILY_MX ? SDQ_FMT_E4M3 : SDQ_FMT_INT8;
  c.metric = metric;
  c.decomp = decomp;
  c.order = order;
  c.sfmt_i = sfmt;
  c.y_dtype = SDQ_DTYPE_F32;
  return c;
}

// A heap buffer of exactly n bytes (n = 0 still gets a distinct pointer), so
// that ASan sees a write one past its end.
struct Buf {
  std::unique_ptr<uint8_t[]> p;
  size_t n;
  explicit Buf(size_t bytes) : p(new uint8_t[bytes ? bytes : 1]), n(bytes) { std::memset(p.get(), 0xA5, n ? n : 1); }
  uint8_t* get() { return p.get(); }
};

void run(const sdq_config& c, long N, long K, std::mt19937& rng) {
  std::normal_distribution<float> nd(0.f, 0.02f);
  std::vector<float> W(size_t(N) * K), an(K);
  for (auto& w : W) w = nd(rng);
  for (long k = 0; k < K; ++k) an[k] = 0.5f + float(k % 7);
  if (N > 2) std::fill(W.begin() + K, W.begin() + 2 * K, 0.f);  // an all-zero row
  if (N > 3)
    for (long k = 0; k < K; ++k) W[3 * K + k] = (k % 3) ? 0.01f : -0.01f;  // ties
  W[0] = 0.5f;                                                           // an outlier
  size_t bytes = 0, lbytes = 0;
  expect(sdq_pack_size(&c, N, K, &bytes) == SDQ_OK && bytes > 0, "pack_size", c, N, K);
  expect(sdq_logical_bytes(&c, N, K, &lbytes) == SDQ_OK && lbytes > 0, "logical_bytes", c, N, K);
  Buf p1(bytes), p5(bytes);
  expect(sdq_pack(&c, W.data(), N, K, an.data(), p1.get(), bytes, 1) == SDQ_OK, "pack 1 thread", c, N, K);
  expect(sdq_pack(&c, W.data(), N, K, an.data(), p5.get(), bytes, 5) == SDQ_OK, "pack 5 threads", c, N, K);
  expect(std::memcmp(p1.get(), p5.get(), bytes) == 0, "pack thread independence", c, N, K);
  expect(sdq_pack(&c, W.data(), N, K, an.data(), p1.get(), bytes - 1, 2) == SDQ_ERR_BUFFER_TOO_SMALL,
         "pack small buffer", c, N, K);
  expect(sdq_pack(&c, nullptr, N, K, an.data(), p1.get(), bytes, 2) == SDQ_ERR_NULL, "pack NULL", c, N, K);

  const bool mx = c.family == SDQ_FAMILY_MX, dual = c.family == SDQ_FAMILY_DUAL;
  const long go = c.n_o ? K / c.m_o * c.n_o : 0, gi = K / 8 * c.n_i;
  const size_t so_bytes = mx ? size_t(N) * (K / 32) : size_t(N) * 4;
  const size_t si_bytes = (mx || dual) ? size_t(N) * (K / 32)
                                       : size_t(N) * (K / 16) * (c.sfmt_i == SDQ_SCALE_E4M3 ? 1 : 2);
  Buf po(size_t(N) * go), co(size_t(N) * go), so(so_bytes), pi(size_t(N) * gi), ci(size_t(N) * gi),
      si(si_bytes), sr(size_t(N) * 4);
  expect(sdq_pack_logical(&c, W.data(), N, K, an.data(), c.n_o ? po.get() : nullptr, c.n_o ? co.get() : nullptr,
                          so.get(), pi.get(), ci.get(), si.get(), reinterpret_cast<float*>(sr.get()), 3) == SDQ_OK,
         "pack_logical", c, N, K);
  Buf cod(size_t(N) * K), cid(size_t(N) * K), so2(so_bytes), si2(si_bytes), sr2(size_t(N) * 4);
  expect(sdq_unpack_dense(&c, p1.get(), bytes, N, K, cod.get(), cid.get(), so2.get(), si2.get(),
                          reinterpret_cast<float*>(sr2.get())) == SDQ_OK,
         "unpack_dense", c, N, K);
  expect(std::memcmp(so.get(), so2.get(), so_bytes) == 0, "outlier scales round trip", c, N, K);
  expect(std::memcmp(si.get(), si2.get(), si_bytes) == 0, "inlier scales round trip", c, N, K);
  // every logical slot's code sits at its position in the dense unpacked form
  for (long n = 0; n < N; ++n)
    for (long g = 0; g < K / 8; ++g)
      for (int j = 0; j < c.n_i; ++j) {
        const size_t s = (size_t(n) * (K / 8) + g) * c.n_i + j;
        const uint8_t code = ci.get()[s], pos = pi.get()[s];
        const uint8_t got = cid.get()[size_t(n) * K + g * 8 + pos];
        const uint8_t mask = (mx || dual) ? 0x0F : 0xFF;
        if (pos >= 8 || (got & mask) != (code & mask)) {
          expect(false, "inlier slot round trip", c, N, K);
          return;
        }
      }
  if (c.n_o) {  // a NaN anywhere is refused
    std::vector<float> Wn = W;
    Wn[size_t(N) * K / 2] = std::nanf("");
    expect(sdq_pack(&c, Wn.data(), N, K, an.data(), p1.get(), bytes, 2) == SDQ_ERR_VALUE, "pack NaN", c, N, K);
  }
}

}  // namespace

int main() {
  std::mt19937 rng(7);
  const std::vector<sdq_config> cfgs = {
      cfg(SDQ_FAMILY_INT, 1, 8, SDQ_FMT_E4M3, 3),
      cfg(SDQ_FAMILY_INT, 1, 8, SDQ_FMT_INT8, 3),
      cfg(SDQ_FAMILY_INT, 1, 16, SDQ_FMT_E4M3, 2),
      cfg(SDQ_FAMILY_INT, 0, 8, SDQ_FMT_E4M3, 3),
      cfg(SDQ_FAMILY_INT, 1, 8, SDQ_FMT_E4M3, 3, SDQ_METRIC_MAGNITUDE, SDQ_DECOMP_SAME, SDQ_ORDER_LARGE,
          SDQ_SCALE_E4M3),
      cfg(SDQ_FAMILY_INT, 1, 8, SDQ_FMT_E4M3, 3, SDQ_METRIC_PRODUCT, SDQ_DECOMP_OUTPUT_ERROR),
      cfg(SDQ_FAMILY_INT, 1, 16, SDQ_FMT_INT8, 3, SDQ_METRIC_MAGNITUDE, SDQ_DECOMP_ERROR, SDQ_ORDER_SMALL),
      cfg(SDQ_FAMILY_MX, 1, 8, SDQ_FMT_E4M3, 2),
      cfg(SDQ_FAMILY_MX, 1, 16, SDQ_FMT_E4M3, 3, SDQ_METRIC_PRODUCT),
      cfg(SDQ_FAMILY_MX, 0, 8, SDQ_FMT_E4M3, 2),
      cfg(SDQ_FAMILY_DUAL, 1, 8, SDQ_FMT_INT8, 6),
      cfg(SDQ_FAMILY_DUAL, 0, 8, SDQ_FMT_INT8, 8),
  };
  const long shapes[][2] = {{1, 128}, {33, 256}, {70, 384}, {5, 1024}};
  for (const auto& c : cfgs)
    for (const auto& s : shapes) run(c, s[0], s[1], rng);
  if (failures) {
    std::printf("%d failures\n", failures);
    return 1;
  }
  std::printf("packer sanitized run ok\n");
  return 0;
}
