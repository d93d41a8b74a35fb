// Host-side checks of the packer, the blob validation and the pruning
// helpers, built with AddressSanitizer and UndefinedBehaviorSanitizer (CPU
// only; tests/test_sanitize.py compiles and runs it).
//
//   * seeded random layers (shapes, pattern libraries of 1..12 masks,
//     connectivity, fp32 / bf16 storage, strides, pads, dilations) are
//     packed and must validate, with the kept-kernel count the connectivity
//     mask gives;
//   * every packed blob is then handed to pp_blob_info truncated (at every
//     length of its header and at random lengths beyond) and with random bit
//     flips and byte overwrites: the call must return (OK or an error code)
//     without reading outside the buffer, which the sanitizers check;
//   * the pruning helpers run on random inputs and on their error paths.
//
// Exit status 0 when every check holds; a sanitizer report aborts.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "pp.h"

namespace {

// splitmix64: a counter-based generator for the seeded draws
struct Rng {
  uint64_t s;
  explicit Rng(uint64_t seed) : s(seed) {}
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  uint32_t below(uint32_t n) { return static_cast<uint32_t>(next() % n); }
  float normal() {   // sum of uniforms: enough for weights
    float t = 0.0f;
    for (int i = 0; i < 4; ++i) t += static_cast<float>(next() >> 40) / static_cast<float>(1 << 24);
    return t - 2.0f;
  }
};

int g_fail = 0;
#define CHECK(c)                                                    \
  do {                                                              \
    if (!(c)) {                                                     \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      ++g_fail;                                                     \
    }                                                               \
  } while (0)

// pp_blob_info on an exact-size copy of the first n bytes (so that any read
// past n leaves the allocation)
pp_status info_of(const std::vector<uint8_t>& b, size_t n) {
  std::vector<uint8_t> c(b.begin(), b.begin() + static_cast<long>(n));
  pp_layer_desc d;
  int32_t kept = 0;
  int64_t nwt = 0;
  return pp_blob_info(n ? c.data() : reinterpret_cast<const uint8_t*>(""), n, &d, &kept, &nwt);
}

void fuzz_blob(Rng& r, const std::vector<uint8_t>& blob) {
  const size_t n = blob.size();
  // truncations
  for (size_t k = 0; k < 96 && k < n; ++k) CHECK(info_of(blob, k) != PP_OK);
  for (int t = 0; t < 8; ++t) {
    const size_t k = r.below(static_cast<uint32_t>(n));
    CHECK(info_of(blob, k) != PP_OK);
  }
  CHECK(info_of(blob, n) == PP_OK);
  // bit flips and byte overwrites: any status, no out-of-bounds access
  for (int t = 0; t < 24; ++t) {
    std::vector<uint8_t> c = blob;
    const int nflip = 1 + static_cast<int>(r.below(8));
    for (int f = 0; f < nflip; ++f) {
      const size_t at = (t % 3 == 0) ? r.below(96) : r.below(static_cast<uint32_t>(n));
      if (t % 2) c[at] ^= static_cast<uint8_t>(1u << r.below(8));
      else c[at] = static_cast<uint8_t>(r.next());
    }
    (void)info_of(c, n);
  }
}

void random_layers(int count) {
  Rng r(2004011250ull);
  for (int it = 0; it < count; ++it) {
    pp_layer_desc d;
    d.c_out = 1 + static_cast<int32_t>(r.below(40));
    d.c_in = 1 + static_cast<int32_t>(r.below(40));
    d.stride = 1 + static_cast<int32_t>(r.below(2));
    d.dilation = 1 + static_cast<int32_t>(r.below(2));
    d.pad = static_cast<int32_t>(r.below(3));
    d.wdtype = r.below(2) ? PP_BF16 : PP_F32;
    const int np = 1 + static_cast<int>(r.below(12));
    std::vector<uint16_t> masks(np);
    for (auto& m : masks) m = static_cast<uint16_t>(1 + r.below(511));
    const size_t k = static_cast<size_t>(d.c_out) * d.c_in;
    std::vector<float> w(k * 9), bias(d.c_out);
    for (auto& v : w) v = r.normal();
    for (auto& v : bias) v = r.normal();
    std::vector<uint8_t> pid(k), conn(k);
    int kept = 0;
    const uint32_t keep_per_mille = r.below(1001);
    for (size_t i = 0; i < k; ++i) {
      pid[i] = static_cast<uint8_t>(r.below(static_cast<uint32_t>(np)));
      conn[i] = r.below(1000) < keep_per_mille ? 1 : 0;
      kept += conn[i];
    }
    size_t bytes = 0;
    CHECK(pp_pack(&d, w.data(), it % 5 ? bias.data() : nullptr, pid.data(), conn.data(), masks.data(), np, nullptr,
                  &bytes) == PP_OK);
    std::vector<uint8_t> blob(bytes);
    size_t cap = bytes;
    CHECK(pp_pack(&d, w.data(), bias.data(), pid.data(), conn.data(), masks.data(), np, blob.data(), &cap) ==
          PP_OK);
    CHECK(cap == bytes);
    // capacity one byte short
    size_t small = bytes - 1;
    CHECK(pp_pack(&d, w.data(), bias.data(), pid.data(), conn.data(), masks.data(), np, blob.data(), &small) ==
          PP_ESIZE);
    pp_layer_desc got;
    int32_t nk = -1;
    int64_t nwt = -1;
    CHECK(pp_blob_info(blob.data(), blob.size(), &got, &nk, &nwt) == PP_OK);
    CHECK(nk == kept);
    CHECK(got.c_out == d.c_out && got.c_in == d.c_in && got.wdtype == d.wdtype);
    fuzz_blob(r, blob);
    // bad arguments
    std::vector<uint8_t> bad = conn;
    bad[r.below(static_cast<uint32_t>(k))] = 2;
    CHECK(pp_pack(&d, w.data(), bias.data(), pid.data(), bad.data(), masks.data(), np, nullptr, &bytes) ==
          PP_EINVAL);
    CHECK(pp_pack(&d, nullptr, bias.data(), pid.data(), conn.data(), masks.data(), np, nullptr, &bytes) ==
          PP_EINVAL);
    CHECK(pp_pack(&d, w.data(), bias.data(), pid.data(), conn.data(), masks.data(), 0, nullptr, &bytes) ==
          PP_EINVAL);
  }
}

void projections(int count) {
  Rng r(77);
  const uint16_t canon[8] = {0x03A, 0x0B2, 0x0B8, 0x09A, 0x01B, 0x036, 0x0D8, 0x1B0};
  for (int it = 0; it < count; ++it) {
    const int co = 1 + static_cast<int>(r.below(24)), ci = 1 + static_cast<int>(r.below(24));
    const size_t k = static_cast<size_t>(co) * ci;
    std::vector<float> w(k * 9);
    for (auto& v : w) v = r.normal();
    std::vector<uint8_t> pid(k), conn(k);
    std::vector<double> energy(k);
    CHECK(pp_project_patterns(w.data(), co, ci, canon, 8, pid.data(), energy.data()) == PP_OK);
    for (size_t i = 0; i < k; ++i) CHECK(pid[i] < 8 && energy[i] >= 0.0);
    const int64_t keep = r.below(static_cast<uint32_t>(k + 1));
    CHECK(pp_project_connectivity(energy.data(), co, ci, keep, conn.data()) == PP_OK);
    int64_t nk = 0;
    for (auto v : conn) nk += v;
    CHECK(nk == keep);
    CHECK(pp_project_connectivity(energy.data(), co, ci, static_cast<int64_t>(k) + 1, conn.data()) == PP_EINVAL);
    std::vector<uint16_t> col(ci), lib(255);
    const int64_t ncol = r.below(static_cast<uint32_t>(9 * ci + 1));
    CHECK(pp_project_columns(w.data(), co, ci, ncol, col.data()) == PP_OK);
    int64_t bits = 0;
    for (auto m : col) bits += __builtin_popcount(m);
    CHECK(bits == ncol);
    int32_t npat = 0;
    const pp_status st = pp_column_library(col.data(), co, ci, lib.data(), &npat, pid.data(), conn.data());
    CHECK(st == PP_OK || st == PP_EUNSUPPORTED);
    std::vector<float> bias(co), g(co), b(co), m(co), v(co);
    for (int o = 0; o < co; ++o) {
      g[o] = r.normal();
      b[o] = r.normal();
      m[o] = r.normal();
      v[o] = std::fabs(r.normal()) + 0.5f;
    }
    CHECK(pp_fold_bn(w.data(), bias.data(), co, ci * 9, g.data(), b.data(), m.data(), v.data(), 1e-5f) == PP_OK);
    v[0] = -1.0f;
    CHECK(pp_fold_bn(w.data(), bias.data(), co, ci * 9, g.data(), b.data(), m.data(), v.data(), 0.0f) == PP_EINVAL);
    CHECK(pp_project_patterns(nullptr, co, ci, canon, 8, pid.data(), nullptr) == PP_EINVAL);
  }
  // bf16 rounding over every exponent
  std::vector<float> f(4096);
  std::vector<uint16_t> h(4096);
  for (size_t i = 0; i < f.size(); ++i) {
    const uint32_t u = static_cast<uint32_t>(r.next());
    std::memcpy(&f[i], &u, 4);
  }
  CHECK(pp_round_bf16(f.data(), h.data(), f.size()) == PP_OK);
}

}  // namespace

int main() {
  random_layers(2000);
  projections(500);
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("host fuzz: all checks passed\n");
  return 0;
}
