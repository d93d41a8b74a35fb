// project.cpp -- host-side pruning-structure helpers: the Euclidean
// projections of ADMM-based structured pruning (Sec. 2) onto pattern,
// connectivity and column structure, the column-pruned layer as a pattern
// library, and batch-norm folding (the conv + BatchNorm fusion of Sec. 3).
// Energies are double sums in ascending tap (filter) order, so the integer
// decisions they drive do not depend on the build.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <numeric>
#include <vector>

#include "ppk1.hpp"

using namespace pp;

namespace {

bool mask_ok(const uint16_t* lib, int32_t n) {
  for (int32_t p = 0; p < n; ++p)
    if (lib[p] == 0 || lib[p] > 0x1FF) return false;
  return true;
}

// indices of v sorted by value descending, then index ascending; the first n
void top_n(const std::vector<double>& v, int64_t n, std::vector<uint8_t>& keep) {
  std::vector<int64_t> idx(v.size());
  std::iota(idx.begin(), idx.end(), int64_t{0});
  std::sort(idx.begin(), idx.end(), [&](int64_t a, int64_t b) { return v[a] > v[b] || (v[a] == v[b] && a < b); });
  keep.assign(v.size(), 0);
  for (int64_t i = 0; i < n; ++i) keep[idx[i]] = 1;
}

}  // namespace

extern "C" pp_status pp_project_patterns(const float* w, int32_t c_out, int32_t c_in, const uint16_t* lib_masks,
                                         int32_t n_patterns, uint8_t* pattern_id, double* kept_energy) {
  clear_error();
  if (!w || !lib_masks || !pattern_id) return fail(PP_EINVAL, "NULL argument");
  if (c_out < 1 || c_in < 1 || c_out > 65535 || c_in > 65535) return fail(PP_EINVAL, "bad channel counts");
  if (n_patterns < 1 || n_patterns > 255) return fail(PP_EINVAL, "n_patterns must be 1..255");
  if (!mask_ok(lib_masks, n_patterns)) return fail(PP_EINVAL, "pattern masks must be in 1..511");
  const size_t nk = static_cast<size_t>(c_out) * c_in;
  for (size_t k = 0; k < nk; ++k) {
    const float* kw = w + 9 * k;
    double best = -1.0;
    int bp = 0;
    for (int32_t p = 0; p < n_patterns; ++p) {
      double e = 0.0;
      for (int t = 0; t < 9; ++t)
        if ((lib_masks[p] >> t) & 1u) e += static_cast<double>(kw[t]) * static_cast<double>(kw[t]);
      if (e > best) {   // strictly larger: ties keep the lower pattern
        best = e;
        bp = p;
      }
    }
    pattern_id[k] = static_cast<uint8_t>(bp);
    if (kept_energy) kept_energy[k] = best;
  }
  return PP_OK;
}

extern "C" pp_status pp_project_connectivity(const double* energy, int32_t c_out, int32_t c_in, int64_t n_keep,
                                             uint8_t* conn) {
  clear_error();
  if (!energy || !conn) return fail(PP_EINVAL, "NULL argument");
  if (c_out < 1 || c_in < 1 || c_out > 65535 || c_in > 65535) return fail(PP_EINVAL, "bad channel counts");
  const int64_t nk = static_cast<int64_t>(c_out) * c_in;
  if (n_keep < 0 || n_keep > nk) return fail(PP_EINVAL, "n_keep must be 0..c_out*c_in");
  std::vector<double> v(energy, energy + nk);
  for (double e : v)
    if (!(e >= 0.0)) return fail(PP_EINVAL, "energies must be >= 0 (and not NaN)");
  std::vector<uint8_t> keep;
  top_n(v, n_keep, keep);
  std::copy(keep.begin(), keep.end(), conn);
  return PP_OK;
}

extern "C" pp_status pp_project_columns(const float* w, int32_t c_out, int32_t c_in, int64_t n_keep,
                                        uint16_t* col_mask) {
  clear_error();
  if (!w || !col_mask) return fail(PP_EINVAL, "NULL argument");
  if (c_out < 1 || c_in < 1 || c_out > 65535 || c_in > 65535) return fail(PP_EINVAL, "bad channel counts");
  const int64_t ncol = static_cast<int64_t>(c_in) * 9;
  if (n_keep < 0 || n_keep > ncol) return fail(PP_EINVAL, "n_keep must be 0..9*c_in");
  std::vector<double> e(ncol, 0.0);
  for (int32_t o = 0; o < c_out; ++o) {
    const float* fw = w + static_cast<size_t>(o) * ncol;
    for (int64_t j = 0; j < ncol; ++j) e[j] += static_cast<double>(fw[j]) * static_cast<double>(fw[j]);
  }
  std::vector<uint8_t> keep;
  top_n(e, n_keep, keep);
  for (int32_t c = 0; c < c_in; ++c) {
    uint16_t m = 0;
    for (int t = 0; t < 9; ++t)
      if (keep[9 * static_cast<int64_t>(c) + t]) m = static_cast<uint16_t>(m | (1u << t));
    col_mask[c] = m;
  }
  return PP_OK;
}

extern "C" pp_status pp_column_library(const uint16_t* col_mask, int32_t c_out, int32_t c_in, uint16_t* lib_masks,
                                       int32_t* n_patterns, uint8_t* pattern_id, uint8_t* conn) {
  clear_error();
  if (!col_mask || !lib_masks || !n_patterns || !pattern_id || !conn) return fail(PP_EINVAL, "NULL argument");
  if (c_out < 1 || c_in < 1 || c_out > 65535 || c_in > 65535) return fail(PP_EINVAL, "bad channel counts");
  std::vector<uint16_t> lib;
  for (int32_t c = 0; c < c_in; ++c) {
    if (col_mask[c] > 0x1FF) return fail(PP_EINVAL, "column masks must be 9-bit");
    if (col_mask[c]) lib.push_back(col_mask[c]);
  }
  std::sort(lib.begin(), lib.end());
  lib.erase(std::unique(lib.begin(), lib.end()), lib.end());
  if (lib.size() > 255) return fail(PP_EUNSUPPORTED, "more than 255 distinct column masks");
  if (lib.empty()) lib.push_back(1);   // a layer with no column left still needs a library
  std::copy(lib.begin(), lib.end(), lib_masks);
  *n_patterns = static_cast<int32_t>(lib.size());
  for (int32_t c = 0; c < c_in; ++c) {
    const uint8_t p = col_mask[c] ? static_cast<uint8_t>(std::lower_bound(lib.begin(), lib.end(), col_mask[c]) -
                                                         lib.begin())
                                  : 0;
    for (int32_t o = 0; o < c_out; ++o) {
      pattern_id[static_cast<size_t>(o) * c_in + c] = p;
      conn[static_cast<size_t>(o) * c_in + c] = col_mask[c] ? 1 : 0;
    }
  }
  return PP_OK;
}

extern "C" pp_status pp_fold_bn(float* w, float* bias, int32_t c_out, int32_t k_elems, const float* gamma,
                                const float* beta, const float* mean, const float* var, float eps) {
  clear_error();
  if (!w || !bias || !gamma || !beta || !mean || !var) return fail(PP_EINVAL, "NULL argument");
  if (c_out < 1 || k_elems < 1) return fail(PP_EINVAL, "bad sizes");
  for (int32_t o = 0; o < c_out; ++o) {
    const double d = static_cast<double>(var[o]) + static_cast<double>(eps);
    if (!(d > 0.0)) return fail(PP_EINVAL, "var + eps must be > 0");
  }
  for (int32_t o = 0; o < c_out; ++o) {
    const double s = static_cast<double>(gamma[o]) / std::sqrt(static_cast<double>(var[o]) + static_cast<double>(eps));
    float* fw = w + static_cast<size_t>(o) * k_elems;
    for (int32_t j = 0; j < k_elems; ++j) fw[j] = static_cast<float>(static_cast<double>(fw[j]) * s);
    bias[o] = static_cast<float>((static_cast<double>(bias[o]) - static_cast<double>(mean[o])) * s +
                                 static_cast<double>(beta[o]));
  }
  return PP_OK;
}
