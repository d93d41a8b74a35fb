// ppk1.hpp -- layout constants and host-side view of a PPK1 packed layer.
//
// The layout (documented in pp.h) is the compact pruned-weight storage of
// the paper (Sec. 3, "sparse model storage"): only kept taps are stored, and
// the positions of the taps follow from the kernel's pattern id, so there is
// no per-weight index.  Filters are reordered (Sec. 3, "matrix reorder") and
// grouped eight to a slot group; per (group, input channel) one byte per slot
// gives the pattern id of that kernel or 0xFF when connectivity pruning
// removed it.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>

#include "pp.h"

namespace pp {

constexpr uint32_t kMagic = 0x314B5050u;   // "PPK1"
constexpr uint32_t kVersion = 2;
constexpr uint32_t kMaxWt = (1u << 24) - 1;   // woff keeps the kept-slot mask in bits 24..31
constexpr int kGroup = 8;                  // filters per slot group
constexpr int kAlign = 64;                 // section alignment in bytes
constexpr int kHeaderWords = 24;
constexpr uint8_t kPruned = 0xFF;
constexpr uint32_t kNoFilter = 0xFFFFFFFFu;

enum HeaderField {
  H_MAGIC = 0, H_VERSION, H_COUT, H_CIN, H_STRIDE, H_PAD, H_DIL, H_NPAT, H_GROUP, H_NGROUPS,
  H_NKEPT, H_NWT, H_OFF_MASKS, H_OFF_PERM, H_OFF_CODES, H_OFF_WOFF, H_OFF_W, H_OFF_BIAS,
  H_TOTAL
};

// Parsed, validated view of a host blob (pointers into the caller's bytes).
struct BlobView {
  int c_out = 0, c_in = 0, stride = 0, pad = 0, dil = 0, n_patterns = 0, n_groups = 0;
  int wdtype = 0;
  int64_t n_kept = 0, n_wt = 0;
  uint32_t off_masks = 0, off_perm = 0, off_codes = 0, off_woff = 0, off_w = 0, off_bias = 0;
  size_t total = 0;
  const uint16_t* masks = nullptr;
  const uint32_t* perm = nullptr;
  const uint8_t* codes = nullptr;
  const uint32_t* woff = nullptr;
  const float* bias = nullptr;
  int max_taps = 0;            // largest pattern size in the library
  bool all_four_taps = false;  // every pattern has exactly 4 taps
};

// Validation of a host blob; fills `v` on success.  `full` also checks every
// code, woff entry and perm entry (O(blob size)); without it only the header,
// the section layout and the pattern library are checked (O(1) + library),
// which is all the kernels rely on: they clamp every offset they read from
// the device copy, so a device blob whose body differs from a valid header
// can give wrong numbers but never reads or writes out of bounds.
pp_status parse_blob(const void* blob, size_t bytes, BlobView* v, bool full = true);

// Thread-local error detail (pp_last_error).
pp_status fail(pp_status s, const std::string& msg);
void clear_error();

inline size_t align_up(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }

}  // namespace pp
