// pack.cpp -- host packer (pp_pack), blob validation (pp_blob_info) and
// status strings.  No HIP dependency: this file also builds with g++ alone.
//
// pp_pack performs the offline part of the method: the projection of dense
// weights onto the pruning structure (pattern + connectivity, Sec. 2), the
// filter reorder (Sec. 3, "matrix reorder") and the compact storage without
// zero weights or per-weight indices (Sec. 3, "sparse model storage").
#include <algorithm>
#include <cstring>
#include <numeric>
#include <vector>

#include "ppk1.hpp"

namespace pp {

namespace {
thread_local std::string g_err;

int popcount9(uint32_t m) { return __builtin_popcount(m & 0x1FFu); }

// fp32 -> bf16 bits, round to nearest, ties to even (inputs are finite).
uint16_t to_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  uint32_t lsb = (u >> 16) & 1u;
  uint64_t r = (static_cast<uint64_t>(u) + 0x7FFFu + lsb) >> 16;
  return static_cast<uint16_t>(r & 0xFFFFu);
}

void put32(std::vector<uint8_t>& b, size_t off, uint32_t v) { std::memcpy(b.data() + off, &v, 4); }
}  // namespace

pp_status fail(pp_status s, const std::string& msg) {
  g_err = msg;
  return s;
}
void clear_error() { g_err.clear(); }

pp_status parse_blob(const void* blob, size_t bytes, BlobView* v, bool full) {
  if (!blob) return fail(PP_EINVAL, "blob is NULL");
  if (bytes < static_cast<size_t>(kHeaderWords) * 4) return fail(PP_EBLOB, "blob shorter than header");
  uint32_t h[kHeaderWords];
  std::memcpy(h, blob, sizeof(h));
  if (h[H_MAGIC] != kMagic) return fail(PP_EBLOB, "bad magic");
  if ((h[H_VERSION] & 0xFFFFu) != kVersion) return fail(PP_EBLOB, "unsupported version");
  const uint32_t wd = h[H_VERSION] >> 16;
  if (wd != PP_F32 && wd != PP_BF16) return fail(PP_EBLOB, "bad weight dtype");
  for (int i = H_TOTAL + 1; i < kHeaderWords; ++i)
    if (h[i] != 0) return fail(PP_EBLOB, "reserved header word nonzero");
  const uint64_t c_out = h[H_COUT], c_in = h[H_CIN], npat = h[H_NPAT], ng = h[H_NGROUPS];
  if (c_out < 1 || c_out > 65535 || c_in < 1 || c_in > 65535) return fail(PP_EBLOB, "bad channel counts");
  if (h[H_STRIDE] < 1 || h[H_STRIDE] > 16 || h[H_DIL] < 1 || h[H_DIL] > 16 || h[H_PAD] > 16)
    return fail(PP_EBLOB, "bad stride/pad/dilation");
  if (npat < 1 || npat > 255) return fail(PP_EBLOB, "bad pattern count");
  if (h[H_GROUP] != static_cast<uint32_t>(kGroup)) return fail(PP_EBLOB, "bad group size");
  if (ng != (c_out + kGroup - 1) / kGroup) return fail(PP_EBLOB, "bad group count");
  const uint64_t slots = ng * kGroup;
  const uint64_t n_wt = h[H_NWT];
  if (n_wt > kMaxWt) return fail(PP_EBLOB, "n_wt too large");
  const uint64_t wsz = (wd == PP_BF16) ? 2 : 4;
  const uint64_t total = h[H_TOTAL];
  if (total != bytes) return fail(PP_EBLOB, "total_bytes does not match blob size");
  if (total % kAlign) return fail(PP_EBLOB, "total_bytes not aligned");
  // sections must be aligned, ordered and inside the blob
  struct Sec { uint32_t off; uint64_t len; } secs[] = {
      {h[H_OFF_MASKS], 2 * npat},           {h[H_OFF_PERM], 4 * slots},
      {h[H_OFF_CODES], ng * c_in * kGroup}, {h[H_OFF_WOFF], 4 * (ng * c_in + 1)},
      {h[H_OFF_W], wsz * n_wt},             {h[H_OFF_BIAS], 4 * slots}};
  uint64_t prev_end = static_cast<uint64_t>(kHeaderWords) * 4;
  for (const Sec& s : secs) {
    if (s.off % kAlign || s.off < prev_end) return fail(PP_EBLOB, "section offset out of order");
    if (s.off + s.len > total) return fail(PP_EBLOB, "section beyond end of blob");
    prev_end = s.off + s.len;
  }
  const uint8_t* base = static_cast<const uint8_t*>(blob);
  v->c_out = static_cast<int>(c_out);
  v->c_in = static_cast<int>(c_in);
  v->stride = static_cast<int>(h[H_STRIDE]);
  v->pad = static_cast<int>(h[H_PAD]);
  v->dil = static_cast<int>(h[H_DIL]);
  v->n_patterns = static_cast<int>(npat);
  v->n_groups = static_cast<int>(ng);
  v->wdtype = static_cast<int>(wd);
  v->n_kept = h[H_NKEPT];
  v->n_wt = static_cast<int64_t>(n_wt);
  v->off_masks = h[H_OFF_MASKS];
  v->off_perm = h[H_OFF_PERM];
  v->off_codes = h[H_OFF_CODES];
  v->off_woff = h[H_OFF_WOFF];
  v->off_w = h[H_OFF_W];
  v->off_bias = h[H_OFF_BIAS];
  v->total = total;
  v->masks = reinterpret_cast<const uint16_t*>(base + v->off_masks);
  v->perm = reinterpret_cast<const uint32_t*>(base + v->off_perm);
  v->codes = base + v->off_codes;
  v->woff = reinterpret_cast<const uint32_t*>(base + v->off_woff);
  v->bias = reinterpret_cast<const float*>(base + v->off_bias);

  // library
  int max_taps = 0;
  bool four = true;
  std::vector<int> wper(npat);
  for (uint64_t p = 0; p < npat; ++p) {
    uint16_t m;
    std::memcpy(&m, v->masks + p, 2);
    if (m < 1 || m > 0x1FF) return fail(PP_EBLOB, "bad pattern mask");
    int k = popcount9(m);
    max_taps = std::max(max_taps, k);
    four = four && k == 4;
    wper[p] = (wd == PP_BF16) ? (k + 1) / 2 * 2 : k;
  }
  v->max_taps = max_taps;
  v->all_four_taps = four;
  if (!full) return PP_OK;
  // perm: a permutation of 0..c_out-1 followed by padding markers
  std::vector<uint8_t> seen(c_out, 0);
  for (uint64_t i = 0; i < slots; ++i) {
    uint32_t o;
    std::memcpy(&o, v->perm + i, 4);
    if (i < c_out) {
      if (o >= c_out || seen[o]) return fail(PP_EBLOB, "perm is not a permutation");
      seen[o] = 1;
    } else if (o != kNoFilter) {
      return fail(PP_EBLOB, "padding slot has a filter");
    }
  }
  // codes and woff must agree with each other and with n_kept / n_wt
  uint64_t pos = 0, kept = 0;
  for (uint64_t e = 0; e < ng * c_in; ++e) {
    uint32_t wo;
    std::memcpy(&wo, v->woff + e, 4);
    if ((wo & kMaxWt) != pos) return fail(PP_EBLOB, "woff inconsistent with codes");
    const uint64_t g = e / c_in;
    uint32_t mask = 0;
    for (int s = 0; s < kGroup; ++s) {
      uint8_t p = v->codes[e * kGroup + s];
      if (p == kPruned) continue;
      if (p >= npat) return fail(PP_EBLOB, "pattern id out of range");
      if (g * kGroup + s >= c_out) return fail(PP_EBLOB, "kernel in a padding slot");
      pos += wper[p];
      mask |= 1u << s;
      ++kept;
    }
    if ((wo >> 24) != mask) return fail(PP_EBLOB, "kept-slot mask inconsistent with codes");
  }
  uint32_t wend;
  std::memcpy(&wend, v->woff + ng * c_in, 4);
  if (wend != pos || pos != n_wt) return fail(PP_EBLOB, "n_wt inconsistent");
  if (kept != v->n_kept) return fail(PP_EBLOB, "n_kept inconsistent");
  // the kernels read up to 16 bytes past any weight block; the bias section
  // (>= 32 bytes) follows the weights, so such reads stay inside the blob
  if (v->off_bias < v->off_w + wsz * n_wt) return fail(PP_EBLOB, "bias overlaps weights");
  return PP_OK;
}

}  // namespace pp

using namespace pp;

extern "C" pp_status pp_pack(const pp_layer_desc* d, const float* w, const float* bias,
                             const uint8_t* pattern_id, const uint8_t* conn,
                             const uint16_t* lib_masks, int32_t n_patterns, void* out,
                             size_t* inout_bytes) {
  clear_error();
  if (!d || !w || !pattern_id || !conn || !lib_masks || !inout_bytes)
    return fail(PP_EINVAL, "NULL argument");
  const int c_out = d->c_out, c_in = d->c_in;
  if (c_out < 1 || c_out > 65535 || c_in < 1 || c_in > 65535) return fail(PP_EINVAL, "c_out/c_in out of range");
  if (d->stride < 1 || d->stride > 16 || d->dilation < 1 || d->dilation > 16 || d->pad < 0 || d->pad > 16)
    return fail(PP_EINVAL, "stride/dilation/pad out of range");
  if (d->wdtype != PP_F32 && d->wdtype != PP_BF16) return fail(PP_EINVAL, "bad weight dtype");
  if (n_patterns < 1 || n_patterns > 255) return fail(PP_EINVAL, "n_patterns must be 1..255");
  for (int p = 0; p < n_patterns; ++p)
    if (lib_masks[p] < 1 || lib_masks[p] > 0x1FF) return fail(PP_EINVAL, "pattern mask must be 1..511");
  const size_t kk = static_cast<size_t>(c_out) * c_in;
  for (size_t i = 0; i < kk; ++i) {
    if (conn[i] > 1) return fail(PP_EINVAL, "conn must be 0 or 1");
    if (conn[i] && pattern_id[i] >= n_patterns) return fail(PP_EINVAL, "pattern id out of range");
  }
  const bool bf = d->wdtype == PP_BF16;

  // ---- matrix reorder: kept count desc, pattern histogram desc, index asc
  std::vector<int> kept(c_out, 0);
  std::vector<int> hist(static_cast<size_t>(c_out) * n_patterns, 0);
  for (int o = 0; o < c_out; ++o)
    for (int c = 0; c < c_in; ++c) {
      size_t i = static_cast<size_t>(o) * c_in + c;
      if (conn[i]) {
        ++kept[o];
        ++hist[static_cast<size_t>(o) * n_patterns + pattern_id[i]];
      }
    }
  std::vector<int> order(c_out);
  std::iota(order.begin(), order.end(), 0);
  std::sort(order.begin(), order.end(), [&](int a, int b) {
    if (kept[a] != kept[b]) return kept[a] > kept[b];
    for (int p = 0; p < n_patterns; ++p) {
      int ha = hist[static_cast<size_t>(a) * n_patterns + p];
      int hb = hist[static_cast<size_t>(b) * n_patterns + p];
      if (ha != hb) return ha > hb;
    }
    return a < b;
  });

  const int ng = (c_out + kGroup - 1) / kGroup;
  const int slots = ng * kGroup;
  std::vector<int> wper(n_patterns);
  for (int p = 0; p < n_patterns; ++p) {
    int k = popcount9(lib_masks[p]);
    wper[p] = bf ? (k + 1) / 2 * 2 : k;
  }
  // ---- sizes
  uint64_t n_wt = 0, n_kept = 0;
  for (int g = 0; g < ng; ++g)
    for (int s = 0; s < kGroup; ++s) {
      int slot = g * kGroup + s;
      if (slot >= c_out) continue;
      int o = order[slot];
      for (int c = 0; c < c_in; ++c) {
        size_t i = static_cast<size_t>(o) * c_in + c;
        if (conn[i]) {
          n_wt += wper[pattern_id[i]];
          ++n_kept;
        }
      }
    }
  if (n_wt > kMaxWt) return fail(PP_EINVAL, "layer has too many weights for 24-bit offsets");
  const uint64_t wsz = bf ? 2 : 4;
  const size_t off_masks = align_up(kHeaderWords * 4);
  const size_t off_perm = align_up(off_masks + 2 * static_cast<size_t>(n_patterns));
  const size_t off_codes = align_up(off_perm + 4 * static_cast<size_t>(slots));
  const size_t off_woff = align_up(off_codes + static_cast<size_t>(ng) * c_in * kGroup);
  const size_t off_w = align_up(off_woff + 4 * (static_cast<size_t>(ng) * c_in + 1));
  const size_t off_bias = align_up(off_w + wsz * n_wt);
  const size_t total = align_up(off_bias + 4 * static_cast<size_t>(slots));
  if (total > 0xFFFFFFFFull) return fail(PP_EINVAL, "blob larger than 4 GiB");
  if (!out) {
    *inout_bytes = total;
    return PP_OK;
  }
  if (*inout_bytes < total) {
    *inout_bytes = total;
    return fail(PP_ESIZE, "output buffer too small");
  }
  std::vector<uint8_t> b(total, 0);
  const uint32_t hdr[kHeaderWords] = {
      kMagic, kVersion | (static_cast<uint32_t>(d->wdtype) << 16), static_cast<uint32_t>(c_out),
      static_cast<uint32_t>(c_in), static_cast<uint32_t>(d->stride), static_cast<uint32_t>(d->pad),
      static_cast<uint32_t>(d->dilation), static_cast<uint32_t>(n_patterns), kGroup,
      static_cast<uint32_t>(ng), static_cast<uint32_t>(n_kept), static_cast<uint32_t>(n_wt),
      static_cast<uint32_t>(off_masks), static_cast<uint32_t>(off_perm), static_cast<uint32_t>(off_codes),
      static_cast<uint32_t>(off_woff), static_cast<uint32_t>(off_w), static_cast<uint32_t>(off_bias),
      static_cast<uint32_t>(total), 0, 0, 0, 0, 0};
  std::memcpy(b.data(), hdr, sizeof(hdr));
  std::memcpy(b.data() + off_masks, lib_masks, 2 * static_cast<size_t>(n_patterns));
  for (int i = 0; i < slots; ++i)
    put32(b, off_perm + 4 * i, i < c_out ? static_cast<uint32_t>(order[i]) : kNoFilter);
  // ---- codes, woff, weights: entry (g, c), kept slots ascending, taps ascending
  uint8_t* codes = b.data() + off_codes;
  uint64_t pos = 0;
  for (int g = 0; g < ng; ++g)
    for (int c = 0; c < c_in; ++c) {
      const size_t e = static_cast<size_t>(g) * c_in + c;
      const uint64_t pos0 = pos;
      uint32_t kept_mask = 0;
      for (int s = 0; s < kGroup; ++s) {
        uint8_t code = kPruned;
        const int slot = g * kGroup + s;
        if (slot < c_out) {
          const int o = order[slot];
          const size_t i = static_cast<size_t>(o) * c_in + c;
          if (conn[i]) {
            const int p = pattern_id[i];
            code = static_cast<uint8_t>(p);
            const float* wk = w + i * 9;
            int written = 0;
            for (int t = 0; t < 9; ++t) {
              if (!((lib_masks[p] >> t) & 1u)) continue;
              if (bf) {
                uint16_t hv = to_bf16(wk[t]);
                std::memcpy(b.data() + off_w + 2 * (pos + written), &hv, 2);
              } else {
                std::memcpy(b.data() + off_w + 4 * (pos + written), &wk[t], 4);
              }
              ++written;
            }
            pos += wper[p];   // bf16 padding element stays zero
            kept_mask |= 1u << s;
          }
        }
        codes[e * kGroup + s] = code;
      }
      put32(b, off_woff + 4 * e, static_cast<uint32_t>(pos0) | (kept_mask << 24));
    }
  put32(b, off_woff + 4 * (static_cast<size_t>(ng) * c_in), static_cast<uint32_t>(pos));
  for (int i = 0; i < slots; ++i) {
    float bv = (i < c_out && bias) ? bias[order[i]] : 0.0f;
    std::memcpy(b.data() + off_bias + 4 * i, &bv, 4);
  }
  std::memcpy(out, b.data(), total);
  *inout_bytes = total;
  return PP_OK;
}

extern "C" pp_status pp_blob_info(const void* h_blob, size_t bytes, pp_layer_desc* d, int32_t* n_kept,
                                  int64_t* n_wt) {
  clear_error();
  BlobView v;
  pp_status st = parse_blob(h_blob, bytes, &v);
  if (st != PP_OK) return st;
  if (d) {
    d->c_out = v.c_out;
    d->c_in = v.c_in;
    d->stride = v.stride;
    d->pad = v.pad;
    d->dilation = v.dil;
    d->wdtype = v.wdtype;
  }
  if (n_kept) *n_kept = static_cast<int32_t>(v.n_kept);
  if (n_wt) *n_wt = v.n_wt;
  return PP_OK;
}

extern "C" pp_status pp_round_bf16(const float* src, uint16_t* dst, size_t count) {
  clear_error();
  if (count && (!src || !dst)) return fail(PP_EINVAL, "NULL src or dst");
  for (size_t i = 0; i < count; ++i) {
    uint32_t u;
    std::memcpy(&u, src + i, 4);
    // a NaN keeps its sign and top payload bits, made quiet (rounding could
    // carry it into infinity)
    dst[i] = (u & 0x7FFFFFFFu) > 0x7F800000u ? static_cast<uint16_t>((u >> 16) | 0x40u) : to_bf16(src[i]);
  }
  return PP_OK;
}

extern "C" const char* pp_status_str(pp_status s) {
  switch (s) {
    case PP_OK: return "ok";
    case PP_EINVAL: return "invalid argument";
    case PP_ESIZE: return "buffer too small";
    case PP_EBLOB: return "malformed packed blob";
    case PP_EUNSUPPORTED: return "unsupported configuration";
    case PP_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

extern "C" const char* pp_last_error(void) { return pp::g_err.c_str(); }
