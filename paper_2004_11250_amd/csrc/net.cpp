// net.cpp -- pp_net_workspace / pp_net_fwd: run a flat op list (one entry
// per fused layer, the layer-wise representation of Sec. 3) on one stream.
// Slot 0 is the input, slot 1 the output, slots 2.. live in the caller's
// workspace at fixed 256-byte-aligned offsets.  Validation of the whole list
// happens before the first launch.  A pruned conv whose output only feeds
// the op right after it -- a 2 x 2 max pool, a residual add or a pixel
// shuffle -- runs as one fused launch (graph-level fusion, Sec. 3): that op
// is taken in the conv's store; an x2 upsample whose output only feeds the
// pruned conv right after it is taken in the conv's loads.  Logical slots
// map to workspace buffers, and a fused pair may leave two slots with
// swapped buffers:
//   - a pool or shuffle that writes the conv's input slot (ping-pong slot
//     use) is written to the conv's output buffer instead;
//   - an add dst = src + conv(x) whose skip operand src is dead afterwards
//     accumulates into src's buffer in place, which becomes dst's;
//   - a conv that reads an upsample's input slot and writes that slot
//     writes the upsample's unused output buffer instead.
#include <dlfcn.h>
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

#include <string>
#include <vector>

#include "api_internal.hpp"
#include "dense.hpp"
#include "ppk1.hpp"

namespace pp {
namespace {

struct Shape {
  int c = 0, h = 0, w = 0;
  bool defined = false;
};

struct Plan {
  std::vector<Shape> in, in2, out;
  std::vector<BlobView> views;
  // op i is a pruned conv fused with op i + 1: the conv's extra flag
  // (PP_MAXPOOL2, PP_ACCUMULATE or PP_PIXSHUF2), else 0
  std::vector<uint32_t> fuse;
  // op i is a pruned conv that reads the input of the upsample at i - 1
  // (PP_UPSAMPLE2); that upsample does not run
  std::vector<char> up_in;
  // per op: the buffers (0 = x, 1 = y, >= 2 workspace) of src, src2, dst
  std::vector<int> b_src, b_src2, b_dst;
  size_t buf_bytes[PP_MAX_SLOTS] = {};
  size_t buf_off[PP_MAX_SLOTS] = {};
  size_t ws_bytes = 0;
  // scratch of the pruned convs' channel splits (partial sums), after the slots
  size_t scratch_off = 0, scratch_bytes = 0;
  Shape final_shape;
};

pp_status bad(int i, const std::string& msg) { return fail(PP_EINVAL, "op " + std::to_string(i) + ": " + msg); }

// device: the op list is for a launch (device pointers must be set); a plan
// query reads host memory only
pp_status make_plan(const pp_net_op* ops, int n_ops, int n, int c, int h, int w, int act, Plan* pl,
                    bool device = true) {
  if (!ops || n_ops < 1) return fail(PP_EINVAL, "empty op list");
  if (n < 1 || c < 1 || h < 1 || w < 1) return fail(PP_EINVAL, "bad input shape");
  if (act != PP_F32 && act != PP_BF16) return fail(PP_EINVAL, "bad activation dtype");
  const size_t esz = act == PP_BF16 ? 2 : 4;
  Shape slots[PP_MAX_SLOTS];
  slots[0] = Shape{c, h, w, true};
  pl->in.resize(n_ops);
  pl->in2.resize(n_ops);
  pl->out.resize(n_ops);
  pl->views.resize(n_ops);
  pl->fuse.assign(n_ops, 0);
  pl->up_in.assign(n_ops, 0);
  std::vector<Shape> writes1;
  size_t part_max = 0;
  for (int i = 0; i < n_ops; ++i) {
    const pp_net_op& op = ops[i];
    if (op.src < 0 || op.src >= PP_MAX_SLOTS || op.dst < 1 || op.dst >= PP_MAX_SLOTS) return bad(i, "slot out of range");
    if (op.dst == op.src) return bad(i, "dst equals src");
    if (!slots[op.src].defined) return bad(i, "src slot not written yet");
    const Shape s = slots[op.src];
    Shape o;
    switch (op.kind) {
      case PP_OP_CONV_PP: {
        pp_status st = parse_blob(op.h_blob, op.blob_bytes, &pl->views[i], /*full=*/false);
        if (st != PP_OK) return st;
        if (device && !op.d_blob) return bad(i, "d_blob is NULL");
        const BlobView& v = pl->views[i];
        if (v.c_in != s.c) return bad(i, "input channels do not match the blob");
        {
          const size_t pb = conv_scratch_bytes(v, n, s.h, s.w, act);
          if (pb > part_max) part_max = pb;
        }
        if (op.flags & ~static_cast<uint32_t>(PP_RELU)) return bad(i, "unknown flags");
        int ho = 0, wo = 0;
        st = conv_check(v, n, s.h, s.w, act, &ho, &wo);
        if (st != PP_OK) return st;
        o = Shape{v.c_out, ho, wo, true};
        break;
      }
      case PP_OP_CONV_DENSE: {
        if (op.k != 1 && op.k != 3 && op.k != 9) return fail(PP_EUNSUPPORTED, "dense conv: k must be 1, 3 or 9");
        if (op.stride != 1 || op.dilation != 1) return fail(PP_EUNSUPPORTED, "dense conv: stride and dilation 1 only");
        if (op.pad < 0 || op.pad > op.k) return bad(i, "bad pad");
        if (op.c_in != s.c || op.c_out < 1) return bad(i, "channel mismatch");
        if (device && !op.d_w) return bad(i, "d_w is NULL");
        const int ho = s.h + 2 * op.pad - op.k + 1, wo = s.w + 2 * op.pad - op.k + 1;
        if (ho < 1 || wo < 1) return bad(i, "input smaller than the kernel");
        o = Shape{op.c_out, ho, wo, true};
        break;
      }
      case PP_OP_DECONV: {
        if (op.k != 4 || op.stride != 2 || op.pad != 1)
          return fail(PP_EUNSUPPORTED, "transposed conv: kernel 4, stride 2, pad 1 only");
        if (op.c_in != s.c || op.c_out < 1) return bad(i, "channel mismatch");
        if (device && !op.d_w) return bad(i, "d_w is NULL");
        o = Shape{op.c_out, 2 * s.h, 2 * s.w, true};
        {
          // (the weights laid out per parity class, in the scratch)
          const size_t db = deconv_scratch_bytes(op.c_in, op.c_out, act == PP_BF16);
          if (db > part_max) part_max = db;
        }
        break;
      }
      case PP_OP_MAXPOOL2:
        if (s.h < 2 || s.w < 2) return bad(i, "maxpool input smaller than 2x2");
        o = Shape{s.c, s.h / 2, s.w / 2, true};
        break;
      case PP_OP_UPSAMPLE2:
        o = Shape{s.c, 2 * s.h, 2 * s.w, true};
        break;
      case PP_OP_PIXSHUF2:
        if (s.c % 4) return bad(i, "pixel shuffle needs a multiple of 4 channels");
        o = Shape{s.c / 4, 2 * s.h, 2 * s.w, true};
        break;
      case PP_OP_ADD: {
        if (op.src2 < 0 || op.src2 >= PP_MAX_SLOTS || !slots[op.src2].defined) return bad(i, "src2 not written yet");
        if (op.dst == op.src2) return bad(i, "dst equals src2");
        const Shape s2 = slots[op.src2];
        if (s2.c != s.c || s2.h != s.h || s2.w != s.w) return bad(i, "add operands differ in shape");
        pl->in2[i] = s2;
        o = s;
        break;
      }
      default:
        return bad(i, "unknown op kind");
    }
    const double elems = static_cast<double>(n) * o.c * o.h * o.w;
    if (elems > static_cast<double>(1LL << 40)) return bad(i, "activation too large");
    pl->in[i] = s;
    pl->out[i] = o;
    slots[op.dst] = o;
    if (op.dst == 1) writes1.push_back(o);
  }
  if (!slots[1].defined) return fail(PP_EINVAL, "no op writes the output slot 1");
  auto dead_after = [&](int slot, int j0) {
    for (int j = j0; j < n_ops; ++j) {
      if (ops[j].src == slot || (ops[j].kind == PP_OP_ADD && ops[j].src2 == slot)) return false;
      if (ops[j].dst == slot) return true;   // rewritten: later reads see the new value
    }
    return true;
  };
  // upsample + conv: the conv reads the upsample's output slot v (not slot
  // 1), which no later op reads before rewriting it.  A conv that writes the
  // upsample's input slot u (which it now reads) writes v's buffer instead,
  // which then becomes u's (u in the workspace; no op after the conv fused)
  for (int i = 0; i + 1 < n_ops; ++i) {
    const pp_net_op& us = ops[i];
    const pp_net_op& cv = ops[i + 1];
    if (us.kind != PP_OP_UPSAMPLE2 || cv.kind != PP_OP_CONV_PP || cv.src != us.dst || us.dst == 1 ||
        (cv.dst == us.src && cv.dst < 2) || !dead_after(us.dst, i + 2))
      continue;
    if (conv_fusable(pl->views[i + 1], n, pl->in[i + 1].h, pl->in[i + 1].w, act, PP_UPSAMPLE2, true)) {
      pl->up_in[i + 1] = 1;
      ++i;
    }
  }
  // the slot a pruned conv reads
  auto read_slot = [&](int i) { return pl->up_in[i] ? ops[i - 1].src : ops[i].src; };
  // conv fusion.  The op after the conv reads the conv's output slot, which
  // is not slot 1 and which no later op reads before rewriting it:
  //   - max pool / pixel shuffle: one that writes the slot the conv reads
  //     needs that slot in the workspace (its buffer is swapped);
  //   - add of a skip slot r (both in the workspace, as is the add's dst)
  //     that the conv does not read and that is dead after the add as well.
  for (int i = 0; i + 1 < n_ops; ++i) {
    const pp_net_op& cv = ops[i];
    const pp_net_op& nx = ops[i + 1];
    if (cv.kind != PP_OP_CONV_PP || cv.dst == 1) continue;
    const int cs = read_slot(i);
    if (cs == cv.dst) continue;   // upsample + conv writing its own input slot: no third op
    uint32_t f = 0;
    if ((nx.kind == PP_OP_MAXPOOL2 || nx.kind == PP_OP_PIXSHUF2) && nx.src == cv.dst && !(nx.dst == cs && cs < 2)) {
      f = nx.kind == PP_OP_MAXPOOL2 ? PP_MAXPOOL2 : PP_PIXSHUF2;
    } else if (nx.kind == PP_OP_ADD && (nx.src == cv.dst) != (nx.src2 == cv.dst)) {
      const int r = nx.src == cv.dst ? nx.src2 : nx.src;
      if (r >= 2 && nx.dst >= 2 && r != cs && dead_after(r, i + 2)) f = PP_ACCUMULATE;
    }
    const uint32_t fin = pl->up_in[i] ? PP_UPSAMPLE2 : 0u;
    if (f && dead_after(cv.dst, i + 2) &&
        conv_fusable(pl->views[i], n, pl->in[i].h, pl->in[i].w, act, f | fin, true)) {
      pl->fuse[i] = f;
      ++i;   // the second op is taken; it cannot start another pair
    }
  }
  // buffers: each op reads and writes the buffers its slots map to now.  A
  // fused pair whose pool / shuffle writes the conv's input slot writes the
  // conv's output buffer and then swaps the two slots' buffers (the conv's
  // output slot is dead after the pair, the input slot is overwritten by
  // it); a fused add writes the skip slot's buffer and then swaps it with
  // the add's dst (the skip slot is dead after the add).  A conv that takes
  // the upsample before it reads that upsample's input buffer; the upsample
  // writes nothing, and a conv that writes the upsample's input slot writes
  // the upsample's output buffer and then swaps the two slots' buffers.
  int buf[PP_MAX_SLOTS];
  for (int s = 0; s < PP_MAX_SLOTS; ++s) buf[s] = s;
  pl->b_src.assign(n_ops, 0);
  pl->b_src2.assign(n_ops, 0);
  pl->b_dst.assign(n_ops, 0);
  for (int i = 0; i < n_ops; ++i) {
    const pp_net_op& op = ops[i];
    if (i + 1 < n_ops && pl->up_in[i + 1]) continue;   // taken by the conv after it
    pl->b_src[i] = buf[pl->up_in[i] ? ops[i - 1].src : op.src];
    pl->b_src2[i] = op.kind == PP_OP_ADD ? buf[op.src2] : 0;
    Shape o = pl->out[i];
    int swap_a = -1, swap_b = -1;   // slots whose buffers swap after the op
    if (pl->fuse[i]) {
      const pp_net_op& nx = ops[i + 1];
      if (pl->fuse[i] == PP_ACCUMULATE) {
        const int r = nx.src == op.dst ? nx.src2 : nx.src;
        pl->b_dst[i] = buf[r];
        swap_a = r;
        swap_b = nx.dst;
      } else if (nx.dst == read_slot(i)) {
        pl->b_dst[i] = buf[op.dst];
        swap_a = op.dst;
        swap_b = nx.dst;
      } else {
        pl->b_dst[i] = buf[nx.dst];
      }
      o = pl->out[i + 1];
    } else if (pl->up_in[i] && op.dst == ops[i - 1].src) {
      pl->b_dst[i] = buf[ops[i - 1].dst];   // the upsample's (unwritten) output buffer
      swap_a = op.dst;
      swap_b = ops[i - 1].dst;
    } else {
      pl->b_dst[i] = buf[op.dst];
    }
    const size_t bytes = static_cast<size_t>(n) * o.c * o.h * o.w * esz;
    if (bytes > pl->buf_bytes[pl->b_dst[i]]) pl->buf_bytes[pl->b_dst[i]] = bytes;
    if (swap_a >= 0) {
      const int t = buf[swap_a];
      buf[swap_a] = buf[swap_b];
      buf[swap_b] = t;
    }
    if (pl->fuse[i]) ++i;
  }
  for (const Shape& s : writes1)
    if (s.c != slots[1].c || s.h != slots[1].h || s.w != slots[1].w)
      return fail(PP_EINVAL, "slot 1 is written with different shapes");
  pl->final_shape = slots[1];
  size_t off = 0;
  for (int b = 2; b < PP_MAX_SLOTS; ++b) {
    pl->buf_off[b] = off;
    off += (pl->buf_bytes[b] + 255) / 256 * 256;
  }
  pl->scratch_off = off;
  pl->scratch_bytes = (part_max + 255) / 256 * 256;
  pl->ws_bytes = off + pl->scratch_bytes;
  return PP_OK;
}

}  // namespace
}  // namespace pp

using namespace pp;

extern "C" pp_status pp_net_workspace(const pp_net_op* ops, int32_t n_ops, int32_t n, int32_t c, int32_t h, int32_t w,
                                      int32_t act_dtype, size_t* bytes, int32_t* out_c, int32_t* out_h,
                                      int32_t* out_w) {
  clear_error();
  Plan pl;
  pp_status st = make_plan(ops, n_ops, n, c, h, w, act_dtype, &pl);
  if (st != PP_OK) return st;
  if (bytes) *bytes = pl.ws_bytes;
  if (out_c) *out_c = pl.final_shape.c;
  if (out_h) *out_h = pl.final_shape.h;
  if (out_w) *out_w = pl.final_shape.w;
  return PP_OK;
}

extern "C" pp_status pp_net_plan(const pp_net_op* ops, int32_t n_ops, int32_t n, int32_t c, int32_t h, int32_t w,
                                 int32_t act_dtype, uint32_t* op_flags, int32_t* recipe) {
  clear_error();
  if (!op_flags) return fail(PP_EINVAL, "NULL op_flags");
  Plan pl;
  pp_status st = make_plan(ops, n_ops, n, c, h, w, act_dtype, &pl, /*device=*/false);
  if (st != PP_OK) return st;
  for (int i = 0; i < n_ops; ++i) {
    op_flags[i] = 0;
    if (recipe) recipe[i] = -1;
  }
  for (int i = 0; i < n_ops; ++i) {
    if (ops[i].kind != PP_OP_CONV_PP) continue;
    const uint32_t f = pl.fuse[i] | (pl.up_in[i] ? PP_UPSAMPLE2 : 0u);
    op_flags[i] = f;
    if (pl.up_in[i]) op_flags[i - 1] = PP_NET_TAKEN;
    if (pl.fuse[i]) op_flags[i + 1] = PP_NET_TAKEN;
    if (recipe) {
      // the conv reads the stored (not upsampled) input of a taken upsample
      const Shape& s = pl.up_in[i] ? pl.in[i - 1] : pl.in[i];
      recipe[i] = conv_recipe(pl.views[i], n, s.h, s.w, act_dtype, ops[i].flags | f, pl.scratch_bytes);
    }
  }
  return PP_OK;
}

// PP_TRACE (environment, read once per process; set and not "0"): the
// launches of each op, or fused pair, inside a named roctx range ("pp op <i>
// <kind>"), for rocprofv3 --marker-trace.  The roctx library is loaded at run
// time (none is linked in); when it is not found there are no ranges.
namespace {
struct Tracer {
  int (*push)(const char*) = nullptr;
  int (*pop)() = nullptr;
  Tracer() {
    const char* e = std::getenv("PP_TRACE");
    if (!e || !*e || (e[0] == '0' && !e[1])) return;
    void* h = dlopen("librocprofiler-sdk-roctx.so.1", RTLD_NOW | RTLD_LOCAL);
    if (!h) h = dlopen("libroctx64.so.4", RTLD_NOW | RTLD_LOCAL);
    if (!h) return;
    push = reinterpret_cast<int (*)(const char*)>(dlsym(h, "roctxRangePushA"));
    pop = reinterpret_cast<int (*)()>(dlsym(h, "roctxRangePop"));
    if (!push || !pop) push = nullptr, pop = nullptr;
  }
};
const Tracer& tracer() {
  static const Tracer t;
  return t;
}
const char* op_kind_name(int kind) {
  switch (kind) {
    case PP_OP_CONV_PP: return "conv3 (pruned)";
    case PP_OP_CONV_DENSE: return "conv (dense)";
    case PP_OP_DECONV: return "deconv";
    case PP_OP_MAXPOOL2: return "maxpool2";
    case PP_OP_UPSAMPLE2: return "upsample2";
    case PP_OP_PIXSHUF2: return "pixshuf2";
    case PP_OP_ADD: return "add";
    default: return "op";
  }
}
}  // namespace

extern "C" pp_status pp_net_fwd(const pp_net_op* ops, int32_t n_ops, const void* x, void* y, int32_t n, int32_t c,
                                int32_t h, int32_t w, int32_t act_dtype, void* workspace, size_t ws_bytes,
                                void* hip_stream) {
  clear_error();
  Plan pl;
  pp_status st = make_plan(ops, n_ops, n, c, h, w, act_dtype, &pl);
  if (st != PP_OK) return st;
  if (!x || !y) return fail(PP_EINVAL, "NULL x or y");
  if (ws_bytes < pl.ws_bytes) return fail(PP_ESIZE, "workspace smaller than pp_net_workspace");
  if (pl.ws_bytes && !workspace) return fail(PP_EINVAL, "NULL workspace");
  if (reinterpret_cast<uintptr_t>(workspace) % 256) return fail(PP_EINVAL, "workspace must be 256-byte aligned");
  const bool bf = act_dtype == PP_BF16;
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  auto buf_ptr = [&](int b) -> void* {
    if (b == 0) return const_cast<void*>(x);
    if (b == 1) return y;
    return static_cast<uint8_t*>(workspace) + pl.buf_off[b];
  };
  void* scratch = pl.scratch_bytes ? static_cast<uint8_t*>(workspace) + pl.scratch_off : nullptr;
  for (int i = 0; i < n_ops; ++i) {
    const pp_net_op& op = ops[i];
    if (i + 1 < n_ops && pl.up_in[i + 1]) continue;   // the upsample runs in the conv after it
    const Shape& si = pl.up_in[i] ? pl.in[i - 1] : pl.in[i];   // the input as stored
    const Shape& so = pl.out[i];
    void* dst = buf_ptr(pl.b_dst[i]);
    const void* src = buf_ptr(pl.b_src[i]);
    hipError_t e = hipSuccess;
    const Tracer& tr = tracer();
    if (tr.push) {
      char name[96];
      std::snprintf(name, sizeof(name), "pp op %d %s%s%s%s", i, pl.up_in[i] ? "upsample2 + " : "", op_kind_name(op.kind),
                    pl.fuse[i] ? " + " : "", pl.fuse[i] && i + 1 < n_ops ? op_kind_name(ops[i + 1].kind) : "");
      tr.push(name);
    }
    switch (op.kind) {
      case PP_OP_CONV_PP: {
        // with the upsample before it (PP_UPSAMPLE2) and / or the pool, add or
        // shuffle after it (then op i + 1 is taken too)
        const uint32_t fl = op.flags | pl.fuse[i] | (pl.up_in[i] ? PP_UPSAMPLE2 : 0u);
        // a layer the net runs in its matrix-core form reads the caller's
        // prepared weights (d_w) instead of expanding the blob into the
        // scratch
        if (op.d_w && act_dtype == PP_BF16 &&
            conv_recipe(pl.views[i], n, si.h, si.w, act_dtype, fl, pl.scratch_bytes) == kRecipeMfma) {
          st = conv_enqueue(pl.views[i], op.d_blob, src, dst, n, si.h, si.w, act_dtype, fl | PP_PREPARED,
                            const_cast<void*>(op.d_w), prepared_bytes(pl.views[i]), stream);
        } else if (op.d_w) {
          // the lean kernel's part of the prepared weights (if the layer has
          // one), with the net's scratch for a split
          st = conv_enqueue(pl.views[i], op.d_blob, src, dst, n, si.h, si.w, act_dtype, fl, scratch, pl.scratch_bytes,
                            stream, lean_prepared(pl.views[i], op.d_w));
        } else {
          st = conv_enqueue(pl.views[i], op.d_blob, src, dst, n, si.h, si.w, act_dtype, fl, scratch, pl.scratch_bytes,
                            stream);
        }
        if (st != PP_OK) {
          if (tr.push) tr.pop();
          return st;
        }
        if (pl.fuse[i]) ++i;
        break;
      }
      case PP_OP_CONV_DENSE:
      case PP_OP_DECONV: {
        DenseParams p;
        p.x = src;
        p.y = dst;
        p.wt = op.d_w;
        p.bias = op.d_b;
        p.n = n;
        p.c_in = si.c;
        p.h = si.h;
        p.w = si.w;
        p.c_out = so.c;
        p.ho = so.h;
        p.wo = so.w;
        p.k = op.k;
        p.stride = op.stride;
        p.pad = op.pad;
        p.relu = (op.flags & PP_RELU) ? 1 : 0;
        if (op.kind == PP_OP_DECONV && pl.scratch_bytes >= deconv_scratch_bytes(si.c, so.c, bf)) p.scratch = scratch;
        e = op.kind == PP_OP_CONV_DENSE ? launch_dense_conv(p, bf, stream) : launch_deconv(p, bf, stream);
        break;
      }
      default: {
        GlueParams p;
        p.op = op.kind == PP_OP_MAXPOOL2 ? kGlueMaxPool2
             : op.kind == PP_OP_UPSAMPLE2 ? kGlueUp2
             : op.kind == PP_OP_PIXSHUF2 ? kGluePixShuf2 : kGlueAdd;
        p.x = src;
        p.x2 = op.kind == PP_OP_ADD ? buf_ptr(pl.b_src2[i]) : nullptr;
        p.y = dst;
        p.n = n;
        p.c_in = si.c;
        p.h = si.h;
        p.w = si.w;
        p.c_out = so.c;
        p.ho = so.h;
        p.wo = so.w;
        e = launch_glue(p, bf, stream);
        break;
      }
    }
    if (tr.push) tr.pop();
    if (e != hipSuccess) return fail(PP_EHIP, "op " + std::to_string(i) + ": " + hipGetErrorString(e));
  }
  return PP_OK;
}
