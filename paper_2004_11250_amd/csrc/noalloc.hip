// noalloc.hip -- pp_conv2d_fwd_noalloc: the pruned 3x3 conv with its device
// scratch (a channel split's partial sums, or the bf16 matrix-core form's
// expanded weights) in a file-scope device array instead of a caller
// workspace, for callers that cannot allocate device memory.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "api_internal.hpp"
#include "ppk1.hpp"

namespace pp {
namespace {

// the scratch of every pp_conv2d_fwd_noalloc call on a device (each device
// holds its own copy until the process ends)
constexpr size_t kScratchBytes = size_t(16) << 20;
__device__ __align__(256) uint8_t scratch[kScratchBytes];

// the array's device address, per device: the name is a host-side stand-in
// and must never be passed to a kernel itself
constexpr int kMaxDevices = 64;
void* g_scratch[kMaxDevices] = {};
std::once_flag g_once[kMaxDevices];
hipError_t g_err[kMaxDevices] = {};

pp_status scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(PP_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(PP_EUNSUPPORTED, "device index beyond 63");
  std::call_once(g_once[dev], [dev] {
    void* p = nullptr;
    g_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (g_err[dev] == hipSuccess) g_scratch[dev] = p;
  });
  if (g_err[dev] != hipSuccess || !g_scratch[dev])
    return fail(PP_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(g_err[dev]));
  *out = g_scratch[dev];
  return PP_OK;
}

}  // namespace
}  // namespace pp

using namespace pp;

extern "C" pp_status pp_conv2d_fwd_noalloc(const void* h_blob, size_t blob_bytes, const void* d_blob, const void* x,
                                           void* y, int32_t n, int32_t h, int32_t w, int32_t act_dtype,
                                           uint32_t flags, void* hip_stream) {
  clear_error();
  BlobView v;
  pp_status s = parse_blob(h_blob, blob_bytes, &v, /*full=*/false);
  if (s != PP_OK) return s;
  if (flags & PP_PREPARED) return fail(PP_EINVAL, "PP_PREPARED needs the prepared weights as a workspace");
  // the scratch pp_conv2d_fwd would use with a pp_conv2d_workspace()-sized
  // workspace (that call sizes a PP_UPSAMPLE2 conv by its upsampled input)
  const bool up = (flags & PP_UPSAMPLE2) != 0;
  if (up && (h < 1 || w < 1 || h > (1 << 29) || w > (1 << 29))) return fail(PP_EINVAL, "bad h, w");
  size_t need = 0;
  s = pp_conv2d_workspace(h_blob, blob_bytes, n, up ? 2 * h : h, up ? 2 * w : w, act_dtype, &need);
  if (s != PP_OK) return s;
  if (need > kScratchBytes)
    return fail(PP_ESIZE, "the layer needs " + std::to_string(need) + " bytes of scratch, more than the " +
                              std::to_string(kScratchBytes) + " the allocation-free call holds; use pp_conv2d_fwd " +
                              "with a workspace");
  void* sp = nullptr;
  if (need > 0) {
    s = scratch_address(&sp);
    if (s != PP_OK) return s;
  }
  return conv_enqueue(v, d_blob, x, y, n, h, w, act_dtype, flags, sp, need, static_cast<hipStream_t>(hip_stream));
}
