// jit.cpp -- run-time specialisation of the wave-pipeline kernel for a
// layer's own library of 4-tap patterns (hipRTC).  The canonical library's
// kernels branch on a pattern code into cases whose tap offsets are
// compile-time constants; any other library runs on the generic kernel,
// which tests taps against run-time masks.  A library of up to 8 patterns of
// exactly 4 taps has the canonical library's form, so the same kernel source
// compiled with that library as its tap table (PP_JIT_LIBRARY) runs it at the
// canonical speed: the per-layer code generation of the paper's compiler
// (Sec. 3), done by the device compiler at run time.
#include <hip/hip_runtime.h>
#include <hip/hiprtc.h>

#include <array>
#include <cstdio>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "api_internal.hpp"
#include "conv_pp.hpp"
#include "jit_sources.inc"   // kJitHeaders / kJitHeaderNames: the kernel headers, embedded at build time

namespace pp {
namespace {

struct JitKey {
  std::array<uint16_t, 8> masks{};
  int n_patterns = 0, stride = 0, dil = 0, recipe = 0, bf16 = 0, device = 0;
  bool operator<(const JitKey& o) const {
    return std::tie(masks, n_patterns, stride, dil, recipe, bf16, device) <
           std::tie(o.masks, o.n_patterns, o.stride, o.dil, o.recipe, o.bf16, o.device);
  }
};

struct JitKernels {
  hipModule_t module = nullptr;
  hipFunction_t conv = nullptr, reduce = nullptr;
};

std::mutex g_mu;
std::map<JitKey, JitKernels> g_cache;   // modules stay loaded for the life of the process

// what the run-time compiler lacks from the host headers
const char* kPrelude =
    "typedef __hip_internal::int8_t int8_t; typedef __hip_internal::uint8_t uint8_t;\n"
    "typedef __hip_internal::int16_t int16_t; typedef __hip_internal::uint16_t uint16_t;\n"
    "typedef __hip_internal::int32_t int32_t; typedef __hip_internal::uint32_t uint32_t;\n"
    "typedef __hip_internal::int64_t int64_t; typedef __hip_internal::uint64_t uint64_t;\n"
    "typedef __hip_internal::uint64_t uintptr_t;\n"
    "namespace std {\n"
    "template <class T, T v> struct integral_constant {\n"
    "  static constexpr T value = v;\n"
    "  constexpr operator T() const { return v; }\n"
    "};\n"
    "using true_type = integral_constant<bool, true>;\n"
    "using false_type = integral_constant<bool, false>;\n"
    "}\n";

std::string kernel_names(const JitKey& k, std::string* conv, std::string* reduce) {
  const RecipeInfo r = recipe_info(k.recipe);
  const int sh = (4 - k.dil % 4) % 4;   // the compiled padding is pad = dilation
  const char* ta = k.bf16 ? "uint16_t" : "float";
  char b[256];
  std::snprintf(b, sizeof b, "pp::kern::pp_conv3x3_wave_kernel<%d, %d, %d, %d, %d, %d, %d, %d, %s, %s>", kLibCanon8,
                k.stride, k.dil, r.r, r.cc, r.lw, r.ws, sh, r.pipe ? "true" : "false", ta);
  *conv = b;
  std::snprintf(b, sizeof b, "pp::kern::pp_split_reduce_kernel<%d, %d, %d, %s>", r.r, r.cc, r.lw, ta);
  *reduce = b;
  std::string src = kPrelude;
  src += "#define PP_JIT_LIBRARY ";
  for (int i = 0; i < 8; ++i) {
    std::snprintf(b, sizeof b, "%s0x%03X", i ? ", " : "", k.masks[i]);
    src += b;
  }
  src += "\n#include \"conv_pp_wave.hpp\"\n";
  src += "template __global__ void " + *conv + "(pp::ConvParams);\n";
  src += "template __global__ void " + *reduce + "(pp::ConvParams);\n";
  return src;
}

pp_status compile(const JitKey& k, JitKernels* out) {
  std::string conv, reduce;
  const std::string src = kernel_names(k, &conv, &reduce);
  hiprtcProgram prog;
  if (hiprtcCreateProgram(&prog, src.c_str(), "pp_jit.hip", kJitHeaderCount, kJitHeaders, kJitHeaderNames) !=
      HIPRTC_SUCCESS)
    return fail(PP_EHIP, "hiprtcCreateProgram failed");
  hiprtcAddNameExpression(prog, conv.c_str());
  hiprtcAddNameExpression(prog, reduce.c_str());
  // the library's own build flags (no packed FP32; see build.py)
  const char* opts[] = {"--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
                        "-packed-fp32-ops", "-mllvm", "-structurizecfg-skip-uniform-regions", "-mllvm",
                        "-simplifycfg-sink-common=false", "-Wno-pass-failed"};
  const hiprtcResult cr = hiprtcCompileProgram(prog, static_cast<int>(sizeof opts / sizeof opts[0]), opts);
  if (cr != HIPRTC_SUCCESS) {
    size_t n = 0;
    hiprtcGetProgramLogSize(prog, &n);
    std::string log(n, '\0');
    if (n) hiprtcGetProgramLog(prog, &log[0]);
    hiprtcDestroyProgram(&prog);
    return fail(PP_EHIP, "run-time compilation failed: " + log.substr(0, 400));
  }
  const char *lc = nullptr, *lr = nullptr;
  hiprtcGetLoweredName(prog, conv.c_str(), &lc);
  hiprtcGetLoweredName(prog, reduce.c_str(), &lr);
  const std::string nc = lc ? lc : "", nr = lr ? lr : "";
  size_t size = 0;
  hiprtcGetCodeSize(prog, &size);
  std::vector<char> code(size);
  hiprtcGetCode(prog, code.data());
  hiprtcDestroyProgram(&prog);
  if (nc.empty() || nr.empty() || !size) return fail(PP_EHIP, "run-time compilation gave no kernels");
  JitKernels kk;
  hipError_t e = hipModuleLoadData(&kk.module, code.data());
  if (e == hipSuccess) e = hipModuleGetFunction(&kk.conv, kk.module, nc.c_str());
  if (e == hipSuccess) e = hipModuleGetFunction(&kk.reduce, kk.module, nr.c_str());
  if (e != hipSuccess) return fail(PP_EHIP, std::string("loading the compiled kernels: ") + hipGetErrorString(e));
  *out = kk;
  return PP_OK;
}

bool make_key(const BlobView& v, const ConvPlan& plan, bool bf16, JitKey* k) {
  if (!jit_library4(v)) return false;
  for (int i = 0; i < 8; ++i) k->masks[i] = v.masks[i < v.n_patterns ? i : v.n_patterns - 1];
  k->n_patterns = v.n_patterns;
  k->stride = v.stride;
  k->dil = v.dil;
  k->recipe = plan.recipe;
  k->bf16 = bf16 ? 1 : 0;
  hipGetDevice(&k->device);
  return true;
}

}  // namespace

bool jit_library4(const BlobView& v) {
  return v.n_patterns >= 1 && v.n_patterns <= 8 && v.all_four_taps && library_kind(v) == kLibGeneric;
}

pp_status jit_prepare(const BlobView& v, const ConvPlan& plan, bool bf16) {
  JitKey k;
  if (!make_key(v, plan, bf16, &k)) return fail(PP_EUNSUPPORTED, "not a library of up to 8 four-tap patterns");
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_cache.count(k)) return PP_OK;
  JitKernels kk;
  const pp_status s = compile(k, &kk);
  if (s != PP_OK) return s;
  g_cache[k] = kk;
  return PP_OK;
}

bool jit_ready(const BlobView& v, const ConvPlan& plan, bool bf16) {
  JitKey k;
  if (!make_key(v, plan, bf16, &k)) return false;
  std::lock_guard<std::mutex> lock(g_mu);
  return g_cache.count(k) != 0;
}

bool jit_launch(const BlobView& v, const ConvPlan& plan, ConvParams p, bool bf16, hipStream_t st, hipError_t* err) {
  JitKey k;
  if (!make_key(v, plan, bf16, &k)) return false;
  JitKernels kk;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    auto it = g_cache.find(k);
    if (it == g_cache.end()) return false;
    kk = it->second;
  }
  // the geometry of launch_wave_tiling for this recipe
  const RecipeInfo r = recipe_info(plan.recipe);
  const int th = (64 / r.lw) * r.r, tw = r.lw * r.cc;
  p.ksplit = plan.ksplit;
  p.tiles_x = (p.wo + tw - 1) / tw;
  p.tiles_y = (p.ho + th - 1) / th;
  p.n_ftiles = p.n_groups;
  const size_t nb = static_cast<size_t>(p.n_groups) * p.tiles_x * p.tiles_y * p.n * p.ksplit;
  if (p.pad != p.dil || tw % 4 != 0 || nb == 0 || nb > 0x7FFFFFFFull || (p.ksplit > 1 && !p.part)) {
    *err = hipErrorInvalidConfiguration;
    return true;
  }
  void* args[] = {&p};
  hipError_t e = hipModuleLaunchKernel(kk.conv, static_cast<uint32_t>(nb), 1, 1, r.ws * 64, 1, 1, 0, st, args, nullptr);
  if (e == hipSuccess && p.ksplit > 1)
    e = hipModuleLaunchKernel(kk.reduce, static_cast<uint32_t>(nb / p.ksplit), 1, 1, 256, 1, 1, 0, st, args, nullptr);
  *err = e;
  return true;
}

}  // namespace pp
