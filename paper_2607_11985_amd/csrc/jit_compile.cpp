// jit_compile.cpp -- hiprtc compilation of one generated kernel for gfx950.
// Linked into the library and into the vqc_jitc helper, which runs it in a
// process of its own so that the kernels of one circuit compile in parallel
// (the run-time compiler serializes the compilations of one process).
#include <hip/hiprtc.h>

#include "vqc.h"
#include "vqc_internal.h"

namespace vqc {

// Shared headers embedded at build time (generated from vqc_structs.h and
// vqc_device.h).
extern const int kJitHeaderCount;
extern const char* const kJitHeaderNames[];
extern const char* const kJitHeaderSources[];

namespace {
const char* const kJitOptions[] = {
    "--offload-arch=gfx950", "-O3", "-std=c++17",
    // no packed FP32 instructions in any device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    // keep the near-identical register cases apart (see build.py)
    "-mllvm", "-simplifycfg-sink-common=false", "-mllvm", "-simplifycfg-hoist-common=false"};
}  // namespace

int compile_source(const std::string& src, std::vector<char>& code, std::string& log) {
  hiprtcProgram prog;
  if (hiprtcCreateProgram(&prog, src.c_str(), "vqc_jit.hip", kJitHeaderCount, kJitHeaderSources,
                          kJitHeaderNames) != HIPRTC_SUCCESS) {
    log = "hiprtcCreateProgram failed";
    return VQC_ERR_UNSUPPORTED;
  }
  const int nopt = (int)(sizeof(kJitOptions) / sizeof(kJitOptions[0]));
  const hiprtcResult rc = hiprtcCompileProgram(prog, nopt, kJitOptions);
  size_t n = 0;
  hiprtcGetProgramLogSize(prog, &n);
  log.assign(n, '\0');
  if (n) hiprtcGetProgramLog(prog, &log[0]);
  if (rc != HIPRTC_SUCCESS) {
    hiprtcDestroyProgram(&prog);
    return VQC_ERR_UNSUPPORTED;
  }
  size_t sz = 0;
  hiprtcGetCodeSize(prog, &sz);
  code.resize(sz);
  hiprtcGetCode(prog, code.data());
  hiprtcDestroyProgram(&prog);
  return VQC_OK;
}

}  // namespace vqc
