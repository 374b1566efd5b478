// hipRTC compilation of one specialised kernel source against the embedded
// headers (see jit.h): used by the library itself and by the compile helper
// program (jitc_main.cpp).
#include <hip/hiprtc.h>

#include <string>
#include <vector>

#include "jit.h"

namespace dg {

// Text of the device headers, embedded at build time.
extern const char* const kJitProgramH;
extern const char* const kJitCoreH;
extern const char* const kJitKernelsDevH;
extern const char* const kJitDagProgramH;
extern const char* const kJitDagCoreH;
extern const char* const kJitDagDevH;

bool jit_compile_source(const std::string& src, std::vector<char>* code, std::string* log) {
  hiprtcProgram prog;
  const char* headers[] = {kJitProgramH, kJitCoreH, kJitKernelsDevH, kJitDagProgramH, kJitDagCoreH, kJitDagDevH};
  const char* names[] = {"program.h", "core.h", "kernels_dev.h", "dag_program.h", "dag_core.h", "dag_dev.h"};
  if (hiprtcCreateProgram(&prog, src.c_str(), "dg_plan.hip", 6, headers, names) != HIPRTC_SUCCESS) {
    *log = "hiprtcCreateProgram failed";
    return false;
  }
  const char* const* opts = jit_compile_options();
  int nopt = 0;
  while (opts[nopt]) ++nopt;
  hiprtcResult r = hiprtcCompileProgram(prog, nopt, const_cast<const char**>(opts));
  size_t n = 0;
  hiprtcGetProgramLogSize(prog, &n);
  if (n > 1) {
    std::string l(n, '\0');
    hiprtcGetProgramLog(prog, &l[0]);
    *log = l;
  }
  if (r != HIPRTC_SUCCESS) {
    hiprtcDestroyProgram(&prog);
    return false;
  }
  size_t sz = 0;
  hiprtcGetCodeSize(prog, &sz);
  code->resize(sz);
  hiprtcGetCode(prog, code->data());
  hiprtcDestroyProgram(&prog);
  return true;
}

}  // namespace dg
