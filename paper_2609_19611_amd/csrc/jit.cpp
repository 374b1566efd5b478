// Run-time specialisation of the per-location kernels (see jit.h).
#include "jit.h"

#include <hip/hiprtc.h>

#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <sstream>

namespace dg {

// Text of program.h, core.h and kernels_dev.h, embedded at build time.
extern const char* const kJitProgramH;
extern const char* const kJitCoreH;
extern const char* const kJitKernelsDevH;

namespace {

std::mutex g_mu;
// Loaded modules: (device, source) -> module and the number of holders.
struct Loaded {
  hipModule_t mod = nullptr;
  int refs = 0;
};
std::map<std::pair<int, std::string>, Loaded> g_modules;
// Compiled code objects by source, with a use stamp; at most kCodeCache are
// kept (least recently used dropped first).
struct Code {
  std::vector<char> bytes;
  uint64_t stamp = 0;
};
const size_t kCodeCache = 128;
std::map<std::string, Code> g_code;
uint64_t g_clock = 0;

void remember_code(const std::string& source, const std::vector<char>& code) {  // g_mu held
  Code& c = g_code[source];
  c.bytes = code;
  c.stamp = ++g_clock;
  while (g_code.size() > kCodeCache) {
    auto oldest = g_code.begin();
    for (auto it = g_code.begin(); it != g_code.end(); ++it)
      if (it->second.stamp < oldest->second.stamp) oldest = it;
    g_code.erase(oldest);
  }
}

bool compile(const std::string& src, std::vector<char>* code, std::string* log) {
  hiprtcProgram prog;
  const char* headers[] = {kJitProgramH, kJitCoreH, kJitKernelsDevH};
  const char* names[] = {"program.h", "core.h", "kernels_dev.h"};
  if (hiprtcCreateProgram(&prog, src.c_str(), "dg_plan.hip", 3, headers, names) != HIPRTC_SUCCESS) {
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

}  // namespace

bool jit_enabled() {
  const char* e = std::getenv("DIRIGO_JIT");
  return !(e && std::strcmp(e, "0") == 0);
}

bool jit_load(const std::string& source, JitModule* out, std::string* log) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    *log = "hipGetDevice failed";
    return false;
  }
  std::vector<char> code;
  out->mod = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    auto mit = g_modules.find({dev, source});
    if (mit != g_modules.end()) {
      ++mit->second.refs;
      out->mod = mit->second.mod;
    } else {
      auto it = g_code.find(source);
      if (it != g_code.end()) {
        code = it->second.bytes;
        it->second.stamp = ++g_clock;
      }
    }
  }
  if (!out->mod) {
    if (code.empty()) {
      if (!compile(source, &code, log)) return false;
      std::lock_guard<std::mutex> lock(g_mu);
      remember_code(source, code);
    }
    hipModule_t m = nullptr;
    hipError_t e = hipModuleLoadData(&m, code.data());
    if (e != hipSuccess) {
      *log = std::string("hipModuleLoadData: ") + hipGetErrorString(e);
      return false;
    }
    std::lock_guard<std::mutex> lock(g_mu);
    Loaded& L = g_modules[{dev, source}];
    if (L.mod) {
      (void)hipModuleUnload(m);  // another thread loaded it meanwhile
    } else {
      L.mod = m;
    }
    ++L.refs;
    out->mod = L.mod;
  }
  out->dev = dev;
  out->source = source;
  // A module holds either the enumeration kernels or the comparison kernel;
  // a name it lacks leaves a null function.  The failed lookup also sets
  // the thread's last HIP error, which is cleared here so that it is not
  // reported by the next launch check.
  auto get = [&](const char* name, hipFunction_t* f) {
    if (hipModuleGetFunction(f, out->mod, name) != hipSuccess) {
      *f = nullptr;
      (void)hipGetLastError();
    }
  };
  get("dg_sizes", &out->sizes);
  get("dg_fill", &out->fill);
  get("dg_enumerate", &out->enumerate);
  get("dg_compare", &out->compare);
  get("dg_enumerate_wide", &out->enumerate_wide);
  return true;
}

void jit_release(JitModule* m) {
  if (!m || !m->mod) return;
  std::lock_guard<std::mutex> lock(g_mu);
  auto it = g_modules.find({m->dev, m->source});
  if (it != g_modules.end() && --it->second.refs == 0) {
    int cur = -1;
    const bool have = hipGetDevice(&cur) == hipSuccess;
    if (hipSetDevice(m->dev) == hipSuccess) (void)hipModuleUnload(it->second.mod);
    if (have) (void)hipSetDevice(cur);
    g_modules.erase(it);
  }
  *m = JitModule{};
}

}  // namespace dg
