// Per-graph specialised kernels, compiled at run time with hipRTC.
//
// The compiled plan of a graph (or of a pair of graphs for a comparison) is
// written into a small HIP source as __constant__ data and the kernel bodies
// of kernels_dev.h are instantiated against it, so every instruction field,
// op dispatch and trip count is a compile-time constant.  Code objects are
// cached per process by source text; modules are loaded per device.
#pragma once

#include <cstdint>
#include <memory>
#include <string>
#include <vector>

#include "compile.h"

namespace dg {

// Source of the specialised enumeration kernels (dg_sizes, dg_fill,
// dg_enumerate) of one plan for blocks of `block` threads.
std::string jit_enum_source(const Plan& p, int block);
// Source of the specialised 64-bit enumeration kernel (dg_enumerate_wide).
std::string jit_wide_source(const Plan& p, int block);
// Source of the specialised comparison kernel (dg_compare) of a pair.
std::string jit_compare_source(const Plan& a, const Plan& b, const dgc::PairPlan& pp, int block);

// Source of the specialised expression-DAG kernels (dg_dag_sizes,
// dg_dag_fill, dg_dag_onepass) of one DAG program for blocks of `block` threads: the
// program's ops are walked unrolled, and only the ways of taking a group
// that its groups use are compiled.
std::string jit_dag_source(const DagProgram& p, int block);

// hipRTC options of the specialised kernels (null-terminated list).
const char* const* jit_compile_options();

// Compiles one specialised source with the runtime compiler linked into the
// calling program; true and the code object, or false and the log.
bool jit_compile_source(const std::string& src, std::vector<char>* code, std::string* log);

}  // namespace dg

#if defined(__HIP_PLATFORM_AMD__) || defined(__HIPCC__)
#include <hip/hip_runtime.h>

namespace dg {

// Compiles (or takes from the cache) and loads on the current device.
// Returns true and the module; on failure a message in *log.  Modules are
// shared by every caller that loads the same source on the same device and
// counted: each successful jit_load is matched by one jit_release, and the
// last release unloads the module.  Compiled code objects stay in a small
// host-side cache (the most recently used few) so that a graph built again
// from the same text is not compiled again.
struct JitModule {
  hipModule_t mod = nullptr;
  hipFunction_t sizes = nullptr, fill = nullptr, enumerate = nullptr, compare = nullptr, enumerate_wide = nullptr;
  hipFunction_t dag_sizes = nullptr, dag_fill = nullptr, dag_onepass = nullptr;
  int dev = -1;        // device the module is loaded on
  std::string source;  // its source (the key of the shared module)
};
bool jit_load(const std::string& source, JitModule* out, std::string* log);
void jit_release(JitModule* m);

// Whether run-time specialisation is enabled (environment DIRIGO_JIT=0
// turns it off; the precompiled kernels then run every graph).
bool jit_enabled();

}  // namespace dg
#endif
