// dg_enumerate_noalloc: the single-pass enumeration for callers that cannot
// allocate device memory.  Its workspace (error word, ticket counter and the
// look-back status words of every location) is a file-scope device array,
// one copy per GPU, held until the process ends.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>

#include "../../include/dirigo_rocm.h"
#include "abi_internal.h"

namespace {

// Room for the workspace of DG_NOALLOC_MAX_LOCATIONS locations: 8 bytes of
// status per location plus the fixed header words and scan area.
constexpr size_t kScratchBytes = (size_t(16) << 20) + (size_t(64) << 10);

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

std::mutex g_mu;
std::map<int, void*> g_scratch;  // device -> address of that device's copy of `scratch`

// The device address of the current device's copy of `scratch`, looked up
// once per device.  (In host code `scratch` only names the symbol; its
// address there is not a device address.)
dg_status scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return dg_internal::fail(DG_E_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  std::lock_guard<std::mutex> lock(g_mu);
  auto it = g_scratch.find(dev);
  if (it != g_scratch.end()) {
    *out = it->second;
    return DG_OK;
  }
  void* p = nullptr;
  e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !p)
    return dg_internal::fail(DG_E_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
  g_scratch[dev] = p;
  *out = p;
  return DG_OK;
}

}  // namespace

extern "C" dg_status dg_enumerate_noalloc(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_offsets,
                                          uint32_t* d_ids, uint32_t* d_counts, int64_t capacity, int64_t* h_total,
                                          void* stream) {
  if (!g || !d_offsets || !h_total || n < 0 || capacity < 0 || (n > 0 && !d_locs) ||
      (capacity > 0 && (!d_ids || !d_counts)))
    return dg_internal::fail(DG_E_INVALID_ARG, "bad argument");
  if (n > DG_NOALLOC_MAX_LOCATIONS || dg_internal::workspace_bytes(n) > kScratchBytes)
    return dg_internal::fail(DG_E_WORKSPACE, "dg_enumerate_noalloc takes at most " +
                                                 std::to_string(DG_NOALLOC_MAX_LOCATIONS) + " locations per call");
  void* ws = nullptr;
  dg_status st = scratch_address(&ws);
  if (st != DG_OK) return st;
  return dg_internal::enumerate_resident(g, d_locs, n, d_offsets, d_ids, d_counts, capacity, ws, h_total, stream);
}
