// Entry points of abi.cpp used by other files of the library (not part of
// the C ABI).
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <string>

#include "../../include/dirigo_rocm.h"

namespace dg_internal {

// Records msg as the calling thread's last error and returns code.
dg_status fail(dg_status code, const std::string& msg);

// Bytes of workspace one call over n locations uses (dg_workspace_size).
size_t workspace_bytes(int64_t n);

// dg_enumerate on a graph already resident on the current device (its plan
// and, with specialisation on, its kernels loaded by an earlier call there),
// with d_ws as the workspace; allocates and loads nothing.  DG_E_INVALID_ARG
// when the graph is not resident.
dg_status enumerate_resident(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_offsets,
                             uint32_t* d_ids, uint32_t* d_counts, int64_t capacity, void* d_ws, int64_t* h_total,
                             void* stream);

}  // namespace dg_internal
