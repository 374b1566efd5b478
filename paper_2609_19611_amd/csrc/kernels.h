// Launchers of the HIP kernels (kernels.hip), called by the C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "core.h"
#include "order.h"

namespace dgk {

hipError_t launch_sizes(const uint8_t* blob, dgc::LocSrc locs, int64_t n, int64_t* offsets, uint32_t* err,
                        int block, uint32_t lds, hipStream_t s);
// Row i is written at [offsets[i] - base, offsets[i+1] - base) of ids/cnt.
hipError_t launch_fill(const uint8_t* blob, dgc::LocSrc locs, int64_t n, const int64_t* offsets, int64_t base,
                       uint32_t* ids, uint32_t* cnt, uint32_t* err, int block, uint32_t lds, hipStream_t s);
// dst[i] = src[i] - base for i < count.
hipError_t launch_rebase(const int64_t* src, int64_t* dst, int64_t count, int64_t base, hipStream_t s);
// pp: device copy of the pair plan; lds: pp's lds_bytes.  found: a word
// counting mismatching locations (cleared by the caller); with limit > 0,
// locations that start after `limit` mismatches were found are skipped.
hipError_t launch_compare(const uint8_t* blob_a, const uint8_t* blob_b, const dgc::PairPlan* pp, uint32_t lds,
                          dgc::LocSrc locs, int64_t n, uint8_t* status, int64_t* flags, uint64_t* found,
                          uint64_t limit, uint32_t* err, int block, hipStream_t s);
// In-place scan: v[1..n] holds sizes on entry, running totals on exit, v[0] = 0.
hipError_t launch_scan(int64_t* v, int64_t n, int64_t* sums, hipStream_t s);
int64_t scan_temp_entries(int64_t n);
// Single pass over n locations: offsets[0..n] and the rows (written only
// where they fit `capacity` entries).  status: n words, ticket: one word,
// both cleared by the caller before the first launch.  One launch runs
// `blocks` blocks, each taking the next location from the ticket; launches
// whose blocks add up to n cover every location.
hipError_t launch_enumerate(const uint8_t* blob, dgc::LocSrc locs, int64_t n, int64_t blocks, int64_t* offsets,
                            uint32_t* ids, uint32_t* cnt, uint64_t capacity, uint64_t* status, uint64_t* ticket,
                            uint32_t* err, int block, uint32_t lds, hipStream_t s);
// The same with 64-bit ids and counts.
hipError_t launch_enumerate_wide(const uint8_t* blob, dgc::LocSrc locs, int64_t n, int64_t blocks,
                                 int64_t* offsets, uint64_t* ids, uint64_t* cnt, uint64_t capacity, uint64_t* status,
                                 uint64_t* ticket, uint32_t* err, int block, uint32_t lds, hipStream_t s);
// Expression DAGs (dag_program.h, DgdHeader; lds: the program's lds_bytes):
// node and edge counts of location i into nodes_n[i + 1], edges_n[i + 1];
// then nodes and edges at node_off[i], edge_off[i]; each block takes
// per_block consecutive locations.
hipError_t launch_dag_sizes(const uint8_t* dblob, dgc::LocSrc locs, int64_t n, int per_block, int64_t* nodes_n,
                            int64_t* edges_n, uint32_t* err, int block, uint32_t lds, hipStream_t s);
// One pass (sizes, offsets by look-back, DAGs) over n locations in a grid
// of `blocks` blocks taking tickets (a list longer than one grid runs as
// several launches); the stage follows the walk's LDS area.
hipError_t launch_dag_onepass(const uint8_t* dblob, dgc::LocSrc locs, int64_t n, int64_t blocks, int64_t* node_off,
                              int64_t* edge_off, uint32_t* nodes, uint32_t* node_edge, uint32_t* edges,
                              uint32_t* mults, uint64_t node_cap, uint64_t edge_cap, uint32_t stage_off,
                              uint32_t stage_nodes, uint32_t stage_edges, uint64_t* st_nodes, uint64_t* st_edges,
                              uint64_t* ticket, uint32_t* err, int block, uint32_t lds, hipStream_t s);
hipError_t launch_dag_fill(const uint8_t* dblob, dgc::LocSrc locs, int64_t n, int per_block, const int64_t* node_off,
                           const int64_t* edge_off, uint32_t* nodes, uint32_t* node_edge, uint32_t* edges,
                           uint32_t* mults, uint32_t* err, int block, uint32_t lds, hipStream_t s);
// Location order: positions [first, first + count) of the keyed
// permutation K (order.h) into out, leaving out the sorted excluded
// positions pos[0..m) (all inside the range) and closing the gaps.
hipError_t launch_order(const DgPermKey& K, const int64_t* pos, int64_t m, int64_t first, int64_t count,
                        int64_t* out, hipStream_t s);
// Clears count 64-bit words.
hipError_t launch_zero_u64(uint64_t* p, int64_t count, hipStream_t s);
// Clears one error word (a kernel, so it may be recorded in a captured graph).
hipError_t launch_zero(uint32_t* p, hipStream_t s);
hipError_t launch_scatter_mismatch(const uint8_t* status, const int64_t* pos, int64_t n, int64_t* out,
                                   hipStream_t s);

}  // namespace dgk
