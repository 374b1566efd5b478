// Host compiler: graph IR -> per-location plan (program.h).
#pragma once
#include <cstdint>
#include <string>
#include <vector>

#include "core.h"
#include "graph.h"
#include "program.h"
#include "view.h"

namespace dg {

// Exact rational number (small numerators and denominators).
struct Frac {
  int64_t n = 0, d = 1;
};

// Where a factor's coordinate range can lie, for every location: each value
// v it covers satisfies  A(r) + lo <= v <= A(r) + hi,  with A a rational
// linear form in the output coordinates r (root dim -> coefficient).  Two
// factors with the same A have a hull of at most floor(hi - lo) + 1
// coordinates however the location moves.
struct FactorPos {
  bool known = false;
  std::vector<std::pair<int, Frac>> a;  // sorted by root dim, no zero coefficients
  Frac lo, hi;
};

struct Plan {
  std::vector<uint8_t> blob;  // DgpHeader followed by the instruction, factor, leaf and term arrays
  int64_t max_row_size = 0;   // static bound on entries per row
  uint64_t count_bound = 0;   // static bound on one path count
  int max_leaf_terms = 0;
  std::vector<FactorPos> fpos;  // per factor (host side only)
  DimPartition part;            // merged dims of every tensor (view.h)
  std::vector<std::vector<int>> leaf_part;  // the leaves' partitions, in declaration order

  const DgpHeader& header() const { return *reinterpret_cast<const DgpHeader*>(blob.data()); }
};

// Compiles the back-projection of one (symbolic) output location over the
// graph's merged-dim view (view.h; `start` forces at least those merges).
// Throws Failure(DG_E_UNSUPPORTED_OP) for reads the view cannot make
// separable and Failure(DG_E_OVERFLOW) if the static path-count bound
// reaches 2^63.  Leaves in the plan have the merged shapes; their ids and
// row order are those of the original shapes.
Plan compile_plan(const GraphIR& g, const DimPartition* start = nullptr);

// Plans of two graphs over the same leaves for a comparison: both view each
// leaf with the same merged dims (the join of what each needs).
void compile_pair_plans(const GraphIR& a, const GraphIR& b, Plan* pa, Plan* pb);

// Local data share bytes one location of this plan needs with a block of
// `nthreads` threads (word_bytes 4: 32-bit ids and counts, 8: 64-bit).
uint32_t plan_lds_bytes(const Plan& p, int nthreads, uint32_t word_bytes = 4);

// Combined per-leaf emission shapes and LDS layout for comparing two plans
// location by location (same leaves in the same order).
void pair_plan(const Plan& a, const Plan& b, int nthreads, dgc::PairPlan* out);

// Expression-DAG program of a graph (DgdHeader and its arrays) for blocks of
// `nthreads` threads.  Throws Failure(DG_E_OVERFLOW) when the element ids of
// all tensors need more than 32 bits and Failure(DG_E_CAPACITY) when a
// frontier bound is unreasonably large.
struct DagProgram {
  std::vector<uint8_t> blob;
  uint32_t lds_bytes = 0;      // LDS area of one location
  uint32_t vars_off = 0;
  int max_vars = 0;
  int64_t max_nodes = 0;       // static bounds for one location
  int64_t max_edges = 0;
  int64_t max_frontier = 0;    // largest frontier capacity (nodes of one op, bound)
  std::vector<uint64_t> gid;   // global id of element 0 per tensor
};
DagProgram compile_dag(const GraphIR& g, int nthreads);

// Text listing of a plan's instructions and leaf terms.
std::string plan_listing(const Plan& p);

}  // namespace dg
