// Host emulation of the device kernels, for CPU tests only.
//
// Runs the same per-location plan (compile.cpp) and the same block code
// (core.h) with a block of one thread on the host, so the compiler and the
// kernel logic can be checked against the oracle without a GPU.  The
// library's entry points never call this; it is built as a separate test
// library.
#include <cstdint>
#include <cstring>
#include <cstdlib>
#include <string>
#include <vector>

#include "../../include/dirigo_rocm.h"
#include "compile.h"
#include "core.h"
#include "dag_core.h"
#include "graph.h"
#include "jit.h"

namespace {

struct HostCtx {
  int tid() const { return 0; }
  int nthreads() const { return 1; }
  int lane() const { return 0; }
  int lanes() const { return 1; }
  int wave() const { return 0; }
  int nwaves() const { return 1; }
  void wave_sync() const {}
  uint32_t wave_prefix(bool f, uint32_t* total) const {
    *total = f ? 1u : 0u;
    return 0u;
  }
  uint64_t scan_add(uint64_t v, uint64_t* total) const {
    *total = v;
    return 0u;
  }
  uint64_t ballot(bool f) const { return f ? 1u : 0u; }
  uint32_t bcast(uint32_t v, int) const { return v; }
  void atomic_or32(uint32_t* p, uint32_t v) const { *p |= v; }
  void reduce_min32(uint32_t* p, uint32_t v) const {
    if (v < *p) *p = v;
  }
  void reduce_max32(uint32_t* p, uint32_t v) const {
    if (v > *p) *p = v;
  }
  uint64_t wave_sum64(uint64_t v) const { return v; }
  uint32_t wave_scan(uint32_t v, uint32_t* total) const {
    *total = v;
    return 0u;
  }
  void sync() const {}
  void atomic_add(uint64_t* p, uint64_t v) const { *p += v; }
  void atomic_max(uint64_t* p, uint64_t v) const {
    if (v > *p) *p = v;
  }
  uint32_t atomic_inc(uint32_t* p) const { return (*p)++; }
  void store(uint32_t* p, uint32_t v) const { *p = v; }
  void store_cached(uint32_t* p, uint32_t v) const { *p = v; }
  void store2(uint32_t* p, uint32_t a, uint32_t b) const {
    p[0] = a;
    p[1] = b;
  }
  void store3(uint32_t* p, uint32_t a, uint32_t b, uint32_t c) const {
    p[0] = a;
    p[1] = b;
    p[2] = c;
  }
  void store(uint64_t* p, uint64_t v) const { *p = v; }
  void reduce_add(uint64_t* p, uint64_t v) const { *p += v; }
  void reduce_max(uint64_t* p, uint64_t v) const {
    if (v > *p) *p = v;
  }
  uint32_t prefix(bool f, uint32_t* total) const {
    *total = f ? 1u : 0u;
    return 0u;
  }
  bool any(bool f) const { return f; }
  int first(bool f) const { return f ? 0 : -1; }
};

thread_local std::string g_err;

int fail_with(const dg::Failure& e) {
  g_err = e.what();
  return e.code;
}

int bits_status(uint32_t bits) {
  if (bits & DGP_ERR_RANGE) { g_err = "location out of range"; return DG_E_RANGE; }
  if (bits & DGP_ERR_OVERFLOW) { g_err = "path count overflow"; return DG_E_OVERFLOW; }
  if (bits & DGP_ERR_CAPACITY) { g_err = "capacity exceeded"; return DG_E_CAPACITY; }
  if (bits & DGP_ERR_SIZE) { g_err = "row size mismatch"; return DG_E_INVALID_ARG; }
  return 0;
}

}  // namespace

extern "C" {

const char* dgh_error(void) { return g_err.c_str(); }

// Row sizes into offsets[0..n] (running totals).
int dgh_sizes(const char* text, int64_t len, const int64_t* locs, int64_t n, int64_t* offsets) {
  try {
    dg::GraphIR ir = dg::parse_dgir(std::string(text, (size_t)len));
    dg::Plan plan = dg::compile_plan(ir);
    std::vector<uint64_t> area((dg::plan_lds_bytes(plan, 1) + 7) / 8 + 1);
    HostCtx c;
    uint32_t err = 0;
    offsets[0] = 0;
    for (int64_t i = 0; i < n; ++i) {
      std::memset(area.data(), 0xA5, area.size() * 8);  // no reliance on zeroed LDS
      uint64_t r = dgc::location_row<HostCtx, dgc::EMIT_COUNT>(c, plan.blob.data(), locs[i],
                                                               reinterpret_cast<uint8_t*>(area.data()), nullptr,
                                                               nullptr, 0, &err);
      offsets[i + 1] = offsets[i] + (int64_t)r;
    }
    return bits_status(err);
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

int dgh_fill(const char* text, int64_t len, const int64_t* locs, int64_t n, const int64_t* offsets, uint32_t* ids,
             uint32_t* cnt) {
  try {
    dg::GraphIR ir = dg::parse_dgir(std::string(text, (size_t)len));
    dg::Plan plan = dg::compile_plan(ir);
    std::vector<uint64_t> area((dg::plan_lds_bytes(plan, 1) + 7) / 8 + 1);
    HostCtx c;
    uint32_t err = 0;
    for (int64_t i = 0; i < n; ++i) {
      std::memset(area.data(), 0x5A, area.size() * 8);
      uint64_t r = dgc::location_row<HostCtx, dgc::EMIT_FILL>(c, plan.blob.data(), locs[i],
                                                              reinterpret_cast<uint8_t*>(area.data()),
                                                              ids + offsets[i], cnt + offsets[i],
                                                              (uint64_t)(offsets[i + 1] - offsets[i]), &err);
      if ((int64_t)r != offsets[i + 1] - offsets[i]) err |= DGP_ERR_SIZE;
    }
    return bits_status(err);
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

int dgh_compare(const char* ta, int64_t la, const char* tb, int64_t lb, const int64_t* locs, int64_t n,
                uint8_t* status) {
  try {
    dg::GraphIR ia = dg::parse_dgir(std::string(ta, (size_t)la));
    dg::GraphIR ib = dg::parse_dgir(std::string(tb, (size_t)lb));
    dg::Plan pa, pb;
    dg::compile_pair_plans(ia, ib, &pa, &pb);
    dgc::PairPlan pp;
    dg::pair_plan(pa, pb, 1, &pp);
    std::vector<uint64_t> area(pp.lds_bytes / 8 + 1);
    HostCtx c;
    uint32_t err = 0;
    for (int64_t i = 0; i < n; ++i) {
      std::memset(area.data(), 0x33, area.size() * 8);
      status[i] = (uint8_t)dgc::location_compare(c, pa.blob.data(), pb.blob.data(), &pp, locs[i],
                                                 reinterpret_cast<uint8_t*>(area.data()), &err);
    }
    return bits_status(err);
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

// Source of the specialised kernels of a graph (for tests and tuning).
int dgh_jit_source(const char* text, int64_t len, int block, char* out, int64_t cap) {
  try {
    dg::GraphIR ir = dg::parse_dgir(std::string(text, (size_t)len));
    dg::Plan plan = dg::compile_plan(ir);
    std::string s = dg::jit_enum_source(plan, block);
    snprintf(out, (size_t)cap, "%s", s.c_str());
    return (int)s.size();
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

// Expression DAGs: node and edge counts as running totals (n + 1 entries
// each), then the DAGs themselves (as the device's dg_dag_sizes / dg_dag_fill).
int dgh_dag_sizes(const char* text, int64_t len, const int64_t* locs, int64_t n, int64_t* node_off,
                  int64_t* edge_off) {
  try {
    dg::GraphIR ir = dg::parse_dgir(std::string(text, (size_t)len));
    dg::DagProgram p = dg::compile_dag(ir, 1);
    std::vector<uint64_t> area(p.lds_bytes / 8 + 1);
    HostCtx c;
    uint32_t err = 0;
    node_off[0] = edge_off[0] = 0;
    dgc::DagOut o{nullptr, nullptr, nullptr, nullptr, 0, 0};
    for (int64_t i = 0; i < n; ++i) {
      std::memset(area.data(), 0xA5, area.size() * 8);
      uint64_t nn = 0, ne = 0;
      dgc::location_dag<HostCtx, dgc::DAG_COUNT>(c, p.blob.data(), locs[i], reinterpret_cast<uint8_t*>(area.data()),
                                                 o, &nn, &ne, &err);
      node_off[i + 1] = node_off[i] + (int64_t)nn;
      edge_off[i + 1] = edge_off[i] + (int64_t)ne;
    }
    return bits_status(err);
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

int dgh_dag_fill(const char* text, int64_t len, const int64_t* locs, int64_t n, const int64_t* node_off,
                 const int64_t* edge_off, uint32_t* nodes, uint32_t* node_edge, uint32_t* edges, uint32_t* mults) {
  try {
    dg::GraphIR ir = dg::parse_dgir(std::string(text, (size_t)len));
    dg::DagProgram p = dg::compile_dag(ir, 1);
    std::vector<uint64_t> area(p.lds_bytes / 8 + 1);
    HostCtx c;
    uint32_t err = 0;
    for (int64_t i = 0; i < n; ++i) {
      std::memset(area.data(), 0x5A, area.size() * 8);
      dgc::DagOut o{nodes + node_off[i], node_edge + node_off[i], edges + edge_off[i], mults + edge_off[i],
                    (uint64_t)(node_off[i + 1] - node_off[i]), (uint64_t)(edge_off[i + 1] - edge_off[i])};
      uint64_t nn = 0, ne = 0;
      dgc::location_dag<HostCtx, dgc::DAG_FILL>(c, p.blob.data(), locs[i], reinterpret_cast<uint8_t*>(area.data()),
                                                o, &nn, &ne, &err);
      if ((int64_t)nn != node_off[i + 1] - node_off[i] || (int64_t)ne != edge_off[i + 1] - edge_off[i])
        err |= DGP_ERR_SIZE;
    }
    return bits_status(err);
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

// How the DAG program takes each read group: per group, four int32 values
// (op index, 1 if the op is pointwise, 1 if the group is taken per variable,
// the number of list variables).  Returns the group count (at most cap are
// written) or a negative status.
// The frontier dedup over a tensor of the given shape: cand[0..n) made
// sorted and unique in place through the bounding-box bitmap with ws_words
// words of scratch; returns the number kept, or -1 when the bitmap does not
// apply (cand untouched).
int64_t dgh_box_unique(int rank, const int64_t* shape, uint32_t* cand, uint32_t n, uint32_t ws_words) {
  DgdTensor X;
  std::memset(&X, 0, sizeof(X));
  X.rank = rank;
  uint64_t st = 1;
  for (int d = rank - 1; d >= 0; --d) {
    X.shape[d] = (int32_t)shape[d];
    X.stride[d] = (uint32_t)st;
    X.magic[d] = shape[d] <= 1 ? 0 : ~0ull / (uint64_t)shape[d] + 1;
    st *= (uint64_t)shape[d];
  }
  std::vector<uint32_t> ws(ws_words + 1);
  HostCtx c;
  const uint32_t k = dgc::box_unique(c, X, cand, n, ws.data(), ws_words);
  return k == ~0u ? -1 : (int64_t)k;
}

int dgh_dag_groups(const char* text, int64_t len, int32_t* out, int64_t cap) {
  try {
    dg::GraphIR ir = dg::parse_dgir(std::string(text, (size_t)len));
    dg::DagProgram p = dg::compile_dag(ir, 64);
    const DgdHeader* h = reinterpret_cast<const DgdHeader*>(p.blob.data());
    const DgdOp* O = reinterpret_cast<const DgdOp*>(p.blob.data() + h->op_off);
    const DgdGroup* G = reinterpret_cast<const DgdGroup*>(p.blob.data() + h->group_off);
    int64_t k = 0;
    for (int o = 0; o < h->nop; ++o)
      for (int q = 0; q < O[o].ng; ++q, ++k) {
        if (k >= cap) continue;
        const DgdGroup& g = G[O[o].g0 + q];
        int lists = 0;  // variables with an exact division (progression step > 1)
        for (int v = 0; v < g.nwin; ++v) lists += g.fast && g.mpair[v] >= 0 ? 1 : 0;
        out[4 * k] = o;
        out[4 * k + 1] = O[o].pointwise;
        out[4 * k + 2] = g.fast;
        out[4 * k + 3] = lists;
      }
    return (int)k;
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

// Static bounds of a graph's DAG program for blocks of `block` threads:
// out = {nodes, edges, largest frontier, LDS bytes} of one location.
int dgh_dag_bounds(const char* text, int64_t len, int block, int64_t* out) {
  try {
    dg::GraphIR ir = dg::parse_dgir(std::string(text, (size_t)len));
    dg::DagProgram p = dg::compile_dag(ir, block);
    out[0] = p.max_nodes;
    out[1] = p.max_edges;
    out[2] = p.max_frontier;
    out[3] = (int64_t)p.lds_bytes;
    return 0;
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

// Source of the specialised expression-DAG kernels of a graph (its DAG
// program for blocks of `block` threads).
int dgh_jit_dag_source(const char* text, int64_t len, int block, char* out, int64_t cap) {
  try {
    dg::GraphIR ir = dg::parse_dgir(std::string(text, (size_t)len));
    dg::DagProgram p = dg::compile_dag(ir, block);
    std::string s = dg::jit_dag_source(p, block);
    snprintf(out, (size_t)cap, "%s", s.c_str());
    return (int)s.size();
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

// Source of the specialised 64-bit enumeration kernel of a graph.
int dgh_jit_wide_source(const char* text, int64_t len, int block, char* out, int64_t cap) {
  try {
    dg::GraphIR ir = dg::parse_dgir(std::string(text, (size_t)len));
    dg::Plan plan = dg::compile_plan(ir);
    std::string s = dg::jit_wide_source(plan, block);
    snprintf(out, (size_t)cap, "%s", s.c_str());
    return (int)s.size();
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

// Source of the specialised comparison kernel of a pair of graphs.
int dgh_jit_compare_source(const char* ta, int64_t la, const char* tb, int64_t lb, int block, char* out,
                           int64_t cap) {
  try {
    dg::GraphIR ia = dg::parse_dgir(std::string(ta, (size_t)la));
    dg::GraphIR ib = dg::parse_dgir(std::string(tb, (size_t)lb));
    dg::Plan pa, pb;
    dg::compile_pair_plans(ia, ib, &pa, &pb);
    dgc::PairPlan pp;
    dg::pair_plan(pa, pb, block, &pp);
    std::string s = dg::jit_compare_source(pa, pb, pp, block);
    snprintf(out, (size_t)cap, "%s", s.c_str());
    return (int)s.size();
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

// hipRTC options of the specialised kernels, space separated.
int dgh_jit_options(char* out, int64_t cap) {
  std::string s;
  for (const char* const* o = dg::jit_compile_options(); *o; ++o) s += std::string(s.empty() ? "" : " ") + *o;
  snprintf(out, (size_t)cap, "%s", s.c_str());
  return (int)s.size();
}

// Human-readable listing of a graph's compiled plan (for tests and tuning).
int dgh_dump(const char* text, int64_t len, char* out, int64_t cap) {
  try {
    dg::GraphIR ir = dg::parse_dgir(std::string(text, (size_t)len));
    dg::Plan plan = dg::compile_plan(ir);
    std::string s = dg::plan_listing(plan);
    snprintf(out, (size_t)cap, "%s", s.c_str());
    return (int)s.size();
  } catch (const dg::Failure& e) {
    return fail_with(e);
  }
}

}  // extern "C"
