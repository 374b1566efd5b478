// C ABI of libdirigo_rocm (declared in include/dirigo_rocm.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <tuple>
#include <vector>
#include <cstring>
#include <map>
#include <memory>
#include <cstdlib>
#include <mutex>
#include <new>
#include <string>

#include "../../include/dirigo_rocm.h"
#include "compile.h"
#include "graph.h"
#include "jit.h"
#include "kernels.h"
#include "order.h"
#include "merge.h"

// Specialised kernels of a graph on one device.
struct DevKernels {
  bool tried = false;
  bool ok = false;
  dg::JitModule jm;
  std::string log;
};

struct dg_graph {
  dg::GraphIR ir;
  dg::Plan plan;
  int block = 64;
  uint32_t lds = 0;
  std::mutex mu;
  std::map<int, uint8_t*> dev_blob;  // compiled plan per device
  std::map<int, DevKernels> jit;     // specialised kernels per device
  std::map<int, DevKernels> jit_wide;  // specialised 64-bit enumeration per device
  uint32_t lds_wide = 0;             // LDS per location with 64-bit ids and counts
  uint64_t serial = 0;               // unique per graph in the process
  // Expression-DAG program, compiled on first use (dag_status: DG_OK or
  // the failure, with its message).
  bool dag_tried = false;
  dg_status dag_status = DG_OK;
  std::string dag_error;
  dg::DagProgram dag;
  int dag_block = 256;
  std::map<int, uint8_t*> dev_dag;  // DAG program per device
  std::map<int, DevKernels> jit_dag;  // specialised DAG kernels per device
};

namespace {

thread_local std::string g_last_error;

// Specialised comparison kernels of graph pairs: (serial of a, serial of b,
// device, block) -> kernels.  Released when either graph is destroyed.
// Each entry has its own lock, so that different pairs compile at once.
struct PairKernels {
  std::mutex mu;
  DevKernels k;
};
std::mutex g_pair_mu;
std::map<std::tuple<uint64_t, uint64_t, int, int>, std::shared_ptr<PairKernels>> g_pair_jit;

// Plans of a pair whose graphs view some leaf with different merged dims
// (each graph's own plan is then not comparable with the other's): both
// recompiled over the joint view, with their device copies per device.
struct PairPlans {
  dg::Plan a, b;
  std::map<int, std::pair<uint8_t*, uint8_t*>> dev;
};
std::map<std::pair<uint64_t, uint64_t>, PairPlans> g_pair_plans;  // under g_pair_mu

// Most locations one call takes (the helper kernels run flat grids of one
// thread per location).
constexpr int64_t kMaxLocations = int64_t(1) << 31;

dg_status set_error(dg_status code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

dg_status hip_error(hipError_t e, const char* where) {
  return set_error(DG_E_HIP, std::string(where) + ": " + hipGetErrorString(e));
}

#define DG_HIP(call, where)              \
  do {                                   \
    hipError_t e_ = (call);              \
    if (e_ != hipSuccess) return hip_error(e_, where); \
  } while (0)

int max_lds_per_block() {
  int dev = 0, v = 65536;
  if (hipGetDevice(&dev) == hipSuccess) {
    int x = 0;
    if (hipDeviceGetAttribute(&x, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess && x > 0) v = x;
  }
  return v;
}

// Finishes a freshly parsed graph: compile, pick the block size and the LDS
// footprint of one location.
dg_status finalize(dg_graph* g) {
  static std::atomic<uint64_t> next_serial{1};
  g->serial = next_serial++;
  g->plan = dg::compile_plan(g->ir);
  g->block = g->plan.max_row_size >= 4096 ? 256 : 64;
  // Tuning override of the block size (specialised kernels only).
  if (const char* e = std::getenv("DIRIGO_BLOCK")) {
    const int b = std::atoi(e);
    if (b == 64 || b == 128 || b == 256 || b == 512 || b == 1024) g->block = b;
  }
  g->lds = dg::plan_lds_bytes(g->plan, g->block);
  g->lds_wide = dg::plan_lds_bytes(g->plan, g->block, 8);
  return DG_OK;
}

dg_status device_blob(const dg_graph* cg, const uint8_t** out) {
  dg_graph* g = const_cast<dg_graph*>(cg);
  int dev = 0;
  DG_HIP(hipGetDevice(&dev), "hipGetDevice");
  std::lock_guard<std::mutex> lock(g->mu);
  auto it = g->dev_blob.find(dev);
  if (it != g->dev_blob.end()) {
    *out = it->second;
    return DG_OK;
  }
  void* p = nullptr;
  const size_t bytes = g->plan.blob.size();
  DG_HIP(hipMalloc(&p, bytes), "hipMalloc(plan)");
  hipError_t e = hipMemcpy(p, g->plan.blob.data(), bytes, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(p);
    return hip_error(e, "hipMemcpy(plan)");
  }
  g->dev_blob[dev] = static_cast<uint8_t*>(p);
  *out = static_cast<uint8_t*>(p);
  return DG_OK;
}

// The graph's expression-DAG program (compiled on first use) and its device
// copy on the current device.
dg_status dag_program(const dg_graph* cg, const uint8_t** out) {
  dg_graph* g = const_cast<dg_graph*>(cg);
  std::lock_guard<std::mutex> lock(g->mu);
  if (!g->dag_tried) {
    g->dag_tried = true;
    try {
      // Small DAGs (a few thousand references per location) run on one wave.
      dg::DagProgram probe = dg::compile_dag(g->ir, 64);
      // Four waves when some op has more than four waves' worth of nodes
      // (the batches of nodes then run side by side) and the DAG is large;
      // one wave otherwise (its barriers are nearly free).
      g->dag_block = probe.max_edges >= 4096 && probe.max_frontier > 256 ? 256 : 64;
      g->dag = g->dag_block == 64 ? std::move(probe) : dg::compile_dag(g->ir, g->dag_block);
    } catch (const dg::Failure& f) {
      g->dag_status = (dg_status)f.code;
      g->dag_error = f.what();
    }
  }
  if (g->dag_status != DG_OK) return set_error(g->dag_status, g->dag_error);
  if (!out) return DG_OK;
  int dev = 0;
  DG_HIP(hipGetDevice(&dev), "hipGetDevice");
  auto it = g->dev_dag.find(dev);
  if (it != g->dev_dag.end()) {
    *out = it->second;
    return DG_OK;
  }
  void* p = nullptr;
  const size_t bytes = g->dag.blob.size();
  DG_HIP(hipMalloc(&p, bytes), "hipMalloc(DAG program)");
  hipError_t e = hipMemcpy(p, g->dag.blob.data(), bytes, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(p);
    return hip_error(e, "hipMemcpy(DAG program)");
  }
  g->dev_dag[dev] = static_cast<uint8_t*>(p);
  *out = static_cast<uint8_t*>(p);
  return DG_OK;
}

// The graph's specialised kernels on the current device, compiled on first
// use; nullptr when specialisation is off or failed (the precompiled
// kernels then run the plan).
const dg::JitModule* graph_jit(const dg_graph* cg) {
  if (!dg::jit_enabled()) return nullptr;
  dg_graph* g = const_cast<dg_graph*>(cg);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  std::lock_guard<std::mutex> lock(g->mu);
  DevKernels& k = g->jit[dev];
  if (!k.tried) {
    k.tried = true;
    k.ok = dg::jit_load(dg::jit_enum_source(g->plan, g->block), &k.jm, &k.log) && k.jm.sizes && k.jm.fill &&
           k.jm.enumerate;
  }
  return k.ok ? &k.jm : nullptr;
}

// Specialised comparison kernel of the pair (a, b) on the current device;
// nullptr when specialisation is off or failed.
const dg::JitModule* pair_jit(const dg_graph* ca, const dg_graph* b, const dg::Plan& plan_a, const dg::Plan& plan_b,
                              const dgc::PairPlan& pp, int block) {
  if (!dg::jit_enabled()) return nullptr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  std::shared_ptr<PairKernels> e;
  {
    std::lock_guard<std::mutex> lock(g_pair_mu);
    auto& slot = g_pair_jit[std::make_tuple(ca->serial, b->serial, dev, block)];
    if (!slot) slot = std::make_shared<PairKernels>();
    e = slot;
  }
  std::lock_guard<std::mutex> lock(e->mu);
  DevKernels& k = e->k;
  if (!k.tried) {
    k.tried = true;
    k.ok = dg::jit_load(dg::jit_compare_source(plan_a, plan_b, pp, block), &k.jm, &k.log) && k.jm.compare;
  }
  return k.ok ? &k.jm : nullptr;
}

// Specialised 64-bit enumeration kernel of g on the current device, or null.
const dg::JitModule* graph_jit_wide(const dg_graph* cg) {
  if (!dg::jit_enabled()) return nullptr;
  dg_graph* g = const_cast<dg_graph*>(cg);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  std::lock_guard<std::mutex> lock(g->mu);
  DevKernels& k = g->jit_wide[dev];
  if (!k.tried) {
    k.tried = true;
    k.ok = dg::jit_load(dg::jit_wide_source(g->plan, g->block), &k.jm, &k.log) && k.jm.enumerate_wide;
  }
  return k.ok ? &k.jm : nullptr;
}

// Calls whose static edge bound (locations times the per-location bound)
// reaches this many edges take the specialised DAG kernels by default:
// below it the compile time (seconds, once per graph and device) outweighs
// the gain.  Both passes gain from them: the sizes pass most (its per-op
// and per-group bookkeeping folds into constants), the fill by a few per
// cent for DAGs of millions of edges per location (timed against the
// precompiled fill in the same processes) up to 3.4x for small ones.
constexpr double kDagJitEdges = double(1 << 26);

// The specialised DAG kernels of g on the current device for a call over n
// locations, compiled on first use; nullptr when the precompiled kernels
// run the call: specialisation off or failed, a call below kDagJitEdges,
// or more than 64 KiB of LDS per location.  DIRIGO_DAG_JIT=1 specialises
// every call, DIRIGO_DAG_JIT=0 none.  The DAG program must be compiled.
const dg::JitModule* dag_jit(const dg_graph* cg, int64_t n) {
  if (!dg::jit_enabled()) return nullptr;
  dg_graph* g = const_cast<dg_graph*>(cg);
  const char* env = std::getenv("DIRIGO_DAG_JIT");
  const int mode = env && env[0] == '1' ? 1 : env && env[0] == '0' ? 0 : -1;
  if (mode == 0 || g->dag.lds_bytes > 65536u) return nullptr;
  if (mode < 0 && (double)n * (double)g->dag.max_edges < kDagJitEdges) return nullptr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  std::lock_guard<std::mutex> lock(g->mu);
  DevKernels& k = g->jit_dag[dev];
  if (!k.tried) {
    k.tried = true;
    k.ok = dg::jit_load(dg::jit_dag_source(g->dag, g->dag_block), &k.jm, &k.log) && k.jm.dag_sizes && k.jm.dag_fill;
  }
  return k.ok ? &k.jm : nullptr;
}

// Consecutive locations per block of the DAG sizes and fill kernels: 8 for
// small DAGs in one-wave blocks (at most 4,096 edges per location, static
// bound), whose one-block rows are too short for a block's start and end to
// vanish beside its writes (a plain writer of 4.6 KB rows in two arrays,
// the size of a 3x3, 64-channel conv2d node's DAG: 3.7 TB/s with one row per
// block, 5.0 with 8), else 1.
int dag_per_block(const dg_graph* g) { return g->dag_block == 64 && g->dag.max_edges <= 4096 ? 8 : 1; }

// Leaf ids of g fit 32 bits.
bool narrow_ids(const dg_graph* g) { return g->ir.leaf_total <= 0xFFFFFFFFull; }

// What an allocation-free call may use on the current device: the plan's
// device copy and the specialised kernels, only if an earlier call put them
// there (DG_E_INVALID_ARG otherwise).  *jm is null when specialisation is
// off or failed (the precompiled kernels then run the plan).
dg_status resident(const dg_graph* cg, bool wide, const uint8_t** blob, const dg::JitModule** jm) {
  dg_graph* g = const_cast<dg_graph*>(cg);
  int dev = 0;
  DG_HIP(hipGetDevice(&dev), "hipGetDevice");
  std::lock_guard<std::mutex> lock(g->mu);
  auto b = g->dev_blob.find(dev);
  if (b == g->dev_blob.end())
    return set_error(DG_E_INVALID_ARG, "the graph is not resident on this device: make one ordinary enumeration "
                                       "call with it on this device first");
  *blob = b->second;
  *jm = nullptr;
  if (dg::jit_enabled()) {
    auto& tab = wide ? g->jit_wide : g->jit;
    auto k = tab.find(dev);
    if (k == tab.end() || !k->second.tried)
      return set_error(DG_E_INVALID_ARG, "the graph's kernels are not loaded on this device: make one ordinary "
                                         "enumeration call with it on this device first");
    if (k->second.ok) *jm = &k->second.jm;
  }
  return DG_OK;
}

// One block per location, in launches of at most kGridLimit / block blocks
// (a grid holds fewer than 2^32 work-items per dimension).  launch(first,
// m) launches blocks for locations first .. first + m - 1.
constexpr int64_t kGridLimit = (int64_t(1) << 32) - 1;

template <class F>
hipError_t per_location(int64_t n, int block, F launch) {
  const int64_t step = kGridLimit / block;
  for (int64_t first = 0; first < n; first += step) {
    hipError_t e = launch(first, std::min(step, n - first));
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// The locations of src from position `first` on.
dgc::LocSrc shifted(dgc::LocSrc src, int64_t first) {
  return src.locs ? dgc::LocSrc{src.locs + first, 0} : dgc::LocSrc{nullptr, src.first + first};
}

hipError_t launch_module(hipFunction_t f, int64_t n, int block, uint32_t lds, hipStream_t s, void** args) {
  if (n <= 0) return hipSuccess;
  if (n > kGridLimit / block) return hipErrorInvalidConfiguration;
  return hipModuleLaunchKernel(f, (unsigned)n, 1, 1, (unsigned)block, 1, 1, lds, s, args, nullptr);
}

// The fill kernel of g (specialised or precompiled): rows of the n
// locations of src at [offsets[i] - base, offsets[i+1] - base).
hipError_t fill_launch(const dg_graph* g, const uint8_t* blob, dgc::LocSrc src, int64_t n, const int64_t* offsets,
                       int64_t base, uint32_t* ids, uint32_t* cnt, uint32_t* err, hipStream_t s) {
  const dg::JitModule* jm = graph_jit(g);
  return per_location(n, g->block, [&](int64_t first, int64_t m) {
    dgc::LocSrc part = shifted(src, first);
    const int64_t* off = offsets + first;
    if (jm) {
      void* args[] = {&part, &m, (void*)&off, &base, &ids, &cnt, &err};
      return launch_module(jm->fill, m, g->block, g->lds, s, args);
    }
    return dgk::launch_fill(blob, part, m, off, base, ids, cnt, err, g->block, g->lds, s);
  });
}

struct WsLayout {
  size_t err, ticket, found, pair, sums, flags, total;
};

// Workspace: error word | comparison pair plan | scan tile sums | flags.
WsLayout ws_layout(int64_t n) {
  WsLayout w;
  w.err = 0;
  w.ticket = 8;
  w.found = 16;
  w.pair = 256;
  w.sums = (w.pair + sizeof(dgc::PairPlan) + 255) & ~size_t(255);
  w.flags = w.sums + 8 * (size_t)dgk::scan_temp_entries(n < 0 ? 0 : n);
  w.flags = (w.flags + 255) & ~size_t(255);
  w.total = w.flags + 8 * (size_t)((n < 0 ? 0 : n) + 1);
  w.total = (w.total + 255) & ~size_t(255);
  return w;
}

// Workspace of the one-pass DAG call: error word | ticket | one status word
// per location for the node counts, then one for the edge counts.
struct DagWsLayout {
  size_t err, ticket, st_nodes, st_edges, total;
};
DagWsLayout dag_ws_layout(int64_t n) {
  const size_t words = (size_t)((n < 0 ? 0 : n) + 1);
  DagWsLayout w;
  w.err = 0;
  w.ticket = 8;
  w.st_nodes = 256;
  w.st_edges = (w.st_nodes + 8 * words + 255) & ~size_t(255);
  w.total = (w.st_edges + 8 * words + 255) & ~size_t(255);
  return w;
}

dg_status device_errors(uint32_t bits) {
  if (bits & DGP_ERR_RANGE) return set_error(DG_E_RANGE, "a location lies outside the output tensor");
  if (bits & DGP_ERR_OVERFLOW) return set_error(DG_E_OVERFLOW, "a path count does not fit 32 bits");
  if (bits & DGP_ERR_CAPACITY)
    return set_error(DG_E_CAPACITY, "a per-location factor outgrew its compiled capacity");
  if (bits & DGP_ERR_SIZE) return set_error(DG_E_INVALID_ARG, "offsets do not match this graph and locations");
  if (bits & DGP_ERR_SHAPE) return set_error(DG_E_HIP, "a specialised DAG kernel lacks code for one of the graph's groups");
  if (bits & DGP_ERR_TIMEOUT) return set_error(DG_E_HIP, "single pass: a predecessor's row size never arrived");
  if (bits & DGP_ERR_BUFFER) return set_error(DG_E_BUFFER, "the rows need more entries than the output buffers hold");
  return DG_OK;
}

template <class F>
dg_status guarded(F f) {
  try {
    return f();
  } catch (const dg::Failure& e) {
    return set_error(e.code, e.what());
  } catch (const std::bad_alloc&) {
    return set_error(DG_E_INVALID_ARG, "out of host memory");
  } catch (const std::exception& e) {
    return set_error(DG_E_INVALID_ARG, e.what());
  }
}

}  // namespace

extern "C" {

const char* dg_last_error(void) { return g_last_error.c_str(); }

dg_status dg_graph_parse(const char* text, size_t len, dg_graph** out) {
  if (!text || !out) return set_error(DG_E_INVALID_ARG, "null argument");
  return guarded([&]() -> dg_status {
    dg_graph* g = new dg_graph;
    try {
      g->ir = dg::parse_dgir(std::string(text, len));
      finalize(g);
    } catch (...) {
      delete g;
      throw;
    }
    *out = g;
    return DG_OK;
  });
}

dg_status dg_graph_build(const dg_tensor_desc* tensors, int32_t nt, const dg_op_desc* ops, int32_t nops,
                         int32_t output_tensor, dg_graph** out) {
  if (!out || nt <= 0 || nops < 0 || !tensors || (nops > 0 && !ops))
    return set_error(DG_E_INVALID_ARG, "bad descriptor arguments");
  return guarded([&]() -> dg_status {
    dg_graph* g = new dg_graph;
    try {
      for (int32_t i = 0; i < nt; ++i) {
        const dg_tensor_desc& t = tensors[i];
        if (!t.name || !t.shape || t.rank <= 0 || t.rank > DG_MAX_RANK)
          throw dg::Failure(DG_E_INVALID_ARG, "bad tensor descriptor " + std::to_string(i));
        dg::add_leaf(g->ir, t.name, dg::Dims(t.shape, t.shape + t.rank));
      }
      for (int32_t i = 0; i < nops; ++i) {
        const dg_op_desc& o = ops[i];
        if (!o.name || !o.kind || o.n_inputs < 0 || (o.n_inputs > 0 && !o.inputs))
          throw dg::Failure(DG_E_INVALID_ARG, "bad op descriptor " + std::to_string(i));
        std::vector<int> in(o.inputs, o.inputs + o.n_inputs);
        for (int t : in)
          if (t < 0 || t >= nt + i) throw dg::Failure(DG_E_INVALID_ARG, "op operand refers to a later tensor");
        dg::add_op(g->ir, o.name, o.kind, in, o.attrs ? o.attrs : "");
      }
      dg::set_output(g->ir, output_tensor, nullptr);
      dg::finish(g->ir);
      finalize(g);
    } catch (...) {
      delete g;
      throw;
    }
    *out = g;
    return DG_OK;
  });
}

void dg_graph_destroy(dg_graph* g) {
  if (!g) return;
  for (auto& kv : g->jit) dg::jit_release(&kv.second.jm);
  for (auto& kv : g->jit_wide) dg::jit_release(&kv.second.jm);
  for (auto& kv : g->jit_dag) dg::jit_release(&kv.second.jm);
  {
    std::lock_guard<std::mutex> lock(g_pair_mu);
    for (auto it = g_pair_jit.begin(); it != g_pair_jit.end();) {
      if (std::get<0>(it->first) == g->serial || std::get<1>(it->first) == g->serial) {
        std::shared_ptr<PairKernels> e = it->second;  // outlives the erase below
        {
          std::lock_guard<std::mutex> el(e->mu);
          dg::jit_release(&e->k.jm);
        }
        it = g_pair_jit.erase(it);
      } else {
        ++it;
      }
    }
    for (auto it = g_pair_plans.begin(); it != g_pair_plans.end();) {
      if (it->first.first == g->serial || it->first.second == g->serial) {
        int cur = 0;
        const bool have = hipGetDevice(&cur) == hipSuccess;
        for (auto& d : it->second.dev)
          if (hipSetDevice(d.first) == hipSuccess) {
            (void)hipFree(d.second.first);
            (void)hipFree(d.second.second);
          }
        if (have) (void)hipSetDevice(cur);
        it = g_pair_plans.erase(it);
      } else {
        ++it;
      }
    }
  }
  int cur = 0;
  bool have = hipGetDevice(&cur) == hipSuccess;
  for (auto& kv : g->dev_blob) {
    if (hipSetDevice(kv.first) == hipSuccess) (void)hipFree(kv.second);
  }
  for (auto& kv : g->dev_dag) {
    if (hipSetDevice(kv.first) == hipSuccess) (void)hipFree(kv.second);
  }
  if (have) (void)hipSetDevice(cur);
  delete g;
}

dg_status dg_graph_info(const dg_graph* g, dg_graph_info_t* out) {
  if (!g || !out) return set_error(DG_E_INVALID_ARG, "null argument");
  std::memset(out, 0, sizeof(*out));
  const dg::Tensor& o = g->ir.tensors[g->ir.output];
  out->n_leaves = (int32_t)g->ir.leaves.size();
  out->output_rank = (int32_t)o.shape.size();
  for (size_t d = 0; d < o.shape.size(); ++d) out->output_shape[d] = o.shape[d];
  out->output_numel = dg::numel(o.shape);
  out->leaf_total = g->ir.leaf_total;
  out->max_row_size = g->plan.max_row_size;
  out->count_bound = g->plan.count_bound;
  out->n_instructions = g->plan.header().ninstr;
  out->lds_bytes = (int32_t)g->lds;
  out->lds_wide_bytes = (int32_t)g->lds_wide;
  out->block_threads = g->block;
  out->max_leaf_terms = g->plan.max_leaf_terms;
  out->n_tensors = (int32_t)g->ir.tensors.size();
  out->specialized = -1;
  if (!dg::jit_enabled()) {
    out->specialized = 0;
  } else {
    int dev = 0;
    if (hipGetDevice(&dev) == hipSuccess) {
      dg_graph* mg = const_cast<dg_graph*>(g);
      std::lock_guard<std::mutex> lock(mg->mu);
      auto it = mg->jit.find(dev);
      if (it != mg->jit.end() && it->second.tried) out->specialized = it->second.ok ? 1 : 0;
    }
  }
  out->dag_specialized = dg::jit_enabled() ? -1 : 0;
  {
    int dev = 0;
    if (hipGetDevice(&dev) == hipSuccess) {
      dg_graph* mg = const_cast<dg_graph*>(g);
      std::lock_guard<std::mutex> lock(mg->mu);
      auto it = mg->jit_dag.find(dev);
      if (it != mg->jit_dag.end() && it->second.tried) out->dag_specialized = it->second.ok ? 1 : 0;
    }
  }
  {
    dg_graph* mg = const_cast<dg_graph*>(g);
    std::lock_guard<std::mutex> lock(mg->mu);
    if (mg->dag_tried && mg->dag_status == DG_OK) {
      out->dag_block_threads = mg->dag_block;
      out->dag_lds_bytes = (int32_t)mg->dag.lds_bytes;
      out->dag_edge_bound = mg->dag.max_edges;
    }
  }
  return DG_OK;
}

dg_status dg_graph_leaf(const dg_graph* g, int32_t i, dg_leaf_info_t* out) {
  if (!g || !out) return set_error(DG_E_INVALID_ARG, "null argument");
  if (i < 0 || i >= (int32_t)g->ir.leaves.size()) return set_error(DG_E_INVALID_ARG, "leaf index out of range");
  std::memset(out, 0, sizeof(*out));
  const dg::Tensor& t = g->ir.tensors[g->ir.leaves[i]];
  std::snprintf(out->name, DG_NAME_LEN, "%s", t.name.c_str());
  out->rank = (int32_t)t.shape.size();
  for (size_t d = 0; d < t.shape.size(); ++d) out->shape[d] = t.shape[d];
  out->base = t.base;
  out->numel = dg::numel(t.shape);
  return DG_OK;
}

dg_status dg_graph_tensor(const dg_graph* g, int32_t i, dg_tensor_info_t* out) {
  if (!g || !out) return set_error(DG_E_INVALID_ARG, "null argument");
  if (i < 0 || i >= (int32_t)g->ir.tensors.size()) return set_error(DG_E_INVALID_ARG, "tensor index out of range");
  std::memset(out, 0, sizeof(*out));
  const dg::Tensor& t = g->ir.tensors[i];
  std::snprintf(out->name, DG_NAME_LEN, "%s", t.name.c_str());
  out->rank = (int32_t)t.shape.size();
  for (size_t d = 0; d < t.shape.size(); ++d) out->shape[d] = t.shape[d];
  out->numel = dg::numel(t.shape);
  out->leaf = t.leaf;
  out->producer = t.producer;
  if (t.producer >= 0) std::snprintf(out->kind, sizeof(out->kind), "%s", g->ir.ops[t.producer].kind.c_str());
  // Global id of element 0: leaves keep theirs, op outputs follow all leaves
  // in SSA order.
  uint64_t gid = g->ir.leaf_total;
  if (t.leaf >= 0) {
    gid = t.base;
  } else {
    for (int k = 0; k < t.producer; ++k) gid += (uint64_t)dg::numel(g->ir.tensors[g->ir.ops[k].out].shape);
  }
  out->gid = gid;
  return DG_OK;
}

dg_status dg_workspace_size(const dg_graph* g, int64_t n_locs, size_t* bytes) {
  if (!g || !bytes || n_locs < 0) return set_error(DG_E_INVALID_ARG, "bad argument");
  *bytes = std::max(ws_layout(n_locs).total, dag_ws_layout(n_locs).total);
  return DG_OK;
}

namespace {

// Row sizes and offsets of the locations of `src` (synchronous).
dg_status sizes_impl(const dg_graph* g, dgc::LocSrc src, int64_t n, int64_t* d_offsets, void* d_ws,
                     int64_t* h_total, hipStream_t s) {
  if (!d_ws) return set_error(DG_E_WORKSPACE, "workspace is required");
  if (g->lds > (uint32_t)max_lds_per_block())
    return set_error(DG_E_CAPACITY, "one location needs " + std::to_string(g->lds) + " bytes of LDS");
  const uint8_t* blob = nullptr;
  dg_status st = device_blob(g, &blob);
  if (st != DG_OK) return st;
  WsLayout w = ws_layout(n);
  uint8_t* ws = static_cast<uint8_t*>(d_ws);
  uint32_t* err = reinterpret_cast<uint32_t*>(ws + w.err);
  DG_HIP(dgk::launch_zero(err, s), "zero");
  const dg::JitModule* jm = graph_jit(g);
  DG_HIP(per_location(n, g->block,
                      [&](int64_t first, int64_t m) {
                        dgc::LocSrc part = shifted(src, first);
                        int64_t* off = d_offsets + first;
                        if (jm) {
                          void* args[] = {&part, &m, &off, &err};
                          return launch_module(jm->sizes, m, g->block, g->lds, s, args);
                        }
                        return dgk::launch_sizes(blob, part, m, off, err, g->block, g->lds, s);
                      }),
         "sizes kernel");
  DG_HIP(dgk::launch_scan(d_offsets, n, reinterpret_cast<int64_t*>(ws + w.sums), s), "scan");
  int64_t total = 0;
  uint32_t bits = 0;
  DG_HIP(hipMemcpyAsync(&total, d_offsets + n, sizeof(int64_t), hipMemcpyDeviceToHost, s), "copy total");
  DG_HIP(hipMemcpyAsync(&bits, err, sizeof(uint32_t), hipMemcpyDeviceToHost, s), "copy flags");
  DG_HIP(hipStreamSynchronize(s), "sizes sync");
  st = device_errors(bits);
  if (st != DG_OK) return st;
  *h_total = total;
  return DG_OK;
}

}  // namespace

dg_status dg_enumerate_sizes(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_offsets, void* d_ws,
                             int64_t* h_total, void* stream) {
  if (!g || !d_offsets || !h_total || n < 0 || n > kMaxLocations || (n > 0 && !d_locs)) return set_error(DG_E_INVALID_ARG, "bad argument");
  return sizes_impl(g, dgc::LocSrc{d_locs, 0}, n, d_offsets, d_ws, h_total, static_cast<hipStream_t>(stream));
}

dg_status dg_enumerate_fill(const dg_graph* g, const int64_t* d_locs, int64_t n, const int64_t* d_offsets,
                            uint32_t* d_ids, uint32_t* d_counts, void* d_ws, void* stream) {
  if (!g || n < 0 || n > kMaxLocations || (n > 0 && (!d_locs || !d_offsets || !d_ids || !d_counts)))
    return set_error(DG_E_INVALID_ARG, "bad argument");
  if (!d_ws) return set_error(DG_E_WORKSPACE, "workspace is required");
  if (!narrow_ids(g)) return set_error(DG_E_OVERFLOW, "leaf ids need 64 bits: use dg_enumerate_wide");
  if (n == 0) return DG_OK;
  if (g->lds > (uint32_t)max_lds_per_block())
    return set_error(DG_E_CAPACITY, "one location needs " + std::to_string(g->lds) + " bytes of LDS");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint8_t* blob = nullptr;
  dg_status st = device_blob(g, &blob);
  if (st != DG_OK) return st;
  uint32_t* err = reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(d_ws) + ws_layout(n).err);
  DG_HIP(dgk::launch_zero(err, s), "zero");
  DG_HIP(fill_launch(g, blob, dgc::LocSrc{d_locs, 0}, n, d_offsets, 0, d_ids, d_counts, err, s), "fill kernel");
  return DG_OK;
}

namespace {

// Single pass over the locations of `src` (a list or a flat range), with
// 32-bit (Word = uint32_t) or 64-bit ids and counts.
// With `no_alloc`, only what resident() allows is used: the call allocates
// nothing and loads nothing.
extern "C++" template <class Word>
dg_status enumerate_impl(const dg_graph* g, dgc::LocSrc src, int64_t n, int64_t* d_offsets, Word* d_ids,
                         Word* d_counts, int64_t capacity, void* d_ws, int64_t* h_total, void* stream,
                         bool no_alloc = false) {
  constexpr bool wide = sizeof(Word) == 8;
  if (!d_ws) return set_error(DG_E_WORKSPACE, "workspace is required");
  if (!wide && !narrow_ids(g))
    return set_error(DG_E_OVERFLOW, "leaf ids need 64 bits: use dg_enumerate_wide");
  const uint32_t lds = wide ? g->lds_wide : g->lds;
  if (lds > (uint32_t)max_lds_per_block())
    return set_error(DG_E_CAPACITY, "one location needs " + std::to_string(lds) + " bytes of LDS");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (n == 0) {
    DG_HIP(dgk::launch_scan(d_offsets, 0, nullptr, s), "offsets");
    DG_HIP(hipStreamSynchronize(s), "sync");
    *h_total = 0;
    return DG_OK;
  }
  const uint8_t* blob = nullptr;
  const dg::JitModule* jm = nullptr;
  if (no_alloc) {
    dg_status st = resident(g, wide, &blob, &jm);
    if (st != DG_OK) return st;
  } else {
    dg_status st = device_blob(g, &blob);
    if (st != DG_OK) return st;
    jm = wide ? graph_jit_wide(g) : graph_jit(g);
  }
  WsLayout w = ws_layout(n);
  uint8_t* ws = static_cast<uint8_t*>(d_ws);
  uint32_t* err = reinterpret_cast<uint32_t*>(ws + w.err);
  DG_HIP(dgk::launch_zero(err, s), "zero");
  uint64_t* status = reinterpret_cast<uint64_t*>(ws + w.flags);
  uint64_t* ticket = reinterpret_cast<uint64_t*>(ws + w.ticket);
  uint64_t cap = (uint64_t)capacity;
  // Blocks take their locations from a ticket counter, so a list longer
  // than one grid runs as several launches of the same kernel on the
  // stream: the blocks of a later launch take the next tickets and look
  // back over words the earlier launches have finished.
  DG_HIP(dgk::launch_zero_u64(status, n, s), "zero status");
  DG_HIP(dgk::launch_zero_u64(ticket, 1, s), "zero ticket");
  DG_HIP(per_location(n, g->block,
                      [&](int64_t, int64_t m) {
                        if (jm) {
                          void* args[] = {&src, &n, &d_offsets, &d_ids, &d_counts, &cap, &status, &ticket, &err};
                          return launch_module(wide ? jm->enumerate_wide : jm->enumerate, m, g->block, lds, s, args);
                        }
                        if constexpr (wide)
                          return dgk::launch_enumerate_wide(blob, src, n, m, d_offsets, d_ids, d_counts, cap, status,
                                                            ticket, err, g->block, lds, s);
                        else
                          return dgk::launch_enumerate(blob, src, n, m, d_offsets, d_ids, d_counts, cap, status,
                                                       ticket, err, g->block, lds, s);
                      }),
         "enumerate kernel");
  int64_t total = 0;
  uint32_t bits = 0;
  DG_HIP(hipMemcpyAsync(&total, d_offsets + n, sizeof(int64_t), hipMemcpyDeviceToHost, s), "copy total");
  DG_HIP(hipMemcpyAsync(&bits, err, sizeof(uint32_t), hipMemcpyDeviceToHost, s), "copy flags");
  DG_HIP(hipStreamSynchronize(s), "enumerate sync");
  *h_total = total;
  return device_errors(bits);
}

}  // namespace

extern "C++" {
namespace dg_internal {

dg_status fail(dg_status code, const std::string& msg) { return set_error(code, msg); }

size_t workspace_bytes(int64_t n) { return ws_layout(n).total; }

dg_status enumerate_resident(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_offsets,
                             uint32_t* d_ids, uint32_t* d_counts, int64_t capacity, void* d_ws, int64_t* h_total,
                             void* stream) {
  return enumerate_impl(g, dgc::LocSrc{d_locs, 0}, n, d_offsets, d_ids, d_counts, capacity, d_ws, h_total, stream,
                        true);
}

}  // namespace dg_internal
}  // extern "C++"

namespace {

// Whether [first, first + n) lies inside the output of g.
bool range_ok(const dg_graph* g, int64_t first, int64_t n) {
  const int64_t numel = g->plan.header().out_numel;
  return first >= 0 && n >= 0 && first <= numel && n <= numel - first;
}

}  // namespace

dg_status dg_enumerate(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_offsets, uint32_t* d_ids,
                       uint32_t* d_counts, int64_t capacity, void* d_ws, int64_t* h_total, void* stream) {
  if (!g || !d_offsets || !h_total || n < 0 || n > kMaxLocations || capacity < 0 || (n > 0 && !d_locs) ||
      (capacity > 0 && (!d_ids || !d_counts)))
    return set_error(DG_E_INVALID_ARG, "bad argument");
  return enumerate_impl(g, dgc::LocSrc{d_locs, 0}, n, d_offsets, d_ids, d_counts, capacity, d_ws, h_total, stream);
}

dg_status dg_enumerate_wide(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_offsets,
                            uint64_t* d_ids, uint64_t* d_counts, int64_t capacity, void* d_ws, int64_t* h_total,
                            void* stream) {
  if (!g || !d_offsets || !h_total || n < 0 || n > kMaxLocations || capacity < 0 || (n > 0 && !d_locs) ||
      (capacity > 0 && (!d_ids || !d_counts)))
    return set_error(DG_E_INVALID_ARG, "bad argument");
  return enumerate_impl(g, dgc::LocSrc{d_locs, 0}, n, d_offsets, d_ids, d_counts, capacity, d_ws, h_total, stream);
}

dg_status dg_enumerate_range(const dg_graph* g, int64_t first, int64_t n, int64_t* d_offsets, uint32_t* d_ids,
                             uint32_t* d_counts, int64_t capacity, void* d_ws, int64_t* h_total, void* stream) {
  if (!g || !d_offsets || !h_total || n < 0 || n > kMaxLocations || capacity < 0 || (capacity > 0 && (!d_ids || !d_counts)))
    return set_error(DG_E_INVALID_ARG, "bad argument");
  if (!range_ok(g, first, n)) return set_error(DG_E_RANGE, "the location range leaves the output");
  return enumerate_impl(g, dgc::LocSrc{nullptr, first}, n, d_offsets, d_ids, d_counts, capacity, d_ws, h_total,
                        stream);
}

dg_status dg_enumerate_stream(const dg_graph* g, int64_t first, int64_t n, void* d_buf, size_t buf_bytes,
                              int64_t max_chunk, dg_chunk_fn fn, void* user, void* stream_a, void* stream_b) {
  if (!g || !d_buf || !fn || n < 0 || n > kMaxLocations || max_chunk <= 0) return set_error(DG_E_INVALID_ARG, "bad argument");
  if (!range_ok(g, first, n)) return set_error(DG_E_RANGE, "the location range leaves the output");
  if (!narrow_ids(g)) return set_error(DG_E_OVERFLOW, "leaf ids need 64 bits: use dg_enumerate_wide");
  if (n == 0) return DG_OK;
  return guarded([&]() -> dg_status {
    // Buffer: offsets of the whole range | sizes workspace | two halves of
    // (chunk offsets from 0 | fill workspace | ids | counts).
    auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
    uint8_t* p = static_cast<uint8_t*>(d_buf);
    int64_t* g_off = reinterpret_cast<int64_t*>(p);
    size_t used_bytes = up(8 * (size_t)(n + 1));
    void* s_ws = p + used_bytes;
    used_bytes += up(ws_layout(n).total);
    max_chunk = std::min(max_chunk, n);
    const size_t rel_bytes = up(8 * (size_t)(max_chunk + 1));
    const size_t fws_bytes = up(ws_layout(max_chunk).total);
    if (buf_bytes < used_bytes + 2 * (rel_bytes + fws_bytes + 512))
      return set_error(DG_E_BUFFER, "buffer too small for the range's offsets and two chunks");
    const size_t half = ((buf_bytes - used_bytes) / 2) & ~size_t(255);
    const int64_t cap = (int64_t)((half - rel_bytes - fws_bytes) / 8) & ~int64_t(63);
    hipStream_t st[2] = {static_cast<hipStream_t>(stream_a), static_cast<hipStream_t>(stream_b)};
    const uint8_t* blob = nullptr;
    dg_status rc = device_blob(g, &blob);
    if (rc != DG_OK) return rc;
    // 1. Row sizes and offsets of the whole range, then chunks cut exactly
    //    where the rows stop fitting a half.
    int64_t total = 0;
    rc = sizes_impl(g, dgc::LocSrc{nullptr, first}, n, g_off, s_ws, &total, st[0]);
    if (rc != DG_OK) return rc;
    std::vector<int64_t> h_off((size_t)n + 1);
    DG_HIP(hipMemcpy(h_off.data(), g_off, 8 * (size_t)(n + 1), hipMemcpyDeviceToHost), "copy offsets");
    // 2. Chunks alternate halves and streams; the fills are asynchronous.
    bool used[2] = {false, false};
    uint32_t bits = 0;
    auto retire = [&](int h) -> dg_status {  // the half's fill and consumer have finished
      uint8_t* base = p + used_bytes + h * half;
      uint32_t b = 0;
      DG_HIP(hipStreamSynchronize(st[h]), "chunk sync");
      DG_HIP(hipMemcpy(&b, base + rel_bytes + ws_layout(max_chunk).err, 4, hipMemcpyDeviceToHost), "copy flags");
      bits |= b;
      used[h] = false;
      return DG_OK;
    };
    int64_t pos = 0;
    for (int c = 0; pos < n; ++c) {
      const int h = c & 1;
      if (used[h]) {
        rc = retire(h);
        if (rc != DG_OK) break;
        if (bits) break;
      }
      const int64_t lim = std::min(n, pos + max_chunk);
      const int64_t end = (int64_t)(std::upper_bound(h_off.begin() + pos, h_off.begin() + lim + 1, h_off[pos] + cap) -
                                    h_off.begin()) - 1;
      const int64_t m = end - pos;
      if (m <= 0) {
        rc = set_error(DG_E_BUFFER, "one location's row does not fit half of the buffer");
        break;
      }
      uint8_t* base = p + used_bytes + h * half;
      int64_t* rel = reinterpret_cast<int64_t*>(base);
      uint8_t* fws = base + rel_bytes;
      uint32_t* ids = reinterpret_cast<uint32_t*>(base + rel_bytes + fws_bytes);
      uint32_t* cnt = ids + cap;
      uint32_t* err = reinterpret_cast<uint32_t*>(fws + ws_layout(max_chunk).err);
      DG_HIP(dgk::launch_zero(err, st[h]), "zero");
      DG_HIP(fill_launch(g, blob, dgc::LocSrc{nullptr, first + pos}, m, g_off + pos, h_off[pos], ids, cnt, err,
                         st[h]),
             "fill kernel");
      DG_HIP(dgk::launch_rebase(g_off + pos, rel, m + 1, h_off[pos], st[h]), "chunk offsets");
      used[h] = true;
      if (fn(user, first + pos, m, rel, ids, cnt, h_off[end] - h_off[pos], st[h]) != 0) {
        rc = set_error(DG_E_STOPPED, "the chunk consumer stopped the stream");
        break;
      }
      pos = end;
    }
    for (int h = 0; h < 2; ++h)
      if (used[h]) {
        dg_status r2 = retire(h);
        if (rc == DG_OK) rc = r2;
      }
    if (rc == DG_OK && bits) rc = device_errors(bits);
    return rc;
  });
}

namespace {

// The joint plans of (a, b) and their copies on the current device,
// compiled and uploaded on first use.
dg_status joint_plans(const dg_graph* a, const dg_graph* b, const dg::Plan** pa, const dg::Plan** pb,
                      const uint8_t** ba, const uint8_t** bb) {
  int dev = 0;
  DG_HIP(hipGetDevice(&dev), "hipGetDevice");
  std::lock_guard<std::mutex> lock(g_pair_mu);
  const auto key = std::make_pair(a->serial, b->serial);
  auto it = g_pair_plans.find(key);
  if (it == g_pair_plans.end()) {
    PairPlans P;
    dg::compile_pair_plans(a->ir, b->ir, &P.a, &P.b);
    it = g_pair_plans.emplace(key, std::move(P)).first;
  }
  PairPlans& P = it->second;
  auto d = P.dev.find(dev);
  if (d == P.dev.end()) {
    uint8_t* p[2] = {nullptr, nullptr};
    const dg::Plan* src[2] = {&P.a, &P.b};
    for (int k = 0; k < 2; ++k) {
      void* q = nullptr;
      hipError_t e = hipMalloc(&q, src[k]->blob.size());
      if (e == hipSuccess) e = hipMemcpy(q, src[k]->blob.data(), src[k]->blob.size(), hipMemcpyHostToDevice);
      if (e != hipSuccess) {
        if (q) (void)hipFree(q);
        if (k == 1) (void)hipFree(p[0]);
        return hip_error(e, "pair plan upload");
      }
      p[k] = static_cast<uint8_t*>(q);
    }
    d = P.dev.emplace(dev, std::make_pair(p[0], p[1])).first;
  }
  *pa = &P.a;
  *pb = &P.b;
  *ba = d->second.first;
  *bb = d->second.second;
  return DG_OK;
}

dg_status compare_impl(const dg_graph* a, const dg_graph* b, dgc::LocSrc src, int64_t n, uint64_t limit,
                       uint8_t* d_status, int64_t* d_mismatch, int64_t* h_n_mismatch, void* d_ws, void* stream) {
  if (!d_ws) return set_error(DG_E_WORKSPACE, "workspace is required");
  return guarded([&]() -> dg_status {
    // MERGE's input/output matching: same leaves (names, shapes, order) and
    // the same output shape.
    const dg::GraphIR &A = a->ir, &B = b->ir;
    if (A.leaves.size() != B.leaves.size()) return set_error(DG_E_SIGNATURE, "leaf count differs");
    for (size_t i = 0; i < A.leaves.size(); ++i) {
      const dg::Tensor &x = A.tensors[A.leaves[i]], &y = B.tensors[B.leaves[i]];
      if (x.name != y.name || x.shape != y.shape)
        return set_error(DG_E_SIGNATURE, "leaf " + std::to_string(i) + " ('" + x.name + "') differs");
    }
    if (A.tensors[A.output].shape != B.tensors[B.output].shape)
      return set_error(DG_E_SIGNATURE, "output shape differs");
    // Comparison rows are compared in LDS, not written: one wave per
    // location keeps its many barriers cheap.
    int block = 64;
    if (const char* e = std::getenv("DIRIGO_CMP_BLOCK")) {
      const int v = std::atoi(e);
      if (v == 64 || v == 128 || v == 256) block = v;
    }
    // Both plans must view each leaf with the same merged dims; when the
    // graphs' own plans do not, the pair's joint plans are used.
    const dg::Plan* plan_a = &a->plan;
    const dg::Plan* plan_b = &b->plan;
    const uint8_t *ba = nullptr, *bb = nullptr;
    dg_status st = DG_OK;
    if (a->plan.leaf_part != b->plan.leaf_part) {
      st = joint_plans(a, b, &plan_a, &plan_b, &ba, &bb);
      if (st != DG_OK) return st;
    } else {
      st = device_blob(a, &ba);
      if (st != DG_OK) return st;
      st = device_blob(b, &bb);
      if (st != DG_OK) return st;
    }
    dgc::PairPlan pp;
    dg::pair_plan(*plan_a, *plan_b, block, &pp);
    if (pp.lds_bytes > (uint32_t)max_lds_per_block())
      return set_error(DG_E_CAPACITY, "comparison needs " + std::to_string(pp.lds_bytes) + " bytes of LDS");
    hipStream_t s = static_cast<hipStream_t>(stream);
    WsLayout w = ws_layout(n);
    uint8_t* ws = static_cast<uint8_t*>(d_ws);
    uint32_t* err = reinterpret_cast<uint32_t*>(ws + w.err);
    int64_t* flags = reinterpret_cast<int64_t*>(ws + w.flags);
    DG_HIP(dgk::launch_zero(err, s), "zero");
    uint64_t* found = reinterpret_cast<uint64_t*>(ws + w.found);
    DG_HIP(dgk::launch_zero_u64(found, 1, s), "zero count");
    const dg::JitModule* jm = pair_jit(a, b, *plan_a, *plan_b, pp, block);
    dgc::PairPlan* d_pp = reinterpret_cast<dgc::PairPlan*>(ws + w.pair);
    if (!jm) {
      if (block != 64 && block != 256) return set_error(DG_E_INVALID_ARG, "block size needs specialised kernels");
      // Pageable source: the copy has completed when the call returns.
      DG_HIP(hipMemcpyAsync(d_pp, &pp, sizeof(pp), hipMemcpyHostToDevice, s), "copy pair plan");
    }
    DG_HIP(per_location(n, block,
                        [&](int64_t first, int64_t m) {
                          dgc::LocSrc part = shifted(src, first);
                          uint8_t* st_part = d_status + first;
                          int64_t* fl_part = flags + first;
                          if (jm) {
                            void* args[] = {&part, &m, &st_part, &fl_part, &found, &limit, &err};
                            return launch_module(jm->compare, m, block, pp.lds_bytes, s, args);
                          }
                          return dgk::launch_compare(ba, bb, d_pp, pp.lds_bytes, part, m, st_part, fl_part, found,
                                                     limit, err, block, s);
                        }),
           "compare kernel");
    DG_HIP(dgk::launch_scan(flags, n, reinterpret_cast<int64_t*>(ws + w.sums), s), "scan");
    DG_HIP(dgk::launch_scatter_mismatch(d_status, flags, n, d_mismatch, s), "scatter");
    int64_t total = 0;
    uint32_t bits = 0;
    DG_HIP(hipMemcpyAsync(&total, flags + n, sizeof(int64_t), hipMemcpyDeviceToHost, s), "copy count");
    DG_HIP(hipMemcpyAsync(&bits, err, sizeof(uint32_t), hipMemcpyDeviceToHost, s), "copy flags");
    DG_HIP(hipStreamSynchronize(s), "compare sync");
    st = device_errors(bits);
    if (st != DG_OK) return st;
    *h_n_mismatch = total;
    return DG_OK;
  });
}

}  // namespace

dg_status dg_dag_sizes(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_node_offsets,
                       int64_t* d_edge_offsets, void* d_ws, int64_t* h_nodes, int64_t* h_edges, void* stream) {
  if (!g || !d_node_offsets || !d_edge_offsets || !h_nodes || !h_edges || n < 0 || n > kMaxLocations || (n > 0 && !d_locs))
    return set_error(DG_E_INVALID_ARG, "bad argument");
  if (!d_ws) return set_error(DG_E_WORKSPACE, "workspace is required");
  return guarded([&]() -> dg_status {
    const uint8_t* dblob = nullptr;
    dg_status st = dag_program(g, &dblob);
    if (st != DG_OK) return st;
    if (g->dag.lds_bytes > (uint32_t)max_lds_per_block())
      return set_error(DG_E_CAPACITY, "one location's DAG frontiers need " + std::to_string(g->dag.lds_bytes) +
                                          " bytes of LDS");
    hipStream_t s = static_cast<hipStream_t>(stream);
    WsLayout w = ws_layout(n);
    uint8_t* ws = static_cast<uint8_t*>(d_ws);
    uint32_t* err = reinterpret_cast<uint32_t*>(ws + w.err);
    DG_HIP(dgk::launch_zero(err, s), "zero");
    const dg::JitModule* jm = dag_jit(g, n);
    int k = dag_per_block(g);
    DG_HIP(per_location(n, g->dag_block,
                        [&](int64_t first, int64_t m) {
                          dgc::LocSrc part{d_locs + first, 0};
                          int64_t* nn = d_node_offsets + first;
                          int64_t* en = d_edge_offsets + first;
                          if (jm) {
                            void* args[] = {&part, &m, &k, &nn, &en, &err};
                            return launch_module(jm->dag_sizes, (m + k - 1) / k, g->dag_block, g->dag.lds_bytes, s,
                                                 args);
                          }
                          return dgk::launch_dag_sizes(dblob, part, m, k, nn, en, err, g->dag_block,
                                                       g->dag.lds_bytes, s);
                        }),
           "DAG sizes kernel");
    int64_t* sums = reinterpret_cast<int64_t*>(ws + w.sums);
    DG_HIP(dgk::launch_scan(d_node_offsets, n, sums, s), "scan");
    DG_HIP(dgk::launch_scan(d_edge_offsets, n, sums, s), "scan");
    int64_t tn = 0, te = 0;
    uint32_t bits = 0;
    DG_HIP(hipMemcpyAsync(&tn, d_node_offsets + n, sizeof(int64_t), hipMemcpyDeviceToHost, s), "copy total");
    DG_HIP(hipMemcpyAsync(&te, d_edge_offsets + n, sizeof(int64_t), hipMemcpyDeviceToHost, s), "copy total");
    DG_HIP(hipMemcpyAsync(&bits, err, sizeof(uint32_t), hipMemcpyDeviceToHost, s), "copy flags");
    DG_HIP(hipStreamSynchronize(s), "DAG sizes sync");
    st = device_errors(bits);
    if (st != DG_OK) return st;
    *h_nodes = tn;
    *h_edges = te;
    return DG_OK;
  });
}

dg_status dg_dag_fill(const dg_graph* g, const int64_t* d_locs, int64_t n, const int64_t* d_node_offsets,
                      const int64_t* d_edge_offsets, uint32_t* d_nodes, uint32_t* d_node_edge, uint32_t* d_edges,
                      uint32_t* d_mults, void* d_ws, void* stream) {
  if (!g || n < 0 || n > kMaxLocations || (n > 0 && (!d_locs || !d_node_offsets || !d_edge_offsets || !d_nodes || !d_node_edge ||
                                !d_edges || !d_mults)))
    return set_error(DG_E_INVALID_ARG, "bad argument");
  if (!d_ws) return set_error(DG_E_WORKSPACE, "workspace is required");
  return guarded([&]() -> dg_status {
    const uint8_t* dblob = nullptr;
    dg_status st = dag_program(g, &dblob);
    if (st != DG_OK) return st;
    if (g->dag.lds_bytes > (uint32_t)max_lds_per_block())
      return set_error(DG_E_CAPACITY, "one location's DAG frontiers need " + std::to_string(g->dag.lds_bytes) +
                                          " bytes of LDS");
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint32_t* err = reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(d_ws) + ws_layout(n).err);
    DG_HIP(dgk::launch_zero(err, s), "zero");
    const dg::JitModule* jm = dag_jit(g, n);
    int k = dag_per_block(g);
    DG_HIP(per_location(n, g->dag_block,
                        [&](int64_t first, int64_t m) {
                          dgc::LocSrc part{d_locs + first, 0};
                          const int64_t* no = d_node_offsets + first;
                          const int64_t* eo = d_edge_offsets + first;
                          if (jm) {
                            void* args[] = {&part, &m, &k, (void*)&no, (void*)&eo, &d_nodes, &d_node_edge, &d_edges,
                                            &d_mults, &err};
                            return launch_module(jm->dag_fill, (m + k - 1) / k, g->dag_block, g->dag.lds_bytes, s,
                                                 args);
                          }
                          return dgk::launch_dag_fill(dblob, part, m, k, no, eo, d_nodes, d_node_edge, d_edges,
                                                      d_mults, err, g->dag_block, g->dag.lds_bytes, s);
                        }),
           "DAG fill kernel");
    uint32_t bits = 0;
    DG_HIP(hipMemcpyAsync(&bits, err, sizeof(uint32_t), hipMemcpyDeviceToHost, s), "copy flags");
    DG_HIP(hipStreamSynchronize(s), "DAG fill sync");
    return device_errors(bits);
  });
}

namespace {

// Where the one-pass DAG kernels stage a location's DAG in LDS (after the
// walk's area) and the LDS a block then needs: node and edge slots of the
// program's static bounds, two words each.  0 when that exceeds 64 KiB or
// the device's limit (the call then takes the two passes).
uint32_t dag_stage_off(const dg_graph* g) { return (g->dag.lds_bytes + 15u) & ~15u; }

// Calls of at most this many locations take the one pass: it saves the
// host round trip between the two passes, but a location costs more than
// its two passes at scale (the DAGs of a 3x3, 64-channel conv2d with an
// affine and a relu: 0.15 against 0.19 ms at 1,024 locations, 0.23 against
// 0.21 ms at 4,096, 3.3 against 0.97 ms at 262,144).
// DIRIGO_DAG_ONEPASS=1 takes it whenever the stage fits,
// DIRIGO_DAG_ONEPASS=0 never.
constexpr int64_t kDagOnePassMax = 2048;
bool dag_onepass_wanted(int64_t n) {
  const char* env = std::getenv("DIRIGO_DAG_ONEPASS");
  if (env && env[0] == '1') return true;
  if (env && env[0] == '0') return false;
  return n <= kDagOnePassMax;
}
uint32_t dag_onepass_lds(const dg_graph* g) {
  const uint64_t words = 2ull * (uint64_t)g->dag.max_nodes + 2ull * (uint64_t)g->dag.max_edges;
  const uint64_t lds = (uint64_t)dag_stage_off(g) + 4ull * words;
  return lds <= std::min<uint64_t>(65536u, (uint64_t)max_lds_per_block()) ? (uint32_t)lds : 0u;
}

}  // namespace

dg_status dg_dag(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_node_offsets, int64_t* d_edge_offsets,
                 uint32_t* d_nodes, uint32_t* d_node_edge, uint32_t* d_edges, uint32_t* d_mults, int64_t node_capacity,
                 int64_t edge_capacity, void* d_ws, int64_t* h_nodes, int64_t* h_edges, void* stream) {
  if (!g || !d_node_offsets || !d_edge_offsets || !h_nodes || !h_edges || n < 0 || n > kMaxLocations ||
      node_capacity < 0 || edge_capacity < 0 || (n > 0 && !d_locs) ||
      (node_capacity > 0 && (!d_nodes || !d_node_edge)) || (edge_capacity > 0 && (!d_edges || !d_mults)))
    return set_error(DG_E_INVALID_ARG, "bad argument");
  if (!d_ws) return set_error(DG_E_WORKSPACE, "workspace is required");
  return guarded([&]() -> dg_status {
    const uint8_t* dblob = nullptr;
    dg_status st = dag_program(g, &dblob);
    if (st != DG_OK) return st;
    if (g->dag.lds_bytes > (uint32_t)max_lds_per_block())
      return set_error(DG_E_CAPACITY, "one location's DAG frontiers need " + std::to_string(g->dag.lds_bytes) +
                                          " bytes of LDS");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (n == 0) {
      DG_HIP(dgk::launch_scan(d_node_offsets, 0, nullptr, s), "offsets");
      DG_HIP(dgk::launch_scan(d_edge_offsets, 0, nullptr, s), "offsets");
      DG_HIP(hipStreamSynchronize(s), "sync");
      *h_nodes = 0;
      *h_edges = 0;
      return DG_OK;
    }
    const uint32_t lds = dag_onepass_wanted(n) ? dag_onepass_lds(g) : 0u;
    if (lds == 0) {
      // The two passes: sizes, then the fill when it fits.
      int64_t tn = 0, te = 0;
      st = dg_dag_sizes(g, d_locs, n, d_node_offsets, d_edge_offsets, d_ws, &tn, &te, stream);
      if (st != DG_OK) return st;
      *h_nodes = tn;
      *h_edges = te;
      if (tn > node_capacity || te > edge_capacity)
        return set_error(DG_E_BUFFER, "the DAGs need more nodes or edges than the output buffers hold");
      return dg_dag_fill(g, d_locs, n, d_node_offsets, d_edge_offsets, d_nodes, d_node_edge, d_edges, d_mults, d_ws,
                         stream);
    }
    DagWsLayout w = dag_ws_layout(n);
    uint8_t* ws = static_cast<uint8_t*>(d_ws);
    uint32_t* err = reinterpret_cast<uint32_t*>(ws + w.err);
    uint64_t* ticket = reinterpret_cast<uint64_t*>(ws + w.ticket);
    uint64_t* st_n = reinterpret_cast<uint64_t*>(ws + w.st_nodes);
    uint64_t* st_e = reinterpret_cast<uint64_t*>(ws + w.st_edges);
    DG_HIP(dgk::launch_zero(err, s), "zero");
    DG_HIP(dgk::launch_zero_u64(st_n, n, s), "zero status");
    DG_HIP(dgk::launch_zero_u64(st_e, n, s), "zero status");
    DG_HIP(dgk::launch_zero_u64(ticket, 1, s), "zero ticket");
    const dg::JitModule* jm = dag_jit(g, n);
    if (jm && !jm->dag_onepass) jm = nullptr;
    dgc::LocSrc src{d_locs, 0};
    uint64_t ncap = (uint64_t)node_capacity, ecap = (uint64_t)edge_capacity;
    uint32_t stage_off = dag_stage_off(g), stage_nodes = (uint32_t)g->dag.max_nodes,
             stage_edges = (uint32_t)g->dag.max_edges;
    // Blocks take their locations from a ticket counter (as for
    // dg_enumerate), so a list longer than one grid runs as several
    // launches of the same kernel.
    DG_HIP(per_location(n, g->dag_block,
                        [&](int64_t, int64_t m) {
                          if (jm) {
                            void* args[] = {&src, &n, &d_node_offsets, &d_edge_offsets, &d_nodes, &d_node_edge,
                                            &d_edges, &d_mults, &ncap, &ecap, &stage_off, &stage_nodes,
                                            &stage_edges, &st_n, &st_e, &ticket, &err};
                            return launch_module(jm->dag_onepass, m, g->dag_block, lds, s, args);
                          }
                          return dgk::launch_dag_onepass(dblob, src, n, m, d_node_offsets, d_edge_offsets, d_nodes,
                                                         d_node_edge, d_edges, d_mults, ncap, ecap, stage_off,
                                                         stage_nodes, stage_edges, st_n, st_e, ticket, err,
                                                         g->dag_block, lds, s);
                        }),
           "DAG one-pass kernel");
    int64_t tn = 0, te = 0;
    uint32_t bits = 0;
    DG_HIP(hipMemcpyAsync(&tn, d_node_offsets + n, sizeof(int64_t), hipMemcpyDeviceToHost, s), "copy total");
    DG_HIP(hipMemcpyAsync(&te, d_edge_offsets + n, sizeof(int64_t), hipMemcpyDeviceToHost, s), "copy total");
    DG_HIP(hipMemcpyAsync(&bits, err, sizeof(uint32_t), hipMemcpyDeviceToHost, s), "copy flags");
    DG_HIP(hipStreamSynchronize(s), "DAG one-pass sync");
    *h_nodes = tn;
    *h_edges = te;
    st = device_errors(bits);
    if (st == DG_E_BUFFER)
      return set_error(DG_E_BUFFER, "the DAGs need more nodes or edges than the output buffers hold");
    return st;
  });
}

dg_status dg_graph_text(const dg_graph* g, char* buf, size_t cap, size_t* len) {
  if (!g || !len || (cap > 0 && !buf)) return set_error(DG_E_INVALID_ARG, "bad argument");
  return guarded([&]() -> dg_status {
    const std::string t = dg::graph_text(g->ir);
    *len = t.size();
    if (cap > 0) {
      const size_t n = std::min(cap - 1, t.size());
      std::memcpy(buf, t.data(), n);
      buf[n] = '\0';
    }
    return DG_OK;
  });
}

dg_status dg_graph_merge(const dg_graph* a, const dg_graph* b, int32_t trim_prefix, dg_graph** a_out,
                         dg_graph** b_out, int32_t* n_trimmed) {
  if (!a || !b || !a_out || !b_out) return set_error(DG_E_INVALID_ARG, "bad argument");
  *a_out = *b_out = nullptr;
  dg_status st = guarded([&]() -> dg_status {
    const dg::Merged m = dg::merge_graphs(a->ir, b->ir, trim_prefix != 0);
    dg_status s = dg_graph_parse(m.a_text.c_str(), m.a_text.size(), a_out);
    if (s != DG_OK) return s;
    s = dg_graph_parse(m.b_text.c_str(), m.b_text.size(), b_out);
    if (s != DG_OK) return s;
    if (n_trimmed) *n_trimmed = m.trimmed;
    return DG_OK;
  });
  if (st != DG_OK) {
    if (*a_out) dg_graph_destroy(*a_out);
    if (*b_out) dg_graph_destroy(*b_out);
    *a_out = *b_out = nullptr;
  }
  return st;
}

dg_status dg_order_prefix(const dg_graph* g, int32_t block_threads, int32_t warp, int64_t* h_prefix, int64_t cap,
                          int64_t* h_count) {
  if (!g || !h_count || cap < 0 || (cap > 0 && !h_prefix)) return set_error(DG_E_INVALID_ARG, "bad argument");
  return guarded([&]() -> dg_status {
    const std::vector<int64_t> p = dg::order_prefix(g->ir, block_threads, warp);
    *h_count = (int64_t)p.size();
    for (int64_t i = 0; i < (int64_t)p.size() && i < cap; ++i) h_prefix[i] = p[(size_t)i];
    return DG_OK;
  });
}

dg_status dg_order_workspace_size(int64_t n_exclude, size_t* bytes) {
  if (!bytes || n_exclude < 0) return set_error(DG_E_INVALID_ARG, "bad argument");
  *bytes = 8 * (size_t)std::max<int64_t>(1, n_exclude);
  return DG_OK;
}

dg_status dg_order_permute(int64_t n_out, uint64_t seed, const int64_t* h_exclude, int64_t n_exclude, int64_t first,
                           int64_t count, int64_t* d_out, int64_t* h_written, void* d_ws, size_t ws_bytes,
                           void* stream) {
  if (!h_written || n_out < 0 || n_out > ((int64_t)1 << 62) || n_exclude < 0 || first < 0 || count < 0 ||
      first > n_out || count > n_out - first || (n_exclude > 0 && !h_exclude) || (count > 0 && !d_out))
    return set_error(DG_E_INVALID_ARG, "bad argument");
  return guarded([&]() -> dg_status {
    const DgPermKey K = dg_perm_key(n_out, seed);
    // Positions of the excluded values inside the range, sorted.
    std::vector<int64_t> pos;
    for (int64_t j = 0; j < n_exclude; ++j) {
      const int64_t v = h_exclude[j];
      if (v < 0 || v >= n_out) return set_error(DG_E_INVALID_ARG, "an excluded value is outside [0, n_out)");
      const int64_t p = dg_perm_position((uint64_t)v, K);
      if (p >= first && p - first < count) pos.push_back(p);
    }
    std::sort(pos.begin(), pos.end());
    pos.erase(std::unique(pos.begin(), pos.end()), pos.end());
    if (!pos.empty() && (!d_ws || ws_bytes < 8 * pos.size()))
      return set_error(DG_E_WORKSPACE, "workspace smaller than dg_order_workspace_size");
    hipStream_t s = static_cast<hipStream_t>(stream);
    int64_t* d_pos = static_cast<int64_t*>(d_ws);
    if (!pos.empty())
      DG_HIP(hipMemcpyAsync(d_pos, pos.data(), 8 * pos.size(), hipMemcpyHostToDevice, s), "copy positions");
    DG_HIP(dgk::launch_order(K, d_pos, (int64_t)pos.size(), first, count, d_out, s), "order kernel");
    DG_HIP(hipStreamSynchronize(s), "order sync");
    *h_written = count - (int64_t)pos.size();
    return DG_OK;
  });
}

dg_status dg_compare(const dg_graph* a, const dg_graph* b, const int64_t* d_locs, int64_t n, uint8_t* d_status,
                     int64_t* d_mismatch, int64_t* h_n_mismatch, void* d_ws, void* stream) {
  if (!a || !b || !h_n_mismatch || n < 0 || n > kMaxLocations || (n > 0 && (!d_locs || !d_status || !d_mismatch)))
    return set_error(DG_E_INVALID_ARG, "bad argument");
  return compare_impl(a, b, dgc::LocSrc{d_locs, 0}, n, 0, d_status, d_mismatch, h_n_mismatch, d_ws, stream);
}

dg_status dg_compare_range(const dg_graph* a, const dg_graph* b, int64_t first, int64_t n, int64_t max_mismatch,
                           uint8_t* d_status, int64_t* d_mismatch, int64_t* h_n_mismatch, void* d_ws,
                           void* stream) {
  if (!a || !b || !h_n_mismatch || n < 0 || n > kMaxLocations || max_mismatch < 0 || (n > 0 && (!d_status || !d_mismatch)))
    return set_error(DG_E_INVALID_ARG, "bad argument");
  if (!range_ok(a, first, n)) return set_error(DG_E_RANGE, "the location range leaves the output");
  return compare_impl(a, b, dgc::LocSrc{nullptr, first}, n, (uint64_t)max_mismatch, d_status, d_mismatch,
                      h_n_mismatch, d_ws, stream);
}

}  // extern "C"
