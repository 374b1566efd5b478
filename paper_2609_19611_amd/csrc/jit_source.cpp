// Sources of the per-graph specialised kernels (see jit.h).  Host-only
// code: no HIP runtime calls.
#include <cstring>
#include <sstream>

#include "dag_program.h"
#include "jit.h"

namespace dg {

namespace {

void emit_bytes(std::ostringstream& o, const char* name, const std::vector<uint8_t>& b) {
  o << "static __constant__ __attribute__((aligned(16))) const unsigned char " << name << "[" << b.size()
    << "] = {";
  for (size_t i = 0; i < b.size(); ++i) {
    if (i % 32 == 0) o << "\n";
    o << (unsigned)b[i] << ",";
  }
  o << "};\n";
}

const char* kPrelude =
    "#define DG_JIT 1\n"
    "#define DGC __device__ __forceinline__\n"
    "#include \"kernels_dev.h\"\n";

// Same code-generation footing as the precompiled kernels: packed FP32
// instructions stay off.
const char* const kOptions[] = {"--offload-arch=gfx950", "-O3",     "-std=c++17",      "-mllvm",
                                "-amdgpu-early-inline-all=true",   "-Wno-pass-failed", "-Xclang",
                                "-target-feature",                 "-Xclang",          "-packed-fp32-ops",
                                nullptr};

}  // namespace

const char* const* jit_compile_options() { return kOptions; }

std::string jit_enum_source(const Plan& p, int block) {
  std::ostringstream o;
  o << kPrelude;
  emit_bytes(o, "dg_plan", p.blob);
  o << "#define DG_B " << block << "\n"
    << "extern \"C\" __global__ __launch_bounds__(DG_B) void dg_sizes(dgc::LocSrc locs, int64_t n,\n"
    << "    int64_t* __restrict__ offsets, uint32_t* __restrict__ err) {\n"
    << "  dgk_dev::sizes_body<DG_B>(dg_plan, locs, n, offsets, err);\n}\n"
    << "extern \"C\" __global__ __launch_bounds__(DG_B) void dg_fill(dgc::LocSrc locs, int64_t n,\n"
    << "    const int64_t* __restrict__ offsets, int64_t base, uint32_t* __restrict__ ids,\n"
    << "    uint32_t* __restrict__ cnt, uint32_t* __restrict__ err) {\n"
    << "  dgk_dev::fill_body<DG_B>(dg_plan, locs, n, offsets, base, ids, cnt, err);\n}\n"
    << "extern \"C\" __global__ __launch_bounds__(DG_B) void dg_enumerate(dgc::LocSrc locs, int64_t n,\n"
    << "    int64_t* __restrict__ offsets, uint32_t* __restrict__ ids, uint32_t* __restrict__ cnt, uint64_t capacity,\n"
    << "    uint64_t* __restrict__ status, unsigned long long* __restrict__ ticket, uint32_t* __restrict__ err) {\n"
    << "  dgk_dev::enumerate_body<DG_B>(dg_plan, locs, n, offsets, ids, cnt, capacity, status, ticket, err);\n}\n";
  return o.str();
}

std::string jit_wide_source(const Plan& p, int block) {
  std::ostringstream o;
  o << kPrelude;
  emit_bytes(o, "dg_plan", p.blob);
  o << "#define DG_B " << block << "\n"
    << "extern \"C\" __global__ __launch_bounds__(DG_B) void dg_enumerate_wide(dgc::LocSrc locs, int64_t n,\n"
    << "    int64_t* __restrict__ offsets, uint64_t* __restrict__ ids, uint64_t* __restrict__ cnt,\n"
    << "    uint64_t capacity, uint64_t* __restrict__ status, unsigned long long* __restrict__ ticket,\n"
    << "    uint32_t* __restrict__ err) {\n"
    << "  dgk_dev::enumerate_body<DG_B, uint64_t>(dg_plan, locs, n, offsets, ids, cnt, capacity, status, ticket,"
       " err);\n}\n";
  return o.str();
}

std::string jit_compare_source(const Plan& a, const Plan& b, const dgc::PairPlan& pp, int block) {
  std::ostringstream o;
  o << kPrelude;
  emit_bytes(o, "dg_plan_a", a.blob);
  emit_bytes(o, "dg_plan_b", b.blob);
  std::vector<uint8_t> ppb(sizeof(pp));
  std::memcpy(ppb.data(), &pp, sizeof(pp));
  emit_bytes(o, "dg_pair", ppb);
  o << "#define DG_B " << block << "\n"
    << "extern \"C\" __global__ __launch_bounds__(DG_B) void dg_compare(dgc::LocSrc locs, int64_t n,\n"
    << "    uint8_t* __restrict__ status, int64_t* __restrict__ flags, unsigned long long* __restrict__ found,\n"
    << "    uint64_t limit, uint32_t* __restrict__ err) {\n"
    << "  dgk_dev::compare_body<DG_B>(dg_plan_a, dg_plan_b, (const dgc::PairPlan*)dg_pair, locs, n, status, flags,"
       " found, limit, err);\n}\n";
  return o.str();
}

std::string jit_dag_source(const DagProgram& p, int block) {
  const DgdHeader* h = reinterpret_cast<const DgdHeader*>(p.blob.data());
  const DgdOp* O = reinterpret_cast<const DgdOp*>(p.blob.data() + h->op_off);
  const DgdGroup* G = reinterpret_cast<const DgdGroup*>(p.blob.data() + h->group_off);
  // The ways of taking a group that the program's groups use (dag_core.h).
  unsigned fast = 0, node = 0;
  int slow = 0, box = 0, pw = 0;
  for (int k = 0; k < h->nop; ++k) {
    if (O[k].pointwise) {
      pw = 1;
      continue;
    }
    for (int q = 0; q < O[k].ng; ++q) {
      const DgdGroup& g = G[O[k].g0 + q];
      if (g.points == 0) continue;
      if (!g.fast) {
        box = 1;
      } else if (g.steps24 && g.nop >= 1 && g.nop <= 3 && g.nwin >= 0 && g.nwin <= 4) {
        fast |= 1u << ((g.nop - 1) * 5 + g.nwin);
      } else {
        slow = 1;
        if (g.nop >= 1 && g.nop <= 3 && g.nwin >= 1 && g.nwin <= 4) node |= 1u << ((g.nop - 1) * 4 + g.nwin - 1);
      }
    }
  }
  std::ostringstream o;
  o << "#define DG_JIT 1\n"
    << "#define DGC __device__ __forceinline__\n"
    << "#define DG_DAG_FAST " << fast << "u\n"
    << "#define DG_DAG_NODE " << node << "u\n"
    << "#define DG_DAG_SLOW " << slow << "\n"
    << "#define DG_DAG_BOX " << box << "\n"
    << "#define DG_DAG_PW " << pw << "\n"
    << "#define DG_DAG_NOPS " << h->nop << "\n"
    << "#include \"dag_dev.h\"\n";
  emit_bytes(o, "dg_dag", p.blob);
  o << "#define DG_B " << block << "\n"
    << "extern \"C\" __global__ __launch_bounds__(DG_B) void dg_dag_sizes(dgc::LocSrc locs, int64_t n, int per_block,\n"
    << "    int64_t* __restrict__ nodes_n, int64_t* __restrict__ edges_n, uint32_t* __restrict__ err) {\n"
    << "  dgk_dev::dag_sizes_body<DG_B>(dg_dag, locs, n, per_block, nodes_n, edges_n, err);\n}\n"
    << "extern \"C\" __global__ __launch_bounds__(DG_B) void dg_dag_fill(dgc::LocSrc locs, int64_t n, int per_block,\n"
    << "    const int64_t* __restrict__ node_off, const int64_t* __restrict__ edge_off, uint32_t* __restrict__ nodes,\n"
    << "    uint32_t* __restrict__ node_edge, uint32_t* __restrict__ edges, uint32_t* __restrict__ mults,\n"
    << "    uint32_t* __restrict__ err) {\n"
    << "  dgk_dev::dag_fill_body<DG_B>(dg_dag, locs, n, per_block, node_off, edge_off, nodes, node_edge, edges, mults,\n"
    << "      err);\n}\n"
    << "extern \"C\" __global__ __launch_bounds__(DG_B) void dg_dag_onepass(dgc::LocSrc locs, int64_t n,\n"
    << "    int64_t* __restrict__ node_off, int64_t* __restrict__ edge_off, uint32_t* __restrict__ nodes,\n"
    << "    uint32_t* __restrict__ node_edge, uint32_t* __restrict__ edges, uint32_t* __restrict__ mults,\n"
    << "    uint64_t node_cap, uint64_t edge_cap, uint32_t stage_off, uint32_t stage_nodes, uint32_t stage_edges,\n"
    << "    uint64_t* __restrict__ st_nodes, uint64_t* __restrict__ st_edges, unsigned long long* __restrict__ ticket,\n"
    << "    uint32_t* __restrict__ err) {\n"
    << "  dgk_dev::dag_onepass_body<DG_B>(dg_dag, locs, n, node_off, edge_off, nodes, node_edge, edges, mults,\n"
    << "      node_cap, edge_cap, stage_off, stage_nodes, stage_edges, st_nodes, st_edges, ticket, err);\n}\n";
  return o.str();
}

}  // namespace dg
