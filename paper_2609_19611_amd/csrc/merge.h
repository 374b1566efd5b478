// MERGE (Sec. 3.2): input matching and common-prefix trimming of two graphs
// (see merge.cpp), and the dgir text of a graph.
#pragma once
#include <string>
#include <vector>

#include "graph.h"

namespace dg {

struct Merged {
  std::string a_text, b_text;       // the two trimmed graphs, same leaves
  int trimmed = 0;                  // ops in the common prefix
  std::vector<std::string> shared;  // prefix results that became leaves
};

// Throws Failure(DG_E_SIGNATURE) when the inputs cannot be matched or the
// output shapes differ.  trim_prefix = false matches the inputs only.
Merged merge_graphs(const GraphIR& a, const GraphIR& b, bool trim_prefix);

// dgir v1 text of a graph (leaves, ops in SSA order, output).
std::string graph_text(const GraphIR& g);

}  // namespace dg
