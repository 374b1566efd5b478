// MERGE (Sec. 3.2): one checking obligation from two programs.  The inputs
// of the two programs are matched, so that the same inputs should give the
// same output, and a common prefix of ops is trimmed.  The trimmed ops'
// results that are still read become shared inputs.  Only the prefix is
// trimmed, never a common suffix, as the paper does.
//
// Input matching.  A leaf of B matches the leaf of A with the same name and
// shape; the leaves left over match in declaration order among leaves of the
// same shape.  Any leaf left without a partner, in either graph, is an error
// (the two programs would not take the same inputs).
//
// Prefix.  Op i of A and op i of B match when they have the same kind, the
// same attributes and operands that match (matched leaves, or results of
// earlier matched ops).  The prefix is the longest run of matching ops from
// the first.
//
// Result.  Two graphs over the same leaves, in A's order and under A's
// names: A's leaves, then the prefix results that an op left in either graph
// reads, or that is an output, in prefix order.  The ops after the prefix
// follow in each graph; B's own tensors keep their names unless one clashes
// with a leaf name, which then gets a suffix.
#include <map>
#include <set>
#include <sstream>
#include <string>
#include <vector>

#include "../../include/dirigo_rocm.h"
#include "merge.h"

namespace dg {

namespace {

std::string csv(const Dims& d) {
  std::ostringstream o;
  for (size_t i = 0; i < d.size(); ++i) o << (i ? "," : "") << d[i];
  return o.str();
}

std::string attr_text(const OpNode& op) {
  std::ostringstream o;
  bool first = true;
  for (const auto& kv : op.ints) {
    o << (first ? "" : " ") << kv.first << "=" << csv(kv.second);
    first = false;
  }
  for (const auto& kv : op.exprs) {
    o << (first ? "" : " ") << kv.first << "=";
    for (size_t i = 0; i < kv.second.size(); ++i) o << (i ? "," : "") << kv.second[i];
    first = false;
  }
  return o.str();
}

bool same_op(const OpNode& x, const OpNode& y) {
  return x.kind == y.kind && x.ints == y.ints && x.exprs == y.exprs && x.in.size() == y.in.size();
}

}  // namespace

std::string graph_text(const GraphIR& g) {
  std::ostringstream o;
  o << "dgir 1\n";
  for (int t : g.leaves) o << "leaf " << g.tensors[t].name << " " << csv(g.tensors[t].shape) << "\n";
  for (const OpNode& op : g.ops) {
    o << "op " << g.tensors[op.out].name << " " << op.kind;
    for (int t : op.in) o << " " << g.tensors[t].name;
    const std::string a = attr_text(op);
    if (!a.empty()) o << " ; " << a;
    o << "\n";
  }
  o << "output " << g.tensors[g.output].name << " " << csv(g.tensors[g.output].shape) << "\n";
  return o.str();
}

Merged merge_graphs(const GraphIR& a, const GraphIR& b, bool trim_prefix) {
  // Inputs: by name and shape first, then by shape in declaration order.
  std::vector<int> b_of_a(a.leaves.size(), -1), a_of_b(b.leaves.size(), -1);
  for (size_t j = 0; j < b.leaves.size(); ++j) {
    const Tensor& tb = b.tensors[b.leaves[j]];
    for (size_t i = 0; i < a.leaves.size(); ++i) {
      const Tensor& ta = a.tensors[a.leaves[i]];
      if (b_of_a[i] < 0 && ta.name == tb.name && ta.shape == tb.shape) {
        b_of_a[i] = (int)j;
        a_of_b[j] = (int)i;
        break;
      }
    }
  }
  for (size_t j = 0; j < b.leaves.size(); ++j) {
    if (a_of_b[j] >= 0) continue;
    const Tensor& tb = b.tensors[b.leaves[j]];
    for (size_t i = 0; i < a.leaves.size(); ++i)
      if (b_of_a[i] < 0 && a.tensors[a.leaves[i]].shape == tb.shape) {
        b_of_a[i] = (int)j;
        a_of_b[j] = (int)i;
        break;
      }
    if (a_of_b[j] < 0)
      throw Failure(DG_E_SIGNATURE, "input '" + tb.name + "' of the second graph has no partner of its shape");
  }
  for (size_t i = 0; i < a.leaves.size(); ++i)
    if (b_of_a[i] < 0)
      throw Failure(DG_E_SIGNATURE, "input '" + a.tensors[a.leaves[i]].name + "' of the first graph has no partner");
  if (a.tensors[a.output].shape != b.tensors[b.output].shape) throw Failure(DG_E_SIGNATURE, "output shape differs");

  // Tensor of A that each tensor of B stands for (leaves, prefix results).
  std::vector<int> a_for(b.tensors.size(), -1);
  for (size_t j = 0; j < b.leaves.size(); ++j) a_for[b.leaves[j]] = a.leaves[a_of_b[j]];
  size_t k = 0;
  while (trim_prefix && k < a.ops.size() && k < b.ops.size()) {
    const OpNode &x = a.ops[k], &y = b.ops[k];
    bool ok = same_op(x, y);
    for (size_t q = 0; ok && q < x.in.size(); ++q) ok = a_for[y.in[q]] == x.in[q];
    if (!ok) break;
    a_for[y.out] = x.out;
    ++k;
  }

  // Prefix results still needed: read after the prefix, or an output.
  std::set<int> need;  // tensors of A
  for (size_t i = k; i < a.ops.size(); ++i)
    for (int t : a.ops[i].in)
      if (a.tensors[t].producer >= 0 && a.tensors[t].producer < (int)k) need.insert(t);
  for (size_t i = k; i < b.ops.size(); ++i)
    for (int t : b.ops[i].in)
      if (b.tensors[t].producer >= 0 && b.tensors[t].producer < (int)k) need.insert(a_for[t]);
  if (a.tensors[a.output].producer >= 0 && a.tensors[a.output].producer < (int)k) need.insert(a.output);
  if (b.tensors[b.output].producer >= 0 && b.tensors[b.output].producer < (int)k) need.insert(a_for[b.output]);

  Merged m;
  m.trimmed = (int)k;
  std::ostringstream la;  // the shared leaf block
  std::set<std::string> leaf_names;
  for (int t : a.leaves) {
    la << "leaf " << a.tensors[t].name << " " << csv(a.tensors[t].shape) << "\n";
    leaf_names.insert(a.tensors[t].name);
  }
  for (size_t i = 0; i < k; ++i) {
    const int t = a.ops[i].out;
    if (!need.count(t)) continue;
    la << "leaf " << a.tensors[t].name << " " << csv(a.tensors[t].shape) << "\n";
    leaf_names.insert(a.tensors[t].name);
    m.shared.push_back(a.tensors[t].name);
  }

  // A after the prefix.
  std::ostringstream oa;
  oa << "dgir 1\n" << la.str();
  for (size_t i = k; i < a.ops.size(); ++i) {
    const OpNode& op = a.ops[i];
    oa << "op " << a.tensors[op.out].name << " " << op.kind;
    for (int t : op.in) oa << " " << a.tensors[t].name;
    const std::string at = attr_text(op);
    if (!at.empty()) oa << " ; " << at;
    oa << "\n";
  }
  oa << "output " << a.tensors[a.output].name << " " << csv(a.tensors[a.output].shape) << "\n";
  m.a_text = oa.str();

  // B after the prefix, its inputs under A's names.
  std::vector<std::string> bname(b.tensors.size());
  std::set<std::string> used = leaf_names;
  for (size_t t = 0; t < b.tensors.size(); ++t) {
    if (a_for[t] >= 0) {
      bname[t] = a.tensors[a_for[t]].name;
      continue;
    }
    std::string nm = b.tensors[t].name;
    for (int s = 1; used.count(nm); ++s) nm = b.tensors[t].name + "_" + std::to_string(s);
    used.insert(nm);
    bname[t] = nm;
  }
  std::ostringstream ob;
  ob << "dgir 1\n" << la.str();
  for (size_t i = k; i < b.ops.size(); ++i) {
    const OpNode& op = b.ops[i];
    ob << "op " << bname[op.out] << " " << op.kind;
    for (int t : op.in) ob << " " << bname[t];
    const std::string at = attr_text(op);
    if (!at.empty()) ob << " ; " << at;
    ob << "\n";
  }
  ob << "output " << bname[b.output] << " " << csv(b.tensors[b.output].shape) << "\n";
  m.b_text = ob.str();
  return m;
}

}  // namespace dg
