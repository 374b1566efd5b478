// Order in which output locations are checked (Sec. 4, "Search
// Heuristic"): a ranked prefix of corner and boundary locations, then a
// seeded random permutation of the others.  This file builds the prefix on
// the host; the permutation runs on the device (kernels.hip).
//
// Corners.  Every op is taken as one kernel launch writing its output in
// row-major order, one element per thread, `block_threads` threads per
// block.  The corner threads are the first and last thread of the first
// and last block and the lanes `warp - 1` and `warp` of block 0 (where a
// warp-level reduction would change lanes).  A corner thread's element
// becomes an output location when the path from its tensor to the output
// runs through reads that permute dims only (each consumer element reads
// exactly that one element, and no other consumer element reads it): the
// location is then unique along a path, and the smallest over paths is
// taken.  Ops are ranked in reverse SSA order (later launches first), each
// op's corners in the order (thread 0, block 0), (last thread, block 0),
// (thread 0, last block), (last thread, last block), lanes warp - 1 and
// warp of block 0.  The first and last output location follow, then the
// permutation; a location is listed once, at its first rank.
#include <algorithm>
#include <set>
#include <vector>

#include "../../include/dirigo_rocm.h"
#include "order.h"

namespace dg {

namespace {

// Output dim read at each dim of operand `o` of group G when the read is a
// dim permutation of an op output of shape `out` (-1 for a unit dim of the
// operand read at 0; window variables must have one value); false
// otherwise.
bool permuting_read(const ReadGroup& G, const Operand& o, const Dims& tshape, const Dims& out,
                    std::vector<int>* perm) {
  const int R = (int)out.size();
  if (numel(tshape) != numel(out) || o.idx.size() != tshape.size()) return false;
  for (size_t q = 0; q < G.wlo.size(); ++q)
    if (G.whi[q] - G.wlo[q] != 1) return false;
  perm->assign(tshape.size(), -1);
  std::vector<bool> used(R, false);
  for (size_t d = 0; d < o.idx.size(); ++d) {
    const IndexFn& f = o.idx[d];
    if (f.mode != 0) return false;
    int64_t c = f.c;
    int var = -1;
    for (const IndexFn::Term& t : f.terms) {
      if (t.var >= R) {
        const int64_t w = G.wlo[t.var - R];
        if (t.vdiv != 1 && w < 0) return false;
        c += t.coef * (t.vdiv == 1 ? w : w / t.vdiv);
      } else {
        if (t.coef != 1 || t.vdiv != 1 || var >= 0) return false;
        var = t.var;
      }
    }
    if (var < 0 && c == 0 && tshape[d] == 1) continue;  // a unit dim of the operand
    if (c != 0 || var < 0 || used[var] || out[var] != tshape[d]) return false;
    used[var] = true;
    (*perm)[d] = var;
  }
  return true;
}

// An index function whose value lies in [0, size) at every output element
// (a constant in range, or one output variable whose extent fits).
bool always_valid(const ReadGroup& G, const IndexFn& f, const Dims& out, int64_t size) {
  const int R = (int)out.size();
  if (f.mode != 0) return false;
  int64_t lo = f.c, hi = f.c;
  for (const IndexFn::Term& t : f.terms) {
    int64_t a, b;
    if (t.var >= R) {
      a = b = G.wlo[t.var - R];
      if (G.whi[t.var - R] - G.wlo[t.var - R] != 1 || a < 0) return false;
    } else {
      a = 0;
      b = out[t.var] - 1;
    }
    if (t.vdiv != 1) {
      a /= t.vdiv;
      b /= t.vdiv;
    }
    lo += std::min(t.coef * a, t.coef * b);
    hi += std::max(t.coef * a, t.coef * b);
  }
  return lo >= 0 && hi < size;
}

// The dim permutation by which op j reads tensor t element for element, if
// every read of t by op j is that one permutation and the other operands of
// those reads are valid everywhere.
bool op_permutes(const GraphIR& g, const OpNode& op, int t, std::vector<int>* perm) {
  const Dims& out = g.tensors[op.out].shape;
  bool any = false;
  for (const ReadGroup& G : op.groups) {
    bool reads = false;
    for (const Operand& o : G.ops) reads = reads || o.tensor == t;
    if (!reads) continue;
    for (const Operand& o : G.ops) {
      const Dims& s = g.tensors[o.tensor].shape;
      if (o.tensor == t) {
        std::vector<int> p;
        if (!permuting_read(G, o, s, out, &p)) return false;
        if (any && p != *perm) return false;
        *perm = p;
        any = true;
      } else {
        for (size_t d = 0; d < o.idx.size(); ++d)
          if (!always_valid(G, o.idx[d], out, s[d])) return false;
      }
    }
  }
  return any;
}

// Smallest output location reached from element e of tensor t through dim
// permutations; -1 for none.
int64_t forward_location(const GraphIR& g, int t, int64_t e) {
  if (t == g.output) return e;
  int64_t best = -1;
  const Dims& ts = g.tensors[t].shape;
  std::vector<int64_t> coord(ts.size());
  int64_t r = e;
  for (int d = (int)ts.size() - 1; d >= 0; --d) {
    coord[d] = r % ts[d];
    r /= ts[d];
  }
  for (const OpNode& op : g.ops) {
    if (op.kind == "reshape") {
      // A reshape keeps the flat index: element e of its operand is
      // element e of its result, and no other result element reads it.
      if (op.in[0] != t) continue;
      const int64_t l = forward_location(g, op.out, e);
      if (l >= 0 && (best < 0 || l < best)) best = l;
      continue;
    }
    std::vector<int> perm;
    if (!op_permutes(g, op, t, &perm)) continue;
    const Dims& os = g.tensors[op.out].shape;
    std::vector<int64_t> oc(os.size(), 0);
    for (size_t d = 0; d < perm.size(); ++d)
      if (perm[d] >= 0) oc[perm[d]] = coord[d];
    int64_t o = 0;
    for (size_t d = 0; d < os.size(); ++d) o = o * os[d] + oc[d];
    const int64_t l = forward_location(g, op.out, o);
    if (l >= 0 && (best < 0 || l < best)) best = l;
  }
  return best;
}

}  // namespace

std::vector<int64_t> order_prefix(const GraphIR& g, int64_t block_threads, int64_t warp) {
  if (block_threads < 1 || warp < 1) throw Failure(DG_E_INVALID_ARG, "block_threads and warp must be positive");
  std::vector<int64_t> out;
  std::set<int64_t> seen;
  auto add = [&](int64_t l) {
    if (l >= 0 && seen.insert(l).second) out.push_back(l);
  };
  for (int k = (int)g.ops.size() - 1; k >= 0; --k) {
    const int t = g.ops[k].out;
    const int64_t m = numel(g.tensors[t].shape);
    if (m == 0) continue;
    const int64_t blocks = (m + block_threads - 1) / block_threads;
    const int64_t last = (blocks - 1) * block_threads;
    const int64_t elems[6] = {0, block_threads - 1, last, last + block_threads - 1, warp - 1, warp};
    for (int q = 0; q < 6; ++q) {
      const int64_t e = elems[q];
      if (q >= 4 && e >= block_threads) continue;  // lanes of block 0 only
      if (e < m) add(forward_location(g, t, e));
    }
  }
  const int64_t n = numel(g.tensors[g.output].shape);
  if (n > 0) {
    add(0);
    add(n - 1);
  }
  return out;
}

}  // namespace dg
