// Merged-dim views of a graph (see view.h).
#include "view.h"

#include <algorithm>
#include <map>
#include <numeric>

#include "../../include/dirigo_rocm.h"

namespace dg {

namespace {

[[noreturn]] void fail(const std::string& m) { throw Failure(DG_E_UNSUPPORTED_OP, m); }

int64_t floor_div(int64_t a, int64_t b) {
  int64_t q = a / b;
  if ((a % b) != 0 && ((a < 0) != (b < 0))) --q;
  return q;
}

struct UnionFind {
  std::vector<int> p;
  explicit UnionFind(int n) : p(n) { std::iota(p.begin(), p.end(), 0); }
  int find(int x) { return p[x] == x ? x : p[x] = find(p[x]); }
  void unite(int a, int b) { p[find(a)] = find(b); }
};

// [first dim, end dim) of every group of a partition.
std::vector<std::pair<int, int>> groups_of(const std::vector<int>& part) {
  std::vector<std::pair<int, int>> g;
  for (int d = 0; d < (int)part.size(); ++d) {
    if (d == 0 || part[d] != part[d - 1]) g.push_back({d, d + 1});
    else g.back().second = d + 1;
  }
  return g;
}

bool is_identity(const std::vector<int>& part) {
  for (int d = 0; d < (int)part.size(); ++d)
    if (part[d] != d) return false;
  return true;
}

// Terms of one variable and divisor added up; zero terms dropped.
IndexFn combined(const IndexFn& f) {
  IndexFn r;
  r.c = f.c;
  r.mode = f.mode;
  r.s = f.s;
  for (const auto& t : f.terms) {
    bool found = false;
    for (auto& u : r.terms)
      if (u.var == t.var && u.vdiv == t.vdiv) {
        u.coef += t.coef;
        found = true;
      }
    if (!found) r.terms.push_back(t);
  }
  r.terms.erase(std::remove_if(r.terms.begin(), r.terms.end(), [](const IndexFn::Term& t) { return t.coef == 0; }),
                r.terms.end());
  return r;
}

bool same_fn(const IndexFn& a, const IndexFn& b) {
  if (a.c != b.c || a.mode != b.mode || a.s != b.s || a.terms.size() != b.terms.size()) return false;
  for (size_t q = 0; q < a.terms.size(); ++q)
    if (a.terms[q].var != b.terms[q].var || a.terms[q].coef != b.terms[q].coef || a.terms[q].vdiv != b.terms[q].vdiv)
      return false;
  return true;
}

// Range of f over the variables' boxes (as the plan compiler bounds it).
std::pair<int64_t, int64_t> fn_range(const IndexFn& f, const std::vector<int64_t>& vmin,
                                     const std::vector<int64_t>& vmax) {
  int64_t lo = f.c, hi = f.c;
  for (const auto& t : f.terms) {
    int64_t a = floor_div(vmin[t.var], t.vdiv), b = floor_div(vmax[t.var], t.vdiv);
    if (t.coef >= 0) {
      lo += t.coef * a;
      hi += t.coef * b;
    } else {
      lo += t.coef * b;
      hi += t.coef * a;
    }
  }
  if (f.mode == 1) return {-floor_div(-lo, f.s), floor_div(hi, f.s)};
  if (f.mode == 2) return {floor_div(lo, f.s), floor_div(hi, f.s)};
  return {lo, hi};
}

// Range of a division-free index function over the merged output
// coordinates [0, size) and the group's window boxes.
std::pair<int64_t, int64_t> var_range(const IndexFn& f, const std::vector<int64_t>& oc_size, const ReadGroup& G) {
  const int Rc = (int)oc_size.size();
  std::vector<int64_t> vmin, vmax;
  for (int64_t n : oc_size) {
    vmin.push_back(0);
    vmax.push_back(n - 1);
  }
  for (size_t b = 0; b < G.wlo.size(); ++b) {
    vmin.push_back(G.wlo[b]);
    vmax.push_back(G.whi[b] - 1);
  }
  (void)Rc;
  return fn_range(f, vmin, vmax);
}

// The graph over partition P.
GraphIR build(const GraphIR& g, const DimPartition& P) {
  GraphIR c = g;
  for (size_t t = 0; t < g.tensors.size(); ++t) {
    Dims s;
    for (auto& gr : groups_of(P[t])) {
      int64_t n = 1;
      for (int d = gr.first; d < gr.second; ++d) n *= g.tensors[t].shape[d];
      if (n >= (int64_t(1) << 31)) fail("a merged dim of '" + g.tensors[t].name + "' holds 2^31 or more elements");
      s.push_back(n);
    }
    c.tensors[t].shape = s;
  }
  for (size_t k = 0; k < g.ops.size(); ++k) {
    const OpNode& op = g.ops[k];
    const int R = (int)g.tensors[op.out].shape.size();
    const std::vector<int>& Po = P[op.out];
    const auto og = groups_of(Po);
    const int Rc = (int)og.size();
    const Dims& oshape = g.tensors[op.out].shape;
    // Output coordinate a in terms of the merged coordinate m of its group.
    auto subst = [&](const IndexFn& f) {
      IndexFn r;
      r.c = f.c;
      r.mode = f.mode;
      r.s = f.s;
      for (const auto& t : f.terms) {
        if (t.var >= R) {
          r.terms.push_back({t.var - R + Rc, t.coef, t.vdiv});
          continue;
        }
        const int a = t.var, m = Po[a];
        const int ga = og[m].first, gb = og[m].second;
        if (gb - ga == 1) {
          r.terms.push_back({m, t.coef, t.vdiv});
          continue;
        }
        int64_t st = 1;
        for (int e = a + 1; e < gb; ++e) st *= oshape[e];
        const int64_t sa = oshape[a];
        if (t.vdiv == 1) {
          r.terms.push_back({m, t.coef, st});
          if (a != ga) r.terms.push_back({m, -t.coef * sa, st * sa});
        } else if (a == ga) {
          r.terms.push_back({m, t.coef, st * t.vdiv});
        } else if (sa % t.vdiv == 0) {
          // floor((floor(m / st) mod sa) / q) = floor(m / (st q)) mod (sa / q)
          r.terms.push_back({m, t.coef, st * t.vdiv});
          r.terms.push_back({m, -t.coef * (sa / t.vdiv), st * sa});
        } else {
          fail(op.kind + ": a merged output coordinate is divided inside its group");
        }
      }
      return combined(r);
    };
    OpNode& cop = c.ops[k];
    std::vector<int64_t> oc_size;  // extent of each merged output coordinate
    for (auto& gr : og) {
      int64_t n = 1;
      for (int d = gr.first; d < gr.second; ++d) n *= oshape[d];
      oc_size.push_back(n);
    }
    for (size_t gi = 0; gi < op.groups.size(); ++gi) {
      const ReadGroup& G = op.groups[gi];
      ReadGroup& CG = cop.groups[gi];
      CG.guards.clear();
      auto add_guard = [&](const IndexFn& f, int64_t size) {
        // (A constant guard is kept too: out of range, it makes the group
        // read nothing.)
        for (const auto& e : CG.guards)
          if (e.second == size && same_fn(e.first, f)) return;
        CG.guards.push_back({f, size});
      };
      for (const auto& gd : G.guards) add_guard(subst(gd.first), gd.second);
      for (size_t r = 0; r < G.ops.size(); ++r) {
        const Operand& o = G.ops[r];
        const Dims& us = g.tensors[o.tensor].shape;
        std::vector<IndexFn> sf;
        for (const IndexFn& f : o.idx) sf.push_back(subst(f));
        Operand& co = CG.ops[r];
        co.idx.clear();
        for (auto& gr : groups_of(P[o.tensor])) {
          if (gr.second - gr.first == 1) {
            co.idx.push_back(sf[gr.first]);
            continue;
          }
          IndexFn m;
          int64_t w = 1;
          for (int d = gr.second - 1; d >= gr.first; --d) {
            IndexFn f = sf[d];
            if (f.mode != 0 && !f.terms.empty()) {
              // An index (e)/s or (e)//s inside a merged dim: its quotient
              // becomes a window variable q of the group, pinned by the
              // guard e - s q in [0, 1) (exact) or [0, s) (floor).
              IndexFn inner = f;
              inner.mode = 0;
              inner.s = 1;
              auto rg = var_range(inner, oc_size, CG);
              const int q = Rc + (int)CG.wlo.size();
              CG.wlo.push_back(floor_div(rg.first, f.s));
              CG.whi.push_back(floor_div(rg.second, f.s) + 1);
              inner.terms.push_back({q, -f.s, 1});
              add_guard(inner, f.mode == 1 ? 1 : f.s);
              f = IndexFn::var(q);
            } else if (f.mode != 0) {
              // A constant: evaluate the division here.
              const int64_t v = f.c;
              if (f.mode == 1 && floor_div(v, f.s) * f.s != v) {
                f = IndexFn::constant(-1);  // not divisible: reads nothing
              } else {
                f = IndexFn::constant(floor_div(v, f.s));
              }
            }
            for (const auto& t : f.terms) m.terms.push_back({t.var, t.coef * w, t.vdiv});
            m.c += f.c * w;
            add_guard(f, us[d]);
            w *= us[d];
          }
          co.idx.push_back(combined(m));
        }
      }
    }
  }
  return c;
}

// Grows P where a read of the graph over P couples two merged dims of one
// operand; returns whether anything changed.
bool grow(const GraphIR& c, DimPartition& P) {
  for (const OpNode& op : c.ops) {
    const Dims& oshape = c.tensors[op.out].shape;
    const int R = (int)oshape.size();
    for (const ReadGroup& G : op.groups) {
      const int Q = (int)G.wlo.size(), NV = R + Q;
      std::vector<int64_t> vmin(NV), vmax(NV);
      bool empty = false;
      for (int a = 0; a < R; ++a) {
        vmin[a] = 0;
        vmax[a] = oshape[a] - 1;
      }
      for (int b = 0; b < Q; ++b) {
        if (G.whi[b] <= G.wlo[b]) empty = true;
        vmin[R + b] = G.wlo[b];
        vmax[R + b] = G.whi[b] - 1;
      }
      if (empty) continue;
      // The validity predicates of the whole group, as the plan compiler
      // takes them: index functions not valid everywhere.
      std::vector<const IndexFn*> preds;
      auto consider = [&](const IndexFn& f, int64_t size) {
        if (f.terms.empty()) return;
        auto rg = fn_range(f, vmin, vmax);
        const bool trivial = (f.mode != 1 || f.s == 1) && rg.first >= 0 && rg.second <= size - 1;
        if (!trivial) preds.push_back(&f);
      };
      for (const Operand& o : G.ops) {
        const Dims& s = c.tensors[o.tensor].shape;
        for (size_t d = 0; d < s.size(); ++d) consider(o.idx[d], s[d]);
      }
      for (const auto& gd : G.guards) consider(gd.first, gd.second);
      for (const Operand& o : G.ops) {
        UnionFind uf(NV);
        for (const IndexFn* p : preds)
          for (size_t q = 1; q < p->terms.size(); ++q) uf.unite(p->terms[0].var, p->terms[q].var);
        for (const IndexFn& f : o.idx)
          for (size_t q = 1; q < f.terms.size(); ++q) uf.unite(f.terms[0].var, f.terms[q].var);
        std::map<int, std::vector<int>> dims;  // component root -> merged dims of o it feeds
        for (size_t d = 0; d < o.idx.size(); ++d)
          if (!o.idx[d].terms.empty()) dims[uf.find(o.idx[d].terms[0].var)].push_back((int)d);
        for (auto& e : dims) {
          if (e.second.size() < 2) continue;
          // Merge groups lo..hi of the operand (and the groups between).
          const int lo = e.second.front(), hi = e.second.back();
          std::vector<int>& part = P[o.tensor];
          for (int& x : part) {
            if (x > lo && x <= hi) x = lo;
            else if (x > hi) x -= hi - lo;
          }
          return true;  // group numbers moved: look again over the new view
        }
      }
    }
  }
  return false;
}

}  // namespace

DimPartition identity_partition(const GraphIR& g) {
  DimPartition P(g.tensors.size());
  for (size_t t = 0; t < g.tensors.size(); ++t) {
    P[t].resize(g.tensors[t].shape.size());
    std::iota(P[t].begin(), P[t].end(), 0);
  }
  return P;
}

MergedView merged_view(const GraphIR& g, const DimPartition* start) {
  MergedView v;
  v.part = start ? *start : identity_partition(g);
  bool all_identity = true;
  for (const auto& p : v.part) all_identity = all_identity && is_identity(p);
  GraphIR c = all_identity ? g : build(g, v.part);
  // Merging only ever coarsens a partition, so this ends.
  while (grow(c, v.part)) c = build(g, v.part);
  v.ir = std::move(c);
  return v;
}

std::vector<int> join_partition(const std::vector<int>& a, const std::vector<int>& b) {
  // A group boundary stays only where both partitions have one.
  std::vector<int> r(a.size());
  for (size_t d = 0; d < a.size(); ++d) {
    const bool cut = d == 0 || (a[d] != a[d - 1] && b[d] != b[d - 1]);
    r[d] = d == 0 ? 0 : r[d - 1] + (cut ? 1 : 0);
  }
  return r;
}

}  // namespace dg
