// Host compiler of the expression-DAG program (dag_program.h, DgdHeader): the
// ops of a graph as read groups with device index functions, element ids of
// every tensor, and static frontier capacities for one location.
#include <algorithm>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/dirigo_rocm.h"
#include "compile.h"
#include "dag_program.h"

namespace dg {

namespace {

[[noreturn]] void fail(int code, const std::string& m) { throw Failure(code, m); }

int32_t i32(int64_t v, const char* what) {
  if (v < INT32_MIN || v > INT32_MAX) fail(DG_E_UNSUPPORTED_OP, std::string(what) + " exceeds 32 bits");
  return (int32_t)v;
}

DgpIFn device_fn(const IndexFn& f, int64_t size) {
  DgpIFn d;
  std::memset(&d, 0, sizeof(d));
  if (f.terms.size() > DGP_MAX_FTERMS) fail(DG_E_UNSUPPORTED_OP, "index function with more than 4 terms");
  d.nterm = (int32_t)f.terms.size();
  for (size_t q = 0; q < f.terms.size(); ++q) {
    d.var[q] = f.terms[q].var;
    d.coef[q] = i32(f.terms[q].coef, "index coefficient");
    d.vdiv[q] = i32(f.terms[q].vdiv, "index divisor");
  }
  d.c = i32(f.c, "index constant");
  d.mode = f.mode;
  d.s = i32(f.s, "index divisor");
  d.size = i32(size, "tensor dimension");
  return d;
}

// floor(2^64 / d) + 1 = ceil(2^64 / d) for d >= 2: the quotient of any
// 32-bit n by d is then the high 64 bits of n * magic (Lemire, Kaser and
// Kurz, "Faster remainder by direct computation", 2019).  0 for d = 1.
uint64_t quotient_magic(int64_t d) { return d <= 1 ? 0 : ~0ull / (uint64_t)d + 1; }

// The one window variable (index into the window) of an index function of a
// group with R output variables; -1 for none, -2 for two or more.
int window_var(const IndexFn& f, int R) {
  int w = -1;
  for (const IndexFn::Term& t : f.terms)
    if (t.var >= R) {
      if (w >= 0 && w != t.var - R) return -2;
      w = t.var - R;
    }
  return w;
}

// Coefficient of window variable q in f when f is c0 + k * w (mode 0) or
// (c0 + k * w) / s exactly (mode 1) with a single unit-divisor term in w;
// 0 otherwise.
int64_t progression_coef(const IndexFn& f, int R, int q) {
  if (f.mode != 0 && f.mode != 1) return 0;
  int n = 0;
  int64_t k = 0;
  for (const IndexFn::Term& t : f.terms)
    if (t.var == R + q) {
      if (t.vdiv != 1) return 0;
      k = t.coef;
      ++n;
    }
  return n == 1 ? k : 0;
}

int64_t gcd64(int64_t a, int64_t b) {
  a = a < 0 ? -a : a;
  b = b < 0 ? -b : b;
  while (b) {
    int64_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

// Inverse of a modulo m (gcd(a, m) = 1, m >= 1); 0 for m = 1.
int64_t mod_inverse(int64_t a, int64_t m) {
  if (m == 1) return 0;
  a %= m;
  if (a < 0) a += m;
  for (int64_t x = 1; x < m; ++x)
    if ((a * x) % m == 1) return x;
  fail(DG_E_UNSUPPORTED_OP, "no modular inverse");
}

// Whether index function f of a group can leave its valid range at some
// node and window point (or, with an exact division and no window
// variable, fail to divide): interval bounds over every output coordinate
// of an op with output shape `out` and every point of the window [wlo,
// whi).  A function that cannot only enters the element indices.
bool can_bind(const IndexFn& f, const Dims& out, const ReadGroup& G, int64_t size, bool window) {
  const int R = (int)out.size();
  int64_t lo = f.c, hi = f.c;
  for (const IndexFn::Term& t : f.terms) {
    int64_t vlo, vhi;
    if (t.var < R) {
      vlo = 0;
      vhi = out[t.var] - 1;
    } else {
      const int q = t.var - R;
      if (q >= (int)G.wlo.size()) return true;
      vlo = G.wlo[q];
      vhi = G.whi[q] - 1;
    }
    if (vhi < vlo) return true;
    if (t.vdiv != 1) {
      // (The device truncates; variables are non-negative.)
      if (vlo < 0 || t.vdiv <= 0) return true;
      vlo /= t.vdiv;
      vhi /= t.vdiv;
    }
    const int64_t a = t.coef * vlo, b = t.coef * vhi;
    lo += std::min(a, b);
    hi += std::max(a, b);
  }
  if (f.mode == 0) return !(lo >= 0 && hi <= size - 1);
  if (f.mode == 1 && window) return !(lo >= 0 && hi <= f.s * (size - 1));  // divisibility: the progression's
  if (f.mode == 1) return f.s != 1 || !(lo >= 0 && hi <= size - 1);
  return true;
}

}  // namespace

DagProgram compile_dag(const GraphIR& g, int nthreads) {
  // Waves of 64 lanes on the device; the host emulation runs one thread.
  const int lanes = nthreads >= 64 ? 64 : 1;
  const int nwaves = nthreads / lanes;
  const int nt = (int)g.tensors.size(), nop = (int)g.ops.size();
  // Element ids: leaves keep theirs, op outputs follow in SSA order.
  std::vector<uint64_t> gid(nt, 0);
  uint64_t next = g.leaf_total;
  for (int t = 0; t < nt; ++t)
    if (g.tensors[t].leaf >= 0) gid[t] = g.tensors[t].base;
  for (const OpNode& op : g.ops) {
    gid[op.out] = next;
    next += (uint64_t)numel(g.tensors[op.out].shape);
  }
  if (next > 0xFFFFFFFFull) fail(DG_E_OVERFLOW, "DAG element ids need more than 32 bits");

  // Static frontier bounds for one location, in reverse SSA order: a
  // tensor's candidate list receives, from every node of a consumer, one
  // entry per window point of every group operand that reads it.
  std::vector<uint64_t> appends(nt, 0), nodes(nt, 0);
  if (g.tensors[g.output].leaf < 0) appends[g.output] = 1;
  DagProgram p;
  int max_vars = 1;
  for (int k = nop - 1; k >= 0; --k) {
    const OpNode& op = g.ops[k];
    const uint64_t n = std::min<uint64_t>(appends[op.out], (uint64_t)numel(g.tensors[op.out].shape));
    nodes[op.out] = n;
    p.max_nodes += (int64_t)n;
    const int R = (int)g.tensors[op.out].shape.size();
    for (const ReadGroup& G : op.groups) {
      uint64_t pts = 1;
      for (size_t q = 0; q < G.wlo.size(); ++q) pts *= (uint64_t)std::max<int64_t>(0, G.whi[q] - G.wlo[q]);
      max_vars = std::max(max_vars, R + (int)G.wlo.size());
      p.max_edges += (int64_t)(n * pts * G.ops.size());
      for (const Operand& o : G.ops)
        if (g.tensors[o.tensor].leaf < 0) appends[o.tensor] += n * pts;
    }
  }

  // Layout of one location's LDS area: frontiers (u32 entries, sorted in
  // place), then one counter per tensor, the per-thread variable tables, the
  // per-node edge counts, the per-thread node slots and the per-wave prefix
  // arrays.
  std::vector<DgdTensor> T(nt);
  uint64_t lds = 0;
  for (int t = 0; t < nt; ++t) {
    DgdTensor& d = T[t];
    std::memset(&d, 0, sizeof(d));
    const Tensor& x = g.tensors[t];
    d.rank = (int32_t)x.shape.size();
    d.leaf = x.leaf >= 0 ? 1 : 0;
    d.gid = (uint32_t)gid[t];
    d.numel = i32(numel(x.shape), "tensor size");
    int64_t st = 1;
    for (int q = (int)x.shape.size() - 1; q >= 0; --q) {
      d.shape[q] = (int32_t)x.shape[q];
      d.stride[q] = (uint32_t)st;
      d.magic[q] = quotient_magic(x.shape[q]);
      st *= x.shape[q];
    }
    d.lds = -1;
    if (!d.leaf && appends[t] > 0) {
      const uint64_t cap = appends[t];
      if (cap > (1u << 20)) fail(DG_E_CAPACITY, "DAG frontier of '" + x.name + "' exceeds 2^20 elements");
      d.cap = (int32_t)cap;
      d.lds = (int32_t)lds;
      lds += 4 * cap;
    }
  }
  // Edge counts: one per node of a pointwise op, one per batch of `lanes`
  // nodes otherwise.
  for (int t = 0; t < nt; ++t) p.max_frontier = std::max<int64_t>(p.max_frontier, T[t].cap);
  int64_t ncount_cap = 1;
  for (const OpNode& op : g.ops) {
    bool pointwise = true;
    for (const ReadGroup& G : op.groups)
      if (!G.wlo.empty()) pointwise = false;
    const int64_t cap = T[op.out].cap;
    ncount_cap = std::max<int64_t>(ncount_cap, pointwise ? cap : (cap + lanes - 1) / lanes);
  }
  const uint64_t count_off = lds;
  lds += 4 * (uint64_t)nt;
  lds = (lds + 7) & ~7ull;
  p.vars_off = (uint32_t)lds;
  p.max_vars = max_vars;
  lds += 4ull * (uint64_t)max_vars * (uint64_t)nthreads;
  const uint64_t ncount_off = lds;
  lds += 4ull * (uint64_t)ncount_cap;

  std::vector<DgdOp> O(nop);
  std::vector<DgdGroup> Gs;
  int max_win = 1, max_opnd = 1;
  std::vector<DgdOperand> Ps;
  for (int k = 0; k < nop; ++k) {
    const OpNode& op = g.ops[k];
    DgdOp& d = O[k];
    std::memset(&d, 0, sizeof(d));
    d.out = op.out;
    d.g0 = (int32_t)Gs.size();
    d.ng = (int32_t)op.groups.size();
    for (const ReadGroup& G : op.groups) {
      DgdGroup e;
      std::memset(&e, 0, sizeof(e));
      if (G.wlo.size() > DGD_MAX_WIN) fail(DG_E_UNSUPPORTED_OP, op.kind + ": window with more than 8 dims");
      if (G.ops.size() > DGD_MAX_OPERANDS) fail(DG_E_UNSUPPORTED_OP, op.kind + ": more than 8 operands in a group");
      e.nwin = (int32_t)G.wlo.size();
      e.nop = (int32_t)G.ops.size();
      e.op0 = (int32_t)Ps.size();
      const int R = (int)g.tensors[op.out].shape.size();
      // Progressions: every index function uses at most one window
      // variable, in a single unit-divisor term, with no floor division;
      // at most one exact division per variable.
      bool fast = true;
      int npair = 0;
      for (int q = 0; q < (int)G.wlo.size(); ++q) {
        e.step[q] = 1;
        e.mpair[q] = -1;
      }
      for (size_t a = 0; a < G.ops.size(); ++a)
        for (size_t d = 0; d < G.ops[a].idx.size(); ++d) {
          const IndexFn& f = G.ops[a].idx[d];
          const int q = window_var(f, R);
          if (q == -2) {
            fast = false;
            continue;
          }
          if (npair < DGD_MAX_PAIRS) {
            const int64_t size = g.tensors[G.ops[a].tensor].shape[d];
            const bool bind = can_bind(f, g.tensors[op.out].shape, G, size, q >= 0);
            DgdPair pr;
            std::memset(&pr, 0, sizeof(pr));
            pr.a = (int32_t)a;
            pr.d = (int32_t)d;
            pr.q = (int32_t)q;
            pr.bind = bind ? 1 : 0;
            int64_t st = 1;
            for (size_t d2 = d + 1; d2 < g.tensors[G.ops[a].tensor].shape.size(); ++d2)
              st *= g.tensors[G.ops[a].tensor].shape[d2];
            pr.stride = (uint32_t)st;
            e.pair[npair] = pr;
          }
          if (q >= 0) {
            const int64_t k = progression_coef(f, R, q);
            if (k == 0) {
              fast = false;
            } else if (f.mode == 1) {
              if (e.mpair[q] >= 0) fast = false;
              const int64_t gk = gcd64(k, f.s);
              e.mpair[q] = npair;
              e.step[q] = (int32_t)(f.s / gk);
              e.minv[q] = (int32_t)mod_inverse(k / gk, f.s / gk);
            }
          }
          ++npair;
        }
      if (npair > DGD_MAX_PAIRS) fast = false;
      e.fast = fast ? 1 : 0;
      e.npair = fast ? npair : 0;
      if (fast) {
        // The pairs that can bind first (in their order), the others after;
        // the exact-division pairs renumbered to match.
        std::vector<int> order;
        for (int pi = 0; pi < npair; ++pi)
          if (e.pair[pi].bind) order.push_back(pi);
        e.nbind = (int32_t)order.size();
        for (int pi = 0; pi < npair; ++pi)
          if (!e.pair[pi].bind) order.push_back(pi);
        std::vector<int> where(npair);
        DgdPair sorted[DGD_MAX_PAIRS];
        std::memset(sorted, 0, sizeof(sorted));
        for (int k2 = 0; k2 < npair; ++k2) {
          sorted[k2] = e.pair[order[k2]];
          where[order[k2]] = k2;
        }
        std::memcpy(e.pair, sorted, sizeof(sorted));
        for (size_t q = 0; q < G.wlo.size(); ++q)
          if (e.mpair[q] >= 0) e.mpair[q] = where[e.mpair[q]];
      }
      if (fast) {
        // Element-index steps per progression step.
        for (size_t a = 0; a < G.ops.size(); ++a) {
          const Dims& sh = g.tensors[G.ops[a].tensor].shape;
          int64_t st = 1;
          for (int d = (int)sh.size() - 1; d >= 0; --d) {
            const IndexFn& f = G.ops[a].idx[d];
            const int q = window_var(f, R);
            if (q >= 0) {
              const int64_t k = progression_coef(f, R, q);
              const int64_t per = f.mode == 1 ? k * e.step[q] / f.s : k * e.step[q];
              e.astep[a][q] += (uint32_t)(st * per);
            }
            st *= sh[d];
          }
        }
        e.steps24 = 1;
        for (size_t a = 0; a < G.ops.size(); ++a)
          for (size_t q = 0; q < G.wlo.size(); ++q) {
            const int32_t v = (int32_t)e.astep[a][q];
            if (v < -(1 << 23) || v >= (1 << 23)) e.steps24 = 0;
          }
        max_win = std::max(max_win, (int)G.wlo.size());
        max_opnd = std::max(max_opnd, (int)G.ops.size());
      }
      int64_t pts = 1;
      for (size_t q = 0; q < G.wlo.size(); ++q) {
        e.wlo[q] = i32(G.wlo[q], "window bound");
        e.whi[q] = i32(G.whi[q], "window bound");
        pts *= std::max<int64_t>(0, G.whi[q] - G.wlo[q]);
      }
      e.points = pts;
      d.refs += pts * (int64_t)G.ops.size();
      for (const Operand& o : G.ops) {
        DgdOperand P;
        std::memset(&P, 0, sizeof(P));
        P.tensor = o.tensor;
        if (g.tensors[o.tensor].leaf < 0) d.nonleaf = 1;
        if (o.mult > 0xFFFFFFFFull) fail(DG_E_OVERFLOW, op.kind + ": multiplicity exceeds 32 bits");
        P.mult = (uint32_t)o.mult;
        const Dims& s = g.tensors[o.tensor].shape;
        for (size_t q = 0; q < s.size(); ++q) P.idx[q] = device_fn(o.idx[q], s[q]);
        Ps.push_back(P);
      }
      Gs.push_back(e);
    }
    d.pointwise = 1;
    for (const ReadGroup& G : op.groups)
      if (!G.wlo.empty()) d.pointwise = 0;
  }
  // Per-thread node slots (per window variable: first value and count; per
  // operand: element index at the first point; the 64-bit first edge), then
  // one prefix word per lane of every wave.
  const int slot_words = 2 * max_win + max_opnd + 2;
  const uint64_t slot_off = lds;
  lds += 4ull * (uint64_t)slot_words * (uint64_t)nthreads;
  const uint64_t wave_off = lds;
  lds += 4ull * (uint64_t)lanes * (uint64_t)nwaves;
  if (lds > (1u << 30)) fail(DG_E_CAPACITY, "DAG frontiers too large");

  DgdHeader h;
  std::memset(&h, 0, sizeof(h));
  h.magic = DGD_MAGIC;
  h.ntensor = nt;
  h.nop = nop;
  h.ngroup = (int32_t)Gs.size();
  h.noperand = (int32_t)Ps.size();
  size_t off = (sizeof(DgdHeader) + 15) & ~(size_t)15;
  h.tensor_off = (int32_t)off;
  off += sizeof(DgdTensor) * T.size();
  off = (off + 15) & ~(size_t)15;
  h.op_off = (int32_t)off;
  off += sizeof(DgdOp) * O.size();
  off = (off + 15) & ~(size_t)15;
  h.group_off = (int32_t)off;
  off += sizeof(DgdGroup) * Gs.size();
  off = (off + 15) & ~(size_t)15;
  h.operand_off = (int32_t)off;
  off += sizeof(DgdOperand) * Ps.size();
  h.blob_bytes = (int32_t)off;
  h.output = g.output;
  h.count_off = (int32_t)count_off;
  h.lds_bytes = (int32_t)lds;
  h.vars_off = (int32_t)p.vars_off;
  h.max_vars = max_vars;
  h.out_numel = numel(g.tensors[g.output].shape);
  h.ncount_off = (int32_t)ncount_off;
  h.ncount_cap = (int32_t)ncount_cap;
  h.slot_off = (int32_t)slot_off;
  h.slot_words = slot_words;
  h.wave_off = (int32_t)wave_off;
  h.max_win = max_win;
  h.max_opnd = max_opnd;
  p.blob.assign(off, 0);
  std::memcpy(p.blob.data(), &h, sizeof(h));
  if (!T.empty()) std::memcpy(p.blob.data() + h.tensor_off, T.data(), sizeof(DgdTensor) * T.size());
  if (!O.empty()) std::memcpy(p.blob.data() + h.op_off, O.data(), sizeof(DgdOp) * O.size());
  if (!Gs.empty()) std::memcpy(p.blob.data() + h.group_off, Gs.data(), sizeof(DgdGroup) * Gs.size());
  if (!Ps.empty()) std::memcpy(p.blob.data() + h.operand_off, Ps.data(), sizeof(DgdOperand) * Ps.size());
  p.lds_bytes = (uint32_t)lds;
  p.gid = gid;
  return p;
}

}  // namespace dg
