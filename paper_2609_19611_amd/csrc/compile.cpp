// Host compiler: graph IR -> per-location plan of separable terms.
//
// The back-projection res(y[l]) of Sec. 3.4 is evaluated symbolically once
// for a generic location.  The path-count function of each reached tensor is
// a sum of terms coef * prod_d f_d(i_d).  Substituting op k's per-element
// equation into a term of T_k: for a read group (window box W, operands) and
// an operand r, the count at r's index is
//     sum over output coords o and window points w with r's index = i and
//     every operand index valid, of coef * prod_a f_a(o_a).
// The variables (o_a, w_b) split into components linked by the validity
// predicates and by r's own index functions; each component carries at most
// one dimension of r (else the dataflow is not separable and the graph is
// rejected), so the sum factors into one vector per dimension of r times
// scalar sums.  Terms that agree in all but one factor are merged, which
// keeps the term count small (e.g. a softmax row plus its own element, or a
// normalisation's statistics set plus its own element).
#include "compile.h"
#include "view.h"

#include <algorithm>
#include <array>
#include <climits>
#include <cmath>
#include <cstring>
#include <map>
#include <numeric>
#include <sstream>

#include "../../include/dirigo_rocm.h"

namespace dg {

namespace {

[[noreturn]] void fail(int code, const std::string& m) { throw Failure(code, m); }

const int kMaxTensorTerms = 64;
const int64_t kLincombFullDim = 4096;  // dims up to this size get full-extent merged factors
const int64_t kMaxTableEntries = 8192;
const int64_t kMaxTableWords = 24576;

int64_t floor_div(int64_t a, int64_t b) {
  int64_t q = a / b;
  if ((a % b) != 0 && ((a < 0) != (b < 0))) --q;
  return q;
}
int64_t ceil_div(int64_t a, int64_t b) { return -floor_div(-a, b); }

struct Coef {
  uint64_t k = 1;
  std::vector<int> slots;  // scalar slots, multiplied
};

struct SymTerm {
  Coef coef;
  std::vector<int> f;  // factor slot per dim
};

struct UnionFind {
  std::vector<int> p;
  explicit UnionFind(int n) : p(n) { std::iota(p.begin(), p.end(), 0); }
  int find(int x) { return p[x] == x ? x : p[x] = find(p[x]); }
  void unite(int a, int b) { p[find(a)] = find(b); }
};

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
  if (f.mode == 1) return {ceil_div(lo, f.s), floor_div(hi, f.s)};
  if (f.mode == 2) return {floor_div(lo, f.s), floor_div(hi, f.s)};
  return {lo, hi};
}

// Largest magnitude of any partial sum while evaluating f (int32 safety).
int64_t fn_magnitude(const IndexFn& f, const std::vector<int64_t>& vmin, const std::vector<int64_t>& vmax) {
  int64_t m = std::llabs(f.c);
  for (const auto& t : f.terms) {
    int64_t v = std::max(std::llabs(vmin[t.var]), std::llabs(vmax[t.var]));
    m += std::llabs(t.coef) * (v / t.vdiv + 1);
  }
  return m;
}

bool fn_uses(const IndexFn& f, int v) {
  for (const auto& t : f.terms)
    if (t.var == v) return true;
  return false;
}

// Static bounds are unsigned 64-bit integers that saturate at kBoundMax
// (a bound that large means "2^64 - 1 or more").
const uint64_t kBoundMax = ~uint64_t(0);
uint64_t bmul(uint64_t a, uint64_t b) {
  uint64_t r;
  return __builtin_mul_overflow(a, b, &r) ? kBoundMax : r;
}
uint64_t badd(uint64_t a, uint64_t b) {
  uint64_t r;
  return __builtin_add_overflow(a, b, &r) ? kBoundMax : r;
}

// ------------------------------------------------- anchored coordinate ranges
// Static capacities of factors and of a leaf's per-dim unions.  A factor's
// range is bounded relative to a linear form of the output coordinates (see
// FactorPos); merging factors with the same form (a linear combination, a
// union of terms) then costs the hull of their offsets instead of the whole
// dimension.  The bounds mirror the device's range computation (core.h
// ifn_range, target_range): each index term is bounded on its own, floor
// divisions widen by (q - 1) / q, clamping to the tensor only shrinks.

Frac frac(int64_t n, int64_t d = 1) {
  if (d < 0) {
    n = -n;
    d = -d;
  }
  int64_t g = std::gcd(n < 0 ? -n : n, d);
  if (g > 1) {
    n /= g;
    d /= g;
  }
  return Frac{n, d};
}
Frac operator+(Frac a, Frac b) { return frac(a.n * b.d + b.n * a.d, a.d * b.d); }
Frac operator-(Frac a, Frac b) { return frac(a.n * b.d - b.n * a.d, a.d * b.d); }
Frac operator*(Frac a, int64_t k) { return frac(a.n * k, a.d); }
Frac operator/(Frac a, int64_t k) { return frac(a.n, a.d * k); }
bool operator<(Frac a, Frac b) { return a.n * b.d < b.n * a.d; }
bool operator==(Frac a, Frac b) { return a.n == b.n && a.d == b.d; }
int64_t floor_frac(Frac a) { return floor_div(a.n, a.d); }

using Anchor = std::vector<std::pair<int, Frac>>;

Anchor anchor_axpy(const Anchor& x, Frac k, const Anchor& y) {  // x + k*y
  std::map<int, Frac> m;
  for (const auto& e : x) m[e.first] = e.second;
  for (const auto& e : y) {
    Frac v = m.count(e.first) ? m[e.first] : Frac{0, 1};
    m[e.first] = v + Frac{e.second.n * k.n, 1} / (e.second.d * k.d);
  }
  Anchor r;
  for (const auto& e : m)
    if (e.second.n != 0) r.push_back({e.first, frac(e.second.n, e.second.d)});
  return r;
}

bool same_anchor(const Anchor& a, const Anchor& b) {
  if (a.size() != b.size()) return false;
  for (size_t i = 0; i < a.size(); ++i)
    if (a[i].first != b[i].first || !(a[i].second == b[i].second)) return false;
  return true;
}

// Coordinates a hull of positions can span; -1 when unbounded (unknown
// position or different anchors).
int64_t hull_bound(const std::vector<const FactorPos*>& ps) {
  if (ps.empty()) return -1;
  Frac lo = ps[0]->lo, hi = ps[0]->hi;
  for (const FactorPos* p : ps) {
    if (!p->known || !same_anchor(p->a, ps[0]->a)) return -1;
    if (p->lo < lo) lo = p->lo;
    if (hi < p->hi) hi = p->hi;
  }
  return floor_frac(hi - lo) + 1;
}

// Canonical forms of factors that are the same at every location whenever
// their forms are equal (two such factors then share one slot, and terms
// that differ only in such factors merge).  Two kinds:
//  - kind 0, a pattern placed at the location: value(x) = coef[x - anchor]
//    for x in [0, size), anchor = the location's coordinate `dim` (or 0 for
//    dim = -1: location independent);
//  - kind 1, fixed positions whose values depend on one coordinate r of the
//    location (dim, extent `span`): value(x) = step[x](r), each a step
//    function over [0, span) kept as (interval start, value) with adjacent
//    values different; positions whose function is zero are dropped.
// A kind 1 form with only constant functions is written as kind 0 with
// dim = -1, so that equal factors always get equal forms.  `unclipped`
// (kind 0): no offset ever leaves [0, size) wherever the anchor is, so the
// pattern can be shifted again.
struct CanonForm {
  bool known = false;
  int kind = 0;
  int dim = -1;
  int64_t size = 0;
  int64_t span = 0;
  std::map<int64_t, uint64_t> coef;
  std::map<int64_t, std::vector<std::pair<int64_t, uint64_t>>> step;
  bool unclipped = false;
};

std::string canon_key(const CanonForm& f) {
  std::ostringstream k;
  k << "CF" << f.kind << " " << f.dim << " " << f.size << " " << f.span << " " << (f.unclipped ? 1 : 0);
  for (const auto& e : f.coef) k << " " << e.first << ":" << e.second;
  for (const auto& e : f.step) {
    k << " @" << e.first;
    for (const auto& iv : e.second) k << "," << iv.first << "=" << iv.second;
  }
  return k.str();
}

// Step functions from per-position difference arrays (position -> (r ->
// change of value at r)) over [0, span); fails (false) on overflow.
bool steps_from_deltas(const std::map<int64_t, std::map<int64_t, int64_t>>& d, int64_t span,
                       std::map<int64_t, std::vector<std::pair<int64_t, uint64_t>>>* out) {
  out->clear();
  for (const auto& e : d) {
    std::vector<std::pair<int64_t, uint64_t>> fn;
    int64_t v = 0;
    bool nonzero = false;
    for (const auto& c : e.second) {
      if (c.first >= span) break;
      if (__builtin_add_overflow(v, c.second, &v) || v < 0) return false;
      if (c.second == 0) continue;
      if (!fn.empty() && fn.back().first == c.first) fn.back().second = (uint64_t)v;
      else fn.push_back({c.first, (uint64_t)v});
    }
    // Intervals start at 0 and adjacent values differ.
    if (fn.empty() || fn.front().first != 0) fn.insert(fn.begin(), {0, 0});
    std::vector<std::pair<int64_t, uint64_t>> m;
    for (const auto& iv : fn)
      if (m.empty() || m.back().second != iv.second) m.push_back(iv);
    for (const auto& iv : m) nonzero = nonzero || iv.second != 0;
    if (nonzero) (*out)[e.first] = m;
  }
  return true;
}

// Kind 1 forms with constant functions become kind 0 at dim -1.
void normalise(CanonForm* f) {
  if (!f->known || f->kind != 1) return;
  for (const auto& e : f->step)
    if (e.second.size() != 1) return;
  CanonForm r;
  r.known = true;
  r.kind = 0;
  r.dim = -1;
  r.size = f->size;
  r.unclipped = true;
  for (const auto& e : f->step) r.coef[e.first] = e.second[0].second;
  *f = r;
}

// A form as difference arrays over the anchor coordinate (kind 1, or a
// location-independent kind 0 form on the given anchor).
bool as_deltas(const CanonForm& f, std::map<int64_t, std::map<int64_t, int64_t>>* d) {
  d->clear();
  if (f.kind == 0) {
    if (f.dim >= 0) return false;
    for (const auto& e : f.coef) (*d)[e.first][0] += (int64_t)e.second;
    return true;
  }
  for (const auto& e : f.step) {
    uint64_t prev = 0;
    for (const auto& iv : e.second) {
      (*d)[e.first][iv.first] += (int64_t)iv.second - (int64_t)prev;
      prev = iv.second;
    }
  }
  return true;
}

class Compiler {
 public:
  explicit Compiler(const GraphIR& g) : g_(g) {}
  Plan run();

 private:
  const GraphIR& g_;
  std::vector<DgpInstr> ins_;
  std::vector<DgpFactor> fac_;
  std::vector<FactorPos> pos_;
  // Per factor: number of coordinates it covers when every value is 1 and
  // the range does not depend on the location (a single point: ROOT,
  // CONST; a window mapped one-to-one: length of its clamped image), else 0.
  std::vector<int64_t> unit_len_;
  std::vector<uint64_t> fbound_;
  std::vector<uint64_t> sbound_;
  std::map<std::string, int> memo_;
  std::vector<CanonForm> cf_;  // per factor
  std::vector<std::vector<SymTerm>> terms_;

  int new_factor(int64_t cap, int64_t size, uint64_t bound) {
    DgpFactor f{};
    f.cap = (int32_t)std::max<int64_t>(1, cap);
    f.size = (int32_t)size;
    fac_.push_back(f);
    cf_.push_back(CanonForm{});
    pos_.push_back(FactorPos{});
    unit_len_.push_back(0);
    fbound_.push_back(bound);
    return (int)fac_.size() - 1;
  }
  int new_scalar(uint64_t bound) {
    sbound_.push_back(bound);
    return (int)sbound_.size() - 1;
  }
  DgpInstr blank(int opcode) {
    DgpInstr i;
    std::memset(&i, 0, sizeof(i));
    i.opcode = opcode;
    i.f1 = i.f2 = i.k1 = i.k2 = -1;
    return i;
  }

  int root_factor(int a) {
    std::string key = "ROOT " + std::to_string(a);
    auto it = memo_.find(key);
    if (it != memo_.end()) return it->second;
    int f = new_factor(1, g_.tensors[g_.output].shape[a], 1);
    cf_[f].known = true;
    cf_[f].dim = a;
    cf_[f].size = g_.tensors[g_.output].shape[a];
    cf_[f].coef[0] = 1;
    cf_[f].unclipped = true;
    memo_[canon_key(cf_[f])] = f;
    unit_len_[f] = 1;
    pos_[f].known = true;
    pos_[f].a = {{a, Frac{1, 1}}};
    DgpInstr i = blank(DGP_ROOT);
    i.dst = f;
    i.a = a;
    ins_.push_back(i);
    return memo_[key] = f;
  }

  int const_factor(int64_t v, int64_t size) {
    std::string key = "CONST " + std::to_string(v) + " " + std::to_string(size);
    auto it = memo_.find(key);
    if (it != memo_.end()) return it->second;
    int f = new_factor(1, size, 1);
    if (v >= 0 && v < size) {
      cf_[f].known = true;
      cf_[f].size = size;
      cf_[f].coef[v] = 1;
      cf_[f].unclipped = true;
      memo_[canon_key(cf_[f])] = f;
    }
    unit_len_[f] = 1;
    pos_[f].known = true;
    pos_[f].lo = pos_[f].hi = frac(v);
    DgpInstr i = blank(DGP_CONST);
    i.dst = f;
    i.a = (int32_t)v;
    ins_.push_back(i);
    return memo_[key] = f;
  }

  uint64_t coef_bound(const Coef& c) {
    uint64_t b = c.k;
    for (int s : c.slots) b = bmul(b, sbound_[s]);
    return b;
  }

  // Materialises the product of a coefficient's scalar slots: (slot or -1, constant).
  std::pair<int, uint64_t> coef_slot(const Coef& c) {
    if (c.slots.empty()) return {-1, c.k};
    if (c.slots.size() == 1) return {c.slots[0], c.k};
    std::vector<int> s = c.slots;
    std::sort(s.begin(), s.end());
    std::ostringstream key;
    key << "SMUL";
    for (int x : s) key << " " << x;
    auto it = memo_.find(key.str());
    int slot;
    if (it != memo_.end()) {
      slot = it->second;
    } else {
      if (s.size() > 8) fail(DG_E_UNSUPPORTED_OP, "coefficient with more than 8 scalar factors");
      uint64_t b = 1;
      for (int x : s) b = bmul(b, sbound_[x]);
      slot = new_scalar(b);
      DgpInstr i = blank(DGP_SMUL);
      i.dst = slot;
      i.dst_is_scalar = 1;
      i.ns = (int32_t)s.size();
      for (size_t q = 0; q < s.size(); ++q) i.s[q] = s[q];
      i.cst = 1;
      ins_.push_back(i);
      memo_[key.str()] = slot;
    }
    return {slot, c.k};
  }

  Coef coef_add(const Coef& a, const Coef& b) {
    if (a.slots.empty() && b.slots.empty()) {
      uint64_t k;
      if (!__builtin_add_overflow(a.k, b.k, &k)) return Coef{k, {}};
    }
    auto sa = coef_slot(a), sb = coef_slot(b);
    std::ostringstream key;
    key << "SADD " << sa.first << " " << sa.second << " " << sb.first << " " << sb.second;
    auto it = memo_.find(key.str());
    int slot;
    if (it != memo_.end()) {
      slot = it->second;
    } else {
      slot = new_scalar(badd(coef_bound(a), coef_bound(b)));
      DgpInstr i = blank(DGP_SADD);
      i.dst = slot;
      i.dst_is_scalar = 1;
      i.f1 = sa.first;
      i.c1 = sa.second;
      i.f2 = sb.first;
      i.c2 = sb.second;
      ins_.push_back(i);
      memo_[key.str()] = slot;
    }
    return Coef{1, {slot}};
  }

  // The PATTERN instruction writing factor `dst` of canonical form cf, if
  // the pattern fits one instruction (at most DGP_MAX_PAT runs or entries,
  // values below 2^32, coordinates in int32).
  bool pattern_instr(const CanonForm& cf, int dst, DgpInstr* out) {
    DgpInstr P = blank(DGP_PATTERN);
    P.dst = dst;
    P.a = cf.dim;
    P.pkind = cf.kind;
    std::vector<std::array<int64_t, 4>> e;
    if (cf.kind == 0) {
      // Maximal runs of one value over consecutive offsets.
      for (const auto& c : cf.coef) {
        if (!e.empty() && e.back()[1] == c.first && (uint64_t)e.back()[3] == c.second) {
          e.back()[1] = c.first + 1;
        } else {
          e.push_back({c.first, c.first + 1, 0, (int64_t)c.second});
        }
      }
    } else {
      for (const auto& c : cf.step)
        for (size_t i = 0; i < c.second.size(); ++i) {
          if (c.second[i].second == 0) continue;
          const int64_t hi = i + 1 < c.second.size() ? c.second[i + 1].first : cf.span;
          e.push_back({c.first, c.second[i].first, hi, (int64_t)c.second[i].second});
        }
    }
    if (e.empty() || e.size() > DGP_MAX_PAT) return false;
    int64_t pmin = INT64_MAX, pmax = INT64_MIN;
    for (const auto& x : e) {
      if (x[3] <= 0 || x[3] > (int64_t)UINT32_MAX) return false;
      for (int q = 0; q < 3; ++q)
        if (x[q] < INT32_MIN / 2 || x[q] > INT32_MAX / 2) return false;
      pmin = std::min(pmin, x[0]);
      pmax = std::max(pmax, cf.kind == 0 ? x[1] : x[0] + 1);
    }
    P.npat = (int32_t)e.size();
    P.pmin = (int32_t)pmin;
    P.pmax = (int32_t)pmax;
    for (size_t i = 0; i < e.size(); ++i)
      for (int q = 0; q < 4; ++q) P.pat[i][q] = (int32_t)(uint32_t)e[i][q];
    const int64_t span = std::min<int64_t>(pmax - pmin, fac_[(size_t)dst].size);
    fac_[(size_t)dst].cap = (int32_t)std::max<int64_t>(1, std::min<int64_t>(fac_[(size_t)dst].cap, span));
    *out = P;
    return true;
  }

  // Canonical form of k1 f1 + k2 f2 with constant k1, k2, when both have one.
  CanonForm lincomb_form(int f1, std::pair<int, uint64_t> s1, int f2, std::pair<int, uint64_t> s2, int64_t size) {
    CanonForm none;
    const CanonForm &a = cf_[f1], &b = cf_[f2];
    if (s1.first >= 0 || s2.first >= 0 || !a.known || !b.known || a.size != size || b.size != size) return none;
    CanonForm r;
    r.known = true;
    r.size = size;
    if (a.kind == 0 && b.kind == 0 && a.dim == b.dim) {
      r.dim = a.dim;
      r.unclipped = a.unclipped && b.unclipped;
      for (int q = 0; q < 2; ++q)
        for (const auto& e : (q ? b : a).coef) {
          uint64_t v;
          if (__builtin_mul_overflow(e.second, q ? s2.second : s1.second, &v) ||
              __builtin_add_overflow(r.coef[e.first], v, &r.coef[e.first]))
            return none;
        }
      for (auto it = r.coef.begin(); it != r.coef.end();) it = it->second == 0 ? r.coef.erase(it) : std::next(it);
      return r;
    }
    // Fixed positions over one anchor coordinate.
    const CanonForm& anchored = a.kind == 1 ? a : b;
    if (anchored.kind != 1) return none;
    for (const CanonForm* f : {&a, &b})
      if (f->kind == 1 && (f->dim != anchored.dim || f->span != anchored.span)) return none;
    std::map<int64_t, std::map<int64_t, int64_t>> da, db, sum;
    if (!as_deltas(a, &da) || !as_deltas(b, &db)) return none;
    for (int q = 0; q < 2; ++q) {
      const uint64_t k = q ? s2.second : s1.second;
      if (k > (uint64_t)INT64_MAX) return none;
      for (const auto& e : (q ? db : da))
        for (const auto& c : e.second) {
          int64_t v;
          if (__builtin_mul_overflow(c.second, (int64_t)k, &v) ||
              __builtin_add_overflow(sum[e.first][c.first], v, &sum[e.first][c.first]))
            return none;
        }
    }
    da.swap(sum);
    r.kind = 1;
    r.dim = anchored.dim;
    r.span = anchored.span;
    if (!steps_from_deltas(da, r.span, &r.step)) return none;
    normalise(&r);
    return r;
  }

  int lincomb(int f1, const Coef& c1, int f2, const Coef& c2, int64_t size) {
    auto s1 = coef_slot(c1), s2 = coef_slot(c2);
    std::ostringstream key;
    key << "LIN " << f1 << " " << s1.first << " " << s1.second << " " << f2 << " " << s2.first << " " << s2.second
        << " " << size;
    auto it = memo_.find(key.str());
    if (it != memo_.end()) return it->second;
    const CanonForm cf = lincomb_form(f1, s1, f2, s2, size);
    if (cf.known) {
      auto hit = memo_.find(canon_key(cf));
      if (hit != memo_.end()) return memo_[key.str()] = hit->second;
    }
    int64_t cap = size <= kLincombFullDim ? size : std::min<int64_t>(size, (int64_t)fac_[f1].cap + fac_[f2].cap);
    const int64_t hb = hull_bound({&pos_[f1], &pos_[f2]});
    if (hb > 0) cap = std::min(cap, hb);
    FactorPos hp;
    if (hb > 0) {
      hp = pos_[f1];
      if (pos_[f2].lo < hp.lo) hp.lo = pos_[f2].lo;
      if (hp.hi < pos_[f2].hi) hp.hi = pos_[f2].hi;
    }
    int f = new_factor(cap, size, badd(bmul(fbound_[f1], coef_bound(c1)), bmul(fbound_[f2], coef_bound(c2))));
    pos_[f] = hp;
    if (cf.known) {
      cf_[f] = cf;
      memo_[canon_key(cf)] = f;
    }
    DgpInstr i = blank(DGP_LINCOMB);
    i.dst = f;
    i.f1 = f1;
    i.k1 = s1.first;
    i.c1 = s1.second;
    i.f2 = f2;
    i.k2 = s2.first;
    i.c2 = s2.second;
    ins_.push_back(i);
    return memo_[key.str()] = f;
  }

  // Merges terms equal in all factors (coefficients add) or in all but one
  // (that factor becomes a linear combination).  `shape` is the tensor's.
  void merge_terms(std::vector<SymTerm>& ts, const Dims& shape) {
    bool again = true;
    while (again) {
      again = false;
      for (size_t i = 0; i < ts.size() && !again; ++i) {
        for (size_t j = i + 1; j < ts.size() && !again; ++j) {
          int ndiff = 0, dim = -1;
          for (size_t d = 0; d < ts[i].f.size(); ++d)
            if (ts[i].f[d] != ts[j].f[d]) {
              ++ndiff;
              dim = (int)d;
            }
          if (ndiff == 0) {
            ts[i].coef = coef_add(ts[i].coef, ts[j].coef);
          } else if (ndiff == 1) {
            ts[i].f[dim] = lincomb(ts[i].f[dim], ts[i].coef, ts[j].f[dim], ts[j].coef, shape[dim]);
            ts[i].coef = Coef{1, {}};
          } else {
            continue;
          }
          ts.erase(ts.begin() + j);
          again = true;
        }
      }
    }
  }

  DgpIFn to_dev(const IndexFn& f, const std::vector<int>& local, int64_t size) {
    DgpIFn d;
    std::memset(&d, 0, sizeof(d));
    if (f.terms.size() > DGP_MAX_FTERMS) fail(DG_E_UNSUPPORTED_OP, "index function with more than 4 terms");
    d.nterm = (int32_t)f.terms.size();
    for (size_t q = 0; q < f.terms.size(); ++q) {
      d.var[q] = local[f.terms[q].var];
      d.coef[q] = (int32_t)f.terms[q].coef;
      d.vdiv[q] = (int32_t)f.terms[q].vdiv;
    }
    d.c = (int32_t)f.c;
    d.mode = f.mode;
    d.s = (int32_t)f.s;
    d.size = (int32_t)size;
    return d;
  }

  static void key_fn(std::ostringstream& k, const IndexFn& f, const std::vector<int>& local, int64_t size) {
    k << "[" << f.c << "," << f.mode << "," << f.s << "," << size;
    for (const auto& t : f.terms) k << ";" << local[t.var] << "," << t.coef << "," << t.vdiv;
    k << "]";
  }

  // Position of a component's target index (see FactorPos), from the
  // positions of its factor variables and the ranges of its window
  // variables.
  FactorPos target_pos(const IndexFn& f, const SymTerm& t, const std::vector<int>& vars, int R, const ReadGroup& G) {
    FactorPos r;
    Anchor A;
    Frac L = frac(f.c), H = frac(f.c);
    for (const auto& tm : f.terms) {
      const int v = tm.var;
      if (std::find(vars.begin(), vars.end(), v) == vars.end()) return FactorPos{};
      Anchor va;
      Frac vlo, vhi;
      bool may_be_negative = false;
      if (v < R) {
        const FactorPos& p = pos_[t.f[v]];
        if (!p.known) return FactorPos{};
        va = p.a;
        vlo = p.lo;
        vhi = p.hi;
      } else {
        vlo = frac(G.wlo[v - R]);
        vhi = frac(G.whi[v - R] - 1);
        may_be_negative = G.wlo[v - R] < 0;
      }
      const int64_t q = tm.vdiv;
      Frac lo = vlo, hi = vhi;
      if (q != 1) {
        // Device: truncating division of a value in [vlo, vhi].
        const Frac w = frac(q - 1, q);
        lo = vlo / q - w;
        hi = may_be_negative ? vhi / q + w : vhi / q;
      }
      A = anchor_axpy(A, frac(tm.coef, q), va);
      if (tm.coef >= 0) {
        L = L + lo * tm.coef;
        H = H + hi * tm.coef;
      } else {
        L = L + hi * tm.coef;
        H = H + lo * tm.coef;
      }
    }
    if (f.mode == 1 || f.mode == 2) {
      A = anchor_axpy(Anchor{}, frac(1, f.s), A);
      L = L / f.s;
      H = H / f.s;
      if (f.mode == 2) L = L - frac(f.s - 1, f.s);
    }
    r.known = true;
    r.a = A;
    r.lo = L;
    r.hi = H;
    return r;
  }

  // How many points of a component sum can land on one target value: all of
  // them, except that a variable occurring in exactly one target term is
  // pinned by the others.  With the others fixed, one target value leaves K
  // inner values (1 without an outer division or with an exact one, s with
  // a floor division by s), so at most ceil(K / |coef|) values of that
  // term's quotient, each taken by at most vdiv values of the variable
  // (2 vdiv - 1 where it can be negative: the division truncates).
  uint64_t collisions(const IndexFn& target, const std::vector<int>& vars, const std::vector<int64_t>& width, int R,
                      const ReadGroup& G) {
    uint64_t points = 1;
    for (int64_t w : width) points = bmul(points, (uint64_t)std::max<int64_t>(w, 0));
    const int64_t K = target.mode == 2 ? target.s : 1;
    uint64_t best = points;
    for (size_t q = 0; q < vars.size(); ++q) {
      const IndexFn::Term* only = nullptr;
      int uses = 0;
      for (const auto& tm : target.terms)
        if (tm.var == vars[q]) {
          only = &tm;
          ++uses;
        }
      if (uses != 1 || only->coef == 0 || width[q] <= 0) continue;
      const bool negative = vars[q] >= R && G.wlo[vars[q] - R] < 0;
      const int64_t per = only->vdiv == 1 ? 1 : (negative ? 2 * only->vdiv - 1 : only->vdiv);
      const int64_t pin = std::min<int64_t>(width[q], ceil_div(K, std::llabs(only->coef)) * per);
      uint64_t others = 1;  // the other variables' widths
      for (size_t r = 0; r < vars.size(); ++r)
        if (r != q) others = bmul(others, (uint64_t)std::max<int64_t>(width[r], 0));
      best = std::min(best, bmul(others, (uint64_t)pin));
    }
    return best;
  }

  // Canonical form of a component sum into a factor, when it has one.  At
  // most one factor variable, whose factor has an unclipped kind 0 form;
  // every index function linear with undivided terms.  Either the target
  // takes the factor variable with coefficient 1 and there is no predicate
  // but the target's own validity (kind 0: the pattern shifted by every
  // window point), or the target takes window variables only (kind 1:
  // fixed positions, each valid for an interval of the anchor coordinate).
  CanonForm component_form(const SymTerm& t, const std::vector<int>& vars, const std::vector<const IndexFn*>& preds,
                           const std::vector<int64_t>& psize, const IndexFn& target, int64_t tsize, int R,
                           const ReadGroup& G) {
    CanonForm none;
    auto linear = [](const IndexFn& f) {
      if (f.mode != 0) return false;
      for (const auto& tm : f.terms)
        if (tm.vdiv != 1) return false;
      return true;
    };
    if (!linear(target)) return none;
    for (const IndexFn* p : preds)
      if (!linear(*p)) return none;
    int fvar = -1;
    std::vector<int> wvars;
    for (int v : vars) {
      if (v < R) {
        if (fvar >= 0) return none;
        fvar = v;
      } else {
        wvars.push_back(v);
      }
    }
    auto coef_of = [](const IndexFn& f, int v) {
      int64_t a = 0;
      for (const auto& tm : f.terms) a += tm.var == v ? tm.coef : 0;
      return a;
    };
    for (const auto& tm : target.terms)
      if (tm.var < R && tm.var != fvar) return none;
    CanonForm src;
    if (fvar >= 0) {
      src = cf_[t.f[fvar]];
      if (!src.known || src.kind != 0 || !src.unclipped) return none;
    } else {
      src.known = true;
      src.dim = -1;
      src.coef[0] = 1;
    }
    int64_t box = 1;
    for (int v : wvars) box *= G.whi[v - R] - G.wlo[v - R];
    if (box <= 0 || box * (int64_t)src.coef.size() > 4096) return none;
    // Every window point, as values of wvars.
    std::vector<std::vector<int64_t>> points{{}};
    for (int v : wvars) {
      std::vector<std::vector<int64_t>> next;
      for (const auto& p0 : points)
        for (int64_t w = G.wlo[v - R]; w < G.whi[v - R]; ++w) {
          next.push_back(p0);
          next.back().push_back(w);
        }
      points.swap(next);
    }
    auto window_part = [&](const IndexFn& f, const std::vector<int64_t>& pt) {
      int64_t x = f.c;
      for (size_t q = 0; q < wvars.size(); ++q) x += coef_of(f, wvars[q]) * pt[q];
      return x;
    };
    const int64_t tf = fvar >= 0 ? coef_of(target, fvar) : 0;
    if (fvar < 0 || tf != 0) {
      // Kind 0 (a location-independent pattern without a factor variable).
      if (fvar >= 0 && tf != 1) return none;
      for (size_t p = 0; p < preds.size(); ++p)
        if (preds[p] != &target || psize[p] != tsize) return none;
      CanonForm r;
      r.known = true;
      r.dim = src.dim;
      r.size = tsize;
      r.unclipped = src.dim < 0;  // a location-independent pattern is clipped here
      for (const auto& e : src.coef)
        for (const auto& pt : points) {
          const int64_t off = e.first + window_part(target, pt);
          if (src.dim < 0 && (off < 0 || off >= tsize)) continue;
          if (__builtin_add_overflow(r.coef[off], e.second, &r.coef[off])) return none;
        }
      for (auto it = r.coef.begin(); it != r.coef.end();) it = it->second == 0 ? r.coef.erase(it) : std::next(it);
      return r;
    }
    // Kind 1: the target is fixed by the window point; each predicate
    // bounds the anchor coordinate r (the factor variable is r + offset).
    if (fvar < 0 || src.dim < 0) return none;
    const int64_t span = g_.tensors[g_.output].shape[src.dim];
    std::map<int64_t, std::map<int64_t, int64_t>> delta;
    for (const auto& e : src.coef)
      for (const auto& pt : points) {
        const int64_t pos = window_part(target, pt);
        if (pos < 0 || pos >= tsize) continue;
        int64_t lo = 0, hi = span;  // r in [lo, hi)
        for (size_t p = 0; p < preds.size(); ++p) {
          const int64_t a = coef_of(*preds[p], fvar);
          const int64_t c = window_part(*preds[p], pt) + a * e.first;  // value = a r + c
          if (a == 0) {
            if (c < 0 || c >= psize[p]) lo = hi;
          } else if (a > 0) {
            lo = std::max(lo, ceil_div(-c, a));
            hi = std::min(hi, floor_div(psize[p] - 1 - c, a) + 1);
          } else {
            lo = std::max(lo, ceil_div(psize[p] - 1 - c, a));
            hi = std::min(hi, floor_div(-c, a) + 1);
          }
        }
        if (lo >= hi) continue;
        if (__builtin_add_overflow(delta[pos][lo], (int64_t)e.second, &delta[pos][lo]) ||
            __builtin_sub_overflow(delta[pos][hi], (int64_t)e.second, &delta[pos][hi]))
          return none;
      }
    CanonForm r;
    r.known = true;
    r.kind = 1;
    r.dim = src.dim;
    r.size = tsize;
    r.span = span;
    if (!steps_from_deltas(delta, span, &r.step)) return none;
    normalise(&r);
    return r;
  }

  // Sum over one component.  Returns a factor slot (target != nullptr) or a
  // scalar slot; a component of window variables without predicates and
  // without a target folds into `folded` and returns -1.
  int component(const SymTerm& t, const std::vector<int>& vars, const std::vector<const IndexFn*>& preds,
                const std::vector<int64_t>& psize, const IndexFn* target, int64_t tsize, int R,
                const ReadGroup& G, uint64_t* folded) {
    // Identity transfer: the target index is exactly one output coordinate.
    if (target && preds.empty() && vars.size() == 1 && vars[0] < R && target->terms.size() == 1 &&
        target->terms[0].coef == 1 && target->terms[0].vdiv == 1 && target->c == 0 && target->mode == 0)
      return t.f[vars[0]];
    // A sum without predicates or target over window variables and over
    // factors whose values are all 1 on a location-independent number of
    // coordinates is that product of counts: fold it into the coefficient.
    if (!target && preds.empty()) {
      uint64_t n = 1;
      bool foldable = true;
      for (int v : vars) {
        const int64_t k = v < R ? unit_len_[t.f[v]] : G.whi[v - R] - G.wlo[v - R];
        if (k <= 0) foldable = false;
        else n *= (uint64_t)k;
      }
      if (foldable) {
        *folded = n;
        return -1;
      }
    }
    if (vars.size() > DGP_MAX_VARS) fail(DG_E_UNSUPPORTED_OP, "component with more than 8 variables");
    if (preds.size() > DGP_MAX_PREDS) fail(DG_E_UNSUPPORTED_OP, "component with more than 12 predicates");
    int nv_total = R + (int)G.wlo.size();
    std::vector<int> local(nv_total, -1);
    for (size_t q = 0; q < vars.size(); ++q) local[vars[q]] = (int)q;
    std::ostringstream key;
    key << "COMP";
    uint64_t points = 1, weight = 1;
    std::vector<int64_t> width(vars.size());
    for (size_t q = 0; q < vars.size(); ++q) {
      int v = vars[q];
      if (v < R) {
        key << " o" << t.f[v];
        width[q] = fac_[t.f[v]].cap;
        weight = bmul(weight, fbound_[t.f[v]]);
      } else {
        key << " w" << G.wlo[v - R] << ":" << G.whi[v - R];
        width[q] = G.whi[v - R] - G.wlo[v - R];
      }
      points = bmul(points, (uint64_t)std::max<int64_t>(width[q], 0));
    }
    if (points > 2147483647u) fail(DG_E_UNSUPPORTED_OP, "component sum over more than 2^31 points");
    key << " P";
    for (size_t p = 0; p < preds.size(); ++p) key_fn(key, *preds[p], local, psize[p]);
    if (target) {
      key << " T";
      key_fn(key, *target, local, tsize);
    } else {
      key << " S";
    }
    auto it = memo_.find(key.str());
    if (it != memo_.end()) return it->second;
    const CanonForm cf = target ? component_form(t, vars, preds, psize, *target, tsize, R, G) : CanonForm{};
    if (cf.known) {
      auto hit = memo_.find(canon_key(cf));
      if (hit != memo_.end()) return memo_[key.str()] = hit->second;
    }

    DgpInstr i = blank(DGP_COMP);
    i.nvar = (int32_t)vars.size();
    for (size_t q = 0; q < vars.size(); ++q) {
      int v = vars[q];
      if (v < R) {
        i.var_src[q] = t.f[v];
      } else {
        i.var_src[q] = -1;
        i.wlo[q] = (int32_t)G.wlo[v - R];
        i.whi[q] = (int32_t)G.whi[v - R];
      }
    }
    i.npred = (int32_t)preds.size();
    for (size_t p = 0; p < preds.size(); ++p) i.pred[p] = to_dev(*preds[p], local, psize[p]);
    int slot;
    if (target) {
      // Capacity: how many integer values the target can take over the
      // variables' ranges (widths from the static factor capacities).
      int64_t span = 0;
      for (const auto& tm : target->terms) {
        int64_t w = width[local[tm.var]];
        span += std::llabs(tm.coef) * ceil_div(w - 1, tm.vdiv);
      }
      int64_t count = (target->mode ? ceil_div(span, target->s) : span) + 1;
      FactorPos tp = target_pos(*target, t, vars, R, G);
      if (tp.known) count = std::min(count, floor_frac(tp.hi - tp.lo) + 1);
      slot = new_factor(std::min(count, tsize), tsize, bmul(collisions(*target, vars, width, R, G), weight));
      pos_[slot] = tp;
      if (preds.empty() && vars.size() == 1 && vars[0] >= R && target->mode == 0 && target->terms.size() == 1 &&
          target->terms[0].vdiv == 1 && (target->terms[0].coef == 1 || target->terms[0].coef == -1)) {
        // Each window point lands on its own coordinate with count 1.
        const int64_t a = target->terms[0].coef * G.wlo[vars[0] - R] + target->c;
        const int64_t b = target->terms[0].coef * (G.whi[vars[0] - R] - 1) + target->c;
        const int64_t lo = std::max<int64_t>(0, std::min(a, b)), hi = std::min<int64_t>(tsize - 1, std::max(a, b));
        unit_len_[slot] = hi >= lo ? hi - lo + 1 : 0;
      }
      i.target = to_dev(*target, local, tsize);
      i.dst_is_scalar = 0;
      if (cf.known) {
        cf_[slot] = cf;
        memo_[canon_key(cf)] = slot;
      }
    } else {
      slot = new_scalar(bmul(points, weight));
      i.dst_is_scalar = 1;
    }
    i.dst = slot;
    ins_.push_back(i);
    return memo_[key.str()] = slot;
  }

  void propagate(const SymTerm& t, const OpNode& op, const ReadGroup& G) {
    const Dims& oshape = g_.tensors[op.out].shape;
    int R = (int)oshape.size(), Q = (int)G.wlo.size(), NV = R + Q;
    std::vector<int64_t> vmin(NV), vmax(NV);
    for (int a = 0; a < R; ++a) {
      vmin[a] = 0;
      vmax[a] = oshape[a] - 1;
    }
    for (int b = 0; b < Q; ++b) {
      if (G.whi[b] <= G.wlo[b]) return;  // empty window: reads nothing
      vmin[R + b] = G.wlo[b];
      vmax[R + b] = G.whi[b] - 1;
    }
    // Validity predicates of the whole group (joint over the operands).
    std::vector<const IndexFn*> preds;
    std::vector<int64_t> psize;
    for (const Operand& r : G.ops) {
      const Dims& s = g_.tensors[r.tensor].shape;
      for (size_t d = 0; d < s.size(); ++d) {
        const IndexFn& f = r.idx[d];
        if (fn_magnitude(f, vmin, vmax) >= (int64_t(1) << 30))
          fail(DG_E_UNSUPPORTED_OP, op.kind + ": index arithmetic exceeds 32 bits");
        if (f.terms.empty()) {
          int64_t v = f.c;
          if (f.mode == 1 && floor_div(v, f.s) * f.s != v) return;
          if (f.mode) v = floor_div(v, f.s);
          if (v < 0 || v >= s[d]) return;  // constant index out of range: nothing is read
          continue;
        }
        auto rg = fn_range(f, vmin, vmax);
        bool trivial = (f.mode != 1 || f.s == 1) && rg.first >= 0 && rg.second <= s[d] - 1;
        if (!trivial) {
          preds.push_back(&f);
          psize.push_back(s[d]);
        }
      }
    }
    // Guards of merged dims: each merged dim's own index must be valid too.
    for (const auto& gd : G.guards) {
      const IndexFn& f = gd.first;
      if (fn_magnitude(f, vmin, vmax) >= (int64_t(1) << 30))
        fail(DG_E_UNSUPPORTED_OP, op.kind + ": index arithmetic exceeds 32 bits");
      if (f.terms.empty()) {
        int64_t v = f.c;
        if (f.mode == 1 && floor_div(v, f.s) * f.s != v) return;
        if (f.mode) v = floor_div(v, f.s);
        if (v < 0 || v >= gd.second) return;  // a merged dim's constant index out of range: nothing is read
        continue;
      }
      auto rg = fn_range(f, vmin, vmax);
      bool trivial = (f.mode != 1 || f.s == 1) && rg.first >= 0 && rg.second <= gd.second - 1;
      if (!trivial) {
        preds.push_back(&f);
        psize.push_back(gd.second);
      }
    }
    for (const Operand& r : G.ops) {
      const Dims& s = g_.tensors[r.tensor].shape;
      UnionFind uf(NV);
      for (const IndexFn* p : preds)
        for (size_t q = 1; q < p->terms.size(); ++q) uf.unite(p->terms[0].var, p->terms[q].var);
      for (const IndexFn& f : r.idx)
        for (size_t q = 1; q < f.terms.size(); ++q) uf.unite(f.terms[0].var, f.terms[q].var);
      // Group variables by component.
      std::map<int, std::vector<int>> comp_vars;
      for (int v = 0; v < NV; ++v) comp_vars[uf.find(v)].push_back(v);
      std::map<int, int> comp_dim;  // component root -> dim of r
      SymTerm out;
      out.coef = t.coef;
      out.f.assign(s.size(), -1);
      uint64_t kmul = r.mult;
      for (size_t d = 0; d < s.size(); ++d) {
        const IndexFn& f = r.idx[d];
        if (f.terms.empty()) {
          int64_t v = f.mode ? floor_div(f.c, f.s) : f.c;
          out.f[d] = const_factor(v, s[d]);
          continue;
        }
        int root = uf.find(f.terms[0].var);
        if (comp_dim.count(root))
          fail(DG_E_UNSUPPORTED_OP, op.kind + ": dims " + std::to_string(comp_dim[root]) + " and " +
                                        std::to_string(d) + " of an operand depend on one coupled set of "
                                        "variables (dataflow not separable)");
        comp_dim[root] = (int)d;
      }
      for (auto& cv : comp_vars) {
        int root = cv.first;
        std::vector<const IndexFn*> cp;
        std::vector<int64_t> cs;
        for (size_t p = 0; p < preds.size(); ++p)
          if (uf.find(preds[p]->terms[0].var) == root) {
            cp.push_back(preds[p]);
            cs.push_back(psize[p]);
          }
        uint64_t folded = 1;
        auto dit = comp_dim.find(root);
        if (dit != comp_dim.end()) {
          int d = dit->second;
          out.f[d] = component(t, cv.second, cp, cs, &r.idx[d], s[d], R, G, &folded);
        } else {
          int slot = component(t, cv.second, cp, cs, nullptr, 0, R, G, &folded);
          if (slot >= 0) out.coef.slots.push_back(slot);
          else if (__builtin_mul_overflow(kmul, folded, &kmul))
            fail(DG_E_OVERFLOW, "static path-count bound exceeds 64 bits");
        }
      }
      if (__builtin_mul_overflow(out.coef.k, kmul, &out.coef.k))
        fail(DG_E_OVERFLOW, "static path-count bound exceeds 64 bits");
      terms_[r.tensor].push_back(out);
    }
  }
};

Plan Compiler::run() {
  const GraphIR& g = g_;
  terms_.assign(g.tensors.size(), {});
  const Dims& oshape = g.tensors[g.output].shape;
  SymTerm root;
  for (size_t a = 0; a < oshape.size(); ++a) root.f.push_back(root_factor((int)a));
  terms_[g.output].push_back(root);
  for (int k = (int)g.ops.size() - 1; k >= 0; --k) {
    const OpNode& op = g.ops[k];
    std::vector<SymTerm> ts;
    ts.swap(terms_[op.out]);
    if (ts.empty()) continue;
    merge_terms(ts, g.tensors[op.out].shape);
    if ((int)ts.size() > kMaxTensorTerms)
      fail(DG_E_UNSUPPORTED_OP, "tensor '" + g.tensors[op.out].name + "' needs more than 64 separable terms");
    for (const SymTerm& t : ts)
      for (const ReadGroup& G : op.groups) propagate(t, op, G);
  }

  std::vector<DgpLeaf> leaves;
  std::vector<DgpTerm> dterms;
  Plan plan;
  int64_t max_row = 0, emit_entries = 0, union_entries = 0;
  uint64_t cbound = 0;
  for (int li = 0; li < (int)g.leaves.size(); ++li) {
    const Tensor& T = g.tensors[g.leaves[li]];
    std::vector<SymTerm>& ts = terms_[g.leaves[li]];
    merge_terms(ts, T.shape);
    if ((int)ts.size() > DGP_MAX_LEAF_TERMS)
      fail(DG_E_UNSUPPORTED_OP, "leaf '" + T.name + "' needs more than 32 separable terms");
    DgpLeaf L;
    std::memset(&L, 0, sizeof(L));
    L.rank = (int32_t)T.shape.size();
    L.nterm = (int32_t)ts.size();
    L.term0 = (int32_t)dterms.size();
    L.base = T.base;
    uint64_t stride = 1;
    for (int d = L.rank - 1; d >= 0; --d) {
      L.shape[d] = (int32_t)T.shape[d];
      L.stride[d] = stride;
      stride *= (uint64_t)T.shape[d];
    }
    uint64_t lb = 0;
    if (ts.size() == 1)
      for (int d = 0; d < L.rank; ++d) fac_[ts[0].f[d]].stat = 1;
    for (const SymTerm& t : ts) {
      DgpTerm dt;
      std::memset(&dt, 0, sizeof(dt));
      auto cs = coef_slot(t.coef);
      dt.coef_slot = cs.first;
      dt.coef_const = cs.second;
      uint64_t b = coef_bound(t.coef);
      for (int d = 0; d < L.rank; ++d) {
        dt.factor[d] = t.f[d];
        b = bmul(b, fbound_[t.f[d]]);
      }
      lb = badd(lb, b);
      dterms.push_back(dt);
    }
    cbound = std::max(cbound, lb);
    int64_t ucount = 0, cells = ts.empty() ? 0 : 1;
    for (int d = 0; d < L.rank; ++d) {
      int64_t u = 0;
      std::vector<const FactorPos*> ps;
      for (const SymTerm& t : ts) {
        u += fac_[t.f[d]].cap;
        ps.push_back(&pos_[t.f[d]]);
      }
      const int64_t hb = hull_bound(ps);
      if (hb > 0) u = std::min(u, hb);
      u = std::min<int64_t>(u, T.shape[d]);
      L.ucap[d] = (int32_t)std::max<int64_t>(u, 1);
      ucount += L.ucap[d];
      cells *= L.ucap[d];
    }
    max_row += cells;
    // Emission tables: dims [0, split) outer, [split, rank) inner.
    int best = -1;
    int64_t best_entries = 0;
    for (int s = 0; s <= L.rank; ++s) {
      int64_t o = 1, in = 1;
      for (int d = 0; d < s; ++d) o *= L.ucap[d];
      for (int d = s; d < L.rank; ++d) in *= L.ucap[d];
      if (o > kMaxTableEntries || in > kMaxTableEntries) continue;
      if (best < 0 || o + in < best_entries) {
        best = s;
        best_entries = o + in;
        L.outer_cap = (int32_t)o;
        L.inner_cap = (int32_t)in;
      }
    }
    int64_t words = best_entries * (1 + std::max<int64_t>(1, ts.size()));
    if (best < 0 || words > kMaxTableWords) {
      L.split = -1;  // per-cell decomposition, no tables
      L.outer_cap = L.inner_cap = 0;
      words = 0;
    } else {
      L.split = best;
    }
    emit_entries = std::max(emit_entries, words);
    union_entries = std::max(union_entries, ucount);
    leaves.push_back(L);
    plan.max_leaf_terms = std::max(plan.max_leaf_terms, (int)ts.size());
  }
  const uint64_t k2_63 = uint64_t(1) << 63;
  if (cbound >= k2_63) fail(DG_E_OVERFLOW, "static path-count bound reaches 2^63");
  for (uint64_t b : fbound_)
    if (b >= k2_63) fail(DG_E_OVERFLOW, "static path-count bound reaches 2^63");
  for (uint64_t b : sbound_)
    if (b >= k2_63) fail(DG_E_OVERFLOW, "static path-count bound reaches 2^63");

  // Factors with canonical forms are written directly from their pattern
  // (one PATTERN instruction, no sources); then every instruction whose
  // result no leaf term reads, directly or through others, is dropped, and
  // its factor keeps no values.
  for (DgpInstr& I : ins_) {
    const bool to_factor = (I.opcode == DGP_COMP && !I.dst_is_scalar) || I.opcode == DGP_LINCOMB;
    if (to_factor && cf_[I.dst].known) {
      DgpInstr P;
      if (pattern_instr(cf_[I.dst], I.dst, &P)) I = P;
    }
  }
  {
    std::vector<char> flive(fac_.size(), 0), slive(sbound_.size(), 0);
    for (const DgpLeaf& L : leaves)
      for (int t = 0; t < L.nterm; ++t) {
        const DgpTerm& T = dterms[(size_t)(L.term0 + t)];
        if (T.coef_slot >= 0) slive[(size_t)T.coef_slot] = 1;
        for (int d = 0; d < L.rank; ++d) flive[(size_t)T.factor[d]] = 1;
      }
    std::vector<char> keep(ins_.size(), 0);
    for (int k = (int)ins_.size() - 1; k >= 0; --k) {
      const DgpInstr& I = ins_[k];
      if (!(I.dst_is_scalar ? slive[(size_t)I.dst] : flive[(size_t)I.dst])) continue;
      keep[(size_t)k] = 1;
      auto f = [&](int x) {
        if (x >= 0) flive[(size_t)x] = 1;
      };
      auto sc = [&](int x) {
        if (x >= 0) slive[(size_t)x] = 1;
      };
      if (I.opcode == DGP_COMP) {
        for (int q = 0; q < I.nvar; ++q) f(I.var_src[q]);
      } else if (I.opcode == DGP_LINCOMB) {
        f(I.f1);
        f(I.f2);
        sc(I.k1);
        sc(I.k2);
      } else if (I.opcode == DGP_SMUL) {
        for (int q = 0; q < I.ns; ++q) sc(I.s[q]);
      } else if (I.opcode == DGP_SADD) {
        sc(I.f1);
        sc(I.f2);
      }
    }
    std::vector<DgpInstr> kept;
    for (size_t k = 0; k < ins_.size(); ++k)
      if (keep[k]) kept.push_back(ins_[k]);
    ins_.swap(kept);
    for (size_t f = 0; f < fac_.size(); ++f)
      if (!flive[f]) fac_[f].cap = 0;
  }

  // Levels: an instruction runs one level after the latest instruction it
  // reads; within a level the order is free.  Component sums over more than
  // two variables get a level of their own.
  const int nins = (int)ins_.size();
  std::vector<int> fprod(fac_.size(), -1), sprod(sbound_.size(), -1), lev(nins, 0);
  for (int k = 0; k < nins; ++k) {
    const DgpInstr& I = ins_[k];
    auto dep_f = [&](int f) {
      if (f >= 0 && fprod[f] >= 0) lev[k] = std::max(lev[k], lev[fprod[f]] + 1);
    };
    auto dep_s = [&](int x) {
      if (x >= 0 && sprod[x] >= 0) lev[k] = std::max(lev[k], lev[sprod[x]] + 1);
    };
    if (I.opcode == DGP_COMP) {
      for (int q = 0; q < I.nvar; ++q) dep_f(I.var_src[q]);
    } else if (I.opcode == DGP_LINCOMB) {
      dep_f(I.f1);
      dep_f(I.f2);
      dep_s(I.k1);
      dep_s(I.k2);
    } else if (I.opcode == DGP_SMUL) {
      for (int q = 0; q < I.ns; ++q) dep_s(I.s[q]);
    } else if (I.opcode == DGP_SADD) {
      dep_s(I.f1);
      dep_s(I.f2);
    }
    if (I.dst_is_scalar) sprod[I.dst] = k;
    else fprod[I.dst] = k;
  }
  int serial_vars = 0;
  std::vector<std::pair<std::pair<int, int>, int>> order;  // ((level, serial rank), instruction)
  for (int k = 0; k < nins; ++k) {
    bool serial = ins_[k].opcode == DGP_COMP && ins_[k].nvar > 2;
    if (serial) serial_vars = std::max(serial_vars, (int)ins_[k].nvar);
    order.push_back({{lev[k], serial ? k + 1 : 0}, k});
  }
  std::stable_sort(order.begin(), order.end(),
                   [](const std::pair<std::pair<int, int>, int>& a, const std::pair<std::pair<int, int>, int>& b) {
                     return a.first < b.first;
                   });
  std::vector<DgpInstr> sorted;
  std::vector<int32_t> level_start;
  std::pair<int, int> cur{-1, -1};
  for (auto& o : order) {
    if (o.first != cur) {
      level_start.push_back((int32_t)sorted.size());
      cur = o.first;
    }
    sorted.push_back(ins_[o.second]);
  }
  level_start.push_back((int32_t)sorted.size());
  ins_.swap(sorted);

  // Factor value offsets: the factors leaf terms read first, then those of
  // intermediate tensors only.
  std::vector<char> live(fac_.size(), 0);
  for (const DgpLeaf& L : leaves)
    for (int t = 0; t < L.nterm; ++t)
      for (int d = 0; d < L.rank; ++d) {
        const int f = dterms[(size_t)(L.term0 + t)].factor[d];
        if (f >= 0 && f < (int)fac_.size()) live[(size_t)f] = 1;
      }
  int64_t fval = 0;
  for (int pass = 1; pass >= 0; --pass)
    for (size_t i = 0; i < fac_.size(); ++i)
      if (live[i] == pass) {
        fac_[i].off = (int32_t)fval;
        fval += fac_[i].cap;
      }
  int64_t fval_live = 0;
  for (size_t i = 0; i < fac_.size(); ++i)
    if (live[i]) fval_live += fac_[i].cap;
  DgpHeader h;
  std::memset(&h, 0, sizeof(h));
  h.magic = DGP_MAGIC;
  h.out_rank = (int32_t)oshape.size();
  h.out_numel = numel(oshape);
  int64_t st = 1;
  for (int d = h.out_rank - 1; d >= 0; --d) {
    h.out_shape[d] = oshape[d];
    h.out_stride[d] = st;
    st *= oshape[d];
  }
  h.ninstr = (int32_t)ins_.size();
  h.nfactor = (int32_t)fac_.size();
  h.nscalar = (int32_t)sbound_.size();
  h.nleaf = (int32_t)leaves.size();
  h.nterm = (int32_t)dterms.size();
  h.fval_entries = (int32_t)fval;
  h.fval_live = (int32_t)fval_live;
  h.max_leaf_terms = plan.max_leaf_terms;
  h.emit_entries = (int32_t)emit_entries;
  h.union_entries = (int32_t)union_entries;
  h.nlevel = (int32_t)level_start.size() - 1;
  h.serial_vars = serial_vars;
  h.no_overflow = cbound <= 4294967295u ? 1 : 0;
  size_t off = (sizeof(DgpHeader) + 15) & ~size_t(15);
  h.instr_off = (int32_t)off;
  off += ins_.size() * sizeof(DgpInstr);
  off = (off + 15) & ~size_t(15);
  h.factor_off = (int32_t)off;
  off += fac_.size() * sizeof(DgpFactor);
  off = (off + 15) & ~size_t(15);
  h.leaf_off = (int32_t)off;
  off += leaves.size() * sizeof(DgpLeaf);
  off = (off + 15) & ~size_t(15);
  h.term_off = (int32_t)off;
  off += dterms.size() * sizeof(DgpTerm);
  off = (off + 15) & ~size_t(15);
  h.level_off = (int32_t)off;
  off += level_start.size() * sizeof(int32_t);
  h.blob_bytes = (int32_t)off;
  plan.blob.assign(off, 0);
  std::memcpy(plan.blob.data(), &h, sizeof(h));
  if (!ins_.empty()) std::memcpy(plan.blob.data() + h.instr_off, ins_.data(), ins_.size() * sizeof(DgpInstr));
  if (!fac_.empty()) std::memcpy(plan.blob.data() + h.factor_off, fac_.data(), fac_.size() * sizeof(DgpFactor));
  if (!leaves.empty()) std::memcpy(plan.blob.data() + h.leaf_off, leaves.data(), leaves.size() * sizeof(DgpLeaf));
  if (!dterms.empty()) std::memcpy(plan.blob.data() + h.term_off, dterms.data(), dterms.size() * sizeof(DgpTerm));
  std::memcpy(plan.blob.data() + h.level_off, level_start.data(), level_start.size() * sizeof(int32_t));
  plan.max_row_size = max_row;
  plan.count_bound = cbound;
  plan.fpos = pos_;
  return plan;
}

}  // namespace

Plan compile_plan(const GraphIR& g, const DimPartition* start) {
  const MergedView v = merged_view(g, start);
  Plan p = Compiler(v.ir).run();
  p.part = v.part;
  for (int t : g.leaves) p.leaf_part.push_back(v.part[t]);
  return p;
}

void compile_pair_plans(const GraphIR& a, const GraphIR& b, Plan* pa, Plan* pb) {
  if (a.leaves.size() != b.leaves.size()) fail(DG_E_SIGNATURE, "leaf count differs");
  *pa = compile_plan(a);
  *pb = compile_plan(b);
  // Both must view every leaf with the same merged dims: start both from
  // the join of their leaf partitions until they agree (each round only
  // coarsens, so this ends).
  while (pa->leaf_part != pb->leaf_part) {
    DimPartition sa = pa->part, sb = pb->part;
    for (size_t i = 0; i < a.leaves.size(); ++i) {
      if (pa->leaf_part[i].size() != pb->leaf_part[i].size()) fail(DG_E_SIGNATURE, "leaf ranks differ");
      const std::vector<int> j = join_partition(pa->leaf_part[i], pb->leaf_part[i]);
      sa[a.leaves[i]] = j;
      sb[b.leaves[i]] = j;
    }
    *pa = compile_plan(a, &sa);
    *pb = compile_plan(b, &sb);
  }
}

uint32_t plan_lds_bytes(const Plan& p, int nthreads, uint32_t word_bytes) {
  const DgpHeader& h = p.header();
  dgc::PlanLayout PL = dgc::plan_layout(&h, dgc::vars_bytes(h.serial_vars, nthreads));
  dgc::EmitLayout E = dgc::emit_layout(PL.end, h.max_leaf_terms, h.union_entries, h.emit_entries, word_bytes);
  return (E.end + 15u) & ~15u;
}

void pair_plan(const Plan& a, const Plan& b, int nthreads, dgc::PairPlan* pp) {
  const DgpHeader& ha = a.header();
  const DgpHeader& hb = b.header();
  if (ha.nleaf != hb.nleaf) fail(DG_E_SIGNATURE, "leaf count differs");
  if (ha.nleaf > 16) fail(DG_E_UNSUPPORTED_OP, "compare supports at most 16 leaves");
  std::memset(pp, 0, sizeof(*pp));
  pp->nleaf = ha.nleaf;
  const DgpLeaf* la = reinterpret_cast<const DgpLeaf*>(a.blob.data() + ha.leaf_off);
  const DgpLeaf* lb = reinterpret_cast<const DgpLeaf*>(b.blob.data() + hb.leaf_off);
  const DgpTerm* ta = reinterpret_cast<const DgpTerm*>(a.blob.data() + ha.term_off);
  const DgpTerm* tb = reinterpret_cast<const DgpTerm*>(b.blob.data() + hb.term_off);
  int64_t emit = 0, uni = 0;
  for (int l = 0; l < ha.nleaf; ++l) {
    const DgpLeaf &x = la[l], &y = lb[l];
    int T = x.nterm + y.nterm;
    pp->max_terms = std::max(pp->max_terms, T);
    dgc::LeafShape& S = pp->leaf[l];
    int64_t ucount = 0;
    for (int d = 0; d < DGP_MAX_RANK; ++d) {
      if (d < x.rank) {
        int64_t u = (x.nterm > 0 ? (int64_t)x.ucap[d] : 0) + (y.nterm > 0 ? (int64_t)y.ucap[d] : 0);
        // Both graphs' positions are anchored on the same output
        // coordinates, so their union is bounded by the joint hull.
        std::vector<const FactorPos*> ps;
        for (int t = 0; t < x.nterm; ++t) ps.push_back(&a.fpos[ta[x.term0 + t].factor[d]]);
        for (int t = 0; t < y.nterm; ++t) ps.push_back(&b.fpos[tb[y.term0 + t].factor[d]]);
        const int64_t hb = hull_bound(ps);
        if (hb > 0) u = std::min(u, hb);
        u = std::min<int64_t>(u, x.shape[d]);
        S.ucap[d] = (int32_t)std::max<int64_t>(u, 1);
        ucount += S.ucap[d];
      } else {
        S.ucap[d] = 1;
      }
    }
    int best = -1;
    int64_t best_e = 0;
    for (int s = 0; s <= x.rank; ++s) {
      int64_t o = 1, in = 1;
      for (int d = 0; d < s; ++d) o *= S.ucap[d];
      for (int d = s; d < x.rank; ++d) in *= S.ucap[d];
      if (o > kMaxTableEntries || in > kMaxTableEntries) continue;
      if (best < 0 || o + in < best_e) {
        best = s;
        best_e = o + in;
      }
    }
    int64_t words = best_e * (1 + std::max(T, 1));
    if (best < 0 || words > kMaxTableWords) {
      S.split = -1;
      words = 0;
    } else {
      S.split = best;
    }
    emit = std::max(emit, words);
    uni = std::max(uni, ucount);
  }
  pp->union_entries = (int32_t)uni;
  pp->emit_entries = (int32_t)emit;
  pp->nthreads = nthreads;
  pp->vars = dgc::vars_bytes(std::max(ha.serial_vars, hb.serial_vars), nthreads);
  dgc::PlanLayout PA = dgc::plan_layout(&ha, pp->vars);
  pp->plan_b = dgc::align8(PA.end);
  dgc::PlanLayout PB = dgc::plan_layout(&hb, pp->plan_b);
  dgc::EmitLayout E =
      dgc::emit_layout(dgc::compare_emit_base(&hb, PB), pp->max_terms, pp->union_entries, pp->emit_entries);
  // (B's plan writes up to PB.end before the emission area takes over.)
  pp->lds_bytes = (std::max(E.end, PB.end) + 15u) & ~15u;
}

}  // namespace dg

namespace dg {

namespace {
std::string fn_text(const DgpIFn& f) {
  std::ostringstream o;
  o << "(";
  for (int q = 0; q < f.nterm; ++q) {
    if (q) o << " + ";
    o << f.coef[q] << "*v" << f.var[q];
    if (f.vdiv[q] != 1) o << "/" << f.vdiv[q];
  }
  o << " + " << f.c << ")";
  if (f.mode == 1) o << " /exact " << f.s;
  if (f.mode == 2) o << " //" << f.s;
  o << " in [0," << f.size << ")";
  return o.str();
}
}  // namespace

std::string plan_listing(const Plan& p) {
  const DgpHeader& h = p.header();
  const DgpInstr* ins = reinterpret_cast<const DgpInstr*>(p.blob.data() + h.instr_off);
  const DgpFactor* fac = reinterpret_cast<const DgpFactor*>(p.blob.data() + h.factor_off);
  const DgpLeaf* lv = reinterpret_cast<const DgpLeaf*>(p.blob.data() + h.leaf_off);
  const DgpTerm* tm = reinterpret_cast<const DgpTerm*>(p.blob.data() + h.term_off);
  std::ostringstream o;
  o << "instructions " << h.ninstr << ", factors " << h.nfactor << " (" << h.fval_entries << " values), scalars "
    << h.nscalar << "\n";
  const int32_t* ls = reinterpret_cast<const int32_t*>(p.blob.data() + h.level_off);
  for (int k = 0; k < h.ninstr; ++k) {
    for (int g = 0; g < h.nlevel; ++g)
      if (ls[g] == k) o << "-- level " << g << "\n";
    const DgpInstr& I = ins[k];
    std::string dst = I.dst_is_scalar ? "s" + std::to_string(I.dst)
                                      : "f" + std::to_string(I.dst) + "[cap " + std::to_string(fac[I.dst].cap) + "]";
    o << k << ": ";
    switch (I.opcode) {
      case DGP_ROOT: o << dst << " = ROOT dim " << I.a; break;
      case DGP_CONST: o << dst << " = CONST " << I.a; break;
      case DGP_COMP:
        o << dst << " = COMP vars";
        for (int q = 0; q < I.nvar; ++q) {
          if (I.var_src[q] >= 0) o << " v" << q << "=f" << I.var_src[q];
          else o << " v" << q << "=[" << I.wlo[q] << "," << I.whi[q] << ")";
        }
        for (int e = 0; e < I.npred; ++e) o << " | pred " << fn_text(I.pred[e]);
        if (!I.dst_is_scalar) o << " | target " << fn_text(I.target);
        break;
      case DGP_LINCOMB:
        o << dst << " = LINCOMB s" << I.k1 << "*" << I.c1 << "*f" << I.f1 << " + s" << I.k2 << "*" << I.c2 << "*f" << I.f2;
        break;
      case DGP_SMUL: o << dst << " = SMUL " << I.cst; for (int q = 0; q < I.ns; ++q) o << " *s" << I.s[q]; break;
      case DGP_SADD: o << dst << " = SADD s" << I.f1 << "*" << I.c1 << " + s" << I.f2 << "*" << I.c2; break;
      case DGP_PATTERN:
        o << dst << " = PATTERN kind " << I.pkind << " at " << (I.a >= 0 ? "dim " + std::to_string(I.a) : "0");
        for (int e = 0; e < I.npat; ++e)
          o << " {" << I.pat[e][0] << "," << I.pat[e][1] << "," << I.pat[e][2] << ":" << I.pat[e][3] << "}";
        break;
    }
    o << "\n";
  }
  for (int l = 0; l < h.nleaf; ++l) {
    o << "leaf " << l << " rank " << lv[l].rank << " split " << lv[l].split << " terms " << lv[l].nterm << ":";
    for (int t = 0; t < lv[l].nterm; ++t) {
      const DgpTerm& T = tm[lv[l].term0 + t];
      o << " [s" << T.coef_slot << "*" << T.coef_const;
      for (int d = 0; d < lv[l].rank; ++d) o << " f" << T.factor[d];
      o << "]";
    }
    o << "\n";
  }
  return o.str();
}

}  // namespace dg
