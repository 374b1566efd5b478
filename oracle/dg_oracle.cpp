// Oracle for batched backward dataflow enumeration.
//
// TEST INFRASTRUCTURE ONLY.  This file is the plain, slow CPU definition that
// the GPU library is checked against.  Only the tests, the smoke check and
// the benchmark's CPU-baseline leg may load it; the product path never does.
// It shares no code with the GPU library: it has its own parser, its own
// shape inference and its own per-op read enumeration.
//
// What it computes (Sec. 3.4, "Per-element equations" and "Back-projection"):
// every op k writes one tensor T_k in SSA order, and each element T_k[l] is a
// per-element equation f_k(l) over elements of earlier tensors.  res(y[l])
// substitutes the equations backwards until only input (leaf) elements are
// left.  The footprint of l is the set of leaf elements occurring in
// res(y[l]); the path count of a leaf element is the number of its
// occurrences.  Writing R_k(l) for the multiset of element references in
// f_k(l), occurrences compose as
//     P(T_k[l], x[i]) = sum over r in R_k(l) of P(r, x[i]),   P(x[i], x[i]) = 1,
// which is evaluated here per location as a dynamic program over the tensors
// in reverse SSA order, one std::map per tensor.
//
// Read multisets R_k(l) are the dataflow skeletons of the Torch lowerings
// (Sec. 3.3, "Torch Operations"): every tensor element is a separate
// variable (Sec. 3.4), constants (padding, eps, 1/n) are not variables, an
// activation is one uninterpreted function of its operand, a select (max,
// min, clamp) reads each operand once, floats are reals (Sec. 3.3, "Setup").
// The readings taken where the paper is silent are restated at each op.
//
// Output per location: leaf elements in leaf declaration order, ascending
// element index, as (global id = leaf base + row-major flat index, count).
// Locations are flat row-major indices into the output (Sec. 3.3 "Setup":
// R_y maps flat indices).  Path counts are exact (uint64 with overflow
// checks).  Two result widths (the paper fixes none; ids are a leaf base
// plus a flat index, counts are path counts): the 32-bit form rejects a graph
// with more than 2^32 - 1 leaf elements and a count that does not fit 32
// bits, the 64-bit form holds both in 64 bits.  Graphs are limited to 2^62
// leaf elements, so that every id and every offset is a non-negative int64.

#include <algorithm>
#include <cctype>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <map>
#include <set>
#include <sstream>
#include <stdexcept>
#include <string>
#include <thread>
#include <vector>

namespace {

typedef std::vector<int64_t> Shape;

struct Error : std::runtime_error {
  explicit Error(const std::string& m) : std::runtime_error(m) {}
};

// Element count of a shape; a tensor may hold at most 2^62 elements.
int64_t numel_of(const Shape& s) {
  int64_t n = 1;
  for (int64_t d : s) {
    if (d < 0 || __builtin_mul_overflow(n, d, &n) || n > (int64_t(1) << 62))
      throw Error("tensor element count exceeds 2^62");
  }
  return n;
}

// Row-major flat index <-> multi-index.
Shape unravel(int64_t flat, const Shape& shape) {
  Shape idx(shape.size());
  for (int d = (int)shape.size() - 1; d >= 0; --d) {
    idx[d] = flat % shape[d];
    flat /= shape[d];
  }
  return idx;
}

int64_t ravel(const Shape& idx, const Shape& shape) {
  int64_t flat = 0;
  for (size_t d = 0; d < shape.size(); ++d) flat = flat * shape[d] + idx[d];
  return flat;
}

// ---------------------------------------------------------------------------
// Affine index expressions of affine_gather: sum of coef*o<k>, coef*w<k> and
// a constant, optionally divided by a positive integer (exactly with "/",
// flooring with "//").  This is the inverted affine write set of a custom
// kernel (Sec. 3.4: a thread writes v(tid,bid) to address a(tid,bid); with
// a affine, fixing the written location makes every read index affine).
// ---------------------------------------------------------------------------
struct Expr {
  struct Term { char var; int index; int64_t coef; };
  std::vector<Term> terms;
  int64_t constant = 0;
  int divmode = 0;  // 0 none, 1 exact, 2 floor
  int64_t divisor = 1;
};

Expr parse_linear(const std::string& s) {
  Expr e;
  size_t i = 0;
  if (s.empty()) throw Error("empty index expression");
  while (i < s.size()) {
    int64_t sign = 1;
    if (s[i] == '+' || s[i] == '-') { sign = s[i] == '-' ? -1 : 1; ++i; }
    size_t j = i;
    while (j < s.size() && s[j] != '+' && s[j] != '-') ++j;
    std::string tok = s.substr(i, j - i);
    i = j;
    if (tok.empty()) throw Error("bad index expression '" + s + "'");
    int64_t coef = 1;
    std::string var = tok;
    size_t star = tok.find('*');
    if (star != std::string::npos) {
      coef = std::stoll(tok.substr(0, star));
      var = tok.substr(star + 1);
    }
    if (var[0] == 'o' || var[0] == 'w') {
      if (var.size() < 2) throw Error("bad variable in '" + s + "'");
      for (size_t k = 1; k < var.size(); ++k)
        if (!isdigit((unsigned char)var[k])) throw Error("bad variable in '" + s + "'");
      e.terms.push_back({var[0], std::stoi(var.substr(1)), sign * coef});
    } else {
      for (char ch : var)
        if (!isdigit((unsigned char)ch)) throw Error("bad token '" + var + "'");
      if (star != std::string::npos) throw Error("bad token '" + tok + "'");
      e.constant += sign * std::stoll(var);
    }
  }
  return e;
}

Expr parse_expr(const std::string& s) {
  if (!s.empty() && s[0] == '(') {
    size_t close = s.find(')');
    if (close == std::string::npos) throw Error("unbalanced '(' in '" + s + "'");
    Expr e = parse_linear(s.substr(1, close - 1));
    std::string rest = s.substr(close + 1);
    if (rest.rfind("//", 0) == 0) { e.divmode = 2; rest = rest.substr(2); }
    else if (rest.rfind("/", 0) == 0) { e.divmode = 1; rest = rest.substr(1); }
    else throw Error("expected '/' or '//' after ')' in '" + s + "'");
    e.divisor = std::stoll(rest);
    if (e.divisor <= 0) throw Error("divisor must be positive in '" + s + "'");
    return e;
  }
  return parse_linear(s);
}

int64_t floor_div(int64_t a, int64_t b) {
  int64_t q = a / b;
  if ((a % b != 0) && ((a < 0) != (b < 0))) --q;
  return q;
}

// Evaluates e at (o, w); returns false when an exact division does not divide.
bool eval_expr(const Expr& e, const Shape& o, const Shape& w, int64_t* out) {
  int64_t v = e.constant;
  for (const auto& t : e.terms) v += t.coef * (t.var == 'o' ? o[t.index] : w[t.index]);
  if (e.divmode == 1) {
    if (v % e.divisor != 0) return false;
    v /= e.divisor;
  } else if (e.divmode == 2) {
    v = floor_div(v, e.divisor);
  }
  *out = v;
  return true;
}

// ---------------------------------------------------------------------------
// Graph
// ---------------------------------------------------------------------------
struct Tensor {
  std::string name;
  Shape shape;
  bool leaf = false;
  int leaf_index = -1;
  uint64_t base = 0;  // global id of element 0 (leaves only)
};

struct Op {
  std::string kind;
  std::vector<int> in;
  int out = -1;
  std::map<std::string, std::vector<int64_t>> attr;
  std::vector<std::vector<Expr>> idx;  // affine_gather
  std::map<std::string, std::string> raw;  // attribute text as written (key -> value)
};

struct Graph {
  std::vector<Tensor> tensors;
  std::vector<Op> ops;  // SSA order
  std::vector<int> leaves;
  std::map<std::string, int> by_name;
  int output = -1;
  uint64_t leaf_total = 0;
};

const std::set<std::string> kUnary = {
    "relu", "gelu", "gelu_tanh", "hardtanh", "clamp", "sigmoid", "tanh", "exp", "log",
    "log1p", "square", "sqrt", "rsqrt", "neg", "abs", "identity", "contiguous", "silu",
    "softplus", "erf", "scale", "leaky_relu", "elu", "reciprocal"};
const std::set<std::string> kBinary = {"add", "sub", "mul", "div", "maximum", "minimum", "pow"};
const std::set<std::string> kReduce = {"sum", "mean", "amax", "amin", "prod", "max", "min"};

std::vector<int64_t> get_attr(const Op& op, const std::string& k) {
  auto it = op.attr.find(k);
  if (it == op.attr.end()) throw Error("op " + op.kind + ": missing attribute '" + k + "'");
  return it->second;
}

std::vector<int64_t> get_attr_or(const Op& op, const std::string& k, std::vector<int64_t> dflt) {
  auto it = op.attr.find(k);
  return it == op.attr.end() ? dflt : it->second;
}

int64_t get_scalar(const Op& op, const std::string& k, int64_t dflt, bool required = false) {
  auto it = op.attr.find(k);
  if (it == op.attr.end()) {
    if (required) throw Error("op " + op.kind + ": missing attribute '" + k + "'");
    return dflt;
  }
  if (it->second.size() != 1) throw Error("op " + op.kind + ": attribute '" + k + "' must be one integer");
  return it->second[0];
}

// NumPy broadcasting of two shapes (right-aligned).
Shape broadcast_shapes(const Shape& a, const Shape& b) {
  size_t r = std::max(a.size(), b.size());
  Shape out(r);
  for (size_t i = 0; i < r; ++i) {
    int64_t da = i < r - a.size() ? 1 : a[i - (r - a.size())];
    int64_t db = i < r - b.size() ? 1 : b[i - (r - b.size())];
    if (da != db && da != 1 && db != 1) throw Error("shapes do not broadcast");
    out[i] = std::max(da, db);
  }
  return out;
}

// Index into an operand of shape `s` broadcast to `out` at out-index `o`.
int64_t broadcast_flat(const Shape& o, const Shape& s) {
  size_t off = o.size() - s.size();
  int64_t flat = 0;
  for (size_t d = 0; d < s.size(); ++d) flat = flat * s[d] + (s[d] == 1 ? 0 : o[off + d]);
  return flat;
}

int norm_dim(int64_t d, size_t rank) {
  int64_t r = (int64_t)rank;
  if (d < 0) d += r;
  if (d < 0 || d >= r) throw Error("dimension out of range");
  return (int)d;
}

Shape infer_shape(Graph& g, Op& op) {
  auto S = [&](int i) -> const Shape& { return g.tensors[op.in[i]].shape; };
  const std::string& k = op.kind;
  auto need = [&](size_t lo, size_t hi) {
    if (op.in.size() < lo || op.in.size() > hi) throw Error("op " + k + ": wrong operand count");
  };
  if (kUnary.count(k)) { need(1, 1); return S(0); }
  if (kBinary.count(k)) { need(2, 2); return broadcast_shapes(S(0), S(1)); }
  if (k == "matmul") {
    need(2, 2);
    const Shape &a = S(0), &b = S(1);
    if (a.size() < 2 || b.size() < 2) throw Error("matmul needs rank >= 2 operands");
    if (a[a.size() - 1] != b[b.size() -2]) throw Error("matmul inner dimensions differ");
    Shape ba(a.begin(), a.end() - 2), bb(b.begin(), b.end() - 2);
    Shape out = broadcast_shapes(ba, bb);
    out.push_back(a[a.size() - 2]);
    out.push_back(b[b.size() - 1]);
    return out;
  }
  if (k == "linear") {
    need(2, 3);
    const Shape &x = S(0), &w = S(1);
    if (w.size() != 2 || x.empty() || x.back() != w[1]) throw Error("linear: bad shapes");
    if (op.in.size() == 3 && (S(2).size() != 1 || S(2)[0] != w[0])) throw Error("linear: bad bias");
    Shape out = x;
    out.back() = w[0];
    return out;
  }
  if (k == "conv" || k == "conv_transpose") {
    need(2, 3);
    const Shape &x = S(0), &w = S(1);
    if (x.size() < 3 || w.size() != x.size()) throw Error(k + ": bad ranks");
    size_t nsp = x.size() - 2;
    auto st = get_attr_or(op, "stride", std::vector<int64_t>(nsp, 1));
    auto pd = get_attr_or(op, "pad", std::vector<int64_t>(nsp, 0));
    auto dl = get_attr_or(op, "dilation", std::vector<int64_t>(nsp, 1));
    auto opd = get_attr_or(op, "output_padding", std::vector<int64_t>(nsp, 0));
    int64_t G = get_scalar(op, "groups", 1);
    if (st.size() != nsp || pd.size() != nsp || dl.size() != nsp || opd.size() != nsp)
      throw Error(k + ": attribute lengths must equal the spatial rank");
    if (G <= 0) throw Error(k + ": bad groups");
    Shape out(x.size());
    out[0] = x[0];
    if (k == "conv") {
      if (x[1] != w[1] * G || w[0] % G != 0) throw Error("conv: channel mismatch");
      out[1] = w[0];
      for (size_t d = 0; d < nsp; ++d) {
        int64_t o = (x[2 + d] + 2 * pd[d] - dl[d] * (w[2 + d] - 1) - 1) / st[d] + 1;
        if (o <= 0) throw Error("conv: empty output");
        out[2 + d] = o;
      }
    } else {
      if (x[1] != w[0] || w[0] % G != 0) throw Error("conv_transpose: channel mismatch");
      out[1] = w[1] * G;
      for (size_t d = 0; d < nsp; ++d) {
        int64_t o = (x[2 + d] - 1) * st[d] - 2 * pd[d] + dl[d] * (w[2 + d] - 1) + opd[d] + 1;
        if (o <= 0) throw Error("conv_transpose: empty output");
        out[2 + d] = o;
      }
    }
    if (op.in.size() == 3 && (S(2).size() != 1 || S(2)[0] != out[1])) throw Error(k + ": bad bias");
    return out;
  }
  if (k == "max_pool" || k == "avg_pool") {
    need(1, 1);
    const Shape& x = S(0);
    auto ks = get_attr(op, "kernel");
    size_t nsp = ks.size();
    if (x.size() < nsp) throw Error("pool: rank too small");
    auto st = get_attr_or(op, "stride", ks);
    auto pd = get_attr_or(op, "pad", std::vector<int64_t>(nsp, 0));
    auto dl = get_attr_or(op, "dilation", std::vector<int64_t>(nsp, 1));
    if (st.size() != nsp || pd.size() != nsp || dl.size() != nsp) throw Error("pool: attribute lengths");
    Shape out = x;
    for (size_t d = 0; d < nsp; ++d) {
      size_t a = x.size() - nsp + d;
      int64_t o = (x[a] + 2 * pd[d] - dl[d] * (ks[d] - 1) - 1) / st[d] + 1;
      if (o <= 0) throw Error("pool: empty output");
      out[a] = o;
    }
    return out;
  }
  if (kReduce.count(k)) {
    need(1, 1);
    const Shape& x = S(0);
    auto dims = get_attr(op, "dims");
    bool keep = get_scalar(op, "keepdim", 0) != 0;
    std::vector<bool> red(x.size(), false);
    for (int64_t d : dims) red[norm_dim(d, x.size())] = true;
    Shape out;
    for (size_t d = 0; d < x.size(); ++d) {
      if (!red[d]) out.push_back(x[d]);
      else if (keep) out.push_back(1);
    }
    if (out.empty()) out.push_back(1);  // full reduction: one element
    return out;
  }
  if (k == "softmax" || k == "log_softmax") {
    need(1, 1);
    norm_dim(get_scalar(op, "dim", 0, true), S(0).size());
    return S(0);
  }
  if (k == "group_norm" || k == "batch_norm" || k == "layer_norm") {
    if (op.in.size() != 1 && op.in.size() != 3) throw Error(k + ": takes 1 or 3 operands");
    const Shape& x = S(0);
    Shape affine;
    if (k == "layer_norm") {
      int64_t nd = get_scalar(op, "ndims", 1);
      if (nd <= 0 || nd > (int64_t)x.size()) throw Error("layer_norm: bad ndims");
      affine.assign(x.end() - nd, x.end());
    } else {
      if (x.size() < 2) throw Error(k + ": needs [N, C, ...]");
      affine = {x[1]};
      if (k == "group_norm") {
        int64_t G = get_scalar(op, "groups", 0, true);
        if (G <= 0 || x[1] % G != 0) throw Error("group_norm: groups must divide C");
      }
    }
    if (op.in.size() == 3 && (S(1) != affine || S(2) != affine)) throw Error(k + ": bad affine shapes");
    return x;
  }
  if (k == "channel_affine") {
    need(3, 3);
    const Shape& x = S(0);
    if (x.size() < 2 || S(1) != Shape{x[1]} || S(2) != Shape{x[1]}) throw Error("channel_affine: bad shapes");
    return x;
  }
  if (k == "slice") {
    need(1, 1);
    const Shape& x = S(0);
    int dim = norm_dim(get_scalar(op, "dim", 0, true), x.size());
    int64_t n = x[dim];
    int64_t start = get_scalar(op, "start", 0), end = get_scalar(op, "end", n), step = get_scalar(op, "step", 1);
    if (step <= 0) throw Error("slice: step must be positive");
    if (start < 0) start += n;
    if (end < 0) end += n;
    start = std::min(std::max(start, (int64_t)0), n);
    end = std::min(std::max(end, (int64_t)0), n);
    if (end <= start) throw Error("slice: empty");
    op.attr["start"] = {start};
    op.attr["end"] = {end};
    op.attr["step"] = {step};
    op.attr["dim"] = {dim};
    Shape out = x;
    out[dim] = (end - start + step - 1) / step;
    return out;
  }
  if (k == "permute") {
    need(1, 1);
    const Shape& x = S(0);
    auto p = get_attr(op, "dims");
    if (p.size() != x.size()) throw Error("permute: wrong length");
    std::vector<bool> seen(x.size(), false);
    Shape out(x.size());
    for (size_t i = 0; i < p.size(); ++i) {
      int d = norm_dim(p[i], x.size());
      if (seen[d]) throw Error("permute: repeated dimension");
      seen[d] = true;
      p[i] = d;
      out[i] = x[d];
    }
    op.attr["dims"] = p;
    return out;
  }
  if (k == "reshape") {
    need(1, 1);
    Shape out = get_attr(op, "shape");
    for (int64_t d : out) if (d <= 0) throw Error("reshape: bad shape");
    if (numel_of(out) != numel_of(S(0))) throw Error("reshape: element count differs");
    return out;
  }
  if (k == "expand") {
    need(1, 1);
    Shape out = get_attr(op, "shape");
    const Shape& x = S(0);
    if (out.size() < x.size()) throw Error("expand: rank too small");
    for (size_t d = 0; d < x.size(); ++d) {
      int64_t od = out[out.size() - x.size() + d];
      if (x[d] != od && x[d] != 1) throw Error("expand: incompatible");
    }
    return out;
  }
  if (k == "affine_gather") {
    if (op.in.empty()) throw Error("affine_gather: needs operands");
    Shape out = get_attr(op, "shape");
    auto win = get_attr_or(op, "window", {});
    for (int64_t d : out) if (d <= 0) throw Error("affine_gather: bad shape");
    for (int64_t d : win) if (d <= 0) throw Error("affine_gather: bad window");
    auto mult = get_attr_or(op, "mult", std::vector<int64_t>(op.in.size(), 1));
    if (mult.size() != op.in.size()) throw Error("affine_gather: mult length");
    for (int64_t m : mult) if (m <= 0) throw Error("affine_gather: multiplicity must be positive");
    int64_t wn = numel_of(win);
    auto fl = get_attr_or(op, "flat", {0, wn});
    if (fl.size() != 2 || fl[0] < 0 || fl[1] > wn || fl[0] > fl[1]) throw Error("affine_gather: bad flat range");
    for (size_t j = 0; j < op.in.size(); ++j) {
      if (op.idx[j].size() != S(j).size()) throw Error("affine_gather: index rank differs from operand rank");
      for (const Expr& e : op.idx[j])
        for (const auto& t : e.terms) {
          if (t.var == 'o' && (t.index < 0 || t.index >= (int)out.size())) throw Error("affine_gather: bad o index");
          if (t.var == 'w' && (t.index < 0 || t.index >= (int)win.size())) throw Error("affine_gather: bad w index");
        }
    }
    return out;
  }
  throw Error("unsupported op '" + k + "'");
}

std::vector<std::string> split_ws(const std::string& s) {
  std::vector<std::string> out;
  std::istringstream is(s);
  std::string t;
  while (is >> t) out.push_back(t);
  return out;
}

std::vector<std::string> split_char(const std::string& s, char c) {
  std::vector<std::string> out;
  std::string cur;
  for (char ch : s) {
    if (ch == c) { out.push_back(cur); cur.clear(); }
    else cur.push_back(ch);
  }
  out.push_back(cur);
  return out;
}

std::vector<int64_t> parse_ints(const std::string& s) {
  std::vector<int64_t> v;
  for (const std::string& p : split_char(s, ',')) {
    if (p.empty()) throw Error("empty integer in '" + s + "'");
    size_t pos = 0;
    int64_t x = std::stoll(p, &pos);
    if (pos != p.size()) throw Error("bad integer '" + p + "'");
    v.push_back(x);
  }
  return v;
}

bool valid_name(const std::string& n) {
  if (n.empty() || !(isalpha((unsigned char)n[0]) || n[0] == '_')) return false;
  for (char c : n) if (!(isalnum((unsigned char)c) || c == '_')) return false;
  return true;
}

Graph parse_graph(const std::string& text) {
  Graph g;
  std::istringstream is(text);
  std::string line;
  int lineno = 0;
  bool header = false;
  Shape declared_out;
  while (std::getline(is, line)) {
    ++lineno;
    size_t hash = line.find('#');
    if (hash != std::string::npos) line = line.substr(0, hash);
    auto toks = split_ws(line);
    if (toks.empty()) continue;
    try {
      if (!header) {
        if (toks.size() != 2 || toks[0] != "dgir" || toks[1] != "1") throw Error("expected 'dgir 1' header");
        header = true;
        continue;
      }
      if (g.output >= 0) throw Error("statement after 'output'");
      if (toks[0] == "leaf") {
        if (toks.size() != 3) throw Error("leaf: expected 'leaf <name> <shape>'");
        if (!valid_name(toks[1]) || g.by_name.count(toks[1])) throw Error("leaf: bad or duplicate name");
        Tensor t;
        t.name = toks[1];
        t.shape = parse_ints(toks[2]);
        for (int64_t d : t.shape) if (d <= 0) throw Error("leaf: dimensions must be positive");
        t.leaf = true;
        t.leaf_index = (int)g.leaves.size();
        t.base = g.leaf_total;
        g.leaf_total += (uint64_t)numel_of(t.shape);
        if (g.leaf_total > (1ull << 62)) throw Error("leaf elements exceed 2^62");
        g.by_name[t.name] = (int)g.tensors.size();
        g.leaves.push_back((int)g.tensors.size());
        g.tensors.push_back(t);
      } else if (toks[0] == "op") {
        if (toks.size() < 4) throw Error("op: expected 'op <name> <kind> <operands...>'");
        if (!valid_name(toks[1]) || g.by_name.count(toks[1])) throw Error("op: bad or duplicate name");
        Op op;
        op.kind = toks[2];
        size_t i = 3;
        for (; i < toks.size() && toks[i] != ";"; ++i) {
          auto it = g.by_name.find(toks[i]);
          if (it == g.by_name.end()) throw Error("op: unknown operand '" + toks[i] + "'");
          op.in.push_back(it->second);
        }
        std::map<std::string, std::string> raw;
        if (i < toks.size()) {
          for (++i; i < toks.size(); ++i) {
            size_t eq = toks[i].find('=');
            if (eq == std::string::npos) throw Error("op: expected key=value");
            raw[toks[i].substr(0, eq)] = toks[i].substr(eq + 1);
          }
        }
        op.raw = raw;
        if (op.kind == "affine_gather") {
          op.idx.resize(op.in.size());
          for (size_t j = 0; j < op.in.size(); ++j) {
            auto it = raw.find("idx" + std::to_string(j));
            if (it == raw.end()) throw Error("affine_gather: missing idx" + std::to_string(j));
            for (const std::string& e : split_char(it->second, ',')) op.idx[j].push_back(parse_expr(e));
            raw.erase(it);
          }
        }
        for (auto& kv : raw) op.attr[kv.first] = parse_ints(kv.second);
        Tensor t;
        t.name = toks[1];
        op.out = (int)g.tensors.size();
        t.shape = infer_shape(g, op);
        numel_of(t.shape);  // at most 2^62 elements
        g.by_name[t.name] = (int)g.tensors.size();
        g.tensors.push_back(t);
        g.ops.push_back(op);
      } else if (toks[0] == "output") {
        if (toks.size() != 3) throw Error("output: expected 'output <name> <shape>'");
        auto it = g.by_name.find(toks[1]);
        if (it == g.by_name.end()) throw Error("output: unknown tensor");
        g.output = it->second;
        declared_out = parse_ints(toks[2]);
        if (declared_out != g.tensors[g.output].shape) throw Error("output: declared shape differs from the inferred one");
      } else {
        throw Error("unknown statement '" + toks[0] + "'");
      }
    } catch (const Error& e) {
      throw Error("line " + std::to_string(lineno) + ": " + e.what());
    } catch (const std::exception& e) {
      throw Error("line " + std::to_string(lineno) + ": " + e.what());
    }
  }
  if (!header) throw Error("missing 'dgir 1' header");
  if (g.output < 0) throw Error("missing 'output' statement");
  if (g.leaf_total > (1ull << 62)) throw Error("leaf elements exceed 2^62");
  return g;
}

// ---------------------------------------------------------------------------
// R_k(l): the multiset of element references of op k at its output location l.
// `emit(tensor, flat_index, multiplicity)` is called once per reference group.
// ---------------------------------------------------------------------------
typedef std::function<void(int, int64_t, uint64_t)> Emit;

// Calls f on every multi-index of the box `ext` (row-major order).
void for_box(const Shape& ext, const std::function<void(const Shape&)>& f) {
  for (int64_t e : ext) if (e <= 0) return;
  Shape i(ext.size(), 0);
  while (true) {
    f(i);
    int d = (int)ext.size() - 1;
    for (; d >= 0; --d) {
      if (++i[d] < ext[d]) break;
      i[d] = 0;
    }
    if (d < 0) return;
  }
}

void op_reads(const Graph& g, const Op& op, int64_t loc, const Emit& emit) {
  const Shape& oshape = g.tensors[op.out].shape;
  const Shape o = unravel(loc, oshape);
  auto S = [&](int i) -> const Shape& { return g.tensors[op.in[i]].shape; };
  const std::string& k = op.kind;

  if (kUnary.count(k)) {  // one uninterpreted function of the operand
    emit(op.in[0], loc, 1);
    return;
  }
  if (kBinary.count(k)) {  // each operand at its broadcast index
    emit(op.in[0], broadcast_flat(o, S(0)), 1);
    emit(op.in[1], broadcast_flat(o, S(1)), 1);
    return;
  }
  if (k == "matmul") {  // out[.., i, j] = sum_k A[.., i, k] * B[.., k, j]
    const Shape &a = S(0), &b = S(1);
    size_t r = o.size();
    int64_t i = o[r - 2], j = o[r - 1], K = a[a.size() - 1];
    Shape ob(o.begin(), o.end() - 2);
    Shape ab(a.begin(), a.end() - 2), bb(b.begin(), b.end() - 2);
    int64_t abase = broadcast_flat(ob, ab), bbase = broadcast_flat(ob, bb);
    int64_t M = a[a.size() - 2], N = b[b.size() - 1];
    for (int64_t kk = 0; kk < K; ++kk) {
      emit(op.in[0], (abase * M + i) * K + kk, 1);
      emit(op.in[1], (bbase * K + kk) * N + j, 1);
    }
    return;
  }
  if (k == "linear") {  // y[.., j] = sum_k x[.., k] * W[j, k] + b[j]
    const Shape& w = S(1);
    int64_t K = w[1], j = o.back();
    int64_t xrow = loc / oshape.back();
    for (int64_t kk = 0; kk < K; ++kk) {
      emit(op.in[0], xrow * K + kk, 1);
      emit(op.in[1], j * K + kk, 1);
    }
    if (op.in.size() == 3) emit(op.in[2], j, 1);
    return;
  }
  if (k == "conv") {
    // out[n, co, o..] = sum over ci in co's group, taps t with
    // i = o*s - p + t*d inside x in every dim, of x[n, ci, i..] * W[co, ci_l, t..];
    // plus b[co].  Padding taps read a constant zero: neither x nor W is read.
    const Shape &x = S(0), &w = S(1);
    size_t nsp = x.size() - 2;
    auto st = get_attr_or(op, "stride", std::vector<int64_t>(nsp, 1));
    auto pd = get_attr_or(op, "pad", std::vector<int64_t>(nsp, 0));
    auto dl = get_attr_or(op, "dilation", std::vector<int64_t>(nsp, 1));
    int64_t G = get_scalar(op, "groups", 1);
    int64_t cin_g = x[1] / G, cout_g = w[0] / G;
    int64_t n = o[0], co = o[1], grp = co / cout_g;
    Shape kext(w.begin() + 2, w.end());
    for (int64_t cl = 0; cl < cin_g; ++cl) {
      for_box(kext, [&](const Shape& t) {
        Shape xi(x.size()), wi(w.size());
        xi[0] = n;
        xi[1] = grp * cin_g + cl;
        wi[0] = co;
        wi[1] = cl;
        for (size_t d = 0; d < nsp; ++d) {
          int64_t i = o[2 + d] * st[d] - pd[d] + t[d] * dl[d];
          if (i < 0 || i >= x[2 + d]) return;
          xi[2 + d] = i;
          wi[2 + d] = t[d];
        }
        emit(op.in[0], ravel(xi, x), 1);
        emit(op.in[1], ravel(wi, w), 1);
      });
    }
    if (op.in.size() == 3) emit(op.in[2], co, 1);
    return;
  }
  if (k == "conv_transpose") {
    // Scatter form: input x[n, ci, i..] with W[ci, co_l, t..] lands on
    // out[n, co, i*s - p + t*d ..].  The reads of out[l] are every (ci, i, t)
    // of co's group with i*s - p + t*d == o in every dim and i inside x;
    // plus b[co].  The condition is tested per dim by looping over all taps
    // and input positions of that dim.  Order: ci, then taps ascending in
    // row-major order (the canonical order of the summation, as in conv).
    const Shape &x = S(0), &w = S(1);
    size_t nsp = x.size() - 2;
    auto st = get_attr_or(op, "stride", std::vector<int64_t>(nsp, 1));
    auto pd = get_attr_or(op, "pad", std::vector<int64_t>(nsp, 0));
    auto dl = get_attr_or(op, "dilation", std::vector<int64_t>(nsp, 1));
    int64_t G = get_scalar(op, "groups", 1);
    int64_t cin_g = x[1] / G, cout_g = w[1];
    int64_t n = o[0], co = o[1], grp = co / cout_g, col = co % cout_g;
    std::vector<std::vector<std::pair<int64_t, int64_t>>> pairs(nsp);  // (i, t) per dim
    for (size_t d = 0; d < nsp; ++d)
      for (int64_t t = 0; t < w[2 + d]; ++t)
        for (int64_t i = 0; i < x[2 + d]; ++i)
          if (i * st[d] - pd[d] + t * dl[d] == o[2 + d]) pairs[d].push_back({i, t});
    Shape pext(nsp);
    for (size_t d = 0; d < nsp; ++d) pext[d] = (int64_t)pairs[d].size();
    for (int64_t ci = grp * cin_g; ci < (grp + 1) * cin_g; ++ci) {
      for_box(pext, [&](const Shape& p) {
        Shape xi(x.size()), wi(w.size());
        xi[0] = n;
        xi[1] = ci;
        wi[0] = ci;
        wi[1] = col;
        for (size_t d = 0; d < nsp; ++d) {
          xi[2 + d] = pairs[d][p[d]].first;
          wi[2 + d] = pairs[d][p[d]].second;
        }
        emit(op.in[0], ravel(xi, x), 1);
        emit(op.in[1], ravel(wi, w), 1);
      });
    }
    if (op.in.size() == 3) emit(op.in[2], co, 1);
    return;
  }
  if (k == "max_pool" || k == "avg_pool") {
    // Every in-range window element; padding is never read.
    const Shape& x = S(0);
    auto ks = get_attr(op, "kernel");
    size_t nsp = ks.size();
    auto st = get_attr_or(op, "stride", ks);
    auto pd = get_attr_or(op, "pad", std::vector<int64_t>(nsp, 0));
    auto dl = get_attr_or(op, "dilation", std::vector<int64_t>(nsp, 1));
    size_t lead = x.size() - nsp;
    for_box(Shape(ks.begin(), ks.end()), [&](const Shape& t) {
      Shape xi(x.size());
      for (size_t d = 0; d < lead; ++d) xi[d] = o[d];
      for (size_t d = 0; d < nsp; ++d) {
        int64_t i = o[lead + d] * st[d] - pd[d] + t[d] * dl[d];
        if (i < 0 || i >= x[lead + d]) return;
        xi[lead + d] = i;
      }
      emit(op.in[0], ravel(xi, x), 1);
    });
    return;
  }
  if (kReduce.count(k)) {  // every element of the reduced slice
    const Shape& x = S(0);
    auto dims = get_attr(op, "dims");
    bool keep = get_scalar(op, "keepdim", 0) != 0;
    std::vector<bool> red(x.size(), false);
    for (int64_t d : dims) red[norm_dim(d, x.size())] = true;
    Shape kept;  // x index for kept dims, from o
    size_t oi = 0;
    Shape xi(x.size(), 0);
    Shape rext;
    std::vector<int> rdims;
    bool full = true;
    for (size_t d = 0; d < x.size(); ++d) if (!red[d]) full = false;
    for (size_t d = 0; d < x.size(); ++d) {
      if (red[d]) {
        rdims.push_back((int)d);
        rext.push_back(x[d]);
        if (keep) ++oi;
      } else {
        xi[d] = o[oi++];
      }
    }
    (void)full;
    for_box(rext, [&](const Shape& r) {
      Shape idx = xi;
      for (size_t j = 0; j < rdims.size(); ++j) idx[rdims[j]] = r[j];
      emit(op.in[0], ravel(idx, x), 1);
    });
    return;
  }
  if (k == "softmax" || k == "log_softmax") {
    // Canonical form exp(x[l]) / sum_D exp(x): the slice along D once, and
    // x[l] once more through the numerator (log_softmax: x[l] - log sum exp).
    const Shape& x = S(0);
    int dim = norm_dim(get_scalar(op, "dim", 0, true), x.size());
    Shape xi = o;
    for (int64_t j = 0; j < x[dim]; ++j) {
      xi[dim] = j;
      emit(op.in[0], ravel(xi, x), 1);
    }
    emit(op.in[0], loc, 1);
    return;
  }
  if (k == "group_norm" || k == "batch_norm" || k == "layer_norm") {
    // Decomposition: mu = mean_S(x); d = x - mu; v = mean_S(square(d));
    // r = rsqrt(v + eps); y = d * r * gamma + beta, with S the statistics
    // set of l.  Every s in S is reached once through mu inside d[l], and
    // |S| + 1 times through r (each d[s'] in v reads mu, and d[s] reads
    // x[s]); x[l] once more through d[l].  So x[s] counts |S| + 2, x[l] one
    // more, and gamma, beta at l's channel once each.
    const Shape& x = S(0);
    Shape box_lo(x.size(), 0), box_ext(x.size());
    int64_t aff = 0;
    if (k == "group_norm") {
      int64_t G = get_scalar(op, "groups", 0, true);
      int64_t cg = x[1] / G;
      for (size_t d = 0; d < x.size(); ++d) box_ext[d] = x[d];
      box_lo[0] = o[0];
      box_ext[0] = 1;
      box_lo[1] = (o[1] / cg) * cg;
      box_ext[1] = cg;
      aff = o[1];
    } else if (k == "batch_norm") {
      for (size_t d = 0; d < x.size(); ++d) box_ext[d] = x[d];
      box_lo[1] = o[1];
      box_ext[1] = 1;
      aff = o[1];
    } else {
      int64_t nd = get_scalar(op, "ndims", 1);
      size_t lead = x.size() - nd;
      Shape tail;
      for (size_t d = 0; d < x.size(); ++d) {
        if (d < lead) { box_lo[d] = o[d]; box_ext[d] = 1; }
        else { box_ext[d] = x[d]; tail.push_back(x[d]); }
      }
      Shape ti(o.begin() + lead, o.end());
      aff = ravel(ti, tail);
    }
    uint64_t size = (uint64_t)numel_of(box_ext);
    for_box(box_ext, [&](const Shape& r) {
      Shape idx(x.size());
      for (size_t d = 0; d < x.size(); ++d) idx[d] = box_lo[d] + r[d];
      emit(op.in[0], ravel(idx, x), size + 2);
    });
    emit(op.in[0], loc, 1);
    if (op.in.size() == 3) {
      emit(op.in[1], aff, 1);
      emit(op.in[2], aff, 1);
    }
    return;
  }
  if (k == "channel_affine") {  // x[l] * scale[c] + shift[c]
    emit(op.in[0], loc, 1);
    emit(op.in[1], o[1], 1);
    emit(op.in[2], o[1], 1);
    return;
  }
  if (k == "slice") {
    const Shape& x = S(0);
    int dim = (int)get_scalar(op, "dim", 0);
    Shape xi = o;
    xi[dim] = get_scalar(op, "start", 0) + o[dim] * get_scalar(op, "step", 1);
    emit(op.in[0], ravel(xi, x), 1);
    return;
  }
  if (k == "permute") {  // out[o] = x[i] with i[perm[k]] = o[k]
    const Shape& x = S(0);
    auto p = get_attr(op, "dims");
    Shape xi(x.size());
    for (size_t q = 0; q < p.size(); ++q) xi[p[q]] = o[q];
    emit(op.in[0], ravel(xi, x), 1);
    return;
  }
  if (k == "reshape") {  // same flat index
    emit(op.in[0], loc, 1);
    return;
  }
  if (k == "expand") {
    emit(op.in[0], broadcast_flat(o, S(0)), 1);
    return;
  }
  if (k == "affine_gather") {
    // For every window point w (row-major flat index inside the declared
    // range) compute every operand's index; the point contributes only when
    // all of them are in range (and exactly divisible), as in a product of
    // the operands; then each operand is read with its multiplicity.
    Shape win = get_attr_or(op, "window", {});
    int64_t wn = numel_of(win);
    auto fl = get_attr_or(op, "flat", {0, wn});
    auto mult = get_attr_or(op, "mult", std::vector<int64_t>(op.in.size(), 1));
    for (int64_t f = fl[0]; f < fl[1]; ++f) {
      Shape w = unravel(f, win);
      std::vector<int64_t> flats(op.in.size());
      bool ok = true;
      for (size_t j = 0; j < op.in.size() && ok; ++j) {
        const Shape& s = S((int)j);
        Shape idx(s.size());
        for (size_t d = 0; d < s.size(); ++d) {
          int64_t v;
          if (!eval_expr(op.idx[j][d], o, w, &v) || v < 0 || v >= s[d]) { ok = false; break; }
          idx[d] = v;
        }
        if (ok) flats[j] = ravel(idx, s);
      }
      if (!ok) continue;
      for (size_t j = 0; j < op.in.size(); ++j) emit(op.in[j], flats[j], (uint64_t)mult[j]);
    }
    return;
  }
  throw Error("unsupported op '" + k + "'");
}

uint64_t checked_add(uint64_t a, uint64_t b) {
  uint64_t r;
  if (__builtin_add_overflow(a, b, &r)) throw Error("path count overflows 64 bits");
  return r;
}

uint64_t checked_mul(uint64_t a, uint64_t b) {
  uint64_t r;
  if (__builtin_mul_overflow(a, b, &r)) throw Error("path count overflows 64 bits");
  return r;
}

typedef std::vector<std::pair<uint64_t, uint64_t>> Row;

// Back-projection of one output location to its leaf multiset.
Row enumerate_one(const Graph& g, int64_t loc) {
  int64_t onumel = numel_of(g.tensors[g.output].shape);
  if (loc < 0 || loc >= onumel) throw Error("location out of range");
  std::vector<std::map<int64_t, uint64_t>> F(g.tensors.size());
  F[g.output][loc] = 1;
  for (int k = (int)g.ops.size() - 1; k >= 0; --k) {
    const Op& op = g.ops[k];
    std::map<int64_t, uint64_t> front;
    front.swap(F[op.out]);
    for (const auto& kv : front) {
      uint64_t c = kv.second;
      op_reads(g, op, kv.first, [&](int t, int64_t idx, uint64_t m) {
        uint64_t& slot = F[t][idx];
        slot = checked_add(slot, checked_mul(c, m));
      });
    }
  }
  Row row;
  for (int t : g.leaves) {
    const Tensor& T = g.tensors[t];
    for (const auto& kv : F[t]) row.push_back({T.base + (uint64_t)kv.first, kv.second});
  }
  return row;
}

// The 32-bit form of a row: every count must fit 32 bits (ids do when the
// graph has at most 2^32 - 1 leaf elements, checked once per call).
const Row& narrow(const Row& row) {
  for (const auto& e : row)
    if (e.second > 0xFFFFFFFFull) throw Error("path count exceeds 32 bits");
  return row;
}

void require_narrow_ids(const Graph& g) {
  if (g.leaf_total > 0xFFFFFFFFull) throw Error("leaf ids need 64 bits");
}

struct Result {
  std::vector<int64_t> offsets;
  std::vector<uint64_t> ids, counts;
};

// ---------------------------------------------------------------------------
// Expression DAG of res(y[l]) (Sec. 3.4, "Back-projection"): every tensor
// element in the cone of y[l] is one node, shared wherever it occurs; a leaf
// element is a variable, any other node is its op applied to the element
// references of its per-element equation, in the equation's order.
//
// Global element ids: a leaf element keeps its id (leaf base + flat index);
// the output of op k (SSA order) follows all leaves, at
// leaf_total + sum of the element counts of ops 0..k-1, plus its flat index.
// Nodes: the non-leaf cone elements, ops in reverse SSA order (y[l] first),
// elements ascending within an op.  Edges of a node: R_k(e) in the order the
// read enumeration lists it (operands in equation order; sums over windows
// in row-major window order), as (child id, multiplicity).
// ---------------------------------------------------------------------------
struct Dag {
  std::vector<uint64_t> nodes, node_edge;  // node_edge: first edge, relative to the location's first
  std::vector<uint64_t> edges, mults;
};

std::vector<uint64_t> op_bases(const Graph& g) {
  std::vector<uint64_t> base(g.ops.size());
  uint64_t b = g.leaf_total;
  for (size_t k = 0; k < g.ops.size(); ++k) {
    base[k] = b;
    b += (uint64_t)numel_of(g.tensors[g.ops[k].out].shape);
  }
  return base;
}

Dag dag_one(const Graph& g, const std::vector<uint64_t>& obase, int64_t loc) {
  int64_t onumel = numel_of(g.tensors[g.output].shape);
  if (loc < 0 || loc >= onumel) throw Error("location out of range");
  std::vector<int> producer(g.tensors.size(), -1);
  for (size_t k = 0; k < g.ops.size(); ++k) producer[g.ops[k].out] = (int)k;
  std::vector<std::set<int64_t>> F(g.tensors.size());
  F[g.output].insert(loc);
  Dag d;
  for (int k = (int)g.ops.size() - 1; k >= 0; --k) {
    const Op& op = g.ops[k];
    for (int64_t e : F[op.out]) {
      d.nodes.push_back(obase[k] + (uint64_t)e);
      d.node_edge.push_back(d.edges.size());
      op_reads(g, op, e, [&](int t, int64_t idx, uint64_t m) {
        const Tensor& T = g.tensors[t];
        d.edges.push_back(producer[t] < 0 ? T.base + (uint64_t)idx : obase[producer[t]] + (uint64_t)idx);
        d.mults.push_back(m);
        if (producer[t] >= 0) F[t].insert(idx);
      });
    }
  }
  return d;
}

struct DagResult {
  std::vector<int64_t> node_offsets, edge_offsets;
  std::vector<uint64_t> nodes, node_edge, edges, mults;
};

template <class F>
void parallel_blocks(int64_t n, int nthreads, F f) {
  if (nthreads <= 1 || n < 2) {
    f(0, n, 0);
    return;
  }
  int64_t nt = std::min<int64_t>(nthreads, n);
  std::vector<std::thread> th;
  std::vector<std::string> errs(nt);
  for (int64_t t = 0; t < nt; ++t) {
    int64_t lo = n * t / nt, hi = n * (t + 1) / nt;
    th.emplace_back([&, lo, hi, t] {
      try { f(lo, hi, (int)t); } catch (const std::exception& e) { errs[t] = e.what(); }
    });
  }
  for (auto& x : th) x.join();
  for (auto& e : errs) if (!e.empty()) throw Error(e);
}

Result enumerate_all(const Graph& g, const int64_t* locs, int64_t n, int nthreads, bool wide) {
  if (!wide) require_narrow_ids(g);
  std::vector<Row> rows(n);
  parallel_blocks(n, nthreads, [&](int64_t lo, int64_t hi, int) {
    for (int64_t i = lo; i < hi; ++i) {
      rows[i] = enumerate_one(g, locs[i]);
      if (!wide) narrow(rows[i]);
    }
  });
  Result r;
  r.offsets.resize(n + 1);
  r.offsets[0] = 0;
  for (int64_t i = 0; i < n; ++i) r.offsets[i + 1] = r.offsets[i] + (int64_t)rows[i].size();
  r.ids.reserve(r.offsets[n]);
  r.counts.reserve(r.offsets[n]);
  for (auto& row : rows)
    for (auto& e : row) { r.ids.push_back(e.first); r.counts.push_back(e.second); }
  return r;
}

void check_signature(const Graph& a, const Graph& b) {
  // MERGE's input/output matching (Sec. 3.2): both programs read the same
  // leaves and write an output of the same shape.
  if (a.leaves.size() != b.leaves.size()) throw Error("leaf count differs");
  for (size_t i = 0; i < a.leaves.size(); ++i) {
    const Tensor &x = a.tensors[a.leaves[i]], &y = b.tensors[b.leaves[i]];
    if (x.name != y.name || x.shape != y.shape) throw Error("leaf '" + x.name + "' differs");
  }
  if (a.tensors[a.output].shape != b.tensors[b.output].shape) throw Error("output shape differs");
}

// 0 equal, 1 the id sets differ, 2 same ids but some count differs.
uint8_t compare_rows(const Row& a, const Row& b) {
  if (a.size() != b.size()) return 1;
  for (size_t i = 0; i < a.size(); ++i) if (a[i].first != b[i].first) return 1;
  for (size_t i = 0; i < a.size(); ++i) if (a[i].second != b[i].second) return 2;
  return 0;
}

DagResult dag_all(const Graph& g, const int64_t* locs, int64_t n, int nthreads) {
  const std::vector<uint64_t> obase = op_bases(g);
  std::vector<Dag> dags(n);
  parallel_blocks(n, nthreads, [&](int64_t lo, int64_t hi, int) {
    for (int64_t i = lo; i < hi; ++i) dags[i] = dag_one(g, obase, locs[i]);
  });
  DagResult r;
  r.node_offsets.assign(n + 1, 0);
  r.edge_offsets.assign(n + 1, 0);
  for (int64_t i = 0; i < n; ++i) {
    r.node_offsets[i + 1] = r.node_offsets[i] + (int64_t)dags[i].nodes.size();
    r.edge_offsets[i + 1] = r.edge_offsets[i] + (int64_t)dags[i].edges.size();
  }
  for (auto& d : dags) {
    r.nodes.insert(r.nodes.end(), d.nodes.begin(), d.nodes.end());
    r.node_edge.insert(r.node_edge.end(), d.node_edge.begin(), d.node_edge.end());
    r.edges.insert(r.edges.end(), d.edges.begin(), d.edges.end());
    r.mults.insert(r.mults.end(), d.mults.begin(), d.mults.end());
  }
  return r;
}

thread_local std::string g_err;

}  // namespace

namespace {

// ---- location order (Sec. 4, "Search Heuristic") ---------------------------
// Candidate locations are ranked before the rest: corner locations of every
// kernel launch (later launches first), then the first and last element of
// the output; the remaining locations follow in a random permutation.
// Readings (the paper's launches are CUDA kernels; here every op is one
// launch writing its output row-major, one element per thread):
//  - corner threads: first and last thread of the first and last block,
//    lanes warp-1 and warp of block 0;
//  - a corner element becomes an output location through reads that are one
//    to one (at every output element of the reading op, its reads of the
//    tensor name exactly one element, and distinct output elements name
//    distinct elements); the smallest location over such paths is taken;
//  - a location is listed once, at its first rank.

// Whether `op` reads tensor t one to one; back[o] = the element read at o.
bool reads_one_to_one(const Graph& g, const Op& op, int t, std::vector<int64_t>* back) {
  const int64_t m = numel_of(g.tensors[op.out].shape);
  if (numel_of(g.tensors[t].shape) != m) return false;
  back->assign((size_t)m, -1);
  std::vector<char> hit((size_t)m, 0);
  for (int64_t o = 0; o < m; ++o) {
    int64_t e = -1;
    bool one = true;
    op_reads(g, op, o, [&](int tt, int64_t ii, uint64_t) {
      if (tt != t) return;
      if (e < 0) e = ii;
      else if (e != ii) one = false;
    });
    if (!one || e < 0 || hit[(size_t)e]) return false;
    hit[(size_t)e] = 1;
    (*back)[(size_t)o] = e;
  }
  return true;
}

std::vector<int64_t> order_prefix(const Graph& g, int64_t threads, int64_t warp) {
  if (threads < 1 || warp < 1) throw Error("threads and warp must be positive");
  const int64_t n = numel_of(g.tensors[g.output].shape);
  // loc[t][e]: smallest output location whose chain of one-to-one reads
  // back from the output reaches element e of tensor t (-1: none).  Ops in
  // reverse SSA order: every consumer of an op's output comes first.
  std::map<int, std::vector<int64_t>> loc;
  std::vector<int64_t>& ly = loc[g.output];
  ly.resize((size_t)n);
  for (int64_t l = 0; l < n; ++l) ly[(size_t)l] = l;
  for (int k = (int)g.ops.size() - 1; k >= 0; --k) {
    const Op& op = g.ops[k];
    if (!loc.count(op.out)) continue;
    std::set<int> operands(op.in.begin(), op.in.end());
    for (int t : operands) {
      std::vector<int64_t> back;
      if (!reads_one_to_one(g, op, t, &back)) continue;
      std::vector<int64_t>& lt = loc[t];
      if (lt.empty()) lt.assign((size_t)numel_of(g.tensors[t].shape), -1);
      const std::vector<int64_t>& lo = loc[op.out];
      for (size_t o = 0; o < back.size(); ++o) {
        const int64_t l = lo[o];
        int64_t& dst = lt[(size_t)back[o]];
        if (l >= 0 && (dst < 0 || l < dst)) dst = l;
      }
    }
  }
  std::vector<int64_t> out;
  std::set<int64_t> seen;
  auto add = [&](int64_t l) {
    if (l >= 0 && seen.insert(l).second) out.push_back(l);
  };
  for (int k = (int)g.ops.size() - 1; k >= 0; --k) {
    const int t = g.ops[k].out;
    const int64_t m = numel_of(g.tensors[t].shape);
    if (m == 0) continue;
    const int64_t blocks = (m + threads - 1) / threads, last = (blocks - 1) * threads;
    // (thread 0, block 0), (last thread, block 0), (thread 0, last block),
    // (last thread, last block), then lanes warp-1 and warp of block 0.
    std::vector<int64_t> corner = {0, threads - 1, last, last + threads - 1};
    if (warp - 1 < threads) corner.push_back(warp - 1);
    if (warp < threads) corner.push_back(warp);
    for (int64_t e : corner) {
      if (e >= m) continue;
      auto it = loc.find(t);
      add(it == loc.end() ? -1 : it->second[(size_t)e]);
    }
  }
  if (n > 0) {
    add(0);
    add(n - 1);
  }
  return out;
}

// SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
// generators", 2014): state += golden gamma, then the output mix.
uint64_t splitmix_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Keyed permutation of [0, n): a balanced Feistel network (Luby and
// Rackoff, 1988) of four rounds on 2h bits, h the smallest with 4^h >= n;
// round r maps halves (L, R) to (R, L xor F_r(R)) with F_r(R) the SplitMix64
// output mix of (R xor key_r) cut to h bits and key_r the r-th SplitMix64
// output for `seed`.  Values at or past n are encrypted again until they
// fall below n (cycle walking: Black and Rogaway, "Ciphers with arbitrary
// finite domains", 2002).
struct Permutation {
  int h = 0;
  uint64_t mask = 0, key[4] = {0, 0, 0, 0};
  int64_t n = 0;
  Permutation(int64_t n_, uint64_t seed) : n(n_) {
    while (h < 31 && (1ull << (2 * h)) < (uint64_t)n) ++h;
    mask = (1ull << h) - 1;
    uint64_t state = seed;
    for (int r = 0; r < 4; ++r) {
      state += 0x9E3779B97F4A7C15ull;
      key[r] = splitmix_mix(state);
    }
  }
  uint64_t encrypt(uint64_t x) const {
    uint64_t L = x >> h, R = x & mask;
    for (int r = 0; r < 4; ++r) {
      uint64_t next = L ^ (splitmix_mix(R ^ key[r]) & mask);
      L = R;
      R = next;
    }
    return (L << h) | R;
  }
  uint64_t decrypt(uint64_t x) const {
    uint64_t L = x >> h, R = x & mask;
    for (int r = 3; r >= 0; --r) {
      uint64_t prev = R ^ (splitmix_mix(L ^ key[r]) & mask);
      R = L;
      L = prev;
    }
    return (L << h) | R;
  }
  int64_t at(int64_t i) const {
    uint64_t v = encrypt((uint64_t)i);
    while (v >= (uint64_t)n) v = encrypt(v);
    return (int64_t)v;
  }
};

}  // namespace

// ---------------------------------------------------------------------------
// C interface used by the Python test harness (ctypes).
// Returns 0 on success, -1 on error (message via dgo_error()).
// ---------------------------------------------------------------------------
namespace {

// ---- MERGE (Sec. 3.2): matched inputs, trimmed common prefix ----------------
// The two programs must take the same inputs: a leaf of b pairs with the leaf
// of a of the same name and shape, the others pair in declaration order among
// leaves of one shape.  Then the longest common prefix of ops (same kind,
// same attributes, paired operands) is trimmed; its results that a remaining
// op or an output still uses become inputs shared by both, after a's leaves
// in prefix order.  No suffix is trimmed.
struct Merged {
  std::string a, b;
  int trimmed = 0;
};

std::string shape_text(const Shape& s) {
  std::string o;
  for (size_t i = 0; i < s.size(); ++i) o += (i ? "," : "") + std::to_string(s[i]);
  return o;
}

std::string op_line(const Graph& g, const Op& op, const std::vector<std::string>& name) {
  std::string o = "op " + name[op.out] + " " + op.kind;
  for (int t : op.in) o += " " + name[t];
  if (!op.raw.empty()) {
    o += " ;";
    for (const auto& kv : op.raw) o += " " + kv.first + "=" + kv.second;
  }
  return o + "\n";
}

bool same_attrs(const Op& x, const Op& y) {
  if (x.kind != y.kind || x.in.size() != y.in.size() || x.attr != y.attr) return false;
  for (const auto& kv : x.raw)
    if (kv.first.compare(0, 3, "idx") == 0) {
      auto it = y.raw.find(kv.first);
      if (it == y.raw.end() || it->second != kv.second) return false;
    }
  return true;
}

Merged merge_programs(const Graph& a, const Graph& b, bool trim) {
  const size_t na = a.leaves.size(), nb = b.leaves.size();
  std::vector<int> pa(na, -1), pb(nb, -1);  // partner leaf positions
  for (size_t j = 0; j < nb; ++j)
    for (size_t i = 0; i < na; ++i) {
      const Tensor &x = a.tensors[a.leaves[i]], &y = b.tensors[b.leaves[j]];
      if (pa[i] < 0 && x.name == y.name && x.shape == y.shape) {
        pa[i] = (int)j;
        pb[j] = (int)i;
        break;
      }
    }
  for (size_t j = 0; j < nb; ++j) {
    if (pb[j] >= 0) continue;
    for (size_t i = 0; i < na; ++i)
      if (pa[i] < 0 && a.tensors[a.leaves[i]].shape == b.tensors[b.leaves[j]].shape) {
        pa[i] = (int)j;
        pb[j] = (int)i;
        break;
      }
    if (pb[j] < 0) throw Error("merge: an input of the second program has no partner");
  }
  for (size_t i = 0; i < na; ++i)
    if (pa[i] < 0) throw Error("merge: an input of the first program has no partner");
  if (a.tensors[a.output].shape != b.tensors[b.output].shape) throw Error("merge: output shapes differ");

  std::vector<int> same(b.tensors.size(), -1);  // tensor of a each tensor of b equals
  for (size_t j = 0; j < nb; ++j) same[b.leaves[j]] = a.leaves[pb[j]];
  size_t k = 0;
  for (; trim && k < a.ops.size() && k < b.ops.size(); ++k) {
    const Op &x = a.ops[k], &y = b.ops[k];
    if (!same_attrs(x, y)) break;
    bool operands = true;
    for (size_t q = 0; q < x.in.size(); ++q) operands = operands && same[y.in[q]] == x.in[q];
    if (!operands) break;
    same[y.out] = x.out;
  }
  // Prefix results still used (tensors of a).
  std::vector<int> prefix_op_a(a.tensors.size(), -1), prefix_op_b(b.tensors.size(), -1);
  for (size_t i = 0; i < k; ++i) {
    prefix_op_a[a.ops[i].out] = (int)i;
    prefix_op_b[b.ops[i].out] = (int)i;
  }
  std::set<int> used;
  for (size_t i = k; i < a.ops.size(); ++i)
    for (int t : a.ops[i].in)
      if (prefix_op_a[t] >= 0) used.insert(t);
  for (size_t i = k; i < b.ops.size(); ++i)
    for (int t : b.ops[i].in)
      if (prefix_op_b[t] >= 0) used.insert(same[t]);
  if (prefix_op_a[a.output] >= 0) used.insert(a.output);
  if (prefix_op_b[b.output] >= 0) used.insert(same[b.output]);

  std::string leaves;
  std::set<std::string> taken;
  for (int t : a.leaves) {
    leaves += "leaf " + a.tensors[t].name + " " + shape_text(a.tensors[t].shape) + "\n";
    taken.insert(a.tensors[t].name);
  }
  for (size_t i = 0; i < k; ++i)
    if (used.count(a.ops[i].out)) {
      const Tensor& t = a.tensors[a.ops[i].out];
      leaves += "leaf " + t.name + " " + shape_text(t.shape) + "\n";
      taken.insert(t.name);
    }
  Merged m;
  m.trimmed = (int)k;
  std::vector<std::string> an(a.tensors.size());
  for (size_t t = 0; t < a.tensors.size(); ++t) an[t] = a.tensors[t].name;
  m.a = "dgir 1\n" + leaves;
  for (size_t i = k; i < a.ops.size(); ++i) m.a += op_line(a, a.ops[i], an);
  m.a += "output " + an[a.output] + " " + shape_text(a.tensors[a.output].shape) + "\n";
  std::vector<std::string> bn(b.tensors.size());
  std::set<std::string> names = taken;
  for (size_t t = 0; t < b.tensors.size(); ++t) {
    if (same[t] >= 0) {
      bn[t] = a.tensors[same[t]].name;
      continue;
    }
    std::string nm = b.tensors[t].name;
    for (int s = 1; names.count(nm); ++s) nm = b.tensors[t].name + "_" + std::to_string(s);
    names.insert(nm);
    bn[t] = nm;
  }
  m.b = "dgir 1\n" + leaves;
  for (size_t i = k; i < b.ops.size(); ++i) m.b += op_line(b, b.ops[i], bn);
  m.b += "output " + bn[b.output] + " " + shape_text(b.tensors[b.output].shape) + "\n";
  return m;
}

}  // namespace

extern "C" {

struct dgo_graph { Graph g; };
struct dgo_result { Result r; };

const char* dgo_error(void) { return g_err.c_str(); }

dgo_graph* dgo_parse(const char* text, int64_t len) {
  try {
    auto* h = new dgo_graph;
    h->g = parse_graph(std::string(text, (size_t)len));
    return h;
  } catch (const std::exception& e) {
    g_err = e.what();
    return nullptr;
  }
}

void dgo_free(dgo_graph* g) { delete g; }

int64_t dgo_output_numel(const dgo_graph* g) { return numel_of(g->g.tensors[g->g.output].shape); }
int dgo_output_rank(const dgo_graph* g) { return (int)g->g.tensors[g->g.output].shape.size(); }
int dgo_num_leaves(const dgo_graph* g) { return (int)g->g.leaves.size(); }
int dgo_num_tensors(const dgo_graph* g) { return (int)g->g.tensors.size(); }
uint64_t dgo_leaf_total(const dgo_graph* g) { return g->g.leaf_total; }

// Tensor t: name, rank, shape (up to 8 dims), leaf index (-1 if produced by an op), base id.
int dgo_tensor_info(const dgo_graph* g, int t, char* name, int name_len, int64_t* shape, int* rank,
                    int* leaf_index, uint64_t* base) {
  if (t < 0 || t >= (int)g->g.tensors.size()) { g_err = "bad tensor index"; return -1; }
  const Tensor& T = g->g.tensors[t];
  snprintf(name, (size_t)name_len, "%s", T.name.c_str());
  *rank = (int)T.shape.size();
  for (size_t d = 0; d < T.shape.size() && d < 8; ++d) shape[d] = T.shape[d];
  *leaf_index = T.leaf_index;
  *base = T.base;
  return 0;
}

int dgo_output_tensor(const dgo_graph* g) { return g->g.output; }

// wide = 0: 32-bit ids and counts; wide = 1: 64-bit ids and counts.
dgo_result* dgo_enumerate(const dgo_graph* g, const int64_t* locs, int64_t n, int nthreads, int wide) {
  try {
    auto* r = new dgo_result;
    r->r = enumerate_all(g->g, locs, n, nthreads, wide != 0);
    return r;
  } catch (const std::exception& e) {
    g_err = e.what();
    return nullptr;
  }
}

int64_t dgo_result_total(const dgo_result* r) { return r->r.offsets.back(); }

// Copies a result made with dgo_enumerate(..., wide = 0).
void dgo_result_copy(const dgo_result* r, int64_t* offsets, uint32_t* ids, uint32_t* counts) {
  memcpy(offsets, r->r.offsets.data(), r->r.offsets.size() * sizeof(int64_t));
  for (size_t i = 0; i < r->r.ids.size(); ++i) {
    ids[i] = (uint32_t)r->r.ids[i];
    counts[i] = (uint32_t)r->r.counts[i];
  }
}

// Copies a result made with dgo_enumerate(..., wide = 1).
void dgo_result_copy_wide(const dgo_result* r, int64_t* offsets, uint64_t* ids, uint64_t* counts) {
  memcpy(offsets, r->r.offsets.data(), r->r.offsets.size() * sizeof(int64_t));
  if (!r->r.ids.empty()) {
    memcpy(ids, r->r.ids.data(), r->r.ids.size() * sizeof(uint64_t));
    memcpy(counts, r->r.counts.data(), r->r.counts.size() * sizeof(uint64_t));
  }
}

void dgo_result_free(dgo_result* r) { delete r; }

struct dgo_dag { DagResult r; };

// Global id of element 0 of tensor t (leaf base, or the op output's base).
uint64_t dgo_tensor_gid(const dgo_graph* g, int t) {
  const Graph& G = g->g;
  if (G.tensors[t].leaf_index >= 0) return G.tensors[t].base;
  std::vector<uint64_t> obase = op_bases(G);
  for (size_t k = 0; k < G.ops.size(); ++k) if (G.ops[k].out == t) return obase[k];
  return 0;
}

dgo_dag* dgo_dag_build(const dgo_graph* g, const int64_t* locs, int64_t n, int nthreads) {
  try {
    auto* r = new dgo_dag;
    r->r = dag_all(g->g, locs, n, nthreads);
    return r;
  } catch (const std::exception& e) {
    g_err = e.what();
    return nullptr;
  }
}

void dgo_dag_totals(const dgo_dag* d, int64_t* nodes, int64_t* edges) {
  *nodes = d->r.node_offsets.back();
  *edges = d->r.edge_offsets.back();
}

void dgo_dag_copy(const dgo_dag* d, int64_t* node_offsets, int64_t* edge_offsets, uint64_t* nodes,
                  uint64_t* node_edge, uint64_t* edges, uint64_t* mults) {
  const DagResult& r = d->r;
  memcpy(node_offsets, r.node_offsets.data(), r.node_offsets.size() * sizeof(int64_t));
  memcpy(edge_offsets, r.edge_offsets.data(), r.edge_offsets.size() * sizeof(int64_t));
  if (!r.nodes.empty()) {
    memcpy(nodes, r.nodes.data(), r.nodes.size() * sizeof(uint64_t));
    memcpy(node_edge, r.node_edge.data(), r.node_edge.size() * sizeof(uint64_t));
  }
  if (!r.edges.empty()) {
    memcpy(edges, r.edges.data(), r.edges.size() * sizeof(uint64_t));
    memcpy(mults, r.mults.data(), r.mults.size() * sizeof(uint64_t));
  }
}

void dgo_dag_free(dgo_dag* d) { delete d; }

int dgo_compare(const dgo_graph* a, const dgo_graph* b, const int64_t* locs, int64_t n, int nthreads,
                uint8_t* status) {
  try {
    check_signature(a->g, b->g);
    require_narrow_ids(a->g);
    parallel_blocks(n, nthreads, [&](int64_t lo, int64_t hi, int) {
      for (int64_t i = lo; i < hi; ++i)
        status[i] = compare_rows(narrow(enumerate_one(a->g, locs[i])), narrow(enumerate_one(b->g, locs[i])));
    });
    return 0;
  } catch (const std::exception& e) {
    g_err = e.what();
    return -1;
  }
}

// MERGE of two programs (trim = 0: inputs matched, no op trimmed): the two
// dgir texts, NUL-separated, into
// out (up to cap bytes); returns the bytes needed, or -1 on error.  *trimmed
// receives the number of prefix ops.
int64_t dgo_merge(const dgo_graph* a, const dgo_graph* b, int trim, char* out, int64_t cap, int* trimmed) {
  try {
    Merged m = merge_programs(a->g, b->g, trim != 0);
    std::string s = m.a + std::string(1, '\0') + m.b;
    if ((int64_t)s.size() <= cap) memcpy(out, s.data(), s.size());
    *trimmed = m.trimmed;
    return (int64_t)s.size();
  } catch (const std::exception& e) {
    g_err = e.what();
    return -1;
  }
}

// Ranked prefix of the location order: up to cap locations into out;
// returns the full count, or -1 on error.
int64_t dgo_order_prefix(const dgo_graph* g, int64_t threads, int64_t warp, int64_t* out, int64_t cap) {
  try {
    std::vector<int64_t> p = order_prefix(g->g, threads, warp);
    for (size_t i = 0; i < p.size() && (int64_t)i < cap; ++i) out[i] = p[i];
    return (int64_t)p.size();
  } catch (const std::exception& e) {
    g_err = e.what();
    return -1;
  }
}

// Positions first .. first + count - 1 of the keyed permutation of [0, n).
void dgo_permutation(int64_t n, uint64_t seed, int64_t first, int64_t count, int64_t* out) {
  Permutation p(n, seed);
  for (int64_t i = 0; i < count; ++i) out[i] = p.at(first + i);
}

// The Feistel network alone (no cycle walking) on the 2h-bit domain of n:
// forward (dir = 0) or inverse (dir = 1) images of x[0..count).
void dgo_feistel(int64_t n, uint64_t seed, int dir, const uint64_t* x, int64_t count, uint64_t* out) {
  Permutation p(n, seed);
  for (int64_t i = 0; i < count; ++i) out[i] = dir ? p.decrypt(x[i]) : p.encrypt(x[i]);
}

// First `count` outputs of SplitMix64 for `seed`.
void dgo_splitmix(uint64_t seed, int64_t count, uint64_t* out) {
  uint64_t state = seed;
  for (int64_t i = 0; i < count; ++i) {
    state += 0x9E3779B97F4A7C15ull;
    out[i] = splitmix_mix(state);
  }
}

// R_k(l) of the op producing tensor t, at location loc: up to `cap` triples
// (tensor index, flat index, multiplicity).  Returns the number of triples
// (which may exceed cap), or -1 on error.
int64_t dgo_reads(const dgo_graph* g, int t, int64_t loc, int32_t* tensors, int64_t* idx, uint64_t* mult,
                  int64_t cap) {
  try {
    const Graph& G = g->g;
    int k = -1;
    for (size_t i = 0; i < G.ops.size(); ++i) if (G.ops[i].out == t) k = (int)i;
    if (k < 0) throw Error("tensor is a leaf");
    if (loc < 0 || loc >= numel_of(G.tensors[t].shape)) throw Error("location out of range");
    int64_t n = 0;
    op_reads(G, G.ops[k], loc, [&](int tt, int64_t ii, uint64_t m) {
      if (n < cap) { tensors[n] = tt; idx[n] = ii; mult[n] = m; }
      ++n;
    });
    return n;
  } catch (const std::exception& e) {
    g_err = e.what();
    return -1;
  }
}

}  // extern "C"
