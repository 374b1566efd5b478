// dgir parsing, shape inference and lowering to read groups.
//
// Every op is lowered to the multiset of element references of its
// per-element equation (Sec. 3.4 "Per-element equations"), written as read
// groups: a window box plus, per operand, one index function per operand
// dimension.  The readings follow the Torch lowerings of Sec. 3.3 with every
// tensor element a variable; they are restated at each case below.
#include "graph.h"

#include <algorithm>
#include <map>
#include <cctype>
#include <set>
#include <sstream>

#include "../../include/dirigo_rocm.h"

namespace dg {

// Element count of a shape.  Every tensor of a graph, leaf or op result,
// holds at most 2^62 elements, so a larger product (or one that would
// overflow 64 bits) is an error rather than a wrapped count.
int64_t numel(const Dims& d) {
  int64_t n = 1;
  for (int64_t x : d) {
    if (x < 0 || __builtin_mul_overflow(n, x, &n) || n > (int64_t(1) << 62))
      throw Failure(DG_E_OVERFLOW, "tensor element count exceeds 2^62");
  }
  return n;
}

namespace {

[[noreturn]] void fail(int code, const std::string& m) { throw Failure(code, m); }

const std::set<std::string>& unary_kinds() {
  static const std::set<std::string> s = {
      "relu", "gelu", "gelu_tanh", "hardtanh", "clamp", "sigmoid", "tanh", "exp", "log",
      "log1p", "square", "sqrt", "rsqrt", "neg", "abs", "identity", "contiguous", "silu",
      "softplus", "erf", "scale", "leaky_relu", "elu", "reciprocal"};
  return s;
}
const std::set<std::string>& binary_kinds() {
  static const std::set<std::string> s = {"add", "sub", "mul", "div", "maximum", "minimum", "pow"};
  return s;
}
const std::set<std::string>& reduce_kinds() {
  static const std::set<std::string> s = {"sum", "mean", "amax", "amin", "prod", "max", "min"};
  return s;
}

Dims ints_of(const std::string& s, const std::string& what) {
  Dims v;
  size_t i = 0;
  if (s.empty()) fail(DG_E_PARSE, what + ": empty list");
  while (i <= s.size()) {
    size_t j = s.find(',', i);
    if (j == std::string::npos) j = s.size();
    std::string tok = s.substr(i, j - i);
    if (tok.empty()) fail(DG_E_PARSE, what + ": empty item in '" + s + "'");
    size_t k = (tok[0] == '-' || tok[0] == '+') ? 1 : 0;
    if (k == tok.size()) fail(DG_E_PARSE, what + ": bad integer '" + tok + "'");
    for (size_t q = k; q < tok.size(); ++q)
      if (!isdigit((unsigned char)tok[q])) fail(DG_E_PARSE, what + ": bad integer '" + tok + "'");
    if (tok.size() > 18) fail(DG_E_PARSE, what + ": integer too large");
    v.push_back(std::stoll(tok));
    i = j + 1;
  }
  return v;
}

bool name_ok(const std::string& n) {
  if (n.empty() || !(isalpha((unsigned char)n[0]) || n[0] == '_')) return false;
  for (char c : n)
    if (!(isalnum((unsigned char)c) || c == '_')) return false;
  return n.size() < DG_NAME_LEN;
}

// ---- attribute access -----------------------------------------------------
const Dims* find_attr(const OpNode& op, const char* k) {
  auto it = op.ints.find(k);
  return it == op.ints.end() ? nullptr : &it->second;
}

Dims attr_list(const OpNode& op, const char* k, size_t n, int64_t dflt) {
  const Dims* v = find_attr(op, k);
  if (!v) return Dims(n, dflt);
  if (v->size() != n) fail(DG_E_SHAPE, op.kind + ": '" + k + "' needs " + std::to_string(n) + " values");
  return *v;
}

Dims attr_required(const OpNode& op, const char* k) {
  const Dims* v = find_attr(op, k);
  if (!v) fail(DG_E_SHAPE, op.kind + ": missing '" + k + "'");
  return *v;
}

int64_t attr_int(const OpNode& op, const char* k, int64_t dflt, bool required = false) {
  const Dims* v = find_attr(op, k);
  if (!v) {
    if (required) fail(DG_E_SHAPE, op.kind + ": missing '" + k + "'");
    return dflt;
  }
  if (v->size() != 1) fail(DG_E_SHAPE, op.kind + ": '" + k + "' must be a single integer");
  return (*v)[0];
}

int axis(int64_t d, size_t rank, const std::string& who) {
  int64_t r = (int64_t)rank;
  if (d < -r || d >= r) fail(DG_E_SHAPE, who + ": dimension out of range");
  return (int)(d < 0 ? d + r : d);
}

Dims bcast(const Dims& a, const Dims& b, const std::string& who) {
  size_t r = std::max(a.size(), b.size());
  Dims out(r);
  for (size_t i = 0; i < r; ++i) {
    int64_t x = i + a.size() >= r ? a[i + a.size() - r] : 1;
    int64_t y = i + b.size() >= r ? b[i + b.size() - r] : 1;
    if (x != y && x != 1 && y != 1) fail(DG_E_SHAPE, who + ": shapes do not broadcast");
    out[i] = std::max(x, y);
  }
  return out;
}

// Index functions reading an operand of shape `s` broadcast into an output of
// rank R (right-aligned; size-1 operand dims read coordinate 0).
std::vector<IndexFn> bcast_index(const Dims& s, const Dims& out) {
  std::vector<IndexFn> f;
  size_t off = out.size() - s.size();
  for (size_t d = 0; d < s.size(); ++d)
    f.push_back(s[d] == 1 ? IndexFn::constant(0) : IndexFn::var((int)(d + off)));
  return f;
}

std::vector<IndexFn> identity_index(size_t rank) {
  std::vector<IndexFn> f;
  for (size_t d = 0; d < rank; ++d) f.push_back(IndexFn::var((int)d));
  return f;
}

ReadGroup group_no_window() { return ReadGroup(); }

ReadGroup group_window(const Dims& ext) {
  ReadGroup g;
  g.wlo.assign(ext.size(), 0);
  g.whi = ext;
  return g;
}

// ---- affine_gather expressions ---------------------------------------------
IndexFn parse_gather_expr(const std::string& src, int R, int Q) {
  std::string s = src;
  IndexFn f;
  if (!s.empty() && s[0] == '(') {
    size_t close = s.rfind(')');
    if (close == std::string::npos) fail(DG_E_PARSE, "affine_gather: unbalanced '(' in '" + src + "'");
    std::string tail = s.substr(close + 1);
    if (tail.compare(0, 2, "//") == 0) {
      f.mode = 2;
      tail = tail.substr(2);
    } else if (tail.compare(0, 1, "/") == 0) {
      f.mode = 1;
      tail = tail.substr(1);
    } else {
      fail(DG_E_PARSE, "affine_gather: expected '/' or '//' in '" + src + "'");
    }
    Dims dv = ints_of(tail, "affine_gather divisor");
    if (dv.size() != 1 || dv[0] <= 0) fail(DG_E_PARSE, "affine_gather: divisor must be a positive integer");
    f.s = dv[0];
    s = s.substr(1, close - 1);
  }
  if (s.empty()) fail(DG_E_PARSE, "affine_gather: empty expression");
  size_t i = 0;
  while (i < s.size()) {
    int64_t sign = 1;
    if (s[i] == '+' || s[i] == '-') {
      sign = s[i] == '-' ? -1 : 1;
      ++i;
    }
    size_t j = i;
    while (j < s.size() && s[j] != '+' && s[j] != '-') ++j;
    std::string tok = s.substr(i, j - i);
    i = j;
    if (tok.empty()) fail(DG_E_PARSE, "affine_gather: bad expression '" + src + "'");
    int64_t coef = 1;
    size_t star = tok.find('*');
    std::string v = tok;
    if (star != std::string::npos) {
      Dims c = ints_of(tok.substr(0, star), "affine_gather coefficient");
      coef = c[0];
      v = tok.substr(star + 1);
    }
    if (!v.empty() && (v[0] == 'o' || v[0] == 'w')) {
      Dims k = ints_of(v.substr(1), "affine_gather variable");
      int lim = v[0] == 'o' ? R : Q;
      if (k[0] < 0 || k[0] >= lim) fail(DG_E_SHAPE, "affine_gather: variable '" + v + "' out of range");
      int var = v[0] == 'o' ? (int)k[0] : R + (int)k[0];
      if (coef != 0) f.terms.push_back({var, sign * coef, 1});
    } else {
      if (star != std::string::npos) fail(DG_E_PARSE, "affine_gather: bad term '" + tok + "'");
      f.c += sign * ints_of(v, "affine_gather constant")[0];
    }
  }
  return f;
}

// Splits the row-major flat range [lo, hi) of a box with extents `ext` into
// disjoint sub-boxes (each given as [blo, bhi) per dim).
void split_flat_range(const Dims& ext, size_t d, Dims blo, Dims bhi, int64_t lo, int64_t hi,
                      std::vector<std::pair<Dims, Dims>>& out) {
  if (lo >= hi) return;
  if (d == ext.size()) {
    out.push_back({blo, bhi});
    return;
  }
  int64_t inner = 1;
  for (size_t j = d + 1; j < ext.size(); ++j) inner *= ext[j];
  int64_t first = lo / inner, last = (hi - 1) / inner;
  auto with = [&](int64_t a, int64_t b) {
    Dims l = blo, h = bhi;
    l.push_back(a);
    h.push_back(b);
    return std::make_pair(l, h);
  };
  if (first == last) {
    auto p = with(first, first + 1);
    split_flat_range(ext, d + 1, p.first, p.second, lo - first * inner, hi - first * inner, out);
    return;
  }
  int64_t full_lo = first, full_hi = last + 1;
  if (lo % inner != 0) {
    auto p = with(first, first + 1);
    split_flat_range(ext, d + 1, p.first, p.second, lo - first * inner, inner, out);
    full_lo = first + 1;
  }
  bool tail = hi % inner != 0;
  if (tail) full_hi = last;
  if (full_lo < full_hi) {
    auto p = with(full_lo, full_hi);
    for (size_t j = d + 1; j < ext.size(); ++j) {
      p.first.push_back(0);
      p.second.push_back(ext[j]);
    }
    out.push_back(p);
  }
  if (tail) {
    auto p = with(last, last + 1);
    split_flat_range(ext, d + 1, p.first, p.second, 0, hi - last * inner, out);
  }
}

// ---- shape inference + lowering, one function per op family -----------------
struct Ctx {
  GraphIR& g;
  OpNode& op;
  const Dims& S(int i) const { return g.tensors[op.in[i]].shape; }
  int T(int i) const { return op.in[i]; }
};

void need(const OpNode& op, size_t lo, size_t hi) {
  if (op.in.size() < lo || op.in.size() > hi) fail(DG_E_SHAPE, op.kind + ": wrong number of operands");
}

Dims lower_op(Ctx c) {
  OpNode& op = c.op;
  const std::string& k = op.kind;
  std::vector<ReadGroup>& G = op.groups;

  if (unary_kinds().count(k)) {
    // An activation or other unary op is one uninterpreted function of its
    // operand: x[l] once.
    need(op, 1, 1);
    ReadGroup g = group_no_window();
    g.ops.push_back({c.T(0), 1, identity_index(c.S(0).size())});
    G.push_back(g);
    return c.S(0);
  }
  if (binary_kinds().count(k)) {
    // Each operand once at its broadcast index; a select (maximum, minimum)
    // reads each operand once as well.
    need(op, 2, 2);
    Dims out = bcast(c.S(0), c.S(1), k);
    ReadGroup g = group_no_window();
    g.ops.push_back({c.T(0), 1, bcast_index(c.S(0), out)});
    g.ops.push_back({c.T(1), 1, bcast_index(c.S(1), out)});
    G.push_back(g);
    return out;
  }
  if (k == "matmul") {
    // out[.., i, j] = sum_k A[.., i, k] B[.., k, j]: every k reads one A and
    // one B element.
    need(op, 2, 2);
    const Dims &a = c.S(0), &b = c.S(1);
    if (a.size() < 2 || b.size() < 2) fail(DG_E_SHAPE, "matmul: operands need rank >= 2");
    if (a.back() != b[b.size() - 2]) fail(DG_E_SHAPE, "matmul: inner dimensions differ");
    Dims out = bcast(Dims(a.begin(), a.end() - 2), Dims(b.begin(), b.end() - 2), k);
    out.push_back(a[a.size() - 2]);
    out.push_back(b.back());
    int R = (int)out.size();
    Dims batch(out.begin(), out.end() - 2);
    ReadGroup g = group_window({a.back()});
    auto side = [&](const Dims& s, bool left) {
      Dims sb(s.begin(), s.end() - 2);
      std::vector<IndexFn> f = bcast_index(sb, batch);
      if (left) {
        f.push_back(IndexFn::var(R - 2));
        f.push_back(IndexFn::var(R));
      } else {
        f.push_back(IndexFn::var(R));
        f.push_back(IndexFn::var(R - 1));
      }
      return f;
    };
    g.ops.push_back({c.T(0), 1, side(a, true)});
    g.ops.push_back({c.T(1), 1, side(b, false)});
    G.push_back(g);
    return out;
  }
  if (k == "linear") {
    // y[.., j] = sum_k x[.., k] W[j, k] + b[j].
    need(op, 2, 3);
    const Dims &x = c.S(0), &w = c.S(1);
    if (x.empty() || w.size() != 2 || x.back() != w[1]) fail(DG_E_SHAPE, "linear: bad shapes");
    Dims out = x;
    out.back() = w[0];
    int R = (int)out.size();
    ReadGroup g = group_window({w[1]});
    std::vector<IndexFn> fx;
    for (int d = 0; d < R - 1; ++d) fx.push_back(IndexFn::var(d));
    fx.push_back(IndexFn::var(R));
    g.ops.push_back({c.T(0), 1, fx});
    g.ops.push_back({c.T(1), 1, {IndexFn::var(R - 1), IndexFn::var(R)}});
    G.push_back(g);
    if (op.in.size() == 3) {
      if (c.S(2) != Dims{w[0]}) fail(DG_E_SHAPE, "linear: bias must be [out]");
      ReadGroup gb = group_no_window();
      gb.ops.push_back({c.T(2), 1, {IndexFn::var(R - 1)}});
      G.push_back(gb);
    }
    return out;
  }
  if (k == "conv" || k == "conv1d" || k == "conv2d" || k == "conv3d" || k == "conv_transpose" ||
      k == "conv_transpose1d" || k == "conv_transpose2d" || k == "conv_transpose3d") {
    bool tr = k.compare(0, 14, "conv_transpose") == 0;
    need(op, 2, 3);
    const Dims &x = c.S(0), &w = c.S(1);
    if (x.size() < 3 || w.size() != x.size()) fail(DG_E_SHAPE, k + ": x and W need equal rank >= 3");
    size_t nsp = x.size() - 2;
    if (k.back() >= '1' && k.back() <= '3' && (size_t)(k.back() - '0') != nsp)
      fail(DG_E_SHAPE, k + ": spatial rank differs from the op name");
    Dims st = attr_list(op, "stride", nsp, 1), pd = attr_list(op, "pad", nsp, 0);
    Dims dl = attr_list(op, "dilation", nsp, 1), opd = attr_list(op, "output_padding", nsp, 0);
    int64_t groups = attr_int(op, "groups", 1);
    for (size_t d = 0; d < nsp; ++d)
      if (st[d] <= 0 || dl[d] <= 0 || pd[d] < 0 || opd[d] < 0) fail(DG_E_SHAPE, k + ": bad stride/pad/dilation");
    if (groups <= 0) fail(DG_E_SHAPE, k + ": bad groups");
    Dims out(x.size());
    out[0] = x[0];
    int64_t cin_g, cout_g;
    if (!tr) {
      if (x[1] != w[1] * groups || w[0] % groups) fail(DG_E_SHAPE, k + ": channel mismatch");
      cin_g = w[1];
      cout_g = w[0] / groups;
      out[1] = w[0];
      for (size_t d = 0; d < nsp; ++d) {
        int64_t span = x[2 + d] + 2 * pd[d] - dl[d] * (w[2 + d] - 1) - 1;
        if (span < 0) fail(DG_E_SHAPE, k + ": empty output");
        out[2 + d] = span / st[d] + 1;
      }
    } else {
      if (x[1] != w[0] || w[0] % groups) fail(DG_E_SHAPE, k + ": channel mismatch");
      cin_g = w[0] / groups;
      cout_g = w[1];
      out[1] = w[1] * groups;
      for (size_t d = 0; d < nsp; ++d) {
        int64_t o = (x[2 + d] - 1) * st[d] - 2 * pd[d] + dl[d] * (w[2 + d] - 1) + opd[d] + 1;
        if (o <= 0) fail(DG_E_SHAPE, k + ": empty output");
        out[2 + d] = o;
      }
    }
    int R = (int)out.size();
    // Window: (input channel within the group, taps...), vars R, R+1+d.
    Dims win{cin_g};
    for (size_t d = 0; d < nsp; ++d) win.push_back(w[2 + d]);
    ReadGroup g = group_window(win);
    // Input channel: (co div cout_g) * cin_g + ci_l.
    IndexFn ci = IndexFn::var(R);
    if (groups > 1) ci.plus(1, cin_g, cout_g);
    std::vector<IndexFn> fx{IndexFn::var(0), ci}, fw;
    if (!tr) {
      // i = o*s - p + t*d, read only where i is inside x in every dim: a
      // padding tap multiplies a constant zero and reads neither x nor W.
      for (size_t d = 0; d < nsp; ++d) {
        IndexFn f = IndexFn::var(2 + (int)d, st[d]);
        f.plus(R + 1 + (int)d, dl[d]).offset(-pd[d]);
        fx.push_back(f);
      }
      fw = {IndexFn::var(1), IndexFn::var(R)};
    } else {
      // x[i] meets W[t] at output i*s - p + t*d, so output o reads the
      // (i, t) with i = (o + p - t*d) / s exactly and i inside x.
      for (size_t d = 0; d < nsp; ++d) {
        IndexFn f = IndexFn::var(2 + (int)d);
        f.plus(R + 1 + (int)d, -dl[d]).offset(pd[d]);
        f.mode = 1;
        f.s = st[d];
        fx.push_back(f);
      }
      IndexFn col = IndexFn::var(1);
      if (groups > 1) col.plus(1, -cout_g, cout_g);
      fw = {ci, col};
    }
    for (size_t d = 0; d < nsp; ++d) fw.push_back(IndexFn::var(R + 1 + (int)d));
    g.ops.push_back({c.T(0), 1, fx});
    g.ops.push_back({c.T(1), 1, fw});
    G.push_back(g);
    if (op.in.size() == 3) {
      if (c.S(2) != Dims{out[1]}) fail(DG_E_SHAPE, k + ": bias must be [C_out]");
      ReadGroup gb = group_no_window();
      gb.ops.push_back({c.T(2), 1, {IndexFn::var(1)}});
      G.push_back(gb);
    }
    return out;
  }
  if (k == "max_pool" || k == "avg_pool") {
    // Every in-range window element once; padding is never read.
    need(op, 1, 1);
    const Dims& x = c.S(0);
    Dims ks = attr_required(op, "kernel");
    size_t nsp = ks.size();
    if (nsp == 0 || x.size() < nsp) fail(DG_E_SHAPE, k + ": bad kernel rank");
    Dims st = find_attr(op, "stride") ? attr_list(op, "stride", nsp, 1) : ks;
    Dims pd = attr_list(op, "pad", nsp, 0), dl = attr_list(op, "dilation", nsp, 1);
    Dims out = x;
    size_t lead = x.size() - nsp;
    for (size_t d = 0; d < nsp; ++d) {
      if (ks[d] <= 0 || st[d] <= 0 || dl[d] <= 0 || pd[d] < 0) fail(DG_E_SHAPE, k + ": bad attributes");
      int64_t span = x[lead + d] + 2 * pd[d] - dl[d] * (ks[d] - 1) - 1;
      if (span < 0) fail(DG_E_SHAPE, k + ": empty output");
      out[lead + d] = span / st[d] + 1;
    }
    int R = (int)out.size();
    ReadGroup g = group_window(ks);
    std::vector<IndexFn> f;
    for (size_t d = 0; d < lead; ++d) f.push_back(IndexFn::var((int)d));
    for (size_t d = 0; d < nsp; ++d) {
      IndexFn e = IndexFn::var((int)(lead + d), st[d]);
      e.plus(R + (int)d, dl[d]).offset(-pd[d]);
      f.push_back(e);
    }
    g.ops.push_back({c.T(0), 1, f});
    G.push_back(g);
    return out;
  }
  if (reduce_kinds().count(k)) {
    // Every element of the reduced slice once.
    need(op, 1, 1);
    const Dims& x = c.S(0);
    Dims dims = attr_required(op, "dims");
    bool keep = attr_int(op, "keepdim", 0) != 0;
    std::vector<bool> red(x.size(), false);
    for (int64_t d : dims) red[axis(d, x.size(), k)] = true;
    Dims out, wext;
    std::vector<int> xvar(x.size());
    for (size_t d = 0; d < x.size(); ++d) {
      if (red[d]) {
        if (keep) out.push_back(1);
      } else {
        out.push_back(x[d]);
      }
    }
    bool scalar_out = out.empty();
    if (scalar_out) out.push_back(1);
    int R = (int)out.size();
    int oi = 0, wi = 0;
    std::vector<IndexFn> f;
    for (size_t d = 0; d < x.size(); ++d) {
      if (red[d]) {
        wext.push_back(x[d]);
        f.push_back(IndexFn::var(R + wi++));
        if (keep) ++oi;
      } else {
        f.push_back(IndexFn::var(oi++));
      }
    }
    ReadGroup g = group_window(wext);
    g.ops.push_back({c.T(0), 1, f});
    G.push_back(g);
    return out;
  }
  if (k == "softmax" || k == "log_softmax") {
    // exp(x[l]) / sum_D exp(x): the slice along D once, x[l] once more.
    need(op, 1, 1);
    const Dims& x = c.S(0);
    int D = axis(attr_int(op, "dim", 0, true), x.size(), k);
    int R = (int)x.size();
    ReadGroup g = group_window({x[D]});
    std::vector<IndexFn> f = identity_index(x.size());
    f[D] = IndexFn::var(R);
    g.ops.push_back({c.T(0), 1, f});
    G.push_back(g);
    ReadGroup g2 = group_no_window();
    g2.ops.push_back({c.T(0), 1, identity_index(x.size())});
    G.push_back(g2);
    return x;
  }
  if (k == "group_norm" || k == "batch_norm" || k == "layer_norm") {
    // mu = mean_S(x), d = x - mu, v = mean_S(square(d)), r = rsqrt(v + eps),
    // y = d * r * gamma + beta: x[s] for s in S reaches y[l] |S| + 2 times
    // (once through mu in d[l], |S| + 1 times through r), x[l] once more,
    // gamma and beta at l's channel once.
    if (op.in.size() != 1 && op.in.size() != 3) fail(DG_E_SHAPE, k + ": takes 1 or 3 operands");
    const Dims& x = c.S(0);
    int R = (int)x.size();
    Dims wext, aff_shape;
    std::vector<IndexFn> fx, faff;
    if (k == "group_norm") {
      if (x.size() < 2) fail(DG_E_SHAPE, k + ": needs [N, C, ...]");
      int64_t groups = attr_int(op, "groups", 0, true);
      if (groups <= 0 || x[1] % groups) fail(DG_E_SHAPE, "group_norm: groups must divide C");
      int64_t cg = x[1] / groups;
      wext.push_back(cg);
      fx.push_back(IndexFn::var(0));
      IndexFn ch = IndexFn::var(R);
      if (groups > 1) ch.plus(1, cg, cg);
      fx.push_back(ch);
      for (int d = 2; d < R; ++d) {
        wext.push_back(x[d]);
        fx.push_back(IndexFn::var(R + d - 1));
      }
      aff_shape = {x[1]};
      faff = {IndexFn::var(1)};
    } else if (k == "batch_norm") {
      if (x.size() < 2) fail(DG_E_SHAPE, k + ": needs [N, C, ...]");
      wext.push_back(x[0]);
      fx.push_back(IndexFn::var(R));
      fx.push_back(IndexFn::var(1));
      for (int d = 2; d < R; ++d) {
        wext.push_back(x[d]);
        fx.push_back(IndexFn::var(R + d - 1));
      }
      aff_shape = {x[1]};
      faff = {IndexFn::var(1)};
    } else {
      int64_t nd = attr_int(op, "ndims", 1);
      if (nd <= 0 || nd > R) fail(DG_E_SHAPE, "layer_norm: bad ndims");
      int lead = R - (int)nd;
      for (int d = 0; d < R; ++d) {
        if (d < lead) {
          fx.push_back(IndexFn::var(d));
        } else {
          wext.push_back(x[d]);
          fx.push_back(IndexFn::var(R + d - lead));
          aff_shape.push_back(x[d]);
          faff.push_back(IndexFn::var(d));
        }
      }
    }
    uint64_t S = (uint64_t)numel(wext);
    ReadGroup g = group_window(wext);
    g.ops.push_back({c.T(0), S + 2, fx});
    G.push_back(g);
    ReadGroup g2 = group_no_window();
    g2.ops.push_back({c.T(0), 1, identity_index(x.size())});
    G.push_back(g2);
    if (op.in.size() == 3) {
      if (c.S(1) != aff_shape || c.S(2) != aff_shape) fail(DG_E_SHAPE, k + ": bad affine parameter shapes");
      ReadGroup g3 = group_no_window();
      g3.ops.push_back({c.T(1), 1, faff});
      g3.ops.push_back({c.T(2), 1, faff});
      G.push_back(g3);
    }
    return x;
  }
  if (k == "channel_affine") {
    // x[l] * scale[c] + shift[c] with c the coordinate of dim 1.
    need(op, 3, 3);
    const Dims& x = c.S(0);
    if (x.size() < 2 || c.S(1) != Dims{x[1]} || c.S(2) != Dims{x[1]})
      fail(DG_E_SHAPE, "channel_affine: scale and shift must be [C]");
    ReadGroup g = group_no_window();
    g.ops.push_back({c.T(0), 1, identity_index(x.size())});
    g.ops.push_back({c.T(1), 1, {IndexFn::var(1)}});
    g.ops.push_back({c.T(2), 1, {IndexFn::var(1)}});
    G.push_back(g);
    return x;
  }
  if (k == "slice") {
    need(op, 1, 1);
    const Dims& x = c.S(0);
    int d = axis(attr_int(op, "dim", 0, true), x.size(), k);
    int64_t n = x[d];
    int64_t start = attr_int(op, "start", 0), end = attr_int(op, "end", n), step = attr_int(op, "step", 1);
    if (step <= 0) fail(DG_E_SHAPE, "slice: step must be positive");
    if (start < 0) start += n;
    if (end < 0) end += n;
    start = std::max<int64_t>(0, std::min(start, n));
    end = std::max<int64_t>(0, std::min(end, n));
    if (end <= start) fail(DG_E_SHAPE, "slice: empty result");
    Dims out = x;
    out[d] = (end - start + step - 1) / step;
    std::vector<IndexFn> f = identity_index(x.size());
    f[d] = IndexFn::var(d, step);
    f[d].offset(start);
    ReadGroup g = group_no_window();
    g.ops.push_back({c.T(0), 1, f});
    G.push_back(g);
    return out;
  }
  if (k == "permute") {
    need(op, 1, 1);
    const Dims& x = c.S(0);
    Dims p = attr_required(op, "dims");
    if (p.size() != x.size()) fail(DG_E_SHAPE, "permute: wrong number of dims");
    Dims out(x.size());
    std::vector<IndexFn> f(x.size());
    std::vector<bool> seen(x.size(), false);
    for (size_t q = 0; q < p.size(); ++q) {
      int d = axis(p[q], x.size(), k);
      if (seen[d]) fail(DG_E_SHAPE, "permute: repeated dim");
      seen[d] = true;
      out[q] = x[d];
      f[d] = IndexFn::var((int)q);
    }
    ReadGroup g = group_no_window();
    g.ops.push_back({c.T(0), 1, f});
    G.push_back(g);
    return out;
  }
  if (k == "reshape") {
    // y[o] reads x at the element with the same row-major flat index F.
    // Without unit dims, the dims of x and of y are two mixed-radix
    // factorisations of F; when their strides form one divisibility chain
    // they have a common refinement, and every digit of x is a sum of
    // pieces floor(o_j / a) mod b of single digits of y, which index
    // functions express (a mod is o - b * floor(o / b)).  Two factorisations
    // of one block with no common refinement ([6,4] and [4,6]) are refused.
    need(op, 1, 1);
    const Dims& x = c.S(0);
    Dims out = attr_required(op, "shape");
    for (int64_t v : out)
      if (v <= 0) fail(DG_E_SHAPE, "reshape: dims must be positive");
    if (numel(out) != numel(x)) fail(DG_E_SHAPE, "reshape: element count differs");
    std::vector<int> xo, oo;  // non-unit dims
    for (size_t d = 0; d < x.size(); ++d)
      if (x[d] != 1) xo.push_back((int)d);
    for (size_t d = 0; d < out.size(); ++d)
      if (out[d] != 1) oo.push_back((int)d);
    // Strides of the non-unit dims in the flat index.
    std::map<int, int64_t> xst, ost;
    int64_t st = 1;
    for (int i = (int)xo.size() - 1; i >= 0; --i) {
      xst[xo[i]] = st;
      st *= x[xo[i]];
    }
    st = 1;
    for (int j = (int)oo.size() - 1; j >= 0; --j) {
      ost[oo[j]] = st;
      st *= out[oo[j]];
    }
    const int64_t total = st;
    std::set<int64_t> bp{1, total};
    for (auto& e : xst) bp.insert(e.second);
    for (auto& e : ost) bp.insert(e.second);
    std::vector<int64_t> chain(bp.begin(), bp.end());
    for (size_t q = 1; q < chain.size(); ++q)
      if (chain[q] % chain[q - 1])
        fail(DG_E_UNSUPPORTED_OP, "reshape: the two shapes factor the flat index with no common refinement");
    std::vector<IndexFn> f(x.size(), IndexFn::constant(0));
    for (int d : xo) {
      const int64_t lo = xst[d], hi = xst[d] * x[d];
      IndexFn e;
      for (size_t q = 0; q + 1 < chain.size(); ++q) {
        const int64_t s0 = chain[q], s1 = chain[q + 1];
        if (s0 < lo || s1 > hi) continue;
        // Refined digit floor(F / s0) mod (s1 / s0), inside digit j of y.
        int j = -1;
        for (int jj : oo)
          if (ost[jj] <= s0 && s1 <= ost[jj] * out[jj]) j = jj;
        const int64_t a = s0 / ost[j], b = s1 / s0, w = s0 / lo;
        e.plus(j, w, a);
        if (s1 != ost[j] * out[j]) e.plus(j, -w * b, a * b);
      }
      // Combine terms of the same variable and divisor.
      IndexFn m;
      for (const auto& t : e.terms) {
        bool found = false;
        for (auto& u : m.terms)
          if (u.var == t.var && u.vdiv == t.vdiv) {
            u.coef += t.coef;
            found = true;
          }
        if (!found) m.terms.push_back(t);
      }
      f[d].terms.clear();
      for (const auto& t : m.terms)
        if (t.coef != 0) f[d].terms.push_back(t);
    }
    ReadGroup g = group_no_window();
    g.ops.push_back({c.T(0), 1, f});
    G.push_back(g);
    return out;
  }
  if (k == "expand") {
    need(op, 1, 1);
    const Dims& x = c.S(0);
    Dims out = attr_required(op, "shape");
    if (out.size() < x.size()) fail(DG_E_SHAPE, "expand: rank too small");
    for (size_t d = 0; d < x.size(); ++d) {
      int64_t od = out[out.size() - x.size() + d];
      if (od <= 0 || (x[d] != od && x[d] != 1)) fail(DG_E_SHAPE, "expand: incompatible shape");
    }
    ReadGroup g = group_no_window();
    g.ops.push_back({c.T(0), 1, bcast_index(x, out)});
    G.push_back(g);
    return out;
  }
  if (k == "affine_gather") {
    if (op.in.empty()) fail(DG_E_SHAPE, "affine_gather: needs operands");
    Dims out = attr_required(op, "shape");
    Dims win = find_attr(op, "window") ? *find_attr(op, "window") : Dims();
    for (int64_t v : out)
      if (v <= 0) fail(DG_E_SHAPE, "affine_gather: bad shape");
    for (int64_t v : win)
      if (v <= 0) fail(DG_E_SHAPE, "affine_gather: bad window");
    int R = (int)out.size(), Q = (int)win.size();
    int64_t wn = numel(win);
    Dims fl = find_attr(op, "flat") ? *find_attr(op, "flat") : Dims{0, wn};
    if (fl.size() != 2 || fl[0] < 0 || fl[1] > wn || fl[0] > fl[1]) fail(DG_E_SHAPE, "affine_gather: bad flat range");
    Dims mult = attr_list(op, "mult", op.in.size(), 1);
    for (int64_t m : mult)
      if (m <= 0) fail(DG_E_SHAPE, "affine_gather: multiplicities must be positive");
    std::vector<std::vector<IndexFn>> fs(op.in.size());
    for (size_t j = 0; j < op.in.size(); ++j) {
      auto it = op.exprs.find("idx" + std::to_string(j));
      if (it == op.exprs.end()) fail(DG_E_SHAPE, "affine_gather: missing idx" + std::to_string(j));
      if (it->second.size() != c.S((int)j).size())
        fail(DG_E_SHAPE, "affine_gather: idx" + std::to_string(j) + " must have one expression per operand dim");
      for (const std::string& e : it->second) fs[j].push_back(parse_gather_expr(e, R, Q));
    }
    std::vector<std::pair<Dims, Dims>> boxes;
    split_flat_range(win, 0, Dims(), Dims(), fl[0], fl[1], boxes);
    for (auto& b : boxes) {
      ReadGroup g;
      g.wlo = b.first;
      g.whi = b.second;
      for (size_t j = 0; j < op.in.size(); ++j) g.ops.push_back({c.T((int)j), (uint64_t)mult[j], fs[j]});
      G.push_back(g);
    }
    return out;
  }
  fail(DG_E_UNSUPPORTED_OP, "unsupported op kind '" + k + "'");
}

std::vector<std::string> words(const std::string& line) {
  std::vector<std::string> w;
  std::istringstream is(line);
  std::string t;
  while (is >> t) w.push_back(t);
  return w;
}

}  // namespace

void add_leaf(GraphIR& g, const std::string& name, const Dims& shape) {
  if (!name_ok(name)) fail(DG_E_PARSE, "bad tensor name '" + name + "'");
  for (auto& t : g.tensors)
    if (t.name == name) fail(DG_E_PARSE, "duplicate tensor name '" + name + "'");
  if (!g.ops.empty()) fail(DG_E_PARSE, "leaves must precede ops");
  if (shape.empty() || shape.size() > DG_MAX_RANK) fail(DG_E_SHAPE, "leaf '" + name + "': rank must be 1..8");
  for (int64_t d : shape)
    if (d <= 0 || d >= (int64_t(1) << 31)) fail(DG_E_SHAPE, "leaf '" + name + "': dims must be in [1, 2^31)");
  Tensor t;
  t.name = name;
  t.shape = shape;
  t.leaf = (int)g.leaves.size();
  t.base = g.leaf_total;
  g.leaf_total += (uint64_t)numel(shape);
  if (g.leaf_total > (1ull << 62)) fail(DG_E_OVERFLOW, "leaf elements exceed 2^62");
  g.leaves.push_back((int)g.tensors.size());
  g.tensors.push_back(t);
}

void add_op(GraphIR& g, const std::string& name, const std::string& kind, const std::vector<int>& in,
            const std::string& attrs) {
  if (!name_ok(name)) fail(DG_E_PARSE, "bad tensor name '" + name + "'");
  for (auto& t : g.tensors)
    if (t.name == name) fail(DG_E_PARSE, "duplicate tensor name '" + name + "'");
  OpNode op;
  op.kind = kind;
  op.in = in;
  for (int t : in)
    if (t < 0 || t >= (int)g.tensors.size()) fail(DG_E_INVALID_ARG, "operand index out of range");
  for (const std::string& kv : words(attrs)) {
    size_t eq = kv.find('=');
    if (eq == std::string::npos || eq == 0) fail(DG_E_PARSE, "expected key=value, got '" + kv + "'");
    std::string key = kv.substr(0, eq), val = kv.substr(eq + 1);
    if (kind == "affine_gather" && key.compare(0, 3, "idx") == 0) {
      std::vector<std::string> parts;
      size_t i = 0;
      while (true) {
        size_t j = val.find(',', i);
        parts.push_back(val.substr(i, j == std::string::npos ? std::string::npos : j - i));
        if (j == std::string::npos) break;
        i = j + 1;
      }
      op.exprs[key] = parts;
    } else {
      op.ints[key] = ints_of(val, kind + " attribute '" + key + "'");
    }
  }
  op.out = (int)g.tensors.size();
  g.ops.push_back(op);
  OpNode& ref = g.ops.back();
  Dims shape = lower_op(Ctx{g, ref});
  if (shape.size() > DG_MAX_RANK) fail(DG_E_SHAPE, kind + ": result rank above 8");
  for (int64_t d : shape)
    if (d >= (int64_t(1) << 31)) fail(DG_E_SHAPE, kind + ": result dim too large");
  numel(shape);  // a result of more than 2^62 elements is DG_E_OVERFLOW
  Tensor t;
  t.name = name;
  t.shape = shape;
  t.producer = (int)g.ops.size() - 1;
  g.tensors.push_back(t);
}

void set_output(GraphIR& g, int tensor, const Dims* declared) {
  if (tensor < 0 || tensor >= (int)g.tensors.size()) fail(DG_E_INVALID_ARG, "output tensor out of range");
  if (declared && *declared != g.tensors[tensor].shape)
    fail(DG_E_SHAPE, "output: declared shape differs from the inferred shape");
  g.output = tensor;
}

void finish(GraphIR& g) {
  if (g.output < 0) fail(DG_E_PARSE, "missing output");
  if (g.leaves.empty()) fail(DG_E_SHAPE, "graph has no leaves");
}

GraphIR parse_dgir(const std::string& text) {
  GraphIR g;
  std::istringstream is(text);
  std::string line;
  int lineno = 0;
  bool header = false;
  while (std::getline(is, line)) {
    ++lineno;
    size_t h = line.find('#');
    if (h != std::string::npos) line.resize(h);
    std::vector<std::string> w = words(line);
    if (w.empty()) continue;
    try {
      if (!header) {
        if (w.size() != 2 || w[0] != "dgir" || w[1] != "1") fail(DG_E_PARSE, "expected the 'dgir 1' header");
        header = true;
      } else if (g.output >= 0) {
        fail(DG_E_PARSE, "statement after 'output'");
      } else if (w[0] == "leaf") {
        if (w.size() != 3) fail(DG_E_PARSE, "expected 'leaf <name> <shape>'");
        add_leaf(g, w[1], ints_of(w[2], "leaf shape"));
      } else if (w[0] == "op") {
        if (w.size() < 4) fail(DG_E_PARSE, "expected 'op <name> <kind> <operands...>'");
        std::vector<int> in;
        size_t i = 3;
        for (; i < w.size() && w[i] != ";"; ++i) {
          int found = -1;
          for (size_t t = 0; t < g.tensors.size(); ++t)
            if (g.tensors[t].name == w[i]) found = (int)t;
          if (found < 0) fail(DG_E_PARSE, "unknown operand '" + w[i] + "'");
          in.push_back(found);
        }
        std::string attrs;
        for (size_t j = i + 1; j < w.size(); ++j) attrs += w[j] + " ";
        add_op(g, w[1], w[2], in, attrs);
      } else if (w[0] == "output") {
        if (w.size() != 3) fail(DG_E_PARSE, "expected 'output <name> <shape>'");
        int found = -1;
        for (size_t t = 0; t < g.tensors.size(); ++t)
          if (g.tensors[t].name == w[1]) found = (int)t;
        if (found < 0) fail(DG_E_PARSE, "unknown output tensor '" + w[1] + "'");
        Dims decl = ints_of(w[2], "output shape");
        set_output(g, found, &decl);
      } else {
        fail(DG_E_PARSE, "unknown statement '" + w[0] + "'");
      }
    } catch (const Failure& e) {
      throw Failure(e.code, "line " + std::to_string(lineno) + ": " + e.what());
    }
  }
  if (!header) fail(DG_E_PARSE, "missing 'dgir 1' header");
  finish(g);
  return g;
}

}  // namespace dg
