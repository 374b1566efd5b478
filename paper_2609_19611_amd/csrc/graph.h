// Graph IR of the library: dgir parsing, shape inference, and lowering of
// every op to read groups (the dataflow skeleton of its per-element
// equation, Sec. 3.4 "Per-element equations").
#pragma once
#include <cstdint>
#include <map>
#include <stdexcept>
#include <string>
#include <vector>

namespace dg {

// Error carrying one of the DG_E_* status codes.
struct Failure : std::runtime_error {
  int code;
  Failure(int c, const std::string& m) : std::runtime_error(m), code(c) {}
};

typedef std::vector<int64_t> Dims;

// Index function over a group's variables (output coordinates 0..R-1,
// then window coordinates R..R+Q-1):
//   v = outer(sum coef * floor(var / vdiv) + c), outer in {none, exact /s, floor /s}.
struct IndexFn {
  struct Term {
    int var;
    int64_t coef;
    int64_t vdiv;
  };
  std::vector<Term> terms;
  int64_t c = 0;
  int mode = 0;
  int64_t s = 1;

  static IndexFn var(int v, int64_t coef = 1) {
    IndexFn f;
    f.terms.push_back({v, coef, 1});
    return f;
  }
  static IndexFn constant(int64_t c) {
    IndexFn f;
    f.c = c;
    return f;
  }
  IndexFn& plus(int v, int64_t coef, int64_t vdiv = 1) {
    terms.push_back({v, coef, vdiv});
    return *this;
  }
  IndexFn& offset(int64_t k) {
    c += k;
    return *this;
  }
};

struct Operand {
  int tensor;
  uint64_t mult;
  std::vector<IndexFn> idx;  // one per dim of the operand
};

// One read group: every window point w in the box [wlo, whi) (together with
// the output coordinates) reads each operand once per multiplicity, provided
// every operand index of that point is valid.  `guards` are further index
// functions that must be valid (value in [0, size)) for a point to read;
// lowering never writes them, the plan compiler's view of merged dims does
// (one per merged dim, see compile.cpp).
struct ReadGroup {
  Dims wlo, whi;
  std::vector<Operand> ops;
  std::vector<std::pair<IndexFn, int64_t>> guards;
};

struct Tensor {
  std::string name;
  Dims shape;
  int producer = -1;   // op index, -1 for a leaf
  int leaf = -1;       // leaf index, -1 for an op output
  uint64_t base = 0;   // global id of element 0 (leaves)
};

struct OpNode {
  std::string kind;
  std::vector<int> in;
  int out = -1;
  std::map<std::string, Dims> ints;
  std::map<std::string, std::vector<std::string>> exprs;  // affine_gather idxN
  std::vector<ReadGroup> groups;                           // filled by lowering
};

struct GraphIR {
  std::vector<Tensor> tensors;
  std::vector<OpNode> ops;
  std::vector<int> leaves;
  int output = -1;
  uint64_t leaf_total = 0;
};

int64_t numel(const Dims& d);

// Parses dgir v1 text, infers shapes and lowers every op.
GraphIR parse_dgir(const std::string& text);

// Adds one op (used by the parser and by descriptor-based construction).
void add_leaf(GraphIR& g, const std::string& name, const Dims& shape);
void add_op(GraphIR& g, const std::string& name, const std::string& kind, const std::vector<int>& in,
            const std::string& attrs);
void set_output(GraphIR& g, int tensor, const Dims* declared);
void finish(GraphIR& g);

}  // namespace dg
