// Expression-DAG program: the contract between the host compiler (dag.cpp)
// and the DAG block code (dag_core.h).  Plain data, copied to the device as
// is.
#pragma once
#include <stdint.h>

#include "program.h"

// ---------------------------------------------------------------------------
// Expression-DAG program: the ops of a graph as read groups, for emitting
// the DAG of res(y[l]) (Sec. 3.4, "Back-projection") one location at a time.
// Every non-leaf element of the cone of y[l] is a node; its edges are the
// element references of its per-element equation in the equation's order:
// groups in order, window points in row-major order, a group's operands in
// order at each point (a point whose operand indices are not all valid reads
// nothing).  Element ids: leaves keep their global ids, op outputs follow in
// SSA order (gid of element 0 below).
// ---------------------------------------------------------------------------
#define DGD_MAX_WIN 8       // window variables of one group
#define DGD_MAX_OPERANDS 8  // operands of one group
#define DGD_MAX_PAIRS 64    // (operand, dim) index functions of one group

// A block emits a location's DAG op by op.  Per op, every node's edge count
// is taken first (an exclusive scan gives the nodes' first edges), then the
// edges are written.  Ops whose groups have no window ("pointwise") give
// one thread a node.  The others take their nodes in batches of one wave's
// width, one node per lane, and each group in one of two ways:
//   by progressions (fast == 1): every index function of the group uses at
//     most one window variable, with a unit divisor and no floor division,
//     and each variable has at most one exact division among its
//     functions.  The valid values of each variable are then an arithmetic
//     progression fixed by the node alone, the valid points are the
//     product of the progressions, and each operand's element index is
//     linear in the progression indices (steps computed here).  Each lane
//     sets up its node, then the wave writes the batch's points flattened
//     across its lanes.
//   point by point (fast == 0): one node at a time, every point of the
//     window box is evaluated and the valid ones are compacted within the
//     wave.

struct DgdTensor {
  int32_t rank;
  int32_t leaf;    // 1: a leaf (a variable; never expanded)
  int32_t cap;     // frontier capacity in entries (0 when never reached)
  int32_t lds;     // byte offset of the frontier in the location's LDS area
  uint32_t gid;    // global id of element 0
  int32_t numel;
  int32_t shape[DGP_MAX_RANK];
  uint32_t stride[DGP_MAX_RANK];  // row-major element strides
  uint64_t magic[DGP_MAX_RANK];   // floor(2^64 / shape) + 1 (0 for a unit dim): quotient by multiply-high
};

struct DgdOperand {
  int32_t tensor;
  uint32_t mult;
  DgpIFn idx[DGP_MAX_RANK];  // variables: output coordinates, then window coordinates
};

// One index function of a fast group: operand a, dim d, its window
// variable q (-1: none), and whether it can bind: 0 when the compiler has
// shown that it lies in range at every node and window point of the group
// (then it only enters the element indices, never the progressions or the
// validity of a node).
// (32-bit fields: the scalar unit loads dwords, and a narrower field
// would be read by a vector load, which waits for the wave's stores.)
// `stride` is the element stride of dim d of operand a's tensor.
struct DgdPair {
  int32_t a, d, q, bind;
  uint32_t stride;
  int32_t pad[3];
};

struct DgdGroup {
  int32_t nwin;
  int32_t nop;
  int32_t op0;     // first operand in the operand array
  int32_t fast;    // 1: by progressions (see above)
  int32_t wlo[DGD_MAX_WIN];
  int32_t whi[DGD_MAX_WIN];
  int64_t points;  // window points (1 without a window, 0 for an empty window)
  // Fast groups.
  int32_t npair;
  int32_t steps24;  // 1: every astep below, read as a signed value, lies in [-2^23, 2^23)
  DgdPair pair[DGD_MAX_PAIRS];
  // Per window variable: the step of its progression, and for a variable
  // with an exact division (v = (c0 + k w) / s), that pair and the inverse
  // of k / g modulo s / g (g = gcd(k, s)).
  int32_t step[DGD_MAX_WIN];
  int32_t mpair[DGD_MAX_WIN];
  int32_t minv[DGD_MAX_WIN];
  int32_t nbind;  // the pairs that can bind come first: pair[0 .. nbind)
  // Step of each operand's element index per progression step of each
  // variable (mod 2^32).
  uint32_t astep[DGD_MAX_OPERANDS][DGD_MAX_WIN];
};

struct DgdOp {
  int32_t out;     // tensor written
  int32_t g0, ng;  // read groups
  int32_t pointwise;  // 1: no group has a window (one thread per node)
  int64_t refs;    // element references of one node when every point is valid
  int32_t nonleaf;    // 1: some operand is not a leaf (its elements become nodes)
  int32_t pad;
};

struct DgdHeader {
  uint32_t magic;
  int32_t ntensor, nop, ngroup, noperand;
  int32_t tensor_off, op_off, group_off, operand_off;  // byte offsets in the blob
  int32_t blob_bytes;
  int32_t output;     // output tensor
  int32_t count_off;  // byte offset of the per-tensor frontier counters in the LDS area
  int32_t vars_off;   // byte offset of the per-thread variable tables (max_vars words per thread)
  int32_t max_vars;   // output plus window variables of the largest group
  int32_t lds_bytes;  // LDS area of one location
  int32_t ncount_off; // byte offset of the edge counts (ncount_cap words)
  int32_t ncount_cap; // per node of a pointwise op, per wave-wide batch of nodes otherwise
  int32_t slot_off;   // byte offset of the per-thread node slots (slot_words words per thread)
  int32_t slot_words; // 2 per window variable, 1 per operand, 2 more (see core.h)
  int32_t wave_off;   // byte offset of the per-wave prefix arrays (one word per lane)
  int32_t max_win;    // window variables and operands of the largest fast group
  int32_t max_opnd;
  int64_t out_numel;
};

#define DGD_MAGIC 0x44474433u  // "DGD3"
