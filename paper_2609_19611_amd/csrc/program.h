// Compiled per-location plan: the contract between the host compiler
// (compile.cpp) and the device kernels (core.h, kernels.hip).
//
// A plan evaluates the back-projection of one output location (Sec. 3.4)
// in factored form.  The path-count function of every tensor reached from
// the location is kept as a short sum of separable terms,
//     count(i_0, ..., i_{r-1}) = coef * f_0(i_0) * ... * f_{r-1}(i_{r-1}),
// where each factor f_d is a small dense vector over a contiguous range of
// dimension d.  Substituting an op's per-element equation into a term
// splits the op's read variables (output coordinates and window
// coordinates) into independent components, one per dimension of the read
// operand plus scalar components; every component is summed over its own
// small box.  Instructions below compute those factors and scalars; the
// leaves' terms are then expanded into CSR rows.
//
// All structures are plain data so the blob can be copied to the device
// as is.
#pragma once
#include <stdint.h>

#define DGP_MAX_VARS 8    // variables of one component
#define DGP_MAX_PREDS 12  // validity predicates of one component
#define DGP_MAX_FTERMS 4  // terms of one index function
#define DGP_MAX_RANK 8
#define DGP_MAX_LEAF_TERMS 32

// Index function: v = outer(sum_i coef_i * floor(var_i / vdiv_i) + c),
// outer = identity (mode 0), exact division by s (mode 1: defined only when
// s divides), floor division by s (mode 2).  Valid when 0 <= v < size.
struct DgpIFn {
  int32_t nterm;
  int32_t var[DGP_MAX_FTERMS];
  int32_t coef[DGP_MAX_FTERMS];
  int32_t vdiv[DGP_MAX_FTERMS];
  int32_t c;
  int32_t mode;
  int32_t s;
  int32_t size;
};

enum DgpOpcode : int32_t {
  DGP_ROOT = 1,     // factor = delta at coordinate `a` of the location
  DGP_CONST = 2,    // factor = delta at constant coordinate `a`
  DGP_COMP = 3,     // component sum into a factor (target) or a scalar
  DGP_LINCOMB = 4,  // factor = k1 * f1 + k2 * f2
  DGP_SMUL = 5,     // scalar = cst * prod s[i]
  DGP_SADD = 6,     // scalar = k1 * s1 + k2 * s2
  DGP_PATTERN = 7,  // factor = a fixed pattern placed at the location (see DgpInstr.pat)
};

#define DGP_MAX_PAT 16  // entries of one pattern

struct DgpInstr {
  int32_t opcode;
  int32_t dst;            // factor slot or scalar slot
  int32_t dst_is_scalar;
  int32_t a;              // ROOT: output dim; CONST: coordinate
  // COMP
  int32_t nvar;
  int32_t var_src[DGP_MAX_VARS];  // factor slot of an output variable, -1 for a window variable
  int32_t wlo[DGP_MAX_VARS];      // window variable range [wlo, whi)
  int32_t whi[DGP_MAX_VARS];
  int32_t npred;
  DgpIFn pred[DGP_MAX_PREDS];
  DgpIFn target;
  // LINCOMB: factors f1, f2 scaled by k = (slot < 0 ? 1 : scalar[slot]) * c
  // SADD:    scalars s1 = f1, s2 = f2 with the same scaling
  int32_t f1, f2, k1, k2;
  uint64_t c1, c2;
  // SMUL
  int32_t ns;
  int32_t s[8];
  uint64_t cst;
  // PATTERN: r is the location's coordinate `a` (0 when a < 0); entry e is
  // pat[e] = {p, q, u, value} (value below 2^32):
  //   kind 0: coordinates [r + p, r + q) hold value (entries disjoint);
  //   kind 1: coordinate p holds value when q <= r < u (entries of one
  //           coordinate never hold at the same r).
  // Coordinates outside [0, size) are dropped.  The factor's range is
  // [r + pmin, r + pmax) (kind 0) or [pmin, pmax) (kind 1), clipped.
  int32_t pkind, npat, pmin, pmax;
  int32_t pat[DGP_MAX_PAT][4];
};

struct DgpFactor {
  int32_t cap;   // capacity (entries)
  int32_t off;   // offset of the values in the factor-value area (in uint64 units)
  int32_t size;  // extent of the tensor dimension the factor lives on
  int32_t stat;  // 1: used by a single-term leaf (its nonzero count and maximum are taken)
};

// One separable term of a leaf: coef = (coef_slot < 0 ? 1 : scalar) * coef_const.
struct DgpTerm {
  int32_t coef_slot;
  int32_t pad;
  uint64_t coef_const;
  int32_t factor[DGP_MAX_RANK];
};

struct DgpLeaf {
  int32_t rank;
  int32_t nterm;
  int32_t term0;      // first term in the term array
  int32_t split;      // dims [0, split) form the outer table, [split, rank) the inner
  uint64_t base;      // global id of element 0
  int32_t outer_cap;  // table capacities (entries)
  int32_t inner_cap;
  int32_t shape[DGP_MAX_RANK];
  uint64_t stride[DGP_MAX_RANK];
  int32_t ucap[DGP_MAX_RANK];  // capacity of the per-dim union of nonzero coordinates
};

struct DgpHeader {
  uint32_t magic;
  int32_t out_rank;
  int64_t out_numel;
  int64_t out_shape[DGP_MAX_RANK];
  int64_t out_stride[DGP_MAX_RANK];
  int32_t ninstr, nfactor, nscalar, nleaf, nterm;
  int32_t instr_off, factor_off, leaf_off, term_off;  // byte offsets in the blob
  int32_t fval_entries;  // total factor-value entries (uint64)
  int32_t blob_bytes;
  int32_t max_leaf_terms;
  int32_t emit_entries;  // table area (uint32 words) for the largest leaf
  int32_t union_entries; // union-list area (int32) for the largest leaf
  // Instructions are grouped into levels: a level only reads values written
  // by earlier levels, so the block synchronises once per phase of a level
  // instead of once per instruction.  level_off: byte offset of int32
  // level_start[nlevel + 1] (instruction index of each level's first
  // instruction).  A component sum over more than two variables runs in a
  // level of its own and keeps its variables in LDS (serial_vars: the
  // largest such variable count, 0 if none).
  int32_t nlevel;
  int32_t level_off;
  int32_t serial_vars;
  // 1 when the static bound on every path count is below 2^32: the
  // run-time overflow checks (factor and table maxima) are then skipped.
  int32_t no_overflow;
  // Factor values that leaf terms read come first in the value area:
  // fval_live entries.  The rest belong to intermediate tensors only and are
  // dead once the plan has run.
  int32_t fval_live;
};

#define DGP_MAGIC 0x44475031u  // "DGP1"

// Error bits raised by the kernels (reported after the sizes pass).
#define DGP_ERR_RANGE 1u      // location outside the output
#define DGP_ERR_OVERFLOW 2u   // a path count does not fit 32 bits
#define DGP_ERR_CAPACITY 4u   // a factor or union outgrew its static capacity
#define DGP_ERR_SIZE 8u       // fill found a row size different from the sizes pass
#define DGP_ERR_BUFFER 16u    // single pass: the rows do not fit the output buffers
#define DGP_ERR_TIMEOUT 32u   // single pass: a predecessor's row size never arrived
#define DGP_ERR_SHAPE 64u     // a specialised DAG kernel lacks the code for one of its program's groups
