// Expression DAGs of res(y[l]), written once for a block of cooperating
// threads (`C` supplies tid, nthreads, lanes and waves, barriers, wave-level
// ballots and scans, LDS atomics).  The device kernels (kernels.hip)
// instantiate it with a HIP block; the host emulation used by the CPU tests
// with a single thread.
#pragma once
#include <stdint.h>

#include "core.h"
#include "dag_program.h"

namespace dgc {

// ---------------------------------------------------------------------------
// Expression DAG of res(y[l]) for one location (dag_program.h, DgdHeader).
//
// Frontiers of the non-leaf tensors live in the LDS area: a consumer node
// appends every non-leaf element it references to the operand's candidate
// list; when the ops are walked back to that tensor's producer (reverse SSA
// order, so every consumer has been walked), the list is sorted and made
// unique, giving the tensor's nodes in ascending order.  A node's edges are
// its (group, window point, operand) references in order; a point whose
// operand indices are not all valid is skipped.
//
// Per op, every node's edge count is taken first and an exclusive scan over
// the nodes gives each node its first edge; the edges are then written at
// known positions.  Pointwise ops give one thread a node; the others give
// one wave a node and take each group per variable (the product of per-
// variable valid sets, no per-point test) or point by point (wave-level
// compaction), as the compiler decided.
// ---------------------------------------------------------------------------
enum : int { DAG_COUNT = 0, DAG_FILL = 1 };

// The ways of taking a group that a kernel carries code for.  The
// precompiled kernels carry every way; a kernel specialised for one program
// carries only the ways its groups use, which keeps the per-location code
// of a large program within the instruction cache.  A group whose way a
// kernel lacks stops the location with DGP_ERR_SHAPE (the host derives the
// masks from the same program, so this does not happen).
//   DG_DAG_FAST  register progressions of nop operands and nwin window
//                variables: bit (nop - 1) * 5 + nwin (nop 1..3, nwin 0..4)
//   DG_DAG_NODE  node-major emitters of the other progression groups: bit
//                (nop - 1) * 4 + nwin - 1 (nop 1..3, nwin 1..4)
//   DG_DAG_SLOW  progression groups without a register form
//   DG_DAG_BOX   point-by-point groups
//   DG_DAG_PW    pointwise ops
#ifndef DG_DAG_FAST
#define DG_DAG_FAST 0x7FFFu
#define DG_DAG_NODE 0xFFFu
#define DG_DAG_SLOW 1
#define DG_DAG_BOX 1
#define DG_DAG_PW 1
#endif
// A specialised kernel also defines DG_DAG_NOPS, its program's op count:
// the walk over the ops and each op's loops over its groups are then
// unrolled, so that every op and group field is a constant.
#ifdef DG_DAG_NOPS
#define DG_DAG_UNROLL _Pragma("unroll")
#else
#define DG_DAG_UNROLL
#endif

struct DagOut {
  uint32_t* nodes;      // node ids (global element ids)
  uint32_t* node_edge;  // first edge of each node, relative to the location's first edge
  uint32_t* edges;      // child ids
  uint32_t* mults;      // multiplicities
  uint64_t room_nodes, room_edges;
};

// Sorts the first n entries of f and keeps one of each value; returns the
// number kept.  Bitonic network whose comparators all put the smaller value
// at the lower index (each merge starts by comparing mirrored positions), so
// positions at or past n act as +infinity and their comparators are
// skipped: any n, sorted in place.  All threads call it.
template <class C>
DGC uint32_t sort_unique(C& c, uint32_t* f, uint32_t n) {
  const int tid = c.tid(), nt = c.nthreads();
  for (uint32_t k = 2; (k >> 1) < n; k <<= 1) {
    for (uint32_t j = k >> 1; j > 0; j >>= 1) {
      const uint32_t mask = j == (k >> 1) ? k - 1 : j;  // mirror within the block first
      for (uint32_t i = (uint32_t)tid; i < n; i += (uint32_t)nt) {
        const uint32_t l = i ^ mask;
        if (l > i && l < n) {
          const uint32_t a = f[i], b = f[l];
          if (a > b) {
            f[i] = b;
            f[l] = a;
          }
        }
      }
      c.sync();
    }
  }
  c.sync();
  uint32_t kept = 0;
  for (uint32_t b0 = 0; b0 < n; b0 += (uint32_t)nt) {
    const uint32_t i = b0 + (uint32_t)tid;
    uint32_t v = 0;
    bool keep = false;
    if (i < n) {
      v = f[i];
      keep = i == 0 || f[i - 1] != v;
    }
    uint32_t tot;
    const uint32_t pre = c.prefix(keep, &tot);
    if (keep) f[kept + pre] = v;
    kept += tot;
    c.sync();
  }
  return kept;
}

// Replaces a[0..n) by its exclusive running sums and returns the total.
// All threads call it; ends past a barrier.
template <class C>
DGC uint64_t block_scan(C& c, uint32_t* a, uint32_t n) {
  const uint32_t nt = (uint32_t)c.nthreads(), tid = (uint32_t)c.tid();
  const uint32_t per = (n + nt - 1) / nt;
  const uint32_t b = tid * per < n ? tid * per : n;
  const uint32_t e = b + per < n ? b + per : n;
  uint64_t s = 0;
  for (uint32_t j = b; j < e; ++j) s += a[j];
  uint64_t tot;
  uint64_t run = c.scan_add(s, &tot);
  for (uint32_t j = b; j < e; ++j) {
    const uint32_t v = a[j];
    a[j] = (uint32_t)run;
    run += v;
  }
  c.sync();
  return tot;
}

// Quotient of a 32-bit n by a tensor dim from its magic number m (0: the
// dim is 1): the high 64 bits of n * m, from two 32 x 32-bit products.
DGC uint32_t magic_div(uint32_t n, uint64_t m) {
  if (!m) return n;
  const uint64_t lo = (uint64_t)n * (uint32_t)m;
  const uint64_t hi = (uint64_t)n * (uint32_t)(m >> 32);
  return (uint32_t)((hi + (lo >> 32)) >> 32);
}

// n / d and n % d for n < 2^16 (digits of a lane index or the wave width).
DGC uint32_t small_divmod(uint32_t n, uint32_t d, uint32_t* r) {
#if defined(__HIP_DEVICE_COMPILE__)
  uint32_t q = (uint32_t)((float)n * __builtin_amdgcn_rcpf((float)d));
  int32_t rr = (int32_t)n - (int32_t)(q * d);
  if (rr < 0) {
    --q;
    rr += (int32_t)d;
  } else if (rr >= (int32_t)d) {
    ++q;
    rr -= (int32_t)d;
  }
  *r = (uint32_t)rr;
  return q;
#else
  *r = n % d;
  return n / d;
#endif
}

// Floor and ceiling of a / b for b > 0.
DGC int32_t floor_div(int32_t a, int32_t b) { return fdiv(a, b); }
DGC int32_t ceil_div(int32_t a, int32_t b) { return -fdiv(-a, b); }

DGC int32_t pmod(int32_t a, int32_t m) {
  if ((m & (m - 1)) == 0) return a & (m - 1);  // (a power of two: two's complement)
  const int32_t r = a % m;
  return r < 0 ? r + m : r;
}

// a / m for a >= 0 and m >= 1 (shift for a power of two).
DGC int32_t qpos(int32_t a, int32_t m) {
  if ((m & (m - 1)) == 0) return a >> __builtin_ctz((unsigned)m);
  return a / m;
}

// a / m for a multiple a of m >= 1 of either sign.
DGC int32_t qexact(int32_t a, int32_t m) {
  if ((m & (m - 1)) == 0) return a >> __builtin_ctz((unsigned)m);
  return a / m;
}

// Coordinates of element e of X in registers (row-major, last fastest).
DGC void elem_coords(const DgdTensor& X, uint32_t e, uint32_t* x) {
  DG_UNROLL
  for (int d = DGP_MAX_RANK - 1; d >= 0; --d) {
    x[d] = 0;
    if (d < X.rank) {
      const uint32_t q = magic_div(e, X.magic[d]);
      x[d] = e - q * (uint32_t)X.shape[d];
      e = q;
    }
  }
}

// The frontier F[0..n) of tensor X made sorted and unique through a bitmap
// over the bounding box of its candidates' coordinates: the box's cells in
// row-major order are in ascending element order, so the set cells, read
// word by word with a scan of the words' counts, are the sorted unique
// elements.  Applies when the box's bitmap and counts fit `ws` (LDS words
// free for the call); returns the number kept, or ~0u with F untouched.
// Called by all threads; ends past a barrier.
template <class C>
DGC uint32_t box_unique(C& c, const DgdTensor& X, uint32_t* F, uint32_t n, uint32_t* ws, uint32_t ws_words) {
  const int tid = c.tid(), nt = c.nthreads();
  const int R = X.rank;
  uint32_t* mn = ws;
  uint32_t* mx = ws + DGP_MAX_RANK;
  if (n < 2 || R < 1 || ws_words < 2 * DGP_MAX_RANK + 2) return ~0u;
  for (int d = tid; d < DGP_MAX_RANK; d += nt) {
    mn[d] = 0xFFFFFFFFu;
    mx[d] = 0;
  }
  c.sync();
  uint32_t lmn[DGP_MAX_RANK], lmx[DGP_MAX_RANK];
  DG_UNROLL
  for (int d = 0; d < DGP_MAX_RANK; ++d) {
    lmn[d] = 0xFFFFFFFFu;
    lmx[d] = 0;
  }
  for (uint32_t i = (uint32_t)tid; i < n; i += (uint32_t)nt) {
    uint32_t x[DGP_MAX_RANK];
    elem_coords(X, F[i], x);
    DG_UNROLL
    for (int d = 0; d < DGP_MAX_RANK; ++d) {
      lmn[d] = x[d] < lmn[d] ? x[d] : lmn[d];
      lmx[d] = x[d] > lmx[d] ? x[d] : lmx[d];
    }
  }
  DG_UNROLL
  for (int d = 0; d < DGP_MAX_RANK; ++d)
    if (d < R) {
      c.reduce_min32(&mn[d], lmn[d]);
      c.reduce_max32(&mx[d], lmx[d]);
    }
  c.sync();
  uint32_t lo[DGP_MAX_RANK], e[DGP_MAX_RANK];
  uint64_t V = 1;
  DG_UNROLL
  for (int d = 0; d < DGP_MAX_RANK; ++d) {
    lo[d] = d < R ? mn[d] : 0u;
    e[d] = d < R ? mx[d] - mn[d] + 1u : 1u;
    V *= e[d];
  }
  const uint64_t W = (V + 31) / 32;
  if (V > (1ull << 26) || 2 * DGP_MAX_RANK + 2 * W > (uint64_t)ws_words) {
    c.sync();  // (every thread has read mn and mx)
    return ~0u;
  }
  uint32_t* bm = ws + 2 * DGP_MAX_RANK;
  uint32_t* pre = bm + W;
  for (uint32_t w = (uint32_t)tid; w < (uint32_t)W; w += (uint32_t)nt) bm[w] = 0;
  c.sync();
  // Box strides, row-major over the extents.
  uint32_t bs[DGP_MAX_RANK];
  {
    uint32_t st = 1;
    DG_UNROLL
    for (int d = DGP_MAX_RANK - 1; d >= 0; --d) {
      bs[d] = st;
      st *= e[d];
    }
  }
  for (uint32_t i = (uint32_t)tid; i < n; i += (uint32_t)nt) {
    uint32_t x[DGP_MAX_RANK];
    elem_coords(X, F[i], x);
    uint32_t b = 0;
    DG_UNROLL
    for (int d = 0; d < DGP_MAX_RANK; ++d) b += (x[d] - lo[d]) * bs[d];
    c.atomic_or32(&bm[b >> 5], 1u << (b & 31u));
  }
  c.sync();
  for (uint32_t w = (uint32_t)tid; w < (uint32_t)W; w += (uint32_t)nt) pre[w] = (uint32_t)__builtin_popcount(bm[w]);
  c.sync();
  const uint64_t total = block_scan(c, pre, (uint32_t)W);
  // Each thread expands whole words: the coordinates of the word's first
  // cell, then one cell at a time (last coordinate fastest).
  for (uint32_t w = (uint32_t)tid; w < (uint32_t)W; w += (uint32_t)nt) {
    uint32_t bits = bm[w];
    if (!bits) continue;
    uint32_t pos = pre[w];
    uint32_t o[DGP_MAX_RANK];
    uint32_t r = w * 32u;
    DG_UNROLL
    for (int d = DGP_MAX_RANK - 1; d >= 0; --d) {
      o[d] = r % e[d];
      r /= e[d];
    }
    uint32_t flat = 0;
    DG_UNROLL
    for (int d = 0; d < DGP_MAX_RANK; ++d)
      if (d < R) flat += (lo[d] + o[d]) * X.stride[d];
    for (int k = 0; k < 32 && bits; ++k) {
      if (bits & 1u) F[pos++] = flat;
      bits >>= 1;
      // Next cell: add one to the last coordinate, carrying.
      DG_UNROLL
      for (int d = DGP_MAX_RANK - 1; d >= 0; --d) {
        if (d >= R) continue;
        flat += X.stride[d];
        if (++o[d] < e[d]) break;
        flat -= e[d] * X.stride[d];
        o[d] = 0;
      }
    }
  }
  c.sync();
  return (uint32_t)total;
}

// An index function at the calling thread's variables, as ifn_eval; in a
// specialised kernel its terms are unrolled, so that each term's variable,
// coefficient and divisor are constants (a division by a constant divisor
// instead of the general sequence).
DGC bool ifn_eval_dag(const DgpIFn& f, const int32_t* vt, int nt, int32_t* out) {
#ifdef DG_DAG_NOPS
  int32_t x = f.c;
  DG_DAG_UNROLL
  for (int q = 0; q < DGP_MAX_FTERMS; ++q) {
    if (q < f.nterm) {
      int32_t vv = vt[f.var[q] * nt];
      const int32_t d = f.vdiv[q];
      if (d != 1) vv = vv / d;  // variables are non-negative
      x += f.coef[q] * vv;
    }
  }
  if (f.mode == 1) {
    if (x % f.s != 0) return false;
    x = x / f.s;
  } else if (f.mode == 2) {
    x = fdiv(x, f.s);
  }
  *out = x;
  return x >= 0 && x < f.size;
#else
  return ifn_eval(f, vt, nt, out);
#endif
}

// Coordinates of element e of X into the calling thread's variables 0..R-1.
DGC void node_coords(const DgdTensor& X, uint32_t e, int32_t* vt, int nt) {
  DG_DAG_UNROLL
  for (int d = DGP_MAX_RANK - 1; d >= 0; --d) {
    if (d < X.rank) {
      const uint32_t q = magic_div(e, X.magic[d]);
      vt[d * nt] = (int32_t)(e - q * (uint32_t)X.shape[d]);
      e = q;
    }
  }
}

// Element index of operand P at the calling thread's variables; false if an
// index is invalid.
DGC bool operand_flat(const DgdOperand& P, const DgdTensor& Ta, const int32_t* vt, int nt, uint32_t* flat) {
  uint32_t f = 0;
  bool ok = true;
  DG_DAG_UNROLL
  for (int d = 0; d < DGP_MAX_RANK; ++d) {
    if (d < Ta.rank) {
      int32_t v = 0;
      ok = ifn_eval_dag(P.idx[d], vt, nt, &v) && ok;
      f += Ta.stride[d] * (uint32_t)v;
    }
  }
  *flat = f;
  return ok;
}

// An interval variable's index function at the node as c0 + k * w (w the
// variable with index `wv`).
DGC void ifn_linear(const DgpIFn& f, int wv, const int32_t* vt, int nt, int32_t* c0, int32_t* k) {
  int32_t c = f.c, kk = 0;
  DG_DAG_UNROLL
  for (int t = 0; t < DGP_MAX_FTERMS; ++t) {
    if (t < f.nterm) {
      if (f.var[t] == wv) {
        kk = f.coef[t];
      } else {
        int32_t vv = vt[f.var[t] * nt];
        if (f.vdiv[t] != 1) vv = qpos(vv, f.vdiv[t]);  // (variables are non-negative)
        c += f.coef[t] * vv;
      }
    }
  }
  *c0 = c;
  *k = kk;
}

// Appends element `flat` of non-leaf tensor t to its frontier.
template <class C>
DGC void dag_append(C& c, const DgdTensor& Tc, int t, uint32_t flat, uint8_t* area, uint32_t* cnt, uint32_t* err) {
  const uint32_t slot = c.atomic_inc(&cnt[t]);
  if (slot < (uint32_t)Tc.cap) ((uint32_t*)(area + Tc.lds))[slot] = flat;
  else *err |= DGP_ERR_CAPACITY;
}

struct DagCtx {
  const DgdHeader* h;
  const DgdTensor* T;
  const DgdGroup* Gs;
  const DgdOperand* Ps;
  uint8_t* area;
  uint32_t* cnt;
  int32_t* vt;
  int nt;
  uint32_t* err;
};

// One thread, one node of a pointwise op: the node's edges (written from
// `pos` when `emit`), non-leaf children appended when `append`; returns the
// number of edges.  The node's coordinates are in the thread's variables.
template <class C>
DGC uint32_t pointwise_node(C& c, const DagCtx& x, const DgdOp& op, uint64_t pos, const DagOut& o, bool emit,
                            bool append) {
  uint32_t k = 0;
  DG_DAG_UNROLL
  for (int q = 0; q < op.ng; ++q) {
    const DgdGroup& G = x.Gs[op.g0 + q];
    if (G.points == 0) continue;
    bool ok = true;
    DG_DAG_UNROLL
    for (int a = 0; a < G.nop; ++a) {
      const DgdOperand& P = x.Ps[G.op0 + a];
      uint32_t f;
      ok = operand_flat(P, x.T[P.tensor], x.vt, x.nt, &f) && ok;
    }
    if (!ok) continue;
    DG_DAG_UNROLL
    for (int a = 0; a < G.nop; ++a) {
      const DgdOperand& P = x.Ps[G.op0 + a];
      const DgdTensor& Ta = x.T[P.tensor];
      uint32_t f = 0;
      operand_flat(P, Ta, x.vt, x.nt, &f);
      if (emit && pos + k < o.room_edges) {
        c.store_cached(&o.edges[pos + k], Ta.gid + f);
        c.store_cached(&o.mults[pos + k], P.mult);
      }
      if (append && !Ta.leaf) dag_append(c, Ta, P.tensor, f, x.area, x.cnt, x.err);
      ++k;
    }
  }
  return k;
}

// Digits of v in the mixed radix len[0..Q) (last digit fastest, the first
// one unbounded), for v < 2^16.
DGC void radix_digits(uint32_t v, const uint32_t* len, int Q, uint32_t* dg) {
  DG_UNROLL
  for (int q = DGD_MAX_WIN - 1; q >= 1; --q) {
    if (q < Q) {
      uint32_t r;
      v = small_divmod(v, len[q], &r);
      dg[q] = r;
    } else {
      dg[q] = 0;
    }
  }
  dg[0] = v;
}

// Adds the digits inc to dg (each digit below its radix, the first one
// unbounded).
DGC void radix_add(uint32_t* dg, const uint32_t* inc, const uint32_t* len, int Q) {
  uint32_t carry = 0;
  DG_UNROLL
  for (int q = DGD_MAX_WIN - 1; q >= 1; --q) {
    if (q < Q) {
      const uint32_t t = dg[q] + inc[q] + carry;
      carry = t >= len[q] ? 1u : 0u;
      dg[q] = carry ? t - len[q] : t;
    }
  }
  dg[0] += inc[0] + carry;
}

// Group G of the wave's node point by point over the whole window box: the
// valid points are compacted within the wave; writes from `pos` when
// `emit`, appends non-leaf children when `append`; returns the edge count.
template <class C>
DGC uint64_t box_group(C& c, const DagCtx& x, const DgdGroup& G, int R, uint64_t pos, const DagOut& o, bool emit,
                       bool append) {
  const int lane = c.lane(), L = c.lanes();
  const int Q = G.nwin, nop = G.nop;
  const uint64_t P = (uint64_t)G.points;
  uint32_t len[DGD_MAX_WIN], dg[DGD_MAX_WIN], inc[DGD_MAX_WIN];
  DG_UNROLL
  for (int q = 0; q < DGD_MAX_WIN; ++q) len[q] = q < Q ? (uint32_t)(G.whi[q] - G.wlo[q]) : 1u;
  radix_digits((uint32_t)lane, len, Q, dg);
  radix_digits((uint32_t)L, len, Q, inc);
  uint64_t run = 0;
  for (uint64_t p0 = 0; p0 < P; p0 += (uint64_t)L) {
    bool ok = p0 + (uint64_t)lane < P;
    if (ok) {
      DG_UNROLL
      for (int q = 0; q < DGD_MAX_WIN; ++q)
        if (q < Q) x.vt[(R + q) * x.nt] = G.wlo[q] + (int32_t)dg[q];
      for (int a = 0; a < G.nop; ++a) {
        const DgdOperand& Pa = x.Ps[G.op0 + a];
        uint32_t f;
        ok = operand_flat(Pa, x.T[Pa.tensor], x.vt, x.nt, &f) && ok;
      }
    }
    uint32_t tot;
    const uint32_t pre = c.wave_prefix(ok, &tot);
    if (ok && (emit || append)) {
      for (int a = 0; a < G.nop; ++a) {
        const DgdOperand& Pa = x.Ps[G.op0 + a];
        const DgdTensor& Ta = x.T[Pa.tensor];
        uint32_t f = 0;
        operand_flat(Pa, Ta, x.vt, x.nt, &f);
        const uint64_t at = pos + (run + pre) * (uint64_t)nop + (uint64_t)a;
        if (emit && at < o.room_edges) {
          c.store_cached(&o.edges[at], Ta.gid + f);
          c.store_cached(&o.mults[at], Pa.mult);
        }
        if (append && !Ta.leaf) dag_append(c, Ta, Pa.tensor, f, x.area, x.cnt, x.err);
      }
    }
    run += tot;
    radix_add(dg, inc, len, Q);
  }
  return run * (uint64_t)nop;
}

// Per-thread node slots (DgdHeader.slot_off, stride = block threads): per
// window variable its first valid value and progression length (while
// setting up: its bounds), per operand its element index at the first valid
// point, and the node's 64-bit first edge of the group.
struct Slots {
  uint32_t* s;  // this wave's lane 0 column; lane j's column is s + j
  int nt, MQ, MA;
  DGC uint32_t& first(int j, int q) const { return s[(size_t)q * nt + j]; }
  DGC uint32_t& len(int j, int q) const { return s[(size_t)(MQ + q) * nt + j]; }
  DGC uint32_t& base(int j, int a) const { return s[(size_t)(2 * MQ + a) * nt + j]; }
  DGC uint32_t& glo(int j) const { return s[(size_t)(2 * MQ + MA) * nt + j]; }
  DGC uint32_t& ghi(int j) const { return s[(size_t)(2 * MQ + MA + 1) * nt + j]; }
};


// Progressions of group G at the calling thread's node (coordinates in its
// variables): every window variable's first valid value and length and,
// with `bases`, every operand's element index at the first point, in the
// thread's slot column j.  Returns the number of valid points.
DGC uint64_t ap_setup(const DagCtx& x, const DgdGroup& G, int R, const Slots& S, int j, bool bases) {
  const int Q = G.nwin;
  for (int q = 0; q < Q; ++q) {
    S.first(j, q) = (uint32_t)G.wlo[q];
    S.len(j, q) = (uint32_t)(G.whi[q] - 1);  // inclusive upper bound while constraining
  }
  bool bad = false;
  for (int pi = 0; pi < G.npair; ++pi) {
    const DgdPair pr = G.pair[pi];
    if (!pr.bind) continue;
    const DgdOperand& P = x.Ps[G.op0 + pr.a];
    const DgpIFn& f = P.idx[pr.d];
    if (pr.q < 0) {
      int32_t v;
      if (!ifn_eval_dag(f, x.vt, x.nt, &v)) bad = true;
      continue;
    }
    const int q = pr.q;
    int32_t c0, k;
    ifn_linear(f, R + q, x.vt, x.nt, &c0, &k);
    const int32_t top = f.mode == 1 ? f.s * (f.size - 1) : f.size - 1;
    int32_t l2, h2;
    if (k > 0) {
      l2 = ceil_div(-c0, k);
      h2 = floor_div(top - c0, k);
    } else {
      l2 = ceil_div(c0 - top, -k);
      h2 = floor_div(c0, -k);
    }
    if (l2 > (int32_t)S.first(j, q)) S.first(j, q) = (uint32_t)l2;
    if (h2 < (int32_t)S.len(j, q)) S.len(j, q) = (uint32_t)h2;
  }
  if (bad) return 0;
  uint64_t P = 1;
  for (int q = 0; q < Q; ++q) {
    const int32_t lo = (int32_t)S.first(j, q), hi = (int32_t)S.len(j, q), m = G.step[q];
    int32_t first = lo;
    if (G.mpair[q] >= 0) {
      // The exact division c0 + k w = 0 (mod s): g = s / step must divide
      // c0 (also when the step is 1, i.e. s divides k: then no w helps an
      // indivisible c0), then w = (-c0 / g) * inverse(k / g) (mod step).
      const DgdPair pr = G.pair[G.mpair[q]];
      const DgpIFn& f = x.Ps[G.op0 + pr.a].idx[pr.d];
      int32_t c0, k;
      ifn_linear(f, R + q, x.vt, x.nt, &c0, &k);
      const int32_t g = f.s / m;
      if (c0 % g != 0) return 0;
      if (m > 1) {
        const int32_t r = (int32_t)(((int64_t)pmod(-(c0 / g), m) * G.minv[q]) % m);
        first = lo + pmod(r - lo, m);
      }
    }
    const uint32_t len = first <= hi ? (uint32_t)((hi - first) / m + 1) : 0u;
    S.first(j, q) = (uint32_t)first;
    S.len(j, q) = len;
    P *= len;
  }
  if (P == 0 || !bases) return P;
  for (int a = 0; a < G.nop; ++a) S.base(j, a) = x.T[x.Ps[G.op0 + a].tensor].gid;
  for (int pi = 0; pi < G.npair; ++pi) {
    const DgdPair pr = G.pair[pi];
    const DgdOperand& P = x.Ps[G.op0 + pr.a];
    const DgdTensor& Ta = x.T[P.tensor];
    const DgpIFn& f = P.idx[pr.d];
    int32_t v = 0;
    if (pr.q < 0) {
      ifn_eval_dag(f, x.vt, x.nt, &v);
    } else {
      int32_t c0, k;
      ifn_linear(f, R + pr.q, x.vt, x.nt, &c0, &k);
      v = c0 + k * (int32_t)S.first(j, pr.q);
      if (f.mode == 1) v /= f.s;
    }
    S.base(j, pr.a) += Ta.stride[pr.d] * (uint32_t)v;
  }
  return P;
}

// ---- progressions in registers ---------------------------------------------
// The same progressions for groups of Q window variables and NOP operands
// known at compile time: every value stays in the calling thread's
// registers (the window variable of a pair selects its entry by unrolled
// comparison), the pairs that cannot bind are skipped, and the common
// coefficients (unit k, unit steps, no division) take short paths.
template <int Q, int NOP>
struct NodeAP {
  int32_t first[Q > 0 ? Q : 1];
  uint32_t len[Q > 0 ? Q : 1];
  uint32_t base[NOP];
};

template <int Q, int NOP>
DGC uint64_t ap_setup_reg(const DagCtx& x, const DgdGroup& G, int R, bool bases, NodeAP<Q, NOP>& N) {
  constexpr int QD = Q > 0 ? Q : 1;
  int32_t lo[QD], hi[QD];
  DG_UNROLL
  for (int q = 0; q < Q; ++q) {
    lo[q] = G.wlo[q];
    hi[q] = G.whi[q] - 1;
  }
  const int np = G.npair, nb = G.nbind;
  bool bad = false;
  // Only the pairs that can bind (the first nb).
  for (int pi = 0; pi < nb; ++pi) {
    const DgdPair pr = G.pair[pi];
    const DgpIFn& f = x.Ps[G.op0 + pr.a].idx[pr.d];
    if (pr.q < 0) {
      int32_t v;
      if (!ifn_eval_dag(f, x.vt, x.nt, &v)) bad = true;
      continue;
    }
    int32_t c0, k;
    ifn_linear(f, R + pr.q, x.vt, x.nt, &c0, &k);
    const int32_t top = f.mode == 1 ? f.s * (f.size - 1) : f.size - 1;
    int32_t l2, h2;
    if (k == 1) {
      l2 = -c0;
      h2 = top - c0;
    } else if (k == -1) {
      l2 = c0 - top;
      h2 = c0;
    } else if (k > 0) {
      l2 = ceil_div(-c0, k);
      h2 = floor_div(top - c0, k);
    } else {
      l2 = ceil_div(c0 - top, -k);
      h2 = floor_div(c0, -k);
    }
    DG_UNROLL
    for (int q = 0; q < Q; ++q)
      if (q == pr.q) {
        lo[q] = l2 > lo[q] ? l2 : lo[q];
        hi[q] = h2 < hi[q] ? h2 : hi[q];
      }
  }
  if (bad) return 0;
  uint64_t P = 1;
  DG_UNROLL
  for (int q = 0; q < Q; ++q) {
    const int32_t m = G.step[q];
    int32_t first = lo[q];
    if (G.mpair[q] >= 0) {
      // The exact division c0 + k w = 0 (mod s), as in ap_setup.
      const DgdPair pr = G.pair[G.mpair[q]];
      const DgpIFn& f = x.Ps[G.op0 + pr.a].idx[pr.d];
      int32_t c0, k;
      ifn_linear(f, R + q, x.vt, x.nt, &c0, &k);
      const int32_t g = qexact(f.s, m);
      if (g != 1 && pmod(c0, g) != 0) return 0;
      if (m > 1) {
        const int32_t cg = g != 1 ? qexact(c0, g) : c0;
        // (m is a divisor of the stride: pmod(...) * minv stays below m^2.)
        const int32_t r = m < 46341 ? pmod(pmod(-cg, m) * G.minv[q], m)
                                    : (int32_t)(((int64_t)pmod(-cg, m) * G.minv[q]) % m);
        first = lo[q] + pmod(r - lo[q], m);
      }
    }
    const uint32_t len = first <= hi[q] ? (uint32_t)qpos(hi[q] - first, m) + 1u : 0u;
    N.first[q] = first;
    N.len[q] = len;
    P *= len;
  }
  if (P == 0 || !bases) return P;
  DG_UNROLL
  for (int a = 0; a < NOP; ++a) N.base[a] = x.T[x.Ps[G.op0 + a].tensor].gid;
  // Every pair's element index at the first point.
  for (int pi = 0; pi < np; ++pi) {
    const DgdPair pr = G.pair[pi];
    const DgpIFn& f = x.Ps[G.op0 + pr.a].idx[pr.d];
    int32_t v = 0;
    if (pr.q < 0) {
      ifn_eval_dag(f, x.vt, x.nt, &v);
    } else {
      int32_t c0, k;
      ifn_linear(f, R + pr.q, x.vt, x.nt, &c0, &k);
      int32_t fq = 0;
      DG_UNROLL
      for (int q = 0; q < Q; ++q)
        if (q == pr.q) fq = N.first[q];
      v = c0 + k * fq;
      if (f.mode == 1 && f.s != 1) v = qexact(v, f.s);
    }
    const uint32_t add = pr.stride * (uint32_t)v;
    DG_UNROLL
    for (int a = 0; a < NOP; ++a)
      if (a == pr.a) N.base[a] += add;
  }
  return P;
}

// Valid points of fast group G at the calling thread's node (registers,
// no element indices); groups of more than four window variables take
// ap_setup.
DGC uint64_t ap_count(const DagCtx& x, const DgdGroup& G, int R, const Slots& S, int j) {
  switch (G.nwin) {
    case 0: { NodeAP<0, 1> N; return ap_setup_reg<0, 1>(x, G, R, false, N); }
    case 1: { NodeAP<1, 1> N; return ap_setup_reg<1, 1>(x, G, R, false, N); }
    case 2: { NodeAP<2, 1> N; return ap_setup_reg<2, 1>(x, G, R, false, N); }
    case 3: { NodeAP<3, 1> N; return ap_setup_reg<3, 1>(x, G, R, false, N); }
    case 4: { NodeAP<4, 1> N; return ap_setup_reg<4, 1>(x, G, R, false, N); }
    default: return ap_setup(x, G, R, S, j, false);
  }
}

// A group of one point per node (no window, leaf operands only) that
// follows a windowed group in the op's read order: its edges sit right after
// each node's run of the windowed group.  Written by the node loop right
// after that run (or after the group's flat emission for the lanes whose
// node it did not take), rather than in a pass of its own over the batch
// once every run is out: cache lines that the runs and the point share are
// then filled while still in the cache instead of reaching HBM in parts.
struct PointTail {
  bool on;        // the group after this one is written with it (same on every lane)
  uint32_t P;     // the lane's node: 1 when its point is valid
  int nop;
  uint32_t v[3];  // the point's operand elements (global ids)
  uint32_t m[3];  // their multiplicities
};

template <int NOP>
DGC void point_tail_setup(const DagCtx& x, const DgdGroup& G1, int R, bool has, PointTail& t) {
  NodeAP<0, NOP> N{};
  t.P = has ? (uint32_t)ap_setup_reg<0, NOP>(x, G1, R, true, N) : 0u;
  DG_UNROLL
  for (int a = 0; a < NOP; ++a) {
    t.v[a] = N.base[a];
    t.m[a] = x.Ps[G1.op0 + a].mult;
  }
  t.nop = NOP;
  t.on = true;
}

// The point tail of group q of op (off when the fill does not write, when
// group q has no window or the next group is not such a group, or when its
// shape has no compiled form).  The lane's node coordinates are in its
// variables.
DGC PointTail point_tail(const DagCtx& x, const DgdOp& op, int q, int R, bool has, bool emit) {
  PointTail t{};
  if (!emit || q + 1 >= op.ng) return t;
  const DgdGroup& G = x.Gs[op.g0 + q];
  const DgdGroup& G1 = x.Gs[op.g0 + q + 1];
  if (G.nwin == 0 || !G1.fast || !G1.steps24 || G1.nwin != 0 || G1.points == 0) return t;
  for (int a = 0; a < G1.nop; ++a)
    if (!x.T[x.Ps[G1.op0 + a].tensor].leaf) return t;
  switch (G1.nop) {
    case 1:
      if constexpr ((DG_DAG_FAST) & 1u) point_tail_setup<1>(x, G1, R, has, t);
      break;
    case 2:
      if constexpr (((DG_DAG_FAST) >> 5) & 1u) point_tail_setup<2>(x, G1, R, has, t);
      break;
    case 3:
      if constexpr (((DG_DAG_FAST) >> 10) & 1u) point_tail_setup<3>(x, G1, R, has, t);
      break;
    default: break;
  }
  return t;
}

// The lane's point of a tail at edge `at` (nothing when it has none).
template <class C>
DGC void point_tail_write(C& c, const PointTail& t, const DagOut& o, uint64_t at) {
  if (!t.P) return;
  DG_UNROLL
  for (int a = 0; a < 3; ++a)
    if (a < t.nop && at + (uint64_t)a < o.room_edges) {
      c.store_cached(&o.edges[at + a], t.v[a]);
      c.store_cached(&o.mults[at + a], t.m[a]);
    }
}

// Writes group G's edges for the wave's batch of nodes: lane j's node has
// Pj points (0 for none), set up in slot column j with its first edge.  The
// points of the batch are taken flattened across the lanes: point t belongs
// to the node whose prefix brackets it, and its operands go to that node's
// first edge + p * nop + a.
template <class C>
DGC void flat_emit(C& c, const DagCtx& x, const DgdGroup& G, const Slots& S, uint32_t* WP, uint32_t Pj,
                   const DagOut& o, bool emit, bool append) {
  const int lane = c.lane(), L = c.lanes();
  const int Q = G.nwin, nop = G.nop;
  uint32_t T;
  WP[lane] = c.wave_scan(Pj, &T);
  c.wave_sync();
  for (uint64_t t0 = 0; t0 < (uint64_t)T; t0 += (uint64_t)L) {
    const uint64_t tt = t0 + (uint64_t)lane;
    if (tt < (uint64_t)T) {
      const uint32_t t = (uint32_t)tt;
      int j = 0;
      for (int st = L >> 1; st >= 1; st >>= 1)
        if (WP[j + st] <= t) j += st;
      const uint32_t p0 = t - WP[j];
      uint32_t p = p0, idx[DGD_MAX_WIN];
      DG_UNROLL
      for (int q = DGD_MAX_WIN - 1; q >= 1; --q) {
        idx[q] = 0;
        if (q < Q) {
          const uint32_t len = S.len(j, q);
          uint32_t r, quo;
          if (p < 65536u) {
            quo = small_divmod(p, len, &r);
          } else {
            quo = p / len;
            r = p - quo * len;
          }
          idx[q] = r;
          p = quo;
        }
      }
      idx[0] = p;
      const uint64_t at0 = (((uint64_t)S.ghi(j) << 32) | S.glo(j)) + (uint64_t)p0 * (uint64_t)nop;
      for (int a = 0; a < nop; ++a) {
        const DgdOperand& Pa = x.Ps[G.op0 + a];
        uint32_t child = S.base(j, a);
        DG_UNROLL
        for (int q = 0; q < DGD_MAX_WIN; ++q)
          if (q < Q) child += G.astep[a][q] * idx[q];
        const uint64_t at = at0 + (uint64_t)a;
        if (emit && at < o.room_edges) {
          c.store_cached(&o.edges[at], child);
          c.store_cached(&o.mults[at], Pa.mult);
        }
        if (append) {
          const DgdTensor& Ta = x.T[Pa.tensor];
          if (!Ta.leaf) dag_append(c, Ta, Pa.tensor, child - Ta.gid, x.area, x.cnt, x.err);
        }
      }
    }
  }
  c.wave_sync();
}

// Writes group G's edges of the batch nodes in `mask` (lane columns of
// nodes with at least half a wave of points), one node after another: the
// wave covers a node's points with its lanes, the digits of each lane's
// point advancing by the wave width with carries.  NOP operands and Q
// window variables are compile-time constants, so the steps stay in
// registers; the group's operand fields are read once for all the nodes.
template <class C, int NOP, int Q>
DGC void node_emit(C& c, const DagCtx& x, const DgdGroup& G, const Slots& S, uint64_t mask, const DagOut& o,
                   bool emit, bool append) {
  const int lane = c.lane(), L = c.lanes();
  // The group's operands: the same for every node.
  uint32_t mult[NOP], as[NOP][Q > 0 ? Q : 1];
  bool leaf[NOP];
  DG_UNROLL
  for (int a = 0; a < NOP; ++a) {
    const DgdOperand& Pa = x.Ps[G.op0 + a];
    mult[a] = Pa.mult;
    leaf[a] = x.T[Pa.tensor].leaf != 0;
    DG_UNROLL
    for (int q = 0; q < Q; ++q) as[a][q] = G.astep[a][q];
  }
  while (mask) {
    const int j = (int)__builtin_ctzll(mask);
    mask &= mask - 1;
    uint32_t len[DGD_MAX_WIN], dg[DGD_MAX_WIN], inc[DGD_MAX_WIN];
    uint64_t P = 1;
    DG_UNROLL
    for (int q = 0; q < DGD_MAX_WIN; ++q) {
      len[q] = q < Q ? S.len(j, q) : 1u;
      P *= len[q];
    }
    uint32_t base[NOP];
    DG_UNROLL
    for (int a = 0; a < NOP; ++a) base[a] = S.base(j, a);
    const uint64_t at0 = ((uint64_t)S.ghi(j) << 32) | S.glo(j);
    radix_digits((uint32_t)lane, len, Q, dg);
    radix_digits((uint32_t)L, len, Q, inc);
    for (uint64_t p0 = 0; p0 < P; p0 += (uint64_t)L) {
      const uint64_t p = p0 + (uint64_t)lane;
      if (p < P) {
        const uint64_t at = at0 + p * (uint64_t)NOP;
        DG_UNROLL
        for (int a = 0; a < NOP; ++a) {
          uint32_t child = base[a];
          DG_UNROLL
          for (int q = 0; q < Q; ++q) child += as[a][q] * dg[q];
          if (emit && at + a < o.room_edges) {
            c.store_cached(&o.edges[at + a], child);
            c.store_cached(&o.mults[at + a], mult[a]);
          }
          if (append && !leaf[a]) {
            const DgdOperand& Pa = x.Ps[G.op0 + a];
            const DgdTensor& Ta = x.T[Pa.tensor];
            dag_append(c, Ta, Pa.tensor, child - Ta.gid, x.area, x.cnt, x.err);
          }
        }
      }
      radix_add(dg, inc, len, Q);
    }
  }
}

// Digits of v in the mixed radix len[0..Q) (last digit fastest, the first
// one unbounded), for v < 2^16.
template <int Q>
DGC void digits_q(uint32_t v, const uint32_t* len, uint32_t* dg) {
  DG_UNROLL
  for (int q = Q - 1; q >= 1; --q) {
    uint32_t r;
    v = small_divmod(v, len[q], &r);
    dg[q] = r;
  }
  if (Q > 0) dg[0] = v;
}

// The NOP words of one point (the point's operand elements, or their
// multiplicities) at p (4-byte aligned): one store instruction per point.
template <class C, int NOP>
DGC void store_point(C& c, uint32_t* p, const uint32_t* v) {
  if constexpr (NOP == 2) {
    c.store2(p, v[0], v[1]);
  } else if constexpr (NOP == 3) {
    c.store3(p, v[0], v[1], v[2]);
  } else {
    DG_UNROLL
    for (int a = 0; a < NOP; ++a) c.store_cached(p + a, v[a]);
  }
}

// a * b (mod 2^32) for a and b in [-2^23, 2^23) as signed values: one
// full-rate 24-bit multiply on the device.
DGC uint32_t mul24(uint32_t a, uint32_t b) {
#if defined(__HIP_DEVICE_COMPILE__)
  return (uint32_t)__mul24((int)a, (int)b);
#else
  return (uint32_t)((int64_t)(int32_t)a * (int64_t)(int32_t)b);
#endif
}

// q = n / d and *r = n % d for n < 64 and 1 <= d <= 64 from m = ceil(2^16 / d):
// n * m / 2^16 = n / d + n * (m * d - 2^16) / (2^16 d), and the second term
// stays below 1 / d, so the floor is exact.
DGC uint32_t div64(uint32_t n, uint32_t d, uint32_t m, uint32_t* r) {
  const uint32_t q = mul24(n, m) >> 16;
  *r = n - mul24(q, d);
  return q;
}

// Edges of the batch nodes in `mask` (lanes whose node has at least half a
// wave of points), one node after another, from the registers that
// ap_setup_reg filled: each node's lengths, element indices, point count
// and first edge are read from its lane.
//
// The bounded digits (all but the first) span B = len[1] * ... * len[Q-1]
// points.  When B is at most the wave width, the node is covered with the
// largest multiple of B lanes, W: a lane then keeps its bounded digits at
// every step and only the first digit advances (by W / B), so each
// operand's element index advances by a constant (no digit arithmetic per
// point).  Each lane first derives, for its own node, B, W / B and the
// reciprocals that split a lane index into digits; a node's lanes then
// take its digits by multiplications.  Larger B (rare) advance all digits
// with carries.  A node whose edges all fit the room is written without a
// check per edge.
template <class C, int NOP, int Q>
DGC void node_emit_reg(C& c, const DagCtx& x, const DgdGroup& G, const NodeAP<Q, NOP>& N, uint32_t Pj, uint64_t gpos,
                       uint64_t mask, const DagOut& o, bool emit, bool append, const PointTail& tl) {
  if constexpr (Q == 0) return;  // (a group without a window has one point per node: never emitted here)
  constexpr int QD = Q > 0 ? Q : 1;
  const int lane = c.lane(), L = c.lanes();
  uint32_t mult[NOP], as[NOP][QD];
  bool leaf[NOP], any_nonleaf = false;
  DG_UNROLL
  for (int a = 0; a < NOP; ++a) {
    const DgdOperand& Pa = x.Ps[G.op0 + a];
    mult[a] = Pa.mult;
    leaf[a] = x.T[Pa.tensor].leaf != 0;
    any_nonleaf = any_nonleaf || !leaf[a];
    DG_UNROLL
    for (int q = 0; q < Q; ++q) as[a][q] = G.astep[a][q];
  }
  // The lane's own node, packed for one broadcast per word: B (0 when above
  // the wave width) and the bounded lengths (7 bits each, all at most 64
  // when B is), and the reciprocals ceil(2^16 / d) - 1 of B and of those
  // lengths (16 bits each).
  uint32_t mylens = 0, mym[(QD + 1) / 2];
  {
    uint64_t b = 1;
    DG_UNROLL
    for (int q = 1; q < Q; ++q) b *= N.len[q];
    const uint32_t B = Pj != 0 && b <= (uint64_t)L ? (uint32_t)b : 0u;
    mylens = B;
    uint32_t m[QD];
    const uint32_t bd = B ? B : 1u;
    m[0] = (65536u + bd - 1u) / bd - 1u;
    DG_UNROLL
    for (int q = 1; q < Q; ++q) {
      const uint32_t d = B ? N.len[q] : 1u;
      mylens |= (B ? d : 0u) << (7 * q);
      m[q] = (65536u + d - 1u) / d - 1u;
    }
    DG_UNROLL
    for (int k = 0; k < (QD + 1) / 2; ++k) mym[k] = m[2 * k] | (2 * k + 1 < Q ? m[2 * k + 1] << 16 : 0u);
  }
  while (mask) {
    const int j = (int)__builtin_ctzll(mask);
    mask &= mask - 1;
    uint32_t base[NOP];
    DG_UNROLL
    for (int a = 0; a < NOP; ++a) base[a] = c.bcast(N.base[a], j);
    const uint32_t P = c.bcast(Pj, j);
    const uint64_t at0 = ((uint64_t)c.bcast((uint32_t)(gpos >> 32), j) << 32) | c.bcast((uint32_t)gpos, j);
    const bool fits = at0 + (uint64_t)P * NOP <= o.room_edges;
    uint32_t* eb = o.edges + at0;
    uint32_t* mb = o.mults + at0;
    uint32_t child[NOP];
    const uint32_t lens = c.bcast(mylens, j);
    const uint32_t B = lens & 127u;
    if (B != 0) {
      // Bounded digits of lane % B, first digit lane / B; W = (L / B) * B
      // (L / B = L * m / 2^16 by the same bound as div64, L <= 64).
      uint32_t m[QD];
      DG_UNROLL
      for (int k = 0; k < (QD + 1) / 2; ++k) {
        const uint32_t w = c.bcast(mym[k], j);
        m[2 * k] = (w & 0xFFFFu) + 1u;
        if (2 * k + 1 < QD) m[2 * k + 1] = (w >> 16) + 1u;
      }
      const uint32_t per = ((uint32_t)L * m[0]) >> 16, W = per * B;
      uint32_t rr;
      const uint32_t d0 = div64((uint32_t)lane, B, m[0], &rr);
      DG_UNROLL
      for (int a = 0; a < NOP; ++a) child[a] = base[a] + mul24(as[a][0], d0);
      DG_UNROLL
      for (int q = Q - 1; q >= 1; --q) {
        uint32_t dq;
        rr = div64(rr, (lens >> (7 * q)) & 127u, m[q], &dq);
        DG_UNROLL
        for (int a = 0; a < NOP; ++a) child[a] += mul24(as[a][q], dq);
      }
      uint32_t step[NOP];
      DG_UNROLL
      for (int a = 0; a < NOP; ++a) step[a] = as[a][0] * per;
      const bool act = (uint32_t)lane < W;
      uint32_t off = (uint32_t)lane * NOP;
      if (fits && emit && !(append && any_nonleaf)) {
        for (uint32_t p0 = 0; p0 < P; p0 += W) {
          if (act && p0 + (uint32_t)lane < P) {
            store_point<C, NOP>(c, eb + off, child);
            store_point<C, NOP>(c, mb + off, mult);
          }
          DG_UNROLL
          for (int a = 0; a < NOP; ++a) child[a] += step[a];
          off += W * NOP;
        }
      } else {
        for (uint32_t p0 = 0; p0 < P; p0 += W) {
          if (act && p0 + (uint32_t)lane < P) {
            DG_UNROLL
            for (int a = 0; a < NOP; ++a) {
              if (emit && at0 + off + a < o.room_edges) {
                c.store_cached(&eb[off + a], child[a]);
                c.store_cached(&mb[off + a], mult[a]);
              }
              if (append && !leaf[a]) {
                const int t = x.Ps[G.op0 + a].tensor;
                dag_append(c, x.T[t], t, child[a] - x.T[t].gid, x.area, x.cnt, x.err);
              }
            }
          }
          DG_UNROLL
          for (int a = 0; a < NOP; ++a) child[a] += step[a];
          off += W * NOP;
        }
      }
      if (tl.on && lane == j) point_tail_write(c, tl, o, gpos + (uint64_t)Pj * NOP);
      continue;
    }
    // Every digit advances by those of the wave width, with carries: the
    // element index by a per-node constant plus one correction per carry.
    uint32_t len[QD];
    DG_UNROLL
    for (int q = 0; q < Q; ++q) len[q] = c.bcast(N.len[q], j);
    uint32_t dg[QD], inc[QD];
    digits_q<Q>((uint32_t)lane, len, dg);
    digits_q<Q>((uint32_t)L, len, inc);
    uint32_t dstep[NOP], corr[NOP][QD];
    DG_UNROLL
    for (int a = 0; a < NOP; ++a) {
      child[a] = base[a];
      dstep[a] = 0;
      DG_UNROLL
      for (int q = 0; q < Q; ++q) {
        child[a] += as[a][q] * dg[q];
        dstep[a] += as[a][q] * inc[q];
        corr[a][q] = q > 0 ? as[a][q - 1] - as[a][q] * len[q] : 0u;
      }
    }
    uint32_t off = (uint32_t)lane * NOP;
    for (uint32_t p0 = 0; p0 < P; p0 += (uint32_t)L) {
      if (p0 + (uint32_t)lane < P) {
        DG_UNROLL
        for (int a = 0; a < NOP; ++a) {
          if (emit && (fits || at0 + off + a < o.room_edges)) {
            c.store_cached(&eb[off + a], child[a]);
            c.store_cached(&mb[off + a], mult[a]);
          }
          if (append && !leaf[a]) {
            const int t = x.Ps[G.op0 + a].tensor;
            dag_append(c, x.T[t], t, child[a] - x.T[t].gid, x.area, x.cnt, x.err);
          }
        }
      }
      uint32_t carry = 0;
      DG_UNROLL
      for (int q = Q - 1; q >= 1; --q) {
        const uint32_t t = dg[q] + inc[q] + carry;
        carry = t >= len[q] ? 1u : 0u;
        dg[q] = carry ? t - len[q] : t;
        DG_UNROLL
        for (int a = 0; a < NOP; ++a) child[a] += carry ? corr[a][q] : 0u;
      }
      DG_UNROLL
      for (int a = 0; a < NOP; ++a) child[a] += dstep[a];
      off += (uint32_t)L * NOP;
    }
    if (tl.on && lane == j) point_tail_write(c, tl, o, gpos + (uint64_t)Pj * NOP);
  }
}

// A fast group of NOP operands and Q window variables for the wave's batch
// (lane `has` a node, its coordinates in the lane's variables, its first
// edge of the group at gpos): progressions in registers, the nodes with at
// least half a wave of points emitted node by node; the others get their
// slots written and are left to flat_emit (*small: the lane's point count
// there, 0 otherwise).  Returns the lane's point count.
template <class C, int NOP, int Q>
DGC uint32_t fast_group_reg(C& c, const DagCtx& x, const DgdGroup& G, int R, bool has, uint64_t gpos, const Slots& S,
                            const DagOut& o, bool emit, bool append, const PointTail& tl, uint32_t* small) {
  const int lane = c.lane(), L = c.lanes();
  NodeAP<Q, NOP> N{};
  const uint32_t Pj = has ? (uint32_t)ap_setup_reg<Q, NOP>(x, G, R, true, N) : 0u;
  const bool big = Q > 0 && Pj >= (uint32_t)((L + 1) / 2);
  const uint64_t mask = c.ballot(big);
  if (mask) node_emit_reg<C, NOP, Q>(c, x, G, N, Pj, gpos, mask, o, emit, append, tl);
  *small = big ? 0u : Pj;
  if (*small) {
    DG_UNROLL
    for (int q = 0; q < Q; ++q) S.len(lane, q) = N.len[q];
    DG_UNROLL
    for (int a = 0; a < NOP; ++a) S.base(lane, a) = N.base[a];
    S.glo(lane) = (uint32_t)gpos;
    S.ghi(lane) = (uint32_t)(gpos >> 32);
  }
  return Pj;
}

// fast_group_reg for the group's shape; false when it has no compiled form.
template <class C>
DGC bool fast_group(C& c, const DagCtx& x, const DgdGroup& G, int R, bool has, uint64_t gpos, const Slots& S,
                    const DagOut& o, bool emit, bool append, const PointTail& tl, uint32_t* Pj, uint32_t* small) {
  if (!G.steps24) return false;
  switch (G.nop * 16 + G.nwin) {
#define DG_FAST(NOP, Q)                                                                          \
  case NOP * 16 + Q:                                                                             \
    if constexpr (((DG_DAG_FAST) >> ((NOP - 1) * 5 + Q)) & 1u) {                                 \
      *Pj = fast_group_reg<C, NOP, Q>(c, x, G, R, has, gpos, S, o, emit, append, tl, small);     \
      return true;                                                                               \
    } else {                                                                                     \
      return false;                                                                              \
    }
    DG_FAST(1, 0) DG_FAST(1, 1) DG_FAST(1, 2) DG_FAST(1, 3) DG_FAST(1, 4)
    DG_FAST(2, 0) DG_FAST(2, 1) DG_FAST(2, 2) DG_FAST(2, 3) DG_FAST(2, 4)
    DG_FAST(3, 0) DG_FAST(3, 1) DG_FAST(3, 2) DG_FAST(3, 3) DG_FAST(3, 4)
#undef DG_FAST
    default: return false;
  }
}

// Node-major emission of the batch nodes in `mask` (lane columns) when the
// group's shape has a compiled emitter; false when it has none.
template <class C>
DGC bool emit_nodes(C& c, const DagCtx& x, const DgdGroup& G, const Slots& S, uint64_t mask, const DagOut& o,
                    bool emit, bool append) {
  switch (G.nop * 16 + G.nwin) {
#define DG_NODE(NOP, Q)                                                \
  case NOP * 16 + Q:                                                   \
    if constexpr (((DG_DAG_NODE) >> ((NOP - 1) * 4 + Q - 1)) & 1u) {   \
      node_emit<C, NOP, Q>(c, x, G, S, mask, o, emit, append);         \
      return true;                                                     \
    } else {                                                           \
      return false;                                                    \
    }
    DG_NODE(1, 1) DG_NODE(1, 2) DG_NODE(1, 3) DG_NODE(1, 4)
    DG_NODE(2, 1) DG_NODE(2, 2) DG_NODE(2, 3) DG_NODE(2, 4)
    DG_NODE(3, 1) DG_NODE(3, 2) DG_NODE(3, 3) DG_NODE(3, 4)
#undef DG_NODE
    default: return false;
  }
}

// Edge count of the calling lane's node in the wave's batch starting at
// node b0 (0 past the end): the box groups node by node across the wave,
// the progression groups one node per lane.  Called by all lanes of the
// wave; leaves every lane's variables at its own node.
template <class C>
DGC uint64_t batch_node_count(C& c, const DagCtx& x, const DgdOp& op, const DgdTensor& X, const uint32_t* F,
                              uint32_t n, uint32_t b0, int R, const Slots& S) {
  const int lane = c.lane(), L = c.lanes();
  uint64_t m = 0;
  bool any_box = false;
  DG_DAG_UNROLL
  for (int q = 0; q < op.ng; ++q) any_box = any_box || (!x.Gs[op.g0 + q].fast && x.Gs[op.g0 + q].points > 0);
  if constexpr (!DG_DAG_BOX) {
    if (any_box) *x.err |= DGP_ERR_SHAPE;
  } else if (any_box) {
    for (uint32_t j = 0; j < (uint32_t)L && b0 + j < n; ++j) {
      node_coords(X, F[b0 + j], x.vt, x.nt);
      uint64_t mj = 0;
      DG_DAG_UNROLL
      for (int q = 0; q < op.ng; ++q) {
        const DgdGroup& G = x.Gs[op.g0 + q];
        if (!G.fast && G.points > 0) mj += box_group(c, x, G, R, 0, DagOut{}, false, false);
      }
      if ((uint32_t)lane == j) m += mj;
    }
  }
  const uint32_t i = b0 + (uint32_t)lane;
  if (i < n) {
    node_coords(X, F[i], x.vt, x.nt);
    DG_DAG_UNROLL
    for (int q = 0; q < op.ng; ++q) {
      const DgdGroup& G = x.Gs[op.g0 + q];
      if (G.fast && G.points > 0) m += ap_count(x, G, R, S, lane) * (uint64_t)G.nop;
    }
  }
  return m;
}

// One op of the walk (ops in reverse SSA order): the op's nodes from its
// frontier, each node's edge count, the scan, then the edges and the
// non-leaf children.  *nb and *eb are the location's node and edge counts
// so far.  Returns false when the location stops with an error.  Called by
// every thread of the block.
template <class C, int MODE>
DGC bool dag_op(C& c, const DagCtx& x, const DgdOp& op, uint32_t* NC, const Slots& S, uint32_t* WP, const DagOut& o,
                uint64_t* nb_, uint64_t* eb_) {
  const int tid = c.tid(), nt = c.nthreads();
  const int lane = c.lane(), wv = c.wave(), W = c.nwaves(), L = c.lanes();
  const DgdTensor& X = x.T[op.out];
  const uint32_t got = x.cnt[op.out];
  if (got == 0) return true;
  const uint64_t nb = *nb_, eb = *eb_;
  c.sync();  // every thread has read the counter
  if (got > (uint32_t)X.cap) {
    *x.err |= DGP_ERR_CAPACITY;
    return false;
  }
  uint32_t* F = (uint32_t*)(x.area + X.lds);
  // (The node slots are free until the op's edge counts.)
  uint32_t n = box_unique(c, X, F, got, (uint32_t*)(x.area + x.h->slot_off), (uint32_t)(x.h->slot_words * nt));
  if (n == ~0u) n = sort_unique(c, F, got);
  if (MODE == DAG_FILL) {
    for (uint32_t i = (uint32_t)tid; i < n; i += (uint32_t)nt)
      if (nb + i < o.room_nodes) c.store(&o.nodes[nb + i], X.gid + F[i]);
  }
  const int R = X.rank;
  // Edge counts: per node for pointwise ops, per batch of L nodes (one wave's
  // lanes) otherwise; a node's first edge is then its batch's offset plus a
  // wave scan of the batch's node counts.
  if (op.pointwise) {
    if constexpr (DG_DAG_PW) {
      for (uint32_t i = (uint32_t)tid; i < n; i += (uint32_t)nt) {
        node_coords(X, F[i], x.vt, nt);
        NC[i] = pointwise_node(c, x, op, 0, o, false, false);
      }
    } else {
      *x.err |= DGP_ERR_SHAPE;
      return false;
    }
  } else {
    for (uint32_t b0 = (uint32_t)(wv * L); b0 < n; b0 += (uint32_t)(W * L)) {
      const uint64_t m = batch_node_count(c, x, op, X, F, n, b0, R, S);
      const uint64_t tot = c.wave_sum64(m);
      if (tot > 0xFFFFFFFFull) *x.err |= DGP_ERR_OVERFLOW;
      if (lane == 0) NC[b0 / (uint32_t)L] = (uint32_t)tot;
    }
  }
  c.sync();
  const uint32_t ncount = op.pointwise ? n : (n + (uint32_t)L - 1) / (uint32_t)L;
  const uint64_t total = block_scan(c, NC, ncount);
  if (eb + total > 0xFFFFFFFFull) {
    *x.err |= DGP_ERR_OVERFLOW;
    return false;
  }
  // The edges, and the non-leaf children.
  const bool emit = MODE == DAG_FILL, append = op.nonleaf != 0;
  if (op.pointwise) {
    if constexpr (DG_DAG_PW) {
      for (uint32_t i = (uint32_t)tid; i < n; i += (uint32_t)nt) {
        if (MODE == DAG_FILL && nb + i < o.room_nodes) c.store(&o.node_edge[nb + i], (uint32_t)(eb + NC[i]));
        if (emit || append) {
          node_coords(X, F[i], x.vt, nt);
          pointwise_node(c, x, op, eb + NC[i], o, emit, append);
        }
      }
    }
  } else if (emit || append) {
    for (uint32_t b0 = (uint32_t)(wv * L); b0 < n; b0 += (uint32_t)(W * L)) {
      const uint32_t i = b0 + (uint32_t)lane;
      const bool has = i < n;
      const uint64_t m = batch_node_count(c, x, op, X, F, n, b0, R, S);
      uint32_t tot;
      uint64_t gpos = eb + NC[b0 / (uint32_t)L] + c.wave_scan((uint32_t)m, &tot);
      if (MODE == DAG_FILL && has && nb + i < o.room_nodes) c.store(&o.node_edge[nb + i], (uint32_t)gpos);
      bool taken = false;  // the group was written as the point tail of the one before
      DG_DAG_UNROLL
      for (int q = 0; q < op.ng; ++q) {
        if (taken) {
          taken = false;
          continue;
        }
        const DgdGroup& G = x.Gs[op.g0 + q];
        if (G.points == 0) continue;
        if (G.fast) {
          uint32_t Pj = 0, small = 0;
          if (has) node_coords(X, F[i], x.vt, nt);
          const PointTail tl = point_tail(x, op, q, R, has, emit);
          if (fast_group(c, x, G, R, has, gpos, S, o, emit, append, tl, &Pj, &small)) {
            if (c.ballot(small != 0)) {
              c.wave_sync();
              flat_emit(c, x, G, S, WP, small, o, emit, append);
            }
            if (tl.on) {
              // Nodes the node loop did not take (fewer than half a wave of
              // points) get their point here.
              const uint64_t at = gpos + (uint64_t)Pj * (uint64_t)G.nop;
              if (has && Pj < (uint32_t)((L + 1) / 2)) point_tail_write(c, tl, o, at);
              gpos += (uint64_t)tl.P * (uint64_t)tl.nop;
              taken = true;
            }
          } else if constexpr (DG_DAG_SLOW) {
            if (has) {
              Pj = (uint32_t)ap_setup(x, G, R, S, lane, true);
              S.glo(lane) = (uint32_t)gpos;
              S.ghi(lane) = (uint32_t)(gpos >> 32);
            }
            // Nodes with at least half a wave of points node by node, the
            // others flattened across the lanes.
            const bool big = Pj >= (uint32_t)((L + 1) / 2);
            const uint64_t mask = c.ballot(big);
            c.wave_sync();
            const bool done = mask != 0 && emit_nodes(c, x, G, S, mask, o, emit, append);
            flat_emit(c, x, G, S, WP, done && big ? 0u : Pj, o, emit, append);
          } else {
            *x.err |= DGP_ERR_SHAPE;
          }
          gpos += (uint64_t)Pj * (uint64_t)G.nop;
        } else if constexpr (!DG_DAG_BOX) {
          *x.err |= DGP_ERR_SHAPE;
        } else {
          S.glo(lane) = (uint32_t)gpos;
          S.ghi(lane) = (uint32_t)(gpos >> 32);
          c.wave_sync();
          for (uint32_t j = 0; j < (uint32_t)L && b0 + j < n; ++j) {
            node_coords(X, F[b0 + j], x.vt, nt);
            const uint64_t gj = ((uint64_t)S.ghi((int)j) << 32) | S.glo((int)j);
            const uint64_t mj = box_group(c, x, G, R, gj, o, emit, append);
            if ((uint32_t)lane == j) gpos += mj;
          }
          c.wave_sync();
        }
      }
    }
  }
  c.sync();
  *nb_ = nb + n;
  *eb_ = eb + total;
  return true;
}

// Ops K, K-1, ..., 0 of the walk, unrolled (a specialised kernel).
template <class C, int MODE, int K>
DGC bool dag_walk(C& c, const DagCtx& x, const DgdOp* O, uint32_t* NC, const Slots& S, uint32_t* WP,
                  const DagOut& o, uint64_t* nb, uint64_t* eb) {
  if constexpr (K < 0) {
    return true;
  } else {
    if (!dag_op<C, MODE>(c, x, O[K], NC, S, WP, o, nb, eb)) return false;
    return dag_walk<C, MODE, K - 1>(c, x, O, NC, S, WP, o, nb, eb);
  }
}

// Expression DAG of res(y[loc]).
template <class C, int MODE>
DGC void location_dag(C& c, const uint8_t* dblob, int64_t loc, uint8_t* area, const DagOut& o, uint64_t* n_nodes,
                      uint64_t* n_edges, uint32_t* err) {
  const DgdHeader* h = (const DgdHeader*)dblob;
  const DgdTensor* T = (const DgdTensor*)(dblob + h->tensor_off);
  const DgdOp* O = (const DgdOp*)(dblob + h->op_off);
  const int tid = c.tid(), nt = c.nthreads();
  uint32_t* cnt = (uint32_t*)(area + h->count_off);
  uint32_t* NC = (uint32_t*)(area + h->ncount_off);
  const int wbase = c.wave() * c.lanes();
  const Slots S{(uint32_t*)(area + h->slot_off) + wbase, nt, h->max_win, h->max_opnd};
  uint32_t* WP = (uint32_t*)(area + h->wave_off) + wbase;
  DagCtx x{h, T, (const DgdGroup*)(dblob + h->group_off), (const DgdOperand*)(dblob + h->operand_off), area, cnt,
           (int32_t*)(area + h->vars_off) + tid, nt, err};
  *n_nodes = 0;
  *n_edges = 0;
  if (loc < 0 || loc >= h->out_numel) {
    *err |= DGP_ERR_RANGE;
    return;
  }
  for (int t = tid; t < h->ntensor; t += nt) cnt[t] = 0;
  c.sync();
  const DgdTensor& Ty = T[h->output];
  if (!Ty.leaf) {
    if (tid == 0) {
      ((uint32_t*)(area + Ty.lds))[0] = (uint32_t)loc;
      cnt[h->output] = 1;
    }
  }
  c.sync();
  uint64_t nb = 0, eb = 0;
#ifdef DG_DAG_NOPS
  if (!dag_walk<C, MODE, DG_DAG_NOPS - 1>(c, x, O, NC, S, WP, o, &nb, &eb)) return;
#else
  for (int k = h->nop - 1; k >= 0; --k)
    if (!dag_op<C, MODE>(c, x, O[k], NC, S, WP, o, &nb, &eb)) return;
#endif
  *n_nodes = nb;
  *n_edges = eb;
}

}  // namespace dgc
