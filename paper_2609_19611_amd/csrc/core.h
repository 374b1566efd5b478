// Per-location plan execution and row emission, written once for a block of
// cooperating threads (`C` supplies tid, nthreads, barriers, atomics and
// ordered prefix counts).  The device kernels instantiate it with a HIP
// block; the host emulation used by the CPU tests instantiates it with a
// single thread.
//
// One location is processed by one block:
//   1. plan_exec runs the compiled instructions: every factor is a dense
//      vector over a contiguous coordinate range of one tensor dim, kept in
//      the local data share (LDS) together with the scalars;
//   2. for each leaf in declaration order, the union of its terms' nonzero
//      coordinates is formed per dim (ordered compaction), giving a sorted
//      grid whose row-major order is ascending global id;
//   3. the grid is split into an outer and an inner table of (id part,
//      count part) pairs, so that each entry costs two LDS reads, one add
//      and one multiply before its two coalesced stores.
#pragma once
#include <stdint.h>

#include "program.h"

// The including file defines DGC (device code: __device__ __forceinline__);
// plain host builds get ordinary inline functions.
#ifndef DGC
#define DGC inline
#endif

namespace dgc {

// ---------------------------------------------------------------- layout --
struct PlanLayout {
  uint32_t scal, fmeta, fval, end;  // byte offsets in the block's LDS area
};

// Per-leaf emission view of one separable term.
struct TermRef {
  uint64_t coef;
  int32_t lo[DGP_MAX_RANK];
  int32_t len[DGP_MAX_RANK];
  uint32_t off[DGP_MAX_RANK];  // uint64 index of the factor's values in the LDS area
};

struct EmitLayout {
  uint32_t terms;    // TermRef[max_terms]
  uint32_t ulist;    // int32[union_entries]
  uint32_t tables;   // uint32[emit_entries]
  uint32_t scratch;  // uint64[2 * 64 + 8]
  uint32_t end;
};

DGC uint32_t align8(uint32_t x) { return (x + 7u) & ~7u; }

DGC PlanLayout plan_layout(const DgpHeader* h, uint32_t base) {
  PlanLayout L;
  L.scal = align8(base);
  L.fmeta = L.scal + 8u * (uint32_t)h->nscalar;
  L.fval = L.fmeta + 8u * (uint32_t)h->nfactor;
  L.end = L.fval + 8u * (uint32_t)h->fval_entries;
  return L;
}

DGC EmitLayout emit_layout(uint32_t base, int32_t max_terms, int32_t union_entries, int32_t emit_entries) {
  EmitLayout E;
  E.terms = align8(base);
  E.ulist = E.terms + (uint32_t)sizeof(TermRef) * (uint32_t)(max_terms > 0 ? max_terms : 1);
  E.tables = align8(E.ulist + 4u * (uint32_t)union_entries);
  E.scratch = align8(E.tables + 4u * (uint32_t)emit_entries);
  E.end = E.scratch + 8u * (2u * 64u + 8u);
  return E;
}

// Per-leaf emission shape (the compiled one, or the combined one for a
// two-graph comparison).
struct LeafShape {
  int32_t split;
  int32_t ucap[DGP_MAX_RANK];
};

// ------------------------------------------------------------ arithmetic --
DGC int32_t fdiv(int32_t a, int32_t b) {
  int32_t q = a / b;
  if ((a % b) != 0 && ((a < 0) != (b < 0))) --q;
  return q;
}

// Evaluates an index function at variable values v; false if an exact
// division does not divide or the result is outside [0, size).
DGC bool ifn_eval(const DgpIFn& f, const int32_t* v, int32_t* out) {
  int32_t x = f.c;
  for (int q = 0; q < f.nterm; ++q) {
    int32_t vv = v[f.var[q]];
    if (f.vdiv[q] != 1) vv = vv / f.vdiv[q];  // variables are non-negative
    x += f.coef[q] * vv;
  }
  if (f.mode == 1) {
    if (x % f.s != 0) return false;
    x = x / f.s;
  } else if (f.mode == 2) {
    x = fdiv(x, f.s);
  }
  *out = x;
  return x >= 0 && x < f.size;
}

// Range of an index function over variables v in [vlo, vlo + vn).
DGC void ifn_range(const DgpIFn& f, const int32_t* vlo, const int32_t* vn, int32_t* lo, int32_t* hi) {
  int32_t a = f.c, b = f.c;
  for (int q = 0; q < f.nterm; ++q) {
    int32_t x0 = vlo[f.var[q]], x1 = vlo[f.var[q]] + vn[f.var[q]] - 1;
    if (f.vdiv[q] != 1) {
      x0 /= f.vdiv[q];
      x1 /= f.vdiv[q];
    }
    if (f.coef[q] >= 0) {
      a += f.coef[q] * x0;
      b += f.coef[q] * x1;
    } else {
      a += f.coef[q] * x1;
      b += f.coef[q] * x0;
    }
  }
  if (f.mode == 1) {
    a = -fdiv(-a, f.s);
    b = fdiv(b, f.s);
  } else if (f.mode == 2) {
    a = fdiv(a, f.s);
    b = fdiv(b, f.s);
  }
  *lo = a;
  *hi = b;
}

DGC uint64_t mul_sat(uint64_t a, uint64_t b) {
  if (a == 0 || b == 0) return 0;
  if (a > ~0ull / b) return ~0ull;
  return a * b;
}

// ------------------------------------------------------------ plan_exec --
template <class C>
DGC void plan_exec(C& c, const uint8_t* blob, int64_t loc, uint8_t* area, const PlanLayout& PL, uint32_t* err) {
  const DgpHeader* h = (const DgpHeader*)blob;
  const DgpInstr* ins = (const DgpInstr*)(blob + h->instr_off);
  const DgpFactor* fac = (const DgpFactor*)(blob + h->factor_off);
  uint64_t* scal = (uint64_t*)(area + PL.scal);
  int32_t* meta = (int32_t*)(area + PL.fmeta);
  uint64_t* fval = (uint64_t*)(area + PL.fval);
  const int tid = c.tid(), nt = c.nthreads();
  for (int k = 0; k < h->ninstr; ++k) {
    const DgpInstr& I = ins[k];
    const int op = I.opcode;
    if (op == DGP_ROOT || op == DGP_CONST) {
      if (tid == 0) {
        int32_t x;
        if (op == DGP_ROOT) x = (int32_t)((loc / h->out_stride[I.a]) % h->out_shape[I.a]);
        else x = I.a;
        meta[2 * I.dst] = x;
        meta[2 * I.dst + 1] = 1;
        fval[fac[I.dst].off] = 1;
      }
    } else if (op == DGP_COMP) {
      const int nv = I.nvar;
      int32_t vlo[DGP_MAX_VARS], vn[DGP_MAX_VARS];
      uint32_t P = 1;
      for (int q = 0; q < nv; ++q) {
        int src = I.var_src[q];
        if (src >= 0) {
          vlo[q] = meta[2 * src];
          vn[q] = meta[2 * src + 1];
        } else {
          vlo[q] = I.wlo[q];
          vn[q] = I.whi[q] - I.wlo[q];
        }
        P *= (uint32_t)vn[q];
      }
      int32_t tlo = 0, tlen = 0;
      uint64_t* dv = nullptr;
      if (!I.dst_is_scalar) {
        const DgpFactor F = fac[I.dst];
        int32_t hi;
        ifn_range(I.target, vlo, vn, &tlo, &hi);
        if (tlo < 0) tlo = 0;
        if (hi > F.size - 1) hi = F.size - 1;
        tlen = (P == 0 || hi < tlo) ? 0 : hi - tlo + 1;
        if (tlen > F.cap) {
          *err |= DGP_ERR_CAPACITY;
          tlen = F.cap;
        }
        dv = fval + F.off;
        if (tid == 0) {
          meta[2 * I.dst] = tlo;
          meta[2 * I.dst + 1] = tlen;
        }
        for (int i = tid; i < tlen; i += nt) dv[i] = 0;
      } else if (tid == 0) {
        scal[I.dst] = 0;
      }
      c.sync();
      uint64_t acc = 0;
      for (uint32_t p = (uint32_t)tid; p < P; p += (uint32_t)nt) {
        int32_t v[DGP_MAX_VARS];
        uint32_t rem = p;
        uint64_t w = 1;
        for (int q = nv - 1; q >= 0; --q) {
          uint32_t n = (uint32_t)vn[q];
          uint32_t r = rem % n;
          rem /= n;
          v[q] = vlo[q] + (int32_t)r;
          int src = I.var_src[q];
          if (src >= 0) w *= fval[fac[src].off + r];
        }
        if (w == 0) continue;
        bool ok = true;
        for (int e = 0; e < I.npred && ok; ++e) {
          int32_t t;
          ok = ifn_eval(I.pred[e], v, &t);
        }
        if (!ok) continue;
        if (dv) {
          int32_t t;
          if (!ifn_eval(I.target, v, &t) || t < tlo || t >= tlo + tlen) continue;
          c.atomic_add(&dv[t - tlo], w);
        } else {
          acc += w;
        }
      }
      if (!dv && acc) c.atomic_add(&scal[I.dst], acc);
    } else if (op == DGP_LINCOMB) {
      int32_t lo1 = meta[2 * I.f1], n1 = meta[2 * I.f1 + 1];
      int32_t lo2 = meta[2 * I.f2], n2 = meta[2 * I.f2 + 1];
      uint64_t k1 = (I.k1 < 0 ? 1ull : scal[I.k1]) * I.c1;
      uint64_t k2 = (I.k2 < 0 ? 1ull : scal[I.k2]) * I.c2;
      int32_t lo, hi;
      if (n1 == 0 && n2 == 0) {
        lo = 0;
        hi = 0;
      } else if (n1 == 0) {
        lo = lo2;
        hi = lo2 + n2;
      } else if (n2 == 0) {
        lo = lo1;
        hi = lo1 + n1;
      } else {
        lo = lo1 < lo2 ? lo1 : lo2;
        hi = (lo1 + n1) > (lo2 + n2) ? (lo1 + n1) : (lo2 + n2);
      }
      int32_t len = hi - lo;
      const DgpFactor F = fac[I.dst];
      if (len > F.cap) {
        *err |= DGP_ERR_CAPACITY;
        len = F.cap;
      }
      const uint64_t* a1 = fval + fac[I.f1].off;
      const uint64_t* a2 = fval + fac[I.f2].off;
      uint64_t* dv = fval + F.off;
      if (tid == 0) {
        meta[2 * I.dst] = lo;
        meta[2 * I.dst + 1] = len;
      }
      for (int i = tid; i < len; i += nt) {
        int32_t x = lo + i;
        uint64_t s = 0;
        if (x - lo1 >= 0 && x - lo1 < n1) s += k1 * a1[x - lo1];
        if (x - lo2 >= 0 && x - lo2 < n2) s += k2 * a2[x - lo2];
        dv[i] = s;
      }
    } else if (op == DGP_SMUL) {
      if (tid == 0) {
        uint64_t v = I.cst;
        for (int q = 0; q < I.ns; ++q) v *= scal[I.s[q]];
        scal[I.dst] = v;
      }
    } else if (op == DGP_SADD) {
      if (tid == 0) {
        uint64_t a = (I.f1 < 0 ? 1ull : scal[I.f1]) * I.c1;
        uint64_t b = (I.f2 < 0 ? 1ull : scal[I.f2]) * I.c2;
        scal[I.dst] = a + b;
      }
    }
    c.sync();
  }
}

// Fills TermRef[t0 .. t0 + L.nterm) for leaf `leaf` of a plan.
template <class C>
DGC void leaf_terms(C& c, const uint8_t* blob, int leaf, uint8_t* area, const PlanLayout& PL, TermRef* out) {
  const DgpHeader* h = (const DgpHeader*)blob;
  const DgpLeaf* L = (const DgpLeaf*)(blob + h->leaf_off) + leaf;
  const DgpTerm* T = (const DgpTerm*)(blob + h->term_off) + L->term0;
  const DgpFactor* fac = (const DgpFactor*)(blob + h->factor_off);
  const uint64_t* scal = (const uint64_t*)(area + PL.scal);
  const int32_t* meta = (const int32_t*)(area + PL.fmeta);
  for (int t = c.tid(); t < L->nterm; t += c.nthreads()) {
    TermRef r;
    r.coef = (T[t].coef_slot < 0 ? 1ull : scal[T[t].coef_slot]) * T[t].coef_const;
    for (int d = 0; d < L->rank; ++d) {
      int f = T[t].factor[d];
      r.lo[d] = meta[2 * f];
      r.len[d] = meta[2 * f + 1];
      r.off[d] = (PL.fval >> 3) + (uint32_t)fac[f].off;
    }
    out[t] = r;
  }
}

DGC uint64_t term_val(const TermRef& r, int d, int32_t x, const uint64_t* area64) {
  int32_t i = x - r.lo[d];
  return (i >= 0 && i < r.len[d]) ? area64[r.off[d] + (uint32_t)i] : 0ull;
}

// Builds the sorted union of nonzero coordinates per dim over terms [0, nterm).
// Returns false (leaf empty) if some dim has no nonzero coordinate.
template <class C>
DGC bool build_union(C& c, const TermRef* terms, int nterm, int rank, const int32_t* ucap, int32_t* ulist,
                     int32_t* u, uint8_t* area, uint32_t* err) {
  const uint64_t* a64 = (const uint64_t*)area;
  const int tid = c.tid(), nt = c.nthreads();
  bool empty = false;
  int32_t base_off = 0;
  for (int d = 0; d < rank; ++d) {
    int32_t hlo = 0x7fffffff, hhi = -0x7fffffff;
    for (int t = 0; t < nterm; ++t) {
      if (terms[t].len[d] <= 0) continue;
      if (terms[t].lo[d] < hlo) hlo = terms[t].lo[d];
      if (terms[t].lo[d] + terms[t].len[d] > hhi) hhi = terms[t].lo[d] + terms[t].len[d];
    }
    int32_t count = 0;
    int32_t* ul = ulist + base_off;
    for (int32_t chunk = hlo; chunk < hhi; chunk += nt) {
      int32_t x = chunk + tid;
      bool nz = false;
      if (x < hhi)
        for (int t = 0; t < nterm && !nz; ++t) nz = term_val(terms[t], d, x, a64) != 0;
      uint32_t tot;
      uint32_t pre = c.prefix(nz, &tot);
      if (nz && count + (int32_t)pre < ucap[d]) ul[count + (int32_t)pre] = x;
      count += (int32_t)tot;
    }
    if (count > ucap[d]) {
      *err |= DGP_ERR_CAPACITY;
      count = ucap[d];
    }
    u[d] = count;
    if (count == 0) empty = true;
    base_off += ucap[d];
  }
  c.sync();
  return !empty;
}

// Mode of a leaf pass.
enum { EMIT_COUNT = 0, EMIT_FILL = 1, EMIT_COMPARE = 2 };

struct LeafGeom {
  int32_t rank;
  uint32_t base;
  uint32_t stride[DGP_MAX_RANK];
};

// One leaf of one location.  Terms [0, na) belong to graph A (the graph
// being enumerated), terms [na, na + nb) to graph B (compare only).
//   EMIT_COUNT:   returns the number of nonzero entries.
//   EMIT_FILL:    writes them at ids/cnt and returns their number.
//   EMIT_COMPARE: returns 0 equal, 1 nonzero sets differ, 2 counts differ.
//   `room` bounds the entries EMIT_FILL may write at ids/cnt; a leaf that
//   would need more raises DGP_ERR_SIZE and writes nothing past it.
template <class C, int MODE>
DGC uint64_t leaf_pass(C& c, const LeafGeom& G, const LeafShape& S, const TermRef* terms, int na, int nb,
                       uint8_t* area, const EmitLayout& E, uint32_t* ids, uint32_t* cnt, uint64_t room,
                       uint32_t* err) {
  const int tid = c.tid(), nt = c.nthreads();
  const int nterm = na + nb;
  const int rank = G.rank;
  if (MODE != EMIT_COMPARE && na == 0) return 0;
  if (MODE == EMIT_COMPARE && nterm == 0) return 0;
  int32_t* ulist = (int32_t*)(area + E.ulist);
  int32_t u[DGP_MAX_RANK];
  if (!build_union(c, terms, nterm, rank, S.ucap, ulist, u, area, err)) {
    // Some dim has no nonzero coordinate in any term: the leaf is absent
    // from both rows.
    return 0;
  }
  const uint64_t* a64 = (const uint64_t*)area;
  int32_t uoff[DGP_MAX_RANK];
  {
    int32_t o = 0;
    for (int d = 0; d < rank; ++d) {
      uoff[d] = o;
      o += S.ucap[d];
    }
  }
  uint64_t* scratch = (uint64_t*)(area + E.scratch);
  const int split = S.split;

  if (split >= 0) {
    // Outer table over dims [0, split), inner over [split, rank); an entry is
    // (id part, count part per term).
    const int W = 1 + nterm;
    uint32_t O = 1, In = 1;
    for (int d = 0; d < split; ++d) O *= (uint32_t)u[d];
    for (int d = split; d < rank; ++d) In *= (uint32_t)u[d];
    uint32_t* otab = (uint32_t*)(area + E.tables);
    uint32_t* itab = otab + (uint64_t)O * W;
    for (int i = tid; i < 2 * nterm; i += nt) scratch[i] = 0;
    c.sync();
    for (int side = 0; side < 2; ++side) {
      const int d0 = side == 0 ? 0 : split, d1 = side == 0 ? split : rank;
      const uint32_t n = side == 0 ? O : In;
      uint32_t* tab = side == 0 ? otab : itab;
      for (uint32_t r = (uint32_t)tid; r < n; r += (uint32_t)nt) {
        uint32_t rem = r;
        int32_t x[DGP_MAX_RANK];
        uint32_t pos = side == 0 ? G.base : 0u;
        for (int d = d1 - 1; d >= d0; --d) {
          uint32_t i = rem % (uint32_t)u[d];
          rem /= (uint32_t)u[d];
          x[d] = ulist[uoff[d] + (int32_t)i];
          pos += (uint32_t)x[d] * G.stride[d];
        }
        tab[(uint64_t)r * W] = pos;
        for (int t = 0; t < nterm; ++t) {
          uint64_t v = side == 0 ? terms[t].coef : 1ull;
          for (int d = d0; d < d1 && v; ++d) v = mul_sat(v, term_val(terms[t], d, x[d], a64));
          tab[(uint64_t)r * W + 1 + t] = v > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)v;
          if (v) c.atomic_max(&scratch[2 * t + side], v);
        }
      }
    }
    c.sync();
    // A term whose largest outer and inner parts multiply past 32 bits has a
    // real cell with that count.
    for (int t = tid; t < nterm; t += nt) {
      uint64_t a = scratch[2 * t], b = scratch[2 * t + 1];
      if (a && b && (a > 0xFFFFFFFFull || b > 0xFFFFFFFFull || a * b > 0xFFFFFFFFull)) *err |= DGP_ERR_OVERFLOW;
    }
    const uint64_t total = (uint64_t)O * In;
    if (MODE == EMIT_COUNT && nterm == 1) return total;
    if (MODE == EMIT_FILL && nterm == 1) {
      // Dense single-term grid: every cell is an entry, in order.
      if (total > room) *err |= DGP_ERR_SIZE;
      const uint32_t tot32 = (uint32_t)(total < room ? total : room);
      const uint32_t step = (uint32_t)nt;
      const uint32_t dr = step / In, dj = step % In;
      uint32_t p = (uint32_t)tid;
      uint32_t r = p / In, j = p % In;
      for (; p < tot32; p += step) {
        const uint32_t* o = otab + (uint64_t)r * 2;
        const uint32_t* q = itab + (uint64_t)j * 2;
        c.store(&ids[p], o[0] + q[0]);
        c.store(&cnt[p], o[1] * q[1]);
        j += dj;
        r += dr;
        if (j >= In) {
          j -= In;
          ++r;
        }
      }
      return total;
    }
    // Several terms: evaluate each cell, keep the nonzero ones in order.
    uint64_t written = 0;
    uint32_t flags = 0;
    for (uint64_t chunk = 0; chunk < total; chunk += (uint64_t)nt) {
      uint64_t p = chunk + (uint64_t)tid;
      uint64_t ca = 0, cb = 0;
      uint32_t pos = 0;
      if (p < total) {
        uint32_t r = (uint32_t)(p / In), j = (uint32_t)(p % In);
        const uint32_t* o = otab + (uint64_t)r * W;
        const uint32_t* q = itab + (uint64_t)j * W;
        pos = o[0] + q[0];
        for (int t = 0; t < na; ++t) ca += (uint64_t)o[1 + t] * q[1 + t];
        for (int t = na; t < nterm; ++t) cb += (uint64_t)o[1 + t] * q[1 + t];
      }
      if (MODE == EMIT_COMPARE) {
        if ((ca == 0) != (cb == 0)) flags |= 1u;
        else if (ca != cb) flags |= 2u;
        if (c.any((flags & 1u) != 0)) return 1;
      } else {
        if (ca > 0xFFFFFFFFull) *err |= DGP_ERR_OVERFLOW;
        bool nz = ca != 0;
        uint32_t tot;
        uint32_t pre = c.prefix(nz, &tot);
        if (MODE == EMIT_FILL && nz) {
          if (written + pre < room) {
            c.store(&ids[written + pre], pos);
            c.store(&cnt[written + pre], (uint32_t)ca);
          } else {
            *err |= DGP_ERR_SIZE;
          }
        }
        written += tot;
      }
    }
    if (MODE == EMIT_COMPARE) return c.any((flags & 2u) != 0) ? 2 : 0;
    return written;
  }

  // No tables: decompose every cell of the union grid.
  uint64_t total = 1;
  for (int d = 0; d < rank; ++d) total *= (uint64_t)u[d];
  uint64_t written = 0;
  uint32_t flags = 0;
  for (uint64_t chunk = 0; chunk < total; chunk += (uint64_t)nt) {
    uint64_t p = chunk + (uint64_t)tid;
    uint64_t ca = 0, cb = 0;
    uint32_t pos = G.base;
    if (p < total) {
      int32_t x[DGP_MAX_RANK];
      uint64_t rem = p;
      for (int d = rank - 1; d >= 0; --d) {
        uint64_t i = rem % (uint64_t)u[d];
        rem /= (uint64_t)u[d];
        x[d] = ulist[uoff[d] + (int32_t)i];
        pos += (uint32_t)x[d] * G.stride[d];
      }
      for (int t = 0; t < nterm; ++t) {
        uint64_t v = terms[t].coef;
        for (int d = 0; d < rank && v; ++d) v = mul_sat(v, term_val(terms[t], d, x[d], a64));
        if (t < na) ca = (ca + v < ca) ? ~0ull : ca + v;
        else cb = (cb + v < cb) ? ~0ull : cb + v;
      }
    }
    if (MODE == EMIT_COMPARE) {
      if ((ca == 0) != (cb == 0)) flags |= 1u;
      else if (ca != cb) flags |= 2u;
      if (c.any((flags & 1u) != 0)) return 1;
    } else {
      if (ca > 0xFFFFFFFFull) *err |= DGP_ERR_OVERFLOW;
      bool nz = ca != 0;
      uint32_t tot;
      uint32_t pre = c.prefix(nz, &tot);
      if (MODE == EMIT_FILL && nz) {
        if (written + pre < room) {
          c.store(&ids[written + pre], pos);
          c.store(&cnt[written + pre], (uint32_t)ca);
        } else {
          *err |= DGP_ERR_SIZE;
        }
      }
      written += tot;
    }
  }
  if (MODE == EMIT_COMPARE) return c.any((flags & 2u) != 0) ? 2 : 0;
  return written;
}

DGC LeafGeom leaf_geom(const DgpLeaf& L) {
  LeafGeom G;
  G.rank = L.rank;
  G.base = L.base;
  for (int d = 0; d < DGP_MAX_RANK; ++d) G.stride[d] = d < L.rank ? L.stride[d] : 0u;
  return G;
}

DGC LeafShape leaf_shape(const DgpLeaf& L) {
  LeafShape S;
  S.split = L.split;
  for (int d = 0; d < DGP_MAX_RANK; ++d) S.ucap[d] = d < L.rank ? L.ucap[d] : 1;
  return S;
}

// Row size (EMIT_COUNT) or row contents (EMIT_FILL, at most `room` entries
// written at ids/cnt) of one location.
template <class C, int MODE>
DGC uint64_t location_row(C& c, const uint8_t* blob, int64_t loc, uint8_t* area, uint32_t* ids, uint32_t* cnt,
                          uint64_t room, uint32_t* err) {
  const DgpHeader* h = (const DgpHeader*)blob;
  if (loc < 0 || loc >= h->out_numel) {
    *err |= DGP_ERR_RANGE;
    return 0;
  }
  const PlanLayout PL = plan_layout(h, 0);
  const EmitLayout E = emit_layout(PL.end, h->max_leaf_terms, h->union_entries, h->emit_entries);
  plan_exec(c, blob, loc, area, PL, err);
  const DgpLeaf* leaves = (const DgpLeaf*)(blob + h->leaf_off);
  TermRef* terms = (TermRef*)(area + E.terms);
  uint64_t off = 0;
  for (int l = 0; l < h->nleaf; ++l) {
    const DgpLeaf L = leaves[l];
    if (L.nterm == 0) continue;
    leaf_terms(c, blob, l, area, PL, terms);
    c.sync();
    off += leaf_pass<C, MODE>(c, leaf_geom(L), leaf_shape(L), terms, L.nterm, 0, area, E,
                               ids ? ids + off : nullptr, cnt ? cnt + off : nullptr, off < room ? room - off : 0,
                               err);
    c.sync();
  }
  return off;
}

// Per-leaf combined emission shapes of a two-graph comparison.
struct PairPlan {
  int32_t nleaf;
  int32_t max_terms;
  int32_t union_entries;
  int32_t emit_entries;
  uint32_t plan_b;  // byte offset of graph B's plan area
  uint32_t lds_bytes;
  LeafShape leaf[16];
};

template <class C>
DGC uint32_t location_compare(C& c, const uint8_t* blob_a, const uint8_t* blob_b, const PairPlan& PP, int64_t loc,
                              uint8_t* area, uint32_t* err) {
  const DgpHeader* ha = (const DgpHeader*)blob_a;
  const DgpHeader* hb = (const DgpHeader*)blob_b;
  if (loc < 0 || loc >= ha->out_numel) {
    *err |= DGP_ERR_RANGE;
    return 0;
  }
  const PlanLayout PA = plan_layout(ha, 0);
  const PlanLayout PB = plan_layout(hb, PP.plan_b);
  const EmitLayout E = emit_layout(PB.end, PP.max_terms, PP.union_entries, PP.emit_entries);
  plan_exec(c, blob_a, loc, area, PA, err);
  plan_exec(c, blob_b, loc, area, PB, err);
  const DgpLeaf* la = (const DgpLeaf*)(blob_a + ha->leaf_off);
  const DgpLeaf* lb = (const DgpLeaf*)(blob_b + hb->leaf_off);
  TermRef* terms = (TermRef*)(area + E.terms);
  uint32_t status = 0;
  for (int l = 0; l < PP.nleaf; ++l) {
    const DgpLeaf A = la[l], B = lb[l];
    if (A.nterm + B.nterm == 0) continue;
    leaf_terms(c, blob_a, l, area, PA, terms);
    leaf_terms(c, blob_b, l, area, PB, terms + A.nterm);
    c.sync();
    uint32_t s = (uint32_t)leaf_pass<C, EMIT_COMPARE>(c, leaf_geom(A), PP.leaf[l], terms, A.nterm, B.nterm, area,
                                                      E, nullptr, nullptr, 0, err);
    c.sync();
    if (s == 1) return 1;
    if (s == 2) status = 2;
  }
  return status;
}

}  // namespace dgc
