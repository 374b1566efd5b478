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
//
// Small per-thread arrays are only ever indexed with compile-time indices
// (fully unrolled loops, select chains) so they stay in registers; values
// that are the same for the whole block live in LDS.
#pragma once
#include <stdint.h>

#include "program.h"

// The including file defines DGC (device code: __device__ __forceinline__);
// plain host builds get ordinary inline functions.
#ifndef DGC
#define DGC inline
#endif

#if defined(__HIP_DEVICE_COMPILE__)
#define DG_UNROLL _Pragma("unroll")
#else
#define DG_UNROLL
#endif

// Loops whose trip counts come from the compiled plan (levels,
// instructions, leaves, terms, dims, predicates).  The kernels specialised
// for one graph see the plan as constant data and unroll them completely;
// the precompiled kernels leave them as loops.
#if defined(DG_JIT)
#define DG_PLAN_UNROLL _Pragma("unroll")
#else
#define DG_PLAN_UNROLL
#endif

namespace dgc {

// ---------------------------------------------------------------- layout --
struct PlanLayout {
  uint32_t scal, fmeta, fval, fstat, end;  // byte offsets in the block's LDS area
};

// Per factor, after the plan has run: how many of its values are nonzero
// and the largest value.
struct FStat {
  uint64_t nnz;
  uint64_t vmax;
};

// Per-leaf emission view of one separable term.
struct TermRef {
  uint64_t coef;
  int32_t lo[DGP_MAX_RANK];
  int32_t len[DGP_MAX_RANK];
  uint32_t off[DGP_MAX_RANK];  // uint64 index of the factor's values in the LDS area
  int32_t fid[DGP_MAX_RANK];   // factor of each dim
};

// Values shared by the block while one leaf is emitted.
struct LeafHdr {
  int32_t u[DGP_MAX_RANK];      // union length per dim
  int32_t uoff[DGP_MAX_RANK];   // offset of the dim's union list
  int32_t hlo[DGP_MAX_RANK];    // first coordinate of the dim's hull
  int32_t dense[DGP_MAX_RANK];  // every hull coordinate is nonzero: no list, x = hlo + i
  uint64_t cnt[DGP_MAX_RANK];   // nonzero coordinates per dim (block total)
  int32_t ok;                   // the prepared leaf has entries
  uint32_t O, In;               // outer and inner table lengths
  int32_t notab;                // cells are evaluated from the factors directly (no tables)
};

struct EmitLayout {
  uint32_t terms;   // TermRef[max_terms]
  uint32_t ulist;   // int32[union_entries]
  uint32_t tables;  // uint32[emit_entries]
  uint32_t hdr;     // LeafHdr
  uint32_t tmax;    // uint64[2 * max_terms]: per-term largest outer / inner table value
  uint32_t end;
};

DGC uint32_t align8(uint32_t x) { return (x + 7u) & ~7u; }

// Component-sum scratch at the start of the area, used by sums over more
// than two variables: the block-uniform lower bound, length and factor
// offset of each variable (3 x 8 words), then each thread's variable
// values, variable-major so that a wave reads consecutive banks.
DGC uint32_t vars_bytes(int serial_vars, int nthreads) {
  return serial_vars > 0 ? align8(4u * (uint32_t)(3 * DGP_MAX_VARS + serial_vars * nthreads)) : 0u;
}

DGC PlanLayout plan_layout(const DgpHeader* h, uint32_t base) {
  PlanLayout L;
  L.scal = align8(base);
  L.fmeta = L.scal + 8u * (uint32_t)h->nscalar;
  L.fval = L.fmeta + 8u * (uint32_t)h->nfactor;
  L.fstat = L.fval + 8u * (uint32_t)h->fval_entries;
  L.end = L.fstat + (uint32_t)sizeof(FStat) * (uint32_t)h->nfactor;
  return L;
}

// word_bytes: 4 for 32-bit ids and counts, 8 for 64-bit ones (the tables'
// words have that width).
DGC EmitLayout emit_layout(uint32_t base, int32_t max_terms, int32_t union_entries, int32_t emit_entries,
                           uint32_t word_bytes = 4) {
  EmitLayout E;
  E.terms = align8(base);
  E.ulist = E.terms + (uint32_t)sizeof(TermRef) * (uint32_t)(max_terms > 0 ? max_terms : 1);
  E.tables = (E.ulist + 4u * (uint32_t)union_entries + 15u) & ~15u;
  E.hdr = align8(E.tables + word_bytes * (uint32_t)emit_entries);
  E.tmax = E.hdr + (uint32_t)sizeof(LeafHdr);
  E.end = E.tmax + 16u * (uint32_t)(max_terms > 0 ? max_terms : 1);
  return E;
}

// A comparison's emission area starts right after graph B's live factor
// values: the values of intermediate tensors and the factor statistics
// (which a comparison never reads) are dead once both plans have run, so
// the emission area may overlay them.
DGC uint32_t compare_emit_base(const DgpHeader* hb, const PlanLayout& PB) {
  return align8(PB.fval + 8u * (uint32_t)hb->fval_live);
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

// Evaluates an index function at the calling thread's variable values
// (vt[k * nt] is variable k); false if an exact division does not divide or
// the result is outside [0, size).
DGC bool ifn_eval(const DgpIFn& f, const int32_t* vt, int nt, int32_t* out) {
  int32_t x = f.c;
  const int n = f.nterm;
  for (int q = 0; q < n; ++q) {
    int32_t vv = vt[f.var[q] * nt];
    const int32_t d = f.vdiv[q];
    if (d != 1) vv = vv / d;  // variables are non-negative
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

// Range of an index function over variables k in [vlo[k], vlo[k] + vn[k]).
DGC void ifn_range(const DgpIFn& f, const int32_t* vlo, const int32_t* vn, int32_t* lo, int32_t* hi) {
  int32_t a = f.c, b = f.c;
  const int n = f.nterm;
  for (int q = 0; q < n; ++q) {
    int32_t x0 = vlo[f.var[q]];
    int32_t x1 = x0 + vn[f.var[q]] - 1;
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
  uint64_t r;
  return __builtin_mul_overflow(a, b, &r) ? ~0ull : r;
}

// ------------------------------------------------------------ plan_exec --
// Index function of a component with at most two variables (v0, v1).
DGC bool ifn_eval2(const DgpIFn& f, int32_t v0, int32_t v1, int32_t* out) {
  int32_t x = f.c;
  const int n = f.nterm;
  DG_PLAN_UNROLL
  for (int q = 0; q < n; ++q) {
    int32_t vv = f.var[q] == 0 ? v0 : v1;
    const int32_t d = f.vdiv[q];
    if (d != 1) vv = vv / d;
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

DGC void ifn_range2(const DgpIFn& f, int32_t lo0, int32_t n0, int32_t lo1, int32_t n1, int32_t* lo, int32_t* hi) {
  int32_t a = f.c, b = f.c;
  const int n = f.nterm;
  DG_PLAN_UNROLL
  for (int q = 0; q < n; ++q) {
    int32_t x0 = f.var[q] == 0 ? lo0 : lo1;
    int32_t x1 = x0 + (f.var[q] == 0 ? n0 : n1) - 1;
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

// Variable ranges of a component with at most two variables.
struct Vars2 {
  int32_t lo0, n0, f0, lo1, n1, f1;  // f: factor value offset, -1 for a window variable
};

DGC Vars2 vars2(const DgpInstr& I, const int32_t* meta, const DgpFactor* fac) {
  Vars2 v;
  v.lo0 = 0;
  v.n0 = 1;
  v.f0 = -1;
  v.lo1 = 0;
  v.n1 = 1;
  v.f1 = -1;
  if (I.nvar >= 1) {
    const int s0 = I.var_src[0];
    if (s0 >= 0) {
      v.lo0 = meta[2 * s0];
      v.n0 = meta[2 * s0 + 1];
      v.f0 = fac[s0].off;
    } else {
      v.lo0 = I.wlo[0];
      v.n0 = I.whi[0] - I.wlo[0];
    }
  }
  if (I.nvar >= 2) {
    const int s1 = I.var_src[1];
    if (s1 >= 0) {
      v.lo1 = meta[2 * s1];
      v.n1 = meta[2 * s1 + 1];
      v.f1 = fac[s1].off;
    } else {
      v.lo1 = I.wlo[1];
      v.n1 = I.whi[1] - I.wlo[1];
    }
  }
  return v;
}

// Target range of a component sum clipped to its factor (len 0 if empty).
DGC void target_range(const DgpIFn& t, int32_t lo, int32_t hi, uint32_t P, const DgpFactor& F, int32_t* tlo,
                      int32_t* tlen, uint32_t* err) {
  if (lo < 0) lo = 0;
  if (hi > F.size - 1) hi = F.size - 1;
  int32_t len = (P == 0 || hi < lo) ? 0 : hi - lo + 1;
  if (len > F.cap) {
    *err |= DGP_ERR_CAPACITY;
    len = F.cap;
  }
  *tlo = lo;
  *tlen = len;
}

// Runs the compiled instructions of one location, level by level: phase 1
// sets up every instruction of the level (factor ranges, zeroed outputs,
// and the instructions that need no accumulation), phase 2 accumulates the
// component sums.  One barrier ends each phase.
template <class C>
DGC void plan_exec(C& c, const uint8_t* blob, int64_t loc, uint8_t* area, const PlanLayout& PL, uint32_t* err) {
  const DgpHeader* h = (const DgpHeader*)blob;
  const DgpInstr* ins = (const DgpInstr*)(blob + h->instr_off);
  const DgpFactor* fac = (const DgpFactor*)(blob + h->factor_off);
  const int32_t* level = (const int32_t*)(blob + h->level_off);
  uint64_t* scal = (uint64_t*)(area + PL.scal);
  int32_t* meta = (int32_t*)(area + PL.fmeta);
  uint64_t* fval = (uint64_t*)(area + PL.fval);
  const int tid = c.tid(), nt = c.nthreads();
  // Scratch of the sums over more than two variables.
  int32_t* vlo = (int32_t*)area;
  int32_t* vn = vlo + DGP_MAX_VARS;
  int32_t* foff = vn + DGP_MAX_VARS;
  int32_t* vt = foff + DGP_MAX_VARS + tid;
  FStat* st = (FStat*)(area + PL.fstat);
  for (int f = tid; f < h->nfactor; f += nt) {
    st[f].nnz = 0;
    st[f].vmax = 0;
  }
  const int nlevel = h->nlevel;
  DG_PLAN_UNROLL
  for (int g = 0; g < nlevel; ++g) {
    const int k0 = level[g], k1 = level[g + 1];
    // ---- phase 1
    DG_PLAN_UNROLL
    for (int k = k0; k < k1; ++k) {
      const DgpInstr& I = ins[k];
      const int op = I.opcode;
      if (op == DGP_COMP) {
        if (I.nvar <= 2) {
          const Vars2 V = vars2(I, meta, fac);
          const uint32_t P = (uint32_t)V.n0 * (uint32_t)V.n1;
          if (!I.dst_is_scalar) {
            int32_t lo, hi, tlo, tlen;
            ifn_range2(I.target, V.lo0, V.n0, V.lo1, V.n1, &lo, &hi);
            target_range(I.target, lo, hi, P, fac[I.dst], &tlo, &tlen, err);
            if (tid == 0) {
              meta[2 * I.dst] = tlo;
              meta[2 * I.dst + 1] = tlen;
            }
            uint64_t* dv = fval + fac[I.dst].off;
            for (int i = tid; i < tlen; i += nt) dv[i] = 0;
          } else if (tid == 0) {
            scal[I.dst] = 0;
          }
        } else if (tid == 0) {
          // Serial level: publish the variable ranges and the target range.
          uint32_t P = 1;
          for (int q = 0; q < I.nvar; ++q) {
            const int src = I.var_src[q];
            if (src >= 0) {
              vlo[q] = meta[2 * src];
              vn[q] = meta[2 * src + 1];
              foff[q] = fac[src].off;
            } else {
              vlo[q] = I.wlo[q];
              vn[q] = I.whi[q] - I.wlo[q];
              foff[q] = -1;
            }
            P *= (uint32_t)vn[q];
          }
          if (!I.dst_is_scalar) {
            int32_t lo, hi, tlo, tlen;
            ifn_range(I.target, vlo, vn, &lo, &hi);
            target_range(I.target, lo, hi, P, fac[I.dst], &tlo, &tlen, err);
            meta[2 * I.dst] = tlo;
            meta[2 * I.dst + 1] = tlen;
          } else {
            scal[I.dst] = 0;
          }
        }
      } else if (op == DGP_PATTERN) {
        const int32_t r = I.a >= 0 ? (int32_t)((loc / h->out_stride[I.a]) % h->out_shape[I.a]) : 0;
        const DgpFactor F = fac[I.dst];
        int32_t lo = I.pkind == 0 ? r + I.pmin : I.pmin, hi = I.pkind == 0 ? r + I.pmax : I.pmax;
        if (lo < 0) lo = 0;
        if (hi > F.size) hi = F.size;
        int32_t len = hi > lo ? hi - lo : 0;
        if (len > F.cap) {
          *err |= DGP_ERR_CAPACITY;
          len = F.cap;
        }
        if (tid == 0) {
          meta[2 * I.dst] = lo;
          meta[2 * I.dst + 1] = len;
        }
        uint64_t* dv = fval + F.off;
        for (int i = tid; i < len; i += nt) {
          const int32_t x = lo + i;
          uint64_t v = 0;
          DG_PLAN_UNROLL
          for (int e = 0; e < I.npat; ++e) {
            const int32_t* P = I.pat[e];
            const bool on = I.pkind == 0 ? (x >= r + P[0] && x < r + P[1]) : (x == P[0] && r >= P[1] && r < P[2]);
            if (on) v += (uint32_t)P[3];
          }
          dv[i] = v;
        }
      } else if (op == DGP_ROOT || op == DGP_CONST) {
        if (tid == 0) {
          int32_t x;
          if (op == DGP_ROOT) x = (int32_t)((loc / h->out_stride[I.a]) % h->out_shape[I.a]);
          else x = I.a;
          meta[2 * I.dst] = x;
          meta[2 * I.dst + 1] = 1;
          fval[fac[I.dst].off] = 1;
        }
      } else if (op == DGP_LINCOMB) {
        const int32_t lo1 = meta[2 * I.f1], n1 = meta[2 * I.f1 + 1];
        const int32_t lo2 = meta[2 * I.f2], n2 = meta[2 * I.f2 + 1];
        const uint64_t k1s = (I.k1 < 0 ? 1ull : scal[I.k1]) * I.c1;
        const uint64_t k2s = (I.k2 < 0 ? 1ull : scal[I.k2]) * I.c2;
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
          const int32_t x = lo + i;
          uint64_t sum = 0;
          if (x - lo1 >= 0 && x - lo1 < n1) sum += k1s * a1[x - lo1];
          if (x - lo2 >= 0 && x - lo2 < n2) sum += k2s * a2[x - lo2];
          dv[i] = sum;
        }
      } else if (op == DGP_SMUL) {
        if (tid == 0) {
          uint64_t v = I.cst;
          DG_PLAN_UNROLL
          for (int q = 0; q < I.ns; ++q) v *= scal[I.s[q]];
          scal[I.dst] = v;
        }
      } else if (op == DGP_SADD) {
        if (tid == 0) {
          const uint64_t a = (I.f1 < 0 ? 1ull : scal[I.f1]) * I.c1;
          const uint64_t b = (I.f2 < 0 ? 1ull : scal[I.f2]) * I.c2;
          scal[I.dst] = a + b;
        }
      }
    }
    c.sync();
    // ---- phase 2
    DG_PLAN_UNROLL
    for (int k = k0; k < k1; ++k) {
      const DgpInstr& I = ins[k];
      if (I.opcode != DGP_COMP) continue;
      const bool to_factor = !I.dst_is_scalar;
      const int npred = I.npred;
      uint64_t* dv = to_factor ? fval + fac[I.dst].off : nullptr;
      int32_t tlo = 0, tlen = 0;
      if (to_factor) {
        tlo = meta[2 * I.dst];
        tlen = meta[2 * I.dst + 1];
      }
      uint64_t acc = 0;
      if (I.nvar <= 2) {
        const Vars2 V = vars2(I, meta, fac);
        const uint32_t n1 = (uint32_t)V.n1;
        const uint32_t P = (uint32_t)V.n0 * n1;
        for (uint32_t p = (uint32_t)tid; p < P; p += (uint32_t)nt) {
          const uint32_t i0 = n1 == 1 ? p : p / n1;
          const uint32_t i1 = p - i0 * n1;
          const int32_t v0 = V.lo0 + (int32_t)i0, v1 = V.lo1 + (int32_t)i1;
          uint64_t w = 1;
          if (V.f0 >= 0) w = fval[V.f0 + (int32_t)i0];
          if (V.f1 >= 0) w *= fval[V.f1 + (int32_t)i1];
          if (w == 0) continue;
          bool ok = true;
          DG_PLAN_UNROLL
          for (int e = 0; e < npred; ++e) {
            int32_t t;
            ok = ok && ifn_eval2(I.pred[e], v0, v1, &t);
          }
          if (!ok) continue;
          if (to_factor) {
            int32_t t;
            if (!ifn_eval2(I.target, v0, v1, &t) || t < tlo || t >= tlo + tlen) continue;
            c.atomic_add(&dv[t - tlo], w);
          } else {
            acc += w;
          }
        }
      } else {
        // Serial level (the only instruction): zero the target, then sum.
        const int nv = I.nvar;
        if (to_factor)
          for (int i = tid; i < tlen; i += nt) dv[i] = 0;
        c.sync();
        uint32_t P = 1;
        for (int q = 0; q < nv; ++q) P *= (uint32_t)vn[q];
        for (uint32_t p = (uint32_t)tid; p < P; p += (uint32_t)nt) {
          uint32_t rem = p;
          uint64_t w = 1;
          for (int q = nv - 1; q >= 0; --q) {
            const uint32_t n = (uint32_t)vn[q];
            const uint32_t r = rem % n;
            rem /= n;
            vt[q * nt] = vlo[q] + (int32_t)r;
            const int32_t fo = foff[q];
            if (fo >= 0) w *= fval[fo + (int32_t)r];
          }
          if (w == 0) continue;
          bool ok = true;
          for (int e = 0; e < npred && ok; ++e) {
            int32_t t;
            ok = ifn_eval(I.pred[e], vt, nt, &t);
          }
          if (!ok) continue;
          if (to_factor) {
            int32_t t;
            if (!ifn_eval(I.target, vt, nt, &t) || t < tlo || t >= tlo + tlen) continue;
            c.atomic_add(&dv[t - tlo], w);
          } else {
            acc += w;
          }
        }
      }
      if (!to_factor) c.reduce_add(&scal[I.dst], acc);
    }
    c.sync();
  }
}

// Nonzero count and largest value of the factors used by single-term leaves
// (after plan_exec, whose last barrier also published the zeroed
// statistics).  A single-term leaf is the outer product of its factors, so
// these give its entry count and its largest path count without touching
// the leaf.
template <class C>
DGC void factor_stats(C& c, const uint8_t* blob, uint8_t* area, const PlanLayout& PL) {
  const DgpHeader* h = (const DgpHeader*)blob;
  const DgpFactor* fac = (const DgpFactor*)(blob + h->factor_off);
  const int32_t* meta = (const int32_t*)(area + PL.fmeta);
  const uint64_t* fval = (const uint64_t*)(area + PL.fval);
  FStat* st = (FStat*)(area + PL.fstat);
  const int tid = c.tid(), nt = c.nthreads();
  const int nf = h->nfactor;
  // Factors of at most 64 values are taken by one wave each, in turn.
  const int nwave = nt >= 64 ? nt / 64 : 1;
  const int wave = nt >= 64 ? tid / 64 : 0;
  int small = 0;
  DG_PLAN_UNROLL
  for (int f = 0; f < nf; ++f) {
    if (!fac[f].stat) continue;
    int32_t x0 = tid, step = nt;
    if (nt >= 64 && fac[f].cap <= 64) {
      if (small++ % nwave != wave) continue;
      x0 = tid & 63;
      step = 64;
    }
    const int32_t len = meta[2 * f + 1];
    const uint64_t* v = fval + fac[f].off;
    uint64_t cnt = 0, mx = 0;
    for (int32_t x = x0; x < len; x += step) {
      const uint64_t a = v[x];
      cnt += a != 0 ? 1u : 0u;
      mx = a > mx ? a : mx;
    }
    c.reduce_add(&st[f].nnz, cnt);
    if (!h->no_overflow) c.reduce_max(&st[f].vmax, mx);
  }
  c.sync();
}

// Fills TermRef[0 .. nterm) for leaf `leaf` of a plan.
template <class C>
DGC void leaf_terms(C& c, const uint8_t* blob, int leaf, uint8_t* area, const PlanLayout& PL, TermRef* out) {
  const DgpHeader* h = (const DgpHeader*)blob;
  const DgpLeaf* L = (const DgpLeaf*)(blob + h->leaf_off) + leaf;
  const DgpTerm* T = (const DgpTerm*)(blob + h->term_off) + L->term0;
  const DgpFactor* fac = (const DgpFactor*)(blob + h->factor_off);
  const uint64_t* scal = (const uint64_t*)(area + PL.scal);
  const int32_t* meta = (const int32_t*)(area + PL.fmeta);
  const int rank = L->rank;
  for (int t = c.tid(); t < L->nterm; t += c.nthreads()) {
    TermRef* r = out + t;
    r->coef = (T[t].coef_slot < 0 ? 1ull : scal[T[t].coef_slot]) * T[t].coef_const;
    DG_PLAN_UNROLL
    for (int d = 0; d < rank; ++d) {
      const int f = T[t].factor[d];
      r->lo[d] = meta[2 * f];
      r->len[d] = meta[2 * f + 1];
      r->off[d] = (PL.fval >> 3) + (uint32_t)fac[f].off;
      r->fid[d] = f;
    }
  }
}

DGC uint64_t term_val(const TermRef& r, int d, int32_t x, const uint64_t* area64) {
  const int32_t i = x - r.lo[d];
  return (i >= 0 && i < r.len[d]) ? area64[r.off[d] + (uint32_t)i] : 0ull;
}

// Hull [lo, hi) of dim d over the terms' ranges (hi <= lo if all empty).
DGC void term_hull(const TermRef* terms, int nterm, int d, int32_t* lo, int32_t* hi) {
  int32_t a = 0x7fffffff, b = -0x7fffffff;
  DG_PLAN_UNROLL
  for (int t = 0; t < nterm; ++t) {
    const int32_t l = terms[t].lo[d], n = terms[t].len[d];
    if (n <= 0) continue;
    if (l < a) a = l;
    if (l + n > b) b = l + n;
  }
  *lo = a;
  *hi = b;
}

// Per dim, the union of the terms' nonzero coordinates: its size, whether it
// is the whole hull (dense: coordinate i of the union is hlo + i) and, for
// the other dims when `lists` is set, the sorted coordinates in `ulist`.
// Returns false (leaf empty) if some dim has no nonzero coordinate.
//
// With `st` (a single term), the factor statistics give the counts and the
// counting pass is skipped.
template <class C>
DGC bool build_union(C& c, const TermRef* terms, int nterm, int rank, const int32_t* ucap, int32_t* ulist,
                     LeafHdr* H, bool lists, uint8_t* area, const FStat* st, uint32_t* err) {
  const uint64_t* a64 = (const uint64_t*)area;
  const int tid = c.tid(), nt = c.nthreads();
  if (!st) {
    for (int i = tid; i < DGP_MAX_RANK; i += nt) H->cnt[i] = 0;
    c.sync();
    // Counts: one pass over every dim, one barrier.
    DG_PLAN_UNROLL
    for (int d = 0; d < rank; ++d) {
      int32_t hlo, hhi;
      term_hull(terms, nterm, d, &hlo, &hhi);
      uint64_t cnt = 0;
      for (int32_t x = hlo + tid; x < hhi; x += nt) {
        bool nz = false;
        DG_PLAN_UNROLL
        for (int t = 0; t < nterm; ++t) nz = nz || term_val(terms[t], d, x, a64) != 0;
        cnt += nz ? 1u : 0u;
      }
      c.reduce_add(&H->cnt[d], cnt);
    }
    c.sync();
  }
  bool empty = false;
  int32_t base_off = 0;
  DG_PLAN_UNROLL
  for (int d = 0; d < rank; ++d) {
    int32_t hlo, hhi;
    term_hull(terms, nterm, d, &hlo, &hhi);
    int32_t count = st ? (int32_t)st[terms[0].fid[d]].nnz : (int32_t)H->cnt[d];
    const bool dense = count > 0 && count == hhi - hlo;
    const int32_t cap = ucap[d];
    if (!dense && count > cap) {
      *err |= DGP_ERR_CAPACITY;
      count = cap;
    }
    if (tid == 0) {
      H->u[d] = count;
      H->uoff[d] = base_off;
      H->hlo[d] = hlo;
      H->dense[d] = dense ? 1 : 0;
    }
    if (count == 0) empty = true;
    if (lists && !dense && count > 0) {
      // Ordered compaction of the nonzero coordinates.
      int32_t* ul = ulist + base_off;
      int32_t done = 0;
      for (int32_t chunk = hlo; chunk < hhi; chunk += nt) {
        const int32_t x = chunk + tid;
        bool nz = false;
        if (x < hhi)
          for (int t = 0; t < nterm && !nz; ++t) nz = term_val(terms[t], d, x, a64) != 0;
        uint32_t tot;
        const uint32_t pre = c.prefix(nz, &tot);
        if (nz && done + (int32_t)pre < cap) ul[done + (int32_t)pre] = x;
        done += (int32_t)tot;
      }
    }
    base_off += cap;
  }
  c.sync();
  return !empty;
}

// Coordinate of union entry i of dim d.
DGC int32_t ucoord(const LeafHdr* H, const int32_t* ulist, int d, int32_t i) {
  return H->dense[d] ? H->hlo[d] + i : ulist[H->uoff[d] + i];
}

// Mode of a leaf pass.
enum { EMIT_COUNT = 0, EMIT_FILL = 1, EMIT_COMPARE = 2 };

struct LeafGeom {
  int32_t rank;
  uint64_t base;
  uint64_t stride[DGP_MAX_RANK];
};

// Width of the emitted ids and counts (and of the emission tables' words):
// uint32_t, or uint64_t for outputs whose ids or counts need 64 bits.
template <class Word>
DGC Word to_word(uint64_t v) {
  return sizeof(Word) == 4 ? (Word)(v > 0xFFFFFFFFull ? 0xFFFFFFFFull : v) : (Word)v;
}

// q = n / d and *rem = n % d for n < 2^20, d >= 1.  On the device a float
// reciprocal gives a quotient within one of the exact one (relative error
// below 2^-21, so an absolute error below 1/2 for these n), which one
// correction step fixes; the host divides.
DGC uint32_t table_divmod(uint32_t n, uint32_t d, uint32_t* rem) {
#if defined(__HIP_DEVICE_COMPILE__)
  uint32_t q = (uint32_t)((float)n * __builtin_amdgcn_rcpf((float)d));
  int32_t r = (int32_t)n - (int32_t)(q * d);
  if (r < 0) {
    --q;
    r += (int32_t)d;
  } else if (r >= (int32_t)d) {
    ++q;
    r -= (int32_t)d;
  }
  *rem = (uint32_t)r;
  return q;
#else
  *rem = n % d;
  return n / d;
#endif
}

// Builds one table: entries r < n over dims [d0, d1); entry = (id part,
// count part of every term).  With `tmax`, records each term's largest
// value there (per-thread maxima, combined once per wave and term).
template <class C, class Word>
DGC void build_table(C& c, const LeafGeom& G, const TermRef* terms, int nterm, const int32_t* ulist,
                     const LeafHdr* H, int d0, int d1, bool with_base, uint32_t n, Word* tab, uint64_t* tmax,
                     const uint64_t* a64, bool narrow = false) {
  const int W = 1 + nterm;
  int32_t u[DGP_MAX_RANK];
  DG_UNROLL
  for (int d = 0; d < DGP_MAX_RANK; ++d) u[d] = H->u[d];
  // Coordinates of entry r (row-major over the union lists of [d0, d1);
  // tables hold at most 8192 entries).
  auto coords = [&](uint32_t r, int32_t* x) {
    uint32_t rem = r;
    DG_UNROLL
    for (int d = DGP_MAX_RANK - 1; d >= 0; --d) {
      x[d] = 0;
      if (d >= d0 && d < d1) {
        uint32_t i;
        rem = table_divmod(rem, (uint32_t)u[d], &i);
        x[d] = ucoord(H, ulist, d, (int32_t)i);
      }
    }
  };
  if (nterm == 1) {
    // One pass: id part and count part together.
    uint64_t m = 0;
    for (uint32_t r = (uint32_t)c.tid(); r < n; r += (uint32_t)c.nthreads()) {
      int32_t x[DGP_MAX_RANK];
      coords(r, x);
      uint64_t pos = with_base ? G.base : 0u;
      uint64_t v = with_base ? terms[0].coef : 1ull;
      DG_UNROLL
      for (int d = 0; d < DGP_MAX_RANK; ++d)
        if (d >= d0 && d < d1) {
          pos += (uint64_t)x[d] * G.stride[d];
          if (v) v = mul_sat(v, term_val(terms[0], d, x[d], a64));
        }
      tab[2 * (uint64_t)r] = (Word)pos;
      tab[2 * (uint64_t)r + 1] = to_word<Word>(v);
      m = v > m ? v : m;
    }
    if (tmax) c.reduce_max(&tmax[0], m);
    return;
  }
  if (!tmax) {
    // Several terms and no maxima to record: one pass, each entry's
    // coordinates decoded once for all terms.
    for (uint32_t r = (uint32_t)c.tid(); r < n; r += (uint32_t)c.nthreads()) {
      int32_t x[DGP_MAX_RANK];
      coords(r, x);
      uint64_t pos = with_base ? G.base : 0u;
      DG_UNROLL
      for (int d = 0; d < DGP_MAX_RANK; ++d)
        if (d >= d0 && d < d1) pos += (uint64_t)x[d] * G.stride[d];
      tab[(uint64_t)r * W] = (Word)pos;
      DG_PLAN_UNROLL
      for (int t = 0; t < nterm; ++t) {
        if (narrow) {
          // Every path count is below 2^32 (static bound).  A part of a
          // term that is nonzero somewhere is at most a real count, so 32
          // bits hold it; a part that is never nonzero multiplies only
          // zeros, whatever its bits.
          uint32_t v = with_base ? (uint32_t)terms[t].coef : 1u;
          DG_UNROLL
          for (int d = 0; d < DGP_MAX_RANK; ++d)
            if (d >= d0 && d < d1) v *= (uint32_t)term_val(terms[t], d, x[d], a64);
          tab[(uint64_t)r * W + 1 + t] = (Word)v;
          continue;
        }
        uint64_t v = with_base ? terms[t].coef : 1ull;
        DG_UNROLL
        for (int d = 0; d < DGP_MAX_RANK; ++d)
          if (d >= d0 && d < d1 && v) v = mul_sat(v, term_val(terms[t], d, x[d], a64));
        tab[(uint64_t)r * W + 1 + t] = to_word<Word>(v);
      }
    }
    return;
  }
  for (uint32_t r = (uint32_t)c.tid(); r < n; r += (uint32_t)c.nthreads()) {
    int32_t x[DGP_MAX_RANK];
    coords(r, x);
    uint64_t pos = with_base ? G.base : 0u;
    DG_UNROLL
    for (int d = 0; d < DGP_MAX_RANK; ++d)
      if (d >= d0 && d < d1) pos += (uint64_t)x[d] * G.stride[d];
    tab[(uint64_t)r * W] = (Word)pos;
  }
  DG_PLAN_UNROLL
  for (int t = 0; t < nterm; ++t) {
    uint64_t m = 0;
    for (uint32_t r = (uint32_t)c.tid(); r < n; r += (uint32_t)c.nthreads()) {
      int32_t x[DGP_MAX_RANK];
      coords(r, x);
      uint64_t v = with_base ? terms[t].coef : 1ull;
      DG_UNROLL
      for (int d = 0; d < DGP_MAX_RANK; ++d)
        if (d >= d0 && d < d1 && v) v = mul_sat(v, term_val(terms[t], d, x[d], a64));
      tab[(uint64_t)r * W + 1 + t] = to_word<Word>(v);
      m = v > m ? v : m;
    }
    if (tmax) c.reduce_max(&tmax[t], m);
  }
}

DGC bool prod_overflows(uint64_t a, uint64_t b) {
  return a && b && (a > 0xFFFFFFFFull || b > 0xFFFFFFFFull || a * b > 0xFFFFFFFFull);
}

// Prepares one leaf of one location for emission (block `w`).  Terms [0, na) belong to graph A (the graph being enumerated),
// terms [na, na + nb) to graph B (compare only).  Forms the union of the
// terms' nonzero coordinates and, with a split, the outer and inner tables,
// and publishes in the leaf header: ok (0 when the leaf has no entry), the
// union lengths, and the table lengths O and In.
template <class W, int MODE, class Word = uint32_t>
DGC void leaf_prepare(W& w, const LeafGeom& G, int split, const int32_t* ucap, const TermRef* terms, int na, int nb,
                      uint8_t* area, const EmitLayout& E, const FStat* st, bool checks, uint32_t* err,
                      bool narrow = false) {
  const int tid = w.tid(), nt = w.nthreads();
  const int nterm = na + nb;
  const int rank = G.rank;
  int32_t* ulist = (int32_t*)(area + E.ulist);
  LeafHdr* H = (LeafHdr*)(area + E.hdr);
  const uint64_t* a64 = (const uint64_t*)area;
  const bool single = MODE != EMIT_COMPARE && nterm == 1;
  bool ok = nterm > 0 && !(MODE != EMIT_COMPARE && na == 0);
  // A single term with a zero coefficient is identically zero.
  if (ok && single && terms[0].coef == 0) ok = false;
  bool hull = false;
  if (ok && MODE == EMIT_COMPARE) {
    // A comparison needs no ordered union: it evaluates both graphs on the
    // hull grid of all terms (cells outside every support are zero on both
    // sides), as long as each hull fits the union's capacity.
    bool fits = true, empty = false;
    int32_t hlo[DGP_MAX_RANK], hhi[DGP_MAX_RANK];
    DG_UNROLL
    for (int d = 0; d < DGP_MAX_RANK; ++d) {
      hlo[d] = 0;
      hhi[d] = 1;
      if (d < rank) {
        term_hull(terms, nterm, d, &hlo[d], &hhi[d]);
        if (hhi[d] <= hlo[d]) empty = true;
        else if (hhi[d] - hlo[d] > ucap[d]) fits = false;
      }
    }
    if (empty) {
      ok = false;
      hull = true;
    } else if (fits) {
      if (tid == 0) {
        DG_UNROLL
        for (int d = 0; d < DGP_MAX_RANK; ++d)
          if (d < rank) {
            H->u[d] = hhi[d] - hlo[d];
            H->hlo[d] = hlo[d];
            H->dense[d] = 1;
          }
      }
      w.sync();
      hull = true;
    }
  }
  // A single term's per-dim counts are the factor statistics.
  if (ok && !hull) ok = build_union(w, terms, nterm, rank, ucap, ulist, H, true, area, single ? st : nullptr, err);
  // A comparison grid that one pass of the block covers is evaluated from
  // the factors directly: tables would cost more than they save.
  bool notab = split < 0;
  if (ok && MODE == EMIT_COMPARE && hull) {
    uint64_t cells = 1;
    DG_PLAN_UNROLL
    for (int d = 0; d < rank; ++d) cells *= (uint64_t)H->u[d];
    if (cells <= (uint64_t)nt) notab = true;
  }
  uint32_t O = 1, In = 1;
  if (ok && !notab) {
    // Outer table over dims [0, split), inner over [split, rank).
    int32_t u[DGP_MAX_RANK];
    DG_UNROLL
    for (int d = 0; d < DGP_MAX_RANK; ++d) u[d] = d < rank ? H->u[d] : 1;
    DG_UNROLL
    for (int d = 0; d < DGP_MAX_RANK; ++d) {
      if (d < split) O *= (uint32_t)u[d];
      else if (d < rank) In *= (uint32_t)u[d];
    }
    const int Wd = 1 + nterm;
    Word* otab = (Word*)(area + E.tables);
    Word* itab = otab + (uint64_t)O * Wd;
    uint64_t* tmax = checks ? (uint64_t*)(area + E.tmax) : nullptr;
    if (checks) {
      for (int i = tid; i < 2 * nterm; i += nt) tmax[i] = 0;
      w.sync();
    }
    build_table(w, G, terms, nterm, ulist, H, 0, split, true, O, otab, tmax, a64, narrow);
    build_table(w, G, terms, nterm, ulist, H, split, rank, false, In, itab, checks ? tmax + nterm : nullptr, a64,
                narrow);
    w.sync();
    // A term whose largest outer and inner parts multiply past 32 bits has a
    // real cell with that count.
    if (checks)
      for (int t = tid; t < nterm; t += nt)
        if (prod_overflows(tmax[t], tmax[nterm + t])) *err |= DGP_ERR_OVERFLOW;
  }
  if (tid == 0) {
    H->ok = ok ? 1 : 0;
    H->O = O;
    H->In = In;
    H->notab = notab ? 1 : 0;
  }
}

// Entry r of a single-term table: (id part, count part), one aligned
// 8-byte (narrow) or 16-byte (wide) pair.
DGC void pair_at(const uint32_t* tab, uint32_t r, uint32_t* id, uint32_t* cnt) {
  const uint64_t v = ((const uint64_t*)tab)[r];
  *id = (uint32_t)v;
  *cnt = (uint32_t)(v >> 32);
}
DGC void pair_at(const uint64_t* tab, uint32_t r, uint64_t* id, uint64_t* cnt) {
  struct alignas(16) P2 {
    uint64_t a, b;
  };
  const P2 v = ((const P2*)tab)[r];
  *id = v.a;
  *cnt = v.b;
}

// Emits one prepared leaf (block `c`).
//   EMIT_COUNT:   returns the number of nonzero entries.
//   EMIT_FILL:    writes them at ids/cnt and returns their number.
//   EMIT_COMPARE: returns 0 equal, 1 nonzero sets differ, 2 counts differ.
//   `room` bounds the entries EMIT_FILL may write at ids/cnt; a leaf that
//   would need more raises DGP_ERR_SIZE and writes nothing past it.
template <class C, int MODE, class Word = uint32_t>
DGC uint64_t leaf_emit(C& c, const LeafGeom& G, int split, const TermRef* terms, int na, int nb, uint8_t* area,
                       const EmitLayout& E, Word* ids, Word* cnt, uint64_t room, uint32_t* err,
                       bool narrow = false) {
  const int tid = c.tid(), nt = c.nthreads();
  const int nterm = na + nb;
  const int rank = G.rank;
  const int32_t* ulist = (const int32_t*)(area + E.ulist);
  const LeafHdr* H = (const LeafHdr*)(area + E.hdr);
  const uint64_t* a64 = (const uint64_t*)area;
  if (!H->ok) return 0;
  int32_t u[DGP_MAX_RANK];
  DG_UNROLL
  for (int d = 0; d < DGP_MAX_RANK; ++d) u[d] = d < rank ? H->u[d] : 1;

  if (!H->notab) {
    const int W = 1 + nterm;
    const uint32_t O = H->O, In = H->In;
    const Word* otab = (const Word*)(area + E.tables);
    const Word* itab = otab + (uint64_t)O * W;
    const uint64_t total = (uint64_t)O * In;
    if (MODE == EMIT_FILL && nterm == 1) {
      // Dense single-term grid: every cell is an entry, in order.  Lanes are
      // shifted so that each wave's stores cover whole aligned blocks of 64
      // words of the id array (256 bytes, or 512 with 64-bit words): rows
      // start anywhere, and unaligned wave stores halve the write rate.
      if (total > room) *err |= DGP_ERR_SIZE;
      const int64_t tot = (int64_t)(total < room ? total : room);
      // (Shift by the entries that precede ids in its 64-word block; the
      // shift stays below the block width, so p + step >= 0 below.)
      const int64_t head = nt >= 64 ? (int64_t)((((uintptr_t)ids) / sizeof(Word)) & 63u) : 0;
      const int64_t step = nt;
      int64_t p = (int64_t)tid - head;
      // (Single-term entries are aligned (id part, count part) pairs, read
      // as one 64- or 128-bit LDS access each, which keeps a wave's reads
      // free of bank conflicts.)
      if (p >= 0 && p < tot) {
        const uint32_t r = (uint32_t)(p / In), j = (uint32_t)(p % In);
        Word oi, oc, qi, qc;
        pair_at(otab, r, &oi, &oc);
        pair_at(itab, j, &qi, &qc);
        c.store(&ids[p], (Word)(oi + qi));
        c.store(&cnt[p], (Word)(oc * qc));
      }
      p += step;
      if (p < tot) {
        uint32_t r = (uint32_t)(p / In), j = (uint32_t)(p % In);
        const uint32_t dr = (uint32_t)(step / In), dj = (uint32_t)(step % In);
        for (; p < tot; p += step) {
          Word oi, oc, qi, qc;
          pair_at(otab, r, &oi, &oc);
          pair_at(itab, j, &qi, &qc);
          c.store(&ids[p], (Word)(oi + qi));
          c.store(&cnt[p], (Word)(oc * qc));
          j += dj;
          r += dr;
          if (j >= In) {
            j -= In;
            ++r;
          }
        }
      }
      return total;
    }
    // Several terms: evaluate each cell, keep the nonzero ones in order.
    // Cell p is (outer r, inner j) = (p / In, p % In); (r, j) advances by
    // the block's width each chunk.  (Tables hold fewer than 2^32 cells, so
    // cell indices fit 32 bits.)
    uint64_t written = 0;
    uint32_t flags = 0;
    uint32_t r = (uint32_t)tid / In, j = (uint32_t)tid % In;
    const uint32_t dr = (uint32_t)nt / In, dj = (uint32_t)nt % In;
    for (uint64_t chunk = 0; chunk < total; chunk += (uint64_t)nt) {
      const uint64_t p = chunk + (uint64_t)tid;
      uint64_t ca = 0, cb = 0;
      Word pos = 0;
      if (p < total) {
        const Word* o = otab + (uint64_t)r * W;
        const Word* q = itab + (uint64_t)j * W;
        pos = o[0] + q[0];
        if (narrow) {
          // (Counts below 2^32: each nonzero product and each sum is at
          // most a real count.)
          uint32_t a = 0, b = 0;
          DG_PLAN_UNROLL
          for (int t = 0; t < na; ++t) a += (uint32_t)o[1 + t] * (uint32_t)q[1 + t];
          DG_PLAN_UNROLL
          for (int t = na; t < nterm; ++t) b += (uint32_t)o[1 + t] * (uint32_t)q[1 + t];
          ca = a;
          cb = b;
        } else {
          DG_PLAN_UNROLL
          for (int t = 0; t < na; ++t) ca += (uint64_t)o[1 + t] * q[1 + t];
          DG_PLAN_UNROLL
          for (int t = na; t < nterm; ++t) cb += (uint64_t)o[1 + t] * q[1 + t];
        }
      }
      j += dj;
      r += dr;
      if (j >= In) {
        j -= In;
        ++r;
      }
      if (MODE == EMIT_COMPARE) {
        if ((ca == 0) != (cb == 0)) flags |= 1u;
        else if (ca != cb) flags |= 2u;
        if (c.any((flags & 1u) != 0)) return 1;
      } else {
        if (sizeof(Word) == 4 && ca > 0xFFFFFFFFull) *err |= DGP_ERR_OVERFLOW;
        const bool nz = ca != 0;
        uint32_t tot;
        const uint32_t pre = c.prefix(nz, &tot);
        if (MODE == EMIT_FILL && nz) {
          if (written + pre < room) {
            c.store(&ids[written + pre], pos);
            c.store(&cnt[written + pre], (Word)ca);
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
  DG_UNROLL
  for (int d = 0; d < DGP_MAX_RANK; ++d) total *= (uint64_t)u[d];
  uint64_t written = 0;
  uint32_t flags = 0;
  for (uint64_t chunk = 0; chunk < total; chunk += (uint64_t)nt) {
    const uint64_t p = chunk + (uint64_t)tid;
    uint64_t ca = 0, cb = 0;
    uint64_t pos = G.base;
    if (p < total) {
      int32_t x[DGP_MAX_RANK];
      uint32_t rem = (uint32_t)p;  // (fewer than 2^32 cells)
      DG_UNROLL
      for (int d = DGP_MAX_RANK - 1; d >= 0; --d) {
        x[d] = 0;
        if (d < rank) {
          const uint32_t i = rem % (uint32_t)u[d];
          rem /= (uint32_t)u[d];
          x[d] = ucoord(H, ulist, d, (int32_t)i);
          pos += (uint64_t)x[d] * G.stride[d];
        }
      }
      DG_PLAN_UNROLL
      for (int t = 0; t < nterm; ++t) {
        uint64_t v = terms[t].coef;
        DG_UNROLL
        for (int d = 0; d < DGP_MAX_RANK; ++d)
          if (d < rank && v) v = mul_sat(v, term_val(terms[t], d, x[d], a64));
        if (t < na) ca = (ca + v < ca) ? ~0ull : ca + v;
        else cb = (cb + v < cb) ? ~0ull : cb + v;
      }
    }
    if (MODE == EMIT_COMPARE) {
      if ((ca == 0) != (cb == 0)) flags |= 1u;
      else if (ca != cb) flags |= 2u;
      if (c.any((flags & 1u) != 0)) return 1;
    } else {
      if (sizeof(Word) == 4 && ca > 0xFFFFFFFFull) *err |= DGP_ERR_OVERFLOW;
      const bool nz = ca != 0;
      uint32_t tot;
      const uint32_t pre = c.prefix(nz, &tot);
      if (MODE == EMIT_FILL && nz) {
        if (written + pre < room) {
          c.store(&ids[written + pre], (Word)pos);
          c.store(&cnt[written + pre], (Word)ca);
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
  DG_UNROLL
  for (int d = 0; d < DGP_MAX_RANK; ++d) G.stride[d] = d < L.rank ? L.stride[d] : 0u;
  return G;
}

// ---------------------------------------------------------------- drivers --
// Where the locations of a launch come from: an explicit list, or (list
// null) the contiguous flat range first, first + 1, ...
struct LocSrc {
  const int64_t* locs;
  int64_t first;
};
DGC int64_t loc_at(const LocSrc& s, int64_t i) { return s.locs ? s.locs[i] : s.first + i; }

DGC bool location_in_range(const uint8_t* blob, int64_t loc) {
  const DgpHeader* h = (const DgpHeader*)blob;
  return loc >= 0 && loc < h->out_numel;
}

// Runs the plan of one (in-range) location and the factor statistics.
template <class C>
DGC void location_plan(C& c, const uint8_t* blob, int64_t loc, uint8_t* area, uint32_t* err) {
  const DgpHeader* h = (const DgpHeader*)blob;
  const PlanLayout PL = plan_layout(h, vars_bytes(h->serial_vars, c.nthreads()));
  plan_exec(c, blob, loc, area, PL, err);
  factor_stats(c, blob, area, PL);
}

// Where a row goes: the emission calls `place` once, right before it writes
// the row's first entry (or at the end if the row has none), after the
// first leaf to emit has been prepared.  It returns the row's offset in
// ids/cnt and whether the row may be written.  The single-pass kernel finds
// its offset there, so that the wait for its predecessors overlaps the
// preparation of its first leaf.
struct PlaceAt {
  uint64_t off;
  template <class C>
  DGC uint64_t operator()(C&, bool* go) const {
    *go = true;
    return off;
  }
};

// Leaf passes over a plan already in LDS (the block has synchronised since
// the plan): the row size (EMIT_COUNT) or the row itself (EMIT_FILL, at most
// `room` entries written at ids/cnt + place()).
template <class C, int MODE, class Place, class Word = uint32_t>
DGC uint64_t location_leaves(C& c, const uint8_t* blob, uint8_t* area, Word* ids, Word* cnt, uint64_t room,
                             uint32_t* err, Place& place) {
  const DgpHeader* h = (const DgpHeader*)blob;
  const PlanLayout PL = plan_layout(h, vars_bytes(h->serial_vars, c.nthreads()));
  const EmitLayout E = emit_layout(PL.end, h->max_leaf_terms, h->union_entries, h->emit_entries, sizeof(Word));
  // 64-bit counts cannot overflow: the static bound is below 2^63.
  const bool checks = sizeof(Word) == 4 && !h->no_overflow;
  const DgpLeaf* leaves = (const DgpLeaf*)(blob + h->leaf_off);
  const DgpTerm* T0 = (const DgpTerm*)(blob + h->term_off);
  const uint64_t* scal = (const uint64_t*)(area + PL.scal);
  const FStat* st = (const FStat*)(area + PL.fstat);
  TermRef* terms = (TermRef*)(area + E.terms);
  uint64_t off = 0, base = 0;
  bool placed = false, go = true;
  const int nleaf = h->nleaf;
  DG_PLAN_UNROLL
  for (int l = 0; l < nleaf; ++l) {
    const DgpLeaf& L = leaves[l];
    if (L.nterm == 0) continue;
    if (MODE == EMIT_COUNT && L.nterm == 1) {
      // Entry count of a single term: the product of its factors' nonzero
      // counts (every thread computes it from the statistics, no barrier).
      const DgpTerm& T = T0[L.term0];
      const uint64_t coef = (T.coef_slot < 0 ? 1ull : scal[T.coef_slot]) * T.coef_const;
      if (coef == 0) continue;
      uint64_t n = 1, mx = coef;
      DG_PLAN_UNROLL
      for (int d = 0; d < L.rank; ++d) {
        n *= st[T.factor[d]].nnz;
        if (checks) mx = mul_sat(mx, st[T.factor[d]].vmax);
      }
      if (checks && n && mx > 0xFFFFFFFFull) *err |= DGP_ERR_OVERFLOW;
      off += n;
      continue;
    }
    const LeafGeom G = leaf_geom(L);
    leaf_terms(c, blob, l, area, PL, terms);
    c.sync();
    leaf_prepare<C, MODE, Word>(c, G, L.split, L.ucap, terms, L.nterm, 0, area, E, st, checks, err);
    c.sync();
    if (!placed) {
      base = place(c, &go);
      placed = true;
      if (!go) break;
    }
    off += leaf_emit<C, MODE, Word>(c, G, L.split, terms, L.nterm, 0, area, E, ids ? ids + base + off : nullptr,
                                    cnt ? cnt + base + off : nullptr, off < room ? room - off : 0, err);
    c.sync();
  }
  if (!placed) place(c, &go);
  return off;
}

// Row size (EMIT_COUNT) or row contents (EMIT_FILL, at most `room` entries
// written at ids/cnt) of one location; 0 and DGP_ERR_RANGE when the
// location lies outside the output.
template <class C, int MODE>
DGC uint64_t location_row(C& c, const uint8_t* blob, int64_t loc, uint8_t* area, uint32_t* ids, uint32_t* cnt,
                          uint64_t room, uint32_t* err) {
  if (!location_in_range(blob, loc)) {
    *err |= DGP_ERR_RANGE;
    return 0;
  }
  location_plan(c, blob, loc, area, err);
  c.sync();
  PlaceAt at{0};
  return location_leaves<C, MODE>(c, blob, area, ids, cnt, room, err, at);
}

// Per-leaf combined emission shapes of a two-graph comparison.
struct PairPlan {
  int32_t nleaf;
  int32_t max_terms;
  int32_t union_entries;
  int32_t emit_entries;
  uint32_t plan_b;  // byte offset of graph B's plan area (for `nthreads`)
  int32_t nthreads;
  uint32_t vars;    // bytes of component-sum scratch before graph A's plan area
  uint32_t lds_bytes;
  LeafShape leaf[16];
};

// One factor of a single-term leaf, as the comparison reads it: values
// vals[0 .. len) at coordinates lo .. lo + len - 1 (LDS).
struct FacView {
  int32_t lo, len;
  const uint64_t* vals;
  DGC uint32_t at(int32_t x) const {  // (values below 2^32 here)
    const int32_t i = x - lo;
    return (i >= 0 && i < len) ? (uint32_t)vals[i] : 0u;
  }
};

DGC FacView fac_view(const uint8_t* blob, const uint8_t* area, const PlanLayout& PL, int f) {
  const DgpHeader* h = (const DgpHeader*)blob;
  const DgpFactor* fac = (const DgpFactor*)(blob + h->factor_off);
  const int32_t* meta = (const int32_t*)(area + PL.fmeta);
  FacView v;
  v.lo = meta[2 * f];
  v.len = meta[2 * f + 1];
  v.vals = (const uint64_t*)(area + PL.fval) + fac[f].off;
  return v;
}

DGC uint64_t term_coef(const uint8_t* blob, const uint8_t* area, const PlanLayout& PL, const DgpTerm& T) {
  const uint64_t* scal = (const uint64_t*)(area + PL.scal);
  return (T.coef_slot < 0 ? 1ull : scal[T.coef_slot]) * T.coef_const;
}

// Compares leaf `leaf` of two plans whose leaf is one term each, without
// expanding cells.  A term is coef * prod_d f_d(x_d).  When both have
// entries (nonzero coefficient and a nonzero coordinate in every dim),
// their nonzero cells agree iff every dim's two factors have the same
// nonzero coordinates; then their counts agree iff every dim's two factors
// are proportional there and one cell (the first nonzero coordinate of
// every dim) has the same count.  Factor values and that cell's count are
// real counts below 2^32 (the caller checks the static bounds), so the
// cross products fit 64 bits.  Block-uniform results come from ballots;
// nothing is written.  Returns 0 equal, 1 nonzero sets differ, 2 counts
// differ.
template <class C>
DGC uint32_t compare_single_terms(C& c, const uint8_t* blob_a, const uint8_t* blob_b, int leaf, const uint8_t* area,
                                  const PlanLayout& PA, const PlanLayout& PB) {
  const DgpHeader* ha = (const DgpHeader*)blob_a;
  const DgpHeader* hb = (const DgpHeader*)blob_b;
  const DgpLeaf& La = ((const DgpLeaf*)(blob_a + ha->leaf_off))[leaf];
  const DgpLeaf& Lb = ((const DgpLeaf*)(blob_b + hb->leaf_off))[leaf];
  const DgpTerm& Ta = ((const DgpTerm*)(blob_a + ha->term_off))[La.term0];
  const DgpTerm& Tb = ((const DgpTerm*)(blob_b + hb->term_off))[Lb.term0];
  const int tid = c.tid(), nt = c.nthreads(), rank = La.rank;
  uint64_t ca = term_coef(blob_a, area, PA, Ta), cb = term_coef(blob_b, area, PB, Tb);
  bool empty_a = ca == 0, empty_b = cb == 0, differ = false;
  int32_t x0[DGP_MAX_RANK];
  // Pass 1: first nonzero coordinate of each factor, and whether the
  // nonzero coordinates agree.
  DG_PLAN_UNROLL
  for (int d = 0; d < rank; ++d) {
    const FacView A = fac_view(blob_a, area, PA, Ta.factor[d]);
    const FacView B = fac_view(blob_b, area, PB, Tb.factor[d]);
    int32_t lo = A.lo, hi = A.lo + A.len;
    if (B.len > 0) {
      if (A.len <= 0) {
        lo = B.lo;
        hi = B.lo + B.len;
      } else {
        lo = B.lo < lo ? B.lo : lo;
        hi = B.lo + B.len > hi ? B.lo + B.len : hi;
      }
    }
    int32_t fa = -1, fb = -1;
    bool diff = false;
    for (int32_t base = lo; base < hi; base += nt) {
      const int32_t x = base + tid;
      const bool nza = x < hi && A.at(x) != 0u, nzb = x < hi && B.at(x) != 0u;
      if (fa < 0) {
        const int k = c.first(nza);
        if (k >= 0) fa = base + k;
      }
      if (fb < 0) {
        const int k = c.first(nzb);
        if (k >= 0) fb = base + k;
      }
      diff = diff || nza != nzb;
    }
    empty_a = empty_a || fa < 0;
    empty_b = empty_b || fb < 0;
    differ = differ || c.any(diff);
    x0[d] = fa;
  }
  if (empty_a || empty_b) return empty_a == empty_b ? 0u : 1u;
  if (differ) return 1u;
  // Pass 2: proportional values against the first nonzero coordinate.
  bool unequal = false;
  DG_PLAN_UNROLL
  for (int d = 0; d < rank; ++d) {
    const FacView A = fac_view(blob_a, area, PA, Ta.factor[d]);
    const FacView B = fac_view(blob_b, area, PB, Tb.factor[d]);
    const uint32_t a0 = A.at(x0[d]), b0 = B.at(x0[d]);
    ca *= a0;
    cb *= b0;
    // (Both have the same nonzero coordinates: A's range covers them.)
    for (int32_t x = A.lo + tid; x < A.lo + A.len; x += nt)
      unequal = unequal || (uint64_t)A.at(x) * b0 != (uint64_t)B.at(x) * a0;
  }
  return (c.any(unequal) || ca != cb) ? 2u : 0u;
}

// PP lives in global memory (the kernels read it from the workspace).
template <class C>
DGC uint32_t location_compare(C& c, const uint8_t* blob_a, const uint8_t* blob_b, const PairPlan* PP, int64_t loc,
                              uint8_t* area, uint32_t* err) {
  const DgpHeader* ha = (const DgpHeader*)blob_a;
  const DgpHeader* hb = (const DgpHeader*)blob_b;
  if (!location_in_range(blob_a, loc)) {
    *err |= DGP_ERR_RANGE;
    return 0;
  }
  const PlanLayout PA = plan_layout(ha, PP->vars);
  const PlanLayout PB = plan_layout(hb, PP->plan_b);
  const EmitLayout E = emit_layout(compare_emit_base(hb, PB), PP->max_terms, PP->union_entries, PP->emit_entries);
  plan_exec(c, blob_a, loc, area, PA, err);
  plan_exec(c, blob_b, loc, area, PB, err);
  c.sync();  // (the emission area overlays B's dead values)
  const bool checks = !(ha->no_overflow && hb->no_overflow);
  const DgpLeaf* la = (const DgpLeaf*)(blob_a + ha->leaf_off);
  const DgpLeaf* lb = (const DgpLeaf*)(blob_b + hb->leaf_off);
  TermRef* terms = (TermRef*)(area + E.terms);
  uint32_t status = 0;
  const int nleaf = PP->nleaf;
  for (int l = 0; l < nleaf; ++l) {
    const int na = la[l].nterm, nb = lb[l].nterm;
    if (na + nb == 0) continue;
    if (na == 1 && nb == 1 && !checks) {
      // Two single-term leaves: compared factor by factor.
      const uint32_t s = compare_single_terms(c, blob_a, blob_b, l, area, PA, PB);
      if (s == 1) return 1;
      if (s == 2) status = 2;
      continue;
    }
    const LeafGeom G = leaf_geom(la[l]);
    leaf_terms(c, blob_a, l, area, PA, terms);
    leaf_terms(c, blob_b, l, area, PB, terms + na);
    c.sync();
    leaf_prepare<C, EMIT_COMPARE>(c, G, PP->leaf[l].split, PP->leaf[l].ucap, terms, na, nb, area, E, nullptr,
                                  checks, err, !checks);
    c.sync();
    const uint32_t s = (uint32_t)leaf_emit<C, EMIT_COMPARE, uint32_t>(c, G, PP->leaf[l].split, terms, na, nb, area,
                                                                      E, nullptr, nullptr, 0, err, !checks);
    c.sync();
    if (s == 1) return 1;
    if (s == 2) status = 2;
  }
  return status;
}

}  // namespace dgc
