// Device code of the expression-DAG kernels, shared by the precompiled
// kernels (kernels.hip) and the per-program specialised kernels built at run
// time (jit.cpp): the block context for dag_core.h and the kernel bodies.
// Each body takes the DAG program as a pointer; the specialised kernels pass
// a pointer to a __constant__ copy, so that every op and group field folds
// to a constant.
#pragma once
#include <stdint.h>

#include "kernels_dev.h"
#include "dag_core.h"

namespace dgk_dev {

// Block context for the expression-DAG code (dag_core.h): the enumeration
// context plus lanes and waves, wave-level ballots, scans and sums, a
// block-wide 64-bit scan and ordinary (cached) stores.
template <int BLOCK>
struct DagDevCtx : DevCtx<BLOCK> {
  uint64_t* wsum64;  // LDS, BLOCK / 64 words (scan_add)
  DGC int lane() const { return (int)(threadIdx.x & 63u); }
  DGC int lanes() const { return 64; }
  DGC int wave() const { return (int)(threadIdx.x >> 6); }
  DGC int nwaves() const { return BLOCK / 64; }
  // Orders the wave's LDS accesses before the call against those after it.
  DGC void wave_sync() const {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  DGC uint64_t ballot(bool f) const { return __ballot(f); }
  DGC void atomic_or32(uint32_t* p, uint32_t v) const { atomicOr(p, v); }
  // The minimum (maximum) of v over the wave into *p, one LDS atomic per
  // wave.
  DGC void reduce_min32(uint32_t* p, uint32_t v) const {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const uint32_t u = (uint32_t)__shfl_xor((int)v, o, 64);
      v = u < v ? u : v;
    }
    if ((threadIdx.x & 63u) == 0) atomicMin(p, v);
  }
  DGC void reduce_max32(uint32_t* p, uint32_t v) const {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const uint32_t u = (uint32_t)__shfl_xor((int)v, o, 64);
      v = u > v ? u : v;
    }
    if ((threadIdx.x & 63u) == 0) atomicMax(p, v);
  }
  // Lane j's v (j the same on every lane).
  DGC uint32_t bcast(uint32_t v, int j) const { return (uint32_t)__builtin_amdgcn_readlane((int)v, j); }
  // Exclusive count of set flags among lower lanes of the wave, and the
  // wave's total (no barrier).
  DGC uint32_t wave_prefix(bool f, uint32_t* total) const {
    const uint64_t m = __ballot(f);
    *total = (uint32_t)__popcll(m);
    return (uint32_t)__popcll(m & ((1ull << (threadIdx.x & 63u)) - 1ull));
  }
  // Exclusive sum of v over lower lanes of the wave, and the wave total
  // (no barrier).
  DGC uint32_t wave_scan(uint32_t v, uint32_t* total) const {
    const int ln = (int)(threadIdx.x & 63u);
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(x, (unsigned)o, 64);
      if (ln >= o) x += y;
    }
    *total = __shfl(x, 63, 64);
    return x - v;
  }
  // Sum of v over the wave, in every lane (no barrier).
  DGC uint64_t wave_sum64(uint64_t v) const {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
  }
  // Exclusive sum of v over lower threads of the block, and the block total.
  // Ends with every thread past a barrier.
  DGC uint64_t scan_add(uint64_t v, uint64_t* total) const {
    const int ln = (int)(threadIdx.x & 63u);
    uint64_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint64_t y = __shfl_up(x, (unsigned)o, 64);
      if (ln >= o) x += y;
    }
    if (BLOCK == 64) {
      *total = __shfl(x, 63, 64);
      return x - v;
    }
    const int wave = (int)(threadIdx.x >> 6);
    __syncthreads();
    if (ln == 63) wsum64[wave] = x;
    __syncthreads();
    uint64_t before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < BLOCK / 64; ++w) {
      const uint64_t s = wsum64[w];
      before += w < wave ? s : 0ull;
      tot += s;
    }
    *total = tot;
    return before + x - v;
  }
  // Ordinary store: the DAG's store instructions fill cache lines in parts
  // (edges at stride `nop`, runs at any alignment), which the L2 merges
  // before writing back; non-temporal stores would send each part to HBM.
  DGC void store_cached(uint32_t* p, uint32_t v) const { *p = v; }
  // Two or three consecutive words at a 4-byte aligned p, one store
  // instruction (the hardware needs only dword alignment for them).
  typedef uint32_t u32x2 __attribute__((ext_vector_type(2), aligned(4)));
  typedef uint32_t u32x3 __attribute__((ext_vector_type(3), aligned(4)));
  DGC void store2(uint32_t* p, uint32_t a, uint32_t b) const { *reinterpret_cast<u32x2*>(p) = u32x2{a, b}; }
  DGC void store3(uint32_t* p, uint32_t a, uint32_t b, uint32_t c) const {
    *reinterpret_cast<u32x3*>(p) = u32x3{a, b, c};
  }
};

// Expression DAGs: the sizes pass writes the node and edge counts of
// location i to nodes_n[i + 1] and edges_n[i + 1] (scanned afterwards into
// offsets); the fill pass writes location i's nodes at node_off[i] and its
// edges at edge_off[i].
template <int BLOCK>
// A block takes `per_block` consecutive locations, one after another (small
// DAGs: a block's writes then form one longer run, and its start and end
// are paid once for them all).
DGC void dag_sizes_body(const uint8_t* __restrict__ dblob, dgc::LocSrc locs, int64_t n, int per_block,
                        int64_t* __restrict__ nodes_n, int64_t* __restrict__ edges_n, uint32_t* __restrict__ err) {
  __shared__ uint32_t wsum[BLOCK / 64];
  __shared__ uint64_t wsum64[BLOCK / 64];
  const int64_t i0 = (int64_t)blockIdx.x * per_block;
  const int64_t i1 = i0 + per_block < n ? i0 + per_block : n;
  DagDevCtx<BLOCK> c{{wsum}, wsum64};
  uint32_t e = 0;
  uint8_t* area = reinterpret_cast<uint8_t*>(dg_smem);
  dgc::DagOut o{nullptr, nullptr, nullptr, nullptr, 0, 0};
  for (int64_t i = i0; i < i1; ++i) {
    uint64_t nn = 0, ne = 0;
    dgc::location_dag<DagDevCtx<BLOCK>, dgc::DAG_COUNT>(c, dblob, dgc::loc_at(locs, i), area, o, &nn, &ne, &e);
    if (threadIdx.x == 0) {
      nodes_n[i + 1] = (int64_t)nn;
      edges_n[i + 1] = (int64_t)ne;
    }
    __syncthreads();  // the next location reuses the LDS area
  }
  if (e) atomicOr(err, e);
}

template <int BLOCK>
DGC void dag_fill_body(const uint8_t* __restrict__ dblob, dgc::LocSrc locs, int64_t n, int per_block,
                       const int64_t* __restrict__ node_off, const int64_t* __restrict__ edge_off,
                       uint32_t* __restrict__ nodes, uint32_t* __restrict__ node_edge, uint32_t* __restrict__ edges,
                       uint32_t* __restrict__ mults, uint32_t* __restrict__ err) {
  __shared__ uint32_t wsum[BLOCK / 64];
  __shared__ uint64_t wsum64[BLOCK / 64];
  const int64_t i0 = (int64_t)blockIdx.x * per_block;
  const int64_t i1 = i0 + per_block < n ? i0 + per_block : n;
  DagDevCtx<BLOCK> c{{wsum}, wsum64};
  uint32_t e = 0;
  uint8_t* area = reinterpret_cast<uint8_t*>(dg_smem);
  for (int64_t i = i0; i < i1; ++i) {
    const int64_t n0 = node_off[i], e0 = edge_off[i];
    const int64_t rn = node_off[i + 1] - n0, re = edge_off[i + 1] - e0;
    dgc::DagOut o{nodes + n0, node_edge + n0, edges + e0, mults + e0, rn > 0 ? (uint64_t)rn : 0ull,
                  re > 0 ? (uint64_t)re : 0ull};
    uint64_t nn = 0, ne = 0;
    dgc::location_dag<DagDevCtx<BLOCK>, dgc::DAG_FILL>(c, dblob, dgc::loc_at(locs, i), area, o, &nn, &ne, &e);
    if (threadIdx.x == 0 && ((int64_t)nn != rn || (int64_t)ne != re)) e |= DGP_ERR_SIZE;
    __syncthreads();  // the next location reuses the LDS area
  }
  if (e) atomicOr(err, e);
}

// One pass over the locations for DAGs that fit in LDS: the walk writes the
// location's nodes and edges into an LDS stage after the walk's own area
// (stage_nodes node slots, two words each, then stage_edges edge slots, two
// words each); a node's first edge is relative to its location, so the
// stage does not depend on where the location's DAG lands.  The location's
// node and edge offsets then come from two decoupled look-backs over its
// predecessors' counts (st_nodes and st_edges, as for the single-pass
// enumeration), and the stage is copied out when it fits the capacities.
// Blocks take their locations from a ticket counter, so every lower index
// belongs to a block that is already running.
template <int BLOCK>
DGC void dag_onepass_body(const uint8_t* __restrict__ dblob, dgc::LocSrc locs, int64_t n,
                          int64_t* __restrict__ node_off, int64_t* __restrict__ edge_off,
                          uint32_t* __restrict__ nodes, uint32_t* __restrict__ node_edge,
                          uint32_t* __restrict__ edges, uint32_t* __restrict__ mults, uint64_t node_cap,
                          uint64_t edge_cap, uint32_t stage_off, uint32_t stage_nodes, uint32_t stage_edges,
                          uint64_t* __restrict__ st_nodes, uint64_t* __restrict__ st_edges,
                          unsigned long long* __restrict__ ticket, uint32_t* __restrict__ err) {
  __shared__ uint32_t wsum[BLOCK / 64];
  __shared__ uint64_t wsum64[BLOCK / 64];
  __shared__ int64_t sh_i;
  __shared__ uint64_t sh_noff, sh_eoff;
  if (threadIdx.x == 0) sh_i = (int64_t)atomicAdd(ticket, 1ull);
  __syncthreads();
  const int64_t i = sh_i;
  if (i >= n) return;
  DagDevCtx<BLOCK> c{{wsum}, wsum64};
  uint32_t e = 0;
  uint8_t* area = reinterpret_cast<uint8_t*>(dg_smem);
  uint32_t* sn = reinterpret_cast<uint32_t*>(area + stage_off);
  uint32_t* sne = sn + stage_nodes;
  uint32_t* se = sne + stage_nodes;
  uint32_t* sm = se + stage_edges;
  dgc::DagOut o{sn, sne, se, sm, stage_nodes, stage_edges};
  uint64_t nn = 0, ne = 0;
  dgc::location_dag<DagDevCtx<BLOCK>, dgc::DAG_FILL>(c, dblob, dgc::loc_at(locs, i), area, o, &nn, &ne, &e);
  if (nn > stage_nodes || ne > stage_edges) {
    // (Never for a program whose static bounds size the stage.)
    e |= DGP_ERR_CAPACITY;
    nn = 0;
    ne = 0;
  }
  __syncthreads();  // the stage is complete
  if (threadIdx.x == 0) {
    __hip_atomic_store(&st_nodes[i], (i == 0 ? ST_PREFIX : ST_SIZE) | nn, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&st_edges[i], (i == 0 ? ST_PREFIX : ST_SIZE) | ne, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  bool go_n = false, go_e = false;
  LookBack<BLOCK> lb_n{st_nodes, i, n, nn, node_cap, node_off, &sh_noff, &e};
  const uint64_t n0 = lb_n(c, &go_n);
  LookBack<BLOCK> lb_e{st_edges, i, n, ne, edge_cap, edge_off, &sh_eoff, &e};
  const uint64_t e0 = lb_e(c, &go_e);
  if (go_n)
    for (uint64_t k = threadIdx.x; k < nn; k += BLOCK) {
      nodes[n0 + k] = sn[k];
      node_edge[n0 + k] = sne[k];
    }
  if (go_e)
    for (uint64_t k = threadIdx.x; k < ne; k += BLOCK) {
      edges[e0 + k] = se[k];
      mults[e0 + k] = sm[k];
    }
  if (e) atomicOr(err, e);
}

}  // namespace dgk_dev
