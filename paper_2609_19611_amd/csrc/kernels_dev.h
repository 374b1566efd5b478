// Device code shared by the precompiled kernels (kernels.hip) and the
// per-graph specialised kernels built at run time (jit.cpp): the block
// context for core.h and the bodies of the per-location kernels.  Each body
// takes the compiled plan as a pointer; the specialised kernels pass a
// pointer to a __constant__ copy of the plan so that every instruction field,
// op dispatch and trip count folds to a constant.
#pragma once
#include <stdint.h>

#include "core.h"

namespace dgk_dev {

// Block context for core.h: BLOCK threads cooperating on one location.
template <int BLOCK>
struct DevCtx {
  uint32_t* wsum;  // LDS, BLOCK / 64 words
  DGC int tid() const { return (int)threadIdx.x; }
  DGC int nthreads() const { return BLOCK; }
  DGC void sync() const { __syncthreads(); }
  DGC void atomic_add(uint64_t* p, uint64_t v) const {
    atomicAdd(reinterpret_cast<unsigned long long*>(p), (unsigned long long)v);
  }
  DGC void atomic_max(uint64_t* p, uint64_t v) const {
    atomicMax(reinterpret_cast<unsigned long long*>(p), (unsigned long long)v);
  }
  DGC uint32_t atomic_inc(uint32_t* p) const { return atomicAdd(p, 1u); }
  // Row stores are ordinary stores through the L2.  A wave's runs are
  // whole lines either way, the HBM write traffic is the same, and they
  // measured 2-3 % (32-bit words) and 4-7 % (64-bit words) faster than
  // non-temporal stores for the CSR rows.
  DGC void store(uint32_t* p, uint32_t v) const { *p = v; }
  DGC void store(uint64_t* p, uint64_t v) const { *p = v; }
  // Adds (or takes the maximum of) every thread's v into *p with at most
  // four LDS atomics per wave instead of one per thread: DPP lane permutes
  // (xor 1, xor 2, mirror within 8, mirror within 16) leave every row of 16
  // lanes holding its total, which the row's first lane adds.  A wave with
  // no nonzero value, or a single one, skips the permutes.  Called by all
  // lanes of the wave.
  DGC void reduce_add(uint64_t* p, uint64_t v) const {
    const uint64_t m = __ballot(v != 0);
    if (m == 0) return;
    if ((m & (m - 1)) == 0) {  // one contributor
      if (v) atomic_add(p, v);
      return;
    }
    v += dpp64<0xB1>(v);
    v += dpp64<0x4E>(v);
    v += dpp64<0x141>(v);
    v += dpp64<0x140>(v);
    if ((threadIdx.x & 15u) == 0 && v) atomic_add(p, v);
  }
  DGC void reduce_max(uint64_t* p, uint64_t v) const {
    const uint64_t m = __ballot(v != 0);
    if (m == 0) return;
    if ((m & (m - 1)) == 0) {  // one contributor
      if (v) atomic_max(p, v);
      return;
    }
    v = umax(v, dpp64<0xB1>(v));
    v = umax(v, dpp64<0x4E>(v));
    v = umax(v, dpp64<0x141>(v));
    v = umax(v, dpp64<0x140>(v));
    if ((threadIdx.x & 15u) == 0 && v) atomic_max(p, v);
  }
  DGC static uint64_t umax(uint64_t a, uint64_t b) { return a > b ? a : b; }
  template <int CTRL>
  DGC static uint64_t dpp64(uint64_t v) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, 0xf, 0xf, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL, 0xf, 0xf, false);
    return ((uint64_t)hi << 32) | lo;
  }
  // Exclusive count of set flags among lower threads of the block, and the
  // block total.  Ends with every thread past a barrier.
  DGC uint32_t prefix(bool f, uint32_t* total) const {
    const uint64_t m = __ballot(f);
    const uint32_t lane = threadIdx.x & 63u;
    const uint32_t pre = (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
    if (BLOCK == 64) {
      *total = (uint32_t)__popcll(m);
      return pre;
    }
    const uint32_t wave = threadIdx.x >> 6;
    __syncthreads();
    if (lane == 0) wsum[wave] = (uint32_t)__popcll(m);
    __syncthreads();
    uint32_t before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < BLOCK / 64; ++w) {
      uint32_t x = wsum[w];
      before += (w < (int)wave) ? x : 0u;
      tot += x;
    }
    *total = tot;
    return before + pre;
  }
  // Whether f holds on any thread of the block.  A one-wave block takes
  // the wave's ballot instead of the block-wide reduction.
  DGC bool any(bool f) const {
    if (BLOCK == 64) return __ballot(f) != 0;
    return __syncthreads_or(f) != 0;
  }
  // Lowest thread index of the block with f set, or -1 (the same on every
  // thread).  A one-wave block takes the wave's ballot.
  DGC int first(bool f) const {
    const uint64_t m = __ballot(f);
    if (BLOCK == 64) return m ? (int)__builtin_ctzll(m) : -1;
    const uint32_t wave = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63u) == 0) wsum[wave] = m ? (uint32_t)__builtin_ctzll(m) : 64u;
    __syncthreads();
    int r = -1;
#pragma unroll
    for (int w = BLOCK / 64 - 1; w >= 0; --w) {
      const uint32_t x = wsum[w];
      if (x < 64u) r = w * 64 + (int)x;
    }
    return r;
  }
};

extern __shared__ uint64_t dg_smem[];

template <int BLOCK>
DGC void sizes_body(const uint8_t* __restrict__ blob, dgc::LocSrc locs, int64_t n,
                    int64_t* __restrict__ offsets, uint32_t* __restrict__ err) {
  __shared__ uint32_t wsum[BLOCK / 64];
  const int64_t i = blockIdx.x;
  if (i >= n) return;
  DevCtx<BLOCK> c{wsum};
  uint32_t e = 0;
  uint8_t* area = reinterpret_cast<uint8_t*>(dg_smem);
  const uint64_t rows =
      dgc::location_row<DevCtx<BLOCK>, dgc::EMIT_COUNT>(c, blob, dgc::loc_at(locs, i), area, nullptr, nullptr, 0, &e);
  if (threadIdx.x == 0) offsets[i + 1] = (int64_t)rows;
  if (e) atomicOr(err, e);
}

template <int BLOCK>
DGC void fill_body(const uint8_t* __restrict__ blob, dgc::LocSrc locs, int64_t n,
                   const int64_t* __restrict__ offsets, int64_t base, uint32_t* __restrict__ ids,
                   uint32_t* __restrict__ cnt, uint32_t* __restrict__ err) {
  __shared__ uint32_t wsum[BLOCK / 64];
  const int64_t i = blockIdx.x;
  if (i >= n) return;
  DevCtx<BLOCK> c{wsum};
  uint32_t e = 0;
  uint8_t* area = reinterpret_cast<uint8_t*>(dg_smem);
  // Row i goes to [offsets[i] - base, offsets[i+1] - base) whatever its size.
  const int64_t start = offsets[i] - base;
  const int64_t room = offsets[i + 1] - offsets[i];
  const uint64_t rows = dgc::location_row<DevCtx<BLOCK>, dgc::EMIT_FILL>(
      c, blob, dgc::loc_at(locs, i), area, ids + start, cnt + start, room > 0 ? (uint64_t)room : 0ull, &e);
  if (threadIdx.x == 0 && (int64_t)rows != room) e |= DGP_ERR_SIZE;
  if (e) atomicOr(err, e);
}

// Status of a location the comparison skipped because `limit` mismatching
// locations had already been found.
constexpr uint8_t CMP_SKIPPED = 3;

template <int BLOCK>
DGC void compare_body(const uint8_t* __restrict__ blob_a, const uint8_t* __restrict__ blob_b,
                      const dgc::PairPlan* __restrict__ pp, dgc::LocSrc locs, int64_t n,
                      uint8_t* __restrict__ status, int64_t* __restrict__ flags, unsigned long long* __restrict__ found,
                      uint64_t limit, uint32_t* __restrict__ err) {
  __shared__ uint32_t wsum[BLOCK / 64];
  __shared__ int skip;
  const int64_t i = blockIdx.x;
  if (i >= n) return;
  if (threadIdx.x == 0)
    skip = limit != 0 && __hip_atomic_load(found, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= limit;
  __syncthreads();
  if (skip) {
    if (threadIdx.x == 0) {
      status[i] = CMP_SKIPPED;
      flags[i + 1] = 0;
    }
    return;
  }
  DevCtx<BLOCK> c{wsum};
  uint32_t e = 0;
  uint8_t* area = reinterpret_cast<uint8_t*>(dg_smem);
  const uint32_t s = dgc::location_compare(c, blob_a, blob_b, pp, dgc::loc_at(locs, i), area, &e);
  if (threadIdx.x == 0) {
    status[i] = (uint8_t)s;
    flags[i + 1] = s != 0 ? 1 : 0;
    if (s != 0 && limit != 0) atomicAdd(found, 1ull);
  }
  if (e) atomicOr(err, e);
}

// ---- single pass: sizes, offsets by decoupled look-back, rows -------------
// status[i]: bits 62-63 = 0 not ready, 1 row size of i, 2 offsets[i+1];
// bits 0-61 the value.  A reader needs nothing but the word itself, so the
// accesses are relaxed atomics at device scope (they bypass the non-coherent
// per-XCD caches without invalidating them).  A block takes its location index from a ticket
// counter, so every lower index belongs to a block that is already running
// and the look-back always finishes; the wait is bounded anyway.
constexpr uint64_t ST_SIZE = 1ull << 62, ST_PREFIX = 2ull << 62, ST_VALUE = (1ull << 62) - 1;
constexpr uint32_t LOOKBACK_SPIN_LIMIT = 1u << 24;
constexpr int LB_WORDS = 1;  // status words read per lane and step

// Offset of row i by decoupled look-back (wave 0), once the row's own size
// has been published: the nearest predecessor whose running total is
// published ends the walk, the row sizes above it are added; only those must
// have arrived.  Publishes row i's running total, writes offsets[i] (and
// offsets[n] for the last row) and tells the block whether the row fits in
// `capacity` entries.  Called by every thread of the block.
template <int BLOCK>
struct LookBack {
  uint64_t* status;
  int64_t i, n;
  uint64_t size, capacity;
  int64_t* offsets;
  uint64_t* sh_off;
  uint32_t* e;
  bool fits = false;
  DGC uint64_t operator()(DevCtx<BLOCK>&, bool* go) {
    if (threadIdx.x < 64) {
      // Each lane reads LB_WORDS consecutive status words, so one step of
      // the wave covers 64 * LB_WORDS predecessors.
      const int lane = (int)threadIdx.x;
      uint64_t before = 0;
      int64_t hi = i;  // window [hi - 64 * LB_WORDS, hi)
      uint32_t spins = 0;
      while (hi > 0) {
        const int64_t base = hi - 64 * LB_WORDS + (int64_t)lane * LB_WORDS;
        uint64_t st[LB_WORDS];
        int kp = -1;  // this lane's highest word holding a running total
#pragma unroll
        for (int k = 0; k < LB_WORDS; ++k) {
          const int64_t j = base + k;
          st[k] = j >= 0 ? __hip_atomic_load(&status[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : ST_PREFIX;
          if ((st[k] & ~ST_VALUE) == ST_PREFIX) kp = k;
        }
        bool missing = false;  // a word above kp has not arrived
#pragma unroll
        for (int k = 0; k < LB_WORDS; ++k) missing = missing || (k > kp && (st[k] & ~ST_VALUE) == 0);
        const uint64_t pmask = __ballot(kp >= 0);
        const int top = pmask ? 63 - __clzll((long long)pmask) : -1;
        const uint64_t waiting = __ballot(missing) & (top >= 0 ? ~((1ull << top) - 1ull) : ~0ull);
        if (waiting) {
          if (++spins > LOOKBACK_SPIN_LIMIT) {
            *e |= DGP_ERR_TIMEOUT;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
          continue;
        }
        uint64_t v = 0;
#pragma unroll
        for (int k = 0; k < LB_WORDS; ++k)
          if (lane > top || (lane == top && k >= kp)) v += st[k] & ST_VALUE;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
        before += v;
        if (top >= 0) break;
        hi -= 64 * LB_WORDS;
      }
      if (lane == 0) {
        if (i > 0)
          __hip_atomic_store(&status[i], ST_PREFIX | (before + size), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        offsets[i] = (int64_t)before;
        if (i == n - 1) offsets[n] = (int64_t)(before + size);
        *sh_off = before;
      }
    }
    __syncthreads();
    const uint64_t off = *sh_off;
    fits = off + size <= capacity;
    if (!fits && threadIdx.x == 0 && size > 0) *e |= DGP_ERR_BUFFER;
    *go = fits;
    return off;
  }
};

template <int BLOCK, class Word = uint32_t>
DGC void enumerate_body(const uint8_t* __restrict__ blob, dgc::LocSrc locs, int64_t n,
                                                     int64_t* __restrict__ offsets, Word* __restrict__ ids,
                                                     Word* __restrict__ cnt, uint64_t capacity,
                                                     uint64_t* __restrict__ status,
                                                     unsigned long long* __restrict__ ticket,
                                                     uint32_t* __restrict__ err) {
  __shared__ uint32_t wsum[BLOCK / 64];
  __shared__ int64_t sh_i;
  __shared__ uint64_t sh_off;
  if (threadIdx.x == 0) sh_i = (int64_t)atomicAdd(ticket, 1ull);
  __syncthreads();
  const int64_t i = sh_i;
  if (i >= n) return;
  DevCtx<BLOCK> c{wsum};
  uint32_t e = 0;
  uint8_t* area = reinterpret_cast<uint8_t*>(dg_smem);
  const int64_t loc = dgc::loc_at(locs, i);
  const bool ok = dgc::location_in_range(blob, loc);
  if (!ok) e |= DGP_ERR_RANGE;
  if (ok) dgc::location_plan(c, blob, loc, area, &e);
  __syncthreads();
  dgc::PlaceAt none{0};
  const uint64_t size = ok ? dgc::location_leaves<DevCtx<BLOCK>, dgc::EMIT_COUNT, dgc::PlaceAt, Word>(
                                 c, blob, area, nullptr, nullptr, 0, &e, none)
                           : 0ull;
  if (threadIdx.x == 0) {
    __hip_atomic_store(&status[i], (i == 0 ? ST_PREFIX : ST_SIZE) | size, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // The row's offset is looked up once its first leaf is prepared (or at
  // once when it has nothing to write).
  LookBack<BLOCK> place{status, i, n, size, capacity, offsets, &sh_off, &e};
  if (ok && size > 0) {
    const uint64_t rows = dgc::location_leaves<DevCtx<BLOCK>, dgc::EMIT_FILL, LookBack<BLOCK>, Word>(
        c, blob, area, ids, cnt, size, &e, place);
    if (threadIdx.x == 0 && place.fits && rows != size) e |= DGP_ERR_SIZE;
  } else {
    bool go;
    place(c, &go);
  }
  if (e) atomicOr(err, e);
}

}  // namespace dgk_dev
