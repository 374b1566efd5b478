// HIP kernels for gfx950: per-location plan execution and CSR emission
// (one block per location), the device-wide scan of row sizes, and the
// two-graph comparator with mismatch compaction.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#define DGC __device__ __forceinline__
#include "kernels_dev.h"
#include "dag_dev.h"
#include "kernels.h"
#include "order.h"


namespace {

using dgk_dev::DevCtx;

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_sizes(const uint8_t* __restrict__ blob, dgc::LocSrc locs, int64_t n,
                                                 int64_t* __restrict__ offsets, uint32_t* __restrict__ err) {
  dgk_dev::sizes_body<BLOCK>(blob, locs, n, offsets, err);
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_fill(const uint8_t* __restrict__ blob, dgc::LocSrc locs, int64_t n,
                                                const int64_t* __restrict__ offsets, int64_t base,
                                                uint32_t* __restrict__ ids, uint32_t* __restrict__ cnt,
                                                uint32_t* __restrict__ err) {
  dgk_dev::fill_body<BLOCK>(blob, locs, n, offsets, base, ids, cnt, err);
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_dag_sizes(const uint8_t* __restrict__ dblob, dgc::LocSrc locs, int64_t n,
                                                     int per_block, int64_t* __restrict__ nodes_n,
                                                     int64_t* __restrict__ edges_n, uint32_t* __restrict__ err) {
  dgk_dev::dag_sizes_body<BLOCK>(dblob, locs, n, per_block, nodes_n, edges_n, err);
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_dag_fill(const uint8_t* __restrict__ dblob, dgc::LocSrc locs, int64_t n,
                                                    int per_block, const int64_t* __restrict__ node_off,
                                                    const int64_t* __restrict__ edge_off, uint32_t* __restrict__ nodes,
                                                    uint32_t* __restrict__ node_edge, uint32_t* __restrict__ edges,
                                                    uint32_t* __restrict__ mults, uint32_t* __restrict__ err) {
  dgk_dev::dag_fill_body<BLOCK>(dblob, locs, n, per_block, node_off, edge_off, nodes, node_edge, edges, mults, err);
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_dag_onepass(
    const uint8_t* __restrict__ dblob, dgc::LocSrc locs, int64_t n, int64_t* __restrict__ node_off,
    int64_t* __restrict__ edge_off, uint32_t* __restrict__ nodes, uint32_t* __restrict__ node_edge,
    uint32_t* __restrict__ edges, uint32_t* __restrict__ mults, uint64_t node_cap, uint64_t edge_cap,
    uint32_t stage_off, uint32_t stage_nodes, uint32_t stage_edges, uint64_t* __restrict__ st_nodes,
    uint64_t* __restrict__ st_edges, unsigned long long* __restrict__ ticket, uint32_t* __restrict__ err) {
  dgk_dev::dag_onepass_body<BLOCK>(dblob, locs, n, node_off, edge_off, nodes, node_edge, edges, mults, node_cap,
                                   edge_cap, stage_off, stage_nodes, stage_edges, st_nodes, st_edges, ticket, err);
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_compare(const uint8_t* __restrict__ blob_a,
                                                   const uint8_t* __restrict__ blob_b,
                                                   const dgc::PairPlan* __restrict__ pp, dgc::LocSrc locs,
                                                   int64_t n, uint8_t* __restrict__ status,
                                                   int64_t* __restrict__ flags, unsigned long long* __restrict__ found,
                                                   uint64_t limit, uint32_t* __restrict__ err) {
  dgk_dev::compare_body<BLOCK>(blob_a, blob_b, pp, locs, n, status, flags, found, limit, err);
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_enumerate(const uint8_t* __restrict__ blob, dgc::LocSrc locs, int64_t n,
                                                     int64_t* __restrict__ offsets, uint32_t* __restrict__ ids,
                                                     uint32_t* __restrict__ cnt, uint64_t capacity,
                                                     uint64_t* __restrict__ status,
                                                     unsigned long long* __restrict__ ticket,
                                                     uint32_t* __restrict__ err) {
  dgk_dev::enumerate_body<BLOCK>(blob, locs, n, offsets, ids, cnt, capacity, status, ticket, err);
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_enumerate_wide(const uint8_t* __restrict__ blob, dgc::LocSrc locs,
                                                          int64_t n, int64_t* __restrict__ offsets,
                                                          uint64_t* __restrict__ ids, uint64_t* __restrict__ cnt,
                                                          uint64_t capacity, uint64_t* __restrict__ status,
                                                          unsigned long long* __restrict__ ticket,
                                                          uint32_t* __restrict__ err) {
  dgk_dev::enumerate_body<BLOCK, uint64_t>(blob, locs, n, offsets, ids, cnt, capacity, status, ticket, err);
}

__global__ void k_zero_u64(uint64_t* __restrict__ p, int64_t count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = 0ull;
}

// ---- device-wide inclusive scan of v[1..n] (v[0] = 0 on exit) ---------------
constexpr int SCAN_THREADS = 256;
constexpr int SCAN_ITEMS = 4;
constexpr int SCAN_TILE = SCAN_THREADS * SCAN_ITEMS;

__device__ __forceinline__ int64_t block_inclusive_scan(int64_t x, int64_t* sh, int64_t* total) {
  // Wave-level scan with shuffles, then across the 4 waves.
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int64_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[wave] = x;
  __syncthreads();
  int64_t before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < SCAN_THREADS / 64; ++w) {
    int64_t s = sh[w];
    before += (w < wave) ? s : 0;
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return x + before;
}

__global__ __launch_bounds__(SCAN_THREADS) void k_scan_reduce(const int64_t* __restrict__ v, int64_t n,
                                                              int64_t* __restrict__ sums) {
  __shared__ int64_t sh[SCAN_THREADS / 64];
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE;
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    int64_t i = base + (int64_t)threadIdx.x * SCAN_ITEMS + k;
    if (i < n) s += v[1 + i];
  }
  int64_t tot;
  block_inclusive_scan(s, sh, &tot);
  if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

// One block scans the tile sums (exclusive, in place).
__global__ __launch_bounds__(SCAN_THREADS) void k_scan_sums(int64_t* __restrict__ sums, int64_t m) {
  __shared__ int64_t sh[SCAN_THREADS / 64];
  int64_t carry = 0;
  for (int64_t b = 0; b < m; b += SCAN_THREADS) {
    int64_t i = b + threadIdx.x;
    int64_t x = i < m ? sums[i] : 0;
    int64_t tot;
    int64_t inc = block_inclusive_scan(x, sh, &tot);
    if (i < m) sums[i] = carry + inc - x;
    carry += tot;
  }
}

__global__ __launch_bounds__(SCAN_THREADS) void k_scan_apply(int64_t* __restrict__ v, int64_t n,
                                                             const int64_t* __restrict__ sums) {
  __shared__ int64_t sh[SCAN_THREADS / 64];
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE;
  int64_t x[SCAN_ITEMS];
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    int64_t i = base + (int64_t)threadIdx.x * SCAN_ITEMS + k;
    x[k] = i < n ? v[1 + i] : 0;
    s += x[k];
  }
  int64_t tot;
  int64_t inc = block_inclusive_scan(s, sh, &tot);
  int64_t run = sums[blockIdx.x] + inc - s;
#pragma unroll
  for (int k = 0; k < SCAN_ITEMS; ++k) {
    int64_t i = base + (int64_t)threadIdx.x * SCAN_ITEMS + k;
    run += x[k];
    if (i < n) v[1 + i] = run;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) v[0] = 0;
}

__global__ void k_scatter_mismatch(const uint8_t* __restrict__ status, const int64_t* __restrict__ pos, int64_t n,
                                   int64_t* __restrict__ out) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n && (status[i] == 1 || status[i] == 2)) out[pos[i]] = i;
}

// ---- location order: keyed permutation with excluded positions ------------
// Position i of [first, first + count) writes pi(i) at i - first minus the
// number of excluded positions below i; an excluded position writes nothing.
// pos: the sorted excluded positions inside the range.
__global__ __launch_bounds__(256) void k_order_write(DgPermKey K, const int64_t* __restrict__ pos, int64_t m,
                                                     int64_t first, int64_t count, int64_t* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < count; t += stride) {
    const int64_t i = first + t;
    int64_t lo = 0, hi = m;  // excluded positions below i
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (pos[mid] < i) lo = mid + 1;
      else hi = mid;
    }
    if (lo < m && pos[lo] == i) continue;
    __builtin_nontemporal_store(dg_perm_at((uint64_t)i, K), &out[t - lo]);
  }
}

__global__ void k_zero_offsets(int64_t* __restrict__ v) { v[0] = 0; }

__global__ void k_rebase(const int64_t* __restrict__ src, int64_t* __restrict__ dst, int64_t count, int64_t base) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) dst[i] = src[i] - base;
}

__global__ void k_zero_word(uint32_t* __restrict__ p) { *p = 0u; }

template <class K>
hipError_t allow_lds(K kernel, uint32_t bytes) {
  if (bytes <= 65536u) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

}  // namespace

namespace dgk {

hipError_t launch_sizes(const uint8_t* blob, dgc::LocSrc locs, int64_t n, int64_t* offsets, uint32_t* err,
                        int block, uint32_t lds, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (block != 64 && block != 256) return hipErrorInvalidConfiguration;
  hipError_t e;
  if (block == 256) {
    if ((e = allow_lds(k_sizes<256>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_sizes<256>, dim3((unsigned)n), dim3(256), lds, s, blob, locs, n, offsets, err);
  } else {
    if ((e = allow_lds(k_sizes<64>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_sizes<64>, dim3((unsigned)n), dim3(64), lds, s, blob, locs, n, offsets, err);
  }
  return hipGetLastError();
}

hipError_t launch_fill(const uint8_t* blob, dgc::LocSrc locs, int64_t n, const int64_t* offsets, int64_t base,
                       uint32_t* ids, uint32_t* cnt, uint32_t* err, int block, uint32_t lds, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (block != 64 && block != 256) return hipErrorInvalidConfiguration;
  hipError_t e;
  if (block == 256) {
    if ((e = allow_lds(k_fill<256>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_fill<256>, dim3((unsigned)n), dim3(256), lds, s, blob, locs, n, offsets, base, ids, cnt,
                       err);
  } else {
    if ((e = allow_lds(k_fill<64>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_fill<64>, dim3((unsigned)n), dim3(64), lds, s, blob, locs, n, offsets, base, ids, cnt, err);
  }
  return hipGetLastError();
}

hipError_t launch_dag_sizes(const uint8_t* dblob, dgc::LocSrc locs, int64_t n, int per_block, int64_t* nodes_n,
                            int64_t* edges_n, uint32_t* err, int block, uint32_t lds, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (per_block < 1) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)((n + per_block - 1) / per_block);
  hipError_t e;
  if (block == 256) {
    if ((e = allow_lds(k_dag_sizes<256>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_dag_sizes<256>, dim3(grid), dim3(256), lds, s, dblob, locs, n, per_block, nodes_n, edges_n,
                       err);
  } else if (block == 64) {
    if ((e = allow_lds(k_dag_sizes<64>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_dag_sizes<64>, dim3(grid), dim3(64), lds, s, dblob, locs, n, per_block, nodes_n, edges_n,
                       err);
  } else {
    return hipErrorInvalidConfiguration;
  }
  return hipGetLastError();
}

hipError_t launch_dag_onepass(const uint8_t* dblob, dgc::LocSrc locs, int64_t n, int64_t blocks, int64_t* node_off,
                              int64_t* edge_off, uint32_t* nodes, uint32_t* node_edge, uint32_t* edges,
                              uint32_t* mults, uint64_t node_cap, uint64_t edge_cap, uint32_t stage_off,
                              uint32_t stage_nodes, uint32_t stage_edges, uint64_t* st_nodes, uint64_t* st_edges,
                              uint64_t* ticket, uint32_t* err, int block, uint32_t lds, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  unsigned long long* t = reinterpret_cast<unsigned long long*>(ticket);
  hipError_t e;
  if (block == 256) {
    if ((e = allow_lds(k_dag_onepass<256>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_dag_onepass<256>, dim3((unsigned)blocks), dim3(256), lds, s, dblob, locs, n, node_off,
                       edge_off, nodes, node_edge, edges, mults, node_cap, edge_cap, stage_off, stage_nodes,
                       stage_edges, st_nodes, st_edges, t, err);
  } else if (block == 64) {
    if ((e = allow_lds(k_dag_onepass<64>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_dag_onepass<64>, dim3((unsigned)blocks), dim3(64), lds, s, dblob, locs, n, node_off,
                       edge_off, nodes, node_edge, edges, mults, node_cap, edge_cap, stage_off, stage_nodes,
                       stage_edges, st_nodes, st_edges, t, err);
  } else {
    return hipErrorInvalidConfiguration;
  }
  return hipGetLastError();
}

hipError_t launch_dag_fill(const uint8_t* dblob, dgc::LocSrc locs, int64_t n, int per_block, const int64_t* node_off,
                           const int64_t* edge_off, uint32_t* nodes, uint32_t* node_edge, uint32_t* edges,
                           uint32_t* mults, uint32_t* err, int block, uint32_t lds, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (per_block < 1) return hipErrorInvalidValue;
  const unsigned grid = (unsigned)((n + per_block - 1) / per_block);
  hipError_t e;
  if (block == 256) {
    if ((e = allow_lds(k_dag_fill<256>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_dag_fill<256>, dim3(grid), dim3(256), lds, s, dblob, locs, n, per_block, node_off, edge_off,
                       nodes, node_edge, edges, mults, err);
  } else if (block == 64) {
    if ((e = allow_lds(k_dag_fill<64>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_dag_fill<64>, dim3(grid), dim3(64), lds, s, dblob, locs, n, per_block, node_off, edge_off,
                       nodes, node_edge, edges, mults, err);
  } else {
    return hipErrorInvalidConfiguration;
  }
  return hipGetLastError();
}

hipError_t launch_compare(const uint8_t* blob_a, const uint8_t* blob_b, const dgc::PairPlan* pp, uint32_t lds,
                          dgc::LocSrc locs, int64_t n, uint8_t* status, int64_t* flags, uint64_t* found,
                          uint64_t limit, uint32_t* err, int block, hipStream_t s) {
  unsigned long long* fnd = reinterpret_cast<unsigned long long*>(found);
  if (n <= 0) return hipSuccess;
  hipError_t e;
  if (block == 256) {
    if ((e = allow_lds(k_compare<256>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_compare<256>, dim3((unsigned)n), dim3(256), lds, s, blob_a, blob_b, pp, locs, n, status,
                       flags, fnd, limit, err);
  } else {
    if ((e = allow_lds(k_compare<64>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_compare<64>, dim3((unsigned)n), dim3(64), lds, s, blob_a, blob_b, pp, locs, n, status, flags,
                       fnd, limit, err);
  }
  return hipGetLastError();
}

int64_t scan_temp_entries(int64_t n) { return (n + SCAN_TILE - 1) / SCAN_TILE + 1; }

hipError_t launch_enumerate(const uint8_t* blob, dgc::LocSrc locs, int64_t n, int64_t blocks, int64_t* offsets,
                            uint32_t* ids, uint32_t* cnt, uint64_t capacity, uint64_t* status, uint64_t* ticket,
                            uint32_t* err, int block, uint32_t lds, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  if (block != 64 && block != 256) return hipErrorInvalidConfiguration;
  hipError_t e;
  unsigned long long* t = reinterpret_cast<unsigned long long*>(ticket);
  if (block == 256) {
    if ((e = allow_lds(k_enumerate<256>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_enumerate<256>, dim3((unsigned)blocks), dim3(256), lds, s, blob, locs, n, offsets, ids, cnt,
                       capacity, status, t, err);
  } else {
    if ((e = allow_lds(k_enumerate<64>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_enumerate<64>, dim3((unsigned)blocks), dim3(64), lds, s, blob, locs, n, offsets, ids, cnt,
                       capacity, status, t, err);
  }
  return hipGetLastError();
}

hipError_t launch_rebase(const int64_t* src, int64_t* dst, int64_t count, int64_t base, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_rebase, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, src, dst, count, base);
  return hipGetLastError();
}

hipError_t launch_enumerate_wide(const uint8_t* blob, dgc::LocSrc locs, int64_t n, int64_t blocks,
                                 int64_t* offsets, uint64_t* ids, uint64_t* cnt, uint64_t capacity, uint64_t* status,
                                 uint64_t* ticket, uint32_t* err, int block, uint32_t lds, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  if (block != 64 && block != 256) return hipErrorInvalidConfiguration;
  hipError_t e;
  unsigned long long* t = reinterpret_cast<unsigned long long*>(ticket);
  if (block == 256) {
    if ((e = allow_lds(k_enumerate_wide<256>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_enumerate_wide<256>, dim3((unsigned)blocks), dim3(256), lds, s, blob, locs, n, offsets, ids,
                       cnt, capacity, status, t, err);
  } else {
    if ((e = allow_lds(k_enumerate_wide<64>, lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_enumerate_wide<64>, dim3((unsigned)blocks), dim3(64), lds, s, blob, locs, n, offsets, ids,
                       cnt, capacity, status, t, err);
  }
  return hipGetLastError();
}

hipError_t launch_zero_u64(uint64_t* p, int64_t count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_zero_u64, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, p, count);
  return hipGetLastError();
}

hipError_t launch_zero(uint32_t* p, hipStream_t s) {
  hipLaunchKernelGGL(k_zero_word, dim3(1), dim3(1), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_scan(int64_t* v, int64_t n, int64_t* sums, hipStream_t s) {
  if (n <= 0) {
    hipLaunchKernelGGL(k_zero_offsets, dim3(1), dim3(1), 0, s, v);
    return hipGetLastError();
  }
  const int64_t tiles = (n + SCAN_TILE - 1) / SCAN_TILE;
  hipLaunchKernelGGL(k_scan_reduce, dim3((unsigned)tiles), dim3(SCAN_THREADS), 0, s, v, n, sums);
  hipLaunchKernelGGL(k_scan_sums, dim3(1), dim3(SCAN_THREADS), 0, s, sums, tiles);
  hipLaunchKernelGGL(k_scan_apply, dim3((unsigned)tiles), dim3(SCAN_THREADS), 0, s, v, n, sums);
  return hipGetLastError();
}

hipError_t launch_order(const DgPermKey& K, const int64_t* pos, int64_t m, int64_t first, int64_t count,
                        int64_t* out, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((count + 255) / 256, 1 << 20);
  hipLaunchKernelGGL(k_order_write, dim3((unsigned)blocks), dim3(256), 0, s, K, pos, m, first, count, out);
  return hipGetLastError();
}

hipError_t launch_scatter_mismatch(const uint8_t* status, const int64_t* pos, int64_t n, int64_t* out,
                                   hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_scatter_mismatch, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, status, pos, n, out);
  return hipGetLastError();
}

}  // namespace dgk
