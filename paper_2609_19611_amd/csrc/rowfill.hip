// Measurement reference for the enumeration's write rate (not part of the
// library's ABI): the rows of a CSR output written by a kernel with no
// per-location work, one block per location, lanes shifted so that each
// wave's stores cover aligned 256-byte blocks, as the enumeration writes
// them.  Launched with the enumeration's block size and LDS per block, it
// has the enumeration's grid, occupancy and store pattern: the rate a
// one-block-per-row writer of these rows reaches on the machine at hand.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_row_fill(uint32_t* __restrict__ ids, uint32_t* __restrict__ cnt,
                                                    const int64_t* __restrict__ offsets, int64_t n) {
  const int64_t i = blockIdx.x;
  if (i >= n) return;
  const int64_t lo = offsets[i], hi = offsets[i + 1];
  const int64_t head = lo & 63;  // lanes shifted to 256-byte boundaries
  for (int64_t p = lo - head + (int64_t)threadIdx.x; p < hi; p += BLOCK)
    if (p >= lo) {
      ids[p] = (uint32_t)p;
      cnt[p] = (uint32_t)i;
    }
}

template <int BLOCK>
hipError_t launch(uint32_t* ids, uint32_t* cnt, const int64_t* offsets, int64_t n, uint32_t lds, hipStream_t s) {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_row_fill<BLOCK>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_row_fill<BLOCK>, dim3((unsigned)n), dim3(BLOCK), lds, s, ids, cnt, offsets, n);
  return hipGetLastError();
}

}  // namespace

// Writes rows [offsets[i], offsets[i+1]) of ids and cnt for i < n (device
// pointers; offsets has n + 1 entries) on `stream`, blocks of `block`
// threads (64 or 256) with `lds` bytes of (unused) dynamic LDS each.
// Returns 0, or -1 for a bad argument (n outside [0, 2^31), another block
// size), or the HIP error code of the launch.
extern "C" int dgr_row_fill(uint32_t* ids, uint32_t* cnt, const int64_t* offsets, int64_t n, int block, uint32_t lds,
                            void* stream) {
  if (n < 0 || n >= (int64_t(1) << 31) || !offsets || (n > 0 && (!ids || !cnt)) || (block != 64 && block != 256))
    return -1;
  if (n == 0) return 0;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const hipError_t e = block == 256 ? launch<256>(ids, cnt, offsets, n, lds, s) : launch<64>(ids, cnt, offsets, n, lds, s);
  return e == hipSuccess ? 0 : (int)e;
}
