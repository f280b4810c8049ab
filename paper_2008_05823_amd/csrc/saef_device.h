// Device helpers shared by the kernel translation units of the SAEF library.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "saef_internal.h"

namespace saef {

typedef unsigned long long u64;

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
}

// Streaming accesses: nothing is re-read soon enough to profit from the caches.
__device__ __forceinline__ float ld_nt(const float* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_nt(float* p, float v) { __builtin_nontemporal_store(v, p); }

// Per lane: bit `lane` of the 64-bit mask ? if1 : if0, in one VALU op
// (v_cndmask with the mask as its lane condition).  The mask must be the
// same in every lane (a sign word read at a wave-uniform address); it is
// moved to scalar registers explicitly, which costs nothing when it already
// is in one.
__device__ __forceinline__ uint32_t sel_by_bit(u64 mask, uint32_t if1, uint32_t if0) {
  const uint32_t mlo = __builtin_amdgcn_readfirstlane((uint32_t)mask);
  const uint32_t mhi = __builtin_amdgcn_readfirstlane((uint32_t)(mask >> 32));
  const u64 m = ((u64)mhi << 32) | mlo;
  uint32_t r;
  asm("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(r) : "v"(if0), "v"(if1), "s"(m));
  return r;
}
__device__ __forceinline__ float sel_by_bit(u64 mask, float if1, float if0) {
  return __uint_as_float(sel_by_bit(mask, __float_as_uint(if1), __float_as_uint(if0)));
}

// (1/K) * acc, binary64; inv_k is 1/K when K is a power of two (exact), else 0.
__device__ __forceinline__ double mean_of(double acc, double inv_k, int K) {
  return (inv_k != 0.0) ? acc * inv_k : acc / (double)K;
}

// Host: 1/K when K is a power of two (then acc * inv_k == acc / K exactly), else 0.
inline double inv_pow2(int K) { return (K & (K - 1)) == 0 ? 1.0 / (double)K : 0.0; }

// The (row, tile) of workgroup b when each tile has `rows` workgroups: along
// a run, tile by tile, then the next row on the same run.  ti may be past the
// last tile (the grid is rounded up to whole groups).
__device__ __forceinline__ void run_tile_of(unsigned b, int rows, int s, int& row, int64_t& ti) {
  const unsigned xcd = b % kXcds, r = b / kXcds;
  const unsigned j = r & ((1u << s) - 1u);
  const unsigned u = r >> s;
  row = (int)(u % (unsigned)rows);
  const int64_t grp = u / (unsigned)rows;
  ti = ((grp * kXcds + xcd) << s) + j;
}

// Workgroups of 4 waves, one wave per tile.
inline unsigned per_wave_grid(const DevLayout& lay) {
  return (unsigned)((lay.n_tiles + kWaves - 1) / kWaves);
}

}  // namespace saef

// All launches go through hipExtLaunchKernelGGL so that an optional event
// pair (a LaunchEvents `ev` in scope) is stamped by the dispatch itself.
#define SAEF_LAUNCH(kernel, grid, block, shmem, stream, ...) \
  hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, ev.start, ev.stop, 0, __VA_ARGS__)
