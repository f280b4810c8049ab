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

// Word 3 of a raw buffer descriptor on gfx9 parts (32-bit data format, no
// swizzle, no index stride).  A load through a raw buffer resource of n
// bytes returns 0 for a byte offset at or past n, without touching memory,
// and a store there is dropped.
constexpr int kBufWord3 = 0x00020000;
// Cache policy of a buffer access on gfx940 and later: bit 1 = nt (streaming).
constexpr int kAuxNT = 2;

typedef __amdgpu_buffer_rsrc_t Buf;

// A raw buffer resource over [p, p + bytes), bytes < 2^31.  Accesses through
// it take a 32-bit byte offset (a lane offset in a VGPR plus an immediate),
// so no 64-bit address arithmetic is spent per element, and the range check
// in the hardware replaces the per-lane guards of a ragged tail.
__device__ __forceinline__ Buf buf_of(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, kBufWord3);
}
__device__ __forceinline__ float buf_ld(Buf r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kAuxNT));
}
// x is re-read by the K workers of a tile through one XCD's L2: cached load.
__device__ __forceinline__ float buf_ld_cached(Buf r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ void buf_st(Buf r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, off, 0, kAuxNT);
}
// A 64-bit sign word at a wave-uniform byte offset (passed as the scalar
// offset of the access, so no vector register holds the address).
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u64 buf_ld_word(Buf r, uint32_t off) {
  const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, 0, off, 0);
  return ((u64)v.y << 32) | v.x;
}
__device__ __forceinline__ void buf_st_word(Buf r, uint32_t off, u64 w) {
  u32x2 v;
  v.x = (uint32_t)w;
  v.y = (uint32_t)(w >> 32);
  __builtin_amdgcn_raw_buffer_store_b64(v, r, 0, off, 0);
}

// Sign words of a buffer that no wave writes during the kernel, at a
// wave-uniform address: read through the scalar cache (s_load), straight
// into the scalar registers the inline v_cndmask takes as its mask.
typedef __attribute__((address_space(4))) const u64 ConstWord;
__device__ __forceinline__ u64 ld_word_ro(const uint64_t* p) {
  return *(ConstWord*)p;  // an address-space cast (same address)
}

// n consecutive sign words (n a power of two <= 64) of a buffer that the
// kernel also writes: one vector load, lane i holding word w0 + (i mod n)
// (vector loads see this kernel's own earlier stores; the scalar cache
// would not); word_of picks word u out of it into scalar registers.
__device__ __forceinline__ u64 buf_ld_words(Buf r, int w0, int n) {
  const uint32_t off = (uint32_t)(w0 + (int)(threadIdx.x & (unsigned)(n - 1))) * 8u;
  const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
  return ((u64)v.y << 32) | v.x;
}
__device__ __forceinline__ u64 word_of(u64 v, int u) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, u);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), u);
  return ((u64)hi << 32) | lo;
}

// v in a vector register the compiler cannot trace back to a scalar one: a
// loop-invariant operand of the inline v_cndmask (which takes only vector
// registers besides its mask) then stays in a VGPR instead of being copied
// from an SGPR at every use.
__device__ __forceinline__ float in_vgpr(float v) {
  asm volatile("" : "+v"(v));
  return v;
}

// ---- exact layer-wise L1 sum ------------------------------------------------
// S = sum_i floor(|v_i| 2^80), an integer below 2^127 when every |v_i| < 2^19
// and a tensor has at most 2^28 elements.  Per lane the terms are split in
// binary64 so that two plain fp64 sums stay exact (8 VALU operations per
// value instead of a 128-bit integer addition with shifts):
//   a = |v| (exact in binary64), t = a + 1.5 2^22 rounds a to H, a multiple
//   of 2^-30 (a < 2^21 keeps a + 1.5 2^22 in [2^22, 2^23), whose spacing is
//   2^-30); C - t = -H and a - H = a + (C - t) are exact (Sterbenz),
//   |a - H| <= 2^-31.  floor(a 2^80) = H 2^80 + floor((a - H) 2^80), and
//   the floor is a truncation: a - H < 0 only when a >= 2^-31, where a is a
//   multiple of 2^-80 (fp32 spacing at that size), so (a - H) 2^80 is an
//   integer; below 2^-57 the bits under 2^-80 are truncated as the
//   definition says (H = 0 there, a - H = a >= 0).
// With at most 16 values per lane between flushes, -sum H 2^30 <= 2^53 and
// |sum trunc((a - H) 2^80)| <= 16 2^49 = 2^53: both fp64 sums are exact.
struct ExactSum {
  double nh = 0.0;   // -sum of H
  double lq = 0.0;   // sum of trunc((a - H) 2^80)
  float mx = 0.0f;   // largest |v| seen (range check; NaN shows in nh)
  int terms = 0;     // values since the last flush (wave-uniform)

  __device__ __forceinline__ void add(float v) {
    const double a = (double)fabsf(v);
    const double t = a + 0x1.8p22;
    const double n = 0x1.8p22 - t;
    nh += n;
    lq += trunc((a + n) * 0x1p80);
    mx = fmaxf(mx, fabsf(v));
  }

  // Moves the two fp64 sums into the 128-bit integer (hi, lo) and clears
  // them: S += (-nh) 2^80 + lq = h 2^50 + lq with h = -nh 2^30.
  __device__ __forceinline__ void flush(u64& lo, u64& hi, bool& bad) {
    bad = bad || !(nh == nh) || !(lq == lq);
    const double h = -nh * 0x1p30;  // integer in [0, 2^53]
    const uint32_t h_hi = (uint32_t)(h * 0x1p-32);
    const uint32_t h_lo = (uint32_t)(h - (double)h_hi * 0x1p32);
    const double q_hd = floor(lq * 0x1p-32);  // lq integer in [-2^53, 2^53]
    const int32_t q_hi = (int32_t)q_hd;
    const uint32_t q_lo = (uint32_t)(lq - q_hd * 0x1p32);
    const u64 hv = ((u64)h_hi << 32) | h_lo;
    const u64 qv = (u64)(((int64_t)q_hi << 32) | q_lo);  // two's complement
    // (hi, lo) += hv 2^50 + qv, modulo 2^128 (the lane's total is >= 0)
    const u64 a_lo = hv << 50;
    u64 n_lo = lo + a_lo;
    hi += (hv >> 14) + (n_lo < lo ? 1ull : 0ull);
    const u64 m_lo = n_lo + qv;
    hi += (m_lo < n_lo ? 1ull : 0ull) + (q_hi < 0 ? ~0ull : 0ull);
    lo = m_lo;
    nh = 0.0;
    lq = 0.0;
    terms = 0;
  }

  // After `count` more values: flush when another pass could break the
  // 16-values-per-lane bound.
  __device__ __forceinline__ void added(int count, u64& lo, u64& hi, bool& bad) {
    terms += count;
    if (terms > 8) flush(lo, hi, bad);
  }

  __device__ __forceinline__ void finish(u64& lo, u64& hi, bool& bad) {
    flush(lo, hi, bad);
    bad = bad || !(mx < 0x1p19f);
  }
};

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
