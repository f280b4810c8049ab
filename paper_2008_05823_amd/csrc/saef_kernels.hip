// HIP kernels for the SAEF round on gfx950 (CDNA4, wave64).
//
// Work decomposition: a layout is cut into tiles of at most a few thousand
// elements of one tensor (tile starts are multiples of 64, so one 64-bit sign
// word never spans two tiles).  Inside a tile, wave w handles 64-element
// words w*U .. w*U+U-1, then strides by 4*U words; lane i of a wave owns
// element 64*word + i, so every global load/store of a wave is one contiguous
// 256-byte segment and the sign word of those 64 elements is a single
// wave-wide ballot.
//
// Layer-wise scale (Eq. (2), one scale per tensor): every workgroup adds the
// exact integer sum of floor(|v| 2^80) over its tile to a 128-bit accumulator
// of (worker, tensor) with two 64-bit atomics, then takes an arrival ticket;
// the workgroup that arrives last converts the total into the fp32 scale and
// clears the accumulator for the next launch.  Integer addition is
// associative, so the scale does not depend on the tiling or on the order in
// which workgroups arrive.
//
// Single pass: the error update e = Delta - C(Delta) needs the scale of the
// whole tensor, which is known only after every tile was read.  The kernels
// therefore store Delta (before its correction) and leave the correction
// pending: the next kernel that reads the buffer subtracts
// (bit ? scale : -scale) on the fly.  The materialize kernel applies the
// pending correction for callers that want plain values.
#include "saef_internal.h"

namespace saef {
namespace {

typedef unsigned long long u64;

constexpr uint32_t kAbsLimitBits = 0x49000000u;  // bit pattern of 2^19

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Adds floor(|v| * 2^80) to the 128-bit integer (hi, lo); `a` is the bit
// pattern of |v| and must be below that of 2^19.
__device__ __forceinline__ void add_fixed(uint32_t a, u64& lo, u64& hi) {
  uint32_t ex = a >> 23;
  uint32_t m = a & 0x7FFFFFu;
  if (ex != 0) {
    m |= 0x800000u;
  } else {
    ex = 1;  // subnormal: m * 2^-149
  }
  // |v| = m * 2^(ex - 150), so |v| * 2^80 = m * 2^(ex - 70)
  const int sh = (int)ex - 70;
  u64 vlo, vhi;
  if (sh >= 64) {
    vlo = 0;
    vhi = (u64)m << (sh - 64);
  } else if (sh > 0) {
    vlo = (u64)m << sh;
    vhi = (u64)m >> (64 - sh);
  } else if (sh == 0) {
    vlo = m;
    vhi = 0;
  } else {
    vlo = (sh > -32) ? (u64)(m >> (-sh)) : 0ull;
    vhi = 0;
  }
  lo += vlo;
  hi += vhi + (lo < vlo ? 1ull : 0ull);
}

__device__ __forceinline__ void add128(u64& lo, u64& hi, u64 olo, u64 ohi) {
  const u64 n = lo + olo;
  hi += ohi + (n < lo ? 1ull : 0ull);
  lo = n;
}

__device__ __forceinline__ void wave_sum128(u64& lo, u64& hi) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) {
    const u64 olo = __shfl_xor(lo, off);
    const u64 ohi = __shfl_xor(hi, off);
    add128(lo, hi, olo, ohi);
  }
}

// Nearest binary64 to the 128-bit integer (hi, lo), ties to even.
__device__ double u128_to_f64(u64 hi, u64 lo) {
  if (hi == 0) return (double)lo;
  const int bits = 64 - __clzll((long long)hi);  // significant bits in hi
  u64 top, rest;
  if (bits == 64) {
    top = hi;
    rest = lo;
  } else {
    top = (hi << (64 - bits)) | (lo >> bits);
    rest = lo << (64 - bits);
  }
  // keep the discarded bits as a sticky bit (round to odd at 64 bits), so the
  // single rounding 64 -> 53 bits below is the correct one
  top |= (rest != 0) ? 1ull : 0ull;
  return ldexp((double)top, bits);
}

// Eq. (2) scale ||v||_1 / n from the exact sum S = sum floor(|v| 2^80):
// fp32( fp64( fp64(S) / n ) * 2^-80 ).
__device__ float scale_from_sum(u64 hi, u64 lo, int64_t n) {
  const double s = u128_to_f64(hi, lo);
  const double mean = s / (double)n;
  return (float)(mean * 0x1p-80);
}

__device__ __forceinline__ float corr(bool bit, float s) { return bit ? s : -s; }

__device__ __forceinline__ bool bit_of(u64 word, int lane) {
  return ((word >> lane) & 1ull) != 0;
}

// Reduce the per-lane exact sums of the workgroup, add them to the
// accumulator of (row, l) and, in the last workgroup to arrive, write the
// tensor's scale to *scale_out.
__device__ void block_finish(const DevLayout& lay, int row, int l, u64 lo, u64 hi, bool bad,
                             float* scale_out) {
  __shared__ u64 s_lo[kWaves];
  __shared__ u64 s_hi[kWaves];
  wave_sum128(lo, hi);
  const int w = threadIdx.x / kWave;
  if (lane_id() == 0) {
    s_lo[w] = lo;
    s_hi[w] = hi;
  }
  const int any_bad = __syncthreads_or(bad ? 1 : 0);
  if (threadIdx.x != 0) return;
  u64 tlo = 0, thi = 0;
  for (int i = 0; i < kWaves; ++i) add128(tlo, thi, s_lo[i], s_hi[i]);
  if (any_bad) atomicOr(lay.status, kStatusRange);

  const size_t idx = (size_t)row * lay.L + l;
  u64* a = lay.acc + (idx * kSlots + (blockIdx.x & (kSlots - 1))) * 2;
  const u64 old = atomicAdd(a, tlo);
  const u64 carry = (old + tlo < old) ? 1ull : 0ull;
  atomicAdd(a + 1, thi + carry);
  __threadfence();
  const unsigned ticket = atomicAdd(lay.cnt + idx, 1u);
  if (ticket != (unsigned)lay.tensors[l].ntiles - 1) return;

  // last arrival: every other tile of (row, l) has added its part
  __threadfence();
  u64 slo = 0, shi = 0;
  for (int sl = 0; sl < kSlots; ++sl) {
    u64* as = lay.acc + (idx * kSlots + sl) * 2;
    const u64 plo = atomicExch(as, 0ull);
    const u64 phi = atomicExch(as + 1, 0ull);
    add128(slo, shi, plo, phi);
  }
  atomicExch(lay.cnt + idx, 0u);
  *scale_out = scale_from_sum(shi, slo, lay.tensors[l].n);
}

// ------------------------------------------------------------------ compress
// Grid: n_tiles * K workgroups, workgroup b handles worker b % K of tile b / K.
template <bool kDecode>
__global__ __launch_bounds__(kBlock) void k_compress(DevLayout lay, int K, float lr,
                                                     const float* __restrict__ g,
                                                     float* __restrict__ e,
                                                     uint64_t* __restrict__ signs,
                                                     float* __restrict__ scales) {
  constexpr int U = 4;
  const int64_t b = blockIdx.x;
  const int k = (int)(b % K);
  const Tile tile = lay.tiles[b / K];
  const int l = tile.l;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t row = (int64_t)k * lay.d_pad + tile.start;
  const float* gk = g + row;
  float* ek = e + row;
  uint64_t* sk = signs + (int64_t)k * (lay.d_pad >> 6) + (tile.start >> 6);
  const float s_old = kDecode ? scales[(int64_t)k * lay.L + l] : 0.0f;
  const int nw = (tile.count + 63) >> 6;

  u64 lo = 0, hi = 0;
  bool bad = false;
  for (int w0 = wave * U; w0 < nw; w0 += kWaves * U) {
    float gv[U], ev[U];
    u64 ow[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = (w0 + u) * 64 + lane;
      const bool ok = (w0 + u < nw) && j < tile.count;
      gv[u] = ok ? gk[j] : 0.0f;
      ev[u] = ok ? ek[j] : 0.0f;
      ow[u] = (kDecode && w0 + u < nw) ? sk[w0 + u] : 0ull;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int w = w0 + u;
      if (w >= nw) break;
      const int j = w * 64 + lane;
      const bool ok = j < tile.count;
      float ev2 = ev[u];
      if (kDecode) ev2 = ev2 - corr(bit_of(ow[u], lane), s_old);
      // Delta^(k) = e^(k) + lr * g^(k), one rounding
      const float p = __builtin_fmaf(lr, gv[u], ev2);
      const u64 word = __ballot(ok && p >= 0.0f);
      if (lane == 0) sk[w] = word;
      if (ok) {
        const uint32_t a = __float_as_uint(p) & 0x7FFFFFFFu;
        if (a < kAbsLimitBits) {
          add_fixed(a, lo, hi);
        } else {
          bad = true;
        }
        ek[j] = p;
      }
    }
  }
  block_finish(lay, k, l, lo, hi, bad, scales + (int64_t)k * lay.L + l);
}

// ------------------------------------------------------------------ aggregate
// Grid: n_tiles workgroups.  mean = (sum_k +-scale_k in binary64, k order)/K.
template <int kMode, bool kDecode, bool kAvg>
__global__ __launch_bounds__(kBlock) void k_aggregate(DevLayout lay, int K, double inv_k,
                                                      const uint64_t* __restrict__ signs,
                                                      const float* __restrict__ scales,
                                                      float* __restrict__ avg,
                                                      float* __restrict__ es,
                                                      uint64_t* __restrict__ ss,
                                                      float* __restrict__ sscales,
                                                      float* __restrict__ x) {
  constexpr int U = 2;
  const Tile tile = lay.tiles[blockIdx.x];
  const int l = tile.l;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t W = lay.d_pad >> 6;
  const int64_t gw0 = tile.start >> 6;
  const int nw = (tile.count + 63) >> 6;
  const float s_srv_old = (kMode == 1 && kDecode) ? sscales[l] : 0.0f;

  u64 lo = 0, hi = 0;
  bool bad = false;
  for (int w0 = wave * U; w0 < nw; w0 += kWaves * U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int w = w0 + u;
      if (w >= nw) break;
      const int j = w * 64 + lane;
      const bool ok = j < tile.count;
      const int64_t i = tile.start + j;
      double acc = 0.0;
      for (int k = 0; k < K; ++k) {
        const u64 word = signs[(int64_t)k * W + gw0 + w];
        const float s = scales[(int64_t)k * lay.L + l];
        acc += (double)corr(bit_of(word, lane), s);
      }
      const float mean = (inv_k != 0.0) ? (float)(acc * inv_k) : (float)(acc / (double)K);
      if (kAvg && ok) avg[i] = mean;
      if (kMode == 1) {
        float ev = ok ? es[i] : 0.0f;
        if (kDecode) ev = ev - corr(bit_of(ss[gw0 + w], lane), s_srv_old);
        // Delta = e + (1/K) sum_k C(Delta^(k))
        const float D = ev + mean;
        const u64 word = __ballot(ok && D >= 0.0f);
        if (lane == 0) ss[gw0 + w] = word;
        if (ok) {
          const uint32_t a = __float_as_uint(D) & 0x7FFFFFFFu;
          if (a < kAbsLimitBits) {
            add_fixed(a, lo, hi);
          } else {
            bad = true;
          }
          es[i] = D;
        }
      } else if (ok) {
        x[i] = x[i] - mean;  // single-way: the mean itself comes back
      }
    }
  }
  if (kMode == 1) block_finish(lay, lay.k_max, l, lo, hi, bad, sscales + l);
}

// ------------------------------------------------------------------ step ahead
// Grid: n_tiles workgroups, each handles all K workers of its tile so x is
// read once.
template <bool kDecX, bool kDecE, bool kAverage, bool kXh>
__global__ __launch_bounds__(kBlock) void k_step_ahead(DevLayout lay, int K, double inv_k,
                                                       float* __restrict__ x,
                                                       const uint64_t* __restrict__ ss,
                                                       const float* __restrict__ sscales,
                                                       float* __restrict__ e,
                                                       const uint64_t* __restrict__ signs,
                                                       const float* __restrict__ scales,
                                                       float* __restrict__ xh) {
  constexpr int U = 2;
  const Tile tile = lay.tiles[blockIdx.x];
  const int l = tile.l;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t d_pad = lay.d_pad;
  const int64_t W = d_pad >> 6;
  const int64_t gw0 = tile.start >> 6;
  const int nw = (tile.count + 63) >> 6;
  const float s_srv = kDecX ? sscales[l] : 0.0f;

  for (int w0 = wave * U; w0 < nw; w0 += kWaves * U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int w = w0 + u;
      if (w >= nw) break;
      const int j = w * 64 + lane;
      const bool ok = j < tile.count;
      const int64_t i = tile.start + j;
      float xv = 0.0f;
      if ((kXh || kDecX) && ok) xv = x[i];
      if (kDecX) {
        xv = xv - corr(bit_of(ss[gw0 + w], lane), s_srv);  // pending re-update
        if (ok) x[i] = xv;
      }
      if (kAverage) {
        // e^(k) <- (1/K) sum_k e^(k)
        double acc = 0.0;
        for (int k = 0; k < K; ++k) {
          float ev = ok ? e[(int64_t)k * d_pad + i] : 0.0f;
          if (kDecE) {
            ev = ev - corr(bit_of(signs[(int64_t)k * W + gw0 + w], lane),
                           scales[(int64_t)k * lay.L + l]);
          }
          acc += (double)ev;
        }
        const float m = (inv_k != 0.0) ? (float)(acc * inv_k) : (float)(acc / (double)K);
        if (ok) {
          for (int k = 0; k < K; ++k) {
            e[(int64_t)k * d_pad + i] = m;
            if (kXh) xh[(int64_t)k * d_pad + i] = xv - m;
          }
        }
      } else if (kXh) {
        // x^(k)_{t+1/2} = x_t - e^(k)_t
        for (int k = 0; k < K; ++k) {
          float ev = ok ? e[(int64_t)k * d_pad + i] : 0.0f;
          if (kDecE) {
            ev = ev - corr(bit_of(signs[(int64_t)k * W + gw0 + w], lane),
                           scales[(int64_t)k * lay.L + l]);
          }
          if (ok) xh[(int64_t)k * d_pad + i] = xv - ev;
        }
      }
    }
  }
}

// ------------------------------------------------------------------ materialize
// Grid: n_tiles * rows, rows = K (+1 when the server row is requested); row K
// is the server error and the weights.
__global__ __launch_bounds__(kBlock) void k_materialize(
    DevLayout lay, int K, int rows, int mode, const float* __restrict__ e,
    const uint64_t* __restrict__ signs, const float* __restrict__ scales,
    float* __restrict__ e_out, const float* __restrict__ es, const float* __restrict__ x,
    const uint64_t* __restrict__ ss, const float* __restrict__ sscales,
    float* __restrict__ es_out, float* __restrict__ x_out) {
  const int64_t b = blockIdx.x;
  const int row = (int)(b % rows);
  const Tile tile = lay.tiles[b / rows];
  const int l = tile.l;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int64_t d_pad = lay.d_pad;
  const int64_t gw0 = tile.start >> 6;
  const int nw = (tile.count + 63) >> 6;
  if (row < K) {
    if (e_out == nullptr) return;
    const float s = scales[(int64_t)row * lay.L + l];
    const uint64_t* sk = signs + (int64_t)row * (d_pad >> 6) + gw0;
    for (int w = wave; w < nw; w += kWaves) {
      const int j = w * 64 + lane;
      if (j < tile.count) {
        const int64_t i = (int64_t)row * d_pad + tile.start + j;
        e_out[i] = e[i] - corr(bit_of(sk[w], lane), s);
      }
    }
    return;
  }
  const float s = (mode == 1) ? sscales[l] : 0.0f;
  for (int w = wave; w < nw; w += kWaves) {
    const int j = w * 64 + lane;
    if (j >= tile.count) continue;
    const int64_t i = tile.start + j;
    if (mode == 1) {
      const float c = corr(bit_of(ss[gw0 + w], lane), s);
      if (es_out) es_out[i] = es[i] - c;
      if (x_out) x_out[i] = x[i] - c;
    } else {
      if (es_out) es_out[i] = 0.0f;
      if (x_out) x_out[i] = x[i];
    }
  }
}

double inv_pow2(int K) { return (K & (K - 1)) == 0 ? 1.0 / (double)K : 0.0; }

}  // namespace

hipError_t launch_compress(const DevLayout& lay, int K, float lr, const float* g, float* e,
                           uint64_t* signs, float* scales, bool decode, hipStream_t s) {
  const dim3 grid((unsigned)(lay.n_tiles * K));
  if (decode) {
    hipLaunchKernelGGL(k_compress<true>, grid, dim3(kBlock), 0, s, lay, K, lr, g, e, signs,
                       scales);
  } else {
    hipLaunchKernelGGL(k_compress<false>, grid, dim3(kBlock), 0, s, lay, K, lr, g, e, signs,
                       scales);
  }
  return hipGetLastError();
}

hipError_t launch_aggregate(const DevLayout& lay, int K, int mode, const uint64_t* signs,
                            const float* scales, float* avg, float* e_srv, uint64_t* srv_signs,
                            float* srv_scales, float* x, bool decode, hipStream_t s) {
  const dim3 grid((unsigned)lay.n_tiles);
  const double ik = inv_pow2(K);
#define SAEF_AGG(M, D, A)                                                                  \
  hipLaunchKernelGGL((k_aggregate<M, D, A>), grid, dim3(kBlock), 0, s, lay, K, ik, signs, \
                     scales, avg, e_srv, srv_signs, srv_scales, x)
  const bool a = avg != nullptr;
  if (mode == 1) {
    if (decode) {
      if (a) SAEF_AGG(1, true, true); else SAEF_AGG(1, true, false);
    } else {
      if (a) SAEF_AGG(1, false, true); else SAEF_AGG(1, false, false);
    }
  } else {
    if (a) SAEF_AGG(0, false, true); else SAEF_AGG(0, false, false);
  }
#undef SAEF_AGG
  return hipGetLastError();
}

hipError_t launch_step_ahead(const DevLayout& lay, int K, float* x, const uint64_t* srv_signs,
                             const float* srv_scales, bool decode_x, float* e,
                             const uint64_t* signs, const float* scales, bool decode_e,
                             bool average, float* xh, hipStream_t s) {
  const dim3 grid((unsigned)lay.n_tiles);
  const double ik = inv_pow2(K);
#define SAEF_SA(DX, DE, AV, XH)                                                             \
  hipLaunchKernelGGL((k_step_ahead<DX, DE, AV, XH>), grid, dim3(kBlock), 0, s, lay, K, ik, \
                     x, srv_signs, srv_scales, e, signs, scales, xh)
  const bool h = xh != nullptr;
  if (!decode_x && !decode_e) {
    if (average) {
      if (h) SAEF_SA(false, false, true, true); else SAEF_SA(false, false, true, false);
    } else {
      SAEF_SA(false, false, false, true);
    }
  } else if (decode_x && decode_e) {
    if (average) SAEF_SA(true, true, true, true); else SAEF_SA(true, true, false, true);
  } else if (!decode_x && decode_e) {
    if (average) SAEF_SA(false, true, true, true); else SAEF_SA(false, true, false, true);
  } else {
    return hipErrorInvalidValue;  // decode_x without decode_e is never requested
  }
#undef SAEF_SA
  return hipGetLastError();
}

hipError_t launch_materialize(const DevLayout& lay, int K, int mode, const float* e,
                              const uint64_t* signs, const float* scales, float* e_out,
                              const float* e_srv, const float* x, const uint64_t* srv_signs,
                              const float* srv_scales, float* e_srv_out, float* x_out,
                              hipStream_t s) {
  const int k_rows = e_out != nullptr ? K : 0;
  const int rows = k_rows + ((e_srv_out != nullptr || x_out != nullptr) ? 1 : 0);
  if (rows == 0) return hipSuccess;
  const dim3 grid((unsigned)(lay.n_tiles * rows));
  hipLaunchKernelGGL(k_materialize, grid, dim3(kBlock), 0, s, lay, k_rows, rows, mode, e, signs,
                     scales, e_out, e_srv, x, srv_signs, srv_scales, e_srv_out, x_out);
  return hipGetLastError();
}

}  // namespace saef
