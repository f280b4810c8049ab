// HIP kernels for the SAEF round on gfx950 (CDNA4, wave64).
//
// Work decomposition: a layout is cut into tiles of at most a few thousand
// elements of one tensor (tile starts are multiples of 64, so one 64-bit sign
// word never spans two tiles).  Inside a tile, wave w handles 64-element
// words w*U .. w*U+U-1, then strides by 4*U words; lane i of a wave owns
// element 64*word + i, so every global load/store of a wave is one contiguous
// 256-byte segment and the sign word of those 64 elements is a single
// wave-wide ballot.  Value buffers are streamed with non-temporal loads and
// stores: nothing is re-read soon enough to profit from the caches.
//
// Layer-wise scale (Eq. (2), one scale per tensor): every workgroup reduces
// the exact integer sum of floor(|v| 2^80) over its tile and stores it as a
// 128-bit partial (plain stores, no cross-workgroup atomics: on a multi-XCD
// part those go to memory-side atomics and serialise).  A small finalize
// kernel then adds the partials of each tensor and converts the total into
// the fp32 scale.  Integer addition is associative, so the scale does not
// depend on the tiling or on the order of anything.
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
constexpr int kWPW = 16;  // words per wave held in registers by the K-worker kernels

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ float ld_nt(const float* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_nt(float* p, float v) { __builtin_nontemporal_store(v, p); }

// Adds floor(|v| * 2^80) to the 128-bit integer (hi, lo); `a` is the bit
// pattern of |v| and must be below that of 2^19.
__device__ __forceinline__ void add_fixed(uint32_t a, u64& lo, u64& hi) {
  uint32_t ex = a >> 23;
  uint32_t m = a & 0x7FFFFFu;
  m |= (ex != 0) ? 0x800000u : 0u;
  ex = (ex != 0) ? ex : 1u;  // subnormal: m * 2^-149
  // |v| = m * 2^(ex - 150), so |v| * 2^80 = m * 2^(ex - 70), ex - 70 in [-69, 75]
  const int sh = (int)ex - 70;
  // split as t * 2^(32 q) with t = m * 2^(sh mod 32) < 2^55, q in {0, 1, 2}
  u64 t;
  int q;
  if (sh >= 0) {
    q = sh >> 5;
    t = (u64)m << (sh & 31);
  } else {
    q = 0;
    t = (sh > -32) ? (u64)(m >> (-sh)) : 0ull;
  }
  const u64 vlo = (q == 0) ? t : ((q == 1) ? (t << 32) : 0ull);
  const u64 vhi = (q == 0) ? 0ull : ((q == 1) ? (t >> 32) : t);
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

// The 32-bit half of the sign word at p that holds bit `lane` (a per-lane
// load: one VGPR per word instead of a scalar register pair).
__device__ __forceinline__ uint32_t half_word(const uint64_t* p, int lane) {
  return reinterpret_cast<const uint32_t*>(p)[lane >> 5];
}
__device__ __forceinline__ bool half_bit(uint32_t h, int lane) {
  return ((h >> (lane & 31)) & 1u) != 0;
}

// Adds up the per-lane exact sums of the workgroup and stores the total as
// the partial of (row, tile); raises the range flag if any lane saw a value
// outside the exact-sum range.
__device__ void block_partial(const DevLayout& lay, int row, int64_t tile, u64 lo, u64 hi,
                              bool bad) {
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
  u64* p = lay.part + ((int64_t)row * lay.n_tiles + tile) * 2;
  p[0] = tlo;
  p[1] = thi;
  if (any_bad) atomicOr(lay.status, kStatusRange);
}

// ------------------------------------------------------------------ compress
// Grid: n_tiles * K workgroups, workgroup b handles worker b % K of tile b / K.
template <bool kDecode>
__global__ __launch_bounds__(kBlock) void k_compress(DevLayout lay, int K, float lr,
                                                     const float* __restrict__ g,
                                                     float* __restrict__ e,
                                                     uint64_t* __restrict__ signs,
                                                     const float* __restrict__ scales) {
  constexpr int U = 4;
  const int64_t b = blockIdx.x;
  const int k = (int)(b % K);
  const int64_t ti = b / K;
  const Tile tile = lay.tiles[ti];
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
    uint32_t ow[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = (w0 + u) * 64 + lane;
      const bool ok = (w0 + u < nw) && j < tile.count;
      gv[u] = ok ? ld_nt(gk + j) : 0.0f;
      ev[u] = ok ? ld_nt(ek + j) : 0.0f;
      ow[u] = (kDecode && w0 + u < nw) ? half_word(sk + w0 + u, lane) : 0u;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int w = w0 + u;
      if (w >= nw) break;
      const int j = w * 64 + lane;
      const bool ok = j < tile.count;
      float ev2 = ev[u];
      if (kDecode) ev2 = ev2 - corr(half_bit(ow[u], lane), s_old);
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
        st_nt(ek + j, p);
      }
    }
  }
  block_partial(lay, k, ti, lo, hi, bad);
}

// ------------------------------------------------------------------ finalize
// Grid: rows * L single-wave workgroups; workgroup b adds the tile partials
// of tensor b % L for row b / L (or the server row) and writes the scale.
__global__ __launch_bounds__(kWave) void k_finalize(DevLayout lay, int server,
                                                    float* __restrict__ scales) {
  const int64_t b = blockIdx.x;
  const int l = (int)(b % lay.L);
  const int r = (int)(b / lay.L);
  const int row = server ? lay.k_max : r;
  const TensorInfo t = lay.tensors[l];
  const u64* p = lay.part + ((int64_t)row * lay.n_tiles + t.first_tile) * 2;
  u64 lo = 0, hi = 0;
  for (int i = threadIdx.x; i < t.ntiles; i += kWave) add128(lo, hi, p[2 * i], p[2 * i + 1]);
  wave_sum128(lo, hi);
  if (threadIdx.x == 0) scales[server ? l : (int64_t)r * lay.L + l] = scale_from_sum(hi, lo, t.n);
}

// ------------------------------------------------------------------ aggregate
// One pass of a wave over kWPW words (elements base + 64 u, u < kWPW) of a
// tile: the wave holds the words in registers and walks the K worker
// messages in order, mean = (sum_k +-scale_k in binary64, k order) / K.
// kFull: all kWPW words lie inside the tile (no per-lane guards); otherwise
// only the first nv words are present and element base + 64 u exists iff
// 64 u < lim.
template <int kMode, bool kDecode, bool kAvg, bool kFull, int kN>
__device__ __forceinline__ void aggregate_pass(const DevLayout& lay, int K, double inv_k, int l,
                                               int64_t base, int64_t gw, int nv, int lim,
                                               const uint64_t* __restrict__ signs,
                                               const float* __restrict__ scales,
                                               float* __restrict__ avg, float* __restrict__ es,
                                               uint64_t* __restrict__ ss, float s_srv_old,
                                               float* __restrict__ x, u64& lo, u64& hi,
                                               bool& bad) {
  const int lane = lane_id();
  const int64_t W = lay.d_pad >> 6;
  float v[kN];
#pragma unroll
  for (int u = 0; u < kN; ++u) {
    v[u] = 0.0f;
    if (kFull || (u < nv && u * 64 < lim))
      v[u] = (kMode == 1) ? ld_nt(es + base + u * 64) : ld_nt(x + base + u * 64);
  }
  double acc[kN];
#pragma unroll
  for (int u = 0; u < kN; ++u) acc[u] = 0.0;
  for (int k = 0; k < K; ++k) {
    const double sd = (double)scales[(int64_t)k * lay.L + l];
    const uint64_t* sk = signs + (int64_t)k * W + gw;
    uint32_t hw[kN];
#pragma unroll
    for (int u = 0; u < kN; ++u) hw[u] = (kFull || u < nv) ? half_word(sk + u, lane) : 0u;
#pragma unroll
    for (int u = 0; u < kN; ++u) acc[u] += half_bit(hw[u], lane) ? sd : -sd;
  }
#pragma unroll
  for (int u = 0; u < kN; ++u) {
    if (!kFull && u >= nv) continue;
    const bool ok = kFull || u * 64 < lim;
    const float mean = (inv_k != 0.0) ? (float)(acc[u] * inv_k) : (float)(acc[u] / (double)K);
    const int64_t i = base + u * 64;
    if (kAvg && ok) avg[i] = mean;
    if (kMode == 1) {
      float ev = v[u];
      if (kDecode) ev = ev - corr(half_bit(half_word(ss + gw + u, lane), lane), s_srv_old);
      // Delta = e + (1/K) sum_k C(Delta^(k))
      const float D = ev + mean;
      const u64 word = __ballot(ok && D >= 0.0f);
      if (lane == 0) ss[gw + u] = word;
      if (ok) {
        const uint32_t a = __float_as_uint(D) & 0x7FFFFFFFu;
        if (a < kAbsLimitBits) {
          add_fixed(a, lo, hi);
        } else {
          bad = true;
        }
        st_nt(es + i, D);
      }
    } else if (ok) {
      st_nt(x + i, v[u] - mean);  // single-way: the mean itself comes back
    }
  }
}

// Grid: n_tiles workgroups; wave w takes passes of kWPW words starting at
// word w*kWPW, striding by 4*kWPW words.
template <int kMode, bool kDecode, bool kAvg>
__global__ __launch_bounds__(kBlock) void k_aggregate(DevLayout lay, int K, double inv_k,
                                                      const uint64_t* __restrict__ signs,
                                                      const float* __restrict__ scales,
                                                      float* __restrict__ avg,
                                                      float* __restrict__ es,
                                                      uint64_t* __restrict__ ss,
                                                      const float* __restrict__ sscales,
                                                      float* __restrict__ x) {
  const int64_t ti = blockIdx.x;
  const Tile tile = lay.tiles[ti];
  const int l = tile.l;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int nw = (tile.count + 63) >> 6;
  const float s_srv_old = (kMode == 1 && kDecode) ? sscales[l] : 0.0f;
  u64 lo = 0, hi = 0;
  bool bad = false;
  for (int wb = wave * kWPW; wb < nw; wb += kWaves * kWPW) {
    const int64_t base = tile.start + wb * 64 + lane;
    const int64_t gw = (tile.start >> 6) + wb;
    if ((wb + kWPW) * 64 <= tile.count) {
      aggregate_pass<kMode, kDecode, kAvg, true, kWPW>(lay, K, inv_k, l, base, gw, kWPW, 0, signs,
                                                       scales, avg, es, ss, s_srv_old, x, lo, hi,
                                                       bad);
    } else {
      // tail of the tile: one word at a time, guarded per lane
      const int nv = min(kWPW, nw - wb);
      for (int u = 0; u < nv; ++u) {
        aggregate_pass<kMode, kDecode, kAvg, false, 1>(
            lay, K, inv_k, l, base + u * 64, gw + u, 1, tile.count - (wb + u) * 64 - lane,
            signs, scales, avg, es, ss, s_srv_old, x, lo, hi, bad);
      }
    }
  }
  if (kMode == 1) block_partial(lay, lay.k_max, ti, lo, hi, bad);
}

// ------------------------------------------------------------------ step ahead
// One pass over kWPW words of a tile (same conventions as aggregate_pass):
// x is read once into registers, then the K workers are walked in order.
template <bool kDecX, bool kDecE, bool kAverage, bool kXh, bool kFull, int kN>
__device__ __forceinline__ void step_pass(const DevLayout& lay, int K, double inv_k, int l,
                                          int64_t base, int64_t gw, int nv, int lim,
                                          float* __restrict__ x, const uint64_t* __restrict__ ss,
                                          float s_srv, float* __restrict__ e,
                                          const uint64_t* __restrict__ signs,
                                          const float* __restrict__ scales,
                                          float* __restrict__ xh) {
  const int lane = lane_id();
  const int64_t d_pad = lay.d_pad;
  const int64_t W = d_pad >> 6;
  float xv[kN];
#pragma unroll
  for (int u = 0; u < kN; ++u) {
    xv[u] = 0.0f;
    if ((kXh || kDecX) && (kFull || (u < nv && u * 64 < lim))) xv[u] = ld_nt(x + base + u * 64);
  }
  if (kDecX) {
#pragma unroll
    for (int u = 0; u < kN; ++u) {
      if (!kFull && u >= nv) continue;
      // pending re-update x <- x - C(Delta) of the previous iteration
      xv[u] = xv[u] - corr(half_bit(half_word(ss + gw + u, lane), lane), s_srv);
      if (kFull || u * 64 < lim) st_nt(x + base + u * 64, xv[u]);
    }
  }
  if (kAverage) {
    // e^(k) <- (1/K) sum_k e^(k), binary64 sum in worker order
    double acc[kN];
#pragma unroll
    for (int u = 0; u < kN; ++u) acc[u] = 0.0;
    for (int k = 0; k < K; ++k) {
      const float* ek = e + (int64_t)k * d_pad + base;
      const uint64_t* sk = signs + (int64_t)k * W + gw;
      const float s = kDecE ? scales[(int64_t)k * lay.L + l] : 0.0f;
      float ev[kN];
      uint32_t hw[kN];
#pragma unroll
      for (int u = 0; u < kN; ++u) {
        ev[u] = 0.0f;
        if (kFull || (u < nv && u * 64 < lim)) ev[u] = ld_nt(ek + u * 64);
        hw[u] = (kDecE && (kFull || u < nv)) ? half_word(sk + u, lane) : 0u;
      }
#pragma unroll
      for (int u = 0; u < kN; ++u) {
        if (kDecE) ev[u] = ev[u] - corr(half_bit(hw[u], lane), s);
        acc[u] += (double)ev[u];
      }
    }
    float m[kN];
#pragma unroll
    for (int u = 0; u < kN; ++u)
      m[u] = (inv_k != 0.0) ? (float)(acc[u] * inv_k) : (float)(acc[u] / (double)K);
    for (int k = 0; k < K; ++k) {
      float* ek = e + (int64_t)k * d_pad + base;
      float* hk = xh + (int64_t)k * d_pad + base;
#pragma unroll
      for (int u = 0; u < kN; ++u) {
        if (kFull || (u < nv && u * 64 < lim)) {
          st_nt(ek + u * 64, m[u]);
          if (kXh) st_nt(hk + u * 64, xv[u] - m[u]);
        }
      }
    }
  } else if (kXh) {
    // x^(k)_{t+1/2} = x_t - e^(k)_t
    for (int k = 0; k < K; ++k) {
      const float* ek = e + (int64_t)k * d_pad + base;
      float* hk = xh + (int64_t)k * d_pad + base;
      const uint64_t* sk = signs + (int64_t)k * W + gw;
      const float s = kDecE ? scales[(int64_t)k * lay.L + l] : 0.0f;
      float ev[kN];
      uint32_t hw[kN];
#pragma unroll
      for (int u = 0; u < kN; ++u) {
        ev[u] = 0.0f;
        if (kFull || (u < nv && u * 64 < lim)) ev[u] = ld_nt(ek + u * 64);
        hw[u] = (kDecE && (kFull || u < nv)) ? half_word(sk + u, lane) : 0u;
      }
#pragma unroll
      for (int u = 0; u < kN; ++u) {
        if (kDecE) ev[u] = ev[u] - corr(half_bit(hw[u], lane), s);
        if (kFull || (u < nv && u * 64 < lim)) st_nt(hk + u * 64, xv[u] - ev[u]);
      }
    }
  }
}

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
  const Tile tile = lay.tiles[blockIdx.x];
  const int l = tile.l;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int nw = (tile.count + 63) >> 6;
  const float s_srv = kDecX ? sscales[l] : 0.0f;
  for (int wb = wave * kWPW; wb < nw; wb += kWaves * kWPW) {
    const int64_t base = tile.start + wb * 64 + lane;
    const int64_t gw = (tile.start >> 6) + wb;
    if ((wb + kWPW) * 64 <= tile.count) {
      step_pass<kDecX, kDecE, kAverage, kXh, true, kWPW>(lay, K, inv_k, l, base, gw, kWPW, 0, x,
                                                         ss, s_srv, e, signs, scales, xh);
    } else {
      // tail of the tile: one word at a time, guarded per lane
      const int nv = min(kWPW, nw - wb);
      for (int u = 0; u < nv; ++u) {
        step_pass<kDecX, kDecE, kAverage, kXh, false, 1>(
            lay, K, inv_k, l, base + u * 64, gw + u, 1, tile.count - (wb + u) * 64 - lane, x, ss,
            s_srv, e, signs, scales, xh);
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
    const float s = scales[(int64_t)row * lay.L + l];
    const uint64_t* sk = signs + (int64_t)row * (d_pad >> 6) + gw0;
    for (int w = wave; w < nw; w += kWaves) {
      const int j = w * 64 + lane;
      if (j < tile.count) {
        const int64_t i = (int64_t)row * d_pad + tile.start + j;
        e_out[i] = e[i] - corr(half_bit(half_word(sk + w, lane), lane), s);
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
      const float c = corr(half_bit(half_word(ss + gw0 + w, lane), lane), s);
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
                           uint64_t* signs, const float* scales, bool decode, hipStream_t s) {
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

hipError_t launch_finalize(const DevLayout& lay, int K, bool server, float* scales,
                           hipStream_t s) {
  const dim3 grid((unsigned)((server ? 1 : K) * lay.L));
  hipLaunchKernelGGL(k_finalize, grid, dim3(kWave), 0, s, lay, server ? 1 : 0, scales);
  return hipGetLastError();
}

hipError_t launch_aggregate(const DevLayout& lay, int K, int mode, const uint64_t* signs,
                            const float* scales, float* avg, float* e_srv, uint64_t* srv_signs,
                            const float* srv_scales, float* x, bool decode, hipStream_t s) {
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
