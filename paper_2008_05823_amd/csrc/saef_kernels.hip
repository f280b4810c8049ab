// HIP kernels for the SAEF round on gfx950 (CDNA4, wave64).
//
// Work decomposition: a layout is cut into tiles of 2048 elements of one
// tensor (more for very large tensors; tile starts are multiples of 64, so a
// 64-bit sign word never spans two tiles).  Lane i of a wave owns element
// 64*word + i of the 64-element words it processes, so every global load or
// store of a wave is one contiguous 256-byte segment and the sign word of
// those 64 elements is a single wave-wide ballot.  Value buffers are
// streamed with non-temporal loads and stores (nothing is re-read soon
// enough to profit from the caches), except x, which the K workers of a
// tile read through the L2 of one XCD.
//
// Layer-wise scale (Eq. (2), one scale per tensor): the workgroup (or wave)
// that owns a tile reduces the exact integer sum of floor(|v| 2^80) over it
// and stores it as a 128-bit partial with plain stores -- no cross-workgroup
// atomics, which on a multi-XCD part go to memory-side atomics and
// serialise.  A small finalize kernel adds the partials of each tensor and
// converts the total into the fp32 scale.  Integer addition is associative,
// so the scale does not depend on the tiling or on the order of anything.
//
// Single pass: the error update e = Delta - C(Delta) needs the scale of the
// whole tensor, which is known only after every tile was read.  The kernels
// therefore store Delta (before its correction) and leave the correction
// pending: the next kernel that reads the buffer subtracts
// (bit ? scale : -scale) on the fly.  The materialize kernel applies the
// pending corrections for callers that want plain values.
#include <hip/hip_ext.h>

#include "saef_device.h"
#include "saef_internal.h"

namespace saef {
namespace {

constexpr uint32_t kAbsLimitBits = 0x49000000u;  // bit pattern of 2^19
// Words per wave per pass in the per-(tile, worker) kernels: 8, so that the
// four waves cover a 2048-element tile in one pass (momentum compression
// 727 -> 677 us at resnet50 K = 8 against 4 words; the sign kernels gain 1%).
constexpr int kU = 8;
// Words per wave per pass in the averaging kernel (it keeps kAvgChunk * kUA
// errors and sign words live; 8 was 2% slower).
constexpr int kUA = 4;

// The compression correction C(v)_i = bit ? scale : -scale.
__device__ __forceinline__ float corr(u64 word, float s) { return sel_by_bit(word, s, -s); }

// The 32-bit half of the sign word at p that holds bit `lane`, read per lane
// (a vector register instead of a scalar pair, for kernels that keep many
// words live), and the lane's bit in it.
__device__ __forceinline__ uint32_t half_word(const uint64_t* p, int lane) {
  return reinterpret_cast<const uint32_t*>(p)[lane >> 5];
}
__device__ __forceinline__ bool half_bit(uint32_t h, int lane) {
  return ((h >> (lane & 31)) & 1u) != 0;
}

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

// Exact-sum term of one value: adds it when |v| < 2^19, else flags it.
__device__ __forceinline__ void sum_abs(float v, u64& lo, u64& hi, bool& bad) {
  const uint32_t a = __float_as_uint(v) & 0x7FFFFFFFu;
  if (a < kAbsLimitBits) {
    add_fixed(a, lo, hi);
  } else {
    bad = true;  // |v| >= 2^19, Inf or NaN
  }
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


// Stores the exact partial of (row, tile) summed over the workgroup.
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
// kU words of one worker's tile starting at word w0: with kMom, the momentum
// buffer m <- fma(mu, m, g) first (one rounding); Delta = fma(lr, m or g, e)
// (e decoded when kDecode), sign words by ballot, exact-sum terms, Delta
// stored.  kFull: all kU words are whole words of the tile (no guards).
template <bool kDecode, bool kMom, bool kFull>
__device__ __forceinline__ void compress_words(int w0, int nw, int count, float lr, float mu,
                                               const float* __restrict__ gk,
                                               float* __restrict__ mk,
                                               float* __restrict__ ek,
                                               uint64_t* __restrict__ sk, float s_old, u64& lo,
                                               u64& hi, bool& bad) {
  const int lane = lane_id();
  float gv[kU], ev[kU], mv[kU];
  u64 ow[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int j = (w0 + u) * 64 + lane;
    const bool ok = kFull || ((w0 + u < nw) && j < count);
    gv[u] = ok ? ld_nt(gk + j) : 0.0f;
    ev[u] = ok ? ld_nt(ek + j) : 0.0f;
    mv[u] = (kMom && ok) ? ld_nt(mk + j) : 0.0f;
    ow[u] = (kDecode && (kFull || w0 + u < nw)) ? sk[w0 + u] : 0ull;
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int w = w0 + u;
    if (!kFull && w >= nw) continue;
    const int j = w * 64 + lane;
    const bool ok = kFull || j < count;
    float ev2 = ev[u];
    if (kDecode) ev2 = ev2 - corr(ow[u], s_old);
    float step = gv[u];
    if (kMom) {
      step = __builtin_fmaf(mu, mv[u], gv[u]);  // m^(k)_{t+1} = mu m^(k)_t + grad
      if (ok) st_nt(mk + j, step);
    }
    // Delta^(k) = e^(k) + lr * m^(k)_{t+1}, one rounding (m = grad when mu = 0)
    const float p = __builtin_fmaf(lr, step, ev2);
    const u64 word = __ballot(ok && p >= 0.0f);
    if (lane == 0) sk[w] = word;
    if (ok) {
      sum_abs(p, lo, hi, bad);
      st_nt(ek + j, p);
    }
  }
}

// Grid: n_tiles * K workgroups; workgroup b handles worker b % K of tile
// b / K.  Wave w takes words w*kU .. w*kU+kU-1 of the tile, then strides by
// 4*kU words.
template <bool kDecode, bool kMom>
__global__ __launch_bounds__(kBlock) void k_compress(DevLayout lay, int K, float lr, float mu,
                                                     const float* __restrict__ g,
                                                     float* __restrict__ m,
                                                     float* __restrict__ e,
                                                     uint64_t* __restrict__ signs,
                                                     const float* __restrict__ scales) {
  const unsigned b = blockIdx.x;
  const int k = (int)(b % (unsigned)K);
  const int64_t ti = b / (unsigned)K;
  const Tile tile = lay.tiles[ti];
  const int wave = wave_id();
  const int64_t row = (int64_t)k * lay.d_pad + tile.start;
  const float* gk = g + row;
  float* mk = kMom ? m + row : nullptr;
  float* ek = e + row;
  uint64_t* sk = signs + (int64_t)k * (lay.d_pad >> 6) + (tile.start >> 6);
  const float s_old = kDecode ? scales[(int64_t)k * lay.L + tile.l] : 0.0f;
  const int nw = (tile.count + 63) >> 6;

  u64 lo = 0, hi = 0;
  bool bad = false;
  for (int w0 = wave * kU; w0 < nw; w0 += kWaves * kU) {
    if ((w0 + kU) * 64 <= tile.count) {
      compress_words<kDecode, kMom, true>(w0, nw, tile.count, lr, mu, gk, mk, ek, sk, s_old,
                                          lo, hi, bad);
    } else {
      compress_words<kDecode, kMom, false>(w0, nw, tile.count, lr, mu, gk, mk, ek, sk, s_old,
                                           lo, hi, bad);
    }
  }
  block_partial(lay, k, ti, lo, hi, bad);
}

// ------------------------------------------------------------------ finalize
// Adds the 128-bit values v[0..n) over the workgroup (thread 0 gets the sum).
__device__ void block_sum128(const u64* __restrict__ v, int64_t n, u64& tlo, u64& thi) {
  __shared__ u64 s_lo[kWaves];
  __shared__ u64 s_hi[kWaves];
  u64 lo = 0, hi = 0;
  for (int64_t i = threadIdx.x; i < n; i += kBlock) add128(lo, hi, v[2 * i], v[2 * i + 1]);
  wave_sum128(lo, hi);
  const int w = threadIdx.x / kWave;
  if (lane_id() == 0) {
    s_lo[w] = lo;
    s_hi[w] = hi;
  }
  __syncthreads();
  tlo = 0;
  thi = 0;
  if (threadIdx.x == 0)
    for (int i = 0; i < kWaves; ++i) add128(tlo, thi, s_lo[i], s_hi[i]);
}

// Grid: rows * L * S workgroups (S = lay.fin_split); workgroup b adds the
// tile partials of part s = b % S of tensor (b / S) % L for row b / (S L)
// (or the server row).  With S = 1 it writes the tensor's scale; otherwise
// it stores a second-level partial that k_finalize2 adds up.
__global__ __launch_bounds__(kBlock) void k_finalize(DevLayout lay, int server,
                                                     float* __restrict__ scales) {
  const int S = lay.fin_split;
  const int64_t b = blockIdx.x;
  const int s = (int)(b % S);
  const int l = (int)((b / S) % lay.L);
  const int r = (int)(b / ((int64_t)S * lay.L));
  const int row = server ? lay.k_max : r;
  const TensorInfo t = lay.tensors[l];
  const int per = (t.ntiles + S - 1) / S;
  const int i0 = min(t.ntiles, s * per), i1 = min(t.ntiles, i0 + per);
  u64 tlo, thi;
  block_sum128(lay.part + ((int64_t)row * lay.n_tiles + t.first_tile + i0) * 2, i1 - i0, tlo,
               thi);
  if (threadIdx.x != 0) return;
  if (S == 1) {
    scales[server ? l : (int64_t)r * lay.L + l] = scale_from_sum(thi, tlo, t.n);
  } else {
    u64* q = lay.part2 + (((int64_t)row * lay.L + l) * S + s) * 2;
    q[0] = tlo;
    q[1] = thi;
  }
}

// Grid: rows * L workgroups: the S second-level partials of (row, tensor).
__global__ __launch_bounds__(kBlock) void k_finalize2(DevLayout lay, int server,
                                                      float* __restrict__ scales) {
  const int S = lay.fin_split;
  const int64_t b = blockIdx.x;
  const int l = (int)(b % lay.L);
  const int r = (int)(b / lay.L);
  const int row = server ? lay.k_max : r;
  u64 tlo, thi;
  block_sum128(lay.part2 + ((int64_t)row * lay.L + l) * S * 2, S, tlo, thi);
  if (threadIdx.x != 0) return;
  scales[server ? l : (int64_t)r * lay.L + l] = scale_from_sum(thi, tlo, lay.tensors[l].n);
}

// ------------------------------------------------------------------ step ahead
// kU words of one worker's tile starting at word w0: x^(k)_{t+1/2} = x_t -
// e^(k)_t with the pending corrections of x and e applied on the fly
// (kHasE false: x_t itself, the evaluation point of local error feedback).
// kFull: all kU words are whole words of the tile (no guards).
template <bool kDecX, int kDecE, bool kHasE, bool kFull>
__device__ __forceinline__ void step_words(int w0, int nw, int count,
                                           const float* __restrict__ xt,
                                           const float* __restrict__ ek, float* __restrict__ hk,
                                           const uint64_t* __restrict__ sx,
                                           const uint64_t* __restrict__ sk, float s_x,
                                           float s_e) {
  const int lane = lane_id();
  float xv[kU], ev[kU];
  u64 mx[kU], me[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int j = (w0 + u) * 64 + lane;
    const bool ok = kFull || ((w0 + u < nw) && j < count);
    xv[u] = ok ? (kHasE ? xt[j] : ld_nt(xt + j)) : 0.0f;
    ev[u] = (kHasE && ok) ? ld_nt(ek + j) : 0.0f;
    mx[u] = (kDecX && (kFull || w0 + u < nw)) ? sx[w0 + u] : 0ull;
    me[u] = (kDecE != kDecPlain && (kFull || w0 + u < nw)) ? sk[w0 + u] : 0ull;
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int j = (w0 + u) * 64 + lane;
    if (!kFull && w0 + u >= nw) continue;
    float xc = xv[u], ec = ev[u];
    if (kDecX) xc = xc - corr(mx[u], s_x);  // x_t = x_{t-1} - C(Delta_t)
    if (kDecE == kDecSign) ec = ec - corr(me[u], s_e);  // e_t = Delta - C(Delta)
    if (kDecE == kDecZero) ec = sel_by_bit(me[u], 0.0f, ec);  // kept elements: 0
    if (kFull || j < count) st_nt(hk + j, kHasE ? xc - ec : xc);  // x^(k)_{t+1/2} = x_t - e^(k)_t
  }
}

// Grid: run_padded_tiles(n_tiles) * K workgroups, one per (tile, worker), in
// the XCD-aware tile order of run_tile_of: the K workers of a run of tiles
// follow one another on one XCD, so x is fetched from HBM once and re-read
// from that XCD's L2.  x itself is not written: the pending re-update of x
// is applied here on the fly and materialized by the aggregate kernel.
// kHasE false (K = 1, e unused): xh = x_t.
template <bool kDecX, int kDecE, bool kHasE>
__global__ __launch_bounds__(kBlock) void k_step(DevLayout lay, int K, const float* __restrict__ x,
                                                 const uint64_t* __restrict__ ss,
                                                 const float* __restrict__ sscales,
                                                 const float* __restrict__ e,
                                                 const uint64_t* __restrict__ signs,
                                                 const float* __restrict__ scales,
                                                 float* __restrict__ xh) {
  int k;
  int64_t ti;
  run_tile_of(blockIdx.x, K, tile_run_shift(lay.n_tiles), k, ti);
  if (ti >= lay.n_tiles) return;
  const Tile tile = lay.tiles[ti];
  const int wave = wave_id();
  const int64_t d_pad = lay.d_pad;
  const int64_t gw0 = tile.start >> 6;
  const float* ek = kHasE ? e + (int64_t)k * d_pad + tile.start : nullptr;
  float* hk = xh + (int64_t)k * d_pad + tile.start;
  const float* xt = x + tile.start;
  const uint64_t* sk = signs + (int64_t)k * (d_pad >> 6) + gw0;
  const uint64_t* sx = ss + gw0;
  const float s_e = kDecE == kDecSign ? scales[(int64_t)k * lay.L + tile.l] : 0.0f;
  const float s_x = kDecX ? sscales[tile.l] : 0.0f;
  const int nw = (tile.count + 63) >> 6;
  for (int w0 = wave * kU; w0 < nw; w0 += kWaves * kU) {
    if ((w0 + kU) * 64 <= tile.count) {
      step_words<kDecX, kDecE, kHasE, true>(w0, nw, tile.count, xt, ek, hk, sx, sk, s_x, s_e);
    } else {
      step_words<kDecX, kDecE, kHasE, false>(w0, nw, tile.count, xt, ek, hk, sx, sk, s_x, s_e);
    }
  }
}

// ------------------------------------------------------------------ step ahead with averaging
constexpr int kAvgChunk = 4;  // workers whose loads are issued together

// kN words of one tile starting at word w0, all K workers: the local errors
// are read in worker order (pending corrections applied when kDecE) and
// replaced by their mean (binary64 sum in worker order, /K, fp32); then
// x^(k)_{t+1/2} = x_t - mean for every worker when kXh.  kFull: the kN
// words are whole words of the tile; otherwise kN is 1 and the lane's
// element exists iff `valid`.
template <bool kDecX, int kDecE, bool kXh, bool kFull, int kN>
__device__ __forceinline__ void average_words(const DevLayout& lay, int K, double inv_k, int l,
                                              int w0, bool valid, int64_t start,
                                              const float* __restrict__ x,
                                              const uint64_t* __restrict__ ss, float s_x,
                                              float* __restrict__ e,
                                              const uint64_t* __restrict__ signs,
                                              const float* __restrict__ scales,
                                              float* __restrict__ xh) {
  const int lane = lane_id();
  const int64_t d_pad = lay.d_pad;
  const int64_t W = d_pad >> 6;
  const int64_t gw0 = (start >> 6) + w0;
  const int64_t base = start + w0 * 64 + lane;
  const bool ok = kFull || valid;
  double acc[kN];
#pragma unroll
  for (int u = 0; u < kN; ++u) acc[u] = 0.0;
  for (int k0 = 0; k0 < K; k0 += kAvgChunk) {
    // sign words are fetched per lane as the 32-bit half holding the lane's
    // bit (vector registers: this kernel keeps kAvgChunk * kN words live)
    float ev[kAvgChunk][kN];
    uint32_t hw[kAvgChunk][kN];
#pragma unroll
    for (int c = 0; c < kAvgChunk; ++c) {
      const bool kin = k0 + c < K;
      const float* ek = e + (int64_t)(k0 + c) * d_pad + base;
      const uint64_t* sk = signs + (int64_t)(k0 + c) * W + gw0;
#pragma unroll
      for (int u = 0; u < kN; ++u) {
        ev[c][u] = (kin && ok) ? ld_nt(ek + u * 64) : 0.0f;
        hw[c][u] = (kDecE != kDecPlain && kin) ? half_word(sk + u, lane) : 0u;
      }
    }
#pragma unroll
    for (int c = 0; c < kAvgChunk; ++c) {
      if (k0 + c >= K) continue;
      const float s = kDecE == kDecSign ? scales[(int64_t)(k0 + c) * lay.L + l] : 0.0f;
#pragma unroll
      for (int u = 0; u < kN; ++u) {
        float v = ev[c][u];
        if (kDecE == kDecSign) v = v - (half_bit(hw[c][u], lane) ? s : -s);
        if (kDecE == kDecZero) v = half_bit(hw[c][u], lane) ? 0.0f : v;
        acc[u] += (double)v;
      }
    }
  }
  float mean[kN], xv[kN];
#pragma unroll
  for (int u = 0; u < kN; ++u) {
    mean[u] = (float)mean_of(acc[u], inv_k, K);
    xv[u] = 0.0f;
    if (kXh) {
      const uint32_t hx = kDecX ? half_word(ss + gw0 + u, lane) : 0u;
      if (ok) xv[u] = x[base + u * 64];
      if (kDecX) xv[u] = xv[u] - (half_bit(hx, lane) ? s_x : -s_x);
    }
  }
  if (!ok) return;
  for (int k = 0; k < K; ++k) {
    float* ek = e + (int64_t)k * d_pad + base;
    float* hk = xh + (int64_t)k * d_pad + base;
#pragma unroll
    for (int u = 0; u < kN; ++u) {
      st_nt(ek + u * 64, mean[u]);
      if (kXh) st_nt(hk + u * 64, xv[u] - mean[u]);
    }
  }
}

// Grid: run_padded_tiles(n_tiles) workgroups, one per tile in the XCD-aware
// tile order of run_tile_of; wave w takes words w*kUA .. w*kUA+kUA-1 of the
// tile, then strides by 4*kUA words.
template <bool kDecX, int kDecE, bool kXh>
__global__ __launch_bounds__(kBlock) void k_step_average(DevLayout lay, int K, double inv_k,
                                                         const float* __restrict__ x,
                                                         const uint64_t* __restrict__ ss,
                                                         const float* __restrict__ sscales,
                                                         float* __restrict__ e,
                                                         const uint64_t* __restrict__ signs,
                                                         const float* __restrict__ scales,
                                                         float* __restrict__ xh) {
  int row0;
  int64_t ti;
  run_tile_of(blockIdx.x, 1, tile_run_shift(lay.n_tiles), row0, ti);
  if (ti >= lay.n_tiles) return;
  const Tile tile = lay.tiles[ti];
  const int wave = wave_id();
  const int nw = (tile.count + 63) >> 6;
  const float s_x = kDecX ? sscales[tile.l] : 0.0f;
  for (int w0 = wave * kUA; w0 < nw; w0 += kWaves * kUA) {
    if ((w0 + kUA) * 64 <= tile.count) {
      average_words<kDecX, kDecE, kXh, true, kUA>(lay, K, inv_k, tile.l, w0, true, tile.start, x,
                                                 ss, s_x, e, signs, scales, xh);
    } else {
      // tail of the tile: one word at a time, guarded per lane
      for (int w = w0; w < min(w0 + kUA, nw); ++w) {
        average_words<kDecX, kDecE, kXh, false, 1>(lay, K, inv_k, tile.l, w,
                                                   w * 64 + lane_id() < tile.count, tile.start, x,
                                                   ss, s_x, e, signs, scales, xh);
      }
    }
  }
}

// ------------------------------------------------------------------ aggregate
constexpr int kAggChunk = 4;  // workers whose sign words are loaded together
// One pass of a wave over kN words of a tile: the K worker messages are
// decoded in order, mean = (sum_k +-scale_k in binary64, k order) / K.
// kFull: all kN words lie inside the tile; otherwise element base + 64 u
// exists iff 64 u < lim (kN is then 1).
template <int kMode, bool kDecode, bool kAvg, bool kFull, int kN>
__device__ __forceinline__ void aggregate_pass(const DevLayout& lay, int K, double inv_k, int l,
                                               int64_t base, int64_t gw, int lim,
                                               const uint64_t* __restrict__ signs,
                                               const float* __restrict__ scales,
                                               float* __restrict__ avg, float* __restrict__ es,
                                               uint64_t* __restrict__ ss, float s_old,
                                               float* __restrict__ x, u64& lo, u64& hi,
                                               bool& bad) {
  const int lane = lane_id();
  const int64_t W = lay.d_pad >> 6;
  constexpr bool kUpdX = kMode == 0 || kDecode;  // x is read and written
  float ev[kN], xv[kN];
  u64 mo[kN];
#pragma unroll
  for (int u = 0; u < kN; ++u) {
    const bool ok = kFull || u * 64 < lim;
    ev[u] = (kMode == 1 && ok) ? ld_nt(es + base + u * 64) : 0.0f;
    xv[u] = (kUpdX && ok) ? ld_nt(x + base + u * 64) : 0.0f;
    mo[u] = (kMode == 1 && kDecode) ? ss[gw + u] : 0ull;
  }
  double acc[kN];
#pragma unroll
  for (int u = 0; u < kN; ++u) acc[u] = 0.0;
  // workers in chunks of kAggChunk: the chunk's scales and sign words are all
  // loaded (a worker past K reloads worker K - 1) before the first is used
  for (int k0 = 0; k0 < K; k0 += kAggChunk) {
    float sc[kAggChunk];
    u64 m[kAggChunk][kN];
#pragma unroll
    for (int c = 0; c < kAggChunk; ++c) {
      const int k = min(k0 + c, K - 1);
      sc[c] = scales[(int64_t)k * lay.L + l];
      const uint64_t* sk = signs + (int64_t)k * W + gw;
#pragma unroll
      for (int u = 0; u < kN; ++u) m[c][u] = sk[u];
    }
#pragma unroll
    for (int c = 0; c < kAggChunk; ++c) {
      if (k0 + c >= K) break;  // wave-uniform
      // +-scale_k in binary64: the two values differ only in the sign bit
      const double sd = (double)sc[c];
      const uint32_t pos_hi = (uint32_t)__double2hiint(sd);
      const uint32_t lo_bits = (uint32_t)__double2loint(sd);
      const uint32_t neg_hi = pos_hi ^ 0x80000000u;
#pragma unroll
      for (int u = 0; u < kN; ++u)
        acc[u] += __hiloint2double((int)sel_by_bit(m[c][u], pos_hi, neg_hi), (int)lo_bits);
    }
  }
#pragma unroll
  for (int u = 0; u < kN; ++u) {
    const bool ok = kFull || u * 64 < lim;
    const float mean = (float)mean_of(acc[u], inv_k, K);
    const int64_t i = base + u * 64;
    if (kAvg && ok) avg[i] = mean;
    if (kMode == 1) {
      float evc = ev[u];
      if (kDecode) {
        const float c = corr(mo[u], s_old);
        evc = evc - c;                    // e_t = Delta_t - C(Delta_t)
        if (ok) st_nt(x + i, xv[u] - c);  // re-update x_t = x_{t-1} - C(Delta_t)
      }
      // Delta_{t+1} = e_t + (1/K) sum_k C(Delta^(k))
      const float D = evc + mean;
      const u64 word = __ballot(ok && D >= 0.0f);
      if (lane == 0) ss[gw + u] = word;
      if (ok) {
        sum_abs(D, lo, hi, bad);
        st_nt(es + i, D);
      }
    } else if (ok) {
      st_nt(x + i, xv[u] - mean);  // single-way: the mean itself comes back
    }
  }
}

// Grid: n_tiles workgroups; workgroup b handles tile b.  Wave w takes words
// w*kU .. w*kU+kU-1 of the tile (one pass over a whole tile), then strides by
// 4*kU words.
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
  const int lane = lane_id();
  const int nw = (tile.count + 63) >> 6;
  const float s_old = (kMode == 1 && kDecode) ? sscales[tile.l] : 0.0f;
  u64 lo = 0, hi = 0;
  bool bad = false;
  for (int w0 = wave_id() * kU; w0 < nw; w0 += kWaves * kU) {
    const int64_t base = tile.start + w0 * 64 + lane;
    const int64_t gw = (tile.start >> 6) + w0;
    if ((w0 + kU) * 64 <= tile.count) {
      aggregate_pass<kMode, kDecode, kAvg, true, kU>(lay, K, inv_k, tile.l, base, gw, 0, signs,
                                                     scales, avg, es, ss, s_old, x, lo, hi, bad);
    } else {
      // tail of the tile: one word at a time, guarded per lane
      for (int u = 0; u < min(kU, nw - w0); ++u) {
        aggregate_pass<kMode, kDecode, kAvg, false, 1>(
            lay, K, inv_k, tile.l, base + u * 64, gw + u, tile.count - (w0 + u) * 64 - lane,
            signs, scales, avg, es, ss, s_old, x, lo, hi, bad);
      }
    }
  }
  if (kMode == 1) block_partial(lay, lay.k_max, ti, lo, hi, bad);
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
  const int wave = wave_id();
  const int64_t d_pad = lay.d_pad;
  const int64_t gw0 = tile.start >> 6;
  const int nw = (tile.count + 63) >> 6;
  if (row < K) {
    const float s = scales[(int64_t)row * lay.L + l];
    const uint64_t* sk = signs + (int64_t)row * (d_pad >> 6) + gw0;
    for (int w = wave; w < nw; w += kWaves) {
      const u64 m = sk[w];
      const int j = w * 64 + lane;
      if (j < tile.count) {
        const int64_t i = (int64_t)row * d_pad + tile.start + j;
        e_out[i] = e[i] - corr(m, s);
      }
    }
    return;
  }
  const float s = (mode == 1) ? sscales[l] : 0.0f;
  for (int w = wave; w < nw; w += kWaves) {
    const u64 m = (mode == 1) ? ss[gw0 + w] : 0ull;
    const int j = w * 64 + lane;
    if (j >= tile.count) continue;
    const int64_t i = tile.start + j;
    if (mode == 1) {
      const float c = corr(m, s);
      if (es_out) es_out[i] = es[i] - c;
      if (x_out) x_out[i] = x[i] - c;
    } else {
      if (es_out) es_out[i] = 0.0f;
      if (x_out) x_out[i] = x[i];
    }
  }
}

// ------------------------------------------------------------------ mismatch
// Gradient-mismatch bounds (a diagnostic, "Step Ahead" and "Error Averaging"
// sections with the Lipschitz constant and the variance term left out), per
// element in binary64:
//   ebar = (sum_k e^(k), worker order) / K,   u = e_srv + ebar,
//   a = u^2 (local error feedback),   b = sum_k (u - e^(k))^2 (step ahead).
// Each wave sums a and b over one tile and stores the two doubles in the
// tile's slot of the partial-sum scratch (row 0); k_mfinalize adds them per
// tensor.  The K errors are read twice: the second read finds them in the
// caches (kMisWords words per wave keep the working set small).
constexpr int kMisWords = 4;   // words per pass, two-read path
constexpr int kMisRegK = 16;   // at most this many workers: one read, values kept in registers
constexpr int kMisRegWords = 2;

// Two-read path (any K): the errors are read once for the mean and again
// for the distances.
template <bool kDC, bool kDecE, bool kDecS, bool kFull, int kN>
__device__ __forceinline__ void mismatch_pass(const DevLayout& lay, int K, double inv_k, int l,
                                              int64_t base, int64_t gw, int lim,
                                              const float* __restrict__ e,
                                              const uint64_t* __restrict__ signs,
                                              const float* __restrict__ scales,
                                              const float* __restrict__ es,
                                              const uint64_t* __restrict__ ss, float s_srv,
                                              double& a, double& b) {
  const int64_t W = lay.d_pad >> 6;
  const int64_t d_pad = lay.d_pad;
  double acc[kN];
#pragma unroll
  for (int u = 0; u < kN; ++u) acc[u] = 0.0;
  for (int k = 0; k < K; ++k) {
    const float s = kDecE ? scales[(int64_t)k * lay.L + l] : 0.0f;
    const float* ek = e + (int64_t)k * d_pad + base;
    const uint64_t* sk = signs + (int64_t)k * W + gw;
#pragma unroll
    for (int u = 0; u < kN; ++u) {
      const bool ok = kFull || u * 64 < lim;
      float v = ok ? ek[u * 64] : 0.0f;
      if (kDecE) v = v - corr(sk[u], s);
      acc[u] += (double)v;
    }
  }
  double uu[kN], bs[kN];
#pragma unroll
  for (int u = 0; u < kN; ++u) {
    const bool ok = kFull || u * 64 < lim;
    const double ebar = mean_of(acc[u], inv_k, K);
    float esv = 0.0f;
    if (kDC) {
      esv = ok ? es[base + u * 64] : 0.0f;
      if (kDecS) esv = esv - corr(ss[gw + u], s_srv);
    }
    uu[u] = (double)esv + ebar;
    if (ok) a += uu[u] * uu[u];
    bs[u] = 0.0;
  }
  for (int k = 0; k < K; ++k) {
    const float s = kDecE ? scales[(int64_t)k * lay.L + l] : 0.0f;
    const float* ek = e + (int64_t)k * d_pad + base;
    const uint64_t* sk = signs + (int64_t)k * W + gw;
#pragma unroll
    for (int u = 0; u < kN; ++u) {
      const bool ok = kFull || u * 64 < lim;
      float v = ok ? ek[u * 64] : 0.0f;
      if (kDecE) v = v - corr(sk[u], s);
      const double dk = uu[u] - (double)v;
      bs[u] += dk * dk;
    }
  }
#pragma unroll
  for (int u = 0; u < kN; ++u)
    if (kFull || u * 64 < lim) b += bs[u];
}

// One-read path (K <= kRK <= kMisRegK): the decoded errors stay in
// registers.  All loads of the pass (the kRK workers' errors and sign-word
// halves, e_srv and its word) are issued before the first one is used: rows
// past K and lanes past the tile's end load an element that exists and are
// masked afterwards.  Same arithmetic as mismatch_pass.
template <bool kDC, bool kDecE, bool kDecS, bool kFull, int kN, int kRK>
__device__ __forceinline__ void mismatch_pass_reg(const DevLayout& lay, int K, double inv_k,
                                                  int64_t base, int64_t gw, int lim,
                                                  const float* __restrict__ e,
                                                  const uint64_t* __restrict__ signs,
                                                  const float (&sc)[kRK],
                                                  const float* __restrict__ es,
                                                  const uint64_t* __restrict__ ss, float s_srv,
                                                  double& a, double& b) {
  const int lane = lane_id();
  const int64_t W = lay.d_pad >> 6;
  const int64_t d_pad = lay.d_pad;
  float v[kRK][kN];
  uint32_t hw[kRK][kN];
  float esv[kN];
  uint32_t hs[kN];
#pragma unroll
  for (int u = 0; u < kN; ++u) {
    const bool ok = kFull || u * 64 < lim;
    const int64_t j = base + (ok ? u * 64 : -lane);  // the word's first element exists
    esv[u] = kDC ? ld_nt(es + j) : 0.0f;
    hs[u] = kDecS ? half_word(ss + gw + u, lane) : 0u;
#pragma unroll
    for (int k = 0; k < kRK; ++k) {
      const int64_t row = k < K ? k : 0;
      v[k][u] = ld_nt(e + row * d_pad + j);
      hw[k][u] = kDecE ? half_word(signs + row * W + gw + u, lane) : 0u;
    }
  }
#pragma unroll
  for (int u = 0; u < kN; ++u) {
    const bool ok = kFull || u * 64 < lim;
    double acc = 0.0;
#pragma unroll
    for (int k = 0; k < kRK; ++k) {
      if (kDecE) v[k][u] = v[k][u] - (half_bit(hw[k][u], lane) ? sc[k] : -sc[k]);
      if (k < K) acc += (double)v[k][u];  // worker order
    }
    const double ebar = mean_of(acc, inv_k, K);
    float ev = esv[u];
    if (kDecS) ev = ev - (half_bit(hs[u], lane) ? s_srv : -s_srv);
    const double uu = (double)ev + ebar;
    double bs = 0.0;
#pragma unroll
    for (int k = 0; k < kRK; ++k) {
      if (k < K) {
        const double dk = uu - (double)v[k][u];
        bs += dk * dk;
      }
    }
    if (ok) {
      a += uu * uu;
      b += bs;
    }
  }
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

// Grid: n_tiles workgroups; wave w of workgroup b takes words
// [w kMisWaveWords, (w + 1) kMisWaveWords) of tile b, and the four waves'
// sums are added in wave order.
constexpr int kMisWaveWords = kTileElems / 64 / kWaves;  // 8
template <bool kDC, bool kDecE, bool kDecS, int kRK>
__global__ __launch_bounds__(kBlock) void k_mismatch(DevLayout lay, int K, double inv_k,
                                                     const float* __restrict__ e,
                                                     const uint64_t* __restrict__ signs,
                                                     const float* __restrict__ scales,
                                                     const float* __restrict__ es,
                                                     const uint64_t* __restrict__ ss,
                                                     const float* __restrict__ sscales) {
  static_assert(kMisWaveWords % kMisWords == 0 && kMisWaveWords % kMisRegWords == 0,
                "a wave's words split into whole passes");
  constexpr bool kReg = kRK > 0;
  constexpr int kR = kReg ? kRK : 1;
  __shared__ double s_a[kWaves];
  __shared__ double s_b[kWaves];
  const int64_t ti = blockIdx.x;
  const Tile tile = lay.tiles[ti];
  const int lane = lane_id();
  const int wave = wave_id();
  const int nw = (tile.count + 63) >> 6;
  const float s_srv = kDecS ? sscales[tile.l] : 0.0f;
  float sc[kR];  // the workers' scales of the tile's tensor (register path)
#pragma unroll
  for (int k = 0; k < kR; ++k)
    sc[k] = (kReg && kDecE) ? scales[(int64_t)(k < K ? k : 0) * lay.L + tile.l] : 0.0f;
  constexpr int kW = kReg ? kMisRegWords : kMisWords;
  double a = 0.0, b = 0.0;
  const int wend = min(nw, (wave + 1) * kMisWaveWords);
  for (int wb = wave * kMisWaveWords; wb < wend; wb += kW) {
    const int64_t base = tile.start + wb * 64 + lane;
    const int64_t gw = (tile.start >> 6) + wb;
    if ((wb + kW) * 64 <= tile.count) {
      if constexpr (kReg)
        mismatch_pass_reg<kDC, kDecE, kDecS, true, kW, kR>(lay, K, inv_k, base, gw, 0, e, signs,
                                                           sc, es, ss, s_srv, a, b);
      else
        mismatch_pass<kDC, kDecE, kDecS, true, kW>(lay, K, inv_k, tile.l, base, gw, 0, e, signs,
                                                   scales, es, ss, s_srv, a, b);
    } else {
      for (int u = 0; u < min(kW, nw - wb); ++u) {
        const int lim = tile.count - (wb + u) * 64 - lane;
        if constexpr (kReg)
          mismatch_pass_reg<kDC, kDecE, kDecS, false, 1, kR>(lay, K, inv_k, base + u * 64, gw + u,
                                                             lim, e, signs, sc, es, ss, s_srv, a,
                                                             b);
        else
          mismatch_pass<kDC, kDecE, kDecS, false, 1>(lay, K, inv_k, tile.l, base + u * 64,
                                                     gw + u, lim, e, signs, scales, es, ss,
                                                     s_srv, a, b);
      }
    }
  }
  a = wave_sum_f64(a);
  b = wave_sum_f64(b);
  if (lane == 0) {
    s_a[wave] = a;
    s_b[wave] = b;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double ta = 0.0, tb = 0.0;
    for (int w = 0; w < kWaves; ++w) {
      ta += s_a[w];
      tb += s_b[w];
    }
    u64* p = lay.part + ti * 2;
    p[0] = (u64)__double_as_longlong(ta);
    p[1] = (u64)__double_as_longlong(tb);
  }
}

// Adds the (a, b) double pairs v[0..n) over the workgroup in a fixed order
// (thread 0 gets the sums).
__device__ void block_sum_pairs(const u64* __restrict__ v, int64_t n, double& ta, double& tb) {
  __shared__ double s_a[kWaves];
  __shared__ double s_b[kWaves];
  double a = 0.0, b = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += kBlock) {
    a += __longlong_as_double((long long)v[2 * i]);
    b += __longlong_as_double((long long)v[2 * i + 1]);
  }
  a = wave_sum_f64(a);
  b = wave_sum_f64(b);
  const int w = threadIdx.x / kWave;
  if (lane_id() == 0) {
    s_a[w] = a;
    s_b[w] = b;
  }
  __syncthreads();
  ta = 0.0;
  tb = 0.0;
  if (threadIdx.x == 0)
    for (int i = 0; i < kWaves; ++i) {
      ta += s_a[i];
      tb += s_b[i];
    }
}

// Grid: L * S workgroups (S = lay.fin_split): part s of tensor l's tile sums.
// With S = 1 it writes out[l] = sum a and out[L + l] = (sum b) / K, else a
// second-level pair that k_mfinalize2 adds.
__global__ __launch_bounds__(kBlock) void k_mfinalize(DevLayout lay, int K,
                                                      double* __restrict__ out) {
  const int S = lay.fin_split;
  const int s = (int)(blockIdx.x % S);
  const int l = (int)(blockIdx.x / S);
  const TensorInfo t = lay.tensors[l];
  const int per = (t.ntiles + S - 1) / S;
  const int i0 = min(t.ntiles, s * per), i1 = min(t.ntiles, i0 + per);
  double a, b;
  block_sum_pairs(lay.part + (int64_t)(t.first_tile + i0) * 2, i1 - i0, a, b);
  if (threadIdx.x != 0) return;
  if (S == 1) {
    out[l] = a;
    out[lay.L + l] = b / (double)K;
  } else {
    u64* q = lay.part2 + ((int64_t)l * S + s) * 2;
    q[0] = (u64)__double_as_longlong(a);
    q[1] = (u64)__double_as_longlong(b);
  }
}

__global__ __launch_bounds__(kBlock) void k_mfinalize2(DevLayout lay, int K,
                                                       double* __restrict__ out) {
  const int S = lay.fin_split;
  const int l = blockIdx.x;
  double a, b;
  block_sum_pairs(lay.part2 + (int64_t)l * S * 2, S, a, b);
  if (threadIdx.x != 0) return;
  out[l] = a;
  out[lay.L + l] = b / (double)K;
}


}  // namespace

hipError_t launch_compress(const DevLayout& lay, int K, float lr, float mu, const float* g,
                           float* m, float* e, uint64_t* signs, const float* scales, bool decode,
                           hipStream_t s, const LaunchEvents& ev) {
  const dim3 grid((unsigned)(lay.n_tiles * K));
#define SAEF_CMP(D, M) \
  SAEF_LAUNCH((k_compress<D, M>), grid, dim3(kBlock), 0, s, lay, K, lr, mu, g, m, e, signs, scales)
  if (m != nullptr) {
    if (decode) SAEF_CMP(true, true); else SAEF_CMP(false, true);
  } else {
    if (decode) SAEF_CMP(true, false); else SAEF_CMP(false, false);
  }
#undef SAEF_CMP
  return hipGetLastError();
}

hipError_t launch_finalize(const DevLayout& lay, int K, bool server, float* scales,
                           hipStream_t s, const LaunchEvents& ev) {
  const int rows = server ? 1 : K;
  const dim3 grid1((unsigned)((int64_t)rows * lay.L * lay.fin_split));
  if (lay.fin_split == 1) {
    SAEF_LAUNCH(k_finalize, grid1, dim3(kBlock), 0, s, lay, server ? 1 : 0, scales);
    return hipGetLastError();
  }
  // two kernels: the event pair brackets both
  hipExtLaunchKernelGGL(k_finalize, grid1, dim3(kBlock), 0, s, ev.start, nullptr, 0, lay,
                        server ? 1 : 0, scales);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipExtLaunchKernelGGL(k_finalize2, dim3((unsigned)(rows * lay.L)), dim3(kBlock), 0, s, nullptr,
                        ev.stop, 0, lay, server ? 1 : 0, scales);
  return hipGetLastError();
}

hipError_t launch_aggregate(const DevLayout& lay, int K, int mode, const uint64_t* signs,
                            const float* scales, float* avg, float* e_srv, uint64_t* srv_signs,
                            const float* srv_scales, float* x, bool decode, hipStream_t s, const LaunchEvents& ev) {
  const dim3 grid((unsigned)lay.n_tiles);
  const double ik = inv_pow2(K);
#define SAEF_AGG(M, D, A)                                                                  \
  SAEF_LAUNCH((k_aggregate<M, D, A>), grid, dim3(kBlock), 0, s, lay, K, ik, signs, \
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

hipError_t launch_step_ahead(const DevLayout& lay, int K, const float* x,
                             const uint64_t* srv_signs, const float* srv_scales, bool decode_x,
                             float* e, const uint64_t* signs, const float* scales, int decode_e,
                             bool average, float* xh, hipStream_t s, const LaunchEvents& ev) {
  if (decode_e < kDecPlain || decode_e > kDecZero) return hipErrorInvalidValue;
  if (decode_x && decode_e != kDecSign) return hipErrorInvalidValue;  // never requested
  if (average) {
    const dim3 grid((unsigned)run_padded_tiles(lay.n_tiles));
    const double ik = inv_pow2(K);
#define SAEF_AV(DX, DE, XH)                                                                  \
  SAEF_LAUNCH((k_step_average<DX, DE, XH>), grid, dim3(kBlock), 0, s, lay, K, ik, x, \
                     srv_signs, srv_scales, e, signs, scales, xh)
    if (xh == nullptr) {
      if (decode_x) return hipErrorInvalidValue;  // x is not read without xh
      if (decode_e == kDecSign) SAEF_AV(false, kDecSign, false);
      else if (decode_e == kDecZero) SAEF_AV(false, kDecZero, false);
      else SAEF_AV(false, kDecPlain, false);
    } else if (decode_x) {
      SAEF_AV(true, kDecSign, true);
    } else if (decode_e == kDecSign) {
      SAEF_AV(false, kDecSign, true);
    } else if (decode_e == kDecZero) {
      SAEF_AV(false, kDecZero, true);
    } else {
      SAEF_AV(false, kDecPlain, true);
    }
#undef SAEF_AV
  } else {
    if (xh == nullptr) return hipErrorInvalidValue;
    const dim3 grid((unsigned)(run_padded_tiles(lay.n_tiles) * K));
#define SAEF_ST(DX, DE)                                                                \
  SAEF_LAUNCH((k_step<DX, DE, true>), grid, dim3(kBlock), 0, s, lay, K, x, srv_signs, \
                     srv_scales, e, signs, scales, xh)
    if (decode_x) {
      SAEF_ST(true, kDecSign);
    } else if (decode_e == kDecSign) {
      SAEF_ST(false, kDecSign);
    } else if (decode_e == kDecZero) {
      SAEF_ST(false, kDecZero);
    } else {
      SAEF_ST(false, kDecPlain);
    }
#undef SAEF_ST
  }
  return hipGetLastError();
}

hipError_t launch_weights(const DevLayout& lay, const float* x, const uint64_t* srv_signs,
                          const float* srv_scales, bool decode_x, float* xh, hipStream_t s,
                          const LaunchEvents& ev) {
  const dim3 grid((unsigned)run_padded_tiles(lay.n_tiles));
  if (decode_x) {
    SAEF_LAUNCH((k_step<true, kDecPlain, false>), grid, dim3(kBlock), 0, s, lay, 1, x, srv_signs,
                srv_scales, nullptr, nullptr, nullptr, xh);
  } else {
    SAEF_LAUNCH((k_step<false, kDecPlain, false>), grid, dim3(kBlock), 0, s, lay, 1, x, srv_signs,
                srv_scales, nullptr, nullptr, nullptr, xh);
  }
  return hipGetLastError();
}

hipError_t launch_materialize(const DevLayout& lay, int K, int mode, const float* e,
                              const uint64_t* signs, const float* scales, float* e_out,
                              const float* e_srv, const float* x, const uint64_t* srv_signs,
                              const float* srv_scales, float* e_srv_out, float* x_out,
                              hipStream_t s, const LaunchEvents& ev) {
  const int k_rows = e_out != nullptr ? K : 0;
  const int rows = k_rows + ((e_srv_out != nullptr || x_out != nullptr) ? 1 : 0);
  if (rows == 0) return hipSuccess;
  const dim3 grid((unsigned)(lay.n_tiles * rows));
  SAEF_LAUNCH(k_materialize, grid, dim3(kBlock), 0, s, lay, k_rows, rows, mode, e, signs,
                     scales, e_out, e_srv, x, srv_signs, srv_scales, e_srv_out, x_out);
  return hipGetLastError();
}

hipError_t launch_mismatch(const DevLayout& lay, int K, int mode, const float* e,
                           const uint64_t* signs, const float* scales, bool decode_e,
                           const float* e_srv, const uint64_t* srv_signs,
                           const float* srv_scales, bool decode_s, double* out, hipStream_t s,
                           const LaunchEvents& ev) {
  const dim3 grid((unsigned)lay.n_tiles);
  const double ik = inv_pow2(K);
#define SAEF_MIS2(DC, DE, DS, R)                                                               \
  hipExtLaunchKernelGGL((k_mismatch<DC, DE, DS, R>), grid, dim3(kBlock), 0, s, ev.start,        \
                        nullptr, 0, lay, K, ik, e, signs, scales, e_srv, srv_signs, srv_scales)
#define SAEF_MIS(DC, DE, DS)                                  \
  do {                                                        \
    if (K <= 4) SAEF_MIS2(DC, DE, DS, 4);                     \
    else if (K <= 8) SAEF_MIS2(DC, DE, DS, 8);                \
    else if (K <= kMisRegK) SAEF_MIS2(DC, DE, DS, kMisRegK);  \
    else SAEF_MIS2(DC, DE, DS, 0);                            \
  } while (0)
  if (mode == 1) {
    if (decode_e) {
      if (decode_s) SAEF_MIS(true, true, true); else SAEF_MIS(true, true, false);
    } else {
      if (decode_s) SAEF_MIS(true, false, true); else SAEF_MIS(true, false, false);
    }
  } else {
    if (decode_e) SAEF_MIS(false, true, false); else SAEF_MIS(false, false, false);
  }
#undef SAEF_MIS
#undef SAEF_MIS2
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int S = lay.fin_split;
  // the event pair brackets the element kernel and the one or two sums
  hipExtLaunchKernelGGL(k_mfinalize, dim3((unsigned)(lay.L * S)), dim3(kBlock), 0, s, nullptr,
                        S == 1 ? ev.stop : nullptr, 0, lay, K, out);
  err = hipGetLastError();
  if (err != hipSuccess || S == 1) return err;
  hipExtLaunchKernelGGL(k_mfinalize2, dim3((unsigned)lay.L), dim3(kBlock), 0, s, nullptr, ev.stop,
                        0, lay, K, out);
  return hipGetLastError();
}

}  // namespace saef
