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

// Workgroup shapes.  The compression and the server (and the stream probe,
// which measures the compression's pattern) take a 2048-element tile with
// kSWaves waves of kU words per pass; the step ahead with kTWaves waves of
// kTU words.  Each wave of the compression and the server ends with a
// 128-bit wave reduction of its exact sum, so fewer, longer waves suit them.
#ifndef SAEF_STREAM_WAVES
#define SAEF_STREAM_WAVES 4
#endif
#ifndef SAEF_STREAM_WORDS
#define SAEF_STREAM_WORDS 8
#endif
#ifndef SAEF_STEP_WAVES
#define SAEF_STEP_WAVES 4
#endif
#ifndef SAEF_STEP_WORDS
#define SAEF_STEP_WORDS 4
#endif
constexpr int kSWaves = SAEF_STREAM_WAVES;
constexpr int kSBlock = kSWaves * kWave;
constexpr int kU = SAEF_STREAM_WORDS;
constexpr int kTWaves = SAEF_STEP_WAVES;
constexpr int kTBlock = kTWaves * kWave;
constexpr int kTU = SAEF_STEP_WORDS;
// The step ahead's work unit (kStepElems elements of a tile) is one pass of
// its workgroup: 1024-element units of 4 waves x 4 words against whole
// 2048-element tiles of 4 x 8: 276-286 against 288-292 us at resnet50
// K = 8, 2951 against 3016-3026 us at 2^28 parameters.
static_assert(kTWaves * kTU * 64 <= kStepElems && kStepElems % (kTWaves * kTU * 64) == 0,
              "a step unit is whole passes of the workgroup");
// Words per wave per pass in the averaging kernel (it keeps kAvgChunk * kUA
// errors and sign words live), and its work units per tile: 1024-element
// units of one pass of 4 waves x 4 words, all 8 workers' loads issued
// together, took 451 us at resnet50 K = 8 against 481 us for whole tiles of
// two passes with the workers in chunks of 4 (460 us: one pass of 8 words;
// 479-502 us: 2 words).
#ifndef SAEF_AVG_WORDS
#define SAEF_AVG_WORDS 4
#endif
#ifndef SAEF_AVG_SPLIT
#define SAEF_AVG_SPLIT 2
#endif
constexpr int kUA = SAEF_AVG_WORDS;
constexpr int kAvgSplit = SAEF_AVG_SPLIT;
static_assert(kAvgSplit >= 1 && kAvgSplit <= kStepSplit && kTileElems % (kAvgSplit * 64) == 0,
              "an averaging unit is whole words of a tile, within the step ahead's grid limit");

// The compression correction C(v)_i = bit ? scale : -scale.
__device__ __forceinline__ float corr(u64 word, float s) { return sel_by_bit(word, s, -s); }

// The same with +-scale already held in vector registers (in_vgpr).
struct Corr {
  float pos, neg;
  __device__ __forceinline__ explicit Corr(float s) : pos(in_vgpr(s)), neg(in_vgpr(-s)) {}
  __device__ __forceinline__ float operator()(u64 word) const { return sel_by_bit(word, pos, neg); }
};

// The 32-bit half of the sign word at p that holds bit `lane`, read per lane
// (a vector register instead of a scalar pair, for kernels that keep many
// words live), and the lane's bit in it.
__device__ __forceinline__ uint32_t half_word(const uint64_t* p, int lane) {
  return reinterpret_cast<const uint32_t*>(p)[lane >> 5];
}
__device__ __forceinline__ bool half_bit(uint32_t h, int lane) {
  return ((h >> (lane & 31)) & 1u) != 0;
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
template <int kNW>
__device__ void block_partial(const DevLayout& lay, int row, int64_t tile, u64 lo, u64 hi,
                              bool bad) {
  __shared__ u64 s_lo[kNW];
  __shared__ u64 s_hi[kNW];
  wave_sum128(lo, hi);
  const int w = threadIdx.x / kWave;
  if (lane_id() == 0) {
    s_lo[w] = lo;
    s_hi[w] = hi;
  }
  const int any_bad = __syncthreads_or(bad ? 1 : 0);
  if (threadIdx.x != 0) return;
  u64 tlo = 0, thi = 0;
  for (int i = 0; i < kNW; ++i) add128(tlo, thi, s_lo[i], s_hi[i]);
  u64* p = lay.part + ((int64_t)row * lay.n_tiles + tile) * 2;
  p[0] = tlo;
  p[1] = thi;
  if (any_bad) atomicOr(lay.status, kStatusRange);
}

// ------------------------------------------------------------------ compress
// kU words of one worker's tile starting at word w0 (element offsets
// relative to the tile; the buffer resources cover the tile's elements and
// sign words, so out-of-range loads read 0 and stores are dropped): with
// kMom, the momentum buffer m <- fma(mu, m, g) first (one rounding); Delta =
// fma(lr, m or g, e) (e decoded when kDecode), sign words by ballot,
// exact-sum terms, Delta stored.  kFull: all kU words are whole words of the
// tile (no lane masks).
template <bool kDecode, bool kMom, bool kFull>
__device__ __forceinline__ void compress_words(int w0, int count, float lr, float mu, Buf rg,
                                               Buf rm, Buf re, Buf rs, const Corr& c_old,
                                               ExactSum& acc) {
  const int lane = lane_id();
  const uint32_t off0 = (uint32_t)(w0 * 64 + lane) * 4u;
  float gv[kU], ev[kU], mv[kU];
  // the old words first (every element waits for them; the scheduling
  // barrier keeps the compiler from moving the load behind the others)
  const u64 ow = kDecode ? buf_ld_words(rs, w0, kU) : 0ull;
  if (kDecode) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    mv[u] = kMom ? buf_ld(rm, off0 + 256u * u) : 0.0f;
    gv[u] = buf_ld(rg, off0 + 256u * u);
    ev[u] = buf_ld(re, off0 + 256u * u);
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const uint32_t off = off0 + 256u * u;
    const bool ok = kFull || (w0 + u) * 64 + lane < count;
    float ev2 = ev[u];
    if (kDecode) ev2 = ev2 - c_old(word_of(ow, u));
    float step = gv[u];
    if (kMom) {
      step = __builtin_fmaf(mu, mv[u], gv[u]);  // m^(k)_{t+1} = mu m^(k)_t + grad
      buf_st(rm, off, step);
    }
    // Delta^(k) = e^(k) + lr * m^(k)_{t+1}, one rounding (m = grad when mu = 0)
    float p = __builtin_fmaf(lr, step, ev2);
    if (!kFull) p = ok ? p : 0.0f;
    const u64 word = __ballot(ok && p >= 0.0f);
    if (lane == 0) buf_st_word(rs, (uint32_t)(w0 + u) * 8u, word);
    acc.add(p);
    buf_st(re, off, p);
  }
}

// Grid: n_tiles * K workgroups; workgroup b handles worker b % K of tile
// b / K.  Wave w takes words w*kU .. w*kU+kU-1 of the tile, then strides by
// 4*kU words.
template <bool kDecode, bool kMom>
__device__ __forceinline__ void compress_tile(const DevLayout& lay, int K, float lr, float mu,
                                              const float* __restrict__ g,
                                              float* __restrict__ m, float* __restrict__ e,
                                              uint64_t* __restrict__ signs,
                                              const float* __restrict__ scales) {
  const unsigned b = blockIdx.x;
  const int k = (int)(b % (unsigned)K);
  const int64_t ti = b / (unsigned)K;
  const Tile tile = lay.tiles[ti];
  const int wave = wave_id();
  const int64_t row = (int64_t)k * lay.d_pad + tile.start;
  const uint32_t nbytes = (uint32_t)tile.count * 4u;
  const int nw = (tile.count + 63) >> 6;
  const Buf rg = buf_of(g + row, nbytes);
  const Buf rm = buf_of(kMom ? m + row : g + row, nbytes);
  const Buf re = buf_of(e + row, nbytes);
  const Buf rs = buf_of(signs + (int64_t)k * (lay.d_pad >> 6) + (tile.start >> 6),
                        (uint32_t)nw * 8u);
  const Corr c_old(kDecode ? scales[(int64_t)k * lay.L + tile.l] : 0.0f);

  ExactSum acc;
  u64 lo = 0, hi = 0;
  bool bad = false;
  for (int w0 = wave * kU; w0 < nw; w0 += kSWaves * kU) {
    if ((w0 + kU) * 64 <= tile.count) {
      compress_words<kDecode, kMom, true>(w0, tile.count, lr, mu, rg, rm, re, rs, c_old, acc);
    } else {
      compress_words<kDecode, kMom, false>(w0, tile.count, lr, mu, rg, rm, re, rs, c_old, acc);
    }
    acc.added(kU, lo, hi, bad);
  }
  acc.finish(lo, hi, bad);
  block_partial<kSWaves>(lay, k, ti, lo, hi, bad);
}

template <bool kDecode>
__global__ __launch_bounds__(kSBlock) void k_compress(DevLayout lay, int K, float lr, float mu,
                                                     const float* __restrict__ g,
                                                     float* __restrict__ m,
                                                     float* __restrict__ e,
                                                     uint64_t* __restrict__ signs,
                                                     const float* __restrict__ scales) {
  compress_tile<kDecode, false>(lay, K, lr, mu, g, m, e, signs, scales);
}

// With momentum (three streams in, two out) at most 5 waves per SIMD: 672
// against 696 us at 8 waves (resnet50, K = 8); the sign kernel prefers 8
// (400 against 406 us).
template <bool kDecode>
__global__ __launch_bounds__(kSBlock) __attribute__((amdgpu_waves_per_eu(1, 5))) void
k_compress_mom(DevLayout lay, int K, float lr, float mu, const float* __restrict__ g,
               float* __restrict__ m, float* __restrict__ e, uint64_t* __restrict__ signs,
               const float* __restrict__ scales) {
  compress_tile<kDecode, true>(lay, K, lr, mu, g, m, e, signs, scales);
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
// kTU words of one worker's tile starting at word w0 (offsets relative to the
// tile; buffer resources over the tile's elements and sign words, so the
// ragged tail needs no guards): x^(k)_{t+1/2} = x_t - e^(k)_t with the
// pending corrections of x and e applied on the fly (kHasE false: x_t
// itself, the evaluation point of local error feedback).
// kFull: all kTU words lie inside the tile (their sign words are read
// unconditionally, in one scalar load per buffer; a guarded load per word
// costs a branch and a wait each).
template <bool kDecX, int kDecE, bool kHasE, bool kFull>
__device__ __forceinline__ void step_words(int w0, int nw, Buf rx, Buf re, Buf rh,
                                           const uint64_t* __restrict__ sx,
                                           const uint64_t* __restrict__ se, const Corr& c_x,
                                           const Corr& c_e) {
  const uint32_t off0 = (uint32_t)(w0 * 64 + lane_id()) * 4u;
  float xv[kTU], ev[kTU];
  u64 mx[kTU], me[kTU];
#pragma unroll
  for (int u = 0; u < kTU; ++u) {
    const uint32_t off = off0 + 256u * u;
    const bool wok = kFull || w0 + u < nw;  // wave-uniform: the tile's words only
    xv[u] = kHasE ? buf_ld_cached(rx, off) : buf_ld(rx, off);
    ev[u] = kHasE ? buf_ld(re, off) : 0.0f;
    mx[u] = (kDecX && wok) ? ld_word_ro(sx + w0 + u) : 0ull;
    me[u] = (kDecE != kDecPlain && wok) ? ld_word_ro(se + w0 + u) : 0ull;
  }
#pragma unroll
  for (int u = 0; u < kTU; ++u) {
    float xc = xv[u], ec = ev[u];
    if (kDecX) xc = xc - c_x(mx[u]);  // x_t = x_{t-1} - C(Delta_t)
    if (kDecE == kDecSign) ec = ec - c_e(me[u]);  // e_t = Delta - C(Delta)
    if (kDecE == kDecZero) ec = sel_by_bit(me[u], 0.0f, ec);  // kept elements: 0
    buf_st(rh, off0 + 256u * u, kHasE ? xc - ec : xc);  // x^(k)_{t+1/2} = x_t - e^(k)_t
  }
}

// Grid: run_padded_tiles(n_tiles kStepSplit) * K workgroups, one per (work
// unit, worker), in the XCD-aware order of run_tile_of over the units: the K
// workers of a run of units follow one another on one XCD, so x is fetched
// from HBM once and re-read from that XCD's L2.  x itself is not written:
// the pending re-update of x is applied here on the fly and materialized by
// the aggregate kernel.
// kHasE false (K = 1, e unused): xh = x_t.
template <bool kDecX, int kDecE, bool kHasE>
__global__ __launch_bounds__(kTBlock) void k_step(DevLayout lay, int K, const float* __restrict__ x,
                                                 const uint64_t* __restrict__ ss,
                                                 const float* __restrict__ sscales,
                                                 const float* __restrict__ e,
                                                 const uint64_t* __restrict__ signs,
                                                 const float* __restrict__ scales,
                                                 float* __restrict__ xh) {
  // work unit: kStepElems elements of a tile (the step ahead keeps no
  // per-tile sums, so its units need not be whole tiles)
  int k;
  int64_t unit;
  const int64_t n_units = lay.n_tiles * kStepSplit;
  run_tile_of(blockIdx.x, K, tile_run_shift(n_units), k, unit);
  if (unit >= n_units) return;
  const Tile tile = lay.tiles[unit / kStepSplit];
  const int part = (int)(unit % kStepSplit);
  const int count = min(tile.count - part * kStepElems, kStepElems);
  if (count <= 0) return;  // a short tile's empty part
  const int64_t start = tile.start + (int64_t)part * kStepElems;
  const int wave = wave_id();
  const int64_t d_pad = lay.d_pad;
  const int64_t gw0 = start >> 6;
  const int nw = (count + 63) >> 6;
  const uint32_t nbytes = (uint32_t)count * 4u;
  const Buf rx = buf_of(x + start, nbytes);
  const Buf re = buf_of(kHasE ? e + (int64_t)k * d_pad + start : x + start, nbytes);
  const Buf rh = buf_of(xh + (int64_t)k * d_pad + start, nbytes);
  const uint64_t* sx = kDecX ? ss + gw0 : nullptr;
  const uint64_t* se = kDecE != kDecPlain ? signs + (int64_t)k * (d_pad >> 6) + gw0 : nullptr;
  const Corr c_e(kDecE == kDecSign ? scales[(int64_t)k * lay.L + tile.l] : 0.0f);
  const Corr c_x(kDecX ? sscales[tile.l] : 0.0f);
  for (int w0 = wave * kTU; w0 < nw; w0 += kTWaves * kTU) {
    if (w0 + kTU <= nw)
      step_words<kDecX, kDecE, kHasE, true>(w0, nw, rx, re, rh, sx, se, c_x, c_e);
    else
      step_words<kDecX, kDecE, kHasE, false>(w0, nw, rx, re, rh, sx, se, c_x, c_e);
  }
}

// ------------------------------------------------------------------ step ahead with averaging
#ifndef SAEF_AVG_CHUNK
#define SAEF_AVG_CHUNK 8
#endif
constexpr int kAvgChunk = SAEF_AVG_CHUNK;  // workers whose loads are issued together

// kUA words of one tile starting at word w0 (offsets relative to the tile;
// lanes past the tile's end compute on zeros and their stores are dropped by
// the buffer range check), all K workers: the local errors are read in
// worker order (pending corrections applied when kDecE) and replaced by their
// mean (binary64 sum in worker order, /K, fp32); then x^(k)_{t+1/2} = x_t -
// mean for every worker when kXh.
template <bool kDecX, int kDecE, bool kXh>
__device__ __forceinline__ void average_words(int K, double inv_k, int L, int l, int64_t d_pad,
                                              int w0, int64_t start, uint32_t nbytes,
                                              uint32_t wbytes, Buf rx, Buf rsx, float s_x,
                                              float* __restrict__ e,
                                              const uint64_t* __restrict__ signs,
                                              const float* __restrict__ scales,
                                              float* __restrict__ xh) {
  const int lane = lane_id();
  const int64_t W = d_pad >> 6;
  const int64_t gw0 = start >> 6;
  const uint32_t off0 = (uint32_t)(w0 * 64 + lane) * 4u;
  // a lane reads the 32-bit half of a sign word that holds its bit (vector
  // registers: this kernel keeps kAvgChunk * kUA words live)
  const uint32_t hoff0 = (uint32_t)w0 * 8u + (uint32_t)(lane >> 5) * 4u;
  double acc[kUA];
#pragma unroll
  for (int u = 0; u < kUA; ++u) acc[u] = 0.0;
  for (int k0 = 0; k0 < K; k0 += kAvgChunk) {
    float ev[kAvgChunk][kUA];
    uint32_t hw[kAvgChunk][kUA];
#pragma unroll
    for (int c = 0; c < kAvgChunk; ++c) {
      const int k = min(k0 + c, K - 1);
      const Buf re = buf_of(e + (int64_t)k * d_pad + start, nbytes);
      const Buf rs = buf_of(signs + (int64_t)k * W + gw0, kDecE != kDecPlain ? wbytes : 0u);
#pragma unroll
      for (int u = 0; u < kUA; ++u) {
        ev[c][u] = buf_ld(re, off0 + 256u * u);
        hw[c][u] = kDecE != kDecPlain
                       ? __builtin_amdgcn_raw_buffer_load_b32(rs, hoff0 + 8u * u, 0, 0)
                       : 0u;
      }
    }
#pragma unroll
    for (int c = 0; c < kAvgChunk; ++c) {
      if (k0 + c >= K) continue;
      const float s = kDecE == kDecSign ? scales[(int64_t)(k0 + c) * L + l] : 0.0f;
#pragma unroll
      for (int u = 0; u < kUA; ++u) {
        float v = ev[c][u];
        if (kDecE == kDecSign) v = v - (half_bit(hw[c][u], lane) ? s : -s);
        if (kDecE == kDecZero) v = half_bit(hw[c][u], lane) ? 0.0f : v;
        acc[u] += (double)v;
      }
    }
  }
  float mean[kUA], xv[kUA];
#pragma unroll
  for (int u = 0; u < kUA; ++u) {
    mean[u] = (float)mean_of(acc[u], inv_k, K);
    xv[u] = 0.0f;
    if (kXh) {
      const uint32_t hx =
          kDecX ? __builtin_amdgcn_raw_buffer_load_b32(rsx, hoff0 + 8u * u, 0, 0) : 0u;
      xv[u] = buf_ld_cached(rx, off0 + 256u * u);
      if (kDecX) xv[u] = xv[u] - (half_bit(hx, lane) ? s_x : -s_x);
    }
  }
  for (int k = 0; k < K; ++k) {
    const Buf re = buf_of(e + (int64_t)k * d_pad + start, nbytes);
    const Buf rh = buf_of(kXh ? xh + (int64_t)k * d_pad + start : e, kXh ? nbytes : 0u);
#pragma unroll
    for (int u = 0; u < kUA; ++u) {
      buf_st(re, off0 + 256u * u, mean[u]);
      if (kXh) buf_st(rh, off0 + 256u * u, xv[u] - mean[u]);
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
  int64_t unit;
  const int64_t n_units = lay.n_tiles * kAvgSplit;
  run_tile_of(blockIdx.x, 1, tile_run_shift(n_units), row0, unit);
  if (unit >= n_units) return;
  const Tile tile = lay.tiles[unit / kAvgSplit];
  const int wave = wave_id();
  const int nw = (tile.count + 63) >> 6;
  // the unit's words of the tile
  constexpr int kUnitWords = kTileElems / 64 / kAvgSplit;
  static_assert(kUnitWords % kUA == 0, "a pass stays in its unit");
  const int uw0 = (int)(unit % kAvgSplit) * kUnitWords;
  const int uw1 = min(nw, uw0 + kUnitWords);
  const uint32_t nbytes = (uint32_t)tile.count * 4u;
  const uint32_t wbytes = (uint32_t)nw * 8u;
  const Buf rx = buf_of(kXh ? x + tile.start : e, kXh ? nbytes : 0u);
  const Buf rsx = buf_of(kDecX ? (const void*)(ss + (tile.start >> 6)) : e, kDecX ? wbytes : 0u);
  const float s_x = kDecX ? sscales[tile.l] : 0.0f;
  for (int w0 = uw0 + wave * kUA; w0 < uw1; w0 += kWaves * kUA)
    average_words<kDecX, kDecE, kXh>(K, inv_k, lay.L, tile.l, lay.d_pad, w0, tile.start, nbytes,
                                     wbytes, rx, rsx, s_x, e, signs, scales, xh);
}

// ------------------------------------------------------------------ aggregate
constexpr int kAggGroup = 64 / kU;  // workers whose sign words one vector load brings

// The sign words of workers k0 .. k0 + kAggGroup - 1 for a pass of a wave
// over the kU words starting at w0 (lane i: word w0 + i mod kU of worker
// k0 + i / kU; 0 past K or past the tile), and their scales (lane c: the
// scale of worker k0 + c): one vector load each, read out with v_readlane.
struct AggGroup {
  u64 words;
  float sc;
};
template <bool kFull>
__device__ __forceinline__ AggGroup agg_group_load(int k0, int K, int L, int l, int64_t W,
                                                   int w0, int count,
                                                   const uint64_t* __restrict__ sw,
                                                   const float* __restrict__ scales) {
  const int lane = lane_id();
  const int kl = k0 + lane / kU, ul = lane % kU;
  AggGroup g;
  g.words = 0ull;
  if (kl < K && (kFull || (w0 + ul) * 64 < count)) g.words = sw[(int64_t)kl * W + w0 + ul];
  g.sc = 0.0f;
  if (lane < kAggGroup && k0 + lane < K) g.sc = scales[(int64_t)(k0 + lane) * L + l];
  return g;
}
// One pass of a wave over the kU words starting at word w0 of a tile (offsets
// relative to the tile; buffer resources over the tile's elements and server
// words): the K worker messages are decoded in order, mean = (sum_k +-scale_k
// in binary64, k order) / K.  Worker words come from sw (the tile's first
// word of worker 0; worker k at sw + k W).  kFull: all kU words lie inside
// the tile (no lane masks).
template <int kMode, bool kDecode, bool kAvg, bool kFull>
__device__ __forceinline__ void aggregate_pass(int K, double inv_k, int L, int l, int64_t W,
                                               int w0, int count,
                                               const uint64_t* __restrict__ sw,
                                               const float* __restrict__ scales, Buf ravg,
                                               Buf res, Buf rss, const Corr& c_old, Buf rx,
                                               ExactSum& acc) {
  const int lane = lane_id();
  const uint32_t off0 = (uint32_t)(w0 * 64 + lane) * 4u;
  constexpr bool kUpdX = kMode == 0 || kDecode;  // x is read and written
  // the first group's words and scales go out before the element loads, so
  // that waiting for them (vector loads complete in order) does not wait for
  // the elements
  AggGroup grp = agg_group_load<kFull>(0, K, L, l, W, w0, count, sw, scales);
  __builtin_amdgcn_sched_barrier(0);
  float ev[kU], xv[kU];
  const u64 mo = (kMode == 1 && kDecode) ? buf_ld_words(rss, w0, kU) : 0ull;  // old words
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    ev[u] = kMode == 1 ? buf_ld(res, off0 + 256u * u) : 0.0f;
    xv[u] = kUpdX ? buf_ld(rx, off0 + 256u * u) : 0.0f;
  }
  double acc_m[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) acc_m[u] = 0.0;
  for (int k0 = 0; k0 < K; k0 += kAggGroup) {
    if (k0 > 0) grp = agg_group_load<kFull>(k0, K, L, l, W, w0, count, sw, scales);
#pragma unroll
    for (int c = 0; c < kAggGroup; ++c) {
      if (k0 + c >= K) break;  // wave-uniform
      // +-scale_k in binary64: the two values differ only in the sign bit
      const double sd =
          (double)__uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(grp.sc), c));
      const uint32_t pos_hi = (uint32_t)__double2hiint(sd);
      const uint32_t lo_bits = (uint32_t)__double2loint(sd);
      const uint32_t neg_hi = pos_hi ^ 0x80000000u;
#pragma unroll
      for (int u = 0; u < kU; ++u)
        acc_m[u] += __hiloint2double(
            (int)sel_by_bit(word_of(grp.words, c * kU + u), pos_hi, neg_hi), (int)lo_bits);
    }
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const uint32_t off = off0 + 256u * u;
    const bool ok = kFull || (w0 + u) * 64 + lane < count;
    const float mean = (float)mean_of(acc_m[u], inv_k, K);
    if (kAvg) buf_st(ravg, off, mean);
    if (kMode == 1) {
      float evc = ev[u];
      if (kDecode) {
        const float c = c_old(word_of(mo, u));
        evc = evc - c;                   // e_t = Delta_t - C(Delta_t)
        buf_st(rx, off, xv[u] - c);      // re-update x_t = x_{t-1} - C(Delta_t)
      }
      // Delta_{t+1} = e_t + (1/K) sum_k C(Delta^(k))
      float D = evc + mean;
      if (!kFull) D = ok ? D : 0.0f;
      const u64 word = __ballot(ok && D >= 0.0f);
      if (lane == 0) buf_st_word(rss, (uint32_t)(w0 + u) * 8u, word);
      acc.add(D);
      buf_st(res, off, D);
    } else {
      buf_st(rx, off, xv[u] - mean);  // single-way: the mean itself comes back
    }
  }
}

// Grid: run_padded_tiles(n_tiles) workgroups, one per tile in the XCD-aware
// tile order of run_tile_of (neighbouring tiles, whose sign words share cache
// lines, run on one XCD).  Wave w takes words w*kU .. w*kU+kU-1 of the tile
// (one pass over a whole tile), then strides by 4*kU words.
template <int kMode, bool kDecode, bool kAvg>
__global__ __launch_bounds__(kSBlock) void k_aggregate(DevLayout lay, int K, double inv_k,
                                                      const uint64_t* __restrict__ signs,
                                                      const float* __restrict__ scales,
                                                      float* __restrict__ avg,
                                                      float* __restrict__ es,
                                                      uint64_t* __restrict__ ss,
                                                      const float* __restrict__ sscales,
                                                      float* __restrict__ x) {
  int row0;
  int64_t ti;
  run_tile_of(blockIdx.x, 1, tile_run_shift(lay.n_tiles), row0, ti);
  if (ti >= lay.n_tiles) return;
  const Tile tile = lay.tiles[ti];
  const int nw = (tile.count + 63) >> 6;
  const uint32_t nbytes = (uint32_t)tile.count * 4u;
  const int64_t gw0 = tile.start >> 6;
  const Buf ravg = buf_of(kAvg ? avg + tile.start : x + tile.start, nbytes);
  const Buf res = buf_of(kMode == 1 ? es + tile.start : x + tile.start, nbytes);
  const Buf rss = buf_of(kMode == 1 ? ss + gw0 : signs, (uint32_t)nw * 8u);
  const Buf rx = buf_of(x + tile.start, nbytes);
  const Corr c_old((kMode == 1 && kDecode) ? sscales[tile.l] : 0.0f);
  const int64_t W = lay.d_pad >> 6;
  ExactSum acc;
  u64 lo = 0, hi = 0;
  bool bad = false;
  for (int w0 = wave_id() * kU; w0 < nw; w0 += kSWaves * kU) {
    if ((w0 + kU) * 64 <= tile.count) {
      aggregate_pass<kMode, kDecode, kAvg, true>(K, inv_k, lay.L, tile.l, W, w0, tile.count,
                                                 signs + gw0, scales, ravg, res, rss, c_old, rx,
                                                 acc);
    } else {
      aggregate_pass<kMode, kDecode, kAvg, false>(K, inv_k, lay.L, tile.l, W, w0, tile.count,
                                                  signs + gw0, scales, ravg, res, rss, c_old, rx,
                                                  acc);
    }
    if (kMode == 1) acc.added(kU, lo, hi, bad);
  }
  if (kMode == 1) {
    acc.finish(lo, hi, bad);
    block_partial<kSWaves>(lay, lay.k_max, ti, lo, hi, bad);
  }
}

// ------------------------------------------------------------------ materialize
// Grid: n_tiles * rows, rows = K (+1 when the server row is requested); row K
// is the server error and the weights.
// e_out may be e, es_out es and x_out x (in place): every element is read and
// then written by the same lane, so those pairs are not restrict-qualified.
__global__ __launch_bounds__(kBlock) void k_materialize(
    DevLayout lay, int K, int rows, int mode, const float* e,
    const uint64_t* __restrict__ signs, const float* __restrict__ scales, float* e_out,
    const float* es, const float* x, const uint64_t* __restrict__ ss,
    const float* __restrict__ sscales, float* es_out, float* x_out) {
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
// Every tile holds at most kTileElems elements (a tensor of at most 2^28
// elements never needs larger tiles), so the waves' word ranges cover it.
static_assert((int64_t)kTileElems * kMaxTilesPerTensor >= kMaxTensor,
              "tiles of a maximal tensor hold kTileElems elements");
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


// ------------------------------------------------------------------ stream probe
// The HBM ceiling of the worker compression's access pattern: c = a + b over
// n elements (2 reads + 1 write of fp32), one 256-thread workgroup per
// 2048-element tile, kU words per wave, non-temporal buffer accesses.
// kTwo: c = a + b; else c = a (c may be a: every element is read and then
// written by the same lane, so a and c are not restrict-qualified).
template <bool kTwo>
__global__ __launch_bounds__(kSBlock) void k_stream_probe(const float* a,
                                                         const float* __restrict__ b,
                                                         float* c, int64_t n) {
  const int64_t start = (int64_t)blockIdx.x * kTileElems;
  const uint32_t nbytes = (uint32_t)min((int64_t)kTileElems, n - start) * 4u;
  const Buf ra = buf_of(a + start, nbytes);
  const Buf rb = buf_of(kTwo ? b + start : a + start, nbytes);
  const Buf rc = buf_of(c + start, nbytes);
  for (int w0 = wave_id() * kU; w0 * 256u < nbytes; w0 += kSWaves * kU) {
    const uint32_t off0 = (uint32_t)(w0 * 64 + lane_id()) * 4u;
    float av[kU], bv[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      av[u] = buf_ld(ra, off0 + 256u * u);
      bv[u] = kTwo ? buf_ld(rb, off0 + 256u * u) : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) buf_st(rc, off0 + 256u * u, kTwo ? av[u] + bv[u] : av[u]);
  }
}

}  // namespace

hipError_t launch_stream_probe(const float* a, const float* b, float* c, int64_t n,
                               hipStream_t s) {
  const LaunchEvents ev;
  const dim3 grid((unsigned)((n + kTileElems - 1) / kTileElems));
  if (b != nullptr)
    SAEF_LAUNCH(k_stream_probe<true>, grid, dim3(kSBlock), 0, s, a, b, c, n);
  else
    SAEF_LAUNCH(k_stream_probe<false>, grid, dim3(kSBlock), 0, s, a, b, c, n);
  return hipGetLastError();
}

hipError_t launch_compress(const DevLayout& lay, int K, float lr, float mu, const float* g,
                           float* m, float* e, uint64_t* signs, const float* scales, bool decode,
                           hipStream_t s, const LaunchEvents& ev) {
  const dim3 grid((unsigned)(lay.n_tiles * K));
#define SAEF_CMP(KERNEL, D) \
  SAEF_LAUNCH((KERNEL<D>), grid, dim3(kSBlock), 0, s, lay, K, lr, mu, g, m, e, signs, scales)
  if (m != nullptr) {
    if (decode) SAEF_CMP(k_compress_mom, true); else SAEF_CMP(k_compress_mom, false);
  } else {
    if (decode) SAEF_CMP(k_compress, true); else SAEF_CMP(k_compress, false);
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
  const dim3 grid((unsigned)run_padded_tiles(lay.n_tiles));
  const double ik = inv_pow2(K);
#define SAEF_AGG(M, D, A)                                                                  \
  SAEF_LAUNCH((k_aggregate<M, D, A>), grid, dim3(kSBlock), 0, s, lay, K, ik, signs, \
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
    const dim3 grid((unsigned)run_padded_tiles(lay.n_tiles * kAvgSplit));
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
    const dim3 grid((unsigned)(run_padded_tiles(lay.n_tiles * kStepSplit) * K));
#define SAEF_ST(DX, DE)                                                                \
  SAEF_LAUNCH((k_step<DX, DE, true>), grid, dim3(kTBlock), 0, s, lay, K, x, srv_signs, \
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
  const dim3 grid((unsigned)run_padded_tiles(lay.n_tiles * kStepSplit));
  if (decode_x) {
    SAEF_LAUNCH((k_step<true, kDecPlain, false>), grid, dim3(kTBlock), 0, s, lay, 1, x, srv_signs,
                srv_scales, nullptr, nullptr, nullptr, xh);
  } else {
    SAEF_LAUNCH((k_step<false, kDecPlain, false>), grid, dim3(kTBlock), 0, s, lay, 1, x, srv_signs,
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
