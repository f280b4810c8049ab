// HIP kernels of the layer-wise Top-K compressor on gfx950 (CDNA4, wave64).
//
// C(v) keeps the k_l elements of largest |v| of each tensor (equal
// magnitudes: the lower index first) and zeroes the others.  The kept set is
// found by a radix select on the 31-bit key |v| (the bit pattern of a
// non-negative float orders like its value), per (row, tensor):
//   pass 1  histogram of key bits 30..20 (2048 bins) per 64Ki-element chunk,
//           built with LDS atomics and stored with plain stores; a pick
//           kernel adds the chunk histograms of the tensor and finds the
//           bucket that holds the k-th largest key;
//   pass 2  bits 19..9 of the elements of that bucket;
//   pass 3  bits 8..0: the threshold key tau and how many of the elements
//           equal to tau are kept; if not all, the chunk that holds the cut
//           is scanned in index order for the last kept index iota.
// Emit: kept = key > tau, or key == tau and index <= iota; the selection
// words (one ballot per 64 elements) and the kept count of each tile; an
// exclusive scan of the counts over the tensor's tiles; then the rank words
// and the kept values in index order, and the kept elements of the error set
// to 0 (e = Delta - C(Delta) is Delta elsewhere).  All of it is integer
// counting, so the kept set does not depend on the launch geometry.
//
// The server runs the same passes on its one row (row k_max of the scratch)
// after k_tk_aggregate has formed Delta = e_srv + mean of the K messages.
#include "saef_device.h"
#include "saef_internal.h"

namespace saef {
namespace {

constexpr uint32_t kFiniteLimit = 0x7F800000u;  // keys >= this are Inf or NaN
constexpr int kTkU = 4;                         // words per wave per pass (first pass, server)
constexpr int kTkH = 8;                         // words per wave per pass (later passes)
constexpr int kTkE = 16;                        // words per wave per pass (emit)
constexpr int kBig = 1024;                      // threads of the single-row (server) kernels
#ifndef SAEF_TK_HIST_THREADS
#define SAEF_TK_HIST_THREADS 256
#endif
#ifndef SAEF_TK_NT
#define SAEF_TK_NT 1
#endif
// Guarded loads without a branch: the load of p[ok ? j : 0] is always
// issued (p[0] must exist) and its value replaced by 0 when !ok.  A branch
// around each load makes the compiler wait for it before the next one.
__device__ __forceinline__ float ld_nt_or0(const float* p, int64_t j, bool ok) {
  const float v = __builtin_nontemporal_load(p + (ok ? j : 0));
  return ok ? v : 0.0f;
}
__device__ __forceinline__ float ld_or0(const float* p, int64_t j, bool ok) {
  const float v = p[ok ? j : 0];
  return ok ? v : 0.0f;
}
// loads of the later passes (the error was just written by the first pass)
__device__ __forceinline__ float ld_pass_or0(const float* p, int64_t j, bool ok) {
  return SAEF_TK_NT ? ld_nt_or0(p, j, ok) : ld_or0(p, j, ok);
}
constexpr int kAggK = 4;                        // workers whose messages are read together

__device__ __forceinline__ uint32_t key_of(float v) { return __float_as_uint(v) & 0x7FFFFFFFu; }

__device__ __forceinline__ u64 lanemask_lt(int lane) {
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Lane of the n-th (1-based) set bit of m; m has at least n set bits.
__device__ __forceinline__ int nth_set_bit(u64 m, int n) {
  for (int i = 1; i < n; ++i) m &= m - 1;
  return __builtin_ctzll(m);
}

// The digit of each radix pass and the prefix an element must match.
template <int kPass>
struct Digit;
template <>
struct Digit<1> {
  static constexpr int kBins = kTkBins;
  static constexpr int kBits = 11;
  __device__ static uint32_t get(uint32_t key) { return key >> 20; }
  __device__ static bool match(uint32_t, uint32_t) { return true; }
};
template <>
struct Digit<2> {
  static constexpr int kBins = kTkBins;
  static constexpr int kBits = 11;
  __device__ static uint32_t get(uint32_t key) { return (key >> 9) & (kTkBins - 1); }
  __device__ static bool match(uint32_t key, uint32_t prefix) { return (key >> 20) == prefix; }
};
template <>
struct Digit<3> {
  static constexpr int kBins = kTkBins3;
  static constexpr int kBits = 9;
  __device__ static uint32_t get(uint32_t key) { return key & (kTkBins3 - 1); }
  __device__ static bool match(uint32_t key, uint32_t prefix) { return (key >> 9) == prefix; }
};

template <int kBins>
__device__ __forceinline__ void hist_clear(uint32_t* h) {
  for (int i = threadIdx.x; i < kBins; i += blockDim.x) h[i] = 0;
  __syncthreads();
}

// Stores the workgroup's LDS histogram (plain stores).
template <int kBins>
__device__ __forceinline__ void hist_store(const uint32_t* h, uint32_t* out) {
  __syncthreads();
  for (int i = threadIdx.x; i < kBins; i += blockDim.x) out[i] = h[i];
}

__device__ __forceinline__ uint32_t* chunk_hist(const TkDev& tk, int row, int64_t ci) {
  return tk.hist + ((int64_t)row * tk.n_chunks + ci) * kTkBins;
}

// ------------------------------------------------------------------ pass 1 (workers)
// kTkU words of one worker's chunk: m <- fma(mu, m, g) with kMom, Delta =
// fma(lr, m or g, e), Delta stored into e, pass-1 histogram of its key.
template <bool kMom, bool kFull>
__device__ __forceinline__ void delta_words(int w0, int nw, int count, float lr, float mu,
                                            const float* __restrict__ gk, float* __restrict__ mk,
                                            float* __restrict__ ek, uint32_t* h, bool& bad) {
  const int lane = lane_id();
  float gv[kTkU], ev[kTkU], mv[kTkU];
#pragma unroll
  for (int u = 0; u < kTkU; ++u) {
    const int j = (w0 + u) * 64 + lane;
    const bool ok = kFull || ((w0 + u < nw) && j < count);
    gv[u] = ld_nt_or0(gk, j, ok);
    ev[u] = ld_nt_or0(ek, j, ok);
    mv[u] = kMom ? ld_nt_or0(mk, j, ok) : 0.0f;
  }
#pragma unroll
  for (int u = 0; u < kTkU; ++u) {
    const int j = (w0 + u) * 64 + lane;
    const bool ok = kFull || ((w0 + u < nw) && j < count);
    if (!ok) continue;
    float step = gv[u];
    if (kMom) {
      step = __builtin_fmaf(mu, mv[u], gv[u]);  // m^(k)_{t+1} = mu m^(k)_t + grad
      st_nt(mk + j, step);
    }
    const float p = __builtin_fmaf(lr, step, ev[u]);  // Delta^(k) = e^(k) + lr m^(k)_{t+1}
    st_nt(ek + j, p);
    const uint32_t key = key_of(p);
    bad |= key >= kFiniteLimit;
    atomicAdd(&h[Digit<1>::get(key)], 1u);
  }
}

// Grid: n_chunks * K workgroups; workgroup b handles worker b % K of chunk b / K.
template <bool kMom>
__global__ __launch_bounds__(kBlock) void k_tk_delta(DevLayout lay, TkDev tk, int K, float lr,
                                                     float mu, const float* __restrict__ g,
                                                     float* __restrict__ m,
                                                     float* __restrict__ e) {
  __shared__ uint32_t h[kTkBins];
  const int k = (int)(blockIdx.x % (unsigned)K);
  const int64_t ci = blockIdx.x / (unsigned)K;
  const TkChunk c = tk.chunks[ci];
  hist_clear<kTkBins>(h);
  const int64_t row = (int64_t)k * lay.d_pad + c.start;
  const float* gk = g + row;
  float* mk = kMom ? m + row : nullptr;
  float* ek = e + row;
  const int nw = (c.count + 63) >> 6;
  bool bad = false;
  for (int w0 = wave_id() * kTkU; w0 < nw; w0 += kWaves * kTkU) {
    if ((w0 + kTkU) * 64 <= c.count)
      delta_words<kMom, true>(w0, nw, c.count, lr, mu, gk, mk, ek, h, bad);
    else
      delta_words<kMom, false>(w0, nw, c.count, lr, mu, gk, mk, ek, h, bad);
  }
  if (__ballot(bad) != 0 && lane_id() == 0) atomicOr(lay.status, kStatusRange);
  hist_store<kTkBins>(h, chunk_hist(tk, k, ci));
}

// ------------------------------------------------------------------ passes 2 and 3
// Grid: n_chunks * R workgroups of kThreads (R rows from row0; data row r at
// data + r d_pad).
template <int kPass, int kThreads>
__global__ __launch_bounds__(kThreads) void k_tk_hist(DevLayout lay, TkDev tk, int R, int row0,
                                                      const float* __restrict__ data) {
  constexpr int B = Digit<kPass>::kBins;
  constexpr int kW = kThreads / kWave;
  __shared__ uint32_t h[B];
  const int r = (int)(blockIdx.x % (unsigned)R);
  const int64_t ci = blockIdx.x / (unsigned)R;
  const TkChunk c = tk.chunks[ci];
  const uint32_t prefix = tk.sel[(int64_t)(row0 + r) * lay.L + c.l].prefix;
  hist_clear<B>(h);
  const float* dr = data + (int64_t)r * lay.d_pad + c.start;
  const int lane = lane_id();
  const int nw = (c.count + 63) >> 6;
  for (int w0 = wave_id() * kTkH; w0 < nw; w0 += kW * kTkH) {
    float v[kTkH];
#pragma unroll
    for (int u = 0; u < kTkH; ++u) {
      const int j = (w0 + u) * 64 + lane;
      v[u] = ld_pass_or0(dr, j, w0 + u < nw && j < c.count);
    }
#pragma unroll
    for (int u = 0; u < kTkH; ++u) {
      const int j = (w0 + u) * 64 + lane;
      const uint32_t key = key_of(v[u]);
      if (w0 + u < nw && j < c.count && Digit<kPass>::match(key, prefix))
        atomicAdd(&h[Digit<kPass>::get(key)], 1u);
    }
  }
  hist_store<B>(h, chunk_hist(tk, row0 + r, ci));
}

// ------------------------------------------------------------------ reduce and pick
// Grid: R * L * red_split workgroups: group s adds the chunk histograms
// [s kTkRedChunks, (s+1) kTkRedChunks) of the tensor (those that exist).
template <int kPass>
__global__ __launch_bounds__(kBlock) void k_tk_sum(DevLayout lay, TkDev tk, int row0) {
  constexpr int B = Digit<kPass>::kBins;
  constexpr int kPer = B / kBlock;
  const int S = tk.red_split;
  const int s = (int)(blockIdx.x % S);
  const int l = (int)((blockIdx.x / S) % lay.L);
  const int r = (int)(blockIdx.x / ((unsigned)S * lay.L));
  const int row = row0 + r;
  const TkTensor t = tk.tens[l];
  const int c0 = min(t.nchunks, s * kTkRedChunks), c1 = min(t.nchunks, c0 + kTkRedChunks);
  uint32_t acc[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) acc[j] = 0;
  for (int c = c0; c < c1; ++c) {
    const uint32_t* src = chunk_hist(tk, row, t.first_chunk + c) + threadIdx.x * kPer;
#pragma unroll
    for (int j = 0; j < kPer; ++j) acc[j] += src[j];
  }
  uint32_t* dst = tk.hist2 + (((int64_t)row * lay.L + l) * S + s) * kTkBins + threadIdx.x * kPer;
#pragma unroll
  for (int j = 0; j < kPer; ++j) dst[j] = acc[j];
}

// Grid: R * L workgroups.  Adds the tensor's histograms (the chunk
// histograms, or the red_split partial sums), finds the bin that holds the
// need-th largest key counted from the top, and updates the selection state.
// After pass 3 the prefix is the threshold key tau; when only some of the
// elements equal to tau are kept, the chunk of the cut and the rank in it
// are located from the chunk histograms.
template <int kPass>
__global__ __launch_bounds__(kBlock) void k_tk_pick(DevLayout lay, TkDev tk, int row0) {
  constexpr int B = Digit<kPass>::kBins;
  constexpr int kPer = B / kBlock;
  __shared__ uint32_t s_tot[kBlock];
  __shared__ uint32_t s_above[kBlock];
  const int l = (int)(blockIdx.x % lay.L);
  const int r = (int)(blockIdx.x / lay.L);
  const int row = row0 + r;
  const TkTensor t = tk.tens[l];
  TkSel* st = tk.sel + (int64_t)row * lay.L + l;
  const int S = tk.red_split;
  uint32_t cnt[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) cnt[j] = 0;
  if (S > 1) {
    const uint32_t* src = tk.hist2 + ((int64_t)row * lay.L + l) * S * kTkBins + threadIdx.x * kPer;
    for (int s = 0; s < S; ++s)
#pragma unroll
      for (int j = 0; j < kPer; ++j) cnt[j] += src[(int64_t)s * kTkBins + j];
  } else {
    for (int c = 0; c < t.nchunks; ++c) {
      const uint32_t* src = chunk_hist(tk, row, t.first_chunk + c) + threadIdx.x * kPer;
#pragma unroll
      for (int j = 0; j < kPer; ++j) cnt[j] += src[j];
    }
  }
  uint32_t tot = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) tot += cnt[j];
  s_tot[threadIdx.x] = tot;
  const int64_t need = (kPass == 1) ? t.keep : st->need;
  const uint32_t prefix = (kPass == 1) ? 0u : st->prefix;
  __syncthreads();
  if (threadIdx.x == 0) {
    // elements in the bins above each thread's range (a tensor has < 2^32)
    uint32_t run = 0;
    for (int i = kBlock - 1; i >= 0; --i) {
      s_above[i] = run;
      run += s_tot[i];
    }
  }
  __syncthreads();
  int64_t run = s_above[threadIdx.x];
  if (run >= need || run + tot < need) return;  // the need-th key is not in this range
  for (int j = kPer - 1; j >= 0; --j) {
    if (run + cnt[j] >= need) {
      const uint32_t bin = (uint32_t)(threadIdx.x * kPer + j);
      const uint32_t np = (prefix << Digit<kPass>::kBits) | bin;
      const int64_t left = need - run;  // to take from this bin
      st->prefix = np;
      st->need = left;
      if (kPass == 3) {
        if (left == (int64_t)cnt[j]) {
          st->cut_chunk = -1;
          st->iota = INT64_MAX;  // every element equal to tau is kept
        } else {
          int64_t before = 0;
          for (int c = 0; c < t.nchunks; ++c) {
            const int64_t in_c = chunk_hist(tk, row, t.first_chunk + c)[bin];
            if (before + in_c >= left) {
              st->cut_chunk = c;
              st->cut_rank = left - before;
              break;
            }
            before += in_c;
          }
        }
      }
      return;
    }
    run += cnt[j];
  }
}

// ------------------------------------------------------------------ ties
// Grid: R * L workgroups of kBig threads.  When only part of the elements
// equal to tau are kept, finds the cut_rank-th of them in index order in the
// chunk of the cut; its absolute element index becomes iota.  Each wave
// counts the ties of its own contiguous slice of the chunk, a prefix over
// the waves names the slice of the cut, and that wave scans its slice again
// (from the caches) to place it.
__global__ __launch_bounds__(kBig) void k_tk_ties(DevLayout lay, TkDev tk, int row0,
                                                  const float* __restrict__ data) {
  constexpr int kW = kBig / kWave;
  __shared__ uint32_t s_cnt[kW];
  const int l = (int)(blockIdx.x % lay.L);
  const int r = (int)(blockIdx.x / lay.L);
  TkSel* st = tk.sel + (int64_t)(row0 + r) * lay.L + l;
  if (st->cut_chunk < 0) return;  // uniform over the workgroup
  const TkTensor t = tk.tens[l];
  const TkChunk c = tk.chunks[t.first_chunk + st->cut_chunk];
  const uint32_t tau = st->prefix;
  const int64_t target = st->cut_rank;
  const float* dr = data + (int64_t)r * lay.d_pad + c.start;
  const int lane = lane_id();
  const int wave = wave_id();
  const int nw = (c.count + 63) >> 6;
  const int per = (nw + kW - 1) / kW;  // words of each wave's slice
  const int w_lo = min(nw, wave * per), w_hi = min(nw, w_lo + per);
  uint32_t mine = 0;
  for (int w0 = w_lo; w0 < w_hi; w0 += kTkE) {
    float v[kTkE];
#pragma unroll
    for (int u = 0; u < kTkE; ++u) {
      const int j = (w0 + u) * 64 + lane;
      v[u] = ld_nt_or0(dr, j, w0 + u < w_hi && j < c.count);
    }
#pragma unroll
    for (int u = 0; u < kTkE; ++u) {
      const int j = (w0 + u) * 64 + lane;
      mine += (uint32_t)__popcll(__ballot(w0 + u < w_hi && j < c.count && key_of(v[u]) == tau));
    }
  }
  if (lane == 0) s_cnt[wave] = mine;
  __syncthreads();
  int64_t before = 0;
  for (int i = 0; i < wave; ++i) before += s_cnt[i];
  if (!(before < target && target <= before + mine)) return;
  // this wave's slice holds the cut
  for (int w0 = w_lo; w0 < w_hi; w0 += kTkE) {
    float v[kTkE];
#pragma unroll
    for (int u = 0; u < kTkE; ++u) {
      const int j = (w0 + u) * 64 + lane;
      v[u] = ld_or0(dr, j, w0 + u < w_hi && j < c.count);
    }
#pragma unroll
    for (int u = 0; u < kTkE; ++u) {
      const int j = (w0 + u) * 64 + lane;
      const u64 m = __ballot(w0 + u < w_hi && j < c.count && key_of(v[u]) == tau);
      const int n = (int)__popcll(m);
      if (before < target && target <= before + n) {
        const int b = nth_set_bit(m, (int)(target - before));
        if (lane == 0) st->iota = c.start + (int64_t)(w0 + u) * 64 + b;
      }
      before += n;
    }
  }
}

// ------------------------------------------------------------------ emit
// Grid: per_wave_grid(lay) * R workgroups; wave w of workgroup b owns tile
// 4 (b / R) + w of row b % R.  Writes the selection words of the tile and
// its kept count.
__global__ __launch_bounds__(kBlock) void k_tk_emit1(DevLayout lay, TkDev tk, int R, int row0,
                                                     const float* __restrict__ data,
                                                     uint64_t* __restrict__ sel) {
  const int r = (int)(blockIdx.x % (unsigned)R);
  const int64_t ti = (int64_t)(blockIdx.x / (unsigned)R) * kWaves + wave_id();
  if (ti >= lay.n_tiles) return;
  const Tile tile = lay.tiles[ti];
  const TkSel st = tk.sel[(int64_t)(row0 + r) * lay.L + tile.l];
  const uint32_t tau = st.prefix;
  const int64_t iota = st.iota;
  const int lane = lane_id();
  const int nw = (tile.count + 63) >> 6;
  const float* dr = data + (int64_t)r * lay.d_pad + tile.start;
  uint64_t* sr = sel + (int64_t)r * (lay.d_pad >> 6) + (tile.start >> 6);
  uint32_t cnt = 0;
  for (int w0 = 0; w0 < nw; w0 += kTkE) {
    float v[kTkE];
#pragma unroll
    for (int u = 0; u < kTkE; ++u) {
      const int j = (w0 + u) * 64 + lane;
      v[u] = ld_pass_or0(dr, j, w0 + u < nw && j < tile.count);
    }
#pragma unroll
    for (int u = 0; u < kTkE; ++u) {
      const int w = w0 + u;
      if (w >= nw) continue;
      const int j = w * 64 + lane;
      const uint32_t key = key_of(v[u]);
      const bool kept = j < tile.count &&
                        (key > tau || (key == tau && tile.start + j <= iota));
      const u64 word = __ballot(kept);
      if (lane == 0) sr[w] = word;
      cnt += (uint32_t)__popcll(word);
    }
  }
  if (lane == 0) tk.tile_cnt[(int64_t)(row0 + r) * lay.n_tiles + ti] = cnt;
}

// Grid: R * L workgroups: exclusive prefix of the kept counts over the
// tensor's tiles, in tile order, in place.
__global__ __launch_bounds__(kBlock) void k_tk_scan(DevLayout lay, TkDev tk, int row0) {
  __shared__ uint32_t s[kBlock];
  const int l = (int)(blockIdx.x % lay.L);
  const int r = (int)(blockIdx.x / lay.L);
  const TensorInfo t = lay.tensors[l];
  uint32_t* cnt = tk.tile_cnt + (int64_t)(row0 + r) * lay.n_tiles + t.first_tile;
  uint32_t carry = 0;
  for (int b = 0; b < t.ntiles; b += kBlock) {
    const int i = b + threadIdx.x;
    const uint32_t v = i < t.ntiles ? cnt[i] : 0u;
    s[threadIdx.x] = v;
    __syncthreads();
    // inclusive scan (Hillis-Steele) in LDS
    for (int off = 1; off < kBlock; off <<= 1) {
      const uint32_t add = (int)threadIdx.x >= off ? s[threadIdx.x - off] : 0u;
      __syncthreads();
      s[threadIdx.x] += add;
      __syncthreads();
    }
    if (i < t.ntiles) cnt[i] = carry + s[threadIdx.x] - v;
    const uint32_t total = s[kBlock - 1];
    __syncthreads();
    carry += total;
  }
}

// Grid: per_wave_grid(lay) * R workgroups, tiles as in k_tk_emit1.  Rank
// words, the kept values in index order, the kept elements of data set to
// 0; kX (server): x <- x - Delta at the kept elements (C(Delta) is zero
// elsewhere).
template <bool kX>
__global__ __launch_bounds__(kBlock) void k_tk_emit2(DevLayout lay, TkDev tk, int R, int row0,
                                                     float* __restrict__ data,
                                                     const uint64_t* __restrict__ sel,
                                                     uint32_t* __restrict__ rank,
                                                     float* __restrict__ vals,
                                                     float* __restrict__ x) {
  const int r = (int)(blockIdx.x % (unsigned)R);
  const int64_t ti = (int64_t)(blockIdx.x / (unsigned)R) * kWaves + wave_id();
  if (ti >= lay.n_tiles) return;
  const Tile tile = lay.tiles[ti];
  const TkTensor t = tk.tens[tile.l];
  const int lane = lane_id();
  const int nw = (tile.count + 63) >> 6;
  const int64_t W = lay.d_pad >> 6;
  float* dr = data + (int64_t)r * lay.d_pad + tile.start;
  const uint64_t* sr = sel + (int64_t)r * W + (tile.start >> 6);
  uint32_t* rr = rank + (int64_t)r * W + (tile.start >> 6);
  float* vr = vals + (int64_t)r * tk.total_keep + t.voff;
  float* xt = kX ? x + tile.start : nullptr;
  uint32_t run = tk.tile_cnt[(int64_t)(row0 + r) * lay.n_tiles + ti];
  const u64 lt = lanemask_lt(lane);
  for (int w0 = 0; w0 < nw; w0 += kTkE) {
    u64 m[kTkE];
#pragma unroll
    for (int u = 0; u < kTkE; ++u) {
      const u64 word = sr[min(w0 + u, nw - 1)];  // always in the tile; masked below
      m[u] = (w0 + u < nw) ? word : 0ull;
    }
    // all loads of the kept elements first, then the stores
    float v[kTkE];
    uint32_t pos[kTkE];
    bool kept[kTkE];
#pragma unroll
    for (int u = 0; u < kTkE; ++u) {
      pos[u] = run + (uint32_t)__popcll(m[u] & lt);
      kept[u] = ((m[u] >> lane) & 1ull) && pos[u] < (uint32_t)t.keep;  // pos < keep always holds
      v[u] = ld_or0(dr, (w0 + u) * 64 + lane, kept[u]);
      run += (uint32_t)__popcll(m[u]);
    }
    float xv[kTkE];
#pragma unroll
    for (int u = 0; u < kTkE; ++u) xv[u] = kX ? ld_or0(xt, (w0 + u) * 64 + lane, kept[u]) : 0.0f;
#pragma unroll
    for (int u = 0; u < kTkE; ++u) {
      const int w = w0 + u;
      if (w >= nw) continue;
      if (lane == 0) rr[w] = pos[u];  // lane 0: the kept count before this word
      if (kept[u]) {
        const int j = w * 64 + lane;
        vr[pos[u]] = v[u];
        dr[j] = 0.0f;  // e = Delta - C(Delta) = 0 at a kept element
        if (kX) xt[j] = xv[u] - v[u];
      }
    }
  }
}

// ------------------------------------------------------------------ server aggregation
// kTkU words of a chunk: mean of the K decoded messages (binary64, worker
// order, /K, fp32); mode 1: Delta = e_srv + mean stored into e_srv and its
// pass-1 histogram; mode 0: x <- x - mean.
template <int kMode, bool kAvg, bool kFull>
__device__ __forceinline__ void tk_aggregate_words(
    const DevLayout& lay, const TkDev& tk, int K, double inv_k, int64_t voff, uint32_t keep,
    int64_t start,
    int w0, int nw, int count, const uint64_t* __restrict__ sel,
    const uint32_t* __restrict__ rank, const float* __restrict__ vals, float* __restrict__ avg,
    float* __restrict__ es, float* __restrict__ x, uint32_t* h, bool& bad) {
  const int lane = lane_id();
  const int64_t W = lay.d_pad >> 6;
  const int64_t gw0 = (start >> 6) + w0;
  const u64 lt = lanemask_lt(lane);
  float dv[kTkU];
#pragma unroll
  for (int u = 0; u < kTkU; ++u) {
    const int j = (w0 + u) * 64 + lane;
    const bool ok = kFull || ((w0 + u < nw) && j < count);
    dv[u] = ld_nt_or0((kMode == 1 ? es : x) + start, j, ok);
  }
  double acc[kTkU];
#pragma unroll
  for (int u = 0; u < kTkU; ++u) acc[u] = 0.0;
  for (int k0 = 0; k0 < K; k0 += kAggK) {
    // the words and ranks of kAggK workers, then all their value gathers
    u64 m[kAggK][kTkU];
    uint32_t rb[kAggK][kTkU];
#pragma unroll
    for (int c = 0; c < kAggK; ++c) {
      const bool kin = k0 + c < K;
      const int64_t row = kin ? (int64_t)(k0 + c) * W : 0;  // absent workers read worker 0
#pragma unroll
      for (int u = 0; u < kTkU; ++u) {
        const bool w_ok = kin && (kFull || w0 + u < nw);
        // always issued at a word of the chunk that exists, masked after
        const int64_t at = gw0 + row + ((kFull || w0 + u < nw) ? u : 0);
        const u64 mw = sel[at];
        const uint32_t rw = rank[at];
        m[c][u] = w_ok ? mw : 0ull;
        rb[c][u] = w_ok ? rw : 0u;
      }
    }
    float cv[kAggK][kTkU];
#pragma unroll
    for (int c = 0; c < kAggK; ++c) {
      const int kk = (k0 + c < K) ? k0 + c : 0;
      const float* vk = vals + (int64_t)kk * tk.total_keep + voff;
#pragma unroll
      for (int u = 0; u < kTkU; ++u) {
        const uint32_t pos = rb[c][u] + (uint32_t)__popcll(m[c][u] & lt);
        cv[c][u] = ld_or0(vk, pos, ((m[c][u] >> lane) & 1ull) && pos < keep);
      }
    }
#pragma unroll
    for (int c = 0; c < kAggK; ++c)
#pragma unroll
      for (int u = 0; u < kTkU; ++u) acc[u] += (double)cv[c][u];  // worker order; absent: +0
  }
#pragma unroll
  for (int u = 0; u < kTkU; ++u) {
    const int j = (w0 + u) * 64 + lane;
    const bool ok = kFull || ((w0 + u < nw) && j < count);
    if (!ok) continue;
    const float mean = (float)mean_of(acc[u], inv_k, K);
    if (kAvg) avg[start + j] = mean;
    if (kMode == 1) {
      const float D = dv[u] + mean;  // Delta_{t+1} = e_t + (1/K) sum_k C(Delta^(k))
      st_nt(es + start + j, D);
      const uint32_t key = key_of(D);
      bad |= key >= kFiniteLimit;
      atomicAdd(&h[Digit<1>::get(key)], 1u);
    } else {
      st_nt(x + start + j, dv[u] - mean);  // single-way: the mean itself comes back
    }
  }
}

// Grid: n_chunks workgroups.
template <int kMode, bool kAvg>
__global__ __launch_bounds__(kBig) void k_tk_aggregate(DevLayout lay, TkDev tk, int K,
                                                         double inv_k,
                                                         const uint64_t* __restrict__ sel,
                                                         const uint32_t* __restrict__ rank,
                                                         const float* __restrict__ vals,
                                                         float* __restrict__ avg,
                                                         float* __restrict__ es,
                                                         float* __restrict__ x) {
  __shared__ uint32_t h[kTkBins];
  const int64_t ci = blockIdx.x;
  const TkChunk c = tk.chunks[ci];
  const int64_t voff = tk.tens[c.l].voff;
  const uint32_t keep = (uint32_t)tk.tens[c.l].keep;
  if (kMode == 1) hist_clear<kTkBins>(h);
  const int nw = (c.count + 63) >> 6;
  bool bad = false;
  for (int w0 = wave_id() * kTkU; w0 < nw; w0 += (kBig / kWave) * kTkU) {
    if ((w0 + kTkU) * 64 <= c.count)
      tk_aggregate_words<kMode, kAvg, true>(lay, tk, K, inv_k, voff, keep, c.start, w0, nw, c.count,
                                            sel, rank, vals, avg, es, x, h, bad);
    else
      tk_aggregate_words<kMode, kAvg, false>(lay, tk, K, inv_k, voff, keep, c.start, w0, nw, c.count,
                                             sel, rank, vals, avg, es, x, h, bad);
  }
  if (kMode == 1) {
    if (__ballot(bad) != 0 && lane_id() == 0) atomicOr(lay.status, kStatusRange);
    hist_store<kTkBins>(h, chunk_hist(tk, lay.k_max, ci));
  }
}

// ------------------------------------------------------------------ host side
struct Launcher {
  const DevLayout& lay;
  const TkDev& tk;
  hipStream_t s;

  template <int kPass>
  hipError_t reduce_pick(int R, int row0) const {
    const LaunchEvents ev;
    if (tk.red_split > 1) {
      SAEF_LAUNCH((k_tk_sum<kPass>), dim3((unsigned)(R * lay.L * tk.red_split)), dim3(kBlock), 0,
                  s, lay, tk, row0);
      const hipError_t err = hipGetLastError();
      if (err != hipSuccess) return err;
    }
    SAEF_LAUNCH((k_tk_pick<kPass>), dim3((unsigned)(R * lay.L)), dim3(kBlock), 0, s, lay, tk,
                row0);
    return hipGetLastError();
  }

  // one histogram pass over R rows: 256-thread workgroups when there are
  // several rows, 1024-thread ones for a single row (the server)
  template <int kPass>
  hipError_t hist(int R, int row0, const float* data) const {
    const LaunchEvents ev;
    const dim3 grid((unsigned)(tk.n_chunks * R));
    if (R > 1)
      SAEF_LAUNCH((k_tk_hist<kPass, SAEF_TK_HIST_THREADS>), grid, dim3(SAEF_TK_HIST_THREADS), 0, s,
                  lay, tk, R, row0, data);
    else
      SAEF_LAUNCH((k_tk_hist<kPass, kBig>), grid, dim3(kBig), 0, s, lay, tk, R, row0, data);
    return hipGetLastError();
  }

  // passes 2 and 3, ties, emit of R rows of `data` (pass 1 already done)
  hipError_t select_and_emit(int R, int row0, float* data, uint64_t* sel, uint32_t* rank,
                             float* vals, float* x, const LaunchEvents& last) const {
    const LaunchEvents ev;
    hipError_t err = reduce_pick<1>(R, row0);
    if (err != hipSuccess) return err;
    if ((err = hist<2>(R, row0, data)) != hipSuccess) return err;
    if ((err = reduce_pick<2>(R, row0)) != hipSuccess) return err;
    if ((err = hist<3>(R, row0, data)) != hipSuccess) return err;
    if ((err = reduce_pick<3>(R, row0)) != hipSuccess) return err;
    SAEF_LAUNCH(k_tk_ties, dim3((unsigned)(R * lay.L)), dim3(kBig), 0, s, lay, tk, row0, data);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    const dim3 tiles((unsigned)(per_wave_grid(lay) * R));
    SAEF_LAUNCH(k_tk_emit1, tiles, dim3(kBlock), 0, s, lay, tk, R, row0, data, sel);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    SAEF_LAUNCH(k_tk_scan, dim3((unsigned)(R * lay.L)), dim3(kBlock), 0, s, lay, tk, row0);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    // the last kernel stamps the caller's stop event
    if (x != nullptr)
      hipExtLaunchKernelGGL((k_tk_emit2<true>), tiles, dim3(kBlock), 0, s, nullptr, last.stop, 0,
                            lay, tk, R, row0, data, sel, rank, vals, x);
    else
      hipExtLaunchKernelGGL((k_tk_emit2<false>), tiles, dim3(kBlock), 0, s, nullptr, last.stop, 0,
                            lay, tk, R, row0, data, sel, rank, vals, x);
    return hipGetLastError();
  }
};

}  // namespace

hipError_t launch_topk_compress(const DevLayout& lay, const TkDev& tk, int K, float lr, float mu,
                                const float* g, float* m, float* e, uint64_t* sel,
                                uint32_t* rank, float* vals, hipStream_t s,
                                const LaunchEvents& ev) {
  const dim3 grid((unsigned)(tk.n_chunks * K));
  // the first kernel stamps the start event, the last one the stop event
  if (m != nullptr)
    hipExtLaunchKernelGGL((k_tk_delta<true>), grid, dim3(kBlock), 0, s, ev.start, nullptr, 0, lay,
                          tk, K, lr, mu, g, m, e);
  else
    hipExtLaunchKernelGGL((k_tk_delta<false>), grid, dim3(kBlock), 0, s, ev.start, nullptr, 0,
                          lay, tk, K, lr, mu, g, m, e);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  return Launcher{lay, tk, s}.select_and_emit(K, 0, e, sel, rank, vals, nullptr, ev);
}

hipError_t launch_topk_aggregate(const DevLayout& lay, const TkDev& tk, int K, int mode,
                                 const uint64_t* sel, const uint32_t* rank, const float* vals,
                                 float* avg, float* e_srv, uint64_t* srv_sel, uint32_t* srv_rank,
                                 float* srv_vals, float* x, hipStream_t s,
                                 const LaunchEvents& ev) {
  const dim3 grid((unsigned)tk.n_chunks);
  const double ik = inv_pow2(K);
  hipEvent_t stop0 = mode == 1 ? nullptr : ev.stop;
#define SAEF_TKA(M, A)                                                                          \
  hipExtLaunchKernelGGL((k_tk_aggregate<M, A>), grid, dim3(kBig), 0, s, ev.start, stop0, 0, \
                        lay, tk, K, ik, sel, rank, vals, avg, e_srv, x)
  if (mode == 1) {
    if (avg != nullptr) SAEF_TKA(1, true); else SAEF_TKA(1, false);
  } else {
    if (avg != nullptr) SAEF_TKA(0, true); else SAEF_TKA(0, false);
  }
#undef SAEF_TKA
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess || mode != 1) return err;
  return Launcher{lay, tk, s}.select_and_emit(1, lay.k_max, e_srv, srv_sel, srv_rank, srv_vals,
                                              x, ev);
}

}  // namespace saef
