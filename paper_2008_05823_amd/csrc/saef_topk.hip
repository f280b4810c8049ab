// HIP kernels of the layer-wise Top-K compressor on gfx950 (CDNA4, wave64).
//
// C(v) keeps the k_l elements of largest |v| of each tensor (equal
// magnitudes: the lower index first) and zeroes the others.  The kept set of
// each (row, tensor) is found on the 31-bit key |v| (the bit pattern of a
// non-negative float orders like its value):
//   histogram  the pass that forms Delta (one workgroup per tile and row)
//              also counts the keys into a tile histogram (LDS atomics,
//              16-bit counts stored): 64 bins per binade over a window of
//              four binades placed around the (row, tensor)'s previous
//              threshold, one bin per binade for seven binades below it,
//              one for the keys further down and one above the window;
//   sum        tile histograms are added per group of 64 tiles (and groups
//              per super-group for very large tensors);
//   pick       a workgroup per (row, tensor) finds the bin b1 that holds the
//              k-th largest key and each group's first candidate slot;
//   offsets    each tile's first candidate slot (a scan inside its group);
//   gather     one wave per tile: elements above b1 are kept for sure
//              (their count to the tile's kept count); the elements of b1
//              (the candidates) go to the tile's slots as (key, index in the
//              tensor), in index order.  Taken from the tile's speculative
//              list (written by the Delta pass: the elements at or above a
//              bound just below the previous threshold) when its bound lies
//              at or below b1, else from one more read of Delta, which also
//              gives the selection words of the sure elements;
//   select     a workgroup per (row, tensor) finds, among the candidates only,
//              the threshold key tau and the last kept index iota of the
//              elements equal to tau (radix passes on the key bits below
//              b1's prefix, then on the index), and places the next call's
//              window around tau; the same workgroup then counts each
//              tile's kept elements (its definite ones, from the gather, and
//              its kept candidates) and turns the counts into each tile's
//              first rank;
//   emit       one wave per tile adds its kept candidates to its selection
//              words, then writes the rank words and the kept values in
//              index order, and sets the kept elements of the error to 0
//              (e = Delta - C(Delta) is Delta elsewhere); a tile the gather
//              took from its list is emitted from the list alone.
// All of it is integer counting, so the kept set does not depend on the
// launch geometry.
//
// The streaming passes (Delta, gather) run one short-lived workgroup or wave
// per 2048-element tile: on MI355X a 2-read/1-write stream reaches about
// 6.1 TB/s that way and about 5.1 TB/s when each workgroup walks 64Ki
// elements.
//
// The server runs the same steps on its one row (row k_max of the scratch)
// after k_tk_aggregate has formed Delta = e_srv + mean of the K messages.
#include "saef_device.h"
#include "saef_topk.h"

namespace saef {
namespace {

constexpr uint32_t kFiniteLimit = 0x7F800000u;  // keys >= this are Inf or NaN
constexpr int kTkU = 8;                         // words per wave per pass (Delta pass: one pass)
constexpr int kTileWords = kTkTileElems / 64;     // 32
constexpr int kBig = 1024;                      // threads of the per-(row, tensor) kernels
static_assert(kTileWords <= kWave, "one selection word of a tile per lane");
// Guarded loads without a branch: the load of p[ok ? j : 0] is always
// issued (p[0] must exist) and its value replaced by 0 when !ok.  A branch
// around each load makes the compiler wait for it before the next one.
__device__ __forceinline__ float ld_nt_or0(const float* p, int64_t j, bool ok) {
  const float v = __builtin_nontemporal_load(p + (ok ? j : 0));
  return ok ? v : 0.0f;
}
// Word 3 of a raw buffer descriptor on gfx9 parts (32-bit data format, no
// swizzle, no index stride).  A load through a raw buffer resource of n
// bytes returns 0 for a byte offset at or past n, without touching memory.
constexpr int kBufWord3 = 0x00020000;

__device__ __forceinline__ uint32_t key_of(float v) { return __float_as_uint(v) & 0x7FFFFFFFu; }

// Pass-1 bin of a key for the window [win, win + 4 binades) (win a multiple
// of 2^23, its binade wb): below it, bin kTkLo - j for binade wb - j (j <
// kTkLo) and bin 0 for all lower keys; kTkLo .. kTkLo + kTkWin - 1 inside it
// (key bits 22..17 within each binade); kTkLo + kTkWin above it.  Bins order
// like the keys.
__device__ __forceinline__ uint32_t hist_bin(uint32_t key, uint32_t win) {
  const int32_t s = (int32_t)(key - win);  // keys and win are below 2^31
  const uint32_t d = (uint32_t)s >> kTkSubShift;
  if (d < (uint32_t)kTkWin) return (uint32_t)kTkLo + d;
  if (s >= 0) return (uint32_t)(kTkLo + kTkWin);
  const int32_t j = s >> 23;  // -(binades below the window's first): <= -1 (win is 2^23-aligned)
  return (uint32_t)max(j + kTkLo, 0);
}

// The window for the next call: the binade of tau is the third of four.
__device__ __forceinline__ uint32_t window_for(uint32_t tau) {
  const uint32_t b = tau >> 23;
  return (b >= 2u ? b - 2u : 0u) << 23;
}

__device__ __forceinline__ uint16_t* tile_hist(const TkDev& tk, const DevLayout& lay, int row,
                                               int64_t ti) {
  return tk.thist + ((int64_t)row * lay.n_tiles + ti) * kTkHistPad;
}

// Stores an LDS histogram of kTkHistPad bins as 16-bit counts, two per store,
// with `spec` (the tile's speculative list count) in slot kTkSpecSlot.
__device__ __forceinline__ void store_hist16(const uint32_t* h, uint16_t* out, uint32_t spec) {
  for (int i = threadIdx.x; i < kTkHistPad / 2; i += blockDim.x)
    reinterpret_cast<uint32_t*>(out)[i] =
        2 * i == kTkSpecSlot ? spec : (h[2 * i] & 0xFFFFu) | (h[2 * i + 1] << 16);
}

// Lower key bound of the speculative lists of a (row, tensor): the previous
// threshold key minus the margin; 2^31 (no element) before the first
// threshold or when the tensor keeps no lists.
__device__ __forceinline__ uint32_t spec_floor(const TkSel& st) {
  if (st.tau == 0u || st.lists == 0u) return 0x80000000u;
  return st.tau > kTkSpecMargin ? st.tau - kTkSpecMargin : 0u;
}

// ------------------------------------------------------------------ pass 1 (workers)
// kTkU words of one worker's tile: m <- fma(mu, m, g) with kMom, Delta =
// fma(lr, m or g, e), Delta stored into e, its key counted.
template <bool kMom, bool kPend, bool kFull>
__device__ __forceinline__ void delta_words(int w0, int nw, int count, float lr, float mu,
                                            const float* __restrict__ gk, float* __restrict__ mk,
                                            float* __restrict__ ek,
                                            const uint64_t* __restrict__ pk, uint32_t win,
                                            uint32_t lo, uint32_t* h, uint32_t (&bits)[kTkU],
                                            u64 (&lm)[kTkU], bool& bad) {
  const int lane = lane_id();
  float gv[kTkU], ev[kTkU], mv[kTkU];
  u64 pw[kTkU];
#pragma unroll
  for (int u = 0; u < kTkU; ++u) {
    const int j = (w0 + u) * 64 + lane;
    const bool ok = kFull || ((w0 + u < nw) && j < count);
    gv[u] = ld_nt_or0(gk, j, ok);
    ev[u] = ld_nt_or0(ek, j, ok);
    mv[u] = kMom ? ld_nt_or0(mk, j, ok) : 0.0f;
    pw[u] = (kPend && (kFull || w0 + u < nw)) ? pk[w0 + u] : 0ull;
  }
  // the previous call left its kept elements pending: they are 0
#pragma unroll
  for (int u = 0; u < kTkU; ++u)
    if (kPend) ev[u] = sel_by_bit(pw[u], 0.0f, ev[u]);
#pragma unroll
  for (int u = 0; u < kTkU; ++u) {
    const int j = (w0 + u) * 64 + lane;
    const bool ok = kFull || ((w0 + u < nw) && j < count);
    float step = gv[u];
    if (kMom) {
      step = __builtin_fmaf(mu, mv[u], gv[u]);  // m^(k)_{t+1} = mu m^(k)_t + grad
      if (ok) st_nt(mk + j, step);
    }
    const float p = __builtin_fmaf(lr, step, ev[u]);  // Delta^(k) = e^(k) + lr m^(k)_{t+1}
    const uint32_t key = key_of(p);
    bits[u] = __float_as_uint(p);
    lm[u] = __ballot(ok && key >= lo);
    if (!ok) continue;
    st_nt(ek + j, p);
    bad |= key >= kFiniteLimit;
    atomicAdd(&h[hist_bin(key, win)], 1u);
  }
}

// Grid: (p.t1 - p.t0) * R workgroups; workgroup b handles row row0 + b % R of
// tile p.t0 + b / R.
// Each wave takes kTkU words of the tile (one pass); the tile's speculative
// list is written in index order (wave by wave) when it fits.  kPend: e
// holds the previous call's Delta with its kept elements (selection words
// psel) still to be set to 0; they are read as 0.
template <bool kMom, bool kPend>
__global__ __launch_bounds__(kBlock) void k_tk_delta(DevLayout lay, TkDev tk, TkPart p, int R,
                                                     int row0,
                                                     float lr, float mu,
                                                     const float* __restrict__ g,
                                                     float* __restrict__ m,
                                                     float* __restrict__ e,
                                                     const uint64_t* __restrict__ psel) {
  static_assert(kWaves * kTkU == kTileWords, "one pass of the four waves covers a tile");
  __shared__ uint32_t h[kTkHistPad];
  __shared__ uint32_t s_cnt[kWaves];
  const int k = row0 + (int)(blockIdx.x % (unsigned)R);
  const int64_t ti = p.t0 + (int64_t)(blockIdx.x / (unsigned)R);
  const Tile tile = lay.tiles[ti];
  const TkSel* st = tk.sel + (int64_t)k * lay.L + tile.l;
  const uint32_t win = st->win;
  const uint32_t lo = spec_floor(*st);
  for (int i = threadIdx.x; i < kTkHistPad; i += kBlock) h[i] = 0;
  __syncthreads();
  const int64_t row = (int64_t)k * lay.d_pad + tile.start;
  const float* gk = g + row;
  float* mk = kMom ? m + row : nullptr;
  float* ek = e + row;
  const int nw = (tile.count + 63) >> 6;
  const int wave = wave_id();
  const int w0 = wave * kTkU;
  bool bad = false;
  uint32_t bits[kTkU];  // Delta's bit patterns
  u64 lm[kTkU];
#pragma unroll
  for (int u = 0; u < kTkU; ++u) lm[u] = 0ull;
  const uint64_t* pk = kPend ? psel + (int64_t)k * (lay.d_pad >> 6) + (tile.start >> 6) : nullptr;
  if (w0 < nw) {
    if ((w0 + kTkU) * 64 <= tile.count)
      delta_words<kMom, kPend, true>(w0, nw, tile.count, lr, mu, gk, mk, ek, pk, win, lo, h, bits,
                                     lm, bad);
    else
      delta_words<kMom, kPend, false>(w0, nw, tile.count, lr, mu, gk, mk, ek, pk, win, lo, h,
                                      bits, lm, bad);
  }
  if (__ballot(bad) != 0 && lane_id() == 0) atomicOr(lay.status, kStatusRange);
  uint32_t mine = 0;
#pragma unroll
  for (int u = 0; u < kTkU; ++u) mine += (uint32_t)__popcll(lm[u]);
  if (lane_id() == 0) s_cnt[wave] = mine;
  __syncthreads();
  uint32_t before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    before += w < wave ? s_cnt[w] : 0u;
    total += s_cnt[w];
  }
  // no list (kTkSpecNone) before the first threshold, for a tensor without
  // lists, or when the tile has more than kTkSpecCap such elements
  const bool fits = lo != 0x80000000u && total <= (uint32_t)kTkSpecCap;
  store_hist16(h, tile_hist(tk, lay, k, ti), fits ? total : kTkSpecNone);
  if (fits && mine != 0u) {
    u64* out = tk.spec + ((int64_t)k * lay.n_tiles + ti) * kTkSpecCap;
    const int lane = lane_id();
#pragma unroll
    for (int u = 0; u < kTkU; ++u) {
      const uint32_t pos =
          before + __builtin_amdgcn_mbcnt_hi((uint32_t)(lm[u] >> 32),
                                             __builtin_amdgcn_mbcnt_lo((uint32_t)lm[u], 0u));
      if ((lm[u] >> lane) & 1ull)  // pos < total <= kTkSpecCap
        out[pos] = (u64)bits[u] | ((u64)((w0 + u) * 64 + lane) << 32);
      before += (uint32_t)__popcll(lm[u]);
    }
  }
}

// ------------------------------------------------------------------ sums
// Grid: R * n workgroups, n the part's groups (kSuper: super-groups).
// Workgroup b adds the tile histograms of the part's group b % n (or the
// group sums of its super-group b % n) of row row0 + b / n.
template <bool kSuper>
__global__ __launch_bounds__(kBlock) void k_tk_sum(DevLayout lay, TkDev tk, TkPart p, int row0) {
  const int64_t n = kSuper ? p.s1 - p.s0 : p.g1 - p.g0;
  const int64_t gi = (kSuper ? p.s0 : p.g0) + (int64_t)(blockIdx.x % n);
  const int row = row0 + (int)(blockIdx.x / n);
  const TkGroup gr = (kSuper ? tk.sgroups : tk.groups)[gi];
  uint32_t* dst = (kSuper ? tk.sghist + ((int64_t)row * tk.n_sgroups + gi) * kTkHistPad
                          : tk.ghist + ((int64_t)row * tk.n_groups + gi) * kTkHistPad);
  for (int b = threadIdx.x; b < kTkHistPad; b += kBlock) {
    uint32_t acc = 0;
    if (kSuper) {
      const uint32_t* src = tk.ghist + ((int64_t)row * tk.n_groups + gr.first) * kTkHistPad + b;
#pragma unroll 8
      for (int i = 0; i < gr.n; ++i) acc += src[(int64_t)i * kTkHistPad];
    } else {
      const uint16_t* src = tile_hist(tk, lay, row, gr.first) + b;
#pragma unroll 8
      for (int i = 0; i < gr.n; ++i) acc += src[(int64_t)i * kTkHistPad];
    }
    dst[b] = acc;
  }
}

// ------------------------------------------------------------------ block helpers
// Exclusive prefix sum of v over the workgroup (threads in order); *total
// receives the sum.  s must hold blockDim.x / 64 entries.
__device__ uint32_t block_excl_scan(uint32_t v, uint32_t* s, uint32_t* total) {
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int nwaves = blockDim.x / kWave;
  uint32_t x = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == kWave - 1) s[wave] = x;
  __syncthreads();
  uint32_t before = 0, all = 0;
  for (int i = 0; i < nwaves; ++i) {
    if (i < wave) before += s[i];
    all += s[i];
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

// Over the LDS histogram h[0..nb), the bin that holds the need-th element
// counted from the top (kTop) or from the bottom (1 <= need <= total).
// Returns to every thread the bin, how many to take inside it and its count.
template <bool kTop>
__device__ void find_bin(const uint32_t* h, int nb, int64_t need, uint32_t* s_scan,
                         uint32_t* s_res, uint32_t& bin, int64_t& left, uint32_t& count) {
  const int per = (nb + (int)blockDim.x - 1) / (int)blockDim.x;
  if (threadIdx.x == 0) {  // defined result even if need exceeded the total
    s_res[0] = 0;
    s_res[1] = 1;
    s_res[2] = 0;
  }
  // thread t owns positions [t per, (t+1) per) counted in the search direction
  uint32_t tot = 0;
  for (int j = 0; j < per; ++j) {
    const int q = threadIdx.x * per + j;
    if (q < nb) tot += h[kTop ? nb - 1 - q : q];
  }
  uint32_t all;
  const uint32_t before = block_excl_scan(tot, s_scan, &all);
  if ((int64_t)before < need && need <= (int64_t)before + tot) {
    int64_t run = before;
    for (int j = 0; j < per; ++j) {
      const int q = threadIdx.x * per + j;
      if (q >= nb) break;
      const int b = kTop ? nb - 1 - q : q;
      if (run + h[b] >= need) {
        s_res[0] = (uint32_t)b;
        s_res[1] = (uint32_t)(need - run);
        s_res[2] = h[b];
        break;
      }
      run += h[b];
    }
  }
  __syncthreads();
  bin = s_res[0];
  left = s_res[1];
  count = s_res[2];
  __syncthreads();
}

// ------------------------------------------------------------------ pick
// Grid: R * nl workgroups, nl the part's tensors (workgroup b: tensor
// p.l0 + b % nl of row row0 + b / nl).  Adds the tensor's group sums (or super-group
// sums), finds the bin b1 that holds the k-th largest key and how many to
// take from it, and gives each group of the tensor its first candidate slot:
// the elements of b1 go to the (row, tensor)'s candidate area (one slot per
// element of the tensor at most) in tile order.
__global__ __launch_bounds__(kBlock) void k_tk_pick(DevLayout lay, TkDev tk, TkPart p, int row0) {
  __shared__ uint32_t s_scan[kWaves];
  __shared__ uint32_t s_res[3];
  __shared__ uint32_t h[kTkHistPad];
  const int nl = p.l1 - p.l0;
  const int l = p.l0 + (int)(blockIdx.x % (unsigned)nl);
  const int r = (int)(blockIdx.x / (unsigned)nl);
  const int row = row0 + r;
  const TkTensor t = tk.tens[l];
  const bool super = t.nsgroups > 0;
  const uint32_t* src = super
      ? tk.sghist + ((int64_t)row * tk.n_sgroups + t.first_sgroup) * kTkHistPad
      : tk.ghist + ((int64_t)row * tk.n_groups + t.first_group) * kTkHistPad;
  const int ns = super ? t.nsgroups : t.ngroups;
  for (int b = threadIdx.x; b < kTkHistPad; b += kBlock) {
    uint32_t cnt = 0;
    for (int i = 0; i < ns; ++i) cnt += src[(int64_t)i * kTkHistPad + b];
    h[b] = cnt;
  }
  __syncthreads();
  uint32_t b1, n1;
  int64_t left;
  find_bin<true>(h, kTkHist, t.keep, s_scan, s_res, b1, left, n1);
  // first candidate slot of each group, in group order
  uint32_t carry = 0;
  const uint32_t* gh = tk.ghist + ((int64_t)row * tk.n_groups + t.first_group) * kTkHistPad + b1;
  for (int g0 = 0; g0 < t.ngroups; g0 += kBlock) {
    const int gi = g0 + threadIdx.x;
    const uint32_t v = gi < t.ngroups ? gh[(int64_t)gi * kTkHistPad] : 0u;
    uint32_t all;
    const uint32_t before = block_excl_scan(v, s_scan, &all);
    if (gi < t.ngroups) tk.goff[(int64_t)row * tk.n_groups + t.first_group + gi] = carry + before;
    carry += all;
  }
  if (threadIdx.x == 0) {
    TkSel* st = tk.sel + (int64_t)row * lay.L + l;
    st->bin = b1;
    st->need = left;
    st->cand = n1;  // the elements of b1 (the sum of the tile counts)
  }
}

// Grid: R * n workgroups of one wave, n the part's groups: the first
// candidate slot of each tile of the part's group b % n in row row0 + b / n
// (the group's slot plus the b1 counts of the group's earlier tiles).
__global__ __launch_bounds__(kWave) void k_tk_offsets(DevLayout lay, TkDev tk, TkPart p,
                                                      int row0) {
  static_assert(kTkGroup == kWave, "one tile of a group per lane");
  const int64_t n = p.g1 - p.g0;
  const int64_t gi = p.g0 + (int64_t)(blockIdx.x % n);
  const int row = row0 + (int)(blockIdx.x / n);
  const TkGroup gr = tk.groups[gi];
  const uint32_t b1 = tk.sel[(int64_t)row * lay.L + gr.l].bin;
  const int lane = lane_id();
  const uint32_t c = lane < gr.n ? tile_hist(tk, lay, row, gr.first + lane)[b1] : 0u;
  uint32_t x = c;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane < gr.n)
    tk.cand_off[(int64_t)row * lay.n_tiles + gr.first + lane] =
        tk.goff[(int64_t)row * tk.n_groups + gi] + x - c;
}

// ------------------------------------------------------------------ gather
// The smallest key of bin b for the window at win (hist_bin's layout; a
// below bin for a binade under 0 is empty and starts at 0); kTkHist (one
// past the last bin) gives 2^31, above every key.
__device__ __forceinline__ uint32_t bin_floor(uint32_t b, uint32_t win) {
  const int64_t wb = win >> 23;
  if (b == 0u) return 0u;
  if (b >= (uint32_t)kTkHist) return 0x80000000u;
  int64_t f;
  if (b < (uint32_t)kTkLo) {
    const int64_t kb = wb - (kTkLo - (int64_t)b);  // the bin's binade
    f = kb > 0 ? kb << 23 : 0;
  } else if (b < (uint32_t)(kTkLo + kTkWin)) {
    f = (int64_t)win + ((int64_t)(b - kTkLo) << kTkSubShift);
  } else {
    f = (wb + 4) << 23;  // the bin above the window
  }
  return f < 0x80000000ll ? (uint32_t)f : 0x80000000u;
}

// The key bits bin b fixes: keys of the bin are those with key >> open ==
// prefix (open = 17 inside the window, 23 for a one-binade bin, 31 for the
// lowest bin and the one above the window).
__device__ __forceinline__ void bin_prefix(uint32_t b, uint32_t win, uint32_t& prefix, int& open) {
  const uint32_t wb = win >> 23;
  if (b >= (uint32_t)kTkLo && b < (uint32_t)(kTkLo + kTkWin)) {
    prefix = (win >> kTkSubShift) + (b - kTkLo);
    open = kTkSubShift;
  } else if (b >= 1u && b < (uint32_t)kTkLo && wb >= (uint32_t)kTkLo - b) {
    prefix = wb - ((uint32_t)kTkLo - b);
    open = 23;
  } else {
    prefix = 0u;
    open = 31;
  }
}

// The gather's classification of a tile's 32 words (kFull: all 2048
// elements exist): selection words (lane u gets word u) and candidates to
// their slots in index order.
template <bool kFull>
__device__ __forceinline__ void gather_words(const float (&v)[kTileWords], int count, uint32_t lo,
                                             uint32_t up, int64_t rel0, uint32_t nslots,
                                             u64* __restrict__ slots, u64& myw, uint32_t& base) {
  const int lane = lane_id();
#pragma unroll
  for (int u = 0; u < kTileWords; ++u) {
    const int j = u * 64 + lane;
    const bool ok = kFull || j < count;
    const uint32_t key = key_of(v[u]);
    const u64 word = __ballot(ok && key >= up);
    if (lane == u) myw = word;
    const u64 cm = __ballot(ok && key - lo < up - lo);  // lo <= key < up
    if (cm != 0ull) {  // wave-uniform: most words have no candidate
      const uint32_t pos = base + __builtin_amdgcn_mbcnt_hi((uint32_t)(cm >> 32),
                                                            __builtin_amdgcn_mbcnt_lo((uint32_t)cm, 0u));
      if (((cm >> lane) & 1ull) && pos < nslots)  // pos < nslots always holds
        slots[pos] = (u64)key | ((u64)(rel0 + j) << 32);
      base += (uint32_t)__popcll(cm);
    }
  }
}

// The gather from a tile's speculative list (n <= 64 kNC entries: Delta's
// bits | index in the tile << 32, index order), if the list's bound lies at
// or below b1 (then every element with a key >= lo is in it): the count of
// the elements above b1 (per lane, to be added) and the elements of b1 to the
// candidate slots in index order; returns false, having written nothing,
// otherwise.  The list loads are issued before the selection state is waited
// for.  The selection words are left to the emit, which reads the list too.
template <int kNC>
__device__ __forceinline__ bool gather_list(const u64* __restrict__ ent, uint32_t n,
                                            const TkSel* st, const TensorInfo* ten,
                                            const uint32_t* co, int64_t row_cand, int64_t start,
                                            int count, const TkDev& tk, uint32_t& ndef) {
  const int lane = lane_id();
  u64 e[kNC > 0 ? kNC : 1];
#pragma unroll
  for (int c = 0; c < kNC; ++c) {
    const uint32_t i = (uint32_t)(c * kWave + lane);
    e[c] = ent[i < n ? i : 0u];
  }
  const uint32_t b1 = st->bin, win = st->win;
  // bin b1 holds the keys [lo, up): above it kept for sure, inside it candidates
  const uint32_t lo = bin_floor(b1, win), up = bin_floor(b1 + 1u, win);
  if (spec_floor(*st) > lo) return false;
  const int64_t off = ten->off;
  const int64_t rel0 = start - off;  // the tile's first element, index in the tensor
  u64* slots = tk.cand + row_cand + off + *co;
  uint32_t base = 0;  // candidates in the earlier entries
#pragma unroll
  for (int c = 0; c < kNC; ++c) {
    const bool ok = (uint32_t)(c * kWave + lane) < n;
    const uint32_t key = (uint32_t)e[c] & 0x7FFFFFFFu, idx = (uint32_t)(e[c] >> 32);
    const u64 sure = __ballot(ok && key >= up);
    ndef += lane == 0 ? (uint32_t)__popcll(sure) : 0u;
    const u64 cm = __ballot(ok && key - lo < up - lo);  // lo <= key < up
    if (cm != 0ull) {
      const uint32_t pos = base + __builtin_amdgcn_mbcnt_hi((uint32_t)(cm >> 32),
                                                            __builtin_amdgcn_mbcnt_lo((uint32_t)cm, 0u));
      // the tile's slots follow the b1 elements of the earlier tiles of the
      // tensor, so pos < count keeps the store inside the tensor's area
      if (((cm >> lane) & 1ull) && pos < (uint32_t)count)
        slots[pos] = (u64)key | ((u64)(rel0 + idx) << 32);
      base += (uint32_t)__popcll(cm);
    }
  }
  return true;
}

// Grid: ceil((p.t1 - p.t0) / 4) * R workgroups; wave w of workgroup b owns
// tile p.t0 + 4 (b / R) + w of row b % R.  The count of the elements above b1 (kept for
// sure) and the elements of b1 to the tile's candidate slots as key | (index
// in the tensor) << 32, in index order: from the tile's speculative list when
// `spec` is set, the list fits and its bound lies at or below b1 (slot
// kTkSpecSlot + 1 of the tile histogram then says so to the emit), otherwise
// from one read of the tile's Delta (all 32 words at once), which also gives
// the selection words of the elements kept for sure.  At most 64 VGPRs: 8
// waves per SIMD (the kernel is bound by the latency of its dependent loads).
// Without lists (kSpec false) every tile takes the Delta read, with its 32
// loads in flight at once (85 VGPRs: k_tk_gather_full).
template <bool kSpec>
__device__ __forceinline__ void gather_tile(const DevLayout& lay, const TkDev& tk,
                                            const TkPart& p, int R, int row0,
                                            const float* __restrict__ data,
                                            uint64_t* __restrict__ sel) {
  constexpr int spec = kSpec ? 1 : 0;
  const int r = (int)(blockIdx.x % (unsigned)R);
  const int64_t ti = p.t0 + (int64_t)(blockIdx.x / (unsigned)R) * kWaves + wave_id();
  if (ti >= p.t1) return;
  const int row = row0 + r;
  uint16_t* th = tile_hist(tk, lay, row, ti);
  // the list count and the flag slot in one 32-bit word: a scalar load issued
  // together with the tile's (a 16-bit load would be a vector one, waited for
  // before anything else)
  const uint32_t sp = spec ? *reinterpret_cast<const uint32_t*>(th + kTkSpecSlot) : kTkSpecNone;
  const Tile tile = lay.tiles[ti];
  const uint32_t n_spec = sp & 0xFFFFu;
  const TkSel* st = tk.sel + (int64_t)row * lay.L + tile.l;
  const TensorInfo* ten = lay.tensors + tile.l;
  const uint32_t* co = tk.cand_off + (int64_t)row * lay.n_tiles + ti;
  const int64_t row_cand = (int64_t)row * lay.d_pad;
  const int lane = lane_id();
  uint32_t ndef = 0;  // kept for sure (lane 0 holds the list path's count)
  bool listed = false;
  if (n_spec != kTkSpecNone) {
    static_assert(kTkSpecCap == 8 * kWave, "lists of up to 8 loads per lane");
    const u64* ent = tk.spec + ((int64_t)row * lay.n_tiles + ti) * kTkSpecCap;
#define SAEF_GL(NC) \
  listed = gather_list<NC>(ent, n_spec, st, ten, co, row_cand, tile.start, tile.count, tk, ndef)
    switch ((n_spec + kWave - 1) / kWave) {
      case 0: SAEF_GL(0); break;
      case 1: SAEF_GL(1); break;
      case 2: SAEF_GL(2); break;
      case 3: SAEF_GL(3); break;
      case 4: SAEF_GL(4); break;
      case 5: SAEF_GL(5); break;
      case 6: SAEF_GL(6); break;
      case 7: SAEF_GL(7); break;
      default: SAEF_GL(8); break;
    }
#undef SAEF_GL
  }
  if (!listed) {
    const uint32_t b1 = st->bin, win = st->win;
    const uint32_t lo = bin_floor(b1, win), up = bin_floor(b1 + 1u, win);
    const int64_t rel0 = tile.start - ten->off;
    u64* slots = tk.cand + row_cand + ten->off + *co;
    const uint32_t nslots = th[b1];  // elements of b1 in the tile
    const float* dr = data + (int64_t)r * lay.d_pad + tile.start;
    float v[kTileWords];
#pragma unroll
    for (int u = 0; u < kTileWords; ++u) {
      const int j = u * 64 + lane;
      v[u] = ld_nt_or0(dr, j, j < tile.count);
    }
    u64 myw = 0;        // lane u < nw: selection word u
    uint32_t base = 0;  // candidates in the earlier words
    if (tile.count == kTkTileElems)
      gather_words<true>(v, tile.count, lo, up, rel0, nslots, slots, myw, base);
    else
      gather_words<false>(v, tile.count, lo, up, rel0, nslots, slots, myw, base);
    const int nw = (tile.count + 63) >> 6;
    uint64_t* sr = sel + (int64_t)r * (lay.d_pad >> 6) + (tile.start >> 6);
    if (lane < nw) sr[lane] = myw;
    ndef = (uint32_t)__popcll(myw);
  }
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) ndef += __shfl_xor(ndef, off);
  if (lane == 0) {
    tk.tile_cnt[(int64_t)row * lay.n_tiles + ti] = ndef;  // kept for sure
    if (spec) th[kTkSpecSlot + 1] = listed ? 1 : 0;
  }
}

__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(8, 8)))
void k_tk_gather_spec(DevLayout lay, TkDev tk, TkPart p, int R, int row0,
                      const float* __restrict__ data, uint64_t* __restrict__ sel) {
  gather_tile<true>(lay, tk, p, R, row0, data, sel);
}

__global__ __launch_bounds__(kBlock)
void k_tk_gather_full(DevLayout lay, TkDev tk, TkPart p, int R, int row0,
                      const float* __restrict__ data, uint64_t* __restrict__ sel) {
  gather_tile<false>(lay, tk, p, R, row0, data, sel);
}

// ------------------------------------------------------------------ select
// One radix pass over the candidates: histogram (LDS) of digit(e) of those
// with match(e).  Each thread has kIlp candidate loads in flight.
template <typename Match, typename Dig>
__device__ void cand_hist(uint32_t* h, int nb, const u64* __restrict__ cand, int64_t C,
                          Match match, Dig digit) {
  constexpr int kIlp = 8;
  for (int i = threadIdx.x; i < nb; i += blockDim.x) h[i] = 0;
  __syncthreads();
  const int64_t nt = blockDim.x;
  for (int64_t i0 = threadIdx.x; i0 < C; i0 += nt * kIlp) {
    u64 e[kIlp];
#pragma unroll
    for (int u = 0; u < kIlp; ++u) {
      const int64_t i = i0 + u * nt;
      e[u] = cand[i < C ? i : 0];  // C > 0 here
    }
#pragma unroll
    for (int u = 0; u < kIlp; ++u)
      if (i0 + u * nt < C && match(e[u])) atomicAdd(&h[digit(e[u])], 1u);
  }
  __syncthreads();
}

// Grid: R * nl workgroups of kBig threads (as k_tk_pick).  Among the candidates of (row,
// tensor) (the elements of bin b1), takes the `need` largest keys, equal
// keys by lower index: radix passes of up to 11 bits over the key bits that
// b1 leaves open (bits 16..0 inside the window, 22..0 for a one-binade bin,
// all 31 for the lowest bin and the one above) give the threshold key tau and how many of the elements
// equal to tau are kept; if not all, passes on the index in the tensor
// (bits 27..17, 16..6, 5..0) give the last kept index iota.  The next
// call's window is placed around tau.  Then each tile's kept count and first
// rank (tile_ranks).
__device__ void tile_ranks(const DevLayout& lay, const TkDev& tk, int row, int l, int64_t C,
                           const TkSel& st, uint32_t* s_cnt, uint32_t* s_scan);
__global__ __launch_bounds__(kBig) void k_tk_select(DevLayout lay, TkDev tk, TkPart p,
                                                     int row0) {
  __shared__ uint32_t h[kTkBins];
  __shared__ uint32_t s_scan[kBig / kWave];
  __shared__ uint32_t s_res[3];
  const int nl = p.l1 - p.l0;
  const int l = p.l0 + (int)(blockIdx.x % (unsigned)nl);
  const int r = (int)(blockIdx.x / (unsigned)nl);
  const int row = row0 + r;
  TkSel* st = tk.sel + (int64_t)row * lay.L + l;
  const u64* cand = tk.cand + (int64_t)row * lay.d_pad + lay.tensors[l].off;
  const int64_t C = st->cand;
  const uint32_t b1 = st->bin, win = st->win;
  int64_t need = st->need;
  uint32_t prefix;  // key >> open of every candidate
  int open;
  bin_prefix(b1, win, prefix, open);
  uint32_t bin = 0, cnt = 0;
  int64_t left = need;
  while (open > 0) {
    const int d = open > 11 ? 11 : open;
    const int sh = open - d;
    const uint32_t mask = (1u << d) - 1u;
    cand_hist(h, 1 << d, cand, C, [prefix, open](u64 e) { return ((uint32_t)e >> open) == prefix; },
              [sh, mask](u64 e) { return ((uint32_t)e >> sh) & mask; });
    find_bin<true>(h, 1 << d, need, s_scan, s_res, bin, left, cnt);
    prefix = (prefix << d) | bin;
    open = sh;
    need = left;
  }
  const uint32_t tau = prefix;
  int64_t iota = INT64_MAX;  // every element equal to tau is kept
  if (left < (int64_t)cnt) {
    // the left-th smallest index among the elements equal to tau
    need = left;
    cand_hist(h, kTkBins, cand, C, [tau](u64 e) { return (uint32_t)e == tau; },
              [](u64 e) { return (uint32_t)(e >> 49) & 2047u; });
    find_bin<false>(h, kTkBins, need, s_scan, s_res, bin, left, cnt);
    const uint32_t q1 = bin;
    need = left;
    cand_hist(h, kTkBins, cand, C,
              [tau, q1](u64 e) { return (uint32_t)e == tau && (uint32_t)(e >> 49) == q1; },
              [](u64 e) { return (uint32_t)(e >> 38) & 2047u; });
    find_bin<false>(h, kTkBins, need, s_scan, s_res, bin, left, cnt);
    const uint32_t q2 = (q1 << 11) | bin;
    need = left;
    cand_hist(h, 64, cand, C,
              [tau, q2](u64 e) { return (uint32_t)e == tau && (uint32_t)(e >> 38) == q2; },
              [](u64 e) { return (uint32_t)(e >> 32) & 63u; });
    find_bin<false>(h, 64, need, s_scan, s_res, bin, left, cnt);
    iota = ((int64_t)q2 << 6) | bin;
  }
  if (threadIdx.x == 0) {
    st->tau = tau;
    st->iota = iota;
    st->win = window_for(tau);
  }
  // every thread holds tau and iota; h (free once the last find_bin is done)
  // holds the per-tile counts
  static_assert(kTkBins >= kBig, "a count per thread of the workgroup");
  __syncthreads();
  TkSel kept{};
  kept.tau = tau;
  kept.iota = iota;
  tile_ranks(lay, tk, row, l, C, kept, h, s_scan);
}

// ------------------------------------------------------------------ emit
// A tile's candidates: slots [first, first + n) of its (row, tensor)'s
// candidate area (the next tile's first slot, or the candidate total after
// the tensor's last tile).
struct TileCands {
  uint32_t first, n;
};
__device__ __forceinline__ TileCands tile_cands(const DevLayout& lay, const TkDev& tk, int row,
                                                int64_t ti, const TensorInfo& ten, int64_t C) {
  const uint32_t* co = tk.cand_off + (int64_t)row * lay.n_tiles;
  const uint32_t first = co[ti];
  const uint32_t end = ti + 1 < ten.first_tile + ten.ntiles ? co[ti + 1] : (uint32_t)C;
  return TileCands{first, end - first};
}

__device__ __forceinline__ bool cand_kept(u64 e, const TkSel& st) {
  const uint32_t key = (uint32_t)e;
  const int64_t idx = (int64_t)(e >> 32);
  return key > st.tau || (key == st.tau && idx <= st.iota);
}

// Each tile's kept count (the gather's count of definite elements plus its
// kept candidates), then the exclusive prefix over the tensor's tiles in
// tile order, in place, for (row, tensor l) with threshold st.tau / st.iota
// and C candidates.  The candidates of a block of blockDim tiles are
// contiguous: the whole workgroup reads them and counts the kept ones per
// tile in s_cnt (blockDim entries of LDS).
__device__ void tile_ranks(const DevLayout& lay, const TkDev& tk, int row, int l, int64_t C,
                           const TkSel& st, uint32_t* s_cnt, uint32_t* s_scan) {
  constexpr int kIlp = 4;
  const int nt = (int)blockDim.x;
  const TensorInfo ten = lay.tensors[l];
  const u64* cand = tk.cand + (int64_t)row * lay.d_pad + ten.off;
  const uint32_t* co = tk.cand_off + (int64_t)row * lay.n_tiles + ten.first_tile;
  uint32_t* cnt = tk.tile_cnt + (int64_t)row * lay.n_tiles + ten.first_tile;
  uint32_t carry = 0;
  for (int b = 0; b < ten.ntiles; b += nt) {
    s_cnt[threadIdx.x] = 0;
    __syncthreads();
    const uint32_t lo = co[b];
    const uint32_t hi = b + nt < ten.ntiles ? co[b + nt] : (uint32_t)C;
    for (uint32_t c0 = lo + threadIdx.x; c0 < hi; c0 += (uint32_t)(nt * kIlp)) {
      u64 e[kIlp];
#pragma unroll
      for (int u = 0; u < kIlp; ++u) {
        const uint32_t c = c0 + (uint32_t)(u * nt);
        e[u] = cand[c < hi ? c : lo];  // lo < hi here
      }
#pragma unroll
      for (int u = 0; u < kIlp; ++u) {
        const int64_t t = (int64_t)(e[u] >> 32) / kTkTileElems - b;  // tile of the block
        if (c0 + (uint32_t)(u * nt) < hi && cand_kept(e[u], st) && t >= 0 && t < nt)
          atomicAdd(&s_cnt[t], 1u);
      }
    }
    __syncthreads();
    const int i = b + threadIdx.x;
    const uint32_t v = i < ten.ntiles ? cnt[i] + s_cnt[threadIdx.x] : 0u;
    uint32_t all;
    const uint32_t before = block_excl_scan(v, s_scan, &all);  // ends with a barrier
    if (i < ten.ntiles) cnt[i] = carry + before;
    carry += all;
  }
}

// The position of the r-th set bit of w (r counted from 0, r < popcount(w)):
// the 32-bit half that holds it, then five halving steps.
__device__ __forceinline__ int nth_set_bit(u64 w, uint32_t r) {
  uint32_t x = (uint32_t)w;
  int pos = 0;
  const uint32_t c_lo = (uint32_t)__popc(x);
  if (r >= c_lo) {
    r -= c_lo;
    x = (uint32_t)(w >> 32);
    pos = 32;
  }
#pragma unroll
  for (int s = 16; s >= 1; s >>= 1) {
    const uint32_t c = (uint32_t)__popc(x & ((1u << s) - 1u));
    if (r >= c) {
      r -= c;
      x >>= s;
      pos += s;
    }
  }
  return pos;
}

// The emit of a tile that the gather took from its speculative list (n <=
// 64 kNC entries, index order, every kept element among them): an entry is
// kept iff its key is above tau, or equal to it with an index up to iota;
// its value (from the entry) goes to the message at the tile's first rank
// plus the kept entries before it, the error there is set to 0, and the
// selection words (assembled in LDS) and rank words are written.
template <int kNC, bool kX, bool kPend>
__device__ __forceinline__ void emit_list(const u64* __restrict__ ent, uint32_t n,
                                          const TkSel* stp, int64_t rel0, uint32_t base,
                                          uint32_t keep, int count, int nw,
                                          uint64_t* __restrict__ sr, uint32_t* __restrict__ rr,
                                          float* __restrict__ vr, float* __restrict__ dr,
                                          float* __restrict__ xt, u64* s_w) {
  const int lane = lane_id();
  u64 e[kNC > 0 ? kNC : 1];
#pragma unroll
  for (int c = 0; c < kNC; ++c) {
    const uint32_t i = (uint32_t)(c * kWave + lane);
    e[c] = ent[i < n ? i : 0u];
  }
  const uint32_t tau = stp->tau;
  const int64_t iota = stp->iota;
  if (lane < kTileWords) s_w[lane] = 0ull;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  uint32_t run = 0;  // kept entries in the earlier chunks
#pragma unroll
  for (int c = 0; c < kNC; ++c) {
    const bool ok = (uint32_t)(c * kWave + lane) < n;
    const uint32_t raw = (uint32_t)e[c], key = raw & 0x7FFFFFFFu;
    const uint32_t idx = (uint32_t)(e[c] >> 32);  // index in the tile
    const bool kept = ok && (key > tau || (key == tau && rel0 + (int64_t)idx <= iota));
    const u64 km = __ballot(kept);
    if (kept) {
      atomicOr(&s_w[idx >> 6], 1ull << (idx & 63u));
      const uint32_t pos = base + run + __builtin_amdgcn_mbcnt_hi((uint32_t)(km >> 32),
                                                                  __builtin_amdgcn_mbcnt_lo((uint32_t)km, 0u));
      if (pos < keep && idx < (uint32_t)count) {  // both always hold
        vr[pos] = __uint_as_float(raw);
        if (!kPend) st_nt(dr + idx, 0.0f);  // e = Delta - C(Delta) = 0 at a kept element
        if (kX) xt[idx] -= __uint_as_float(raw);
      }
    }
    run += (uint32_t)__popcll(km);
  }
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  __builtin_amdgcn_wave_barrier();
  const u64 mine = lane < nw ? s_w[lane] : 0ull;
  if (lane < nw) sr[lane] = mine;
  const uint32_t cnt = (uint32_t)__popcll(mine);
  uint32_t incl = cnt;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  if (lane < nw) rr[lane] = base + incl - cnt;
}

// Grid: ceil((p.t1 - p.t0) / 4) * R workgroups; wave w of workgroup b owns
// tile p.t0 + 4 (b / R) + w of row b % R.  The tile's kept candidates are added to its
// selection words (LDS), then the rank words, the kept values in index order
// and the kept elements of data set to 0; kX (server): x <- x - Delta at the
// kept elements (C(Delta) is zero elsewhere).  Lane j holds selection word j
// of the tile and a wave scan of the word counts gives every rank word; then
// lane i takes the tile's kept elements i, i + 64, ...: its word by a binary
// search over the scan, its bit by nth_set_bit, so the work follows the kept
// count, not the tile size.
template <bool kX, bool kPend>
__global__ __launch_bounds__(kBlock) void k_tk_emit(DevLayout lay, TkDev tk, TkPart p, int R,
                                                    int row0, int spec,
                                                    float* __restrict__ data,
                                                    uint64_t* __restrict__ sel,
                                                    uint32_t* __restrict__ rank,
                                                    float* __restrict__ vals,
                                                    float* __restrict__ x) {
  static_assert(kTileWords == 32, "five halving steps find a word of the tile");
  __shared__ u64 words[kWaves][kTileWords];  // one row per wave, used by that wave only
  const int r = (int)(blockIdx.x % (unsigned)R);
  const int64_t ti = p.t0 + (int64_t)(blockIdx.x / (unsigned)R) * kWaves + wave_id();
  if (ti >= p.t1) return;
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int row = row0 + r;
  const int64_t W = lay.d_pad >> 6;
  // count and flag of the tile's speculative list (read before the tile so
  // that the two loads overlap)
  const uint32_t sp =
      spec ? *reinterpret_cast<const uint32_t*>(tile_hist(tk, lay, row, ti) + kTkSpecSlot) : 0u;
  const Tile tile = lay.tiles[ti];
  const int nw = (tile.count + 63) >> 6;
  uint64_t* sr = sel + (int64_t)r * W + (tile.start >> 6);
  {
    // a tile the gather took from its speculative list: emit it from the list
    if ((sp >> 16) != 0u) {
      static_assert(kTkSpecSlot % 2 == 0, "count and flag in one 32-bit word");
      const uint32_t n = sp & 0xFFFFu;
      const u64* ent = tk.spec + ((int64_t)row * lay.n_tiles + ti) * kTkSpecCap;
      const uint32_t base = tk.tile_cnt[(int64_t)row * lay.n_tiles + ti];
      const TkSel* stp = tk.sel + (int64_t)row * lay.L + tile.l;
      const int64_t rel0 = tile.start - lay.tensors[tile.l].off;
      const TkTensor* tp = tk.tens + tile.l;
      uint32_t* rr = rank + (int64_t)r * W + (tile.start >> 6);
      float* vr = vals + (int64_t)r * tk.total_keep + tp->voff;
      float* dr = data + (int64_t)r * lay.d_pad + tile.start;
      const uint32_t keep = (uint32_t)tp->keep;
      float* xt = kX ? x + tile.start : nullptr;
#define SAEF_EL(NC)                                                                   \
  emit_list<NC, kX, kPend>(ent, n, stp, rel0, base, keep, tile.count, nw, sr, rr, vr, dr, xt, \
                           words[wave])
      switch ((n + kWave - 1) / kWave) {
        case 0: SAEF_EL(0); break;
        case 1: SAEF_EL(1); break;
        case 2: SAEF_EL(2); break;
        case 3: SAEF_EL(3); break;
        case 4: SAEF_EL(4); break;
        case 5: SAEF_EL(5); break;
        case 6: SAEF_EL(6); break;
        case 7: SAEF_EL(7); break;
        default: SAEF_EL(8); break;
      }
#undef SAEF_EL
      return;
    }
  }
  const TensorInfo ten = lay.tensors[tile.l];
  const TkSel st = tk.sel[(int64_t)row * lay.L + tile.l];
  const TkTensor t = tk.tens[tile.l];
  const TileCands tc = tile_cands(lay, tk, row, ti, ten, st.cand);
  const uint32_t base = tk.tile_cnt[(int64_t)row * lay.n_tiles + ti];
  // lane j: word j of the tile (the gather's elements kept for sure)
  u64 mine = lane < nw ? sr[lane] : 0ull;
  if (tc.n > 0) {  // wave-uniform: add the kept candidates' bits
    if (lane < kTileWords) words[wave][lane] = mine;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    const u64* slots = tk.cand + (int64_t)row * lay.d_pad + ten.off + tc.first;
    const int64_t rel0 = tile.start - ten.off;
    for (uint32_t i = lane; i < tc.n; i += kWave) {
      const u64 e = slots[i];
      const int64_t q = (int64_t)(e >> 32) - rel0;  // element of the tile
      if (cand_kept(e, st) && q >= 0 && q < tile.count)
        atomicOr(&words[wave][q >> 6], 1ull << (q & 63));
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    mine = lane < nw ? words[wave][lane] : 0ull;
    if (lane < nw) sr[lane] = mine;
  }
  float* dr = data + (int64_t)r * lay.d_pad + tile.start;
  uint32_t* rr = rank + (int64_t)r * W + (tile.start >> 6);
  float* vr = vals + (int64_t)r * tk.total_keep + t.voff;
  float* xt = kX ? x + tile.start : nullptr;
  const uint32_t c = (uint32_t)__popcll(mine);
  uint32_t incl = c;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  const uint32_t excl = incl - c;
  if (lane < nw) rr[lane] = base + excl;
  const uint32_t total = (uint32_t)__shfl(incl, kWave - 1);  // kept in the tile
  const uint32_t lo = (uint32_t)mine, hi = (uint32_t)(mine >> 32);
  for (uint32_t i0 = 0; i0 < total; i0 += kWave) {
    const uint32_t i = i0 + (uint32_t)lane;  // the i-th kept element of the tile
    // its word: the number of words whose inclusive count is <= i (words past
    // nw count all of the tile, so the search stays below kTileWords)
    int u = 0;
#pragma unroll
    for (int step = kTileWords / 2; step >= 1; step >>= 1)
      if ((uint32_t)__shfl(incl, u + step - 1) <= i) u += step;
    const uint32_t wlo = (uint32_t)__shfl(lo, u), whi = (uint32_t)__shfl(hi, u);
    const uint32_t wex = (uint32_t)__shfl(excl, u);
    const int j = u * 64 + nth_set_bit(((u64)whi << 32) | wlo, i - wex);
    const uint32_t pos = base + i;
    if (i < total && j < tile.count && pos < (uint32_t)t.keep) {  // the last two always hold
      const float v = dr[j];
      vr[pos] = v;
      if (!kPend) dr[j] = 0.0f;  // e = Delta - C(Delta) = 0 at a kept element
      if (kX) xt[j] -= v;
    }
  }
}

// ------------------------------------------------------------------ server aggregation
// A wave takes whole tiles of a chunk, U selection words (U x 64 elements)
// per pass in word order, and the workers in batches of kWave / U: in a
// batch, lane q loads selection word q % U of worker q / U together with its
// rank word (one vector load each).  The values are gathered per pair (their
// masks and ranks read out of those lanes with v_readlane), per worker for
// dense messages, or over the union of the workers' kept elements (below).
// The words of the next step are loaded before the values of the current one
// are waited for, so one step costs one memory round trip.  The K values of
// an element are added in binary64 in worker order (/K, fp32); mode 1: Delta
// = e_srv + mean stored into e_srv, its pass-1 histogram and the server row's
// speculative lists; mode 0: x <- x - mean.

// A lane's (worker, word) pair: selection word, 4 x rank word (0 for a pair
// that does not exist).
struct AggWords {
  uint32_t lo, hi, rk4;
};
// The pair as loaded, with whether it exists: the words are cleared where
// they are used, in the next step (selects right after the loads made the
// compiler branch around them and wait for them, and so for every load
// issued before them, at once).
struct AggStep {
  u64 s;
  uint32_t r;
  bool ok;
  __device__ __forceinline__ AggWords words() const {
    AggWords a;
    a.lo = ok ? (uint32_t)s : 0u;
    a.hi = ok ? (uint32_t)(s >> 32) : 0u;
    a.rk4 = ok ? r * 4u : 0u;
    return a;
  }
};

template <int U>
__device__ __forceinline__ AggStep agg_words(const uint64_t* __restrict__ sel,
                                             const uint32_t* __restrict__ rank, int64_t W,
                                             int64_t gw, int K, int nw, int w0, int k0,
                                             int lane) {
  const int kq = k0 + lane / U, uq = lane % U;
  AggStep a;
  a.ok = kq < K && w0 + uq < nw;
  // always issued at a word that exists (the chunk's first word of worker 0)
  const int64_t at = a.ok ? (int64_t)kq * W + gw + w0 + uq : gw;
  a.s = sel[at];
  a.r = rank[at];
  return a;
}

// How a pass gathers the K messages' values: per (worker, word) pair, one
// load per worker for dense messages, or over the pass's union (below).
constexpr int kTkAggPairs = 0;
constexpr int kTkAggDense = 1;
constexpr int kTkAggUnion = 2;

// The means of a pass of U words when one batch holds every worker (K <= kWave
// / U; lane q holds the words of worker q / U, word q % U): the elements that
// some worker kept (the union of the K selection words of each word) are
// taken 64 at a time, one per lane, and each lane gathers its element's K
// values (a worker that did not keep it reads past the end of its buffer and
// gets 0), so a sparse pass costs K loads per 64 union elements instead of
// one per (worker, word) pair.  The sum runs over all kWave / U workers in
// order in binary64 (absent ones add +0), as in the per-pair gathers, so the
// means are the same bits.  mb (U x 64 floats, the wave's own) returns them
// per element; an element no worker kept has mean +0.  The wave's pairs go
// to wt (64 entries of 16 bytes) and its union words to ut (U entries): a
// lane reads the entry it needs with one LDS load (lanes of one word read
// one address, and the U entries of a worker are one 16 U-byte span, so the
// loads have no bank conflicts), which keeps the pass off the LDS issue
// limit that one ds_bpermute per word and worker ran into.
template <int U>
__device__ __forceinline__ void union_means(const AggWords& cur, int K, double inv_k,
                                            const float* __restrict__ vals, int64_t total_keep,
                                            uint32_t keep, int lane, float* __restrict__ mb,
                                            uint4* __restrict__ wt, uint4* __restrict__ ut,
                                            float (&mean)[U]) {
  constexpr int kB = kWave / U;
#pragma unroll
  for (int i = 0; i < U; ++i) mb[i * kWave + lane] = 0.0f;
  wt[lane] = make_uint4(cur.lo, cur.hi, cur.rk4, 0u);
  // the union of word q % U in every lane q (absent workers hold empty words)
  uint32_t ulo = cur.lo, uhi = cur.hi;
#pragma unroll
  for (int off = U; off < kWave; off <<= 1) {
    ulo |= (uint32_t)__shfl_xor((int)ulo, off);
    uhi |= (uint32_t)__shfl_xor((int)uhi, off);
  }
  // inclusive scan of the union counts over the U words (every group of U
  // lanes holds the same counts and scans them alike)
  const uint32_t cnt = (uint32_t)(__popc(ulo) + __popc(uhi));
  uint32_t incl = cnt;
#pragma unroll
  for (int off = 1; off < U; off <<= 1) {
    const uint32_t y = (uint32_t)__shfl_up((int)incl, off);
    if ((lane % U) >= off) incl += y;
  }
  if (lane < U) ut[lane] = make_uint4(ulo, uhi, incl - cnt, 0u);
  // the inclusive counts of words 0 .. U - 2, and the pass's union size
  uint32_t inc_s[U - 1];
#pragma unroll
  for (int w = 0; w < U - 1; ++w) inc_s[w] = (uint32_t)__builtin_amdgcn_readlane((int)incl, w);
  const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl, U - 1);
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  for (uint32_t i0 = 0; i0 < total; i0 += kWave) {
    const uint32_t i = i0 + (uint32_t)lane;  // the i-th union element of the pass
    // its word: the number of words whose inclusive count is <= i (at most
    // U - 1, for lanes past the end, which load and store nothing)
    int u = 0;
#pragma unroll
    for (int w = 0; w < U - 1; ++w) u += inc_s[w] <= i ? 1 : 0;
    const uint4 uw = ut[u];  // union word, union elements before it
    const int b = nth_set_bit(((u64)uw.y << 32) | uw.x, i - uw.z);
    const bool live = i < total;
    const u64 below_mask = (1ull << b) - 1ull;
    float v[kB];
#pragma unroll
    for (int kk = 0; kk < kB; ++kk) {
      const int kidx = min(kk, K - 1);  // absent workers have empty words
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          (void*)(vals + (int64_t)kidx * total_keep), 0, (int)(keep * 4u), kBufWord3);
      const uint4 pw = wt[kk * U + u];  // worker kk's selection word, 4 x rank word
      const u64 w = ((u64)pw.y << 32) | pw.x;
      const bool bit = live && ((w >> b) & 1ull) != 0ull;
      const uint32_t off = bit ? pw.z + 4u * (uint32_t)__popcll(w & below_mask) : 0x80000000u;
      v[kk] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0));
    }
    double acc = 0.0;
#pragma unroll
    for (int kk = 0; kk < kB; ++kk) acc += (double)v[kk];  // worker order; absent: +0
    if (live) mb[u * kWave + b] = (float)mean_of(acc, inv_k, K);
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
#pragma unroll
  for (int i = 0; i < U; ++i) mean[i] = mb[i * kWave + lane];
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
}

// Counts each ok lane's bin into the LDS histogram h.  The server's errors
// crowd a few bins (most of them keep last call's residual, and its binade),
// and one 64-lane LDS atomic into one address is serialized lane by lane: the
// lanes that share the first lane's bin add their count with one atomic, the
// others theirs one by one.  At resnet50 K = 8 Top-1% (union gathers) that
// took the iteration from 0.974-0.977 to 0.965-0.968 ms; repeating it for a
// second bin gave 0.976, a third 0.987-0.990 ms.
__device__ __forceinline__ void agg_hist_add(uint32_t* h, uint32_t bin, bool ok, int lane) {
  const u64 todo = __ballot(ok);
  if (todo == 0ull) return;  // wave-uniform
  const int lead = __builtin_ctzll(todo);
  const uint32_t lb = (uint32_t)__builtin_amdgcn_readlane((int)bin, lead);
  const u64 same = __ballot(bin == lb) & todo;
  if (lane == lead)
    atomicAdd(&h[lb], (uint32_t)__popcll(same));
  else if (((todo & ~same) >> lane) & 1ull)
    atomicAdd(&h[bin], 1u);
}

template <int kMode, bool kAvg, int U, int kPath>
__global__ __launch_bounds__(kBig) void k_tk_aggregate(DevLayout lay, TkDev tk, TkPart p,
                                                       int K, double inv_k,
                                                       const uint64_t* __restrict__ sel,
                                                       const uint32_t* __restrict__ rank,
                                                       const float* __restrict__ vals,
                                                       float* __restrict__ avg,
                                                       float* __restrict__ es,
                                                       float* __restrict__ x) {
  constexpr int kB = kWave / U;  // workers per batch
  static_assert(kB * U == kWave, "one (worker, word) pair per lane");
  static_assert(kTileWords % U == 0, "a pass of U words stays in one tile");
  constexpr int kChunkTiles = kTkChunk / kTkTileElems;
  __shared__ uint32_t h[kMode == 1 ? kChunkTiles * kTkHistPad : 1];  // per tile of the chunk
  __shared__ float mb[kPath == kTkAggUnion ? (kBig / kWave) * U * kWave : 1];  // a pass's means
  __shared__ uint4 wt[kPath == kTkAggUnion ? kBig : 1];                 // per wave: its 64 pairs
  __shared__ uint4 ut[kPath == kTkAggUnion ? (kBig / kWave) * U : 1];   // per wave: union words
  static_assert(kPath != kTkAggUnion || U * kWave <= (int)(sizeof(mb) / sizeof(float)),
                "a wave's means");
  const int64_t ci = p.c0 + (int64_t)blockIdx.x;
  const TkChunk c = tk.chunks[ci];
  const int64_t voff = tk.tens[c.l].voff;
  const uint32_t keep = (uint32_t)tk.tens[c.l].keep;
  const TkSel* sst = tk.sel + (int64_t)lay.k_max * lay.L + c.l;  // the server row's state
  const uint32_t win = kMode == 1 ? sst->win : 0u;
  // the server row's speculative lists, as the worker Delta pass writes them:
  // per tile, the elements whose key is at least spec_floor, in index order
  const uint32_t lo_spec = kMode == 1 ? spec_floor(*sst) : 0x80000000u;
  const TensorInfo ten = lay.tensors[c.l];
  const int64_t tile0 = ten.first_tile + (c.start - ten.off) / kTkTileElems;
  if (kMode == 1) {
    for (int i = threadIdx.x; i < kChunkTiles * kTkHistPad; i += kBig) h[i] = 0;
    __syncthreads();
  }
  const int lane = lane_id();
  const int nw = (c.count + 63) >> 6;
  const int64_t W = lay.d_pad >> 6;
  const int64_t gw = c.start >> 6;
  // e_srv (mode 1) or x (mode 0), and the mean, over the chunk's elements:
  // past the chunk a load returns 0 and a store is dropped, so the pass has
  // no per-element branch (a store in one would make the loop wait for every
  // store before the next pass)
  const uint32_t nbytes = (uint32_t)c.count * 4u;
  const Buf rd = buf_of((kMode == 1 ? es : x) + c.start, nbytes);
  const Buf ra = buf_of(kAvg ? avg + c.start : es, kAvg ? nbytes : 0u);
  // Wave w takes the chunk's tiles w, w + kBW, ... one at a time, U words per
  // pass in word order, so that a tile's passes, and its list, are one
  // wave's.
  constexpr int kBW = kBig / kWave;
  const auto next_w0 = [](int w) {
    return (w + U) % kTileWords != 0 ? w + U : w + U + (kBW - 1) * kTileWords;
  };
  bool bad = false;
  uint32_t lc = 0;  // list entries of the wave's tile so far
  // (past the chunk's last word, agg_words issues a load at a word that
  // exists and returns empty words: no branch, so no early wait)
  AggStep cur = agg_words<U>(sel, rank, W, gw, K, nw, wave_id() * kTileWords, 0, lane);
  // wait for the first words here, once: the loop header then knows them
  // loaded on both of its entries and does not wait at every pass for the
  // stores of the one before
  asm volatile("" ::"v"(cur.s), "v"(cur.r));
  for (int w0 = wave_id() * kTileWords; w0 < nw; w0 = next_w0(w0)) {
    float dv[U];
#pragma unroll
    for (int i = 0; i < U; ++i) dv[i] = buf_ld(rd, (uint32_t)((w0 + i) * 64 + lane) * 4u);
    float mean[U];
    if (kPath == kTkAggUnion) {
      // one batch holds every worker: the next pass's words go out first
      const AggStep nxt = agg_words<U>(sel, rank, W, gw, K, nw, next_w0(w0), 0, lane);
      const int wv = wave_id();
      union_means<U>(cur.words(), K, inv_k, vals + voff, tk.total_keep, keep, lane,
                     mb + wv * (U * kWave), wt + wv * kWave, ut + wv * U, mean);
      cur = nxt;
    } else {
      double acc[U];
#pragma unroll
      for (int i = 0; i < U; ++i) acc[i] = 0.0;
      for (int k0 = 0; k0 < K; k0 += kB) {
        // the next step's words go out before this step's values are waited for
        const bool last_b = k0 + kB >= K;
        const int nw0 = last_b ? next_w0(w0) : w0;
        const AggStep nxt =
            agg_words<U>(sel, rank, W, gw, K, nw, nw0, last_b ? 0 : k0 + kB, lane);
        const AggWords cw = cur.words();
        // This step's values, read through a buffer resource over each worker's
        // k_l values (a read past the end gets 0 from the range check, with no
        // memory access).
        bool done = false;
        if (kPath == kTkAggDense) {
          // Dense messages: the kept values of a worker's U words are contiguous
          // in its message; when no worker of the step has more than 64 of them,
          // one load per worker brings them all (lane j: the group's j-th
          // value) and each element takes its own with ds_bpermute.
          uint32_t gcnt = (uint32_t)(__popc(cw.lo) + __popc(cw.hi));
#pragma unroll
          for (int off = 1; off < U; off <<= 1) gcnt += (uint32_t)__shfl_xor((int)gcnt, off);
          if (__ballot(gcnt > (uint32_t)kWave) == 0ull) {  // wave-uniform
            float gv[kB];
#pragma unroll
            for (int kk = 0; kk < kB; ++kk) {
              const int kidx = min(k0 + kk, K - 1);  // absent workers have empty words
              const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                  (void*)(vals + (int64_t)kidx * tk.total_keep + voff), 0, (int)(keep * 4u),
                  kBufWord3);
              const uint32_t g4 = __builtin_amdgcn_readlane(cw.rk4, kk * U);  // group's first rank
              gv[kk] = __uint_as_float(
                  __builtin_amdgcn_raw_buffer_load_b32(rs, g4 + 4u * (uint32_t)lane, 0, 0));
            }
#pragma unroll
            for (int kk = 0; kk < kB; ++kk) {
              const uint32_t g4 = __builtin_amdgcn_readlane(cw.rk4, kk * U);
              // the U shuffles of the worker go out together (distinct
              // registers), then their values are added
              int pv[U];
#pragma unroll
              for (int i = 0; i < U; ++i) {
                const int q = kk * U + i;
                const uint32_t mlo = __builtin_amdgcn_readlane(cw.lo, q);
                const uint32_t mhi = __builtin_amdgcn_readlane(cw.hi, q);
                const uint32_t r4 = __builtin_amdgcn_readlane(cw.rk4, q);
                // the lane's element: its position among the group's kept values
                const uint32_t below =
                    __builtin_amdgcn_mbcnt_hi(mhi, __builtin_amdgcn_mbcnt_lo(mlo, 0u));
                const int src = (int)((r4 - g4) + 4u * below);  // < 4 * 64 for a kept element
                pv[i] = __builtin_amdgcn_ds_bpermute(src, __float_as_int(gv[kk]));
              }
#pragma unroll
              for (int i = 0; i < U; ++i) {
                const int q = kk * U + i;
                const uint32_t mlo = __builtin_amdgcn_readlane(cw.lo, q);
                const uint32_t mhi = __builtin_amdgcn_readlane(cw.hi, q);
                acc[i] += (double)sel_by_bit(((u64)mhi << 32) | mlo, __int_as_float(pv[i]),
                                             0.0f);  // worker order
              }
            }
            done = true;
          }
        }
        if (!done) {
          // Sparse messages (or a worker with more than 64 kept values in the
          // step's words): every (worker, word) pair gathers its values, a lane
          // whose bit is clear reading past the end; the loads go out before the
          // first one is used (dense kernels: one worker at a time, which needs fewer
          // registers next to the dense path).
          constexpr int kW = kPath == kTkAggDense ? 1 : kB;  // workers whose loads go out together
          for (int kw = 0; kw < kB; kw += kW) {
            float cv[kW][U];
#pragma unroll
            for (int kx = 0; kx < kW; ++kx) {
              const int kk = kw + kx;
              const int kidx = min(k0 + kk, K - 1);  // absent workers have empty words
              const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                  (void*)(vals + (int64_t)kidx * tk.total_keep + voff), 0, (int)(keep * 4u),
                  kBufWord3);
#pragma unroll
              for (int i = 0; i < U; ++i) {
                const int q = kk * U + i;
                const uint32_t mlo = __builtin_amdgcn_readlane(cw.lo, q);
                const uint32_t mhi = __builtin_amdgcn_readlane(cw.hi, q);
                const uint32_t r4 = __builtin_amdgcn_readlane(cw.rk4, q);
                // rank of the lane's element among the word's kept ones, in bytes
                const uint32_t below =
                    __builtin_amdgcn_mbcnt_hi(mhi, __builtin_amdgcn_mbcnt_lo(mlo, 0u));
                const uint32_t off =
                    sel_by_bit(((u64)mhi << 32) | mlo, below * 4u + r4, 0x80000000u);
                cv[kx][i] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0));
              }
            }
#pragma unroll
            for (int kx = 0; kx < kW; ++kx)
#pragma unroll
              for (int i = 0; i < U; ++i) acc[i] += (double)cv[kx][i];  // worker order; absent: +0
          }
        }
        cur = nxt;
      }
#pragma unroll
      for (int i = 0; i < U; ++i) mean[i] = (float)mean_of(acc[i], inv_k, K);
    }
    // the tile's list (kTkSpecCap entries; a store past it is dropped)
    const int tl = w0 / kTileWords;  // tile of the chunk
    const Buf rl = buf_of(tk.spec + ((int64_t)lay.k_max * lay.n_tiles + tile0 + tl) * kTkSpecCap,
                          kMode == 1 ? (uint32_t)kTkSpecCap * 8u : 0u);
#pragma unroll
    for (int i = 0; i < U; ++i) {
      const int j = (w0 + i) * 64 + lane;
      const bool ok = j < c.count;
      const uint32_t off = (uint32_t)j * 4u;
      if (kAvg) buf_st(ra, off, mean[i]);
      if (kMode == 1) {
        const float D = dv[i] + mean[i];  // Delta_{t+1} = e_t + (1/K) sum_k C(Delta^(k))
        buf_st(rd, off, D);
        const uint32_t key = key_of(D);
        bad |= ok && key >= kFiniteLimit;
        // list entry: Delta's bits | index in the tile << 32
        const u64 lm = __ballot(ok && key >= lo_spec);
        const uint32_t pos = lc + __builtin_amdgcn_mbcnt_hi((uint32_t)(lm >> 32),
                                                            __builtin_amdgcn_mbcnt_lo((uint32_t)lm, 0u));
        u32x2 ev;
        ev.x = __float_as_uint(D);
        ev.y = (uint32_t)(j - tl * kTkTileElems);
        __builtin_amdgcn_raw_buffer_store_b64(
            ev, rl, ((lm >> lane) & 1ull) && pos < (uint32_t)kTkSpecCap ? pos * 8u : 0x80000000u,
            0, 0);
        lc += (uint32_t)__popcll(lm);
        // a pass stays in one tile; a lane past the chunk adds nothing
        const uint32_t hb = (uint32_t)(w0 / kTileWords) * kTkHistPad + hist_bin(key, win);
        // (the dense gathers lost with the leader: Top-5% 1.122-1.125 against
        // 1.111 ms, Top-10% 1.257 against 1.247-1.249 ms)
        if (kPath == kTkAggUnion)
          agg_hist_add(h, hb, ok, lane);
        else
          atomicAdd(&h[hb], ok ? 1u : 0u);
      } else {
        buf_st(rd, off, dv[i] - mean[i]);  // single-way: the mean itself comes back
      }
    }
    if (kMode == 1 && ((w0 + U) % kTileWords == 0 || w0 + U >= nw)) {
      // the tile's last pass: its list count (none before the first
      // threshold, for a tensor without lists, or past kTkSpecCap entries)
      if (lane == 0)
        h[tl * kTkHistPad + kTkSpecSlot] =
            lo_spec != 0x80000000u && lc <= (uint32_t)kTkSpecCap ? lc : kTkSpecNone;
      lc = 0;
    }
  }
  if (kMode == 1) {
    if (__ballot(bad) != 0 && lane_id() == 0) atomicOr(lay.status, kStatusRange);
    __syncthreads();
    // the tile histograms of the chunk, 16-bit counts, two bins per store
    // (the list count in slot kTkSpecSlot, 0 in the flag slot after it)
    const int ntile = (c.count + kTkTileElems - 1) / kTkTileElems;
    uint32_t* out = reinterpret_cast<uint32_t*>(tile_hist(tk, lay, lay.k_max, tile0));
    for (int i = threadIdx.x; i < ntile * (kTkHistPad / 2); i += kBig)
      out[i] = (h[2 * i] & 0xFFFFu) | (h[2 * i + 1] << 16);
  }
}

// ------------------------------------------------------------------ host side
struct Launcher {
  const DevLayout& lay;
  const TkDev& tk;
  hipStream_t s;

  // The Delta pass of R rows (row0..) over the part's tiles; `start` stamps
  // the dispatch's start when non-null.
  hipError_t delta(const TkPart& p, int R, int row0, float lr, float mu, const float* g,
                   float* m, float* e, const uint64_t* psel, bool pend_in,
                   hipEvent_t start) const {
    const dim3 grid((unsigned)((int64_t)(p.t1 - p.t0) * R));
#define SAEF_TKD(MOM, PEND)                                                                  \
  hipExtLaunchKernelGGL((k_tk_delta<MOM, PEND>), grid, dim3(kBlock), kTkDeltaLdsPad, s, start, \
                        nullptr, 0, lay, tk, p, R, row0, lr, mu, g, m, e, psel)
    if (m != nullptr) {
      if (pend_in) SAEF_TKD(true, true); else SAEF_TKD(true, false);
    } else {
      if (pend_in) SAEF_TKD(false, true); else SAEF_TKD(false, false);
    }
#undef SAEF_TKD
    return hipGetLastError();
  }

  // everything after the first pass for R rows of `data` (rows row0..) over
  // the part's tensors: sums, pick, offsets, gather, select (with the tile
  // ranks), emit.
  // The last kernel stamps the caller's stop event.
  hipError_t select_and_emit(const TkPart& p, int R, int row0, float* data, uint64_t* sel,
                             uint32_t* rank, float* vals, float* x, bool pend_out,
                             const LaunchEvents& last) const {
    const LaunchEvents ev;
    hipError_t err;
    const dim3 groups((unsigned)((int64_t)R * (p.g1 - p.g0)));
    SAEF_LAUNCH(k_tk_sum<false>, groups, dim3(kBlock), 0, s, lay, tk, p, row0);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    if (p.s1 > p.s0) {
      SAEF_LAUNCH(k_tk_sum<true>, dim3((unsigned)((int64_t)R * (p.s1 - p.s0))), dim3(kBlock), 0,
                  s, lay, tk, p, row0);
      if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    const dim3 pairs((unsigned)((int64_t)R * (p.l1 - p.l0)));
    const dim3 tiles((unsigned)((int64_t)(p.t1 - p.t0 + kWaves - 1) / kWaves * R));
    SAEF_LAUNCH(k_tk_pick, pairs, dim3(kBlock), 0, s, lay, tk, p, row0);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    SAEF_LAUNCH(k_tk_offsets, groups, dim3(kWave), 0, s, lay, tk, p, row0);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    // speculative lists (written by the worker Delta pass, and for the
    // server row by the aggregation), if some tensor keeps them
    const int spec = tk.lists != 0 ? 1 : 0;
    if (spec)
      SAEF_LAUNCH(k_tk_gather_spec, tiles, dim3(kBlock), 0, s, lay, tk, p, R, row0, data, sel);
    else
      SAEF_LAUNCH(k_tk_gather_full, tiles, dim3(kBlock), 0, s, lay, tk, p, R, row0, data, sel);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    SAEF_LAUNCH(k_tk_select, pairs, dim3(kBig), 0, s, lay, tk, p, row0);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    if (x != nullptr)
      hipExtLaunchKernelGGL((k_tk_emit<true, false>), tiles, dim3(kBlock), 0, s, nullptr,
                            last.stop, 0, lay, tk, p, R, row0, spec, data, sel, rank, vals, x);
    else if (pend_out)
      hipExtLaunchKernelGGL((k_tk_emit<false, true>), tiles, dim3(kBlock), 0, s, nullptr,
                            last.stop, 0, lay, tk, p, R, row0, spec, data, sel, rank, vals, x);
    else
      hipExtLaunchKernelGGL((k_tk_emit<false, false>), tiles, dim3(kBlock), 0, s, nullptr,
                            last.stop, 0, lay, tk, p, R, row0, spec, data, sel, rank, vals, x);
    return hipGetLastError();
  }

  // The server step over the part's tensors: the aggregation of the K
  // messages, then (mode 1) the server row's selection and message.  The
  // aggregation stamps ev.start; the last kernel ev.stop.
  hipError_t server(const TkPart& p, int K, int mode, const uint64_t* sel, const uint32_t* rank,
                    const float* vals, float* avg, float* e_srv, uint64_t* srv_sel,
                    uint32_t* srv_rank, float* srv_vals, float* x,
                    const LaunchEvents& ev) const {
    const dim3 grid((unsigned)(p.c1 - p.c0));
    const double ik = inv_pow2(K);
    hipEvent_t stop0 = mode == 1 ? nullptr : ev.stop;
    // dense messages (at least 1/32 of the elements kept): one load per worker
    // and step, values handed out with ds_bpermute; sparser ones: gathers over
    // the union of the workers' kept elements when one batch holds every
    // worker (K <= 16), else per-pair gathers.  At resnet50 K = 8 the union
    // took the Top-1% iteration from 1.000 to 0.984 ms (its end, pipelined:
    // 710 -> 680 us); for dense messages it lost to the one-load-per-worker
    // path (Top-5% 1.12 against 1.11 ms, Top-10% 1.29 against 1.25 ms).
    const bool co = tk.total_keep * 32 >= lay.d_pad;
#define SAEF_TKA(M, A, U, C)                                                                 \
  hipExtLaunchKernelGGL((k_tk_aggregate<M, A, U, C>), grid, dim3(kBig), 0, s, ev.start, stop0, \
                        0, lay, tk, p, K, ik, sel, rank, vals, avg, e_srv, x)
#define SAEF_TKA_U(M, A)                                                    \
  do {                                                                      \
    if (K <= 8) {                                                           \
      if (co) SAEF_TKA(M, A, 8, kTkAggDense);                               \
      else SAEF_TKA(M, A, 8, kTkAggUnion);                                  \
    } else if (K <= 16) {                                                   \
      if (co) SAEF_TKA(M, A, 4, kTkAggDense);                               \
      else SAEF_TKA(M, A, 4, kTkAggUnion);                                  \
    } else {                                                                \
      if (co) SAEF_TKA(M, A, 4, kTkAggDense);                               \
      else SAEF_TKA(M, A, 4, kTkAggPairs);                                  \
    }                                                                       \
  } while (0)
    if (mode == 1) {
      if (avg != nullptr) SAEF_TKA_U(1, true); else SAEF_TKA_U(1, false);
    } else {
      if (avg != nullptr) SAEF_TKA_U(0, true); else SAEF_TKA_U(0, false);
    }
#undef SAEF_TKA_U
#undef SAEF_TKA
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess || mode != 1) return err;
    return select_and_emit(p, 1, lay.k_max, e_srv, srv_sel, srv_rank, srv_vals, x, false, ev);
  }
};

}  // namespace

// After a fork, an error still joins: s waits for whatever the side stream
// was given, so no work of this call outlives it on the side stream.
static hipError_t join_side(hipStream_t s, const TkStreams& side, hipError_t err) {
  const hipError_t e1 = hipEventRecord(side.join, side.stream);
  const hipError_t e2 = e1 == hipSuccess ? hipStreamWaitEvent(s, side.join, 0) : e1;
  return err != hipSuccess ? err : e2;
}

hipError_t launch_topk_compress(const DevLayout& lay, const TkDev& tk, const TkPart& all, int K,
                                float lr, float mu, const float* g, float* m, float* e,
                                uint64_t* sel, uint32_t* rank, float* vals, bool pend_in,
                                bool pend_out, hipStream_t s, const TkStreams& side,
                                const LaunchEvents& ev) {
  // The Delta pass of a group of rows is HBM-bound; the selection chain that
  // follows it (sums, pick, offsets, gather, select, scan, emit) is mostly
  // launch- and latency-bound.  With a side stream the workers are taken in
  // two groups: the first group's chain runs on the side stream while the
  // second group's Delta pass streams on s; s waits for the side stream at
  // the end.  The groups' scratch rows are disjoint.
  const bool split = side.stream != nullptr && K >= 2;
  const int R0 = split ? (K + 1) / 2 : K;
  const Launcher main{lay, tk, s};
  const int64_t W = lay.d_pad >> 6;
  // the first Delta pass stamps the start event, the last kernel on s the stop event
  hipError_t err = main.delta(all, R0, 0, lr, mu, g, m, e, sel, pend_in, ev.start);
  if (err != hipSuccess) return err;
  if (!split) return main.select_and_emit(all, K, 0, e, sel, rank, vals, nullptr, pend_out, ev);
  const int R1 = K - R0;
  if ((err = hipEventRecord(side.fork, s)) != hipSuccess) return err;
  if ((err = hipStreamWaitEvent(side.stream, side.fork, 0)) != hipSuccess) return err;
  const Launcher aside{lay, tk, side.stream};
  err = aside.select_and_emit(all, R0, 0, e, sel, rank, vals, nullptr, pend_out, LaunchEvents());
  if (err == hipSuccess) err = main.delta(all, R1, R0, lr, mu, g, m, e, sel, pend_in, nullptr);
  if (err == hipSuccess)
    err = main.select_and_emit(all, R1, R0, e + (int64_t)R0 * lay.d_pad, sel + (int64_t)R0 * W,
                               rank + (int64_t)R0 * W, vals + (int64_t)R0 * tk.total_keep,
                               nullptr, pend_out, ev);
  return join_side(s, side, err);
}

hipError_t launch_topk_round_end(const DevLayout& lay, const TkDev& tk, const TkPart* parts,
                                 int n_parts, int K, float lr, float mu, int mode,
                                 const float* g, float* m, float* e, uint64_t* sel,
                                 uint32_t* rank, float* vals, bool pend_in, float* e_srv,
                                 uint64_t* srv_sel, uint32_t* srv_rank, float* srv_vals,
                                 float* x, hipStream_t s, const TkStreams& side,
                                 const LaunchEvents& ev) {
  // Every step after the Delta pass works tensor by tensor, so the parts are
  // independent once their Delta is formed: the Delta passes of the parts
  // stream one after another on s, and each part but the last, as soon as
  // its Delta is stored, runs its worker selection and messages and its
  // server step on the side stream, under the next parts' Delta passes; the
  // last part's steps run on s, which then waits for the side stream.  All
  // data and scratch of two parts are disjoint (tiles, groups, chunks and
  // (row, tensor) state).
  const Launcher main{lay, tk, s};
  const Launcher aside{lay, tk, side.stream};
  hipError_t err = hipSuccess;
  bool forked = false;
  for (int i = 0; i < n_parts && err == hipSuccess; ++i) {
    const TkPart& p = parts[i];
    const bool last = i == n_parts - 1;
    err = main.delta(p, K, 0, lr, mu, g, m, e, sel, pend_in, i == 0 ? ev.start : nullptr);
    if (err == hipSuccess && !last) {
      err = hipEventRecord(side.fork, s);
      if (err == hipSuccess) err = hipStreamWaitEvent(side.stream, side.fork, 0);
      forked = forked || err == hipSuccess;
    }
    const Launcher& on = last ? main : aside;
    if (err == hipSuccess)
      err = on.select_and_emit(p, K, 0, e, sel, rank, vals, nullptr, true, LaunchEvents());
    LaunchEvents tail;
    if (last) tail.stop = ev.stop;
    if (err == hipSuccess)
      err = on.server(p, K, mode, sel, rank, vals, nullptr, e_srv, srv_sel, srv_rank, srv_vals,
                      x, tail);
  }
  return forked ? join_side(s, side, err) : err;
}

// Grid: n_tiles * K workgroups; workgroup b sets to 0 the elements of worker
// b % K's tile b / K whose selection bit is set (wave w: words w*kTkU ..).
__global__ __launch_bounds__(kBlock) void k_tk_zero(DevLayout lay, int K, float* __restrict__ e,
                                                    const uint64_t* __restrict__ sel) {
  const int k = (int)(blockIdx.x % (unsigned)K);
  const int64_t ti = blockIdx.x / (unsigned)K;
  const Tile tile = lay.tiles[ti];
  const int nw = (tile.count + 63) >> 6;
  const int lane = lane_id();
  const uint64_t* sk = sel + (int64_t)k * (lay.d_pad >> 6) + (tile.start >> 6);
  float* ek = e + (int64_t)k * lay.d_pad + tile.start;
  for (int w = wave_id() * kTkU; w < min(nw, wave_id() * kTkU + kTkU); ++w) {
    const u64 word = sk[w];
    const int j = w * 64 + lane;
    if (((word >> lane) & 1ull) && j < tile.count) ek[j] = 0.0f;
  }
}

hipError_t launch_topk_materialize(const DevLayout& lay, int K, float* e, const uint64_t* sel,
                                   hipStream_t s, const LaunchEvents& ev) {
  const dim3 grid((unsigned)(lay.n_tiles * K));
  SAEF_LAUNCH(k_tk_zero, grid, dim3(kBlock), 0, s, lay, K, e, sel);
  return hipGetLastError();
}

hipError_t launch_topk_aggregate(const DevLayout& lay, const TkDev& tk, const TkPart& all,
                                 int K, int mode, const uint64_t* sel, const uint32_t* rank,
                                 const float* vals, float* avg, float* e_srv, uint64_t* srv_sel,
                                 uint32_t* srv_rank, float* srv_vals, float* x, hipStream_t s,
                                 const LaunchEvents& ev) {
  return Launcher{lay, tk, s}.server(all, K, mode, sel, rank, vals, avg, e_srv, srv_sel,
                                     srv_rank, srv_vals, x, ev);
}

}  // namespace saef
