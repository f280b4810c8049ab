// Internal declarations of the layer-wise Top-K compressor (kernels in
// saef_topk.hip, entry points in saef_api.hip); not part of the public C ABI.
#pragma once

#include "saef_internal.h"

namespace saef {

constexpr int kTkChunk = 65536;    // elements per histogram chunk (multiple of the tile)
constexpr int kTkBins = 2048;      // bins of an 11-bit radix digit
constexpr int kTkBins3 = 512;      // bins of the 9-bit key digit
constexpr int kTkRedChunks = 64;   // chunk histograms one reduce workgroup adds
static_assert(kTkChunk % kTileElems == 0, "a Top-K chunk holds whole tiles");
static_assert((int64_t)kTileElems * kMaxTilesPerTensor >= kMaxTensor,
              "every tensor is cut into tiles of kTileElems elements");

struct TkChunk {
  int64_t start;  // absolute element index (multiple of 64)
  int32_t l;
  int32_t count;
};

struct TkTensor {
  int64_t voff;        // first value of the tensor in a message
  int64_t keep;        // k_l
  int32_t first_chunk;
  int32_t nchunks;
};

// Selection state of one (row, tensor): after the pick, the bin b1 of key
// bits 30..20 that holds the k-th largest key, how many elements to take
// from it and how many it holds (the candidates); after the select, the
// threshold key tau and the last kept index iota (in the tensor) of the
// elements equal to tau.
struct TkSel {
  uint32_t prefix;  // b1, then tau
  uint32_t pad;
  int64_t need;
  int64_t cand;
  int64_t iota;     // elements equal to tau with index <= iota are kept
};

struct TkDev {
  const TkChunk* chunks;
  const TkTensor* tens;
  uint32_t* hist;    // [rows][n_chunks][kTkBins] chunk histograms
  uint32_t* hist2;   // [rows][L][red_split][kTkBins] second-level sums (red_split > 1)
  TkSel* sel;        // [rows][L]
  uint32_t* tile_cnt;  // [rows][n_tiles] kept per tile, then the exclusive prefix
  unsigned long long* cand;  // [rows][d_pad] candidate slots: (row, tensor) at the tensor's offset
  uint32_t* cand_off;  // [rows][n_chunks] first slot of each chunk's candidates
  int64_t n_chunks;
  int64_t total_keep;
  int32_t red_split;   // reduce workgroups per (row, tensor)
};

// Worker Top-K compression of K rows (row k of e, hist row k).  m non-null:
// momentum.  Writes Delta into e (then the kept elements are zeroed), the
// selection words, rank words and values of each row.
hipError_t launch_topk_compress(const DevLayout& lay, const TkDev& tk, int K, float lr, float mu,
                                const float* g, float* m, float* e, uint64_t* sel,
                                uint32_t* rank, float* vals, hipStream_t s,
                                const LaunchEvents& ev = LaunchEvents());

// Server Top-K aggregation: mean of the K decoded messages; mode 1: e_srv
// <- e_srv + mean, its Top-K message, e_srv at kept elements <- 0 and x <- x
// - C(Delta); mode 0: x <- x - mean.  avg written when non-null.
hipError_t launch_topk_aggregate(const DevLayout& lay, const TkDev& tk, int K, int mode,
                                 const uint64_t* sel, const uint32_t* rank, const float* vals,
                                 float* avg, float* e_srv, uint64_t* srv_sel, uint32_t* srv_rank,
                                 float* srv_vals, float* x, hipStream_t s,
                                 const LaunchEvents& ev = LaunchEvents());

}  // namespace saef
