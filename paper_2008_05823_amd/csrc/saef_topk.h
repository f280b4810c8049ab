// Internal declarations of the layer-wise Top-K compressor (kernels in
// saef_topk.hip, entry points in saef_api.hip); not part of the public C ABI.
#pragma once

#include "saef_internal.h"

namespace saef {

// Pass-1 histogram of the key |v| over a window of four binades (exponents)
// of a (row, tensor), placed around the previous call's threshold: 64 bins
// per binade (key bits 22..17) inside the window; below it one bin per binade
// for the kTkLo - 1 binades under the window and one bin for all lower keys;
// one bin above it.  The window only decides how many elements become
// candidates; the kept set is exact wherever the threshold falls.  (With one
// bin below, a threshold that fell more than two binades made every element
// under the window a candidate: at bert_base Top-1% the selection of the word
// embedding then took 10-23 ms.  Above the window there are few elements.)
constexpr int kTkSubShift = 17;                // in-window bin width: 2^17 keys
constexpr int kTkWin = 256;                    // in-window bins (4 binades)
constexpr int kTkLo = 8;                       // bins below the window
constexpr int kTkHist = kTkLo + kTkWin + 1;    // + one above
constexpr int kTkHistPad = 268;                // 16-bit counts per tile (even, 8-byte rows)
constexpr int kTkGroup = 64;      // tile histograms (or group sums) one sum workgroup adds
constexpr int kTkBins = 2048;     // bins of an 11-bit radix digit
constexpr int kTkChunk = 65536;   // elements per server-aggregation workgroup
// Speculative candidate lists: for a tensor that keeps at most 1/8 of its
// elements, the worker Delta pass also writes, per (row, tile), the elements
// whose key is at least the previous call's threshold key minus
// kTkSpecMargin (1/32 binade), in index order, up to kTkSpecCap of them; their
// count goes to slot kTkSpecSlot of the tile histogram (kTkSpecNone when the
// tile had more, or for the server row).  When the bin b1 that this call's
// histogram picks lies at or above that bound, the list holds every element
// the gather needs and the tile's Delta is not read again.  (Under error
// feedback the threshold mostly rises from call to call, and the elements
// just below it pile up: at 1% kept the lists hold about 3% of the elements.)
constexpr int kTkSpecCap = 512;
constexpr int kTkSpecSlot = (kTkHist + 1) & ~1;  // the first even slot past the bins
constexpr uint32_t kTkSpecNone = 0xFFFFu;
constexpr uint32_t kTkSpecMargin = 1u << 18;
constexpr int kTkSpecMaxShare = 8;  // lists when k_l * 8 <= n_l
// Dynamic LDS the Delta pass requests and does not use: with its own 1 KB
// it keeps at most 5 of its workgroups on a CU (160 KB of LDS), so the
// selection kernels of the other rows or tensors, launched on the side
// stream while a Delta pass streams, find free slots.  At resnet50 K = 8
// Top-1% per iteration: 1.014 ms against 1.030 ms uncapped, 1.017 ms with
// only the overlapped pass capped, 1.022 ms at 4 workgroups per CU.
constexpr unsigned kTkDeltaLdsPad = 26624;
// The Top-K kernels take a tile as 32 sign words (one per lane of a gather
// wave): they need the layout's tiles to hold 2048 elements.  A library built
// with another SAEF_TILE_ELEMS (the sign path works with any) refuses Top-K
// plans (saef_topk_create returns SAEF_EINVAL).
constexpr int kTkTileElems = 2048;
constexpr bool kTkUsable = kTileElems == kTkTileElems;
static_assert(kTkHistPad >= kTkSpecSlot + 2 && kTkHistPad % 4 == 0, "padded tile histogram");
static_assert(kTkTileElems < 65536, "a tile's bin counts fit 16 bits");
static_assert(kTkChunk % kTkTileElems == 0, "a server chunk holds whole tiles");
static_assert(kTkSpecSlot < kTkHistPad && kTkSpecSlot % 2 == 0, "a spare, even histogram slot");
static_assert(kTkSpecCap < (int)kTkSpecNone, "list counts fit the slot below the marker");
static_assert((int64_t)kTileElems * kMaxTilesPerTensor >= kMaxTensor,
              "every tensor is cut into tiles of kTileElems elements");

// Up to kTkChunk elements of one tensor (whole tiles): the server's workgroups.
struct TkChunk {
  int64_t start;  // absolute element index (multiple of 64)
  int32_t l;
  int32_t count;
};

// kTkGroup consecutive tiles of one tensor (a group), or kTkGroup consecutive
// groups of one tensor (a super-group).
struct TkGroup {
  int32_t l;
  int32_t first;  // first tile (group) index, global
  int32_t n;      // tiles (groups) in it
  int32_t pad;
};

struct TkTensor {
  int64_t voff;         // first value of the tensor in a message
  int64_t keep;         // k_l
  int32_t first_chunk;  // server chunks
  int32_t nchunks;
  int32_t first_group;  // tile groups
  int32_t ngroups;
  int32_t first_sgroup;  // super-groups, when ngroups > kTkGroup
  int32_t nsgroups;      // 0 otherwise
};

// Selection state of one (row, tensor): the histogram window (kept from one
// call to the next); after the pick, the bin b1 that holds the k-th largest
// key, how many elements to take from it and how many it holds (the
// candidates); after the select, the threshold key tau and the last kept
// index iota (in the tensor) of the elements equal to tau.
struct TkSel {
  uint32_t tau;
  uint32_t win;     // window base key (a multiple of 2^23)
  uint32_t bin;     // b1
  uint32_t lists;   // 1: worker rows of this tensor keep speculative lists (set at creation)
  int64_t need;
  int64_t cand;
  int64_t iota;     // elements equal to tau with index <= iota are kept
};

// A run of whole tensors [l0, l1) with the tiles, tile groups, super-groups
// and server chunks that belong to them: each a contiguous index range, since
// all four are numbered tensor by tensor.  The Top-K kernels work on one
// part; the whole layout is one part.
struct TkPart {
  int32_t l0, l1;  // tensors
  int32_t t0, t1;  // tiles
  int32_t g0, g1;  // tile groups
  int32_t s0, s1;  // super-groups
  int32_t c0, c1;  // server chunks
};

struct TkDev {
  const TkChunk* chunks;
  const TkTensor* tens;
  const TkGroup* groups;
  const TkGroup* sgroups;
  uint16_t* thist;     // [rows][n_tiles][kTkHistPad] tile histograms
  uint32_t* ghist;     // [rows][n_groups][kTkHistPad] group sums
  uint32_t* sghist;    // [rows][n_sgroups][kTkHistPad] super-group sums
  uint32_t* goff;      // [rows][n_groups] first candidate slot of the group in its tensor
  TkSel* sel;          // [rows][L]
  uint32_t* tile_cnt;  // [rows][n_tiles] kept per tile, then the exclusive prefix
  uint32_t* cand_off;  // [rows][n_tiles] first candidate slot of the tile in its tensor
  unsigned long long* cand;  // [rows][d_pad] candidate slots: (row, tensor) at the tensor's offset
  unsigned long long* spec;  // [k_max][n_tiles][kTkSpecCap] key | (index in the tile) << 32
  int64_t n_chunks;
  int64_t n_groups;
  int64_t n_sgroups;
  int64_t total_keep;
  int32_t lists;  // 1: some tensor keeps speculative lists
  int32_t pad;
};

// Worker Top-K compression of K rows (row k of e, histogram row k).  m
// non-null: momentum.  Writes Delta into e, the selection words, rank words
// and values of each row.  pend_in: e holds the previous call's Delta whose
// kept elements (the selection words in sel) are still to be set to 0; they
// are read as 0.  pend_out: this call's kept elements are left as they are
// (pending, for the next reader) instead of being set to 0.
//
// side: a second stream of the plan and two events (fork, join).  When
// given and K >= 2, the rows are compressed in two groups and the first
// group's selection runs on the side stream, overlapping the second group's
// Delta pass; s waits for the side stream before the call returns (an event
// fork and join, so the launches stay capturable in a HIP graph).
struct TkStreams {
  hipStream_t stream = nullptr;
  hipEvent_t fork = nullptr;
  hipEvent_t join = nullptr;
};
// `all`: the part of every tensor.
hipError_t launch_topk_compress(const DevLayout& lay, const TkDev& tk, const TkPart& all, int K,
                                float lr, float mu, const float* g, float* m, float* e,
                                uint64_t* sel, uint32_t* rank, float* vals, bool pend_in,
                                bool pend_out, hipStream_t s, const TkStreams& side,
                                const LaunchEvents& ev = LaunchEvents());

// Sets to 0 the elements of the K rows of e whose selection bit is set.
hipError_t launch_topk_materialize(const DevLayout& lay, int K, float* e, const uint64_t* sel,
                                   hipStream_t s, const LaunchEvents& ev = LaunchEvents());

// Server Top-K aggregation: mean of the K decoded messages; mode 1: e_srv
// <- e_srv + mean, its Top-K message, e_srv at kept elements <- 0 and x <- x
// - C(Delta); mode 0: x <- x - mean.  avg written when non-null.
hipError_t launch_topk_aggregate(const DevLayout& lay, const TkDev& tk, const TkPart& all,
                                 int K, int mode, const uint64_t* sel, const uint32_t* rank,
                                 const float* vals, float* avg, float* e_srv, uint64_t* srv_sel,
                                 uint32_t* srv_rank, float* srv_vals, float* x, hipStream_t s,
                                 const LaunchEvents& ev = LaunchEvents());

// The worker compression (pend_out: its kept elements left pending) and the
// server step of one iteration, pipelined over n_parts >= 2 parts that
// cover the tensors in order: the parts' Delta passes run one after another
// on s, and each part but the last then takes its selection, messages and
// server step on the side stream while the later parts' Delta passes
// stream; s waits for the side stream at the end (an event fork and join).
// The same results as launch_topk_compress then launch_topk_aggregate (avg
// null).  ev: start stamped by the first Delta pass, stop by the last kernel
// on s.
hipError_t launch_topk_round_end(const DevLayout& lay, const TkDev& tk, const TkPart* parts,
                                 int n_parts, int K, float lr, float mu, int mode,
                                 const float* g, float* m, float* e, uint64_t* sel,
                                 uint32_t* rank, float* vals, bool pend_in, float* e_srv,
                                 uint64_t* srv_sel, uint32_t* srv_rank, float* srv_vals,
                                 float* x, hipStream_t s, const TkStreams& side,
                                 const LaunchEvents& ev = LaunchEvents());

}  // namespace saef
