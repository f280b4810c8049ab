// Internal declarations shared by the kernel and host translation units of
// the SAEF library (not part of the public C ABI in include/saef.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace saef {

constexpr int kWave = 64;             // CDNA wavefront width
constexpr int kBlock = 256;           // threads per workgroup (4 waves)
constexpr int kWaves = kBlock / kWave;
#ifndef SAEF_TILE_ELEMS
#define SAEF_TILE_ELEMS 2048
#endif
constexpr int kTileElems = SAEF_TILE_ELEMS;  // default work tile (elements, multiple of 64)
static_assert((SAEF_TILE_ELEMS & (SAEF_TILE_ELEMS - 1)) == 0 && SAEF_TILE_ELEMS >= 64,
              "the tile size is a power of two of at least one sign word");
constexpr int64_t kMaxTensor = int64_t(1) << 28;
constexpr int kMaxTilesPerTensor = (int)(kMaxTensor / kTileElems);  // tiles of a maximal tensor
constexpr int kFinChunk = 4096;              // tile partials per finalize workgroup
// The step ahead keeps no per-tile sums, so it takes a tile in work units of
// kStepElems elements, one workgroup each (1024-element units stream faster
// than whole 2048-element tiles).
constexpr int kStepElems = kTileElems < 1024 ? kTileElems : 1024;
constexpr int kStepSplit = kTileElems / kStepElems;  // units per tile
constexpr int kXcds = 8;  // MI355X: 8 XCDs, workgroups dealt round-robin

// XCD-aware tile order.  Workgroups are dealt to the 8 XCDs round-robin
// (XCD b mod 8); XCD x takes run x of every group of 8 runs of 2^s
// consecutive tiles, so each XCD streams contiguous memory and sees every
// row (worker) of its tiles, which shares x through its L2.  Long runs
// (s = 6, 512 KB of a row) stream best on large layouts (measured: -15% for
// the step ahead at 2^28 parameters); layouts of fewer than 2048 tiles keep
// s = 0, where long runs would leave XCDs idle.
__host__ __device__ inline int tile_run_shift(int64_t n_tiles) { return n_tiles >= 2048 ? 6 : 0; }

// Tiles rounded up to whole groups of 8 runs.
inline int64_t run_padded_tiles(int64_t n_tiles) {
  const int64_t g = (int64_t)kXcds << tile_run_shift(n_tiles);
  return (n_tiles + g - 1) / g * g;
}

// One unit of work: `count` consecutive elements of tensor `l` starting at
// absolute element index `start` (a multiple of 64).
struct Tile {
  int64_t start;
  int32_t l;
  int32_t count;
};

struct TensorInfo {
  int64_t off;
  int64_t n;
  int32_t first_tile;
  int32_t ntiles;
};

// Device-side view of a layout, passed by value to every kernel.
struct DevLayout {
  const Tile* tiles;
  const TensorInfo* tensors;
  unsigned long long* part;  // [(k_max + 1) * n_tiles * 2] exact partial sums (lo, hi) of
                             // each tile; row k_max belongs to the server
  unsigned long long* part2; // [(k_max + 1) * L * fin_split * 2] second-level sums
  int32_t fin_split;         // finalize workgroups per (row, tensor): ceil(max tiles / kFinChunk)
  int* status;               // sticky error flag
  int64_t n_tiles;
  int64_t d_pad;
  int32_t L;
  int32_t k_max;
};

// status flag bits
constexpr int kStatusRange = 1;

// Optional timing of one launch: when set, the kernel's dispatch packet
// records its start and end in these events (no extra queue packets).
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

// ---- kernel launchers (defined in saef_kernels.hip) ----------------------
// All return hipSuccess or the launch error.  Arguments are validated by the
// caller.  Each launcher enqueues one kernel (launch_finalize: one or two).

// Worker compression.  decode: e holds values with a pending correction
// (signs/scales of the previous compression) that is applied on read.  m
// non-null: momentum, m <- fma(mu, m, g) and Delta = fma(lr, m, e); else
// Delta = fma(lr, g, e).  Always writes Delta (before correction) into e,
// the new sign words and the tile partial sums; launch_finalize then writes
// the new scales.
hipError_t launch_compress(const DevLayout& lay, int K, float lr, float mu, const float* g,
                           float* m, float* e, uint64_t* signs, const float* scales, bool decode,
                           hipStream_t s, const LaunchEvents& ev = LaunchEvents());

// Scales from the tile partial sums: worker rows 0..K-1 into scales[k][l]
// (server == false) or the server row into scales[l] (server == true).  One
// kernel, or two when a tensor has more than kFinChunk tiles (fin_split > 1).
hipError_t launch_finalize(const DevLayout& lay, int K, bool server, float* scales,
                           hipStream_t s,
                           const LaunchEvents& ev = LaunchEvents());

// Server aggregation.  mode 1: reads/writes e_srv (Delta before correction),
// writes srv_signs and the server tile partial sums (launch_finalize then
// writes srv_scales); decode applies the pending server correction (old
// srv_signs/srv_scales) to e_srv on read and materializes it into x.
// mode 0: x <- x - mean.  avg written when non-null.
hipError_t launch_aggregate(const DevLayout& lay, int K, int mode, const uint64_t* signs,
                            const float* scales, float* avg, float* e_srv, uint64_t* srv_signs,
                            const float* srv_scales, float* x, bool decode, hipStream_t s,
                           const LaunchEvents& ev = LaunchEvents());

// How the worker errors are read: as stored; with the pending scaled-sign
// correction (e - (bit ? s : -s), sign words and scales); or with the
// pending Top-K zeroing (0 where the selection bit is set).
constexpr int kDecPlain = 0;
constexpr int kDecSign = 1;
constexpr int kDecZero = 2;

// Step ahead / error averaging.  decode_x: apply the pending server
// correction to x on read (x is never written here; the aggregate kernel
// materializes it; requires decode_e == kDecSign).  decode_e: how e is read
// (kDecPlain / kDecSign / kDecZero; `signs` holds the sign or selection
// words).  average: replace every e[k] by the mean and write it back
// (plain).  xh written when non-null (required unless average; without xh,
// x is not read and decode_x must be false).
hipError_t launch_step_ahead(const DevLayout& lay, int K, const float* x,
                             const uint64_t* srv_signs, const float* srv_scales, bool decode_x,
                             float* e, const uint64_t* signs, const float* scales, int decode_e,
                             bool average, float* xh, hipStream_t s,
                           const LaunchEvents& ev = LaunchEvents());

// The weights x_t into xh (one row): the evaluation point of local error
// feedback.  decode_x applies the pending server correction on read.
hipError_t launch_weights(const DevLayout& lay, const float* x, const uint64_t* srv_signs,
                          const float* srv_scales, bool decode_x, float* xh, hipStream_t s,
                          const LaunchEvents& ev = LaunchEvents());

// Apply pending corrections: e_out[k] = e[k] - c_k for k < K (when e_out),
// and, when e_srv_out or x_out is given, e_srv_out = e_srv - c and
// x_out = x - c (mode 1) or plain copies (mode 0; e_srv_out then receives 0).
hipError_t launch_materialize(const DevLayout& lay, int K, int mode, const float* e,
                              const uint64_t* signs, const float* scales, float* e_out,
                              const float* e_srv, const float* x, const uint64_t* srv_signs,
                              const float* srv_scales, float* e_srv_out, float* x_out,
                              hipStream_t s,
                           const LaunchEvents& ev = LaunchEvents());

// Gradient-mismatch bounds of the state (a diagnostic): out[l] = sum over
// tensor l of (e_srv + ebar)^2 and out[L + l] = (1/K) sum_k sum (e_srv + ebar
// - e^(k))^2, binary64 (mode 0: no server error).  decode_e / decode_s apply
// the pending worker / server corrections on read.  Uses the tile
// partial-sum scratch of row 0 (and the second-level scratch).
hipError_t launch_mismatch(const DevLayout& lay, int K, int mode, const float* e,
                           const uint64_t* signs, const float* scales, bool decode_e,
                           const float* e_srv, const uint64_t* srv_signs,
                           const float* srv_scales, bool decode_s, double* out, hipStream_t s,
                           const LaunchEvents& ev = LaunchEvents());

// The HBM ceiling of the compression's access pattern: c = a + b over n
// elements (measurement aid; no layout).
hipError_t launch_stream_probe(const float* a, const float* b, float* c, int64_t n,
                               hipStream_t s);

}  // namespace saef
