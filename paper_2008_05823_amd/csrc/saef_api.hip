// C ABI of the SAEF library: argument checks, the layout object and the
// order in which the kernels of one SAEF iteration are enqueued.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "saef.h"
#include "saef_internal.h"
#include "saef_topk.h"

using saef::DevLayout;
using saef::TensorInfo;
using saef::Tile;

// Kernel kinds timed by saef_profile_enable (step ahead, compression, worker
// scales, aggregation, server scales, averaging, mismatch).
constexpr int kProfileKinds = 7;

struct saef_layout {
  int device = 0;
  int32_t L = 0;
  int32_t k_max = 0;
  int64_t d_pad = 0;
  std::vector<int64_t> off, n;
  std::vector<TensorInfo> tensors;  // host copy of the tensor table (tiles per tensor)
  DevLayout dev{};
  void* mem_tiles = nullptr;
  void* mem_tensors = nullptr;
  void* mem_part = nullptr;
  void* mem_part2 = nullptr;
  void* mem_status = nullptr;
  // measurement: event pairs recorded around the kernels of saef_round
  std::vector<hipEvent_t> ev_start, ev_stop;
  std::vector<int> ev_kind;
  size_t ev_used = 0;
  uint32_t ev_mask = 0;  // kinds being timed
  int32_t ev_every = 1;  // every ev_every-th dispatch of a timed kind is stamped
  int64_t ev_seen[kProfileKinds] = {};  // dispatches of each kind since enable
};

// A Top-K plan: the kept count of every tensor and the selection scratch.
struct saef_topk {
  const saef_layout* layout = nullptr;
  std::vector<int64_t> keep;
  int64_t total_keep = 0;
  saef::TkDev dev{};
  void* mem_chunks = nullptr;
  void* mem_tens = nullptr;
  void* mem_groups = nullptr;
  void* mem_sgroups = nullptr;
  void* mem_thist = nullptr;
  void* mem_ghist = nullptr;
  void* mem_sghist = nullptr;
  void* mem_goff = nullptr;
  void* mem_sel = nullptr;
  void* mem_tile_cnt = nullptr;
  void* mem_cand = nullptr;
  void* mem_cand_off = nullptr;
  void* mem_spec = nullptr;
  // the side stream (default priority) and fork/join events of the worker
  // compression's two row groups and of the pipelined iteration end
  saef::TkStreams side{};
  saef::TkPart all{};               // every tensor
  std::vector<saef::TkPart> pipe;   // the iteration end's parts (empty: not pipelined)
};

namespace {

// ---- scratch of the allocation-free iteration (saef_round_noalloc) --------
// The tile partial sums and their second level live in this file-scope
// device array instead of the layout's buffers.  Host code never uses the
// array's name as an address: saef_layout_create looks up its device
// address once per device (hipGetSymbolAddress, with that device current)
// and saef_round_noalloc passes that address to the kernels.
constexpr size_t kScratchBytes = size_t(32) << 20;
constexpr int kMaxDevices = 64;
__device__ __align__(256) unsigned char scratch[kScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
bool g_scratch_tried[kMaxDevices] = {};

// Looks up `scratch` on the current device (device `dev`) once.
void scratch_init(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_tried[dev]) return;
  g_scratch_tried[dev] = true;
  void* p = nullptr;
  if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess) g_scratch_ptr[dev] = p;
}

void* scratch_of(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  return g_scratch_ptr[dev];
}

// Elements per work tile of a tensor of n elements: kTileElems, or more for
// very large tensors so that no tensor has more than kMaxTilesPerTensor tiles
// (bounds the number of partial sums the finalize kernel adds per tensor).
// The parts of the pipelined Top-K iteration end: runs of whole tensors in
// order (SAEF_TK_PARTS of them, fewer when there are fewer tensors; one part
// means no pipeline), cut where the running element count passes the first
// part's share of d (SAEF_TK_FIRST_PCT percent), then equal shares of the
// rest.  At resnet50 K = 8 Top-1% a 45% share (cut at 48.8% by the tensor
// boundaries) took 1.002-1.004 ms per iteration, 40% 1.005-1.007 ms, 50%
// (57%) 1.011 ms, 35% 1.053-1.057 ms.
#ifndef SAEF_TK_PARTS
#define SAEF_TK_PARTS 2
#endif
#ifndef SAEF_TK_FIRST_PCT
#define SAEF_TK_FIRST_PCT 45
#endif
std::vector<saef::TkPart> pipeline_parts(const saef_layout* layout,
                                         const std::vector<saef::TkTensor>& tens) {
  const int32_t L = layout->L;
  const int parts = std::min<int>(SAEF_TK_PARTS, L);
  std::vector<saef::TkPart> out;
  if (parts < 2) return out;
  int64_t d = 0;
  for (int32_t l = 0; l < L; ++l) d += layout->n[l];
  int32_t l0 = 0;
  int64_t cum = 0;
  for (int i = 0; i < parts; ++i) {
    int32_t l1 = l0;
    if (i == parts - 1) {
      l1 = L;
    } else {
      // the running count's target after part i (in parts of 100 * (parts - 1))
      const int64_t first = SAEF_TK_FIRST_PCT * (parts - 1);
      const int64_t target = first + (100 - SAEF_TK_FIRST_PCT) * i;
      // at least one tensor, and one left for each later part
      while (l1 < L - (parts - 1 - i) && (l1 == l0 || cum * 100 * (parts - 1) < d * target))
        cum += layout->n[l1++];
    }
    const saef::TkTensor& a = tens[l0];
    const saef::TkTensor& b = tens[l1 - 1];
    const saef::TensorInfo& ta = layout->tensors[l0];
    const saef::TensorInfo& tb = layout->tensors[l1 - 1];
    out.push_back(saef::TkPart{l0, l1, ta.first_tile, tb.first_tile + tb.ntiles, a.first_group,
                               b.first_group + b.ngroups, a.first_sgroup,
                               b.first_sgroup + b.nsgroups, a.first_chunk,
                               b.first_chunk + b.nchunks});
    l0 = l1;
  }
  return out;
}

int64_t tile_elems(int64_t n) {
  int64_t t = saef::kTileElems;
  if (n > t * saef::kMaxTilesPerTensor) {
    t = (n + saef::kMaxTilesPerTensor - 1) / saef::kMaxTilesPerTensor;
    t = (t + 63) / 64 * 64;
  }
  return t;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// [p, p + bytes) and [q, q + qbytes) overlap?
bool overlap(const void* p, size_t bytes, const void* q, size_t qbytes) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p), b = reinterpret_cast<uintptr_t>(q);
  return a < b + qbytes && b < a + bytes;
}

// Largest grid (workgroups in x) a launch may use.
constexpr int64_t kMaxGrid = 2147483647;

int check_common(const saef_layout* lay, int32_t K) {
  if (lay == nullptr) return SAEF_EINVAL;
  if (K < 1 || K > lay->k_max) return SAEF_EINVAL;
  // the per-(tile, worker) grids (tiles rounded up to whole groups of runs)
  // must fit the launch limit
  if (saef::run_padded_tiles(lay->dev.n_tiles * saef::kStepSplit) * (int64_t)K > kMaxGrid)
    return SAEF_EINVAL;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SAEF_EHIP;
  if (dev != lay->device) return SAEF_EINVAL;
  return SAEF_OK;
}

bool f32_ok(const float* p) { return p != nullptr && aligned(p, 4); }
bool u64_ok(const uint64_t* p) { return p != nullptr && aligned(p, 8); }

int hip_rc(hipError_t e) { return e == hipSuccess ? SAEF_OK : SAEF_EHIP; }

void release_events(saef_layout* l) {
  for (hipEvent_t e : l->ev_start) (void)hipEventDestroy(e);
  for (hipEvent_t e : l->ev_stop) (void)hipEventDestroy(e);
  l->ev_start.clear();
  l->ev_stop.clear();
  l->ev_kind.clear();
  l->ev_used = 0;
}

// Launches one kernel of saef_round; while the layout is being profiled and
// an event pair is free, the dispatch stamps its start and end into the pair.
template <typename F>
hipError_t timed(const saef_layout* cl, int kind, F&& launch) {
  saef_layout* l = const_cast<saef_layout*>(cl);
  saef::LaunchEvents ev;
  const bool sel = ((l->ev_mask >> kind) & 1u) != 0;
  const bool rec = sel && l->ev_used < l->ev_start.size() && l->ev_seen[kind] % l->ev_every == 0;
  if (rec) {
    ev.start = l->ev_start[l->ev_used];
    ev.stop = l->ev_stop[l->ev_used];
  }
  hipError_t err = launch(ev);
  if (err != hipSuccess) return err;
  if (sel) ++l->ev_seen[kind];
  if (rec) {
    l->ev_kind[l->ev_used] = kind;
    ++l->ev_used;
  }
  return hipSuccess;
}

void free_layout(saef_layout* l) {
  if (l == nullptr) return;
  release_events(l);
  (void)hipFree(l->mem_tiles);
  (void)hipFree(l->mem_tensors);
  (void)hipFree(l->mem_part);
  (void)hipFree(l->mem_part2);
  (void)hipFree(l->mem_status);
  delete l;
}

void free_topk(saef_topk* p) {
  if (p == nullptr) return;
  if (p->side.stream != nullptr) {
    (void)hipStreamSynchronize(p->side.stream);
    (void)hipStreamDestroy(p->side.stream);
  }
  if (p->side.fork != nullptr) (void)hipEventDestroy(p->side.fork);
  if (p->side.join != nullptr) (void)hipEventDestroy(p->side.join);
  for (void* q : {p->mem_chunks, p->mem_tens, p->mem_groups, p->mem_sgroups, p->mem_thist,
                  p->mem_ghist, p->mem_sghist, p->mem_goff, p->mem_sel, p->mem_tile_cnt,
                  p->mem_cand, p->mem_cand_off, p->mem_spec})
    (void)hipFree(q);
  delete p;
}

}  // namespace

extern "C" {

int saef_layout_create(const int64_t* off, const int64_t* n, int32_t L, int64_t d_pad,
                       int32_t k_max, saef_layout** out) {
  if (out == nullptr) return SAEF_EINVAL;
  *out = nullptr;
  if (off == nullptr || n == nullptr || L < 1 || d_pad < 64 || d_pad % 64 != 0) return SAEF_EINVAL;
  if (k_max < 1 || k_max > 4096) return SAEF_EINVAL;
  // tensors: 64-aligned, non-empty, in range, non-overlapping
  std::vector<int32_t> order(L);
  for (int32_t l = 0; l < L; ++l) {
    if (off[l] < 0 || off[l] % 64 != 0) return SAEF_EINVAL;
    if (n[l] < 1 || n[l] > saef::kMaxTensor) return SAEF_EINVAL;
    if (off[l] > d_pad - n[l]) return SAEF_EINVAL;
    order[l] = l;
  }
  std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return off[a] < off[b]; });
  for (int32_t i = 1; i < L; ++i)
    if (off[order[i - 1]] + n[order[i - 1]] > off[order[i]]) return SAEF_EINVAL;

  saef_layout* lay = new (std::nothrow) saef_layout();
  if (lay == nullptr) return SAEF_EHIP;
  if (hipGetDevice(&lay->device) != hipSuccess) {
    delete lay;
    return SAEF_EHIP;
  }
  scratch_init(lay->device);  // the allocation-free iteration's scratch on this device
  lay->L = L;
  lay->k_max = k_max;
  lay->d_pad = d_pad;
  lay->off.assign(off, off + L);
  lay->n.assign(n, n + L);

  std::vector<Tile> tiles;
  std::vector<TensorInfo> tensors(L);
  for (int32_t l = 0; l < L; ++l) {
    const int64_t te = tile_elems(n[l]);
    const int64_t nt = (n[l] + te - 1) / te;
    tensors[l] = TensorInfo{off[l], n[l], (int32_t)tiles.size(), (int32_t)nt};
    for (int64_t j = 0; j < nt; ++j) {
      const int64_t c = std::min(te, n[l] - j * te);
      tiles.push_back(Tile{off[l] + j * te, l, (int32_t)c});
    }
  }
  const size_t n_rows = (size_t)k_max + 1;
  const size_t part_bytes = n_rows * tiles.size() * 2 * sizeof(unsigned long long);
  int32_t max_tiles = 1;
  for (int32_t l = 0; l < L; ++l) max_tiles = std::max(max_tiles, tensors[l].ntiles);
  const int32_t fin_split = (max_tiles + saef::kFinChunk - 1) / saef::kFinChunk;
  const size_t part2_bytes = n_rows * L * fin_split * 2 * sizeof(unsigned long long);
  hipError_t err = hipSuccess;
  err = hipMalloc(&lay->mem_tiles, tiles.size() * sizeof(Tile));
  if (err == hipSuccess) err = hipMalloc(&lay->mem_tensors, tensors.size() * sizeof(TensorInfo));
  if (err == hipSuccess) err = hipMalloc(&lay->mem_part, part_bytes);
  if (err == hipSuccess) err = hipMalloc(&lay->mem_part2, part2_bytes);
  if (err == hipSuccess) err = hipMalloc(&lay->mem_status, sizeof(int));
  if (err == hipSuccess)
    err = hipMemcpy(lay->mem_tiles, tiles.data(), tiles.size() * sizeof(Tile),
                    hipMemcpyHostToDevice);
  if (err == hipSuccess)
    err = hipMemcpy(lay->mem_tensors, tensors.data(), tensors.size() * sizeof(TensorInfo),
                    hipMemcpyHostToDevice);
  if (err == hipSuccess) err = hipMemset(lay->mem_part, 0, part_bytes);
  if (err == hipSuccess) err = hipMemset(lay->mem_status, 0, sizeof(int));
  if (err == hipSuccess) err = hipDeviceSynchronize();
  if (err != hipSuccess) {
    free_layout(lay);
    return SAEF_EHIP;
  }
  DevLayout& d = lay->dev;
  lay->tensors = tensors;
  d.tiles = static_cast<const Tile*>(lay->mem_tiles);
  d.tensors = static_cast<const TensorInfo*>(lay->mem_tensors);
  d.part = static_cast<unsigned long long*>(lay->mem_part);
  d.part2 = static_cast<unsigned long long*>(lay->mem_part2);
  d.fin_split = fin_split;
  d.status = static_cast<int*>(lay->mem_status);
  d.n_tiles = (int64_t)tiles.size();
  d.d_pad = d_pad;
  d.L = L;
  d.k_max = k_max;
  *out = lay;
  return SAEF_OK;
}

int saef_layout_destroy(saef_layout* layout) {
  if (layout == nullptr) return SAEF_EINVAL;
  free_layout(layout);
  return SAEF_OK;
}

int saef_layout_info(const saef_layout* layout, int32_t* L, int64_t* d_pad, int32_t* k_max,
                     int64_t* n_tiles) {
  if (layout == nullptr) return SAEF_EINVAL;
  if (L) *L = layout->L;
  if (d_pad) *d_pad = layout->d_pad;
  if (k_max) *k_max = layout->k_max;
  if (n_tiles) *n_tiles = layout->dev.n_tiles;
  return SAEF_OK;
}

}  // extern "C"

namespace {

// saef_compress / saef_compress_momentum (m == nullptr: no momentum).
int compress_impl(const saef_layout* layout, int32_t K, float lr, float mu, const float* g,
                  float* m, float* e, uint64_t* signs, float* scales, hipStream_t stream) {
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (!f32_ok(g) || !f32_ok(e) || !u64_ok(signs) || !f32_ok(scales) || !std::isfinite(lr))
    return SAEF_EINVAL;
  const size_t vb = (size_t)K * layout->d_pad * sizeof(float);
  if (overlap(g, vb, e, vb)) return SAEF_EINVAL;
  if (m != nullptr && (!f32_ok(m) || overlap(m, vb, g, vb) || overlap(m, vb, e, vb)))
    return SAEF_EINVAL;
  rc = hip_rc(
      saef::launch_compress(layout->dev, K, lr, mu, g, m, e, signs, scales, false, stream));
  if (rc != SAEF_OK) return rc;
  rc = hip_rc(saef::launch_finalize(layout->dev, K, false, scales, stream));
  if (rc != SAEF_OK) return rc;
  return hip_rc(saef::launch_materialize(layout->dev, K, SAEF_MODE_SC, e, signs, scales, e,
                                         nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                         stream));
}

bool mu_ok(float mu) { return mu >= 0.0f && mu < 1.0f; }

}  // namespace

extern "C" {

int saef_compress(const saef_layout* layout, int32_t K, float lr, const float* g, float* e,
                  uint64_t* signs, float* scales, hipStream_t stream) {
  return compress_impl(layout, K, lr, 0.0f, g, nullptr, e, signs, scales, stream);
}

int saef_compress_momentum(const saef_layout* layout, int32_t K, float lr, float mu,
                           const float* g, float* m, float* e, uint64_t* signs, float* scales,
                           hipStream_t stream) {
  if (!mu_ok(mu) || m == nullptr) return SAEF_EINVAL;
  return compress_impl(layout, K, lr, mu, g, m, e, signs, scales, stream);
}

int saef_aggregate(const saef_layout* layout, int32_t K, int32_t mode, const uint64_t* signs,
                   const float* scales, float* avg, float* e_srv, uint64_t* srv_signs,
                   float* srv_scales, float* x, hipStream_t stream) {
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (mode != SAEF_MODE_SC && mode != SAEF_MODE_DC) return SAEF_EINVAL;
  if (!u64_ok(signs) || !f32_ok(scales) || !f32_ok(x)) return SAEF_EINVAL;
  if (avg != nullptr && !aligned(avg, 4)) return SAEF_EINVAL;
  if (mode == SAEF_MODE_DC && (!f32_ok(e_srv) || !u64_ok(srv_signs) || !f32_ok(srv_scales)))
    return SAEF_EINVAL;
  rc = hip_rc(saef::launch_aggregate(layout->dev, K, mode, signs, scales, avg, e_srv, srv_signs,
                                     srv_scales, x, false, stream));
  if (rc != SAEF_OK || mode == SAEF_MODE_SC) return rc;
  rc = hip_rc(saef::launch_finalize(layout->dev, K, true, srv_scales, stream));
  if (rc != SAEF_OK) return rc;
  // e_srv <- Delta - C(Delta), x <- x - C(Delta)
  return hip_rc(saef::launch_materialize(layout->dev, 0, SAEF_MODE_DC, nullptr, nullptr,
                                         nullptr, nullptr, e_srv, x, srv_signs, srv_scales,
                                         e_srv, x, stream));
}

int saef_step_ahead(const saef_layout* layout, int32_t K, const float* x, const float* e,
                    float* xh, hipStream_t stream) {
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (!f32_ok(x) || !f32_ok(e) || !f32_ok(xh)) return SAEF_EINVAL;
  const size_t vb = (size_t)K * layout->d_pad * sizeof(float);
  if (overlap(xh, vb, x, layout->d_pad * sizeof(float)) || overlap(xh, vb, e, vb))
    return SAEF_EINVAL;
  return hip_rc(saef::launch_step_ahead(layout->dev, K, x, nullptr, nullptr, false,
                                        const_cast<float*>(e), nullptr, nullptr, false, false, xh,
                                        stream));
}

int saef_error_average(const saef_layout* layout, int32_t K, float* e, hipStream_t stream) {
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (!f32_ok(e)) return SAEF_EINVAL;
  return hip_rc(saef::launch_step_ahead(layout->dev, K, nullptr, nullptr, nullptr, false, e,
                                        nullptr, nullptr, false, true, nullptr, stream));
}

}  // extern "C"

namespace {

// saef_round / saef_round_momentum (m == nullptr: no momentum).
// The first half of iteration t (Algorithm 1 up to the gradient): error
// averaging when due, the mismatch bounds when requested, then the point
// where the gradient is taken (step ahead, or the weights themselves for
// local error feedback).  The state is in saef_round's pending form.
int round_begin_impl(const saef_layout* layout, int64_t t, int64_t period, int32_t K,
                     int32_t mode, int32_t variant, float* e, const float* e_srv, const float* x,
                     float* xh, const uint64_t* signs, const float* scales,
                     const uint64_t* srv_signs, const float* srv_scales, double* mismatch,
                     hipStream_t stream, const DevLayout* dev = nullptr) {
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (t < 0 || period < 0) return SAEF_EINVAL;
  if (mode != SAEF_MODE_SC && mode != SAEF_MODE_DC) return SAEF_EINVAL;
  if (variant != SAEF_VARIANT_EF && variant != SAEF_VARIANT_SAEF) return SAEF_EINVAL;
  const bool pending = t > 0;  // at t == 0 the state is plain (Algorithm 1 initialisation)
  const bool averaging = period > 0 && (t + 1) % period == 0;
  const bool dc = mode == SAEF_MODE_DC;
  if (!f32_ok(e) || !f32_ok(x) || !f32_ok(xh)) return SAEF_EINVAL;
  if (pending && (!u64_ok(signs) || !f32_ok(scales))) return SAEF_EINVAL;
  if (pending && dc && (!u64_ok(srv_signs) || !f32_ok(srv_scales))) return SAEF_EINVAL;
  if (mismatch != nullptr && (!aligned(mismatch, 8) || (dc && !f32_ok(e_srv))))
    return SAEF_EINVAL;
  const size_t vb = (size_t)K * layout->d_pad * sizeof(float);
  const size_t xb = layout->d_pad * sizeof(float);
  const size_t hb = variant == SAEF_VARIANT_SAEF ? vb : xb;
  if (overlap(xh, hb, x, xb) || overlap(xh, hb, e, vb) ||
      (e_srv != nullptr && overlap(xh, hb, e_srv, xb)))
    return SAEF_EINVAL;
  if (mismatch != nullptr) {
    const size_t mb = 2 * (size_t)layout->L * sizeof(double);
    if (overlap(mismatch, mb, e, vb) || overlap(mismatch, mb, xh, hb) ||
        overlap(mismatch, mb, x, xb) || (e_srv != nullptr && overlap(mismatch, mb, e_srv, xb)))
      return SAEF_EINVAL;
  }
  const DevLayout& d = dev != nullptr ? *dev : layout->dev;
  if (variant == SAEF_VARIANT_SAEF) {
    // error averaging (when due) and step ahead, applying last iteration's
    // pending corrections to e and (double-way) x
    rc = hip_rc(timed(layout, averaging ? 5 : 0, [&](const saef::LaunchEvents& ev) {
      return saef::launch_step_ahead(d, K, x, srv_signs, srv_scales, pending && dc, e, signs,
                                     scales, pending, averaging, xh, stream, ev);
    }));
    if (rc != SAEF_OK) return rc;
  } else if (averaging) {
    // local error feedback with error averaging: average only
    rc = hip_rc(timed(layout, 5, [&](const saef::LaunchEvents& ev) {
      return saef::launch_step_ahead(d, K, x, srv_signs, srv_scales, false, e, signs, scales,
                                     pending, true, nullptr, stream, ev);
    }));
    if (rc != SAEF_OK) return rc;
  }
  if (mismatch != nullptr) {
    // the errors are plain after an averaging step
    rc = hip_rc(timed(layout, 6, [&](const saef::LaunchEvents& ev) {
      return saef::launch_mismatch(d, K, mode, e, signs, scales, pending && !averaging, e_srv,
                                   srv_signs, srv_scales, pending && dc, mismatch, stream, ev);
    }));
    if (rc != SAEF_OK) return rc;
  }
  if (variant == SAEF_VARIANT_SAEF) return SAEF_OK;
  // local error feedback: the gradient is taken at x_t itself (one row)
  return hip_rc(timed(layout, 0, [&](const saef::LaunchEvents& ev) {
    return saef::launch_weights(d, x, srv_signs, srv_scales, pending && dc, xh, stream, ev);
  }));
}

// The second half of iteration t: worker compression (momentum update first
// when m is given), worker scales, server aggregation and compression,
// server scales.  e is plain when the first half averaged it.
int round_end_impl(const saef_layout* layout, int64_t t, int64_t period, int32_t K, float lr,
                   float mu, int32_t mode, const float* g, float* m, float* e, float* e_srv,
                   float* x, uint64_t* signs, float* scales, uint64_t* srv_signs,
                   float* srv_scales, hipStream_t stream, const DevLayout* dev = nullptr) {
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (t < 0 || period < 0 || !std::isfinite(lr)) return SAEF_EINVAL;
  if (mode != SAEF_MODE_SC && mode != SAEF_MODE_DC) return SAEF_EINVAL;
  if (!f32_ok(g) || !f32_ok(e) || !f32_ok(x) || !u64_ok(signs) || !f32_ok(scales))
    return SAEF_EINVAL;
  if (mode == SAEF_MODE_DC && (!f32_ok(e_srv) || !u64_ok(srv_signs) || !f32_ok(srv_scales)))
    return SAEF_EINVAL;
  const size_t vb = (size_t)K * layout->d_pad * sizeof(float);
  const size_t xb = layout->d_pad * sizeof(float);
  if (overlap(g, vb, e, vb) || overlap(g, vb, x, xb) || overlap(e, vb, x, xb)) return SAEF_EINVAL;
  if (m != nullptr && (!f32_ok(m) || overlap(m, vb, g, vb) || overlap(m, vb, e, vb) ||
                       overlap(m, vb, x, xb)))
    return SAEF_EINVAL;

  const bool pending = t > 0;
  const bool averaging = period > 0 && (t + 1) % period == 0;
  const bool dc = mode == SAEF_MODE_DC;
  const DevLayout& d = dev != nullptr ? *dev : layout->dev;
  // [gradient slot: g was computed by the caller at the first half's xh]
  rc = hip_rc(timed(layout, 1, [&](const saef::LaunchEvents& ev) {
    return saef::launch_compress(d, K, lr, mu, g, m, e, signs, scales, pending && !averaging,
                                 stream, ev);
  }));
  if (rc != SAEF_OK) return rc;
  rc = hip_rc(timed(layout, 2, [&](const saef::LaunchEvents& ev) {
    return saef::launch_finalize(d, K, false, scales, stream, ev);
  }));
  if (rc != SAEF_OK) return rc;
  // server aggregation, server compression; x keeps its correction pending
  rc = hip_rc(timed(layout, 3, [&](const saef::LaunchEvents& ev) {
    return saef::launch_aggregate(d, K, mode, signs, scales, nullptr, e_srv, srv_signs,
                                  srv_scales, x, pending && dc, stream, ev);
  }));
  if (rc != SAEF_OK || !dc) return rc;
  return hip_rc(timed(layout, 4, [&](const saef::LaunchEvents& ev) {
    return saef::launch_finalize(d, K, true, srv_scales, stream, ev);
  }));
}

int round_impl(const saef_layout* layout, int64_t t, int64_t period, int32_t K, float lr,
               float mu, int32_t mode, const float* g, float* m, float* e, float* e_srv,
               float* x, float* xh, uint64_t* signs, float* scales, uint64_t* srv_signs,
               float* srv_scales, hipStream_t stream, const DevLayout* dev = nullptr) {
  // check both halves' arguments before anything is enqueued
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (t < 0 || period < 0 || !std::isfinite(lr)) return SAEF_EINVAL;
  if (mode != SAEF_MODE_SC && mode != SAEF_MODE_DC) return SAEF_EINVAL;
  if (!f32_ok(g) || !f32_ok(e) || !f32_ok(x) || !f32_ok(xh) || !u64_ok(signs) || !f32_ok(scales))
    return SAEF_EINVAL;
  if (mode == SAEF_MODE_DC && (!f32_ok(e_srv) || !u64_ok(srv_signs) || !f32_ok(srv_scales)))
    return SAEF_EINVAL;
  const size_t vb = (size_t)K * layout->d_pad * sizeof(float);
  const size_t xb = layout->d_pad * sizeof(float);
  if (overlap(xh, vb, x, xb) || overlap(xh, vb, e, vb) || overlap(xh, vb, g, vb) ||
      overlap(g, vb, e, vb) || overlap(g, vb, x, xb) || overlap(e, vb, x, xb))
    return SAEF_EINVAL;
  if (m != nullptr && (!f32_ok(m) || overlap(m, vb, g, vb) || overlap(m, vb, e, vb) ||
                       overlap(m, vb, xh, vb) || overlap(m, vb, x, xb)))
    return SAEF_EINVAL;
  rc = round_begin_impl(layout, t, period, K, mode, SAEF_VARIANT_SAEF, e, e_srv, x, xh, signs,
                        scales, srv_signs, srv_scales, nullptr, stream, dev);
  if (rc != SAEF_OK) return rc;
  return round_end_impl(layout, t, period, K, lr, mu, mode, g, m, e, e_srv, x, signs, scales,
                        srv_signs, srv_scales, stream, dev);
}

}  // namespace

extern "C" {

int saef_round(const saef_layout* layout, int64_t t, int64_t period, int32_t K, float lr,
               int32_t mode, const float* g, float* e, float* e_srv, float* x, float* xh,
               uint64_t* signs, float* scales, uint64_t* srv_signs, float* srv_scales,
               hipStream_t stream) {
  return round_impl(layout, t, period, K, lr, 0.0f, mode, g, nullptr, e, e_srv, x, xh, signs,
                    scales, srv_signs, srv_scales, stream);
}

int saef_round_noalloc(const saef_layout* layout, int64_t t, int64_t period, int32_t K, float lr,
                       int32_t mode, const float* g, float* e, float* e_srv, float* x, float* xh,
                       uint64_t* signs, float* scales, uint64_t* srv_signs, float* srv_scales,
                       hipStream_t stream) {
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  // the tile partial sums of K worker rows and the server row, and their
  // second level, must fit the static scratch
  const DevLayout& ld = layout->dev;
  const size_t rows = (size_t)K + 1;
  const size_t part_bytes = rows * (size_t)ld.n_tiles * 2 * sizeof(unsigned long long);
  const size_t part2_bytes = rows * (size_t)ld.L * (size_t)ld.fin_split * 2 *
                             sizeof(unsigned long long);
  const size_t part_pad = (part_bytes + 255) / 256 * 256;
  if (part_pad + part2_bytes > kScratchBytes) return SAEF_EINVAL;
  unsigned char* base = static_cast<unsigned char*>(scratch_of(layout->device));
  if (base == nullptr) return SAEF_EHIP;
  DevLayout d = ld;
  d.part = reinterpret_cast<unsigned long long*>(base);
  d.part2 = reinterpret_cast<unsigned long long*>(base + part_pad);
  d.k_max = K;  // the server's partial sums go to row K of the scratch
  return round_impl(layout, t, period, K, lr, 0.0f, mode, g, nullptr, e, e_srv, x, xh, signs,
                    scales, srv_signs, srv_scales, stream, &d);
}

int saef_round_momentum(const saef_layout* layout, int64_t t, int64_t period, int32_t K,
                        float lr, float mu, int32_t mode, const float* g, float* m, float* e,
                        float* e_srv, float* x, float* xh, uint64_t* signs, float* scales,
                        uint64_t* srv_signs, float* srv_scales, hipStream_t stream) {
  if (!mu_ok(mu) || m == nullptr) return SAEF_EINVAL;
  return round_impl(layout, t, period, K, lr, mu, mode, g, m, e, e_srv, x, xh, signs, scales,
                    srv_signs, srv_scales, stream);
}

int saef_round_begin(const saef_layout* layout, int64_t t, int64_t period, int32_t K,
                     int32_t mode, int32_t variant, float* e, const float* e_srv, const float* x,
                     float* xh, const uint64_t* signs, const float* scales,
                     const uint64_t* srv_signs, const float* srv_scales, double* mismatch,
                     hipStream_t stream) {
  return round_begin_impl(layout, t, period, K, mode, variant, e, e_srv, x, xh, signs, scales,
                          srv_signs, srv_scales, mismatch, stream);
}

int saef_round_end(const saef_layout* layout, int64_t t, int64_t period, int32_t K, float lr,
                   float mu, int32_t mode, const float* g, float* m, float* e, float* e_srv,
                   float* x, uint64_t* signs, float* scales, uint64_t* srv_signs,
                   float* srv_scales, hipStream_t stream) {
  if (m == nullptr ? mu != 0.0f : !mu_ok(mu)) return SAEF_EINVAL;
  return round_end_impl(layout, t, period, K, lr, mu, mode, g, m, e, e_srv, x, signs, scales,
                        srv_signs, srv_scales, stream);
}

int saef_materialize(const saef_layout* layout, int32_t K, int32_t mode, const float* e,
                     const float* e_srv, const float* x, const uint64_t* signs,
                     const float* scales, const uint64_t* srv_signs, const float* srv_scales,
                     float* e_out, float* e_srv_out, float* x_out, hipStream_t stream) {
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (mode != SAEF_MODE_SC && mode != SAEF_MODE_DC) return SAEF_EINVAL;
  if (e_out != nullptr && (!f32_ok(e_out) || !f32_ok(e) || !u64_ok(signs) || !f32_ok(scales)))
    return SAEF_EINVAL;
  if (x_out != nullptr && (!f32_ok(x_out) || !f32_ok(x))) return SAEF_EINVAL;
  if (e_srv_out != nullptr && !f32_ok(e_srv_out)) return SAEF_EINVAL;
  if (mode == SAEF_MODE_DC && (e_srv_out != nullptr || x_out != nullptr) &&
      (!u64_ok(srv_signs) || !f32_ok(srv_scales)))
    return SAEF_EINVAL;
  if (mode == SAEF_MODE_DC && e_srv_out != nullptr && !f32_ok(e_srv)) return SAEF_EINVAL;
  return hip_rc(saef::launch_materialize(layout->dev, K, mode, e, signs, scales,
                                         e_out, e_srv, x, srv_signs, srv_scales, e_srv_out,
                                         x_out, stream));
}

int saef_profile_enable(saef_layout* layout, int32_t capacity, uint32_t kind_mask,
                        int32_t every) {
  if (layout == nullptr || capacity < 0 || capacity > (1 << 20) || every < 1) return SAEF_EINVAL;
  release_events(layout);
  layout->ev_mask = kind_mask;
  layout->ev_every = every;
  for (int i = 0; i < kProfileKinds; ++i) layout->ev_seen[i] = 0;
  for (int32_t i = 0; i < capacity; ++i) {
    hipEvent_t a = nullptr, b = nullptr;
    if (hipEventCreate(&a) != hipSuccess) return SAEF_EHIP;
    if (hipEventCreate(&b) != hipSuccess) {
      (void)hipEventDestroy(a);
      return SAEF_EHIP;
    }
    layout->ev_start.push_back(a);
    layout->ev_stop.push_back(b);
    layout->ev_kind.push_back(-1);
  }
  layout->ev_used = 0;
  return SAEF_OK;
}

int saef_stream_probe(const float* a, const float* b, float* c, int64_t n,
                      hipStream_t stream) {
  if (n < 1 || n > (int64_t)saef::kTileElems * 2147483647) return SAEF_EINVAL;
  if (!f32_ok(a) || (b != nullptr && !f32_ok(b)) || !f32_ok(c)) return SAEF_EINVAL;
  const size_t vb = (size_t)n * sizeof(float);
  if (b != nullptr && (overlap(c, vb, a, vb) || overlap(c, vb, b, vb))) return SAEF_EINVAL;
  if (b == nullptr && c != a && overlap(c, vb, a, vb)) return SAEF_EINVAL;
  return hip_rc(saef::launch_stream_probe(a, b, c, n, stream));
}

int saef_profile_read(saef_layout* layout, int32_t* counts, double* total_ms) {
  if (layout == nullptr || counts == nullptr || total_ms == nullptr) return SAEF_EINVAL;
  for (int i = 0; i < kProfileKinds; ++i) {
    counts[i] = 0;
    total_ms[i] = 0.0;
  }
  for (size_t i = 0; i < layout->ev_used; ++i) {
    if (hipEventSynchronize(layout->ev_stop[i]) != hipSuccess) return SAEF_EHIP;
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, layout->ev_start[i], layout->ev_stop[i]) != hipSuccess)
      return SAEF_EHIP;
    const int k = layout->ev_kind[i];
    if (k >= 0 && k < kProfileKinds) {
      counts[k] += 1;
      total_ms[k] += ms;
    }
  }
  layout->ev_used = 0;
  return SAEF_OK;
}

int saef_topk_create(const saef_layout* layout, const int64_t* keep, saef_topk** out) {
  if (out == nullptr) return SAEF_EINVAL;
  *out = nullptr;
  if (layout == nullptr || keep == nullptr) return SAEF_EINVAL;
  if (!saef::kTkUsable) return SAEF_EINVAL;  // a build with other than 2048-element tiles
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SAEF_EHIP;
  if (dev != layout->device) return SAEF_EINVAL;
  const int32_t L = layout->L;
  for (int32_t l = 0; l < L; ++l)
    if (keep[l] < 1 || keep[l] > layout->n[l]) return SAEF_EINVAL;
  saef_topk* p = new (std::nothrow) saef_topk();
  if (p == nullptr) return SAEF_EHIP;
  p->layout = layout;
  p->keep.assign(keep, keep + L);
  // server chunks (kTkChunk elements), tile groups (kTkGroup tiles) and, for
  // tensors with more than kTkGroup groups, super-groups (kTkGroup groups)
  std::vector<saef::TkChunk> chunks;
  std::vector<saef::TkTensor> tens(L);
  std::vector<saef::TkGroup> groups, sgroups;
  for (int32_t l = 0; l < L; ++l) {
    const int64_t n = layout->n[l];
    const int64_t nc = (n + saef::kTkChunk - 1) / saef::kTkChunk;
    const int32_t first_tile = layout->tensors[l].first_tile, ntiles = layout->tensors[l].ntiles;
    const int32_t ng = (ntiles + saef::kTkGroup - 1) / saef::kTkGroup;
    const int32_t nsg = ng > saef::kTkGroup ? (ng + saef::kTkGroup - 1) / saef::kTkGroup : 0;
    tens[l] = saef::TkTensor{p->total_keep,          keep[l],
                             (int32_t)chunks.size(), (int32_t)nc,
                             (int32_t)groups.size(), ng,
                             (int32_t)sgroups.size(), nsg};
    p->total_keep += keep[l];
    for (int64_t c = 0; c < nc; ++c)
      chunks.push_back(saef::TkChunk{layout->off[l] + c * saef::kTkChunk, l,
                                     (int32_t)std::min<int64_t>(saef::kTkChunk,
                                                                n - c * saef::kTkChunk)});
    for (int32_t s = 0; s < nsg; ++s)
      sgroups.push_back(saef::TkGroup{l, (int32_t)groups.size() + s * saef::kTkGroup,
                                      std::min(saef::kTkGroup, ng - s * saef::kTkGroup), 0});
    for (int32_t g = 0; g < ng; ++g)
      groups.push_back(saef::TkGroup{l, first_tile + g * saef::kTkGroup,
                                     std::min(saef::kTkGroup, ntiles - g * saef::kTkGroup), 0});
  }
  p->all = saef::TkPart{0, L, 0, (int32_t)layout->dev.n_tiles, 0, (int32_t)groups.size(),
                        0, (int32_t)sgroups.size(), 0, (int32_t)chunks.size()};
  p->pipe = pipeline_parts(layout, tens);
  const size_t rows = (size_t)layout->k_max + 1;
  if ((int64_t)std::max(chunks.size(), groups.size()) * (int64_t)rows > kMaxGrid) {
    free_topk(p);
    return SAEF_EINVAL;
  }
  const size_t n_tiles = (size_t)layout->dev.n_tiles;
  const size_t thist_bytes = rows * n_tiles * saef::kTkHistPad * sizeof(uint16_t);
  const size_t ghist_bytes = rows * groups.size() * saef::kTkHistPad * sizeof(uint32_t);
  const size_t sghist_bytes = rows * sgroups.size() * saef::kTkHistPad * sizeof(uint32_t);
  const size_t goff_bytes = rows * groups.size() * sizeof(uint32_t);
  const size_t sel_bytes = rows * L * sizeof(saef::TkSel);
  const size_t cnt_bytes = rows * n_tiles * sizeof(uint32_t);
  // candidate slots: at most every element of a tensor (8 B each) per row
  const size_t cand_bytes = rows * (size_t)layout->d_pad * sizeof(unsigned long long);
  const size_t cand_off_bytes = rows * n_tiles * sizeof(uint32_t);
  // speculative candidate lists of the worker rows and the server row
  const size_t spec_bytes =
      (size_t)(layout->k_max + 1) * n_tiles * saef::kTkSpecCap * sizeof(unsigned long long);
  hipError_t err = hipMalloc(&p->mem_chunks, chunks.size() * sizeof(saef::TkChunk));
  if (err == hipSuccess) err = hipMalloc(&p->mem_tens, tens.size() * sizeof(saef::TkTensor));
  if (err == hipSuccess) err = hipMalloc(&p->mem_groups, groups.size() * sizeof(saef::TkGroup));
  if (err == hipSuccess && !sgroups.empty())
    err = hipMalloc(&p->mem_sgroups, sgroups.size() * sizeof(saef::TkGroup));
  if (err == hipSuccess) err = hipMalloc(&p->mem_thist, thist_bytes);
  if (err == hipSuccess) err = hipMalloc(&p->mem_ghist, ghist_bytes);
  if (err == hipSuccess && sghist_bytes) err = hipMalloc(&p->mem_sghist, sghist_bytes);
  if (err == hipSuccess) err = hipMalloc(&p->mem_goff, goff_bytes);
  if (err == hipSuccess) err = hipMalloc(&p->mem_sel, sel_bytes);
  if (err == hipSuccess) err = hipMalloc(&p->mem_tile_cnt, cnt_bytes);
  if (err == hipSuccess) err = hipMalloc(&p->mem_cand, cand_bytes);
  if (err == hipSuccess) err = hipMalloc(&p->mem_cand_off, cand_off_bytes);
  if (err == hipSuccess) err = hipMalloc(&p->mem_spec, spec_bytes);
  if (err == hipSuccess)
    err = hipMemcpy(p->mem_chunks, chunks.data(), chunks.size() * sizeof(saef::TkChunk),
                    hipMemcpyHostToDevice);
  if (err == hipSuccess)
    err = hipMemcpy(p->mem_tens, tens.data(), tens.size() * sizeof(saef::TkTensor),
                    hipMemcpyHostToDevice);
  if (err == hipSuccess)
    err = hipMemcpy(p->mem_groups, groups.data(), groups.size() * sizeof(saef::TkGroup),
                    hipMemcpyHostToDevice);
  if (err == hipSuccess && !sgroups.empty())
    err = hipMemcpy(p->mem_sgroups, sgroups.data(), sgroups.size() * sizeof(saef::TkGroup),
                    hipMemcpyHostToDevice);
  if (err == hipSuccess) {
    // zero state (the first call's window starts at the bottom of the key
    // range), and the per-tensor speculative-list switch
    std::vector<saef::TkSel> sel0(rows * L);
    for (size_t r = 0; r < rows; ++r)
      for (int32_t l = 0; l < L; ++l) {
        saef::TkSel z{};
        z.lists = p->keep[l] * saef::kTkSpecMaxShare <= layout->n[l] ? 1u : 0u;
        sel0[r * L + l] = z;
      }
    err = hipMemcpy(p->mem_sel, sel0.data(), sel_bytes, hipMemcpyHostToDevice);
  }
  if (err == hipSuccess) err = hipStreamCreateWithFlags(&p->side.stream, hipStreamNonBlocking);
  if (err == hipSuccess) err = hipEventCreateWithFlags(&p->side.fork, hipEventDisableTiming);
  if (err == hipSuccess) err = hipEventCreateWithFlags(&p->side.join, hipEventDisableTiming);
  if (err == hipSuccess) err = hipDeviceSynchronize();
  if (err != hipSuccess) {
    free_topk(p);
    return SAEF_EHIP;
  }
  saef::TkDev& d = p->dev;
  d.chunks = static_cast<const saef::TkChunk*>(p->mem_chunks);
  d.tens = static_cast<const saef::TkTensor*>(p->mem_tens);
  d.groups = static_cast<const saef::TkGroup*>(p->mem_groups);
  d.sgroups = static_cast<const saef::TkGroup*>(p->mem_sgroups);
  d.thist = static_cast<uint16_t*>(p->mem_thist);
  d.ghist = static_cast<uint32_t*>(p->mem_ghist);
  d.sghist = static_cast<uint32_t*>(p->mem_sghist);
  d.goff = static_cast<uint32_t*>(p->mem_goff);
  d.sel = static_cast<saef::TkSel*>(p->mem_sel);
  d.tile_cnt = static_cast<uint32_t*>(p->mem_tile_cnt);
  d.cand = static_cast<unsigned long long*>(p->mem_cand);
  d.cand_off = static_cast<uint32_t*>(p->mem_cand_off);
  d.spec = static_cast<unsigned long long*>(p->mem_spec);
  d.n_chunks = (int64_t)chunks.size();
  d.n_groups = (int64_t)groups.size();
  d.n_sgroups = (int64_t)sgroups.size();
  d.total_keep = p->total_keep;
  d.lists = 0;
  for (int32_t l = 0; l < L; ++l)
    if (p->keep[l] * saef::kTkSpecMaxShare <= layout->n[l]) d.lists = 1;
  *out = p;
  return SAEF_OK;
}

int saef_topk_destroy(saef_topk* plan) {
  if (plan == nullptr) return SAEF_EINVAL;
  free_topk(plan);
  return SAEF_OK;
}

int saef_topk_info(const saef_topk* plan, int64_t* total_keep) {
  if (plan == nullptr) return SAEF_EINVAL;
  if (total_keep) *total_keep = plan->total_keep;
  return SAEF_OK;
}

namespace {

// The argument checks of saef_topk_compress.
int topk_compress_check(const saef_topk* plan, int32_t K, float lr, float mu, const float* g,
                        const float* m, const float* e, const uint64_t* sel,
                        const uint32_t* rank, const float* vals) {
  if (plan == nullptr) return SAEF_EINVAL;
  const saef_layout* layout = plan->layout;
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (!std::isfinite(lr) || (m == nullptr ? mu != 0.0f : !mu_ok(mu))) return SAEF_EINVAL;
  if (!f32_ok(g) || !f32_ok(e) || !u64_ok(sel) || rank == nullptr || !aligned(rank, 4) ||
      !f32_ok(vals))
    return SAEF_EINVAL;
  const size_t vb = (size_t)K * layout->d_pad * sizeof(float);
  const size_t wb = (size_t)K * (layout->d_pad / 64) * sizeof(uint64_t);
  const size_t rb = (size_t)K * (layout->d_pad / 64) * sizeof(uint32_t);
  const size_t mb = (size_t)K * plan->total_keep * sizeof(float);
  if (overlap(g, vb, e, vb) || overlap(vals, mb, e, vb) || overlap(vals, mb, g, vb) ||
      overlap(sel, wb, e, vb) || overlap(rank, rb, e, vb) || overlap(rank, rb, vals, mb) ||
      overlap(sel, wb, vals, mb) || overlap(sel, wb, rank, rb))
    return SAEF_EINVAL;
  if (m != nullptr && (!f32_ok(m) || overlap(m, vb, g, vb) || overlap(m, vb, e, vb) ||
                       overlap(m, vb, vals, mb)))
    return SAEF_EINVAL;
  return SAEF_OK;
}

// saef_topk_compress with the pending flags of launch_topk_compress.
int topk_compress(const saef_topk* plan, int32_t K, float lr, float mu, const float* g,
                  float* m, float* e, uint64_t* sel, uint32_t* rank, float* vals, bool pend_in,
                  bool pend_out, hipStream_t stream) {
  const int rc = topk_compress_check(plan, K, lr, mu, g, m, e, sel, rank, vals);
  if (rc != SAEF_OK) return rc;
  const saef_layout* layout = plan->layout;
  return hip_rc(timed(layout, 1, [&](const saef::LaunchEvents& ev) {
    return saef::launch_topk_compress(layout->dev, plan->dev, plan->all, K, lr, mu, g, m, e, sel,
                                      rank, vals, pend_in, pend_out, stream, plan->side, ev);
  }));
}

// The argument checks of saef_topk_aggregate.
int topk_aggregate_check(const saef_topk* plan, int32_t K, int32_t mode, const uint64_t* sel,
                         const uint32_t* rank, const float* vals, const float* avg,
                         const float* e_srv, const uint64_t* srv_sel, const uint32_t* srv_rank,
                         const float* srv_vals, const float* x) {
  if (plan == nullptr) return SAEF_EINVAL;
  const saef_layout* layout = plan->layout;
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (mode != SAEF_MODE_SC && mode != SAEF_MODE_DC) return SAEF_EINVAL;
  if (!u64_ok(sel) || rank == nullptr || !aligned(rank, 4) || !f32_ok(vals) || !f32_ok(x))
    return SAEF_EINVAL;
  if (avg != nullptr && !f32_ok(avg)) return SAEF_EINVAL;
  const size_t xb = layout->d_pad * sizeof(float);
  const size_t wb1 = (layout->d_pad / 64) * sizeof(uint64_t);
  const size_t rb1 = (layout->d_pad / 64) * sizeof(uint32_t);
  const size_t mb1 = plan->total_keep * sizeof(float);
  if (mode == SAEF_MODE_DC) {
    if (!f32_ok(e_srv) || !u64_ok(srv_sel) || srv_rank == nullptr || !aligned(srv_rank, 4) ||
        !f32_ok(srv_vals))
      return SAEF_EINVAL;
    if (overlap(e_srv, xb, x, xb) || overlap(srv_vals, mb1, x, xb) ||
        overlap(srv_vals, mb1, e_srv, xb) || overlap(srv_sel, wb1, x, xb) ||
        overlap(srv_sel, wb1, e_srv, xb) || overlap(srv_rank, rb1, x, xb) ||
        overlap(srv_rank, rb1, e_srv, xb) || overlap(srv_rank, rb1, srv_vals, mb1))
      return SAEF_EINVAL;
  }
  if (avg != nullptr && (overlap(avg, xb, x, xb) || (e_srv && overlap(avg, xb, e_srv, xb))))
    return SAEF_EINVAL;
  return SAEF_OK;
}

}  // namespace

int saef_topk_compress(const saef_topk* plan, int32_t K, float lr, float mu, const float* g,
                       float* m, float* e, uint64_t* sel, uint32_t* rank, float* vals,
                       hipStream_t stream) {
  return topk_compress(plan, K, lr, mu, g, m, e, sel, rank, vals, false, false, stream);
}

int saef_topk_materialize(const saef_topk* plan, int32_t K, float* e, const uint64_t* sel,
                          hipStream_t stream) {
  if (plan == nullptr) return SAEF_EINVAL;
  const saef_layout* layout = plan->layout;
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (!f32_ok(e) || !u64_ok(sel)) return SAEF_EINVAL;
  const size_t vb = (size_t)K * layout->d_pad * sizeof(float);
  const size_t wb = (size_t)K * (layout->d_pad / 64) * sizeof(uint64_t);
  if (overlap(sel, wb, e, vb)) return SAEF_EINVAL;
  return hip_rc(saef::launch_topk_materialize(layout->dev, K, e, sel, stream));
}

int saef_topk_aggregate(const saef_topk* plan, int32_t K, int32_t mode, const uint64_t* sel,
                        const uint32_t* rank, const float* vals, float* avg, float* e_srv,
                        uint64_t* srv_sel, uint32_t* srv_rank, float* srv_vals, float* x,
                        hipStream_t stream) {
  const int rc = topk_aggregate_check(plan, K, mode, sel, rank, vals, avg, e_srv, srv_sel,
                                     srv_rank, srv_vals, x);
  if (rc != SAEF_OK) return rc;
  const saef_layout* layout = plan->layout;
  return hip_rc(timed(layout, 3, [&](const saef::LaunchEvents& ev) {
    return saef::launch_topk_aggregate(layout->dev, plan->dev, plan->all, K, mode, sel, rank,
                                       vals, avg, e_srv, srv_sel, srv_rank, srv_vals, x, stream,
                                       ev);
  }));
}

int saef_topk_round_begin(const saef_topk* plan, int64_t t, int64_t period, int32_t K,
                          int32_t mode, int32_t variant, float* e, const uint64_t* sel,
                          const float* e_srv, const float* x, float* xh, double* mismatch,
                          hipStream_t stream) {
  if (plan == nullptr) return SAEF_EINVAL;
  const saef_layout* layout = plan->layout;
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (t < 0 || period < 0) return SAEF_EINVAL;
  if (mode != SAEF_MODE_SC && mode != SAEF_MODE_DC) return SAEF_EINVAL;
  if (variant != SAEF_VARIANT_EF && variant != SAEF_VARIANT_SAEF) return SAEF_EINVAL;
  if (!f32_ok(e) || !f32_ok(x) || !f32_ok(xh)) return SAEF_EINVAL;
  // after t = 0, e holds the previous iteration's Delta with its kept
  // elements (the selection words sel) pending
  const bool pending = t > 0;
  if (pending && !u64_ok(sel)) return SAEF_EINVAL;
  if (mismatch != nullptr && (!aligned(mismatch, 8) || (mode == SAEF_MODE_DC && !f32_ok(e_srv))))
    return SAEF_EINVAL;
  const size_t vb = (size_t)K * layout->d_pad * sizeof(float);
  const size_t xb = layout->d_pad * sizeof(float);
  const size_t hb = variant == SAEF_VARIANT_SAEF ? vb : xb;
  if (overlap(xh, hb, x, xb) || overlap(xh, hb, e, vb) || overlap(e, vb, x, xb) ||
      (e_srv != nullptr && overlap(xh, hb, e_srv, xb)))
    return SAEF_EINVAL;
  if (mismatch != nullptr) {
    const size_t mb = 2 * (size_t)layout->L * sizeof(double);
    if (overlap(mismatch, mb, e, vb) || overlap(mismatch, mb, xh, hb) ||
        overlap(mismatch, mb, x, xb) || (e_srv != nullptr && overlap(mismatch, mb, e_srv, xb)))
      return SAEF_EINVAL;
  }
  if (pending) {
    const size_t wb = (size_t)K * (layout->d_pad / 64) * sizeof(uint64_t);
    if (overlap(sel, wb, e, vb) || overlap(sel, wb, xh, hb) || overlap(sel, wb, x, xb))
      return SAEF_EINVAL;
  }
  const bool averaging = period > 0 && (t + 1) % period == 0;
  const DevLayout& d = layout->dev;
  const int dec = pending ? saef::kDecZero : saef::kDecPlain;
  if (variant == SAEF_VARIANT_SAEF || averaging) {
    float* h = variant == SAEF_VARIANT_SAEF ? xh : nullptr;
    rc = hip_rc(timed(layout, averaging ? 5 : 0, [&](const saef::LaunchEvents& ev) {
      return saef::launch_step_ahead(d, K, x, nullptr, nullptr, false, e, sel, nullptr, dec,
                                     averaging, h, stream, ev);
    }));
    if (rc != SAEF_OK) return rc;
  }
  if (mismatch != nullptr && pending && !averaging) {
    // the bounds read the plain errors: set the pending elements to 0 in place
    // (the next reader's zeroing of them is then a no-op)
    rc = hip_rc(saef::launch_topk_materialize(d, K, e, sel, stream));
    if (rc != SAEF_OK) return rc;
  }
  if (mismatch != nullptr) {
    rc = hip_rc(timed(layout, 6, [&](const saef::LaunchEvents& ev) {
      return saef::launch_mismatch(d, K, mode, e, nullptr, nullptr, false, e_srv, nullptr,
                                   nullptr, false, mismatch, stream, ev);
    }));
    if (rc != SAEF_OK) return rc;
  }
  if (variant == SAEF_VARIANT_SAEF) return SAEF_OK;
  return hip_rc(timed(layout, 0, [&](const saef::LaunchEvents& ev) {
    return saef::launch_weights(d, x, nullptr, nullptr, false, xh, stream, ev);
  }));
}

int saef_topk_round_end(const saef_topk* plan, int64_t t, int64_t period, int32_t K, float lr,
                        float mu, int32_t mode, const float* g, float* m, float* e, float* e_srv,
                        float* x, uint64_t* sel, uint32_t* rank, float* vals, uint64_t* srv_sel,
                        uint32_t* srv_rank, float* srv_vals, hipStream_t stream) {
  if (plan == nullptr) return SAEF_EINVAL;
  if (t < 0 || period < 0) return SAEF_EINVAL;
  const saef_layout* layout = plan->layout;
  if (layout == nullptr || K < 1 || K > layout->k_max) return SAEF_EINVAL;
  const size_t vb = (size_t)K * layout->d_pad * sizeof(float);
  const size_t xb = layout->d_pad * sizeof(float);
  if (g != nullptr && x != nullptr && e != nullptr &&
      (overlap(g, vb, x, xb) || overlap(e, vb, x, xb)))
    return SAEF_EINVAL;
  // e is pending unless t = 0 or this iteration's averaging wrote it plain;
  // the compression leaves its own kept elements pending
  const bool averaging = period > 0 && (t + 1) % period == 0;
  const bool pend_in = t > 0 && !averaging;
  if (plan->pipe.size() >= 2 && plan->side.stream != nullptr) {
    // pipelined over the plan's parts: one timed span (kind 1) from the
    // first Delta pass to the last kernel on the caller's stream
    int rc = topk_compress_check(plan, K, lr, mu, g, m, e, sel, rank, vals);
    if (rc == SAEF_OK)
      rc = topk_aggregate_check(plan, K, mode, sel, rank, vals, nullptr, e_srv, srv_sel,
                                srv_rank, srv_vals, x);
    if (rc != SAEF_OK) return rc;
    return hip_rc(timed(layout, 1, [&](const saef::LaunchEvents& ev) {
      return saef::launch_topk_round_end(layout->dev, plan->dev, plan->pipe.data(),
                                         (int)plan->pipe.size(), K, lr, mu, mode, g, m, e, sel,
                                         rank, vals, pend_in, e_srv, srv_sel, srv_rank, srv_vals,
                                         x, stream, plan->side, ev);
    }));
  }
  int rc = topk_compress(plan, K, lr, mu, g, m, e, sel, rank, vals, pend_in, true, stream);
  if (rc != SAEF_OK) return rc;
  return saef_topk_aggregate(plan, K, mode, sel, rank, vals, nullptr, e_srv, srv_sel, srv_rank,
                             srv_vals, x, stream);
}

int saef_topk_round(const saef_topk* plan, int64_t t, int64_t period, int32_t K, float lr,
                    float mu, int32_t mode, const float* g, float* m, float* e, float* e_srv,
                    float* x, float* xh, uint64_t* sel, uint32_t* rank, float* vals,
                    uint64_t* srv_sel, uint32_t* srv_rank, float* srv_vals, hipStream_t stream) {
  if (plan == nullptr) return SAEF_EINVAL;
  const saef_layout* layout = plan->layout;
  int rc = check_common(layout, K);
  if (rc != SAEF_OK) return rc;
  if (!f32_ok(xh) || !f32_ok(g)) return SAEF_EINVAL;
  const size_t vb = (size_t)K * layout->d_pad * sizeof(float);
  if (overlap(xh, vb, g, vb)) return SAEF_EINVAL;
  rc = saef_topk_round_begin(plan, t, period, K, mode, SAEF_VARIANT_SAEF, e, sel, e_srv, x, xh,
                             nullptr, stream);
  if (rc != SAEF_OK) return rc;
  // [gradient slot: g was computed by the caller at xh]
  return saef_topk_round_end(plan, t, period, K, lr, mu, mode, g, m, e, e_srv, x, sel, rank,
                             vals, srv_sel, srv_rank, srv_vals, stream);
}

int saef_status(const saef_layout* layout, hipStream_t stream) {
  if (layout == nullptr) return SAEF_EINVAL;
  if (hipStreamSynchronize(stream) != hipSuccess) return SAEF_EHIP;
  int flag = 0;
  if (hipMemcpy(&flag, layout->dev.status, sizeof(int), hipMemcpyDeviceToHost) != hipSuccess)
    return SAEF_EHIP;
  if (flag != 0 && hipMemset(layout->dev.status, 0, sizeof(int)) != hipSuccess) return SAEF_EHIP;
  return (flag & saef::kStatusRange) ? SAEF_ERANGE : SAEF_OK;
}

}  // extern "C"
