/*
 * saef.h -- C ABI of the MI355X (gfx950) library for the per-iteration hot
 * path of Step-Ahead Error Feedback (SAEF).
 *
 * The method (Xu, Huo, Huang, "Step-Ahead Error Feedback for Distributed
 * Training with Compressed Gradient", AAAI 2021), Algorithm 1:
 *   if (t+1) mod p == 0:  e^(k) <- (1/K) sum_k e^(k)          error averaging
 *   x^(k)_{t+1/2} = x_t - e^(k)                                step ahead
 *     (local error feedback, the EF branch: the gradient is taken at x_t)
 *   [gradient g^(k) computed at x^(k)_{t+1/2} by the caller]
 *   m^(k) <- mu m^(k) + g^(k)                                  (mu = 0: m = g)
 *   Delta^(k) = e^(k) + lr m^(k);  e^(k) <- Delta^(k) - C(Delta^(k))   worker
 *   Delta = e + (1/K) sum_k C(Delta^(k));  e <- Delta - C(Delta)       server
 *   x <- x - C(Delta)                                          re-update
 * with the scaled sign compressor
 *   C(v) = (||v||_1 / d) sign(v)                                   Eq. (2)
 * or layer-wise Top-K (the saef_topk_* calls), both applied per parameter
 * tensor (d = tensor size n_l).  The K workers are simulated on one GPU:
 * worker k's vectors are rows of (K, d_pad) device arrays and
 * "send"/"broadcast" are device buffers.
 *
 * ---------------------------------------------------------------- numbers
 * Every fp32 result is defined exactly, so results do not depend on the
 * launch geometry and runs are bit-reproducible:
 *   Delta^(k)   = fma(lr, g, e)                (one rounding)
 *   momentum    m = fma(mu, m, g), Delta^(k) = fma(lr, m, e)  (*_momentum)
 *   sign bit    = (v >= 0)  -- +0 and -0 give +1 (the paper leaves sign(0) open)
 *   ||v||_1     = S = sum floor(|v_i| 2^80) as an exact integer
 *                 (needs |v_i| < 2^19; n_l <= 2^28)
 *   scale       = fp32( fp64( fp64(S) / n_l ) * 2^-80 )
 *   error       = fp32(v - (bit ? scale : -scale))
 *   worker mean = fp32( (sum_{k=0..K-1} in binary64, in k order) / K )
 *   server Delta = fp32(e_srv + fp32(mean));   x, xh: one fp32 subtraction
 *
 * ---------------------------------------------------------------- layout
 * A layout describes L parameter tensors inside a flat vector of d_pad
 * floats: tensor l is elements [off[l], off[l] + n[l]).  off[l] must be a
 * multiple of 64, tensors must not overlap, 1 <= n[l] <= 2^28 and
 * off[l] + n[l] <= d_pad.  Elements outside every tensor (padding) are never
 * read or written.  Sign words: worker k's message is the uint64 row
 * signs[k][d_pad/64]; bit b of word off[l]/64 + j is the sign bit of element
 * 64 j + b of tensor l (1 = the message carries +scale); bits past n[l] are
 * written as 0.  Scales: scales[k][L] (fp32).  The server message uses
 * srv_signs[d_pad/64] and srv_scales[L].
 *
 * ---------------------------------------------------------------- conventions
 * All pointers other than the layout arrays are DEVICE pointers owned by the
 * caller, aligned to their element type (4 bytes for fp32 and uint32 arrays,
 * 8 for uint64 and binary64 ones; a misaligned or NULL required pointer is
 * SAEF_EINVAL; PyTorch allocations are 256-byte aligned).  Every call is asynchronous
 * and ordered on `stream`; nothing allocates or frees device memory except
 * saef_layout_create / saef_layout_destroy.  Calls that use the same layout
 * must not run concurrently (the layout holds the reduction scratch).
 * Return codes: SAEF_OK, SAEF_EINVAL (argument check, nothing enqueued),
 * SAEF_EHIP (a HIP call failed).  Values outside the exact-sum range (|v| >=
 * 2^19, Inf or NaN) set a sticky device flag that saef_status reports as
 * SAEF_ERANGE; the outputs of that call are then unspecified.
 */
#ifndef SAEF_H
#define SAEF_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SAEF_OK 0
#define SAEF_EINVAL (-1)
#define SAEF_ERANGE (-2)
#define SAEF_EHIP (-3)

#define SAEF_MODE_SC 0 /* single-way: the server returns the mean uncompressed */
#define SAEF_MODE_DC 1 /* double-way: Algorithm 1 (server error + server message) */

#define SAEF_VARIANT_EF 0   /* local error feedback: gradient taken at x_t (EF branch) */
#define SAEF_VARIANT_SAEF 1 /* step ahead: gradient taken at x_t - e^(k)_t (SAEF branch) */

typedef struct saef_layout saef_layout;

/* Layer-wise compression needs one scale per tensor (Experiments: all
 * compression is layer-wise).  Copies the host arrays off[L], n[L], builds
 * the tile tables on the current HIP device and allocates the reduction
 * scratch for up to k_max workers.  Synchronous.  *out receives the handle,
 * owned by the caller until saef_layout_destroy. */
int saef_layout_create(const int64_t* off, const int64_t* n, int32_t L, int64_t d_pad,
                       int32_t k_max, saef_layout** out);
int saef_layout_destroy(saef_layout* layout);

/* Worker side of Algorithm 1 (local update, Delta^(k), error update, send):
 * for every worker k < K and tensor l, Delta = fma(lr, g[k], e[k]);
 * scales[k][l] and signs[k] receive C(Delta); e[k] <- Delta - C(Delta).
 * g: (K, d_pad) read only.  e: (K, d_pad) in/out.  signs: (K, d_pad/64) out.
 * scales: (K, L) out.  1 <= K <= k_max. */
int saef_compress(const saef_layout* layout, int32_t K, float lr, const float* g, float* e,
                  uint64_t* signs, float* scales, hipStream_t stream);

/* Worker side of Algorithm 1 with momentum constant mu (0 <= mu < 1, the
 * momentum SGD update of the SAEF branch): m[k] <- fma(mu, m[k], g[k]) (one
 * rounding), then Delta = fma(lr, m[k], e[k]) and everything else as in
 * saef_compress.  m: (K, d_pad) in/out momentum buffers, zero at the start
 * of training (Algorithm 1 initialisation).  SAEF_EINVAL for mu outside
 * [0, 1) or m NULL. */
int saef_compress_momentum(const saef_layout* layout, int32_t K, float lr, float mu,
                           const float* g, float* m, float* e, uint64_t* signs, float* scales,
                           hipStream_t stream);

/* Server side of Algorithm 1 plus the re-update.  mean = (1/K) sum_k C_k
 * decoded from signs/scales.  mode SAEF_MODE_DC: Delta = e_srv + mean,
 * srv_signs/srv_scales <- C(Delta), e_srv <- Delta - C(Delta),
 * x <- x - C(Delta).  mode SAEF_MODE_SC (method notation "SC"):
 * x <- x - mean; e_srv, srv_signs, srv_scales are unused (may be NULL).
 * avg (d_pad) receives the mean when not NULL.  x, e_srv: (d_pad) in/out. */
int saef_aggregate(const saef_layout* layout, int32_t K, int32_t mode, const uint64_t* signs,
                   const float* scales, float* avg, float* e_srv, uint64_t* srv_signs,
                   float* srv_scales, float* x, hipStream_t stream);

/* Step ahead (Algorithm 1, SAEF branch): xh[k] = x - e[k] for k < K.
 * x: (d_pad), e: (K, d_pad) read only; xh: (K, d_pad) out, must not overlap
 * x or e. */
int saef_step_ahead(const saef_layout* layout, int32_t K, const float* x, const float* e,
                    float* xh, hipStream_t stream);

/* Error averaging (Algorithm 1 and the "Error Averaging" section): every
 * e[k] <- (1/K) sum_k e[k], in place.  The caller decides when it is due
 * ((t+1) mod p == 0). */
int saef_error_average(const saef_layout* layout, int32_t K, float* e, hipStream_t stream);

/* One whole iteration t of Algorithm 1 in the paper's order: error averaging
 * when period > 0 and (t+1) mod period == 0 (period 0 = never, p = infinity),
 * step ahead into xh, [the caller's gradient g, already in place], worker
 * compression, server aggregation and re-update.
 *
 * State form: to make each kernel a single streaming pass, saef_round keeps
 * the state with its last compression correction pending.  After a call,
 *   e_true[k]  = e[k]  - (bit_k ? scales[k][l] : -scales[k][l])
 *   e_srv_true = e_srv - (bit ? srv_scales[l] : -srv_scales[l])     (DC)
 *   x_true     = x     - (bit ? srv_scales[l] : -srv_scales[l])     (DC)
 * (SC: x and e_srv hold plain values).  The next saef_round applies the
 * pending corrections as it reads them; saef_materialize produces the plain
 * values.  At t == 0 the buffers are taken as plain (Algorithm 1 starts from
 * e = 0 and x_0) and signs/scales need no initial value; for t > 0 they must
 * hold what the previous call left (a plain state can be entered at t > 0 by
 * setting every scale to 0 and every sign bit to 1).
 * xh holds the plain step-ahead weights x_t - e^(k)_t of iteration t. */
int saef_round(const saef_layout* layout, int64_t t, int64_t period, int32_t K, float lr,
               int32_t mode, const float* g, float* e, float* e_srv, float* x, float* xh,
               uint64_t* signs, float* scales, uint64_t* srv_signs, float* srv_scales,
               hipStream_t stream);

/* saef_round with momentum: the worker compression step is the one of
 * saef_compress_momentum (m in/out, plain values).  Same state form and t
 * conventions as saef_round. */
int saef_round_momentum(const saef_layout* layout, int64_t t, int64_t period, int32_t K,
                        float lr, float mu, int32_t mode, const float* g, float* m, float* e,
                        float* e_srv, float* x, float* xh, uint64_t* signs, float* scales,
                        uint64_t* srv_signs, float* srv_scales, hipStream_t stream);

/* saef_round in two halves around the gradient, for callers that compute
 * the gradient at the evaluation point the first half writes (Algorithm 1,
 * both branches).  Same state form, t conventions and arguments as
 * saef_round; calling saef_round_begin(t, variant SAEF_VARIANT_SAEF) and then
 * saef_round_end(t) with the same t and period gives exactly saef_round(t).
 *
 * saef_round_begin: error averaging when (t+1) mod period == 0 (period 0 =
 * never; both variants, e is then left plain), then the evaluation point:
 *   SAEF_VARIANT_SAEF  xh[k] = x_t - e^(k)_t, xh is (K, d_pad)    step ahead
 *   SAEF_VARIANT_EF    xh    = x_t,          xh is (d_pad)        local EF
 * x and e_srv are read only.  mismatch (device, 2 L doubles, may be NULL):
 * the gradient-mismatch bounds of the "Gradient Mismatch", "Step Ahead" and
 * "Error Averaging" sections without the Lipschitz constant and the
 * variance term, per tensor l, from the state after averaging:
 *   mismatch[l]     = sum_i (e_srv_i + ebar_i)^2          (local error feedback)
 *   mismatch[L + l] = (1/K) sum_k sum_i (e_srv_i + ebar_i - e^(k)_i)^2   (step ahead)
 * in binary64 with ebar_i = (sum_k e^(k)_i, worker order) / K and e_srv = 0
 * in SAEF_MODE_SC (e_srv may then be NULL).  Each element's terms are exact
 * functions of the state; the sums over a tensor are taken in a fixed order
 * of the library's own (deterministic run to run, not the sequential order),
 * so they agree with a sequential binary64 sum to within 2 n_l K 2^-53
 * relative.  Signs/scales (and srv_* in DC) are read only when t > 0.
 *
 * saef_round_end: worker compression (with momentum m, 0 <= mu < 1, when m
 * is not NULL; m == NULL requires mu == 0), server aggregation and
 * compression, re-update.  g holds the gradients the caller computed at the
 * evaluation points of saef_round_begin(t). */
int saef_round_begin(const saef_layout* layout, int64_t t, int64_t period, int32_t K,
                     int32_t mode, int32_t variant, float* e, const float* e_srv, const float* x,
                     float* xh, const uint64_t* signs, const float* scales,
                     const uint64_t* srv_signs, const float* srv_scales, double* mismatch,
                     hipStream_t stream);
int saef_round_end(const saef_layout* layout, int64_t t, int64_t period, int32_t K, float lr,
                   float mu, int32_t mode, const float* g, float* m, float* e, float* e_srv,
                   float* x, uint64_t* signs, float* scales, uint64_t* srv_signs,
                   float* srv_scales, hipStream_t stream);

/* Plain values of a saef_round state: writes e_true to e_out (K, d_pad),
 * e_srv_true to e_srv_out and x_true to x_out (each may be NULL to skip, and
 * may equal its input to convert in place -- the state is then plain and a
 * later saef_round must be told so as described above). */
int saef_materialize(const saef_layout* layout, int32_t K, int32_t mode, const float* e,
                     const float* e_srv, const float* x, const uint64_t* signs,
                     const float* scales, const uint64_t* srv_signs, const float* srv_scales,
                     float* e_out, float* e_srv_out, float* x_out, hipStream_t stream);

/* ---------------------------------------------------------------- Top-K
 * The paper's second compressor (Experiments: Top-K sparsification with the
 * sparsity in percent, layer-wise; "How related to compression?"): C(v)
 * keeps the keep[l] elements of largest |v| of each tensor and sets the
 * others to 0.  Equal magnitudes are kept in index order (lower index
 * first), so the kept set is unique.  Values must be finite (Inf or NaN
 * sets the SAEF_ERANGE flag); no other range limit applies.
 *
 * Message of one sender (worker k: row k of each array; server: one row):
 *   sel[d_pad/64]    uint64 words in the sign-word layout, bit set = kept
 *                    (bits past a tensor's end are 0);
 *   rank[d_pad/64]   uint32 per word: kept elements of the tensor in its
 *                    words before this one;
 *   vals[total]      the kept values of tensor l, in index order, at
 *                    voff_l = keep[0] + ... + keep[l-1]; total = sum keep.
 * After saef_topk_compress and saef_topk_aggregate the state is plain: e =
 * Delta - C(Delta) is Delta with the kept elements set to 0, and x is
 * updated in place; the fused iteration (saef_topk_round, _round_end) leaves
 * the kept worker errors pending instead (below).  The tie rule, encoding and
 * state are the library's own choices; the paper gives none. */
typedef struct saef_topk saef_topk;

/* Top-K plan on a layout: keep[L] (host, 1 <= keep[l] <= n[l]) is copied;
 * the plan owns the selection scratch (tile histograms and their sums,
 * selection state, candidate slots, tile counts: about 8.3 bytes per
 * element of d_pad for each of the k_max + 1 rows; lists of candidate
 * elements, written by the worker Delta pass and the server aggregation: 2
 * bytes per element of d_pad for each of the k_max + 1 rows).  The selection state
 * keeps, per worker row and tensor, where the last call found its threshold:
 * the next call's histogram is placed there, so the first call on a plan (or
 * one after the data scale rose by more than about two binades, or fell by
 * more than about nine) takes longer; the results never depend on it.  The
 * plan also owns a second HIP stream (default priority) and two events:
 * saef_topk_compress and saef_topk_round_end give part of their work to that
 * stream and make the caller's stream wait for it before they return.
 * Calls using one plan must not run concurrently.  Synchronises the device;
 * the layout must outlive the plan. */
int saef_topk_create(const saef_layout* layout, const int64_t* keep, saef_topk** out);
int saef_topk_destroy(saef_topk* plan);
/* total = sum keep, the length of one message's value array. */
int saef_topk_info(const saef_topk* plan, int64_t* total);

/* Worker side with Top-K: Delta = fma(lr, g, e) (with m != NULL: m =
 * fma(mu, m, g), Delta = fma(lr, m, e), 0 <= mu < 1; m == NULL requires mu
 * == 0); writes the message (sel, rank: (K, d_pad/64); vals: (K, total))
 * and e <- Delta - C(Delta) in place. */
int saef_topk_compress(const saef_topk* plan, int32_t K, float lr, float mu, const float* g,
                       float* m, float* e, uint64_t* sel, uint32_t* rank, float* vals,
                       hipStream_t stream);

/* Server side with Top-K: mean = fp32((sum_k C(Delta^(k)), binary64, worker
 * order) / K) decoded from the K messages.  SAEF_MODE_DC: Delta = fp32(e_srv
 * + mean), server message (srv_sel, srv_rank, srv_vals) of C(Delta), e_srv
 * <- Delta - C(Delta), x <- x - C(Delta).  SAEF_MODE_SC: x <- x - mean
 * (e_srv and srv_* may be NULL).  avg (may be NULL) receives the mean. */
int saef_topk_aggregate(const saef_topk* plan, int32_t K, int32_t mode, const uint64_t* sel,
                        const uint32_t* rank, const float* vals, float* avg, float* e_srv,
                        uint64_t* srv_sel, uint32_t* srv_rank, float* srv_vals, float* x,
                        hipStream_t stream);

/* One iteration t of Algorithm 1 with Top-K, in two halves around the
 * gradient.  Worker state between iterations (build-defined, like the
 * pending correction of saef_round): after saef_topk_round_end the worker
 * errors e hold Delta with the kept elements not yet set to 0; the
 * selection words sel written by the same call mark them.  The next
 * iteration (t > 0) reads those elements as 0, and saef_topk_materialize
 * gives the plain errors.  sel must not be changed in between.
 * saef_topk_round_begin: error averaging when (t+1) mod period == 0 (period
 * 0 = never; the errors are then plain), then the evaluation point:
 * SAEF_VARIANT_SAEF xh[k] = x - e[k] ((K, d_pad)), SAEF_VARIANT_EF xh = x
 * ((d_pad)); mismatch (may be NULL): the 2 L bounds of saef_round_begin from
 * the state after averaging (they first set the pending elements to 0 in
 * place).  sel may be NULL at t = 0.
 * saef_topk_round_end: the worker compression of saef_topk_compress (m may be
 * NULL, then mu must be 0), leaving the kept elements pending, and
 * saef_topk_aggregate with the gradient g the caller computed at xh; t and
 * period must be those of the begin call (they tell whether e is pending).
 * With two or more tensors the plan's side stream runs part of it: the
 * tensor list is cut in two runs of whole tensors, and the first run's
 * selection, messages and server step go to the side stream (after an event
 * recorded on `stream`) while the second run's worker pass streams on
 * `stream`, which then waits for the side stream (an event), so the call
 * stays stream-ordered and capturable in a HIP graph.  The results are those
 * of saef_topk_compress then saef_topk_aggregate.  Profiled (kind 1), the
 * whole of it is one timed span, from its first kernel to its last on
 * `stream`; kind 3 is not used.
 * saef_topk_round is begin (SAEF) + end. */
int saef_topk_round_begin(const saef_topk* plan, int64_t t, int64_t period, int32_t K,
                          int32_t mode, int32_t variant, float* e, const uint64_t* sel,
                          const float* e_srv, const float* x, float* xh, double* mismatch,
                          hipStream_t stream);
int saef_topk_round_end(const saef_topk* plan, int64_t t, int64_t period, int32_t K, float lr,
                        float mu, int32_t mode, const float* g, float* m, float* e, float* e_srv,
                        float* x, uint64_t* sel, uint32_t* rank, float* vals, uint64_t* srv_sel,
                        uint32_t* srv_rank, float* srv_vals, hipStream_t stream);
int saef_topk_round(const saef_topk* plan, int64_t t, int64_t period, int32_t K, float lr,
                    float mu, int32_t mode, const float* g, float* m, float* e, float* e_srv,
                    float* x, float* xh, uint64_t* sel, uint32_t* rank, float* vals,
                    uint64_t* srv_sel, uint32_t* srv_rank, float* srv_vals, hipStream_t stream);

/* The plain worker errors after saef_topk_round / saef_topk_round_end: sets
 * to 0, in place, the elements of the K rows of e whose bit in sel (the
 * selection words of the last compression) is set.  Doing it again, or on
 * errors that are already plain, changes nothing. */
int saef_topk_materialize(const saef_topk* plan, int32_t K, float* e, const uint64_t* sel,
                          hipStream_t stream);

/* Synchronises `stream`, then returns and clears the layout's sticky device
 * flag: SAEF_ERANGE if any call since the last saef_status met a value with
 * |v| >= 2^19, Inf or NaN, SAEF_OK otherwise (SAEF_EHIP on a HIP error). */
int saef_status(const saef_layout* layout, hipStream_t stream);

/* Per-kernel timing of saef_round (and its halves), for measurement.
 * saef_profile_enable with capacity > 0 creates that many HIP event pairs;
 * every later saef_round / saef_round_begin / saef_round_end on this layout
 * then has the dispatch of each kernel whose kind bit is set in kind_mask
 * stamp its start and end into a free pair (kind 0 = step ahead, or the
 * copy of x_t for local error feedback, 1 = worker compression, 2 = worker
 * scales from the tile sums, 3 = server aggregation, 4 = server scales, 5 =
 * error averaging (with step ahead in the SAEF variant), 6 = mismatch
 * bounds), until the pairs run out; with every > 1 only the 1st, (every+1)-th,
 * ... dispatch of each timed kind since the call is stamped (a sample spread
 * over the run; every < 1 is SAEF_EINVAL).  saef_profile_read waits for the
 * recorded events and returns, per kind, the number of launches timed
 * (counts[7]) and their summed durations in milliseconds (total_ms[7]), then
 * starts over with all pairs free.  capacity 0 releases
 * the events and stops recording.  Timed dispatches cost a few microseconds
 * each, so time only the kernels of interest. */
int saef_profile_enable(saef_layout* layout, int32_t capacity, uint32_t kind_mask,
                        int32_t every);
int saef_profile_read(saef_layout* layout, int32_t* counts, double* total_ms);

/* For callers that cannot allocate device memory during the iteration
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): saef_round with the same arguments and the same results, whose
 * kernels keep their tile partial sums in a static device array of the
 * library (32 MiB per GPU, held until the process ends) instead of the
 * layout's scratch.  The call allocates nothing.  It needs (K + 1) * n_tiles
 * * 16 bytes (rounded up to 256) plus (K + 1) * L * ceil(max tiles per tensor
 * / 4096) * 16 bytes of that array; a layout and K needing more are
 * SAEF_EINVAL.  Every call on one GPU shares the array, whatever the layout:
 * calls that overlap on one GPU (other streams, other threads) race.  The
 * array's device address is looked up by saef_layout_create (SAEF_EHIP here
 * if that failed). */
int saef_round_noalloc(const saef_layout* layout, int64_t t, int64_t period, int32_t K, float lr,
                       int32_t mode, const float* g, float* e, float* e_srv, float* x, float* xh,
                       uint64_t* signs, float* scales, uint64_t* srv_signs, float* srv_scales,
                       hipStream_t stream);

/* Measurement aid (no paper operation): the HBM ceiling of the streaming
 * pattern the worker compression uses.  c[i] = a[i] + b[i] for i < n (two
 * fp32 reads and one fp32 write per element, 12 bytes), one 256-thread
 * workgroup per 2048-element tile, non-temporal accesses.  a, b, c: device
 * arrays of n floats, c must not overlap a or b (SAEF_EINVAL); n >= 1.
 * b may be NULL: then c[i] = a[i] (one read and one write, 8 bytes), and c
 * may also be a itself (in place: the pattern of the server step's error
 * and weight streams); a partial overlap of c and a is SAEF_EINVAL. */
int saef_stream_probe(const float* a, const float* b, float* c, int64_t n, hipStream_t stream);

/* Host-side query of a layout: tensor count, padded length, worker limit and
 * the number of work tiles the kernels split the tensors into.  Any output
 * pointer may be NULL.  No device work. */
int saef_layout_info(const saef_layout* layout, int32_t* L, int64_t* d_pad, int32_t* k_max,
                     int64_t* n_tiles);

#ifdef __cplusplus
}
#endif

#endif
