/*
 * CPU oracle for the Step-Ahead Error Feedback (SAEF) round with the scaled
 * sign compressor.  TEST INFRASTRUCTURE ONLY: the tests, the smoke check and
 * the benchmark's CPU baseline may load it; the product library never does.
 *
 * Plain, slow, single-threaded C.  It shares no code, header, table or helper
 * with the HIP library.  Every buffer is a host pointer.  Layout convention:
 * L tensors, tensor l occupies elements [off[l], off[l] + n[l]) of a flat
 * vector of d_pad floats; off[l] is a multiple of 64; worker k's vector sits at
 * base + k * d_pad.  Sign words: bit b of word off[l]/64 + j is the sign of
 * element 64*j + b of tensor l (1 means the value >= 0, i.e. the message
 * carries +scale); bits past n[l] are 0.  Elements outside every tensor are
 * never read or written.
 *
 * Return codes: 0 ok, -1 invalid arguments, -2 value out of the exact-sum
 * range (|value| >= 2^19 or not finite) -- outputs are then unspecified.
 */
#ifndef SAEF_ORACLE_H
#define SAEF_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_ERANGE (-2)

/* Exact fixed-point L1 norm: S = sum_i floor(|v_i| * 2^80), returned as two
 * 64-bit halves.  Eq. (2) numerator. */
int oracle_l1_fixed(const float* v, int64_t n, uint64_t* s_hi, uint64_t* s_lo);

/* The scale of Eq. (2) from the exact sum: fp32(fp64(fp64(S) / n) * 2^-80). */
float oracle_scale_from_sum(uint64_t s_hi, uint64_t s_lo, int64_t n);

/* Worker side of Algorithm 1 with mu = 0: Delta = e + lr * g (one rounding),
 * message C(Delta) = (scale, sign words), e <- Delta - C(Delta). */
int oracle_compress(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                    int32_t K, float lr, const float* g, float* e,
                    uint64_t* signs, float* scales);

/* Worker side of Algorithm 1 with momentum constant mu (0 <= mu < 1):
 * m <- mu m + g (one rounding), Delta = e + lr m (one rounding), then the
 * message and error update as in oracle_compress.  m: (K, d_pad) in/out. */
int oracle_compress_momentum(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                             int32_t K, float lr, float mu, const float* g, float* m, float* e,
                             uint64_t* signs, float* scales);

/* Server side of Algorithm 1 and the re-update.  mode 1 = double-way
 * compression (server error and server message), mode 0 = single-way (the
 * average goes back uncompressed).  avg may be NULL.  In mode 0 e_srv,
 * srv_signs and srv_scales may be NULL. */
int oracle_aggregate(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                     int32_t K, int32_t mode, const uint64_t* signs, const float* scales,
                     float* avg, float* e_srv, uint64_t* srv_signs, float* srv_scales,
                     float* x);

/* Step ahead: xh[k] = x - e[k]. */
int oracle_step_ahead(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                      int32_t K, const float* x, const float* e, float* xh);

/* Error averaging: every e[k] <- (1/K) sum_k e[k]. */
int oracle_error_average(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                         int32_t K, float* e);

/* Gradient-mismatch bounds of the "Step Ahead" and "Error Averaging"
 * sections (Lipschitz constant and variance term left out), per tensor l:
 *   ef[l]   = sum_i (e_srv_i + ebar_i)^2                      local error feedback
 *   saef[l] = (1/K) sum_k sum_i (e_srv_i + ebar_i - e[k]_i)^2     step ahead
 * in binary64, ebar_i = (sum_k e[k]_i in worker order) / K.  e_srv NULL
 * means no server error (single-way compression). */
int oracle_mismatch(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                    int32_t K, const float* e, const float* e_srv, double* ef, double* saef);

/* First half of iteration t of Algorithm 1, up to the gradient: error
 * averaging when (t+1) mod period == 0 (period 0 = never), then the point
 * where the gradient is taken: variant 1 (SAEF) xh[k] = x - e[k] for every
 * worker; variant 0 (local error feedback, the EF branch) xh[0..d_pad) = x.
 * mismatch (may be NULL): 2 L doubles, oracle_mismatch of the state after
 * averaging (ef in [0, L), saef in [L, 2 L)); mode 0 ignores e_srv. */
int oracle_round_begin(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                       int64_t t, int64_t period, int32_t K, int32_t mode, int32_t variant,
                       float* e, const float* e_srv, const float* x, float* xh, double* mismatch);

/* Second half: worker compression (oracle_compress_momentum when m is not
 * NULL, else oracle_compress), then oracle_aggregate. */
int oracle_round_end(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                     int32_t K, float lr, float mu, int32_t mode, const float* g, float* m,
                     float* e, float* e_srv, float* x, uint64_t* signs, float* scales,
                     uint64_t* srv_signs, float* srv_scales);

/* One full iteration t of Algorithm 1 (SAEF branch, mu = 0) in the paper's
 * order: error averaging when (t+1) mod period == 0 (period 0 = never),
 * step ahead, [gradient g supplied], worker compression, server, re-update. */
int oracle_round(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                 int64_t t, int64_t period, int32_t K, float lr, int32_t mode,
                 const float* g, float* e, float* e_srv, float* x, float* xh,
                 uint64_t* signs, float* scales, uint64_t* srv_signs, float* srv_scales);

/* oracle_round with momentum: the worker step uses oracle_compress_momentum. */
int oracle_round_momentum(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                          int64_t t, int64_t period, int32_t K, float lr, float mu, int32_t mode,
                          const float* g, float* m, float* e, float* e_srv, float* x, float* xh,
                          uint64_t* signs, float* scales, uint64_t* srv_signs,
                          float* srv_scales);

/* Layer-wise Top-K sparsification (the paper's second compressor, kept
 * count keep[l] per tensor, 1 <= keep[l] <= n[l]): C(v) keeps the keep[l]
 * elements of largest |v| of each tensor (equal magnitudes: lower index
 * first) and zeroes the rest.  Message of a sender: sel words (sign-word
 * layout, bit set = element kept), rank words (uint32 per 64-bit word: kept
 * elements of the tensor in the words before it) and the kept values of
 * tensor l in index order at vals[voff_l ..), voff_l = keep[0] + ... +
 * keep[l-1]; total = sum keep.  Values must be finite (else -2).
 *
 * Worker side: Delta = fma(lr, g, e) (with m: m = fma(mu, m, g), Delta =
 * fma(lr, m, e); m NULL requires mu == 0), message of C(Delta), e <- Delta -
 * C(Delta).  sel, rank: (K, d_pad/64); vals: (K, total). */
int oracle_topk_compress(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                         int32_t K, float lr, float mu, const int64_t* keep, const float* g,
                         float* m, float* e, uint64_t* sel, uint32_t* rank, float* vals);

/* Server side: mean = fp32((sum_k C(Delta^(k)), binary64, worker order) / K),
 * decoded from the messages (sel, vals; rank is not needed to decode).  mode
 * 1: Delta = fp32(e_srv + mean), server message of C(Delta), e_srv <- Delta -
 * C(Delta), x <- x - C(Delta); mode 0: x <- x - mean.  avg may be NULL. */
int oracle_topk_aggregate(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                          int32_t K, int32_t mode, const int64_t* keep, const uint64_t* sel,
                          const float* vals, float* avg, float* e_srv, uint64_t* srv_sel,
                          uint32_t* srv_rank, float* srv_vals, float* x);

/* One iteration of Algorithm 1 (SAEF branch) with the Top-K compressor:
 * oracle_round_begin (SAEF), oracle_topk_compress, oracle_topk_aggregate. */
int oracle_topk_round(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                      int64_t t, int64_t period, int32_t K, float lr, float mu, int32_t mode,
                      const int64_t* keep, const float* g, float* m, float* e, float* e_srv,
                      float* x, float* xh, uint64_t* sel, uint32_t* rank, float* vals,
                      uint64_t* srv_sel, uint32_t* srv_rank, float* srv_vals);

#ifdef __cplusplus
}
#endif

#endif
