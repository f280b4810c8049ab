/*
 * CPU oracle for the SAEF round -- TEST INFRASTRUCTURE ONLY (see saef_oracle.h).
 *
 * What it follows:
 *   - Eq. (2): C(v) = (||v||_1 / d) sign(v), applied layer-wise, i.e. one
 *     scale per parameter tensor (Experiments: "all compression are performed
 *     in a layer-wise way"), so d becomes the tensor size n_l.
 *   - Algorithm 1, SAEF branch, with momentum constant mu = 0 (SAEF-SGD), and
 *     with mu > 0 through the *_momentum entry points (m <- mu m + grad,
 *     Delta^(k) = e^(k) + eta m):
 *       every p iterations the local errors are replaced by their mean,
 *       x_{t+1/2} = x_t - e_t            (step ahead)
 *       m = grad                         (mu = 0)
 *       Delta^(k) = e^(k) + x_{t+1/2} - (x_{t+1/2} - eta m) = e^(k) + eta m
 *       e^(k) <- Delta^(k) - C(Delta^(k))
 *       server: Delta = e + (1/K) sum_k C(Delta^(k));  e <- Delta - C(Delta)
 *       re-update: x <- x - C(Delta)
 *   - Single-way compression (Experiments, method notation): the server sends
 *     its average back uncompressed and keeps no error.
 *
 * Readings where the paper is silent (each one is a fixed rule here):
 *   - sign(0) = +1 for +0 and -0, so ||C(v)||_1 = ||v||_1 always holds.
 *   - ||v||_1 is summed exactly as the integer S = sum floor(|v_i| 2^80)
 *     (requires |v_i| < 2^19 and n <= 2^28); the scale is
 *     fp32( fp64( fp64(S) / n ) * 2^-80 ).
 *   - eta * m + e is formed with one rounding (fused multiply-add), and so
 *     is the momentum update mu * m + grad.
 *   - Means over the K workers are binary64 sums taken in worker order
 *     0..K-1, divided by K in binary64, then rounded once to fp32.
 *   - Delta = fp32(e_server + fp32(average)); every other fp32 result is the
 *     correctly rounded fp32 operation of its two fp32 operands.
 *
 * Built with -O1 -ffp-contract=off and no fast-math so that every float
 * expression below is exactly one IEEE operation.
 */
#include "saef_oracle.h"

#include <math.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;

/* |v| must stay below 2^19 for the 128-bit exact sum of up to 2^28 terms. */
static const float kMaxAbs = 524288.0f; /* 2^19 */
static const int64_t kMaxN = (int64_t)1 << 28;

/* ---- layout checks ------------------------------------------------------ */

static int check_layout(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad)
{
    if (L < 1 || off == NULL || n == NULL || d_pad < 1) return ORACLE_EINVAL;
    for (int32_t l = 0; l < L; ++l) {
        if (off[l] < 0 || off[l] % 64 != 0) return ORACLE_EINVAL;
        if (n[l] < 1 || n[l] > kMaxN) return ORACLE_EINVAL;
        if (off[l] + n[l] > d_pad) return ORACLE_EINVAL;
    }
    /* no two tensors may share an element (quadratic, fine for an oracle) */
    for (int32_t a = 0; a < L; ++a)
        for (int32_t b = a + 1; b < L; ++b)
            if (off[a] < off[b] + n[b] && off[b] < off[a] + n[a]) return ORACLE_EINVAL;
    return ORACLE_OK;
}

static int value_in_range(float v)
{
    /* NaN fails every comparison, so it is out of range too */
    return fabsf(v) < kMaxAbs;
}

/* ---- Eq. (2): the scaled sign compressor on one tensor -------------------- */

int oracle_l1_fixed(const float* v, int64_t n, uint64_t* s_hi, uint64_t* s_lo)
{
    u128 S = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (!value_in_range(v[i])) return ORACLE_ERANGE;
        /* |v| * 2^80 is exact in binary64 (only the exponent changes); the
         * conversion to an integer truncates, i.e. takes the floor. */
        double scaled = ldexp((double)fabsf(v[i]), 80);
        S += (u128)scaled;
    }
    *s_hi = (uint64_t)(S >> 64);
    *s_lo = (uint64_t)S;
    return ORACLE_OK;
}

float oracle_scale_from_sum(uint64_t s_hi, uint64_t s_lo, int64_t n)
{
    u128 S = ((u128)s_hi << 64) | (u128)s_lo;
    double S64 = (double)S;             /* round to nearest even */
    double mean = S64 / (double)n;       /* binary64 division */
    return (float)ldexp(mean, -80);      /* exact scaling, then round to fp32 */
}

/* sign(v) as a bit: 1 for v >= 0 (both zeros included), 0 for v < 0. */
static int sign_bit(float v)
{
    return v >= 0.0f ? 1 : 0;
}

/* One element of C(v) from the message (scale, sign bit). */
static float message_value(float scale, int bit)
{
    return bit ? scale : -scale;
}

static int get_bit(const uint64_t* words, int64_t off, int64_t i)
{
    return (int)((words[off / 64 + i / 64] >> (i % 64)) & 1u);
}

/* Compress the n values v of one tensor: writes the message (scale and the
 * ceil(n/64) sign words starting at words[off/64]) and the residual
 * err = v - C(v) (Algorithm 1, local/server error update).  err may alias v. */
static int compress_tensor(const float* v, int64_t n, int64_t off,
                           float* scale_out, uint64_t* words, float* err)
{
    uint64_t hi, lo;
    int rc = oracle_l1_fixed(v, n, &hi, &lo);
    if (rc != ORACLE_OK) return rc;
    float scale = oracle_scale_from_sum(hi, lo, n);

    int64_t nwords = (n + 63) / 64;
    for (int64_t j = 0; j < nwords; ++j) words[off / 64 + j] = 0;
    for (int64_t i = 0; i < n; ++i)
        if (sign_bit(v[i])) words[off / 64 + i / 64] |= (uint64_t)1 << (i % 64);

    for (int64_t i = 0; i < n; ++i) {
        int bit = get_bit(words, off, i);
        err[i] = v[i] - message_value(scale, bit);
    }
    *scale_out = scale;
    return ORACLE_OK;
}

/* ---- Algorithm 1: worker compression ------------------------------------ */

int oracle_compress(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                    int32_t K, float lr, const float* g, float* e,
                    uint64_t* signs, float* scales)
{
    int rc = check_layout(L, off, n, d_pad);
    if (rc != ORACLE_OK) return rc;
    if (K < 1 || g == NULL || e == NULL || signs == NULL || scales == NULL) return ORACLE_EINVAL;
    int status = ORACLE_OK;
    for (int32_t k = 0; k < K; ++k) {
        const float* gk = g + (int64_t)k * d_pad;
        float* ek = e + (int64_t)k * d_pad;
        uint64_t* wk = signs + (int64_t)k * (d_pad / 64);
        for (int32_t l = 0; l < L; ++l) {
            /* Delta^(k) = e^(k) + eta * m^(k), m = grad (mu = 0) */
            for (int64_t i = 0; i < n[l]; ++i) {
                int64_t j = off[l] + i;
                ek[j] = fmaf(lr, gk[j], ek[j]);
            }
            /* e^(k) <- Delta^(k) - C(Delta^(k)); message goes to the server */
            rc = compress_tensor(ek + off[l], n[l], off[l], &scales[(int64_t)k * L + l],
                                 wk, ek + off[l]);
            if (rc != ORACLE_OK) status = rc;
        }
    }
    return status;
}

int oracle_compress_momentum(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                             int32_t K, float lr, float mu, const float* g, float* m, float* e,
                             uint64_t* signs, float* scales)
{
    int rc = check_layout(L, off, n, d_pad);
    if (rc != ORACLE_OK) return rc;
    if (K < 1 || g == NULL || m == NULL || e == NULL || signs == NULL || scales == NULL)
        return ORACLE_EINVAL;
    if (!(mu >= 0.0f && mu < 1.0f)) return ORACLE_EINVAL;
    int status = ORACLE_OK;
    for (int32_t k = 0; k < K; ++k) {
        const float* gk = g + (int64_t)k * d_pad;
        float* mk = m + (int64_t)k * d_pad;
        float* ek = e + (int64_t)k * d_pad;
        uint64_t* wk = signs + (int64_t)k * (d_pad / 64);
        for (int32_t l = 0; l < L; ++l) {
            for (int64_t i = 0; i < n[l]; ++i) {
                int64_t j = off[l] + i;
                /* m^(k)_{t+1} = mu m^(k)_t + grad */
                mk[j] = fmaf(mu, mk[j], gk[j]);
                /* Delta^(k) = e^(k) + eta * m^(k)_{t+1} */
                ek[j] = fmaf(lr, mk[j], ek[j]);
            }
            /* e^(k) <- Delta^(k) - C(Delta^(k)); message goes to the server */
            rc = compress_tensor(ek + off[l], n[l], off[l], &scales[(int64_t)k * L + l],
                                 wk, ek + off[l]);
            if (rc != ORACLE_OK) status = rc;
        }
    }
    return status;
}

/* ---- Algorithm 1: server aggregation and worker re-update --------------- */

int oracle_aggregate(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                     int32_t K, int32_t mode, const uint64_t* signs, const float* scales,
                     float* avg, float* e_srv, uint64_t* srv_signs, float* srv_scales,
                     float* x)
{
    int rc = check_layout(L, off, n, d_pad);
    if (rc != ORACLE_OK) return rc;
    if (K < 1 || (mode != 0 && mode != 1) || signs == NULL || scales == NULL || x == NULL)
        return ORACLE_EINVAL;
    if (mode == 1 && (e_srv == NULL || srv_signs == NULL || srv_scales == NULL))
        return ORACLE_EINVAL;
    int status = ORACLE_OK;
    for (int32_t l = 0; l < L; ++l) {
        int64_t nl = n[l];
        /* (1/K) sum_k C(Delta^(k)), decoded from the K messages */
        for (int64_t i = 0; i < nl; ++i) {
            double acc = 0.0;
            for (int32_t k = 0; k < K; ++k) {
                const uint64_t* wk = signs + (int64_t)k * (d_pad / 64);
                acc += (double)message_value(scales[(int64_t)k * L + l], get_bit(wk, off[l], i));
            }
            float a = (float)(acc / (double)K);
            if (avg != NULL) avg[off[l] + i] = a;
            if (mode == 1) {
                /* Delta = e + (1/K) sum_k C(Delta^(k)), held in e_srv until compressed */
                e_srv[off[l] + i] = e_srv[off[l] + i] + a;
            } else {
                /* single-way: x <- x - (1/K) sum_k C(Delta^(k)) */
                x[off[l] + i] = x[off[l] + i] - a;
            }
        }
        if (mode == 1) {
            /* e <- Delta - C(Delta); broadcast C(Delta); x <- x - C(Delta) */
            rc = compress_tensor(e_srv + off[l], nl, off[l], &srv_scales[l], srv_signs,
                                 e_srv + off[l]);
            if (rc != ORACLE_OK) { status = rc; continue; }
            for (int64_t i = 0; i < nl; ++i) {
                int bit = get_bit(srv_signs, off[l], i);
                x[off[l] + i] = x[off[l] + i] - message_value(srv_scales[l], bit);
            }
        }
    }
    return status;
}

/* ---- Algorithm 1: step ahead and error averaging ------------------------ */

int oracle_step_ahead(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                      int32_t K, const float* x, const float* e, float* xh)
{
    int rc = check_layout(L, off, n, d_pad);
    if (rc != ORACLE_OK) return rc;
    if (K < 1 || x == NULL || e == NULL || xh == NULL) return ORACLE_EINVAL;
    for (int32_t k = 0; k < K; ++k)
        for (int32_t l = 0; l < L; ++l)
            for (int64_t i = 0; i < n[l]; ++i) {
                int64_t j = off[l] + i;
                /* x^(k)_{t+1/2} = x^(k)_t - e^(k)_t */
                xh[(int64_t)k * d_pad + j] = x[j] - e[(int64_t)k * d_pad + j];
            }
    return ORACLE_OK;
}

int oracle_error_average(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                         int32_t K, float* e)
{
    int rc = check_layout(L, off, n, d_pad);
    if (rc != ORACLE_OK) return rc;
    if (K < 1 || e == NULL) return ORACLE_EINVAL;
    for (int32_t l = 0; l < L; ++l)
        for (int64_t i = 0; i < n[l]; ++i) {
            int64_t j = off[l] + i;
            double acc = 0.0;
            for (int32_t k = 0; k < K; ++k) acc += (double)e[(int64_t)k * d_pad + j];
            float mean = (float)(acc / (double)K);
            for (int32_t k = 0; k < K; ++k) e[(int64_t)k * d_pad + j] = mean;
        }
    return ORACLE_OK;
}

/* ---- gradient-mismatch bounds ("Gradient Mismatch", "Step Ahead" and
 * "Error Averaging" sections, with the Lipschitz constant and the variance
 * term left out) ------------------------------------------------------------
 *
 * With the server error e_t and the mean of the local errors ebar, local
 * error feedback evaluates worker k's gradient at x_t while the auxiliary
 * variable sits at x_t - (e_t + ebar); step ahead evaluates it at x_t - e^(k)_t.
 * The squared distances, summed over the elements of tensor l:
 *   ef[l]   = || e_t + ebar ||^2
 *   saef[l] = (1/K) sum_k || e_t + ebar - e^(k)_t ||^2
 * all in binary64: ebar_i = (sum_k e^(k)_i, worker order) / K. */
int oracle_mismatch(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                    int32_t K, const float* e, const float* e_srv, double* ef, double* saef)
{
    int rc = check_layout(L, off, n, d_pad);
    if (rc != ORACLE_OK) return rc;
    if (K < 1 || e == NULL || ef == NULL || saef == NULL) return ORACLE_EINVAL;
    for (int32_t l = 0; l < L; ++l) {
        double a = 0.0, b = 0.0;
        for (int64_t i = 0; i < n[l]; ++i) {
            int64_t j = off[l] + i;
            double sum = 0.0;
            for (int32_t k = 0; k < K; ++k) sum += (double)e[(int64_t)k * d_pad + j];
            double ebar = sum / (double)K;
            /* single-way compression has no server error (e_srv == NULL) */
            double u = (e_srv != NULL ? (double)e_srv[j] : 0.0) + ebar;
            a += u * u;
            for (int32_t k = 0; k < K; ++k) {
                double dk = u - (double)e[(int64_t)k * d_pad + j];
                b += dk * dk;
            }
        }
        ef[l] = a;
        saef[l] = b / (double)K;
    }
    return ORACLE_OK;
}

/* ---- one iteration of Algorithm 1, in two halves around the gradient ----- */

int oracle_round_begin(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                       int64_t t, int64_t period, int32_t K, int32_t mode, int32_t variant,
                       float* e, const float* e_srv, const float* x, float* xh, double* mismatch)
{
    if (t < 0 || period < 0) return ORACLE_EINVAL;
    if (variant != 0 && variant != 1) return ORACLE_EINVAL;
    int rc = check_layout(L, off, n, d_pad);
    if (rc != ORACLE_OK) return rc;
    if (x == NULL || xh == NULL) return ORACLE_EINVAL;
    if (period > 0 && (t + 1) % period == 0) {
        rc = oracle_error_average(L, off, n, d_pad, K, e);
        if (rc != ORACLE_OK) return rc;
    }
    if (mismatch != NULL) {
        rc = oracle_mismatch(L, off, n, d_pad, K, e, mode == 1 ? e_srv : NULL, mismatch,
                             mismatch + L);
        if (rc != ORACLE_OK) return rc;
    }
    if (variant == 1) /* SAEF: one step ahead */
        return oracle_step_ahead(L, off, n, d_pad, K, x, e, xh);
    /* local error feedback: the gradient is taken at the weights themselves */
    for (int32_t l = 0; l < L; ++l)
        for (int64_t i = 0; i < n[l]; ++i) xh[off[l] + i] = x[off[l] + i];
    return ORACLE_OK;
}

int oracle_round_end(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                     int32_t K, float lr, float mu, int32_t mode, const float* g, float* m,
                     float* e, float* e_srv, float* x, uint64_t* signs, float* scales,
                     uint64_t* srv_signs, float* srv_scales)
{
    /* the gradient at xh is the caller's input g */
    int status = (m != NULL)
        ? oracle_compress_momentum(L, off, n, d_pad, K, lr, mu, g, m, e, signs, scales)
        : oracle_compress(L, off, n, d_pad, K, lr, g, e, signs, scales);
    if (status == ORACLE_EINVAL) return status;
    int rc = oracle_aggregate(L, off, n, d_pad, K, mode, signs, scales, NULL, e_srv,
                              srv_signs, srv_scales, x);
    if (rc != ORACLE_OK) status = rc;
    return status;
}

int oracle_round(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                 int64_t t, int64_t period, int32_t K, float lr, int32_t mode,
                 const float* g, float* e, float* e_srv, float* x, float* xh,
                 uint64_t* signs, float* scales, uint64_t* srv_signs, float* srv_scales)
{
    int rc = oracle_round_begin(L, off, n, d_pad, t, period, K, mode, 1, e, e_srv, x, xh, NULL);
    if (rc != ORACLE_OK) return rc;
    return oracle_round_end(L, off, n, d_pad, K, lr, 0.0f, mode, g, NULL, e, e_srv, x, signs,
                            scales, srv_signs, srv_scales);
}

int oracle_round_momentum(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                          int64_t t, int64_t period, int32_t K, float lr, float mu, int32_t mode,
                          const float* g, float* m, float* e, float* e_srv, float* x, float* xh,
                          uint64_t* signs, float* scales, uint64_t* srv_signs,
                          float* srv_scales)
{
    if (m == NULL) return ORACLE_EINVAL;
    int rc = oracle_round_begin(L, off, n, d_pad, t, period, K, mode, 1, e, e_srv, x, xh, NULL);
    if (rc != ORACLE_OK) return rc;
    return oracle_round_end(L, off, n, d_pad, K, lr, mu, mode, g, m, e, e_srv, x, signs, scales,
                            srv_signs, srv_scales);
}

/* ---- layer-wise Top-K sparsification -------------------------------------
 * The paper's second compressor (Experiments: "Top-K" with the sparsity in
 * percent, layer-wise; "How related to compression?"): C(v) keeps the k_l
 * components of largest magnitude of each tensor and sets the others to 0.
 * Equal magnitudes are ordered by index (the lower index is kept), so the
 * kept set is unique.
 *
 * Message of one sender: sel words (the sign-word layout: bit b of word
 * off[l]/64 + j set when element 64 j + b of tensor l is kept), rank words
 * (rank[w] = kept elements of the tensor in its words before w) and the kept
 * values of tensor l, in index order, at vals[voff_l .. voff_l + k_l) with
 * voff_l = k_0 + ... + k_{l-1}. */

static const float* g_topk_values; /* qsort passes no context */

static int topk_order(const void* pa, const void* pb)
{
    int64_t a = *(const int64_t*)pa, b = *(const int64_t*)pb;
    float ma = fabsf(g_topk_values[a]), mb = fabsf(g_topk_values[b]);
    if (ma > mb) return -1;
    if (ma < mb) return 1;
    return (a < b) ? -1 : (a > b) ? 1 : 0;
}

static int check_keep(int32_t L, const int64_t* n, const int64_t* keep)
{
    if (keep == NULL) return ORACLE_EINVAL;
    for (int32_t l = 0; l < L; ++l)
        if (keep[l] < 1 || keep[l] > n[l]) return ORACLE_EINVAL;
    return ORACLE_OK;
}

/* Keeps the top k of v[0..n) (flags in kept[]), all values finite. */
static int topk_select(const float* v, int64_t n, int64_t k, unsigned char* kept)
{
    int64_t* order = (int64_t*)malloc((size_t)n * sizeof(int64_t));
    if (order == NULL) return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i) order[i] = i;
    g_topk_values = v;
    qsort(order, (size_t)n, sizeof(int64_t), topk_order);
    for (int64_t i = 0; i < n; ++i) kept[i] = 0;
    for (int64_t r = 0; r < k; ++r) kept[order[r]] = 1;
    free(order);
    return ORACLE_OK;
}

/* C(v) of one tensor v[0..n) (v = a vector at base + off): the message, and
 * err[i] = v[i] - C(v)_i.  Returns ERANGE when a value is not finite. */
static int topk_tensor(const float* v, int64_t n, int64_t k, int64_t off, uint64_t* sel,
                       uint32_t* rank, float* vals, float* err, float* applied_to)
{
    for (int64_t i = 0; i < n; ++i)
        if (!isfinite(v[i])) return ORACLE_ERANGE;
    unsigned char* kept = (unsigned char*)malloc((size_t)n);
    if (kept == NULL) return ORACLE_EINVAL;
    int rc = topk_select(v, n, k, kept);
    if (rc != ORACLE_OK) {
        free(kept);
        return rc;
    }
    int64_t nw = (n + 63) / 64, count = 0;
    for (int64_t w = 0; w < nw; ++w) {
        sel[off / 64 + w] = 0;
        rank[off / 64 + w] = (uint32_t)count;
        for (int64_t b = 0; b < 64 && 64 * w + b < n; ++b) {
            int64_t i = 64 * w + b;
            if (kept[i]) {
                sel[off / 64 + w] |= (uint64_t)1 << b;
                vals[count++] = v[i];
            }
        }
    }
    for (int64_t i = 0; i < n; ++i) {
        float c = kept[i] ? v[i] : 0.0f; /* C(v)_i */
        if (applied_to != NULL) applied_to[i] = applied_to[i] - c;
        err[i] = v[i] - c;
    }
    free(kept);
    return ORACLE_OK;
}

int oracle_topk_compress(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                         int32_t K, float lr, float mu, const int64_t* keep, const float* g,
                         float* m, float* e, uint64_t* sel, uint32_t* rank, float* vals)
{
    int rc = check_layout(L, off, n, d_pad);
    if (rc != ORACLE_OK) return rc;
    if (check_keep(L, n, keep) != ORACLE_OK) return ORACLE_EINVAL;
    if (K < 1 || g == NULL || e == NULL || sel == NULL || rank == NULL || vals == NULL)
        return ORACLE_EINVAL;
    if (m == NULL ? mu != 0.0f : !(mu >= 0.0f && mu < 1.0f)) return ORACLE_EINVAL;
    int64_t total = 0;
    for (int32_t l = 0; l < L; ++l) total += keep[l];
    int status = ORACLE_OK;
    float* delta = (float*)malloc((size_t)d_pad * sizeof(float));
    if (delta == NULL) return ORACLE_EINVAL;
    for (int32_t k = 0; k < K; ++k) {
        const float* gk = g + (int64_t)k * d_pad;
        float* ek = e + (int64_t)k * d_pad;
        float* mk = m != NULL ? m + (int64_t)k * d_pad : NULL;
        int64_t voff = 0;
        for (int32_t l = 0; l < L; ++l) {
            for (int64_t i = 0; i < n[l]; ++i) {
                int64_t j = off[l] + i;
                /* Delta^(k) = e^(k) + eta m^(k), m = mu m + grad (m = grad when mu = 0) */
                if (mk != NULL) {
                    mk[j] = fmaf(mu, mk[j], gk[j]);
                    delta[j] = fmaf(lr, mk[j], ek[j]);
                } else {
                    delta[j] = fmaf(lr, gk[j], ek[j]);
                }
            }
            rc = topk_tensor(delta + off[l], n[l], keep[l], off[l],
                             sel + (int64_t)k * (d_pad / 64), rank + (int64_t)k * (d_pad / 64),
                             vals + (int64_t)k * total + voff, ek + off[l], NULL);
            if (rc == ORACLE_EINVAL) {
                free(delta);
                return rc;
            }
            if (rc != ORACLE_OK) status = rc;
            voff += keep[l];
        }
    }
    free(delta);
    return status;
}

/* C(Delta^(k)) of one message, decoded into dense[] (tensor elements only):
 * the kept elements, in index order, take the values in order. */
static void topk_decode(int32_t L, const int64_t* off, const int64_t* n, const int64_t* keep,
                        const uint64_t* sel, const float* vals, float* dense)
{
    int64_t voff = 0;
    for (int32_t l = 0; l < L; ++l) {
        int64_t next = voff;
        for (int64_t i = 0; i < n[l]; ++i)
            dense[off[l] + i] = get_bit(sel, off[l], i) ? vals[next++] : 0.0f;
        voff += keep[l];
    }
}

int oracle_topk_aggregate(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                          int32_t K, int32_t mode, const int64_t* keep, const uint64_t* sel,
                          const float* vals, float* avg, float* e_srv, uint64_t* srv_sel,
                          uint32_t* srv_rank, float* srv_vals, float* x)
{
    int rc = check_layout(L, off, n, d_pad);
    if (rc != ORACLE_OK) return rc;
    if (check_keep(L, n, keep) != ORACLE_OK) return ORACLE_EINVAL;
    if (K < 1 || sel == NULL || vals == NULL || x == NULL) return ORACLE_EINVAL;
    if (mode != 0 && mode != 1) return ORACLE_EINVAL;
    if (mode == 1 && (e_srv == NULL || srv_sel == NULL || srv_rank == NULL || srv_vals == NULL))
        return ORACLE_EINVAL;
    int64_t total = 0;
    for (int32_t l = 0; l < L; ++l) total += keep[l];
    double* acc = (double*)calloc((size_t)d_pad, sizeof(double));
    float* dense = (float*)calloc((size_t)d_pad, sizeof(float));
    float* mean = (float*)calloc((size_t)d_pad, sizeof(float));
    if (acc == NULL || dense == NULL || mean == NULL) {
        free(acc); free(dense); free(mean);
        return ORACLE_EINVAL;
    }
    /* (1/K) sum_k C(Delta^(k)): binary64 sum in worker order, then /K, then fp32 */
    for (int32_t k = 0; k < K; ++k) {
        topk_decode(L, off, n, keep, sel + (int64_t)k * (d_pad / 64), vals + (int64_t)k * total,
                    dense);
        for (int32_t l = 0; l < L; ++l)
            for (int64_t i = 0; i < n[l]; ++i) acc[off[l] + i] += (double)dense[off[l] + i];
    }
    int status = ORACLE_OK;
    for (int32_t l = 0; l < L; ++l)
        for (int64_t i = 0; i < n[l]; ++i) {
            int64_t j = off[l] + i;
            mean[j] = (float)(acc[j] / (double)K);
            if (avg != NULL) avg[j] = mean[j];
        }
    if (mode == 0) {
        /* single-way: the mean comes back uncompressed */
        for (int32_t l = 0; l < L; ++l)
            for (int64_t i = 0; i < n[l]; ++i) x[off[l] + i] = x[off[l] + i] - mean[off[l] + i];
    } else {
        int64_t voff = 0;
        for (int32_t l = 0; l < L; ++l) {
            /* server: Delta = e + mean; e <- Delta - C(Delta); x <- x - C(Delta) */
            for (int64_t i = 0; i < n[l]; ++i)
                e_srv[off[l] + i] = e_srv[off[l] + i] + mean[off[l] + i];
            rc = topk_tensor(e_srv + off[l], n[l], keep[l], off[l], srv_sel, srv_rank,
                             srv_vals + voff, e_srv + off[l], x + off[l]);
            if (rc == ORACLE_EINVAL) status = rc;
            else if (rc != ORACLE_OK && status == ORACLE_OK) status = rc;
            voff += keep[l];
        }
    }
    free(acc);
    free(dense);
    free(mean);
    return status;
}

int oracle_topk_round(int32_t L, const int64_t* off, const int64_t* n, int64_t d_pad,
                      int64_t t, int64_t period, int32_t K, float lr, float mu, int32_t mode,
                      const int64_t* keep, const float* g, float* m, float* e, float* e_srv,
                      float* x, float* xh, uint64_t* sel, uint32_t* rank, float* vals,
                      uint64_t* srv_sel, uint32_t* srv_rank, float* srv_vals)
{
    int rc = oracle_round_begin(L, off, n, d_pad, t, period, K, mode, 1, e, e_srv, x, xh, NULL);
    if (rc != ORACLE_OK) return rc;
    /* the gradient at xh is the caller's input g */
    int status = oracle_topk_compress(L, off, n, d_pad, K, lr, mu, keep, g, m, e, sel, rank,
                                      vals);
    if (status == ORACLE_EINVAL) return status;
    rc = oracle_topk_aggregate(L, off, n, d_pad, K, mode, keep, sel, vals, NULL, e_srv, srv_sel,
                               srv_rank, srv_vals, x);
    if (rc != ORACLE_OK) status = rc;
    return status;
}
