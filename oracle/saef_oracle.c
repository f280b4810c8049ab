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
