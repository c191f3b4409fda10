/*
 * eao.c -- Efficient-Adam oracle (plain single-threaded C).
 *
 * TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the CPU
 * baseline of the benchmark; never by the product library.  Build with
 * -ffp-contract=off so that every a*b+c below is two roundings.
 *
 * Each function names the passage of the paper it follows.  Readings of the
 * paper where it is silent are stated at the function; none of them changes
 * what Algorithms 1 and 2 compute.
 */
#include "eao.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------------------
 * Philox4x32-10 (Salmon et al., SC'11, Section 4: the Philox family).
 * One round multiplies counter words 0 and 2 by two fixed odd constants into
 * 64-bit products; the new counter is (hi1^c1^k0, lo1, hi0^c3^k1, lo0).  The
 * key is bumped by two Weyl increments (golden ratio and sqrt(3)-1 in 32-bit
 * fixed point) between rounds.  Pinned: equals a library implementation of the
 * same generator on random counters and keys, plus uniformity checks.
 * ------------------------------------------------------------------------- */
void eao_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        if (r > 0) { k0 += W0; k1 += W1; }
        uint64_t p0 = (uint64_t)M0 * c0;
        uint64_t p1 = (uint64_t)M1 * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Stochastic-rounding draws (the paper is silent on the random source; this
 * is the build's reading): counter-based, so a draw depends only on
 * (seed, t, stream, n) and never on how the work is split. */
void eao_uniforms(uint64_t seed, uint32_t t, uint32_t stream,
                  int64_t n0, int64_t len, float *u)
{
    const uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
    for (int64_t i = 0; i < len; ++i) {
        const int64_t n = n0 + i;
        const uint64_t j = (uint64_t)n >> 2;
        const uint32_t ctr[4] = { (uint32_t)j, (uint32_t)(j >> 32), t, stream };
        uint32_t r[4];
        eao_philox4x32_10(ctr, key, r);
        u[i] = (float)(r[n & 3] >> 8) * (1.0f / 16777216.0f);
    }
}

/* ---------------------------------------------------------------------------
 * Quantizer descriptions.
 * ------------------------------------------------------------------------- */

/* Example 2 needs one sign bit plus enough bits for the K-k+1 exponents and
 * one extra code for 0 (sign(0) = 0 makes Q(0) = 0). */
static int32_t pow2_bits(int32_t kmin, int32_t kmax)
{
    int32_t mags = kmax - kmin + 2;
    int32_t b = 0;
    while ((1 << b) < mags) ++b;
    return 1 + b;
}

int32_t eao_code_bits(const eao_quant *q)
{
    switch (q->kind) {
    case EAO_Q_NONE:
        return 32;
    case EAO_Q_SCALED_SIGN:
        return 1;
    case EAO_Q_STOCH_UNIFORM:
        if (q->bits == 1 || q->bits == 2 || q->bits == 4 || q->bits == 8) return q->bits;
        return -1;
    case EAO_Q_DET_UNIFORM:
        /* Example 1 with k = bits-1 has 2^(k+1)-1 levels: k+1 bits. */
        if (q->bits >= 2 && q->bits <= 8) return q->bits;
        return -1;
    case EAO_Q_POW2:
        if (q->pow2_kmin < -126 || q->pow2_kmax > 127 || q->pow2_kmin >= q->pow2_kmax) return -1;
        return pow2_bits(q->pow2_kmin, q->pow2_kmax);
    case EAO_Q_TOPK:
    case EAO_Q_RANDK:
        return q->keep >= 1 ? 1 : -1;   /* the code is the kept flag */
    default:
        return -1;
    }
}

static int is_sparse(const eao_quant *q)
{
    return q->kind == EAO_Q_TOPK || q->kind == EAO_Q_RANDK;
}

static int has_scales(const eao_quant *q)
{
    return q->kind == EAO_Q_SCALED_SIGN || q->kind == EAO_Q_STOCH_UNIFORM ||
           q->kind == EAO_Q_DET_UNIFORM;
}

int64_t eao_bucket_len(const eao_quant *q, int64_t d)
{
    if (q->bucket <= 0 || q->bucket >= d) return d;
    return q->bucket;
}

int64_t eao_num_scales(const eao_quant *q, int64_t d, int64_t len)
{
    const int64_t B = eao_bucket_len(q, d);
    if (is_sparse(q)) return (len + B - 1) / B * q->keep;
    if (!has_scales(q)) return 0;
    return (len + B - 1) / B;
}

int64_t eao_msg_words(const eao_quant *q, int64_t len)
{
    const int32_t b = eao_code_bits(q);
    if (b < 0) return -1;
    if (b == 32) return (len + 1) / 2;
    return ((len + 255) / 256) * 4 * b;
}

/* ---------------------------------------------------------------------------
 * Bucket norms.  Sums run in binary64 in element order and are rounded to
 * binary32 once; the maximum is exact.
 * ------------------------------------------------------------------------- */
static double sum_abs(const float *p, int64_t n)
{
    double s = 0.0;
    for (int64_t j = 0; j < n; ++j) s += fabs((double)p[j]);
    return s;
}

static double sum_sq(const float *p, int64_t n)
{
    double s = 0.0;
    for (int64_t j = 0; j < n; ++j) s += (double)p[j] * (double)p[j];
    return s;
}

static float max_abs(const float *p, int64_t n)
{
    float m = 0.0f;
    for (int64_t j = 0; j < n; ++j) {
        const float a = fabsf(p[j]);
        if (a > m) m = a;
    }
    return m;
}

/* Scale of one bucket of n elements: the mean absolute value (scaled sign),
 * the max-norm (stochastic uniform with EAO_SCALE_MAX; Example 1's
 * Q1(||x||_inf), Q1 being the identity on binary32) or the L2 norm
 * (stochastic uniform with EAO_SCALE_L2).  Kinds without a scale give 1. */
static float bucket_scale(const eao_quant *q, int64_t n, const float *p)
{
    switch (q->kind) {
    case EAO_Q_SCALED_SIGN:
        return (float)(sum_abs(p, n) / (double)n);
    case EAO_Q_STOCH_UNIFORM:
        return q->scale == EAO_SCALE_MAX ? max_abs(p, n) : sqrtf((float)sum_sq(p, n));
    case EAO_Q_DET_UNIFORM:
        return max_abs(p, n);
    default:
        return 1.0f;
    }
}

/* Factor applied to both x and s before x/s is formed as x * (1/s): 1 for a
 * normal scale; 2^64 (exact for both) for a scale below 2^-126, whose
 * reciprocal would overflow.  The max-norm of a bucket of subnormal values is
 * such a scale; an L2 norm never is (the square root of the smallest
 * subnormal is about 3.7e-23). */
static float prescale_of(float s)
{
    return s < 0x1p-126f ? 0x1p64f : 1.0f;
}

/* Scaled sign (a Definition 3 compressor): every element of a bucket is sent
 * as +-s with s the mean absolute value of the bucket.  Code 1 means negative;
 * a zero is sent as +s. */
static void q_scaled_sign(int64_t n, const float *p, float s, uint32_t *code, float *deq)
{
    for (int64_t j = 0; j < n; ++j) {
        code[j] = p[j] < 0.0f ? 1u : 0u;
        deq[j] = code[j] ? -s : s;
    }
}

/* Level c of a b-bit uniform grid on [-1, 1]: (2c - L)/L with L = 2^b - 1,
 * rounded once to binary32. */
static float uniform_level(uint32_t c, uint32_t L)
{
    return (float)(2 * (int32_t)c - (int32_t)L) / (float)L;
}

/* Stochastic uniform quantizer: p/s is mapped onto the grid of 2^b levels on
 * [-1, 1] and rounded up with probability equal to its distance above the
 * lower level, so that E[Q(p)] = p.  s is the bucket's max-norm or L2-norm;
 * both bound |p|, so p/s lies in [-1, 1].  A bucket whose scale is zero or not
 * finite is sent as all zeros. */
static void q_stoch_uniform(const eao_quant *q, int64_t n, const float *p, const float *u, float s,
                            uint32_t *code, float *deq)
{
    const uint32_t L = (1u << q->bits) - 1u;
    if (!(s > 0.0f) || isinf(s)) {
        for (int64_t j = 0; j < n; ++j) { code[j] = 0; deq[j] = 0.0f; }
        return;
    }
    const float f = prescale_of(s);
    const float inv = 1.0f / (s * f);
    const float h = (float)L * 0.5f;
    for (int64_t j = 0; j < n; ++j) {
        float y = ((p[j] * f) * inv + 1.0f) * h;
        if (y < 0.0f) y = 0.0f;
        if (y > (float)L) y = (float)L;
        const float lo = floorf(y);
        const float fr = y - lo;
        uint32_t c = (uint32_t)lo + (u[j] < fr ? 1u : 0u);
        if (c > L) c = L;
        code[j] = c;
        deq[j] = s * uniform_level(c, L);
    }
}

/* Example 1: Q(x) = Q1(|x|_inf) * Q2(x / Q1(|x|_inf)), Q2 rounding each
 * coordinate to the nearest of i/(2^k-1), i = -(2^k-1)..(2^k-1); Q(x) = 0 when
 * the max-norm is 0.  Applied per bucket.  Q1 is the identity because the
 * max-norm of binary32 values is a binary32 value.  x/s is formed as x*(1/s)
 * (after prescale_of).  A coordinate exactly half-way between two levels goes
 * to the one nearer 0 (the flooring direction of Remark 1).
 * Code c = i + (2^k - 1). */
static void q_det_uniform(const eao_quant *q, int64_t n, const float *p, float s,
                          uint32_t *code, float *deq)
{
    const int32_t k = q->bits - 1;
    const int32_t L = (1 << k) - 1;
    if (!(s > 0.0f) || isinf(s)) {
        for (int64_t j = 0; j < n; ++j) { code[j] = (uint32_t)L; deq[j] = 0.0f; }
        return;
    }
    const float f = prescale_of(s);
    const float inv = 1.0f / (s * f);
    for (int64_t j = 0; j < n; ++j) {
        float a = (fabsf(p[j]) * f) * inv * (float)L;
        if (a > (float)L) a = (float)L;
        int32_t i = (int32_t)floorf(a);
        if (a - (float)i > 0.5f) i += 1;
        const int32_t si = p[j] < 0.0f ? -i : i;
        code[j] = (uint32_t)(si + L);
        deq[j] = s * ((float)si / (float)L);
    }
}

/* Example 2: Q(x) = sign(x) * argmin over y in {2^kmin..2^kmax} of ||x|-y|,
 * coordinate-wise, no scale.  sign(0) = 0, so a zero is sent as the extra code
 * (kmax-kmin+1) and decodes to 0.  The nearest power of two to |x| in
 * [2^e, 2^(e+1)) is 2^(e+1) exactly when the mantissa exceeds 1.5; a tie
 * (mantissa 1.5) goes to the smaller power.  Values below 2^kmin map to
 * 2^kmin and values above 2^kmax to 2^kmax.  Code = sign<<(b-1) | (j - kmin). */
static void q_pow2(const eao_quant *q, int64_t n, const float *p, uint32_t *code, float *deq)
{
    const int32_t kmin = q->pow2_kmin, kmax = q->pow2_kmax;
    const int32_t b = pow2_bits(kmin, kmax);
    const uint32_t zero_code = (uint32_t)(kmax - kmin + 1);
    for (int64_t j = 0; j < n; ++j) {
        const float x = p[j];
        if (x == 0.0f) { code[j] = zero_code; deq[j] = 0.0f; continue; }
        uint32_t bits;
        memcpy(&bits, &x, sizeof bits);
        const uint32_t neg = bits >> 31;
        const int32_t ex = (int32_t)((bits >> 23) & 0xFFu);
        const uint32_t frac = bits & 0x7FFFFFu;
        int32_t e;
        if (ex == 0) e = -127;                     /* subnormal: below 2^-126 <= 2^kmin */
        else e = ex - 127 + (frac > 0x400000u ? 1 : 0);
        if (e < kmin) e = kmin;
        if (e > kmax) e = kmax;
        code[j] = (neg << (b - 1)) | (uint32_t)(e - kmin);
        const float mag = ldexpf(1.0f, e);
        deq[j] = neg ? -mag : mag;
    }
}

/* Definition 3 sparsifiers (TOPK, RANDK; see eao.h for the ranking).  The
 * ranking is a sort of (key, index) pairs, larger key first, lower index
 * first among equal keys; the first min(keep, n) are kept. */
typedef struct {
    uint32_t key;
    int64_t idx;
} eao_ranked;

static int by_rank(const void *a, const void *b)
{
    const eao_ranked *x = (const eao_ranked *)a, *y = (const eao_ranked *)b;
    if (x->key != y->key) return x->key > y->key ? -1 : 1;
    return x->idx < y->idx ? -1 : (x->idx > y->idx ? 1 : 0);
}

static uint32_t magnitude_key(float x)
{
    uint32_t b;
    memcpy(&b, &x, sizeof b);
    return b & 0x7FFFFFFFu;
}

static int q_sparse(const eao_quant *q, int64_t n, const float *p, const float *u,
                    uint32_t *code, float *deq, float *vals)
{
    eao_ranked *r = (eao_ranked *)malloc((size_t)n * sizeof(eao_ranked));
    if (!r) return -1;
    for (int64_t j = 0; j < n; ++j) {
        /* u = w * 2^-24 for a 24-bit integer w, so u * 2^24 is w exactly. */
        r[j].key = q->kind == EAO_Q_TOPK ? magnitude_key(p[j]) : (uint32_t)(u[j] * 16777216.0f);
        r[j].idx = j;
    }
    qsort(r, (size_t)n, sizeof(eao_ranked), by_rank);
    const int64_t k = q->keep < n ? q->keep : n;
    for (int64_t j = 0; j < n; ++j) code[j] = 0;
    for (int64_t i = 0; i < k; ++i) code[r[i].idx] = 1;
    free(r);
    int64_t slot = 0;
    for (int64_t j = 0; j < n; ++j) {
        if (code[j]) {
            deq[j] = p[j];
            vals[slot++] = p[j];
        } else {
            deq[j] = 0.0f;
        }
    }
    for (; slot < q->keep; ++slot) vals[slot] = 0.0f;
    return 0;
}

/* Full-precision communication ("Ours_full" in Table 2): the code is the
 * binary32 bit pattern itself. */
static void q_none(int64_t n, const float *p, uint32_t *code, float *deq)
{
    for (int64_t j = 0; j < n; ++j) {
        memcpy(&code[j], &p[j], sizeof(uint32_t));
        deq[j] = p[j];
    }
}

/* Codes and dequantized values of one bucket of n elements under scale s. */
static void code_bucket(const eao_quant *q, int64_t n, const float *p, const float *u, float s,
                        uint32_t *code, float *deq)
{
    switch (q->kind) {
    case EAO_Q_SCALED_SIGN:
        q_scaled_sign(n, p, s, code, deq);
        break;
    case EAO_Q_STOCH_UNIFORM:
        q_stoch_uniform(q, n, p, u, s, code, deq);
        break;
    default:
        q_det_uniform(q, n, p, s, code, deq);
        break;
    }
}

static int valid_for_quantize(const eao_quant *q, const float *u)
{
    if (eao_code_bits(q) < 0) return 0;
    if (q->kind == EAO_Q_STOCH_UNIFORM && q->scale != EAO_SCALE_L2 && q->scale != EAO_SCALE_MAX)
        return 0;
    if ((q->kind == EAO_Q_STOCH_UNIFORM || q->kind == EAO_Q_RANDK) && u == NULL) return 0;
    return 1;
}

int eao_quantize(const eao_quant *q, int64_t d, int64_t len, const float *p,
                 const float *u, uint32_t *code, float *deq, float *scales)
{
    if (!valid_for_quantize(q, u)) return -1;
    if (q->kind == EAO_Q_NONE) { q_none(len, p, code, deq); return 0; }
    if (q->kind == EAO_Q_POW2) { q_pow2(q, len, p, code, deq); return 0; }
    const int64_t B = eao_bucket_len(q, d);
    for (int64_t b0 = 0, bi = 0; b0 < len; b0 += B, ++bi) {
        const int64_t n = (len - b0 < B) ? (len - b0) : B;
        if (is_sparse(q)) {
            if (q_sparse(q, n, p + b0, u ? u + b0 : NULL, code + b0, deq + b0, scales + bi * q->keep))
                return -1;
            continue;
        }
        scales[bi] = bucket_scale(q, n, p + b0);
        code_bucket(q, n, p + b0, u ? u + b0 : NULL, scales[bi], code + b0, deq + b0);
    }
    return 0;
}

int eao_quantize_bucket(const eao_quant *q, int64_t n, const float *p, const float *u, float s,
                        uint32_t *code, float *deq)
{
    if (!valid_for_quantize(q, u) || !has_scales(q) || n < 1) return -1;
    code_bucket(q, n, p, u, s, code, deq);
    return 0;
}

int eao_dequantize(const eao_quant *q, int64_t d, int64_t len, const uint32_t *code,
                   const float *scales, float *deq)
{
    const int32_t b = eao_code_bits(q);
    if (b < 0) return -1;
    const int64_t B = eao_bucket_len(q, d);
    if (is_sparse(q)) {
        /* Kept elements take the bucket's values in index order. */
        for (int64_t b0 = 0, bi = 0; b0 < len; b0 += B, ++bi) {
            const int64_t n = (len - b0 < B) ? (len - b0) : B;
            int64_t slot = 0;
            for (int64_t j = 0; j < n; ++j)
                deq[b0 + j] = code[b0 + j] ? scales[bi * q->keep + slot++] : 0.0f;
        }
        return 0;
    }
    for (int64_t j = 0; j < len; ++j) {
        const uint32_t c = code[j];
        switch (q->kind) {
        case EAO_Q_NONE:
            memcpy(&deq[j], &c, sizeof(float));
            break;
        case EAO_Q_SCALED_SIGN: {
            const float s = scales[j / B];
            deq[j] = c ? -s : s;
            break;
        }
        case EAO_Q_STOCH_UNIFORM: {
            const float s = scales[j / B];
            const uint32_t L = (1u << q->bits) - 1u;
            deq[j] = (!(s > 0.0f) || isinf(s)) ? 0.0f : s * uniform_level(c, L);
            break;
        }
        case EAO_Q_DET_UNIFORM: {
            const float s = scales[j / B];
            const int32_t L = (1 << (q->bits - 1)) - 1;
            const int32_t si = (int32_t)c - L;
            deq[j] = (!(s > 0.0f) || isinf(s)) ? 0.0f : s * ((float)si / (float)L);
            break;
        }
        case EAO_Q_POW2: {
            const uint32_t zero_code = (uint32_t)(q->pow2_kmax - q->pow2_kmin + 1);
            const uint32_t mag = c & ((1u << (b - 1)) - 1u);
            if (mag == zero_code) { deq[j] = 0.0f; break; }
            const float v = ldexpf(1.0f, (int32_t)mag + q->pow2_kmin);
            deq[j] = (c >> (b - 1)) ? -v : v;
            break;
        }
        default:
            return -1;
        }
    }
    return 0;
}

/* ---------------------------------------------------------------------------
 * Message layout (the paper gives no encoding; this is the build's format).
 * ------------------------------------------------------------------------- */
void eao_pack(int32_t bits, int64_t len, const uint32_t *code, uint64_t *words)
{
    if (bits == 32) {
        memset(words, 0, (size_t)((len + 1) / 2) * sizeof(uint64_t));
        for (int64_t n = 0; n < len; ++n)
            words[n >> 1] |= (uint64_t)code[n] << (32 * (n & 1));
        return;
    }
    memset(words, 0, (size_t)(((len + 255) / 256) * 4 * bits) * sizeof(uint64_t));
    for (int64_t n = 0; n < len; ++n) {
        const int64_t c = n >> 8;
        const int64_t l = (n >> 2) & 63;
        const int64_t k = n & 3;
        for (int32_t p = 0; p < bits; ++p)
            if ((code[n] >> p) & 1u)
                words[(4 * c + k) * bits + p] |= (uint64_t)1 << l;
    }
}

void eao_unpack(int32_t bits, int64_t len, const uint64_t *words, uint32_t *code)
{
    for (int64_t n = 0; n < len; ++n) {
        if (bits == 32) {
            code[n] = (uint32_t)(words[n >> 1] >> (32 * (n & 1)));
            continue;
        }
        const int64_t c = n >> 8;
        const int64_t l = (n >> 2) & 63;
        const int64_t k = n & 3;
        uint32_t v = 0;
        for (int32_t p = 0; p < bits; ++p)
            v |= (uint32_t)((words[(4 * c + k) * bits + p] >> l) & 1u) << p;
        code[n] = v;
    }
}

/* ---------------------------------------------------------------------------
 * Adam (Algorithm 2, moment lines and the update alpha m / sqrt(v)); no bias
 * correction, v starts at eps and eps is not added in the denominator.
 * ------------------------------------------------------------------------- */
void eao_adam_moments(float beta1, float beta2, float *m, float *v, float g)
{
    const float omb1 = 1.0f - beta1;
    const float omb2 = 1.0f - beta2;
    *v = beta2 * *v + omb2 * (g * g);
    *m = beta1 * *m + omb1 * g;
}

float eao_adam_update(float lr, float m, float v)
{
    if (!(v > 0.0f)) return 0.0f;
    return lr * (m / sqrtf(v));
}

/* ---------------------------------------------------------------------------
 * One round.  ADAM_AT_WORKER follows Algorithm 2 (each worker updates its own
 * moments, sends Q_w(alpha m/sqrt(v) + e)) then Algorithm 1 (the server
 * averages, sends Q_s(avg + e_s), keeps the residual, steps x).
 * ADAM_AT_SERVER moves the moment update to the server: each worker sends
 * Q_w(g + e), and the server runs Adam on the average before its own
 * quantization.  Both keep the two error-feedback residuals of Section IV.
 * The N worker replicas of x are identical (same x_1, same broadcast), so one
 * x is kept.
 * ------------------------------------------------------------------------- */
/* The toy problem of Section V-A: gradient of ||A x - (x* + xi)||^2 is
 * 2 A^T (A x - x* - xi). */
void eao_toy_grad(int64_t d, int32_t N, const float *A, const float *x_star, const float *xi,
                  const float *x, float *g, double *grad_sq)
{
    double *ax = (double *)malloc((size_t)d * sizeof(double));
    double *res = (double *)malloc((size_t)d * sizeof(double));
    for (int64_t k = 0; k < d; ++k) {
        double s = 0.0;
        for (int64_t j = 0; j < d; ++j) s += (double)A[k * d + j] * (double)x[j];
        ax[k] = s;
    }
    for (int32_t i = 0; i < N; ++i) {
        for (int64_t k = 0; k < d; ++k) res[k] = ax[k] - (double)x_star[k] - (double)xi[(int64_t)i * d + k];
        for (int64_t j = 0; j < d; ++j) {
            double s = 0.0;
            for (int64_t k = 0; k < d; ++k) s += (double)A[k * d + j] * res[k];
            g[(int64_t)i * d + j] = (float)(2.0 * s);
        }
    }
    if (grad_sq) {
        double tot = 0.0;
        for (int64_t k = 0; k < d; ++k) res[k] = ax[k] - (double)x_star[k];
        for (int64_t j = 0; j < d; ++j) {
            double s = 0.0;
            for (int64_t k = 0; k < d; ++k) s += (double)A[k * d + j] * res[k];
            s = 2.0 * s;
            tot += s * s;
        }
        *grad_sq = tot;
    }
    free(ax);
    free(res);
}

/* Schedules: Assumption 2's theta_t = 1 - theta/T and alpha_t = alpha/sqrt(T);
 * Section V-B's decay of alpha by a constant factor every `period` steps. */
int eao_schedule_at(const eao_schedule *s, float lr0, float beta2_0, int64_t t,
                    float *lr, float *beta2)
{
    if (t < 1) return -1;
    switch (s->kind) {
    case EAO_SCHED_CONSTANT:
        *lr = lr0;
        *beta2 = beta2_0;
        return 0;
    case EAO_SCHED_ASSUMPTION2: {
        if (s->T < 1 || s->T >= (1 << 24) || !(s->theta > 0.0f) || !(s->theta <= (float)s->T)) return -1;
        const float Tf = (float)s->T;      /* exact: T < 2^24 */
        *lr = s->alpha / sqrtf(Tf);
        *beta2 = 1.0f - s->theta / Tf;
        return 0;
    }
    case EAO_SCHED_STEP_DECAY: {
        if (s->period < 1 || !(s->factor > 0.0f) || !(s->factor <= 1.0f)) return -1;
        int64_t k = (t - 1) / s->period;
        float r = 1.0f, b = s->factor;
        while (k > 0) {
            if (k & 1) r = r * b;
            b = b * b;
            k >>= 1;
        }
        *lr = s->alpha * r;
        *beta2 = beta2_0;
        return 0;
    }
    default:
        return -1;
    }
}

static int check_segment(const eao_quant *q, int64_t d, int64_t n0, int64_t len)
{
    const int64_t B = eao_bucket_len(q, d);
    if (B == d) return (n0 == 0 && len == d) ? 0 : -1;
    if (n0 % B) return -1;
    if (n0 + len != d && len % B) return -1;
    return 0;
}

static int needs_draws(const eao_quant *q)
{
    return q->kind == EAO_Q_STOCH_UNIFORM || q->kind == EAO_Q_RANDK;
}

int eao_step(const eao_config *c, uint32_t t, int64_t n0, int64_t len,
             const float *g, float *e_w, float *m_w, float *v_w,
             float *m, float *v, float *e_s, float *x,
             uint64_t *wcodes, float *wscales, uint64_t *scodes, float *sscales,
             float *srv_in, float *p_w, float *q_s)
{
    const int64_t d = c->d;
    const int32_t N = c->N;
    if (d < 1 || N < 1 || len < 1 || n0 < 0 || n0 + len > d || (n0 & 255)) return -1;
    if (eao_code_bits(&c->qw) < 0 || eao_code_bits(&c->qs) < 0) return -1;
    if (check_segment(&c->qw, d, n0, len) || check_segment(&c->qs, d, n0, len)) return -1;
    const int at_worker = c->placement == EAO_ADAM_AT_WORKER;
    if (at_worker ? (!m_w || !v_w) : (!m || !v)) return -1;

    const int32_t bw = eao_code_bits(&c->qw), bs = eao_code_bits(&c->qs);
    const int64_t words_w = eao_msg_words(&c->qw, len);
    const int64_t scales_w = eao_num_scales(&c->qw, d, len);

    float *p = malloc((size_t)len * sizeof(float));
    float *u = malloc((size_t)len * sizeof(float));
    float *deq = malloc((size_t)len * sizeof(float));
    float *acc = calloc((size_t)len, sizeof(float));
    uint32_t *code = malloc((size_t)len * sizeof(uint32_t));
    if (!p || !u || !deq || !acc || !code) {
        free(p); free(u); free(deq); free(acc); free(code);
        return -1;
    }

    /* Workers (Algorithm 2). */
    for (int32_t i = 0; i < N; ++i) {
        const float *gi = g + (int64_t)i * len;
        float *ei = e_w + (int64_t)i * len;
        if (at_worker) {
            float *mi = m_w + (int64_t)i * len;
            float *vi = v_w + (int64_t)i * len;
            for (int64_t n = 0; n < len; ++n) {
                eao_adam_moments(c->beta1, c->beta2, &mi[n], &vi[n], gi[n]);
                p[n] = eao_adam_update(c->lr, mi[n], vi[n]) + ei[n];
            }
        } else {
            for (int64_t n = 0; n < len; ++n) p[n] = gi[n] + ei[n];
        }
        if (p_w) memcpy(p_w + (int64_t)i * len, p, (size_t)len * sizeof(float));
        if (needs_draws(&c->qw)) eao_uniforms(c->seed, t, (uint32_t)i, n0, len, u);
        if (eao_quantize(&c->qw, d, len, p, u, code, deq, wscales + (int64_t)i * scales_w)) {
            free(p); free(u); free(deq); free(acc); free(code);
            return -1;
        }
        eao_pack(bw, len, code, wcodes + (int64_t)i * words_w);
        for (int64_t n = 0; n < len; ++n) {
            ei[n] = c->qw.error_feedback ? p[n] - deq[n] : 0.0f;
            acc[n] = acc[n] + deq[n];
        }
    }

    /* Server (Algorithm 1): average, [Adam], add residual, quantize. */
    for (int64_t n = 0; n < len; ++n) {
        const float avg = acc[n] / (float)N;
        float a = avg;
        if (!at_worker) {
            eao_adam_moments(c->beta1, c->beta2, &m[n], &v[n], avg);
            a = eao_adam_update(c->lr, m[n], v[n]);
        }
        if (srv_in) srv_in[n] = a;
        p[n] = a + e_s[n];
    }
    if (q_s) memcpy(q_s, p, (size_t)len * sizeof(float));
    if (needs_draws(&c->qs)) eao_uniforms(c->seed, t, 0xFFFFFFFFu, n0, len, u);
    if (eao_quantize(&c->qs, d, len, p, u, code, deq, sscales)) {
        free(p); free(u); free(deq); free(acc); free(code);
        return -1;
    }
    eao_pack(bs, len, code, scodes);
    for (int64_t n = 0; n < len; ++n) {
        e_s[n] = c->qs.error_feedback ? p[n] - deq[n] : 0.0f;
        x[n] = x[n] - deq[n];
    }

    free(p); free(u); free(deq); free(acc); free(code);
    return 0;
}
