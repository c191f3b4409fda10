/*
 * eao.h -- Efficient-Adam oracle: a plain, slow, single-threaded C reference
 * of one optimizer round (paper: "Efficient-Adam: Communication-Efficient
 * Distributed Adam", Chen, Shen, Liu, Luo; Section IV, Algorithms 1 and 2).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this code; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no source with the HIP path.
 *
 * Arithmetic: every value the method communicates is an IEEE binary32 number
 * (Table 2 names 32-bit floats as full precision; Example 1 rounds the scale
 * to binary32), so the oracle computes in binary32 with round-to-nearest-even
 * and no contraction of a*b+c into a fused multiply-add.  Bucket sums are
 * accumulated in binary64 and rounded once.  Quantizer decisions are therefore
 * taken in binary32, the precision the kernels use.  x/s (Example 1, the
 * stochastic quantizer) is formed as x * (1/s); for a scale below 2^-126,
 * whose reciprocal overflows, x and s are first multiplied by 2^64 (exact).
 *
 * Parity status of each function is stated next to it; "parity unpinned"
 * marks a function that no test pins to something other than itself.
 */
#ifndef EAO_H
#define EAO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { EAO_Q_NONE = 0, EAO_Q_SCALED_SIGN = 1, EAO_Q_STOCH_UNIFORM = 2,
       EAO_Q_DET_UNIFORM = 3, EAO_Q_POW2 = 4, EAO_Q_TOPK = 5, EAO_Q_RANDK = 6 };
enum { EAO_SCALE_L1 = 0, EAO_SCALE_L2 = 1, EAO_SCALE_MAX = 2 };
enum { EAO_ADAM_AT_SERVER = 0, EAO_ADAM_AT_WORKER = 1 };

/* One quantization mapping Q (Definition 1 / Definition 3). */
typedef struct {
    int32_t kind;            /* EAO_Q_*                                         */
    int32_t scale;           /* STOCH_UNIFORM: EAO_SCALE_L2 or EAO_SCALE_MAX     */
    int32_t bits;            /* code width in bits (POW2: derived, see below)   */
    int32_t error_feedback;  /* 1: keep the residual e; 0: e is reset to 0      */
    int64_t bucket;          /* elements per scale bucket; 0 or >= d: one bucket */
    int32_t pow2_kmin;       /* Example 2: M = {2^kmin, ..., 2^kmax}            */
    int32_t pow2_kmax;
    int32_t keep;            /* TOPK, RANDK: elements kept per bucket, >= 1     */
    int32_t reserved;        /* 0                                               */
} eao_quant;

/* Definition 3 compressors (the sparsifiers of the works it cites): in each
 * bucket of n elements the k = min(keep, n) highest-ranked elements are kept
 * and the others sent as 0, which meets ||x - Q(x)||^2 <= (1 - k/n) ||x||^2
 * for TOPK (and in expectation, with equality, for RANDK).  Ranking is by a
 * 32-bit key, larger first, equal keys by lower index:
 *   TOPK   key = the binary32 pattern of x with the sign bit cleared, an order
 *          that equals the order of |x| on all non-NaN values (NaN ranks above
 *          infinity);
 *   RANDK  key = u * 2^24 for the element's uniform draw u (the 24-bit word
 *          the draw is made of), so the kept set is the k largest of n
 *          independent uniform keys: a uniformly random k-subset up to equal
 *          keys.
 * Code 1 marks a kept element.  The message's value array holds `keep`
 * binary32 numbers per bucket: the kept values in index order, then zeros
 * (only a last bucket shorter than keep has any). */

typedef struct {
    int64_t d;               /* parameters                                      */
    int32_t N;               /* workers                                         */
    int32_t placement;       /* EAO_ADAM_AT_SERVER or EAO_ADAM_AT_WORKER         */
    float beta1;             /* beta   (Algorithm 2)                            */
    float beta2;             /* theta_t (Algorithm 2)                           */
    float lr;                /* alpha_t (Algorithm 2)                           */
    float eps;               /* v_0 = eps (Algorithm 2, initialization)         */
    uint64_t seed;           /* key of the stochastic-rounding generator        */
    eao_quant qw;            /* Q_w, worker side                                */
    eao_quant qs;            /* Q_s, server side                                */
} eao_config;

/* Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw: "Parallel random
 * numbers: as easy as 1, 2, 3", SC'11).  Pinned against an independent
 * library implementation of the same generator. */
void eao_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* Uniform draws in [0,1) for global elements n0 .. n0+len-1 of one stream:
 * block j = n>>2 gives counter {lo(j), hi(j), t, stream}, key {lo(seed),
 * hi(seed)}; element n takes word n&3, r, and u = (r>>8) * 2^-24. */
void eao_uniforms(uint64_t seed, uint32_t t, uint32_t stream,
                  int64_t n0, int64_t len, float *u);

/* Code width of a quantizer in bits; -1 if the description is invalid. */
int32_t eao_code_bits(const eao_quant *q);
/* Bucket length used for a vector of d elements. */
int64_t eao_bucket_len(const eao_quant *q, int64_t d);
/* Number of per-bucket scales for a segment of len elements (0: none); for
 * TOPK and RANDK the number of values, keep per bucket. */
int64_t eao_num_scales(const eao_quant *q, int64_t d, int64_t len);
/* Number of 64-bit message words for a segment of len elements. */
int64_t eao_msg_words(const eao_quant *q, int64_t len);

/* Quantize a segment p[0..len) that starts on a bucket boundary of a vector
 * of d elements.  u[] holds one uniform draw per element (read only by
 * STOCH_UNIFORM and RANDK; may be NULL otherwise).  Writes one integer code and
 * one dequantized value per element, and one scale per bucket (TOPK, RANDK:
 * keep values per bucket).  Returns 0, or -1
 * on an invalid description. */
int eao_quantize(const eao_quant *q, int64_t d, int64_t len, const float *p,
                 const float *u, uint32_t *code, float *deq, float *scales);

/* One bucket of n elements of a scaled quantizer (SCALED_SIGN,
 * STOCH_UNIFORM, DET_UNIFORM) coded under a given scale s instead of its own
 * norm: the codes and dequantized values eao_quantize would give if the
 * bucket's scale were s.  Test infrastructure for checking a result formed
 * under a scale that differs from the oracle's in its last place.  Returns 0,
 * or -1 on an invalid description. */
int eao_quantize_bucket(const eao_quant *q, int64_t n, const float *p, const float *u, float s,
                        uint32_t *code, float *deq);

/* Dequantize codes back to values (inverse map of the code table). */
int eao_dequantize(const eao_quant *q, int64_t d, int64_t len, const uint32_t *code,
                   const float *scales, float *deq);

/* Pack/unpack per-element codes into the message word layout: element n of a
 * segment that starts at a multiple of 256 lies in chunk c = n>>8, at lane
 * l = (n>>2)&63 and slot k = n&3; bit p of its code is bit l of word
 * (4c + k)*bits + p.  32-bit codes are stored two per word, element n in
 * word n>>1, low half for even n. */
void eao_pack(int32_t bits, int64_t len, const uint32_t *code, uint64_t *words);
void eao_unpack(int32_t bits, int64_t len, const uint64_t *words, uint32_t *code);

/* Adam moments of Algorithm 2 (no bias correction), in place. */
void eao_adam_moments(float beta1, float beta2, float *m, float *v, float g);
/* Adam step alpha * m / sqrt(v); 0 when v is not positive. */
float eao_adam_update(float lr, float m, float v);

/* Step-size schedules.  lr_t and beta2_t (the paper's alpha_t and theta_t)
 * at step t >= 1, in binary32 arithmetic:
 *   CONSTANT     lr0, beta2_0 (the constants of the Section V experiments);
 *   ASSUMPTION2  alpha_t = alpha / sqrt(T), theta_t = 1 - theta / T for a
 *                horizon of T steps (Assumption 2);
 *   STEP_DECAY   alpha_t = alpha * factor^k with k = (t-1) / period (integer
 *                division; Section V-B reduces alpha to 0.2 alpha after every
 *                19,550 iterations), theta_t = beta2_0.  factor^k is formed by
 *                square-and-multiply over the bits of k from the lowest:
 *                r = 1, b = factor; for each bit: if set r = r*b; b = b*b.
 * Pinned by closed forms of both formulas and by the decay boundaries.
 * Returns 0, or -1 for an invalid schedule or t < 1. */
enum { EAO_SCHED_CONSTANT = 0, EAO_SCHED_ASSUMPTION2 = 1, EAO_SCHED_STEP_DECAY = 2 };
typedef struct {
    int32_t kind;            /* EAO_SCHED_*                                     */
    float alpha;             /* base learning rate                              */
    float theta;             /* ASSUMPTION2: theta, 0 < theta <= T              */
    float factor;            /* STEP_DECAY: 0 < factor <= 1                     */
    int64_t T;               /* ASSUMPTION2: horizon, 1 <= T < 2^24             */
    int64_t period;          /* STEP_DECAY: steps between decays, >= 1          */
} eao_schedule;

int eao_schedule_at(const eao_schedule *s, float lr0, float beta2_0, int64_t t,
                    float *lr, float *beta2);

/* Gradients of the toy problem of Section V-A, f(x) = E_xi || A x - (x* + xi) ||^2,
 * for N workers with noise draws xi_i (given):
 *   res_i = A x - x* - xi_i            (A x summed over j in binary64, then the
 *                                       two subtractions in binary64, in order)
 *   g_i   = 2 A^T res_i                (summed over k in binary64, then x2,
 *                                       rounded once to binary32)
 * and, if grad_sq is not NULL, *grad_sq = || 2 A^T (A x - x*) ||^2 in binary64
 * (the full gradient's squared norm, Figure 1's y-axis).  A is d x d,
 * row-major; xi and g are [N][d].  Pinned by finite differences of the
 * objective, the identity matrix case, and the noise-free consistency. */
void eao_toy_grad(int64_t d, int32_t N, const float *A, const float *x_star, const float *xi,
                  const float *x, float *g, double *grad_sq);

/* One full round at step t (1-based) on the segment [n0, n0+len) of the
 * d-vector.  Arrays are segment-local:
 *   g, e_w            [N][len]   gradients; worker residuals (in/out)
 *   m_w, v_w          [N][len]   worker moments, ADAM_AT_WORKER only (else NULL)
 *   m, v              [len]      server moments, ADAM_AT_SERVER only (else NULL)
 *   e_s, x            [len]      server residual, parameters (in/out)
 *   wcodes, wscales   [N][...]   worker messages (out)
 *   scodes, sscales   [...]      server message (out)
 *   srv_in            [len]      optional (NULL to skip): the value the server
 *                                quantizes before adding e_s
 *   p_w               [N][len]   optional (NULL to skip): each worker's
 *                                quantizer input p (after its residual is added)
 *   q_s               [len]      optional (NULL to skip): the server's quantizer
 *                                input (srv_in + e_s)
 * n0 must be a multiple of 256 and of both bucket lengths; a one-bucket
 * quantizer requires n0 == 0 and len == d.  Returns 0, or -1 on bad input. */
int eao_step(const eao_config *c, uint32_t t, int64_t n0, int64_t len,
             const float *g, float *e_w, float *m_w, float *v_w,
             float *m, float *v, float *e_s, float *x,
             uint64_t *wcodes, float *wscales, uint64_t *scodes, float *sscales,
             float *srv_in, float *p_w, float *q_s);

#ifdef __cplusplus
}
#endif
#endif
