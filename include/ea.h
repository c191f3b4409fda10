/*
 * ea.h -- C ABI of libea, the MI355X (gfx950) implementation of one
 * Efficient-Adam round (Chen, Shen, Liu, Luo, "Efficient-Adam:
 * Communication-Efficient Distributed Adam"; Section IV, Algorithms 1-2).
 *
 * N parameter-server workers and the server are simulated on one GPU; the
 * "messages" between them are device buffers in the wire format below.
 *
 * Conventions for every entry point
 *   - Pointers marked (device) are device memory owned by the caller; the
 *     library never allocates, frees or keeps them.  Pointers marked (host)
 *     are host memory read during the call only.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream)
 *     and the call returns without waiting.  Errors raised by the device
 *     surface at the next synchronization of that stream.  The fused round
 *     (ea_step, ea_step_scheduled, ea_run) may run the ragged last tile on a
 *     stream of its own (default priority, one per device, created on first
 *     use), forked from `stream` and joined back to it within the call, so
 *     work queued on `stream` afterwards still sees every result; not while
 *     `stream` is being captured, and never in ea_step_noalloc.
 *   - Return value: EA_OK, or a negative EA_ERR_* code; ea_last_error()
 *     returns a description of the last failure on the calling thread.
 *     Arguments are validated before any device work is enqueued, so an
 *     invalid call enqueues nothing and touches no device state.
 *   - Vectors are IEEE binary32.  Per-worker arrays are row-major [N][d].
 *   - Device pointers must be 4-byte aligned (else EA_ERR_ALIGN).  The whole-
 *     tile kernels need 16-byte aligned rows: every binary32 vector of the
 *     call 16-byte aligned (and an EA_Q_NONE message buffer) and d a multiple
 *     of 4, so that each row of an [N][d] array starts 16-byte aligned.  Any
 *     other accepted layout runs on kernels with per-element bounds checks,
 *     with the same results, about twice as slow.  Rows whose byte length is
 *     a multiple of 128 also share no cache line between tiles.
 *   - Calls that share buffers must be ordered by the caller (same stream).
 *
 * Wire format of a message (the paper defines none)
 *   codes   uint64 words.  For a code width b < 32, element n lies in chunk
 *           c = n>>8, lane l = (n>>2)&63, slot k = n&3; bit p of its code is
 *           bit l of word (4c + k)*b + p.  Bits of elements >= d are zero.
 *           ea_msg_words() = ceil(d/256)*4*b.  For EA_Q_NONE (b = 32) the
 *           words hold the binary32 values themselves, element n in word n>>1
 *           (low half for even n); ea_msg_words() = ceil(d/2).
 *   scales  one binary32 per bucket, in bucket order (none for NONE, POW2).
 *           TOPK, RANDK: `keep` binary32 values per bucket, in bucket order:
 *           the kept values in element order, then zeros (only a last bucket
 *           shorter than keep has any).
 *
 * Code tables
 *   SCALED_SIGN   b=1: code 1 = negative; value +-s, s = mean |p| of the bucket.
 *   STOCH_UNIFORM b in {1,2,4,8}: code c in [0, 2^b-1] is the level
 *                 s*(2c-L)/L, L = 2^b-1; s = bucket max-norm or L2-norm;
 *                 rounding up with probability equal to the fractional
 *                 position (unbiased).
 *   DET_UNIFORM   Example 1 with k = b-1, b in [2, 8]: code c = i + (2^k-1)
 *                 for the level s*i/(2^k-1); s = bucket max-norm.
 *   POW2          Example 2 with M = {2^kmin..2^kmax}: code = sign<<(b-1) |
 *                 (j - kmin) for +-2^j, and the magnitude code kmax-kmin+1
 *                 for 0; b = 1 + ceil(log2(kmax-kmin+2)).
 *   NONE          the value itself ("32-bit floating point", Table 2).
 *   TOPK, RANDK   Definition 3 compressors, b=1: code 1 marks a kept element,
 *                 which is sent exactly; the others are sent as 0.  Each bucket
 *                 of n elements keeps its min(keep, n) highest-ranked elements
 *                 by a 32-bit key, larger first, equal keys by lower index:
 *                 TOPK: the binary32 pattern with the sign cleared (the order
 *                 of |p|; NaN ranks above infinity), so ||p - Q(p)||^2 <=
 *                 (1 - keep/n) ||p||^2;  RANDK: the element's 24-bit draw
 *                 word (see below), a uniformly random subset up to equal
 *                 words.
 *
 * Buckets: `bucket` is 0 (one bucket over the whole vector), >= d (same), or
 * 256, 512, 1024 or 2048 (other sizes return EA_ERR_UNSUPPORTED).  TOPK and RANDK need
 * bucket 256, 512, 1024 or 2048 (a bucket >= d is one short bucket) and
 * 1 <= keep <= bucket.
 *
 * Stochastic rounding draws: element n of stream s at step t uses word n&3
 * of Philox4x32-10 (Salmon et al., SC'11) applied to counter
 * {lo(n>>2), hi(n>>2), t, s} with key {lo(seed), hi(seed)}, as
 * u = (word>>8) * 2^-24; RANDK ranks by word>>8.  Worker i uses stream i, the server 0xFFFFFFFF.
 * Replaying a step t replays its draws.
 */
#ifndef EA_H
#define EA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EA_OK 0
#define EA_ERR_ARG (-1)          /* invalid argument                               */
#define EA_ERR_ALIGN (-2)        /* a device pointer is not 4-byte aligned         */
#define EA_ERR_HIP (-3)          /* the HIP runtime reported an error              */
#define EA_ERR_UNSUPPORTED (-4)  /* valid per the paper, not supported here        */

#define EA_Q_NONE 0
#define EA_Q_SCALED_SIGN 1
#define EA_Q_STOCH_UNIFORM 2
#define EA_Q_DET_UNIFORM 3
#define EA_Q_POW2 4
#define EA_Q_TOPK 5              /* Definition 3: top-k per bucket                 */
#define EA_Q_RANDK 6             /* Definition 3: random-k per bucket              */

#define EA_SCALE_L1 0
#define EA_SCALE_L2 1
#define EA_SCALE_MAX 2

#define EA_ADAM_AT_SERVER 0      /* workers send Q_w(g + e); the server runs Adam  */
#define EA_ADAM_AT_WORKER 1      /* Algorithms 1-2 as printed: workers run Adam    */

/* One quantization mapping (Definition 1) or compressor (Definition 3). */
typedef struct ea_quant {
    int32_t kind;            /* EA_Q_*                                                */
    int32_t scale;           /* STOCH_UNIFORM: EA_SCALE_L2 or EA_SCALE_MAX; else unused */
    int32_t bits;            /* STOCH_UNIFORM, DET_UNIFORM: code width; else unused   */
    int32_t error_feedback;  /* 1: keep the residual e (Alg. 1-2); 0: e stays 0       */
    int64_t bucket;          /* see "Buckets" above                                   */
    int32_t pow2_kmin;       /* POW2: Example 2's k, -126 <= kmin < kmax <= 127       */
    int32_t pow2_kmax;       /* POW2: Example 2's K                                   */
    int32_t keep;            /* TOPK, RANDK: elements kept per bucket; else unused    */
    int32_t reserved;        /* must be 0                                             */
} ea_quant_t;

/* Arguments of the round, following the paper's statement of the problem. */
typedef struct ea_config {
    int64_t d;               /* parameters, d >= 1                                    */
    int32_t N;               /* workers, 1 <= N <= 1024                               */
    int32_t placement;       /* EA_ADAM_AT_SERVER or EA_ADAM_AT_WORKER                */
    float beta1;             /* beta in [0, 1)   (Algorithm 2)                        */
    float beta2;             /* theta_t in [0, 1) (Algorithm 2)                       */
    float lr;                /* alpha_t (Algorithm 2)                                 */
    float eps;               /* v_0 = eps (Algorithm 2, initialization)               */
    uint64_t seed;           /* key of the stochastic-rounding draws                  */
    ea_quant_t qw;           /* Q_w, used by the workers                              */
    ea_quant_t qs;           /* Q_s, used by the server                               */
} ea_config_t;

/* ---- sizes (host-only; never touch the device) --------------------------- */

/* Code width b in bits, or a negative EA_ERR_* for an invalid description. */
int32_t ea_code_bits(const ea_quant_t *q);
/* uint64 words of one message for a d-vector (see "Wire format"). */
int64_t ea_msg_words(const ea_quant_t *q, int64_t d);
/* binary32 scales of one message (0 for NONE and POW2; TOPK, RANDK: keep
 * values per bucket). */
int64_t ea_msg_scales(const ea_quant_t *q, int64_t d);
/* Payload bits of one message: d*b plus 32 per scale (the communication
 * cost counted in Corollary 1 and on the x-axis of Figures 1, 3, 6). */
int64_t ea_msg_bits(const ea_quant_t *q, int64_t d);
/* Device workspace (bytes) that ea_step, ea_worker_compress and
 * ea_server_compress need for one-bucket quantizers; 0 when none is needed. */
int64_t ea_workspace_bytes(const ea_config_t *c);
/* EA_OK if the configuration is valid and supported, else the error code. */
int ea_validate(const ea_config_t *c);
/* Description of the last error on the calling thread ("" if none). */
const char *ea_last_error(void);

/* ---- state ---------------------------------------------------------------- */

/* Initialization lines of Algorithms 1-2: m = 0, v = eps, e = 0.
 *   ADAM_AT_SERVER: m, v (device, d) required; m_w, v_w ignored (may be NULL).
 *   ADAM_AT_WORKER: m_w, v_w (device, N*d) required; m, v ignored.
 *   e_s (device, d) and e_w (device, N*d) are zeroed.  x is not touched. */
int ea_state_init(const ea_config_t *c, float *m, float *v, float *e_s, float *e_w,
                  float *m_w, float *v_w, void *stream);

/* ---- the round, split as in the paper ------------------------------------ */

/* Worker i, step t (Algorithm 2, from the moment update to the residual):
 *   ADAM_AT_SERVER: p = g + e_w;  ADAM_AT_WORKER: m_w, v_w <- Adam moments of g,
 *   p = lr * m_w / sqrt(v_w) + e_w.  Sends codes/scales = Q_w(p) and sets
 *   e_w = p - Q_w(p) (or 0 without error feedback).
 *   g (device, d, read), e_w (device, d, read/write), m_w, v_w (device, d,
 *   read/write; ADAM_AT_WORKER only, else NULL), codes (device,
 *   ea_msg_words(qw)), scales (device, ea_msg_scales(qw)), workspace (device,
 *   ea_workspace_bytes(c) bytes, or NULL when that is 0).
 *   Requires 0 <= i < N and 1 <= t <= 2^32-1. */
int ea_worker_compress(const ea_config_t *c, int32_t i, int64_t t, const float *g, float *e_w,
                       float *m_w, float *v_w, uint64_t *codes, float *scales,
                       void *workspace, void *stream);

/* Server gather (Algorithm 1, averaging line): avg = (sum over i = 0..N-1 of
 * the dequantized worker messages, added in ascending i) / N.
 *   ADAM_AT_SERVER: m, v (device, d, read/write) <- Adam moments of avg and
 *   u_out = lr * m / sqrt(v).  ADAM_AT_WORKER: u_out = avg; m, v ignored.
 *   wcodes (device, N * ea_msg_words(qw)), wscales (device, N *
 *   ea_msg_scales(qw); NULL when that is 0): the N messages, worker-major.
 *   u_out (device, d, write). */
int ea_server_aggregate_adam(const ea_config_t *c, int64_t t, const uint64_t *wcodes,
                             const float *wscales, float *m, float *v, float *u_out,
                             void *stream);

/* Server broadcast (Algorithm 1): q = u + e_s; sends codes/scales = Q_s(q)
 * and sets e_s = q - Q_s(q) (or 0 without error feedback).
 *   u (device, d, read), e_s (device, d, read/write), codes (device,
 *   ea_msg_words(qs)), scales (device, ea_msg_scales(qs)), workspace as above. */
int ea_server_compress(const ea_config_t *c, int64_t t, const float *u, float *e_s,
                       uint64_t *codes, float *scales, void *workspace, void *stream);

/* Every worker (and the server): x <- x - dequantize(server message)
 * (last line of Algorithms 1 and 2).  codes/scales (device, read), x (device,
 * d, read/write). */
int ea_worker_apply(const ea_config_t *c, const uint64_t *codes, const float *scales,
                    float *x, void *stream);

/* ---- the round, fused --------------------------------------------------- */

/* One full round at step t: the N worker compressions, the server gather
 * (+ Adam), the server compression and the update of x, in as few passes
 * over HBM as the buckets allow.  Produces the same messages and state as
 * the four calls above in order, without materializing the average.
 *   g (device, N*d, read); e_w (device, N*d, read/write); m_w, v_w (device,
 *   N*d, ADAM_AT_WORKER only); m, v (device, d, ADAM_AT_SERVER only); e_s, x
 *   (device, d, read/write); wcodes (device, N*ea_msg_words(qw)), wscales
 *   (device, N*ea_msg_scales(qw)), scodes (device, ea_msg_words(qs)),
 *   sscales (device, ea_msg_scales(qs)): the messages (write); workspace as
 *   above. */
int ea_step(const ea_config_t *c, int64_t t, const float *g, float *e_w, float *m_w, float *v_w,
            float *m, float *v, float *e_s, float *x, uint64_t *wcodes, float *wscales,
            uint64_t *scodes, float *sscales, void *workspace, void *stream);

/* ---- for callers that cannot allocate ------------------------------------ */

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): ea_step
 * without the workspace argument.  The workspace that one-bucket quantizers
 * need (ea_workspace_bytes) comes from a device array the library holds on
 * each GPU it runs on, EA_NOALLOC_SCRATCH_BYTES bytes, until the process ends;
 * the call itself allocates nothing (no hipMalloc, no allocating library
 * routine).  Every call on one GPU shares that GPU's array: calls that overlap
 * on one GPU (on different streams, or from different threads without
 * ordering) race and give undefined results.  Nothing in the array needs to
 * start at any value.  Returns EA_ERR_UNSUPPORTED, before any device work,
 * when ea_workspace_bytes(c) exceeds EA_NOALLOC_SCRATCH_BYTES.  Other
 * arguments, results and errors as ea_step. */
#define EA_NOALLOC_SCRATCH_BYTES (16 << 20)
int ea_step_noalloc(const ea_config_t *c, int64_t t, const float *g, float *e_w, float *m_w, float *v_w,
                    float *m, float *v, float *e_s, float *x, uint64_t *wcodes, float *wscales,
                    uint64_t *scodes, float *sscales, void *stream);

/* ---- step-size schedules and multi-step calls ------------------------------ */

/* lr_t and beta2_t (the paper's alpha_t and theta_t) at step t >= 1, in
 * binary32 arithmetic:
 *   EA_SCHED_CONSTANT     c->lr and c->beta2 (the Section V experiments);
 *   EA_SCHED_ASSUMPTION2  alpha_t = alpha / sqrt(T), theta_t = 1 - theta / T for
 *                         a horizon of T steps (Assumption 2); 1 <= T < 2^24,
 *                         0 < theta <= T;
 *   EA_SCHED_STEP_DECAY   alpha_t = alpha * factor^k, k = (t-1) / period, and
 *                         theta_t = c->beta2 (Section V-B: alpha becomes
 *                         0.2 alpha after every 19,550 iterations); factor^k is
 *                         formed by square-and-multiply over the bits of k from
 *                         the lowest; 0 < factor <= 1, period >= 1. */
#define EA_SCHED_CONSTANT 0
#define EA_SCHED_ASSUMPTION2 1
#define EA_SCHED_STEP_DECAY 2

typedef struct ea_schedule {
    int32_t kind;            /* EA_SCHED_*                                            */
    float alpha;             /* base learning rate (ASSUMPTION2, STEP_DECAY)          */
    float theta;             /* ASSUMPTION2                                           */
    float factor;            /* STEP_DECAY                                            */
    int64_t T;               /* ASSUMPTION2: horizon                                  */
    int64_t period;          /* STEP_DECAY: steps between decays                      */
} ea_schedule_t;

/* Host-only: (lr_t, beta2_t) of the schedule at step t >= 1 (host pointers). */
int ea_schedule_at(const ea_config_t *c, const ea_schedule_t *s, int64_t t, float *lr, float *beta2);

/* One round like ea_step, with the step index read on the device and the
 * hyperparameters taken from the schedule:
 *   t_dev (device, one uint32, read/write) holds the step t (>= 1; 0 gives an
 *   undefined round); the round uses t for its draws and lr_t, beta2_t from
 *   `s`, then stores t + 1.  Nothing on the host depends on t, so the call can
 *   be captured once into a HIP graph and replayed, each replay taking the
 *   next step.  Other arguments as ea_step (c->lr, c->beta2 are used by
 *   EA_SCHED_CONSTANT only). */
int ea_step_scheduled(const ea_config_t *c, const ea_schedule_t *s, uint32_t *t_dev, const float *g,
                      float *e_w, float *m_w, float *v_w, float *m, float *v, float *e_s, float *x,
                      uint64_t *wcodes, float *wscales, uint64_t *scodes, float *sscales,
                      void *workspace, void *stream);

/* `steps` rounds at t0, t0+1, ... with lr_t, beta2_t from the schedule,
 * enqueued back to back with the state kept in device memory.  Round t0+k
 * reads its gradients at g + k*g_step_stride (elements; 0: the same [N][d]
 * gradients every round).  The messages of the last round are left in
 * wcodes, wscales, scodes, sscales.  Other arguments as ea_step;
 * 1 <= t0 and t0 + steps - 1 <= 2^32-1. */
int ea_run(const ea_config_t *c, const ea_schedule_t *s, int64_t t0, int64_t steps, const float *g,
           int64_t g_step_stride, float *e_w, float *m_w, float *v_w, float *m, float *v, float *e_s,
           float *x, uint64_t *wcodes, float *wscales, uint64_t *scodes, float *sscales, void *workspace,
           void *stream);

/* ---- the toy problem of Section V-A -------------------------------------- */

/* Device workspace (bytes) of ea_toy_grad and ea_toy_step for dimension d. */
int64_t ea_toy_workspace_bytes(int64_t d);

/* Gradients of f(x) = E_xi || A x - (x* + xi) ||^2 (Section V-A) for N
 * workers: g_i = 2 A^T (A x - x* - xi_i), and, if grad_sq is not NULL, the
 * squared norm of the full gradient 2 A^T (A x - x*) (Figure 1's y-axis).
 *   A (device, d*d, row-major), x_star, x (device, d), xi (device, N*d: the
 *   workers' noise draws, supplied by the caller), g (device, N*d, write),
 *   grad_sq (device, one double, write; NULL to skip), workspace (device,
 *   ea_toy_workspace_bytes(d) bytes, 8-byte aligned).
 *   Products are summed in binary64 and each g_i rounded once to binary32.
 *   1 <= d <= 65536, 1 <= N <= 1024. */
int ea_toy_grad(int64_t d, int32_t N, const float *A, const float *x_star, const float *xi, const float *x,
                float *g, double *grad_sq, void *workspace, void *stream);

/* One round of the toy problem of Section V-A with the workers' gradients
 * formed inside it (Figure 1's setting): g_i = 2 A^T (A x - x* - xi_i) at the
 * current x, then the round of ea_step on those gradients, and, if grad_sq
 * is not NULL, the squared norm of the full gradient 2 A^T (A x - x*) at that
 * x (Figure 1's y-axis).  The gradients are not written to memory unless
 * g_out is given.  Both quantizers must be without scales (EA_Q_POW2,
 * Example 2; EA_Q_NONE), else EA_ERR_UNSUPPORTED: the message of a scaled
 * quantizer would need the whole bucket's gradient first.
 *   A (device, d*d, row-major), x_star (device, d), xi (device, N*d: the
 *   workers' noise draws for this step), e_w, m_w, v_w, m, v, e_s, x, wcodes,
 *   scodes as ea_step (no scales); grad_sq (device, one double, write, or
 *   NULL); g_out (device, N*d, write, or NULL); workspace (device,
 *   ea_toy_workspace_bytes(d) bytes, 8-byte aligned).
 *   The gradients' products are summed in binary64 (with fused multiply-adds,
 *   in the same order as ea_toy_grad's, whose gradients equal these bit for
 *   bit) and each g_i rounded once to binary32.  1 <= d <= 65536, 1 <= N <= 1024, 1 <= t <= 2^32-1. */
int ea_toy_step(const ea_config_t *c, int64_t t, const float *A, const float *x_star, const float *xi, float *e_w,
                float *m_w, float *v_w, float *m, float *v, float *e_s, float *x, uint64_t *wcodes,
                uint64_t *scodes, double *grad_sq, float *g_out, void *workspace, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* EA_H */
