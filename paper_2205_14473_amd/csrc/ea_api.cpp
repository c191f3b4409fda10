// ea_api.cpp -- the C ABI of libea (declared in include/ea.h): argument
// validation, launch geometry and kernel dispatch on the caller's stream.
// No entry point allocates memory or synchronizes.
#include "ea.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "ea_launch.hpp"

namespace {

// Device memory of ea_step_noalloc: the workspace of a round with one-bucket
// quantizers (per-tile partial norms and the server input), held by each GPU
// the library runs on until the process ends.  Every kernel that uses it
// writes each entry before reading it, so nothing needs clearing between
// calls.  In host code the array's name is only a stand-in: its device
// address, which differs per GPU, comes from scratch_ptr().
constexpr int64_t kScratchBytes = EA_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {nullptr};

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int ok()
{
    g_err[0] = '\0';
    return EA_OK;
}

bool kind_has_scales(int32_t kind)
{
    return kind == EA_Q_SCALED_SIGN || kind == EA_Q_STOCH_UNIFORM || kind == EA_Q_DET_UNIFORM;
}

bool kind_is_sparse(int32_t kind)
{
    return kind == EA_Q_TOPK || kind == EA_Q_RANDK;
}

// Code width of a quantizer (validated), or a negative error.
int32_t bits_of(const ea_quant_t* q)
{
    if (!q) return EA_ERR_ARG;
    switch (q->kind) {
    case EA_Q_NONE:
        return 32;
    case EA_Q_SCALED_SIGN:
        return 1;
    case EA_Q_STOCH_UNIFORM:
        return (q->bits == 1 || q->bits == 2 || q->bits == 4 || q->bits == 8) ? q->bits : EA_ERR_ARG;
    case EA_Q_DET_UNIFORM:
        return (q->bits >= 2 && q->bits <= 8) ? q->bits : EA_ERR_ARG;
    case EA_Q_POW2: {
        if (q->pow2_kmin < -126 || q->pow2_kmax > 127 || q->pow2_kmin >= q->pow2_kmax) return EA_ERR_ARG;
        int32_t need = q->pow2_kmax - q->pow2_kmin + 2;  // exponents plus the zero code
        int32_t b = 0;
        while ((1 << b) < need) ++b;
        return 1 + b;
    }
    case EA_Q_TOPK:
    case EA_Q_RANDK:
        return q->keep >= 1 ? 1 : EA_ERR_ARG;
    default:
        return EA_ERR_ARG;
    }
}

bool one_bucket(const ea_quant_t* q, int64_t d)
{
    return kind_has_scales(q->kind) && (q->bucket <= 0 || q->bucket >= d);
}

int64_t bucket_len(const ea_quant_t* q, int64_t d)
{
    return one_bucket(q, d) ? d : q->bucket;
}

int64_t nscales_of(const ea_quant_t* q, int64_t d)
{
    if (kind_is_sparse(q->kind)) return (d + q->bucket - 1) / q->bucket * q->keep;
    if (!kind_has_scales(q->kind)) return 0;
    const int64_t B = bucket_len(q, d);
    return (d + B - 1) / B;
}

int64_t words_of(int32_t b, int64_t d)
{
    return b == 32 ? (d + 1) / 2 : ((d + 255) / 256) * 4 * b;
}

int check_quant(const ea_quant_t* q, int64_t d, const char* side)
{
    const int32_t b = bits_of(q);
    if (b < 0)
        return fail(EA_ERR_ARG, "%s quantizer: invalid kind %d / bits %d / pow2 range [%d, %d] / keep %d", side,
                    q->kind, q->bits, q->pow2_kmin, q->pow2_kmax, q->keep);
    if (q->kind == EA_Q_STOCH_UNIFORM && q->scale != EA_SCALE_L2 && q->scale != EA_SCALE_MAX)
        return fail(EA_ERR_ARG, "%s quantizer: stochastic uniform needs EA_SCALE_L2 or EA_SCALE_MAX", side);
    if (q->error_feedback != 0 && q->error_feedback != 1)
        return fail(EA_ERR_ARG, "%s quantizer: error_feedback must be 0 or 1", side);
    if (q->bucket < 0) return fail(EA_ERR_ARG, "%s quantizer: negative bucket", side);
    if (kind_has_scales(q->kind) && !one_bucket(q, d)) {
        const int64_t B = q->bucket;
        if (B != 256 && B != 512 && B != 1024 && B != 2048)
            return fail(EA_ERR_UNSUPPORTED, "%s quantizer: bucket %lld must be 256, 512, 1024, 2048, 0 or >= d",
                        side, (long long)B);
    }
    if (kind_is_sparse(q->kind)) {
        const int64_t B = q->bucket;
        if (B != 256 && B != 512 && B != 1024 && B != 2048)
            return fail(EA_ERR_UNSUPPORTED, "%s quantizer: top-k / random-k bucket %lld must be 256, 512, 1024 or 2048",
                        side, (long long)B);
        if (q->keep > B)
            return fail(EA_ERR_ARG, "%s quantizer: keep %d must be in [1, bucket %lld]", side, q->keep, (long long)B);
    }
    if (q->reserved != 0) return fail(EA_ERR_ARG, "%s quantizer: reserved field must be 0", side);
    return EA_OK;
}

struct Plan {
    int C;                 // chunks per tile
    int64_t ntiles;
    ea::QDev qw, qs;
    bool wglobal, sglobal; // one-bucket quantizers
    int64_t off_wpart, off_spart, off_ubuf, ws_bytes;
};

ea::QDev make_qdev(const ea_quant_t* q, int64_t d)
{
    ea::QDev r{};
    r.kind = q->kind;
    r.bits = bits_of(q);
    r.ef = q->error_feedback;
    r.norm = q->kind == EA_Q_SCALED_SIGN ? ea::S_L1
           : (q->kind == EA_Q_STOCH_UNIFORM && q->scale == EA_SCALE_L2) ? ea::S_L2 : ea::S_MAX;
    r.B = kind_has_scales(q->kind) ? bucket_len(q, d) : kind_is_sparse(q->kind) ? q->bucket : d;
    r.cpb = ((kind_has_scales(q->kind) && !one_bucket(q, d)) || kind_is_sparse(q->kind)) ? (int32_t)(q->bucket / 256)
                                                                                          : 0;
    r.keep = kind_is_sparse(q->kind) ? q->keep : 0;
    r.cpb_shift = 0;
    while (r.cpb > 0 && (1 << r.cpb_shift) < r.cpb) ++r.cpb_shift;
    r.L = q->kind == EA_Q_STOCH_UNIFORM ? (1 << r.bits) - 1 : q->kind == EA_Q_DET_UNIFORM ? (1 << (r.bits - 1)) - 1 : 0;
    r.kmin = q->pow2_kmin;
    r.kmax = q->pow2_kmax;
    r.nscales = nscales_of(q, d);
    r.words = words_of(r.bits, d);
    return r;
}

int64_t align256(int64_t x)
{
    return (x + 255) / 256 * 256;
}

int validate(const ea_config_t* c)
{
    if (!c) return fail(EA_ERR_ARG, "config is NULL");
    if (c->d < 1) return fail(EA_ERR_ARG, "d must be >= 1 (got %lld)", (long long)c->d);
    if (c->d > ((int64_t)1 << 40)) return fail(EA_ERR_UNSUPPORTED, "d above 2^40 is not supported");
    if (c->N < 1 || c->N > 1024) return fail(EA_ERR_ARG, "N must be in [1, 1024] (got %d)", c->N);
    if (c->placement != EA_ADAM_AT_SERVER && c->placement != EA_ADAM_AT_WORKER)
        return fail(EA_ERR_ARG, "placement must be EA_ADAM_AT_SERVER or EA_ADAM_AT_WORKER");
    if (!(c->beta1 >= 0.0f && c->beta1 < 1.0f)) return fail(EA_ERR_ARG, "beta1 must be in [0, 1)");
    if (!(c->beta2 >= 0.0f && c->beta2 < 1.0f)) return fail(EA_ERR_ARG, "beta2 must be in [0, 1)");
    if (!std::isfinite(c->lr)) return fail(EA_ERR_ARG, "lr must be finite");
    if (!(c->eps >= 0.0f) || !std::isfinite(c->eps)) return fail(EA_ERR_ARG, "eps must be finite and >= 0");
    int rc = check_quant(&c->qw, c->d, "worker");
    if (rc) return rc;
    return check_quant(&c->qs, c->d, "server");
}

int make_plan(const ea_config_t* c, Plan* p)
{
    int rc = validate(c);
    if (rc) return rc;
    p->qw = make_qdev(&c->qw, c->d);
    p->qs = make_qdev(&c->qs, c->d);
    const int cw = p->qw.cpb, cs = p->qs.cpb;
    p->C = cw > cs ? cw : cs;
    if (p->C == 0) p->C = 2;
    const int64_t tile = (int64_t)p->C * ea::kChunk;
    p->ntiles = (c->d + tile - 1) / tile;
    p->wglobal = kind_has_scales(c->qw.kind) && cw == 0;
    p->sglobal = kind_has_scales(c->qs.kind) && cs == 0;
    int64_t off = 0;
    p->off_wpart = off;
    if (p->wglobal) off += align256((int64_t)c->N * p->ntiles * 8);
    p->off_spart = off;
    if (p->sglobal) off += align256(p->ntiles * 8);
    p->off_ubuf = off;
    if (p->sglobal) off += align256(c->d * 4);
    p->ws_bytes = off;
    return EA_OK;
}

bool aligned(const void* ptr, uintptr_t a)
{
    return ((uintptr_t)ptr % a) == 0;
}

// Fills the common part of the kernel argument block.
ea::StepArgs base_args(const ea_config_t* c, const Plan& p, int64_t t)
{
    ea::StepArgs a{};
    a.d = c->d;
    a.N = c->N;
    a.placement = c->placement;
    a.beta1 = c->beta1;
    a.beta2 = c->beta2;
    a.lr = c->lr;
    a.k0 = (uint32_t)c->seed;
    a.k1 = (uint32_t)(c->seed >> 32);
    a.t = (uint32_t)t;
    a.ntiles = p.ntiles;
    a.qw = p.qw;
    a.qs = p.qs;
    return a;
}

int check_t(int64_t t)
{
    if (t < 1 || t > (int64_t)0xFFFFFFFFLL) return fail(EA_ERR_ARG, "t must be in [1, 2^32-1] (got %lld)", (long long)t);
    return EA_OK;
}

// Schedules (declared with their definition in ea.h).
int check_schedule(const ea_schedule_t* s)
{
    if (!s) return fail(EA_ERR_ARG, "schedule is NULL");
    switch (s->kind) {
    case EA_SCHED_CONSTANT:
        return EA_OK;
    case EA_SCHED_ASSUMPTION2:
        if (s->T < 1 || s->T >= ((int64_t)1 << 24))
            return fail(EA_ERR_ARG, "schedule horizon T must be in [1, 2^24) (got %lld)", (long long)s->T);
        if (!(s->theta > 0.0f) || !(s->theta <= (float)s->T))
            return fail(EA_ERR_ARG, "schedule theta must be in (0, T] (got %g)", (double)s->theta);
        break;
    case EA_SCHED_STEP_DECAY:
        if (s->period < 1) return fail(EA_ERR_ARG, "schedule period must be >= 1 (got %lld)", (long long)s->period);
        if (!(s->factor > 0.0f) || !(s->factor <= 1.0f))
            return fail(EA_ERR_ARG, "schedule factor must be in (0, 1] (got %g)", (double)s->factor);
        break;
    default:
        return fail(EA_ERR_ARG, "unknown schedule kind %d", s->kind);
    }
    if (!std::isfinite(s->alpha) || s->alpha < 0.0f)
        return fail(EA_ERR_ARG, "schedule alpha must be finite and >= 0 (got %g)", (double)s->alpha);
    return EA_OK;
}

// lr_t, beta2_t of a validated schedule at step t >= 1, in binary32.
void schedule_values(const ea_schedule_t* s, float lr0, float beta2_0, int64_t t, float* lr, float* beta2)
{
    *lr = lr0;
    *beta2 = beta2_0;
    if (s->kind == EA_SCHED_ASSUMPTION2) {
        const float Tf = (float)s->T;
        *lr = s->alpha / std::sqrt(Tf);
        *beta2 = 1.0f - s->theta / Tf;
    } else if (s->kind == EA_SCHED_STEP_DECAY) {
        int64_t k = (t - 1) / s->period;
        float r = 1.0f, b = s->factor;
        for (; k > 0; k >>= 1) {
            if (k & 1) r = r * b;
            b = b * b;
        }
        *lr = s->alpha * r;
    }
}

int hip_status(hipError_t e, const char* what)
{
    if (e != hipSuccess) return fail(EA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

struct PtrCheck {
    int rc = EA_OK;
    void need(const void* ptr, bool required, uintptr_t align, const char* name)
    {
        if (rc) return;
        if (!ptr) {
            if (required) rc = fail(EA_ERR_ARG, "%s is NULL", name);
            return;
        }
        if (!aligned(ptr, align)) rc = fail(EA_ERR_ALIGN, "%s is not %u-byte aligned", name, (unsigned)align);
    }
};

// Vector path when every float row is 16-byte aligned.
bool vec_ok(int64_t d, std::initializer_list<const void*> ptrs)
{
    if (d % 4) return false;
    for (const void* q : ptrs)
        if (q && !aligned(q, 16)) return false;
    return true;
}

// One fused round.  With t_dev the step is read on the device, lr and beta2
// come from the schedule at that step, and t_dev is advanced afterwards.
int step_impl(const char* name, const ea_config_t* c, int64_t t, uint32_t* t_dev, const ea_schedule_t* sched,
              const float* g, float* e_w, float* m_w, float* v_w, float* m, float* v, float* e_s, float* x,
              uint64_t* wcodes, float* wscales, uint64_t* scodes, float* sscales, void* workspace, void* stream,
              bool side_stream = true)
{
    Plan p;
    int rc = make_plan(c, &p);
    if (rc) return rc;
    if (!t_dev && (rc = check_t(t))) return rc;
    const bool srv = c->placement == EA_ADAM_AT_SERVER;
    PtrCheck pc;
    pc.need(g, true, 4, "g");
    pc.need(e_w, true, 4, "e_w");
    pc.need(m_w, !srv, 4, "m_w");
    pc.need(v_w, !srv, 4, "v_w");
    pc.need(m, srv, 4, "m");
    pc.need(v, srv, 4, "v");
    pc.need(e_s, true, 4, "e_s");
    pc.need(x, true, 4, "x");
    pc.need(wcodes, true, 8, "wcodes");
    pc.need(wscales, p.qw.nscales > 0, 4, "wscales");
    pc.need(scodes, true, 8, "scodes");
    pc.need(sscales, p.qs.nscales > 0, 4, "sscales");
    pc.need(workspace, p.ws_bytes > 0, 256, "workspace");
    if (pc.rc) return pc.rc;
    ea::StepArgs a = base_args(c, p, t);
    if (t_dev) {
        a.t_dev = t_dev;
        a.sched_kind = sched->kind;
        a.sched_alpha = sched->alpha;
        a.sched_theta = sched->theta;
        a.sched_factor = sched->factor;
        a.sched_T = sched->T;
        a.sched_period = sched->period;
    }
    a.g = g;
    a.e_w = e_w;
    a.m_w = srv ? nullptr : m_w;
    a.v_w = srv ? nullptr : v_w;
    a.m = srv ? m : nullptr;
    a.v = srv ? v : nullptr;
    a.e_s = e_s;
    a.x = x;
    a.wcodes = wcodes;
    a.wscales = wscales;
    a.scodes = scodes;
    a.sscales = sscales;
    a.apply = 1;
    if (p.wglobal) a.wpart = (double*)((char*)workspace + p.off_wpart);
    if (p.sglobal) {
        a.spart = (double*)((char*)workspace + p.off_spart);
        a.ubuf = (float*)((char*)workspace + p.off_ubuf);
    }
    // Messages sent as raw values are written as float4 by whole-tile kernels.
    const bool vec = vec_ok(c->d, {g, e_w, a.m_w, a.v_w, a.m, a.v, e_s, x, a.ubuf,
                                   c->qw.kind == EA_Q_NONE ? (const void*)wcodes : nullptr,
                                   c->qs.kind == EA_Q_NONE ? (const void*)scodes : nullptr});
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = hipSuccess;
    if (p.wglobal) {
        e = ea::launch_worker_partials(a, p.C, vec, 0, c->N, s);
        if (e == hipSuccess)
            e = ea::launch_finalize(a.wpart, p.ntiles, p.qw.norm, c->d, wscales, p.qw.nscales, c->N, s);
    }
    if (e == hipSuccess) e = ea::launch_step(a, p.C, vec, s, side_stream);
    if (e == hipSuccess && p.sglobal) {
        e = ea::launch_finalize(a.spart, p.ntiles, p.qs.norm, c->d, sscales, 1, 1, s);
        if (e == hipSuccess) e = ea::launch_server(a, p.C, vec, s);
    }
    if (e == hipSuccess && t_dev) e = ea::launch_advance(t_dev, s);
    return hip_status(e, name);
}

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept.
int scratch_ptr(void** out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(EA_ERR_HIP, "ea_step_noalloc: hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return fail(EA_ERR_UNSUPPORTED, "ea_step_noalloc: device %d outside [0, %d)", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(EA_ERR_HIP, "ea_step_noalloc: hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return EA_OK;
}

}  // namespace

extern "C" {

int32_t ea_code_bits(const ea_quant_t* q)
{
    const int32_t b = bits_of(q);
    if (b < 0) return fail(b, "invalid quantizer description");
    return b;
}

int64_t ea_msg_words(const ea_quant_t* q, int64_t d)
{
    const int32_t b = bits_of(q);
    if (b < 0 || d < 1) return fail(EA_ERR_ARG, "invalid quantizer or d");
    return words_of(b, d);
}

int64_t ea_msg_scales(const ea_quant_t* q, int64_t d)
{
    if (bits_of(q) < 0 || d < 1) return fail(EA_ERR_ARG, "invalid quantizer or d");
    return nscales_of(q, d);
}

int64_t ea_msg_bits(const ea_quant_t* q, int64_t d)
{
    const int32_t b = bits_of(q);
    if (b < 0 || d < 1) return fail(EA_ERR_ARG, "invalid quantizer or d");
    return d * b + 32 * nscales_of(q, d);
}

int64_t ea_workspace_bytes(const ea_config_t* c)
{
    Plan p;
    const int rc = make_plan(c, &p);
    if (rc) return rc;
    return p.ws_bytes;
}

int ea_validate(const ea_config_t* c)
{
    Plan p;
    const int rc = make_plan(c, &p);
    return rc ? rc : ok();
}

const char* ea_last_error(void)
{
    return g_err;
}

int ea_state_init(const ea_config_t* c, float* m, float* v, float* e_s, float* e_w, float* m_w, float* v_w,
                  void* stream)
{
    Plan p;
    int rc = make_plan(c, &p);
    if (rc) return rc;
    const bool srv = c->placement == EA_ADAM_AT_SERVER;
    PtrCheck pc;
    pc.need(e_s, true, 4, "e_s");
    pc.need(e_w, true, 4, "e_w");
    pc.need(m, srv, 4, "m");
    pc.need(v, srv, 4, "v");
    pc.need(m_w, !srv, 4, "m_w");
    pc.need(v_w, !srv, 4, "v_w");
    if (pc.rc) return pc.rc;
    hipStream_t s = (hipStream_t)stream;
    const int64_t d = c->d, Nd = (int64_t)c->N * c->d;
    hipError_t e = ea::launch_fill(e_s, d, 0.0f, s);
    if (e == hipSuccess) e = ea::launch_fill(e_w, Nd, 0.0f, s);
    if (e == hipSuccess && srv) e = ea::launch_fill(m, d, 0.0f, s);
    if (e == hipSuccess && srv) e = ea::launch_fill(v, d, c->eps, s);
    if (e == hipSuccess && !srv) e = ea::launch_fill(m_w, Nd, 0.0f, s);
    if (e == hipSuccess && !srv) e = ea::launch_fill(v_w, Nd, c->eps, s);
    return hip_status(e, "ea_state_init");
}

int ea_worker_compress(const ea_config_t* c, int32_t i, int64_t t, const float* g, float* e_w, float* m_w,
                       float* v_w, uint64_t* codes, float* scales, void* workspace, void* stream)
{
    Plan p;
    int rc = make_plan(c, &p);
    if (rc) return rc;
    if ((rc = check_t(t))) return rc;
    if (i < 0 || i >= c->N) return fail(EA_ERR_ARG, "worker index %d outside [0, %d)", i, c->N);
    const bool atw = c->placement == EA_ADAM_AT_WORKER;
    PtrCheck pc;
    pc.need(g, true, 4, "g");
    pc.need(e_w, true, 4, "e_w");
    pc.need(m_w, atw, 4, "m_w");
    pc.need(v_w, atw, 4, "v_w");
    pc.need(codes, true, 8, "codes");
    pc.need(scales, p.qw.nscales > 0, 4, "scales");
    pc.need(workspace, p.wglobal, 256, "workspace");
    if (pc.rc) return pc.rc;
    ea::StepArgs a = base_args(c, p, t);
    a.g = g;
    a.e_w = e_w;
    a.m_w = atw ? m_w : nullptr;
    a.v_w = atw ? v_w : nullptr;
    a.wcodes = codes;
    a.wscales = scales;
    a.worker = i;
    const bool vec = vec_ok(c->d, {g, e_w, a.m_w, a.v_w});
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = hipSuccess;
    if (p.wglobal) {
        a.wpart = (double*)((char*)workspace + p.off_wpart);
        e = ea::launch_worker_partials(a, p.C, vec, i, i + 1, s);
        if (e == hipSuccess) e = ea::launch_finalize(a.wpart, p.ntiles, p.qw.norm, c->d, scales, 1, 1, s);
    }
    if (e == hipSuccess) e = ea::launch_worker(a, p.C, vec, s);
    return hip_status(e, "ea_worker_compress");
}

int ea_server_aggregate_adam(const ea_config_t* c, int64_t t, const uint64_t* wcodes, const float* wscales,
                             float* m, float* v, float* u_out, void* stream)
{
    Plan p;
    int rc = make_plan(c, &p);
    if (rc) return rc;
    if ((rc = check_t(t))) return rc;
    const bool srv = c->placement == EA_ADAM_AT_SERVER;
    PtrCheck pc;
    pc.need(wcodes, true, 8, "wcodes");
    pc.need(wscales, p.qw.nscales > 0, 4, "wscales");
    pc.need(m, srv, 4, "m");
    pc.need(v, srv, 4, "v");
    pc.need(u_out, true, 4, "u_out");
    if (pc.rc) return pc.rc;
    ea::StepArgs a = base_args(c, p, t);
    a.wcodes = const_cast<uint64_t*>(wcodes);
    a.wscales = const_cast<float*>(wscales);
    a.m = srv ? m : nullptr;
    a.v = srv ? v : nullptr;
    a.ubuf = u_out;
    const bool vec = vec_ok(c->d, {a.m, a.v, u_out});
    return hip_status(ea::launch_aggregate(a, p.C, vec, (hipStream_t)stream), "ea_server_aggregate_adam");
}

int ea_server_compress(const ea_config_t* c, int64_t t, const float* u, float* e_s, uint64_t* codes,
                       float* scales, void* workspace, void* stream)
{
    Plan p;
    int rc = make_plan(c, &p);
    if (rc) return rc;
    if ((rc = check_t(t))) return rc;
    PtrCheck pc;
    pc.need(u, true, 4, "u");
    pc.need(e_s, true, 4, "e_s");
    pc.need(codes, true, 8, "codes");
    pc.need(scales, p.qs.nscales > 0, 4, "scales");
    pc.need(workspace, p.sglobal, 256, "workspace");
    if (pc.rc) return pc.rc;
    ea::StepArgs a = base_args(c, p, t);
    a.ubuf = const_cast<float*>(u);
    a.e_s = e_s;
    a.scodes = codes;
    a.sscales = scales;
    a.apply = 0;
    const bool vec = vec_ok(c->d, {u, e_s});
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = hipSuccess;
    if (p.sglobal) {
        a.spart = (double*)((char*)workspace + p.off_spart);
        e = ea::launch_server_partials(a, p.C, vec, s);
        if (e == hipSuccess) e = ea::launch_finalize(a.spart, p.ntiles, p.qs.norm, c->d, scales, 1, 1, s);
    }
    if (e == hipSuccess) e = ea::launch_server(a, p.C, vec, s);
    return hip_status(e, "ea_server_compress");
}

int ea_worker_apply(const ea_config_t* c, const uint64_t* codes, const float* scales, float* x, void* stream)
{
    Plan p;
    int rc = make_plan(c, &p);
    if (rc) return rc;
    PtrCheck pc;
    pc.need(codes, true, 8, "codes");
    pc.need(scales, p.qs.nscales > 0, 4, "scales");
    pc.need(x, true, 4, "x");
    if (pc.rc) return pc.rc;
    ea::StepArgs a = base_args(c, p, 1);
    a.scodes = const_cast<uint64_t*>(codes);
    a.sscales = const_cast<float*>(scales);
    a.x = x;
    const bool vec = vec_ok(c->d, {x});
    return hip_status(ea::launch_apply(a, p.C, vec, (hipStream_t)stream), "ea_worker_apply");
}

int ea_step(const ea_config_t* c, int64_t t, const float* g, float* e_w, float* m_w, float* v_w, float* m,
            float* v, float* e_s, float* x, uint64_t* wcodes, float* wscales, uint64_t* scodes, float* sscales,
            void* workspace, void* stream)
{
    return step_impl("ea_step", c, t, nullptr, nullptr, g, e_w, m_w, v_w, m, v, e_s, x, wcodes, wscales, scodes,
                     sscales, workspace, stream);
}

int ea_step_noalloc(const ea_config_t* c, int64_t t, const float* g, float* e_w, float* m_w, float* v_w, float* m,
                    float* v, float* e_s, float* x, uint64_t* wcodes, float* wscales, uint64_t* scodes,
                    float* sscales, void* stream)
{
    Plan p;
    int rc = make_plan(c, &p);
    if (rc) return rc;
    if (p.ws_bytes > kScratchBytes)
        return fail(EA_ERR_UNSUPPORTED, "ea_step_noalloc: this configuration needs %lld bytes of scratch memory, more "
                    "than the %lld the library holds (EA_NOALLOC_SCRATCH_BYTES); use ea_step with a workspace",
                    (long long)p.ws_bytes, (long long)kScratchBytes);
    void* ws = nullptr;
    if (p.ws_bytes > 0 && (rc = scratch_ptr(&ws))) return rc;
    // no side stream for the ragged tile: creating one on first use would allocate
    return step_impl("ea_step_noalloc", c, t, nullptr, nullptr, g, e_w, m_w, v_w, m, v, e_s, x, wcodes, wscales,
                     scodes, sscales, ws, stream, false);
}

int ea_schedule_at(const ea_config_t* c, const ea_schedule_t* s, int64_t t, float* lr, float* beta2)
{
    if (!c || !lr || !beta2) return fail(EA_ERR_ARG, "ea_schedule_at: NULL argument");
    int rc = check_schedule(s);
    if (rc) return rc;
    if (t < 1) return fail(EA_ERR_ARG, "t must be >= 1 (got %lld)", (long long)t);
    schedule_values(s, c->lr, c->beta2, t, lr, beta2);
    return ok();
}

int ea_step_scheduled(const ea_config_t* c, const ea_schedule_t* s, uint32_t* t_dev, const float* g, float* e_w,
                      float* m_w, float* v_w, float* m, float* v, float* e_s, float* x, uint64_t* wcodes,
                      float* wscales, uint64_t* scodes, float* sscales, void* workspace, void* stream)
{
    int rc = check_schedule(s);
    if (rc) return rc;
    if (!t_dev || ((uintptr_t)t_dev & 3u)) return fail(EA_ERR_ALIGN, "t_dev must be a 4-byte aligned device pointer");
    return step_impl("ea_step_scheduled", c, 1, t_dev, s, g, e_w, m_w, v_w, m, v, e_s, x, wcodes, wscales, scodes,
                     sscales, workspace, stream);
}

int ea_run(const ea_config_t* c, const ea_schedule_t* s, int64_t t0, int64_t steps, const float* g,
           int64_t g_step_stride, float* e_w, float* m_w, float* v_w, float* m, float* v, float* e_s, float* x,
           uint64_t* wcodes, float* wscales, uint64_t* scodes, float* sscales, void* workspace, void* stream)
{
    if (!c) return fail(EA_ERR_ARG, "config is NULL");
    int rc = check_schedule(s);
    if (rc) return rc;
    if (steps < 0) return fail(EA_ERR_ARG, "steps must be >= 0 (got %lld)", (long long)steps);
    if (g_step_stride < 0) return fail(EA_ERR_ARG, "g_step_stride must be >= 0");
    if ((rc = check_t(t0))) return rc;
    if (steps > 0 && (rc = check_t(t0 + steps - 1))) return rc;
    // Validate before enqueueing anything.  The steps' configurations differ
    // from c only in lr and beta2, and a valid schedule keeps them valid at
    // every step once they are at t0 (the step decay only shrinks a finite,
    // non-negative alpha; the other schedules are constant in t), so one
    // check covers the whole run.
    if (steps > 0) {
        ea_config_t c0 = *c;
        schedule_values(s, c->lr, c->beta2, t0, &c0.lr, &c0.beta2);
        Plan p;
        if ((rc = make_plan(&c0, &p))) return rc;
    }
    for (int64_t k = 0; k < steps; ++k) {
        ea_config_t ck = *c;
        schedule_values(s, c->lr, c->beta2, t0 + k, &ck.lr, &ck.beta2);
        rc = step_impl("ea_run", &ck, t0 + k, nullptr, nullptr, g ? g + k * g_step_stride : nullptr, e_w, m_w, v_w,
                       m, v, e_s, x, wcodes, wscales, scodes, sscales, workspace, stream);
        if (rc) return rc;
    }
    return ok();
}

int64_t ea_toy_workspace_bytes(int64_t d)
{
    if (d < 1 || d > ea::kToyMaxD) return fail(EA_ERR_ARG, "toy gradient needs 1 <= d <= %lld (got %lld)",
                                               (long long)ea::kToyMaxD, (long long)d);
    return ea::toy_workspace_bytes(d);
}

int ea_toy_grad(int64_t d, int32_t N, const float* A, const float* x_star, const float* xi, const float* x,
                float* g, double* grad_sq, void* workspace, void* stream)
{
    if (d < 1 || d > ea::kToyMaxD) return fail(EA_ERR_ARG, "toy gradient needs 1 <= d <= %lld (got %lld)",
                                               (long long)ea::kToyMaxD, (long long)d);
    if (N < 1 || N > 1024) return fail(EA_ERR_ARG, "N must be in [1, 1024] (got %d)", N);
    PtrCheck pc;
    pc.need(A, true, 4, "A");
    pc.need(x_star, true, 4, "x_star");
    pc.need(xi, true, 4, "xi");
    pc.need(x, true, 4, "x");
    pc.need(g, true, 4, "g");
    pc.need(grad_sq, false, 8, "grad_sq");
    pc.need(workspace, true, 8, "workspace");
    if (pc.rc) return pc.rc;
    return hip_status(ea::launch_toy_grad(d, N, A, x_star, xi, x, g, grad_sq, workspace, (hipStream_t)stream),
                      "ea_toy_grad");
}

int ea_toy_step(const ea_config_t* c, int64_t t, const float* A, const float* x_star, const float* xi, float* e_w,
                float* m_w, float* v_w, float* m, float* v, float* e_s, float* x, uint64_t* wcodes, uint64_t* scodes,
                double* grad_sq, float* g_out, void* workspace, void* stream)
{
    Plan p;
    int rc = make_plan(c, &p);
    if (rc) return rc;
    if ((rc = check_t(t))) return rc;
    if (c->d > ea::kToyMaxD)
        return fail(EA_ERR_ARG, "ea_toy_step needs d <= %lld (got %lld)", (long long)ea::kToyMaxD, (long long)c->d);
    const auto scaleless = [](int32_t k) { return k == EA_Q_POW2 || k == EA_Q_NONE; };
    if (!scaleless(c->qw.kind) || !scaleless(c->qs.kind))
        return fail(EA_ERR_UNSUPPORTED, "ea_toy_step: both quantizers must be without scales (EA_Q_POW2 or EA_Q_NONE); "
                    "use ea_toy_grad and ea_step for the others");
    const bool srv = c->placement == EA_ADAM_AT_SERVER;
    PtrCheck pc;
    pc.need(A, true, 4, "A");
    pc.need(x_star, true, 4, "x_star");
    pc.need(xi, true, 4, "xi");
    pc.need(e_w, true, 4, "e_w");
    pc.need(m_w, !srv, 4, "m_w");
    pc.need(v_w, !srv, 4, "v_w");
    pc.need(m, srv, 4, "m");
    pc.need(v, srv, 4, "v");
    pc.need(e_s, true, 4, "e_s");
    pc.need(x, true, 4, "x");
    pc.need(wcodes, true, 8, "wcodes");
    pc.need(scodes, true, 8, "scodes");
    pc.need(grad_sq, false, 8, "grad_sq");
    pc.need(g_out, false, 4, "g_out");
    pc.need(workspace, true, 8, "workspace");
    if (pc.rc) return pc.rc;
    ea::StepArgs a = base_args(c, p, t);
    a.e_w = e_w;
    a.m_w = srv ? nullptr : m_w;
    a.v_w = srv ? nullptr : v_w;
    a.m = srv ? m : nullptr;
    a.v = srv ? v : nullptr;
    a.e_s = e_s;
    a.x = x;
    a.wcodes = wcodes;
    a.scodes = scodes;
    return hip_status(ea::launch_toy_step(a, A, x_star, xi, grad_sq, g_out, workspace, (hipStream_t)stream),
                      "ea_toy_step");
}

}  // extern "C"
