// ea_launch.hpp -- kernel argument block and launchers shared by the C ABI
// (ea_api.cpp) and the kernels (ea_kernels.hip, ea_half_c*.hip, ea_toy.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ea.h"
#include "ea_device.hpp"

namespace ea {

// Everything one launch needs; pointers are device memory.
struct StepArgs {
    int64_t d;
    int32_t N;
    int32_t placement;
    float beta1, beta2, lr;
    uint32_t k0, k1;          // Philox key = seed
    uint32_t t;               // step (Philox counter word 2)
    int64_t ntiles;           // tiles of C chunks covering d
    QDev qw, qs;
    // worker side ([N][d] in ea_step; one row in the split calls)
    const float* g;
    float* e_w;
    float* m_w;
    float* v_w;
    // server side ([d])
    float* m;
    float* v;
    float* e_s;
    float* x;
    // messages
    uint64_t* wcodes;         // [N][qw.words]
    float* wscales;           // [N][qw.nscales]
    uint64_t* scodes;         // [qs.words]
    float* sscales;           // [qs.nscales]
    // one-bucket workspace
    double* wpart;            // [N][ntiles] per-tile partial norms (qw one bucket)
    double* spart;            // [ntiles]    per-tile partial norms (qs one bucket)
    float* ubuf;              // [d] server input / aggregate output
    int64_t tile0, tile1;     // fused round: the launch's tiles [tile0, tile1)
    int32_t worker;           // split calls: worker index (Philox stream)
    int32_t apply;            // server_kernel: also update x
    int32_t one_buffer;       // fused round, more workers than waves: single-buffered handoff
    int32_t xcd_run;          // fused round: blocks of a group of 8*xcd_run take tiles XCD-major (1: none)
    // Step index read on the device (null: `t`, `lr`, `beta2` above hold the
    // step's values); the schedule then gives lr and beta2 at that step.
    const uint32_t* t_dev;
    int32_t sched_kind;       // EA_SCHED_*
    float sched_alpha, sched_theta, sched_factor;
    int64_t sched_T, sched_period;
};

// Launchers; C = chunks per tile (1..8), vec = rows are 16-byte aligned.
// side_stream: the ragged last tile may run on a library-owned stream forked
// from s and joined back to it (created on first use per device).
hipError_t launch_step(const StepArgs& a, int C, bool vec, hipStream_t s, bool side_stream = true);

// Kernels specialized for the worker quantizer only (kind, code bits, norm
// and chunks per bucket fixed; the server quantizer and the Adam placement
// read at run time): the fused round for whole tiles of C = chunks-per-bucket
// chunks, and the split calls on the worker side.  One table per C, each
// compiled in its own translation unit.
struct HalfKernel {
    int C, wkind, wbits, wnorm, wcpb;
    void (*kernel)(StepArgs);
    int tiles;                // tiles per block
    void (*worker)(StepArgs);     // split call: one worker's compression (aligned rows)
    void (*aggregate)(StepArgs);  // split call: decode and average of the N messages
    void (*aggregate_full)(StepArgs);  // the same on tiles that lie wholly inside d
    // The same quantizer on the server side of the split calls (aligned rows):
    void (*server)(StepArgs);     // the server's compression
    void (*apply)(StepArgs);      // x -= the server message
};
// Fully specialized fused-round kernels for the same quantizer on both sides
// with Adam at the server, for wide tiles (C = 4, 8), where a run-time server
// quantizer costs most (its registers set the whole block's).
struct SymKernel {
    int C, kind, bits, norm, cpb;
    void (*kernel)(StepArgs);
    int tiles;
    void (*edge)(StepArgs);   // the last, partial tile (aligned rows)
};
const SymKernel* sym_kernels_c4(int* n);
const SymKernel* sym_kernels_c8(int* n);
const HalfKernel* half_kernels_c1(int* n);
const HalfKernel* half_kernels_c2(int* n);
const HalfKernel* half_kernels_c4(int* n);
const HalfKernel* half_kernels_c8(int* n);
hipError_t launch_worker_partials(const StepArgs& a, int C, bool vec, int i0, int i1, hipStream_t s);
hipError_t launch_server_partials(const StepArgs& a, int C, bool vec, hipStream_t s);
hipError_t launch_finalize(const double* part, int64_t ntiles, int32_t norm, int64_t n, float* out,
                           int64_t out_stride, int nvec, hipStream_t s);
hipError_t launch_worker(const StepArgs& a, int C, bool vec, hipStream_t s);
hipError_t launch_aggregate(const StepArgs& a, int C, bool vec, hipStream_t s);
hipError_t launch_server(const StepArgs& a, int C, bool vec, hipStream_t s);
hipError_t launch_apply(const StepArgs& a, int C, bool vec, hipStream_t s);
hipError_t launch_fill(float* p, int64_t n, float value, hipStream_t s);
// t_dev[0] <- t_dev[0] + 1 (after the kernels of a round that read it).
hipError_t launch_advance(uint32_t* t_dev, hipStream_t s);
// Toy problem of Section V-A: g = 2 A^T (A x - x* - xi_i) for N workers and
// the noise-free gradient's squared norm.  The workspace holds the residual
// and per-block partial norms (toy_workspace_bytes).
constexpr int64_t kToyMaxD = 65536;
int64_t toy_workspace_bytes(int64_t d);
hipError_t launch_toy_grad(int64_t d, int32_t N, const float* A, const float* xs, const float* xi, const float* x,
                           float* g, double* grad_sq, void* workspace, hipStream_t s);
// One round of the toy problem with the gradients formed inside it (the
// quantizers have no scales); `a` carries the configuration, the state and
// the messages.  g_out (nullable) receives the workers' gradients.
hipError_t launch_toy_step(const StepArgs& a, const float* A, const float* xs, const float* xi, double* grad_sq,
                           float* g_out, void* workspace, hipStream_t s);

}  // namespace ea
