// ea_toy.hip -- the toy problem of Section V-A on the device:
// f(x) = E_xi || A x - (x* + xi) ||^2, whose gradient for a noise draw xi_i is
// g_i = 2 A^T (A x - x* - xi_i).  Products are summed in binary64 and each g
// rounded once to binary32, like the oracle.
//
// Two launches for both entry points:
//   1. residual: res[k] = (A x)[k] - x*[k], one wave per row of A (it also
//      clears the counters of the second launch);
//   2. toy_round_kernel: block (b, r) owns columns [64b, 64b+64), one per
//      lane, and the r-th of the splits of the rows of A.  Its 16 waves stage
//      r - xi_i for a tile of rows of every worker in LDS and accumulate all
//      workers' column sums (and the noise-free one) over contiguous row
//      ranges, in binary64 with fused multiply-adds; the 16 partial sums of
//      an output are added in wave order.  With several splits each block
//      publishes its sums, and the last block of the column group to arrive
//      adds the splits' sums in split order and goes on alone (no block
//      waits for another); a small problem thereby spreads over many CUs
//      instead of one block walking every row.  The last column group to
//      finish adds the groups' partial squared norms of the noise-free
//      gradient (lane l those of groups l, l+64, ..., then the wave's sum).
//
// ea_toy_grad writes the gradients and stops there.  ea_toy_step fuses the
// producer into the round (quantizers without scales: Example 2, full
// precision): wave i holds worker i's gradient for the block's columns and
// runs its side of the round (Adam at the worker, the code, the residual);
// its codes fill a 16-bit slice of each message word (the block's 64
// elements are 16 lanes of one 256-element chunk).  The last wave adds the
// workers' dequantized values in ascending order and runs the server side.
// The gradient is not written to HBM unless asked for (g_out).  Both entry
// points sum in the same order, so their gradients agree bit for bit.
#include "ea_launch.hpp"

namespace ea {

namespace {

constexpr int kResWaves = 4;                    // rows per residual block

__global__ __launch_bounds__(kResWaves * kWave) void toy_residual_kernel(int64_t d, const float* __restrict__ A,
                                                                         const float* __restrict__ xs,
                                                                         const float* __restrict__ x,
                                                                         double* __restrict__ res,
                                                                         uint32_t* __restrict__ counter,
                                                                         int32_t ncounter)
{
    if (counter != nullptr && blockIdx.x == 0)
        for (int i = (int)threadIdx.x; i < ncounter; i += (int)blockDim.x) counter[i] = 0u;
    const int64_t k = (int64_t)blockIdx.x * kResWaves + threadIdx.x / kWave;
    if (k >= d) return;
    const int lane = lane_id();
    const float* row = A + k * d;
    double s = 0.0;
    int64_t j = lane;
    for (; j + 3 * kWave < d; j += 4 * kWave) {
        const float a0 = row[j], a1 = row[j + kWave], a2 = row[j + 2 * kWave], a3 = row[j + 3 * kWave];
        const float x0 = x[j], x1 = x[j + kWave], x2 = x[j + 2 * kWave], x3 = x[j + 3 * kWave];
        s += (double)a0 * (double)x0;
        s += (double)a1 * (double)x1;
        s += (double)a2 * (double)x2;
        s += (double)a3 * (double)x3;
    }
    for (; j < d; j += kWave) s += (double)row[j] * (double)x[j];
    s = wave_sum(s);
    if (lane == 0) res[k] = s - (double)xs[k];
}

// ---------------------------------------------------------------------------
// The fused toy round.
// ---------------------------------------------------------------------------
constexpr int kTRWaves = 16;                   // waves per block
constexpr int kTROut = 16;                     // column sums per pass: workers + the noise-free one
constexpr int kTRWorkers = kTROut - 1;         // workers per pass
constexpr int kTRRows = 256;                   // rows of A per staged tile, one split
constexpr int kTRSplitRows = 64;               // the same with several splits: one slot per thread
constexpr int kTRMaxSplits = 8;                // splits of the rows per column group
constexpr int kTRSplitBlocks = 1024;           // column groups x splits aimed at

// Splits of the rows of A for d columns when the workers fit one pass (one
// when the column groups alone fill the GPU), each a whole number of
// kTRSplitRows tiles; `rows` receives the rows per split.
int toy_splits(int64_t d, int64_t* rows)
{
    const int64_t nblk = (d + kWave - 1) / kWave;
    int64_t R = (d + kTRSplitRows - 1) / kTRSplitRows;
    if (R > kTRMaxSplits) R = kTRMaxSplits;
    if (R > kTRSplitBlocks / nblk) R = kTRSplitBlocks / nblk;
    if (R < 2) {
        *rows = d;
        return 1;
    }
    const int64_t per = (d + R - 1) / R;
    *rows = (per + kTRSplitRows - 1) / kTRSplitRows * kTRSplitRows;
    return (int)((d + *rows - 1) / *rows);
}

// Bits 0, 4, 8, ..., 60 of x gathered into bits 0..15.
__device__ __forceinline__ uint32_t every_fourth_bit(uint64_t x)
{
    x &= 0x1111111111111111ull;
    x = (x | (x >> 3)) & 0x0303030303030303ull;
    x = (x | (x >> 6)) & 0x000F000F000F000Full;
    x = (x | (x >> 12)) & 0x000000FF000000FFull;
    x = (x | (x >> 24)) & 0x000000000000FFFFull;
    return (uint32_t)x;
}

// Code and dequantized value of one element for a quantizer without scales.
__device__ __forceinline__ void toy_code(const QDev& q, float p, uint32_t& code, float& deq)
{
    if (q.kind == Q_NONE) {
        code = __float_as_uint(p);
        deq = p;
    } else {
        code = code_of<QRt>(q, p, 0.0f, 0u);
        deq = lut_entry<QRt>(q, (int32_t)code);
    }
}

// The block's 64 elements are lanes l0..l0+15 of chunk `chunk`, all four
// slots.  Bit plane p of slot s is a 16-bit slice (bits l0..l0+15) of message
// word (4 chunk + s) b + p; lane s b + p stores it.  Raw values (b = 32) are
// stored as the binary32 element itself.
__device__ __forceinline__ void toy_store_codes(const QDev& q, uint64_t* __restrict__ msg, int64_t col, bool in,
                                                uint32_t code)
{
    const int lane = lane_id();
    if (q.kind == Q_NONE) {
        if (in) reinterpret_cast<uint32_t*>(msg)[col] = code;
        return;
    }
    const int b = q.bits;
    const int64_t c0 = col - lane;                 // first column of the block (a multiple of 64)
    const int64_t chunk = c0 >> 8;
    const int l0 = (int)((c0 >> 2) & 63);          // 0, 16, 32 or 48
    uint32_t piece = 0;
    for (int s = 0; s < 4; ++s)
        for (int p = 0; p < b; ++p) {
            const uint64_t m = __builtin_amdgcn_ballot_w64(in && ((code >> p) & 1u) != 0u);
            const uint32_t v = every_fourth_bit(m >> s);
            piece = (uint32_t)ea_writelane_i32((int)v, s * b + p, (int)piece);
        }
    if (lane < 4 * b) {
        const int s = lane / b, p = lane % b;
        uint16_t* w = reinterpret_cast<uint16_t*>(msg + (4 * chunk + s) * b + p);
        w[l0 >> 4] = (uint16_t)piece;
    }
}

struct ToyArgs {
    int64_t d;
    int32_t N, placement;
    float beta1, beta2, lr;
    QDev qw, qs;
    const float* A;
    const double* res;      // r = A x - x*
    const float* xi;        // [N][d]
    float *x, *e_w, *m_w, *v_w, *m, *v, *e_s;
    uint64_t *wcodes, *scodes;
    double* part;           // [blocks] partial squared norms of the noise-free gradient
    uint32_t* counter;      // [1 + blocks]: column groups done, then each group's splits
                            // arrived (cleared by the residual launch)
    int32_t splits;         // splits of the rows (gridDim.y); above 1 only with one pass
    int64_t split_rows;     // rows per split
    double* psum;           // [blocks][splits][kTROut][64] the splits' column sums
    double* grad_sq;        // nullable
    float* g_out;           // nullable: [N][d] the workers' gradients, for checking
};

// ROUND: the round follows the gradients; without it the kernel only writes
// the gradients to g_out (ea_toy_grad) and the norm.
template <int ROWS, bool ROUND>
__global__ __launch_bounds__(kTRWaves * kWave) void toy_round_kernel(ToyArgs a)
{
    constexpr int kPer = ROWS / kTRWaves;          // rows of a tile per wave
    static_assert(ROWS % kTRWaves == 0 && ROWS * kTROut <= kTRWaves * kTROut * kWave, "tile shape");
    // Staged tiles (row-major [row][output]), then the waves' partial sums.
    __shared__ __attribute__((aligned(16))) double big[kTRWaves * kTROut * kWave];
    __shared__ float xfer[kTRWorkers * kWave];
    __shared__ int last_split;
    const int lane = lane_id();
    const int w = (int)(threadIdx.x / kWave);
    const int64_t d = a.d;
    const int64_t col = (int64_t)blockIdx.x * kWave + lane;
    const bool in = col < d;
    const int64_t cc = in ? col : d - 1;
    const bool atw = a.placement == AT_WORKER;
    constexpr int kServer = kTRWaves - 1;
    float acc = 0.0f;                              // the server wave's sum of dequantized messages
    // the server's rows of the block's columns (only this block writes them)
    float sm = 0.0f, sv = 0.0f, se = 0.0f, sx = 0.0f;
    if (ROUND && w == kServer && in) {
        if (!atw) {
            sm = a.m[col];
            sv = a.v[col];
        }
        se = a.e_s[col];
        sx = a.x[col];
    }

    for (int g0 = 0; g0 < a.N; g0 += kTRWorkers) {
        const int nw = a.N - g0 < kTRWorkers ? a.N - g0 : kTRWorkers;
        const bool first = g0 == 0;
        const int nout = nw + (first ? 1 : 0);     // output nw is the noise-free gradient (first pass)
        // the worker's rows, loaded now so that they arrive during the sums
        const int64_t wrow = (int64_t)(g0 + (w < nw ? w : 0)) * d + cc;
        float e0 = 0.0f, m0 = 0.0f, v0 = 0.0f;
        if (ROUND && w < nw) {
            e0 = a.e_w[wrow];
            if (atw) {
                m0 = a.m_w[wrow];
                v0 = a.v_w[wrow];
            }
        }
        double s[kTROut];
#pragma unroll
        for (int o = 0; o < kTROut; ++o) s[o] = 0.0;
        const int64_t kb = (int64_t)blockIdx.y * a.split_rows;
        const int64_t ke = d - kb < a.split_rows ? d : kb + a.split_rows;
        for (int64_t k0 = kb; k0 < ke; k0 += ROWS) {
            const int rows = ke - k0 < ROWS ? (int)(ke - k0) : ROWS;
            const int r0 = w * kPer;
            float av[kPer];
#pragma unroll
            for (int j = 0; j < kPer; ++j) av[j] = r0 + j < rows ? a.A[(k0 + r0 + j) * d + cc] : 0.0f;
            __syncthreads();                       // the previous tile has been read
            // every slot of the tile: outputs past nout and rows past the
            // tile's end hold zeros, so the sums below need no guards
            for (int idx = threadIdx.x; idx < kTROut * ROWS; idx += kTRWaves * kWave) {
                const int o = idx / ROWS, kk = idx - o * ROWS;
                double val = 0.0;
                if (kk < rows && o < nout) {
                    const double r = a.res[k0 + kk];
                    val = o < nw ? r - (double)a.xi[(int64_t)(g0 + o) * d + k0 + kk] : r;
                }
                big[kk * kTROut + o] = val;
            }
            __syncthreads();
            const auto row = [&](int j) {
                const double ad = (double)av[j];
                const double2* t = reinterpret_cast<const double2*>(big + (r0 + j) * kTROut);
#pragma unroll
                for (int o2 = 0; o2 < kTROut / 2; ++o2) {
                    const double2 tv = t[o2];
                    s[2 * o2] = fma(ad, tv.x, s[2 * o2]);
                    s[2 * o2 + 1] = fma(ad, tv.y, s[2 * o2 + 1]);
                }
            };
            if (r0 + kPer <= rows) {
#pragma unroll
                for (int j = 0; j < kPer; ++j) row(j);
            } else {
                for (int j = 0; r0 + j < rows; ++j) row(j);
            }
        }
        __syncthreads();                           // every wave is done with the last tile
#pragma unroll
        for (int o = 0; o < kTROut; ++o)
            if (o < nout) big[(w * kTROut + o) * kWave + lane] = s[o];
        __syncthreads();
        double tot = 0.0;
        if (w < nout)
            for (int u = 0; u < kTRWaves; ++u) tot += big[(u * kTROut + w) * kWave + lane];
        if (a.splits > 1) {
            // publish this split's sums; the group's last block adds them all
            constexpr int64_t kSet = kTROut * kWave;
            double* group = a.psum + (int64_t)blockIdx.x * a.splits * kSet;
            // Each wave that stored releases its own stores (a write-back of
            // the L2, no invalidation: the other blocks are still reading A
            // through it); only the group's last block acquires.
            if (w < nout) {
                group[blockIdx.y * kSet + w * kWave + lane] = tot;
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            }
            __syncthreads();
            if (threadIdx.x == 0) {
                const bool last = atomicAdd(a.counter + 1 + blockIdx.x, 1u) == (uint32_t)(a.splits - 1);
                if (last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                last_split = last ? 1 : 0;
            }
            __syncthreads();
            if (!last_split) return;               // the whole block leaves together
            if (w < nout) {
                // all the loads first (one memory latency), then the sums in
                // split order
                const unsigned long long* bits = reinterpret_cast<const unsigned long long*>(group);
                double part[kTRMaxSplits];
#pragma unroll
                for (int r = 0; r < kTRMaxSplits; ++r)
                    part[r] = r < a.splits ? __longlong_as_double((long long)__atomic_load_n(
                                                 bits + r * kSet + w * kWave + lane, __ATOMIC_RELAXED))
                                           : 0.0;
                tot = 0.0;
#pragma unroll
                for (int r = 0; r < kTRMaxSplits; ++r)
                    if (r < a.splits) tot += part[r];
            }
        }
        if (w < nout) {
            const double gd = 2.0 * tot;
            if (w < nw) {
                // worker g0 + w (Algorithm 2 with Adam at the worker, else g + e)
                const float g = (float)gd;
                if (a.g_out != nullptr && in) a.g_out[wrow] = g;
                if constexpr (ROUND) {
                    float p;
                    if (atw) {
                        const float vk = a.beta2 * v0 + (1.0f - a.beta2) * (g * g);
                        const float mk = a.beta1 * m0 + (1.0f - a.beta1) * g;
                        p = (vk > 0.0f ? a.lr * (mk / sqrtf(vk)) : 0.0f) + e0;
                        if (in) {
                            a.m_w[wrow] = mk;
                            a.v_w[wrow] = vk;
                        }
                    } else {
                        p = g + e0;
                    }
                    uint32_t code;
                    float dq;
                    toy_code(a.qw, p, code, dq);
                    if (in) a.e_w[wrow] = a.qw.ef ? p - dq : 0.0f;
                    toy_store_codes(a.qw, a.wcodes + (int64_t)(g0 + w) * a.qw.words, col, in, code);
                    xfer[w * kWave + lane] = dq;
                }
            } else if (a.grad_sq != nullptr) {
                // the noise-free gradient: this column group's share of
                // ||grad F||^2; the last group to get here adds the shares:
                // lane l the shares of groups l, l+64, ... in order (loaded
                // side by side), then the wave's sum
                const double sq = wave_sum(in ? gd * gd : 0.0);
                uint32_t done = 0;
                if (lane == 0) {
                    a.part[blockIdx.x] = sq;
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
                    done = atomicAdd(a.counter, 1u);
                    if (done == gridDim.x - 1) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                }
                done = (uint32_t)__builtin_amdgcn_readfirstlane((int)done);
                if (done == gridDim.x - 1) {
                    double mine = 0.0;
                    const unsigned long long* bits = reinterpret_cast<const unsigned long long*>(a.part);
                    for (uint32_t b = (uint32_t)lane; b < gridDim.x; b += kWave)
                        mine += __longlong_as_double((long long)__atomic_load_n(bits + b, __ATOMIC_RELAXED));
                    const double all = wave_sum(mine);
                    if (lane == 0) *a.grad_sq = all;
                }
            }
        }
        __syncthreads();
        if (ROUND && w == kServer)
            for (int i = 0; i < nw; ++i) acc = acc + xfer[i * kWave + lane];
    }

    if (ROUND && w == kServer) {
        // Algorithm 1: average, [Adam at the server], residual, quantize, apply
        const float fN = (float)a.N;
        const bool pow2 = (a.N & (a.N - 1)) == 0;
        const float avg = pow2 ? acc * (1.0f / fN) : acc / fN;
        float u = avg;
        if (!atw) {
            const float vk = a.beta2 * sv + (1.0f - a.beta2) * (avg * avg);
            const float mk = a.beta1 * sm + (1.0f - a.beta1) * avg;
            u = vk > 0.0f ? a.lr * (mk / sqrtf(vk)) : 0.0f;
            if (in) {
                a.m[col] = mk;
                a.v[col] = vk;
            }
        }
        const float q = u + se;
        uint32_t code;
        float dq;
        toy_code(a.qs, q, code, dq);
        if (in) {
            a.e_s[col] = a.qs.ef ? q - dq : 0.0f;
            a.x[col] = sx - dq;
        }
        toy_store_codes(a.qs, a.scodes, col, in, code);
    }
}

}  // namespace

// r (d doubles), the per-block partial norms (one per 64 columns), the
// fused round's counters (1 + one per column group, as 32-bit words) and its
// splits' column sums.
int64_t toy_workspace_bytes(int64_t d)
{
    const int64_t nblk = (d + kWave - 1) / kWave;
    int64_t rows = 0;
    const int64_t R = toy_splits(d, &rows);
    const int64_t psum = R > 1 ? nblk * R * kTROut * kWave : 0;
    return (d + nblk + (nblk + 2) / 2 + psum) * (int64_t)sizeof(double);
}

namespace {

// The residual launch (which also clears the counters), then the round
// kernel, with the round (ROUND) or writing the gradients only.
template <bool ROUND>
hipError_t launch_toy(ToyArgs& a, const float* xs, const float* x, void* workspace, hipStream_t s)
{
    const int64_t d = a.d;
    const int64_t nblk = (d + kWave - 1) / kWave;
    double* res = static_cast<double*>(workspace);
    a.res = res;
    a.part = res + d;
    a.counter = reinterpret_cast<uint32_t*>(res + d + nblk);
    a.psum = res + d + nblk + (nblk + 2) / 2;
    // several splits only when the workers fit one pass (each pass would
    // need its own sums) and the workspace holds them (toy_workspace_bytes)
    a.splits = a.N <= kTRWorkers ? toy_splits(d, &a.split_rows) : 1;
    if (a.splits == 1) a.split_rows = d;
    hipLaunchKernelGGL(toy_residual_kernel, dim3((unsigned)((d + kResWaves - 1) / kResWaves)),
                       dim3(kResWaves * kWave), 0, s, d, a.A, xs, x, res, a.counter, (int32_t)(1 + nblk));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.splits > 1)
        hipLaunchKernelGGL((toy_round_kernel<kTRSplitRows, ROUND>), dim3((unsigned)nblk, (unsigned)a.splits),
                           dim3(kTRWaves * kWave), 0, s, a);
    else
        hipLaunchKernelGGL((toy_round_kernel<kTRRows, ROUND>), dim3((unsigned)nblk), dim3(kTRWaves * kWave), 0, s,
                           a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_toy_grad(int64_t d, int32_t N, const float* A, const float* xs, const float* xi, const float* x,
                           float* g, double* grad_sq, void* workspace, hipStream_t s)
{
    ToyArgs a{};
    a.d = d;
    a.N = N;
    a.A = A;
    a.xi = xi;
    a.g_out = g;
    a.grad_sq = grad_sq;
    return launch_toy<false>(a, xs, x, workspace, s);
}

hipError_t launch_toy_step(const StepArgs& sa, const float* A, const float* xs, const float* xi, double* grad_sq,
                           float* g_out, void* workspace, hipStream_t s)
{
    ToyArgs a{};
    a.d = sa.d;
    a.N = sa.N;
    a.placement = sa.placement;
    a.beta1 = sa.beta1;
    a.beta2 = sa.beta2;
    a.lr = sa.lr;
    a.qw = sa.qw;
    a.qs = sa.qs;
    a.A = A;
    a.xi = xi;
    a.x = sa.x;
    a.e_w = sa.e_w;
    a.m_w = sa.m_w;
    a.v_w = sa.v_w;
    a.m = sa.m;
    a.v = sa.v;
    a.e_s = sa.e_s;
    a.wcodes = sa.wcodes;
    a.scodes = sa.scodes;
    a.grad_sq = grad_sq;
    a.g_out = g_out;
    return launch_toy<true>(a, xs, sa.x, workspace, s);
}

}  // namespace ea
