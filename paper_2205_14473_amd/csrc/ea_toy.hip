// ea_toy.hip -- gradients of the toy problem of Section V-A on the device:
// f(x) = E_xi || A x - (x* + xi) ||^2, whose gradient for a noise draw xi_i is
// g_i = 2 A^T (A x - x* - xi_i).  Products are summed in binary64 and each g
// rounded once to binary32, like the oracle.  Three launches:
//   1. residual: res[k] = (A x)[k] - x*[k], one wave per row of A;
//   2. columns:  blocks of 64 columns x up to 8 workers; the 16 waves of a
//      block take 16 contiguous ranges of k, their partial sums meet in LDS
//      and are added in wave order; block (b, 0) also forms the noise-free
//      gradient and the partial sum of its squares for its columns;
//   3. norm: the per-block partial sums added in block order.
#include "ea_launch.hpp"

namespace ea {

namespace {

constexpr int kResWaves = 4;                    // rows per residual block
constexpr int kColThreads = 1024;
constexpr int kColWaves = kColThreads / kWave;
constexpr int kToyWorkers = 8;                  // workers per column block
constexpr int kToyOut = kToyWorkers + 1;        // + the noise-free gradient

__global__ __launch_bounds__(kResWaves * kWave) void toy_residual_kernel(int64_t d, const float* __restrict__ A,
                                                                         const float* __restrict__ xs,
                                                                         const float* __restrict__ x,
                                                                         double* __restrict__ res)
{
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

__global__ __launch_bounds__(kColThreads) void toy_columns_kernel(int64_t d, int32_t N, const float* __restrict__ A,
                                                                 const double* __restrict__ res,
                                                                 const float* __restrict__ xi,
                                                                 float* __restrict__ g, double* __restrict__ part)
{
    __shared__ double sums[kColWaves][kToyOut][kWave];
    const int lane = lane_id();
    const int w = (int)(threadIdx.x / kWave);
    const int64_t j = (int64_t)blockIdx.x * kWave + lane;
    const int i0 = (int)blockIdx.y * kToyWorkers;
    const int W = N - i0 < kToyWorkers ? N - i0 : kToyWorkers;
    const bool full = blockIdx.y == 0 && part != nullptr;
    const int64_t per = (d + kColWaves - 1) / kColWaves;
    const int64_t k0 = (int64_t)w * per;
    const int64_t k1 = k0 + per < d ? k0 + per : d;

    double acc[kToyOut];
#pragma unroll
    for (int c = 0; c < kToyOut; ++c) acc[c] = 0.0;
    if (j < d) {
#pragma unroll 4
        for (int64_t k = k0; k < k1; ++k) {
            const double a = (double)A[k * d + j];
            const double r0 = res[k];
            if (full) acc[0] += a * r0;
#pragma unroll
            for (int c = 0; c < kToyWorkers; ++c)
                if (c < W) acc[c + 1] += a * (r0 - (double)xi[(int64_t)(i0 + c) * d + k]);
        }
    }
#pragma unroll
    for (int c = 0; c < kToyOut; ++c) sums[w][c][lane] = acc[c];
    __syncthreads();
    if (w > W) return;
    double s = 0.0;
    for (int u = 0; u < kColWaves; ++u) s += sums[u][w][lane];
    if (w > 0) {
        if (j < d) g[(int64_t)(i0 + w - 1) * d + j] = (float)(2.0 * s);
        return;
    }
    if (!full) return;
    const double gj = 2.0 * s;
    double sq = j < d ? gj * gj : 0.0;
    sq = wave_sum(sq);
    if (lane == 0) part[blockIdx.x] = sq;
}

__global__ __launch_bounds__(kWave) void toy_norm_kernel(int64_t nparts, const double* __restrict__ part,
                                                         double* __restrict__ grad_sq)
{
    if (threadIdx.x != 0) return;
    double s = 0.0;
    for (int64_t b = 0; b < nparts; ++b) s += part[b];
    *grad_sq = s;
}

}  // namespace

int64_t toy_workspace_bytes(int64_t d)
{
    return (d + (d + kWave - 1) / kWave) * (int64_t)sizeof(double);
}

hipError_t launch_toy_grad(int64_t d, int32_t N, const float* A, const float* xs, const float* xi, const float* x,
                           float* g, double* grad_sq, void* workspace, hipStream_t s)
{
    double* res = static_cast<double*>(workspace);
    const int64_t ncol = (d + kWave - 1) / kWave;
    double* part = grad_sq ? res + d : nullptr;
    hipLaunchKernelGGL(toy_residual_kernel, dim3((unsigned)((d + kResWaves - 1) / kResWaves)),
                       dim3(kResWaves * kWave), 0, s, d, A, xs, x, res);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(toy_columns_kernel, dim3((unsigned)ncol, (unsigned)((N + kToyWorkers - 1) / kToyWorkers)),
                       dim3(kColThreads), 0, s, d, N, A, res, xi, g, part);
    e = hipGetLastError();
    if (e != hipSuccess || !grad_sq) return e;
    hipLaunchKernelGGL(toy_norm_kernel, dim3(1), dim3(kWave), 0, s, ncol, part, grad_sq);
    return hipGetLastError();
}

}  // namespace ea
