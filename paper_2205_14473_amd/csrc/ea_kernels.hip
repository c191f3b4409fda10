// ea_kernels.hip -- the generic and fully specialized fused-round kernels,
// the split calls' kernels, and the launchers (dispatch to the kernel that
// matches a configuration).  The round itself is in ea_round.hpp.
#include "ea_round.hpp"

#include <mutex>

namespace ea {

namespace {

// Per-tile partial norms of the worker inputs p for workers [i0, i1), without
// writing any state (one-bucket Q_w).  Rows are [i - i0][d] from a.g etc.
template <int C, bool VEC>
__global__ __launch_bounds__(kBlock) void worker_partials_kernel(StepArgs args, int i0, int i1)
{
    const StepArgs a = with_step(args);
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    const bool atw = a.placement == AT_WORKER;
    for (int i = i0; i < i1; ++i) {
        const int64_t row = (int64_t)(i - i0) * a.d;
        WorkerRows<C> r;
        float4 p[C];
        load_worker<C, VEC, false, -1>(a, a.g + row, a.e_w + row, atw ? a.m_w + row : nullptr,
                                       atw ? a.v_w + row : nullptr, t.base, t.nch, r);
        worker_p<C, -1>(a, r, p);
        const double part = tile_partial<C>(a.qw, p, t.base, t.nch, a.d);
        if (lane_id() == 0) a.wpart[(int64_t)(i - i0) * a.ntiles + t.tile] = part;
    }
}

// Per-tile partial norms of q = u + e_s (one-bucket Q_s, split call).
template <int C, bool VEC>
__global__ __launch_bounds__(kBlock) void server_partials_kernel(StepArgs a)
{
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    const int lane = lane_id();
    float4 q[C];
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        q[ch] = zero4();
        if (ch >= t.nch) continue;
        const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
        q[ch] = add4(ld4<VEC>(a.ubuf, n, a.d), ld4<VEC>(a.e_s, n, a.d));
    }
    const double part = tile_partial<C>(a.qs, q, t.base, t.nch, a.d);
    if (lane == 0) a.spart[t.tile] = part;
}

// Reduce per-tile partials to one scale per vector: block v handles
// part[v*ntiles .. (v+1)*ntiles) and writes out[v*out_stride].
__global__ __launch_bounds__(kBlock) void finalize_kernel(const double* __restrict__ part, int64_t ntiles,
                                                          int32_t norm, int64_t n, float* __restrict__ out,
                                                          int64_t out_stride)
{
    __shared__ double red[kWavesPerBlock];
    const double* pv = part + (int64_t)blockIdx.x * ntiles;
    double acc = 0.0;
    for (int64_t j = threadIdx.x; j < ntiles; j += blockDim.x)
        acc = norm == S_MAX ? fmax(acc, pv[j]) : acc + pv[j];
    if (norm == S_MAX) {
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) acc = fmax(acc, __shfl_xor(acc, o, kWave));
    } else {
        acc = wave_sum(acc);
    }
    if (lane_id() == 0) red[threadIdx.x / kWave] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        double tot = red[0];
        for (int w = 1; w < kWavesPerBlock; ++w) tot = norm == S_MAX ? fmax(tot, red[w]) : tot + red[w];
        out[(int64_t)blockIdx.x * out_stride] = scale_from(norm, tot, (float)tot, n);
    }
}

__global__ void fill_kernel(float* __restrict__ p, int64_t n, float value)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = value;
}

__global__ void advance_kernel(uint32_t* t_dev)
{
    if (threadIdx.x == 0) t_dev[0] = t_dev[0] + 1u;
}

int64_t grid_of(const StepArgs& a)
{
    return (a.ntiles + kWavesPerBlock - 1) / kWavesPerBlock;
}

// Dispatch on (C, VEC) to a generic kernel template instance.
#define EA_DISPATCH(KERNEL, C, VEC, GRID, STREAM, ...)                                              \
    do {                                                                                           \
        switch ((C) * 2 + ((VEC) ? 1 : 0)) {                                                       \
        case 2: hipLaunchKernelGGL((KERNEL<1, false>), dim3(GRID), dim3(kBlock), 0, STREAM, __VA_ARGS__); break; \
        case 3: hipLaunchKernelGGL((KERNEL<1, true>), dim3(GRID), dim3(kBlock), 0, STREAM, __VA_ARGS__); break;  \
        case 4: hipLaunchKernelGGL((KERNEL<2, false>), dim3(GRID), dim3(kBlock), 0, STREAM, __VA_ARGS__); break; \
        case 5: hipLaunchKernelGGL((KERNEL<2, true>), dim3(GRID), dim3(kBlock), 0, STREAM, __VA_ARGS__); break;  \
        case 8: hipLaunchKernelGGL((KERNEL<4, false>), dim3(GRID), dim3(kBlock), 0, STREAM, __VA_ARGS__); break; \
        case 9: hipLaunchKernelGGL((KERNEL<4, true>), dim3(GRID), dim3(kBlock), 0, STREAM, __VA_ARGS__); break;  \
        case 16: hipLaunchKernelGGL((KERNEL<8, false>), dim3(GRID), dim3(kBlock), 0, STREAM, __VA_ARGS__); break; \
        case 17: hipLaunchKernelGGL((KERNEL<8, true>), dim3(GRID), dim3(kBlock), 0, STREAM, __VA_ARGS__); break;  \
        default: return hipErrorInvalidValue;                                                      \
        }                                                                                          \
    } while (0)

// Specialized fused rounds: (chunks per tile, worker traits, server traits,
// placement), chosen when the configuration matches exactly and rows are
// 16-byte aligned.
using SignQ8 = QCt<Q_SCALED_SIGN, 1, S_L1, 8>;
using SignQ4 = QCt<Q_SCALED_SIGN, 1, S_L1, 4>;
using SignQ2 = QCt<Q_SCALED_SIGN, 1, S_L1, 2>;
using Stoch4L2Q2 = QCt<Q_STOCH, 4, S_L2, 2>;
using Stoch2MaxQ2 = QCt<Q_STOCH, 2, S_MAX, 2>;
using Stoch2MaxQ4 = QCt<Q_STOCH, 2, S_MAX, 4>;
using TopKQ2 = QCt<Q_TOPK, 1, S_MAX, 2>;
using RandKQ2 = QCt<Q_RANDK, 1, S_MAX, 2>;

struct Special {
    int C;
    int wkind, wbits, wnorm, wcpb;
    int skind, sbits, snorm, scpb;
    int placement;
    void (*kernel)(StepArgs);   // whole tiles
    void (*edge)(StepArgs);     // the ragged last tile
    int tiles;                  // tiles per block of `kernel`
};

#define EA_SPECIAL(CC, QWT, QST, PLC)                                                               \
    Special{CC, QWT::kind(QDev{}), QWT::bits(QDev{}), QWT::norm(QDev{}), QWT::cpb(QDev{}),         \
            QST::kind(QDev{}), QST::bits(QDev{}), QST::norm(QDev{}), QST::cpb(QDev{}), PLC,         \
            step_kernel<CC, true, true, QWT, QST, PLC>, step_kernel<CC, true, false, QWT, QST, PLC>,         \
            round_tiles_per_block(CC, PLC == AT_SERVER)}

const Special kSpecials[] = {
    EA_SPECIAL(2, Stoch4L2Q2, Stoch4L2Q2, AT_SERVER),
    EA_SPECIAL(2, Stoch4L2Q2, Stoch4L2Q2, AT_WORKER),
    EA_SPECIAL(2, Stoch2MaxQ2, Stoch2MaxQ2, AT_SERVER),
    EA_SPECIAL(2, Stoch2MaxQ2, Stoch2MaxQ2, AT_WORKER),
    EA_SPECIAL(8, SignQ8, SignQ8, AT_SERVER),
    EA_SPECIAL(8, SignQ8, SignQ8, AT_WORKER),
    EA_SPECIAL(4, Stoch2MaxQ4, SignQ4, AT_SERVER),
    EA_SPECIAL(4, Stoch2MaxQ4, SignQ4, AT_WORKER),
    EA_SPECIAL(2, SignQ2, SignQ2, AT_SERVER),
    EA_SPECIAL(2, TopKQ2, TopKQ2, AT_SERVER),
    EA_SPECIAL(2, RandKQ2, RandKQ2, AT_SERVER),
};

const Special* find_special(const StepArgs& a, int C)
{
    for (const Special& s : kSpecials) {
        if (s.C == C && s.placement == a.placement && s.wkind == a.qw.kind && s.wbits == a.qw.bits &&
            s.wnorm == a.qw.norm && s.wcpb == a.qw.cpb && s.skind == a.qs.kind && s.sbits == a.qs.bits &&
            s.snorm == a.qs.norm && s.scpb == a.qs.cpb)
            return &s;
    }
    return nullptr;
}

// The specialized tables' entry for quantizer q at tile size C, when one
// matches: tiles of one bucket of q each, or of any size for a quantizer
// without buckets (Example 2, full precision).  find_half keys on the worker
// quantizer (the fused round and the split worker calls); the split server
// calls key on the server's.
const HalfKernel* find_half_for(const QDev& q, int C)
{
    const bool bucketless = q.kind == Q_POW2 || q.kind == Q_NONE;
    if (q.cpb != (bucketless ? 0 : C)) return nullptr;
    int n = 0;
    const HalfKernel* t = C == 1 ? half_kernels_c1(&n) : C == 2 ? half_kernels_c2(&n)
                        : C == 4 ? half_kernels_c4(&n) : C == 8 ? half_kernels_c8(&n) : nullptr;
    for (int i = 0; i < n; ++i) {
        const HalfKernel& h = t[i];
        if (h.C == C && h.wkind == q.kind && h.wbits == q.bits && h.wnorm == q.norm && h.wcpb == q.cpb) return &h;
    }
    return nullptr;
}

const HalfKernel* find_half(const StepArgs& a, int C)
{
    return find_half_for(a.qw, C);
}

// A fully specialized kernel for a wide tile with the same quantizer on both
// sides and Adam at the server, when one matches.
const SymKernel* find_sym(const StepArgs& a, int C)
{
    if (a.placement != AT_SERVER || (C != 4 && C != 8)) return nullptr;
    const QDev& w = a.qw;
    const QDev& v = a.qs;
    if (w.kind != v.kind || w.bits != v.bits || w.norm != v.norm || w.cpb != v.cpb || w.cpb != C) return nullptr;
    int n = 0;
    const SymKernel* t = C == 4 ? sym_kernels_c4(&n) : sym_kernels_c8(&n);
    for (int i = 0; i < n; ++i)
        if (t[i].kind == w.kind && t[i].bits == w.bits && t[i].norm == w.norm && t[i].cpb == w.cpb) return &t[i];
    return nullptr;
}

}  // namespace

namespace {

hipError_t launch_step_main(const StepArgs& a, int C, int64_t nfull, const Special* sp, const SymKernel* sk,
                            const HalfKernel* hk, size_t limit, hipStream_t s);
hipError_t launch_step_edge(const StepArgs& a, int C, int64_t nfull, const Special* sp, const SymKernel* sk,
                            size_t limit, hipStream_t s);

// Waves per block of a fused-round launch: one per worker up to the tile's
// limit, and at least one per tile of the block, since wave k serves tile k
// (with fewer workers than tiles the other waves only serve).  Fully
// specialized 8-chunk tiles serve a whole-tile server bucket, or a
// sparsifier's server side, on C waves, one chunk each (SplitServe,
// SparseServe; whole and ragged tiles alike), so their blocks have C waves
// at least.
int step_waves(const StepArgs& a, int C, int K, const Special* sp, const SymKernel* sk, size_t limit)
{
    int G = round_waves(a.N, C, K, limit, a.placement);
    if (G < K) G = K;
    const bool scaled = a.qs.cpb == C &&
                        (a.qs.kind == Q_SCALED_SIGN || a.qs.kind == Q_STOCH || a.qs.kind == Q_DET);
    const bool sparse = a.qs.kind == Q_TOPK || a.qs.kind == Q_RANDK;
    const bool split = (sp || sk) && C == 8 && (scaled || sparse);
    return split && G < C ? C : G;
}

// Rows whose byte length is not a multiple of 128 share a cache line between
// adjacent tiles.  Whole-tile launches of one tile per block then deal runs
// of this many adjacent tiles to each XCD (block_slot): ResNet-18-sized
// round 0.2930 -> 0.2847 ms (runs of 8: 0.2880, 32: 0.2863).  With two
// tiles per block the pair's shared line is inside the block already, and
// runs measured slower (ResNet-50-sized 2.108 -> 2.155-2.187 ms).
#ifndef EA_XCD_RUN
#define EA_XCD_RUN 16
#endif

// Tiles per block of the whole-tile launch.
int main_tiles_per_block(int C, const Special* sp, const SymKernel* sk, const HalfKernel* hk)
{
    return sp ? sp->tiles : sk ? sk->tiles : hk ? hk->tiles : round_tiles_per_block(C, false);
}

// A second stream per device for the ragged last tile (see launch_step).
// Default priority, non-blocking with respect to the null stream.
struct SideStream {
    hipStream_t stream = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
    bool tried = false, ok = false;
};
constexpr int kMaxSideDevices = 64;
std::mutex g_side_mu;
SideStream g_side[kMaxSideDevices];

// The current device's side stream, created on first use; nullptr if it
// cannot be had.  Called with g_side_mu held.
SideStream* device_side_stream()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxSideDevices) return nullptr;
    SideStream& ss = g_side[dev];
    if (!ss.tried) {
        ss.tried = true;
        ss.ok = hipStreamCreateWithFlags(&ss.stream, hipStreamNonBlocking) == hipSuccess &&
                hipEventCreateWithFlags(&ss.fork, hipEventDisableTiming) == hipSuccess &&
                hipEventCreateWithFlags(&ss.join, hipEventDisableTiming) == hipSuccess;
    }
    return ss.ok ? &ss : nullptr;
}

// Runs main(s) and edge(t): with `allow` and when s is not being captured, t
// is the device's side stream, forked from s before both launches and joined
// back to s after them; otherwise both go to s in order.  main and edge must
// touch disjoint memory.
template <class Main, class Edge>
hipError_t run_beside(hipStream_t s, bool allow, const Main& main, const Edge& edge)
{
    if (allow) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusActive;
        if (hipStreamIsCapturing(s, &cs) == hipSuccess && cs == hipStreamCaptureStatusNone) {
            std::lock_guard<std::mutex> lock(g_side_mu);
            if (SideStream* ss = device_side_stream()) {
                hipError_t e = hipEventRecord(ss->fork, s);
                if (e == hipSuccess) e = hipStreamWaitEvent(ss->stream, ss->fork, 0);
                if (e != hipSuccess) return e;
                e = edge(ss->stream);
                if (e == hipSuccess) e = main(s);
                // joined even after a failed launch, so that s never runs ahead of the side stream
                const hipError_t r = hipEventRecord(ss->join, ss->stream);
                const hipError_t w = r == hipSuccess ? hipStreamWaitEvent(s, ss->join, 0) : r;
                return e != hipSuccess ? e : w;
            }
        }
    }
    const hipError_t e = main(s);
    return e == hipSuccess ? edge(s) : e;
}

}  // namespace

// Whole tiles go to a kernel without bounds checks: one specialized for both
// quantizers and the placement when one matches, else one specialized for
// the worker quantizer, else the generic one.  The ragged last tile goes to a
// checked kernel, specialized in the first case.  Every tile of rows that are
// not 16-byte aligned goes to the generic checked kernel.
//
// The ragged tile is one block whose latency would add in full to the round
// if it were queued behind the whole-tile launch (about 23 us of a 0.31 ms
// ResNet-18-sized round).  The two launches touch disjoint elements, message
// words and scales, so the ragged tile runs on a side stream forked from the
// caller's stream before both launches and joined back after them; the
// caller's stream then holds both.  That pays while the whole-tile launch is
// short (ResNet-18-sized round 0.306 -> 0.296 ms, ResNet-50-sized 2.160 ->
// 2.130 ms); on the long launches it did not (BERT-sized unchanged at 4.57
// ms, GPT-2-medium-sized 7.83 -> 7.93 ms), so those queue both launches in
// order, as does every launch under stream capture.
constexpr int64_t kSideStreamMaxBlocks = 32768;

hipError_t launch_step(const StepArgs& a, int C, bool vec, hipStream_t s, bool side_stream)
{
    const size_t limit = lds_limit_bytes();
    const Special* sp = vec ? find_special(a, C) : nullptr;
    const SymKernel* sk = vec && !sp ? find_sym(a, C) : nullptr;
    const HalfKernel* hk = vec && !sp && !sk ? find_half(a, C) : nullptr;
    // The whole-tile launch takes a multiple of its tiles per block (its
    // kernels assume full blocks); the whole tiles left over go to the checked
    // launch with the ragged one.
    const int K = main_tiles_per_block(C, sp, sk, hk);
    const int64_t nfull = vec ? a.d / ((int64_t)C * kChunk) / K * K : 0;
    const bool has_main = nfull > 0, has_edge = nfull < a.ntiles;
    const int64_t main_blocks = nfull / K;
    if (has_main && has_edge)
        return run_beside(
            s, side_stream && main_blocks < kSideStreamMaxBlocks,
            [&](hipStream_t t) { return launch_step_main(a, C, nfull, sp, sk, hk, limit, t); },
            [&](hipStream_t t) { return launch_step_edge(a, C, nfull, sp, sk, limit, t); });
    if (has_main) return launch_step_main(a, C, nfull, sp, sk, hk, limit, s);
    return has_edge ? launch_step_edge(a, C, nfull, sp, sk, limit, s) : hipSuccess;
}

namespace {

// One dispatch covers at most 2^32 - 1 work-items, and the fused kernels run
// up to four threads per element (one-chunk tiles, 16 waves, one tile per
// block), so a whole-tile launch is issued in pieces of at most this many
// blocks (2^30 threads): one piece up to d = 2^28 in that shape, 2^30 in
// the BERT-sized one.  Pieces are multiples of 128 blocks, so the XCD runs
// of block_slot keep their groups.
constexpr int64_t kMaxLaunchBlocks = (int64_t)1 << 20;

// The whole tiles [0, nfull) of a round, nfull a multiple of the kernel's
// tiles per block (launch_step).
hipError_t launch_step_main(const StepArgs& a, int C, int64_t nfull, const Special* sp, const SymKernel* sk,
                            const HalfKernel* hk, size_t limit, hipStream_t s)
{
    const int K = main_tiles_per_block(C, sp, sk, hk);
    const int G = step_waves(a, C, K, sp, sk, limit);
    StepArgs b = a;
    const int bufs = handoff_bufs(a.N, C, G, K, limit);
    b.one_buffer = bufs == 1 ? 1 : 0;
    b.xcd_run = (a.d * 4) % 128 != 0 && K == 1 ? EA_XCD_RUN : 1;
    const dim3 block((unsigned)(G * kWave));
    const size_t lds = round_lds_bytes(a.N, C, G, K, bufs);
    const int64_t nblocks = nfull / K;
    for (int64_t b0 = 0; b0 < nblocks; b0 += kMaxLaunchBlocks) {
        const int64_t nb = nblocks - b0 < kMaxLaunchBlocks ? nblocks - b0 : kMaxLaunchBlocks;
        b.tile0 = b0 * K;
        b.tile1 = (b0 + nb) * K;
        const dim3 grid((unsigned)nb);
        if (sp) {
            hipLaunchKernelGGL(sp->kernel, grid, block, lds, s, b);
        } else if (sk) {
            hipLaunchKernelGGL(sk->kernel, grid, block, lds, s, b);
        } else if (hk) {
            hipLaunchKernelGGL(hk->kernel, grid, block, lds, s, b);
        } else {
            switch (C) {
            case 1: hipLaunchKernelGGL((step_kernel<1, true, true, QRt, QRt, -1>), grid, block, lds, s, b); break;
            case 2: hipLaunchKernelGGL((step_kernel<2, true, true, QRt, QRt, -1>), grid, block, lds, s, b); break;
            case 4: hipLaunchKernelGGL((step_kernel<4, true, true, QRt, QRt, -1>), grid, block, lds, s, b); break;
            case 8: hipLaunchKernelGGL((step_kernel<8, true, true, QRt, QRt, -1>), grid, block, lds, s, b); break;
            default: return hipErrorInvalidValue;
            }
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// The tiles [nfull, ntiles) of a round (at most one short of a whole-tile
// block, plus the ragged one), one block each, with bounds checks
// (launch_step).
hipError_t launch_step_edge(const StepArgs& a, int C, int64_t nfull, const Special* sp, const SymKernel* sk,
                            size_t limit, hipStream_t s)
{
    const int G = step_waves(a, C, 1, sp, sk, limit);
    StepArgs b = a;
    const int bufs = handoff_bufs(a.N, C, G, 1, limit);
    b.one_buffer = bufs == 1 ? 1 : 0;
    b.xcd_run = 1;
    const dim3 block((unsigned)(G * kWave));
    const size_t lds = round_lds_bytes(a.N, C, G, 1, bufs);
    // one tile per block; every tile of a round with unaligned rows comes
    // here, so the launch is issued in pieces as the whole-tile one is
    for (int64_t t0 = nfull; t0 < a.ntiles; t0 += kMaxLaunchBlocks) {
        b.tile0 = t0;
        b.tile1 = a.ntiles - t0 < kMaxLaunchBlocks ? a.ntiles : t0 + kMaxLaunchBlocks;
        const dim3 grid((unsigned)(b.tile1 - b.tile0));
        if (sp) {
            hipLaunchKernelGGL(sp->edge, grid, block, lds, s, b);
        } else if (sk) {
            hipLaunchKernelGGL(sk->edge, grid, block, lds, s, b);
        } else {
            switch (C) {
            case 1: hipLaunchKernelGGL((step_kernel<1, false, false, QRt, QRt, -1>), grid, block, lds, s, b); break;
            case 2: hipLaunchKernelGGL((step_kernel<2, false, false, QRt, QRt, -1>), grid, block, lds, s, b); break;
            case 4: hipLaunchKernelGGL((step_kernel<4, false, false, QRt, QRt, -1>), grid, block, lds, s, b); break;
            case 8: hipLaunchKernelGGL((step_kernel<8, false, false, QRt, QRt, -1>), grid, block, lds, s, b); break;
            default: return hipErrorInvalidValue;
            }
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_worker_partials(const StepArgs& a, int C, bool vec, int i0, int i1, hipStream_t s)
{
    EA_DISPATCH(worker_partials_kernel, C, vec, grid_of(a), s, a, i0, i1);
    return hipGetLastError();
}

hipError_t launch_server_partials(const StepArgs& a, int C, bool vec, hipStream_t s)
{
    EA_DISPATCH(server_partials_kernel, C, vec, grid_of(a), s, a);
    return hipGetLastError();
}

hipError_t launch_finalize(const double* part, int64_t ntiles, int32_t norm, int64_t n, float* out,
                           int64_t out_stride, int nvec, hipStream_t s)
{
    hipLaunchKernelGGL(finalize_kernel, dim3(nvec), dim3(kBlock), 0, s, part, ntiles, norm, n, out, out_stride);
    return hipGetLastError();
}

// The split calls on the worker side use a kernel specialized for the worker
// quantizer when one matches and rows are aligned, else the generic one.
hipError_t launch_worker(const StepArgs& a, int C, bool vec, hipStream_t s)
{
    const HalfKernel* hk = vec ? find_half(a, C) : nullptr;
    if (hk) {
        hipLaunchKernelGGL(hk->worker, dim3((unsigned)grid_of(a)), dim3(kBlock), 0, s, a);
        return hipGetLastError();
    }
    EA_DISPATCH(worker_kernel, C, vec, grid_of(a), s, a);
    return hipGetLastError();
}

// Worker-specialized aggregates for tiles of up to four chunks take the tiles
// that lie wholly inside d with a kernel without per-tile checks (BERT-sized
// round, 4-bit codes: 652 -> 585 us) and the ragged last tile with a checked
// one.  For 8-chunk tiles the checked kernel is faster (ResNet-18-sized: 54
// against 62 us): without the per-chunk selects the compiler folds the next
// worker's prefetch into the next iteration, where it is waited for at once.
hipError_t launch_aggregate(const StepArgs& a, int C, bool vec, hipStream_t s)
{
    const HalfKernel* hk = vec ? find_half(a, C) : nullptr;
    if (hk) {
        const int64_t nfull = C <= 4 ? a.d / ((int64_t)C * kChunk) : 0;
        const auto full = [&](hipStream_t t) {
            StepArgs b = a;
            b.tile0 = 0;
            b.ntiles = nfull;
            hipLaunchKernelGGL(hk->aggregate_full, dim3((unsigned)grid_of(b)), dim3(kBlock), 0, t, b);
            return hipGetLastError();
        };
        const auto rest = [&](hipStream_t t) {
            StepArgs b = a;
            b.tile0 = nfull;
            hipLaunchKernelGGL(hk->aggregate, dim3((unsigned)((a.ntiles - nfull + kWavesPerBlock - 1) / kWavesPerBlock)),
                               dim3(kBlock), 0, t, b);
            return hipGetLastError();
        };
        // The ragged tile stays on s after the whole tiles: on a side stream it
        // measured slower (BERT-sized split round 4.447 -> 4.456 ms,
        // ResNet-50-sized 2.024 -> 2.046 ms).
        if (nfull > 0) {
            const hipError_t e = full(s);
            if (e != hipSuccess || nfull == a.ntiles) return e;
        }
        return rest(s);
    }
    EA_DISPATCH(aggregate_kernel, C, vec, grid_of(a), s, a);
    return hipGetLastError();
}

// The split server calls take the worker-specialized tables' kernels for the
// server quantizer when it is one of theirs.
hipError_t launch_server(const StepArgs& a, int C, bool vec, hipStream_t s)
{
    const HalfKernel* hk = vec ? find_half_for(a.qs, C) : nullptr;
    if (hk) {
        hipLaunchKernelGGL(hk->server, dim3((unsigned)grid_of(a)), dim3(kBlock), 0, s, a);
        return hipGetLastError();
    }
    EA_DISPATCH(server_kernel, C, vec, grid_of(a), s, a);
    return hipGetLastError();
}

hipError_t launch_apply(const StepArgs& a, int C, bool vec, hipStream_t s)
{
    const HalfKernel* hk = vec ? find_half_for(a.qs, C) : nullptr;
    if (hk) {
        hipLaunchKernelGGL(hk->apply, dim3((unsigned)grid_of(a)), dim3(kBlock), 0, s, a);
        return hipGetLastError();
    }
    EA_DISPATCH(apply_kernel, C, vec, grid_of(a), s, a);
    return hipGetLastError();
}

hipError_t launch_advance(uint32_t* t_dev, hipStream_t s)
{
    hipLaunchKernelGGL(advance_kernel, dim3(1), dim3(kWave), 0, s, t_dev);
    return hipGetLastError();
}

hipError_t launch_fill(float* p, int64_t n, float value, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    int64_t blocks = (n + 1023) / 1024;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n, value);
    return hipGetLastError();
}

}  // namespace ea
