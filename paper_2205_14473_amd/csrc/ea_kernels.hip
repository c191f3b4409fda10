// ea_kernels.hip -- HIP kernels of one Efficient-Adam round for gfx950.
//
// Work decomposition: one wave64 owns one tile of C chunks (C*256 elements);
// a block holds 4 independent waves.  Bucket norms are reduced inside the
// wave (no LDS, no barrier); codes are bit-plane packed with one ballot per
// 64-element plane word.  The fused step streams the N workers of a tile in
// ascending worker order, keeps the dequantized sum in registers, and runs
// the server's Adam, quantization and the parameter update on the same tile
// (Algorithms 1-2, Section IV).
#include "ea_launch.hpp"

namespace ea {

namespace {

// Number of valid elements among lane's float4 at element n.
__device__ __forceinline__ int nvalid4(int64_t n, int64_t d)
{
    const int64_t r = d - n;
    return r <= 0 ? 0 : (r >= 4 ? 4 : (int)r);
}

// ---------------------------------------------------------------------------
// Quantize one tile: scales (reduced per bucket inside the wave, or given for
// a one-bucket quantizer), codes, bit-plane packing and the dequantized
// values.  codes/scales point at the start of the message.
// ---------------------------------------------------------------------------
template <int C>
__device__ __forceinline__ void quantize_tile(const QDev& q, const float* lut, const float4 (&p)[C],
                                              int64_t base, int nch, int64_t d, uint32_t k0, uint32_t k1,
                                              uint32_t step, uint32_t sid, float given_scale,
                                              uint64_t* __restrict__ codes, float* __restrict__ scales,
                                              float4 (&deq)[C])
{
    const int lane = lane_id();
    float s[C];
    if (has_scale(q)) {
        if (q.cpb == 0) {
#pragma unroll
            for (int ch = 0; ch < C; ++ch) s[ch] = given_scale;
        } else {
            Partial part[C];
#pragma unroll
            for (int ch = 0; ch < C; ++ch) {
                part[ch].sum = 0.0;
                part[ch].mx = 0.0f;
                if (ch < nch) partial_add4(part[ch], q.norm, p[ch], nvalid4(base + ch * kChunk + 4 * lane, d));
            }
#pragma unroll
            for (int ch = 0; ch < C; ++ch) {
                if (ch % q.cpb == 0) {
                    if (ch < nch) {
                        Partial tot;
                        tot.sum = 0.0;
                        tot.mx = 0.0f;
#pragma unroll
                        for (int j = 0; j < C; ++j) {
                            if (j >= ch && j < ch + q.cpb) {
                                tot.sum += part[j].sum;
                                tot.mx = fmaxf(tot.mx, part[j].mx);
                            }
                        }
                        const int64_t b0 = base + (int64_t)ch * kChunk;
                        const int64_t nb = (d - b0) < q.B ? (d - b0) : q.B;
                        const double S = q.norm == S_MAX ? 0.0 : wave_sum(tot.sum);
                        const float M = q.norm == S_MAX ? wave_max(tot.mx) : 0.0f;
                        s[ch] = scale_from(q.norm, S, M, nb);
                        if (lane == 0) scales[b0 / q.B] = s[ch];
                    } else {
                        s[ch] = 0.0f;
                    }
                } else {
                    s[ch] = s[ch > 0 ? ch - 1 : 0];
                }
            }
        }
    } else {
#pragma unroll
        for (int ch = 0; ch < C; ++ch) s[ch] = 1.0f;
    }

    uint32_t c[C][4];
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        const int nv = ch < nch ? nvalid4(n, d) : 0;
        const float sc = s[ch];
        const bool ok = sc > 0.0f && !isinf(sc);
        const float inv = ok ? 1.0f / sc : 0.0f;
        uint4 r = make_uint4(0u, 0u, 0u, 0u);
        if (q.kind == Q_STOCH && ch < nch) {
            const uint64_t j = (uint64_t)n >> 2;
            r = philox10(make_uint4((uint32_t)j, (uint32_t)(j >> 32), step, sid), k0, k1);
        }
        const uint32_t rr[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float x = comp(p[ch], k);
            const bool valid = k < nv;
            const uint32_t cc = valid ? code_of(q, x, inv, ok, u24(rr[k])) : 0u;
            c[ch][k] = cc;
            set_comp(deq[ch], k, valid ? deq_of(q, lut, cc, x, sc, ok) : 0.0f);
        }
    }

    if (q.kind == Q_NONE) {
        float* raw = reinterpret_cast<float*>(codes);
#pragma unroll
        for (int ch = 0; ch < C; ++ch)
            if (ch < nch) st4<false>(raw, base + (int64_t)ch * kChunk + 4 * lane, d, p[ch]);
        return;
    }
    WordSink sink;
    sink.out = codes + (base / kChunk) * 4 * q.bits;
    sink.lo = 0u;
    sink.hi = 0u;
    sink.filled = 0;
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (ch < nch) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                for (int pl = 0; pl < q.bits; ++pl)
                    sink.put(__builtin_amdgcn_ballot_w64(((c[ch][k] >> pl) & 1u) != 0u));
            }
        }
    }
    sink.flush();
}

// Dequantize one tile of a message (the inverse of the code table).
template <int C, bool VEC>
__device__ __forceinline__ void dequant_tile(const QDev& q, const float* lut, const uint64_t* __restrict__ codes,
                                             const float* __restrict__ scales, int64_t base, int nch, int64_t d,
                                             float4 (&deq)[C])
{
    const int lane = lane_id();
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        deq[ch] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (ch >= nch) continue;
        if (q.kind == Q_NONE) {
            deq[ch] = ld4<false>(reinterpret_cast<const float*>(codes), n, d);
            continue;
        }
        const int64_t chunk = (base / kChunk) + ch;
        float sc = 1.0f;
        if (has_scale(q)) sc = scales[(chunk * kChunk) / q.B];
        const bool ok = sc > 0.0f && !isinf(sc);
        const uint64_t* w = codes + chunk * 4 * q.bits;
        const int nv = nvalid4(n, d);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            uint32_t cc = 0;
            for (int pl = 0; pl < q.bits; ++pl) cc |= (uint32_t)((w[k * q.bits + pl] >> lane) & 1u) << pl;
            set_comp(deq[ch], k, k < nv ? deq_of(q, lut, cc, 0.0f, sc, ok) : 0.0f);
        }
    }
}

// p for worker rows: g + e (Adam at the server) or lr*m/sqrt(v) + e after the
// moment update (Adam at the workers).  Moments are written back when asked.
template <int C, bool VEC>
__device__ __forceinline__ void worker_input(const StepArgs& a, const float* __restrict__ g,
                                             const float* __restrict__ e, float* __restrict__ mw,
                                             float* __restrict__ vw, int64_t base, int nch, bool store,
                                             float4 (&p)[C])
{
    const int lane = lane_id();
    const float omb1 = 1.0f - a.beta1, omb2 = 1.0f - a.beta2;
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        if (ch >= nch) {
            p[ch] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            continue;
        }
        const float4 gv = ld4<VEC>(g, n, a.d);
        const float4 ev = ld4<VEC>(e, n, a.d);
        if (a.placement == AT_WORKER) {
            float4 mv = ld4<VEC>(mw, n, a.d);
            float4 vv = ld4<VEC>(vw, n, a.d);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float gk = comp(gv, k);
                const float vk = a.beta2 * comp(vv, k) + omb2 * (gk * gk);
                const float mk = a.beta1 * comp(mv, k) + omb1 * gk;
                set_comp(vv, k, vk);
                set_comp(mv, k, mk);
                const float uk = vk > 0.0f ? a.lr * (mk / sqrtf(vk)) : 0.0f;
                set_comp(p[ch], k, uk + comp(ev, k));
            }
            if (store) {
                st4<VEC>(mw, n, a.d, mv);
                st4<VEC>(vw, n, a.d, vv);
            }
        } else {
            p[ch] = make_float4(gv.x + ev.x, gv.y + ev.y, gv.z + ev.z, gv.w + ev.w);
        }
    }
}

// Server input from the worker average: Adam (at the server) or the average.
template <int C, bool VEC>
__device__ __forceinline__ void server_input(const StepArgs& a, const float4 (&acc)[C], int64_t base, int nch,
                                             float4 (&u)[C])
{
    const int lane = lane_id();
    const float fN = (float)a.N;
    const float omb1 = 1.0f - a.beta1, omb2 = 1.0f - a.beta2;
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        if (ch >= nch) {
            u[ch] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            continue;
        }
        float4 avg = make_float4(acc[ch].x / fN, acc[ch].y / fN, acc[ch].z / fN, acc[ch].w / fN);
        if (a.placement == AT_SERVER) {
            float4 mv = ld4<VEC>(a.m, n, a.d);
            float4 vv = ld4<VEC>(a.v, n, a.d);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float gk = comp(avg, k);
                const float vk = a.beta2 * comp(vv, k) + omb2 * (gk * gk);
                const float mk = a.beta1 * comp(mv, k) + omb1 * gk;
                set_comp(vv, k, vk);
                set_comp(mv, k, mk);
                set_comp(avg, k, vk > 0.0f ? a.lr * (mk / sqrtf(vk)) : 0.0f);
            }
            st4<VEC>(a.m, n, a.d, mv);
            st4<VEC>(a.v, n, a.d, vv);
        }
        u[ch] = avg;
    }
}

// Partial norm of a tile, reduced over the wave (one-bucket quantizers).
template <int C>
__device__ __forceinline__ double tile_partial(const QDev& q, const float4 (&p)[C], int64_t base, int nch,
                                               int64_t d)
{
    Partial a;
    a.sum = 0.0;
    a.mx = 0.0f;
#pragma unroll
    for (int ch = 0; ch < C; ++ch)
        if (ch < nch) partial_add4(a, q.norm, p[ch], nvalid4(base + ch * kChunk + 4 * lane_id(), d));
    return q.norm == S_MAX ? (double)wave_max(a.mx) : wave_sum(a.sum);
}

struct TilePos {
    int64_t tile, base;
    int nch;
};

template <int C>
__device__ __forceinline__ bool tile_pos(const StepArgs& a, TilePos& t)
{
    t.tile = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x / kWave);
    if (t.tile >= a.ntiles) return false;
    t.base = t.tile * C * kChunk;
    const int64_t rem = (a.d - t.base + kChunk - 1) / kChunk;
    t.nch = rem < C ? (int)rem : C;
    return true;
}

// ---------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------

// The fused round.  With a one-bucket Q_w the worker scales are read from
// wscales (computed beforehand); with a one-bucket Q_s the kernel stops after
// the server input, which it leaves in ubuf with per-tile partial norms.
template <int C, bool VEC>
__global__ __launch_bounds__(kBlock) void step_kernel(StepArgs a)
{
    __shared__ float lut_w[kLutSize];
    __shared__ float lut_s[kLutSize];
    fill_lut(a.qw, lut_w);
    fill_lut(a.qs, lut_s);
    __syncthreads();
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    const int lane = lane_id();
    const bool wglobal = has_scale(a.qw) && a.qw.cpb == 0;
    const bool sglobal = has_scale(a.qs) && a.qs.cpb == 0;

    float4 acc[C];
#pragma unroll
    for (int ch = 0; ch < C; ++ch) acc[ch] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);

    for (int i = 0; i < a.N; ++i) {
        const int64_t row = (int64_t)i * a.d;
        float* e = a.e_w + row;
        float4 p[C], dq[C];
        worker_input<C, VEC>(a, a.g + row, e, a.m_w ? a.m_w + row : nullptr, a.v_w ? a.v_w + row : nullptr,
                             t.base, t.nch, true, p);
        const float gs = wglobal ? a.wscales[(int64_t)i * a.qw.nscales] : 0.0f;
        quantize_tile<C>(a.qw, lut_w, p, t.base, t.nch, a.d, a.k0, a.k1, a.t, (uint32_t)i, gs,
                         a.wcodes + (int64_t)i * a.qw.words, a.wscales + (int64_t)i * a.qw.nscales, dq);
#pragma unroll
        for (int ch = 0; ch < C; ++ch) {
            if (ch >= t.nch) continue;
            const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
            float4 r = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            if (a.qw.ef) r = make_float4(p[ch].x - dq[ch].x, p[ch].y - dq[ch].y, p[ch].z - dq[ch].z, p[ch].w - dq[ch].w);
            st4<VEC>(e, n, a.d, r);
            acc[ch] = make_float4(acc[ch].x + dq[ch].x, acc[ch].y + dq[ch].y, acc[ch].z + dq[ch].z,
                                  acc[ch].w + dq[ch].w);
        }
    }

    float4 u[C], q[C], dq[C];
    server_input<C, VEC>(a, acc, t.base, t.nch, u);
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (ch >= t.nch) {
            q[ch] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            continue;
        }
        const float4 es = ld4<VEC>(a.e_s, t.base + (int64_t)ch * kChunk + 4 * lane, a.d);
        q[ch] = make_float4(u[ch].x + es.x, u[ch].y + es.y, u[ch].z + es.z, u[ch].w + es.w);
    }
    if (sglobal) {
#pragma unroll
        for (int ch = 0; ch < C; ++ch)
            if (ch < t.nch) st4<VEC>(a.ubuf, t.base + (int64_t)ch * kChunk + 4 * lane, a.d, u[ch]);
        const double part = tile_partial<C>(a.qs, q, t.base, t.nch, a.d);
        if (lane == 0) a.spart[t.tile] = part;
        return;
    }
    quantize_tile<C>(a.qs, lut_s, q, t.base, t.nch, a.d, a.k0, a.k1, a.t, kServerStream, 0.0f, a.scodes,
                     a.sscales, dq);
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (ch >= t.nch) continue;
        const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
        float4 r = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (a.qs.ef) r = make_float4(q[ch].x - dq[ch].x, q[ch].y - dq[ch].y, q[ch].z - dq[ch].z, q[ch].w - dq[ch].w);
        st4<VEC>(a.e_s, n, a.d, r);
        const float4 xv = ld4<VEC>(a.x, n, a.d);
        st4<VEC>(a.x, n, a.d, make_float4(xv.x - dq[ch].x, xv.y - dq[ch].y, xv.z - dq[ch].z, xv.w - dq[ch].w));
    }
}

// Per-tile partial norms of the worker inputs p for workers [i0, i1), without
// writing any state (one-bucket Q_w).  Rows are [i][d] from a.g / a.e_w.
template <int C, bool VEC>
__global__ __launch_bounds__(kBlock) void worker_partials_kernel(StepArgs a, int i0, int i1)
{
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    for (int i = i0; i < i1; ++i) {
        const int64_t row = (int64_t)(i - i0) * a.d;
        float4 p[C];
        worker_input<C, VEC>(a, a.g + row, a.e_w + row, a.m_w ? a.m_w + row : nullptr,
                             a.v_w ? a.v_w + row : nullptr, t.base, t.nch, false, p);
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
        q[ch] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (ch >= t.nch) continue;
        const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
        const float4 uv = ld4<VEC>(a.ubuf, n, a.d);
        const float4 es = ld4<VEC>(a.e_s, n, a.d);
        q[ch] = make_float4(uv.x + es.x, uv.y + es.y, uv.z + es.z, uv.w + es.w);
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

// Split call: worker a.worker compresses its row (a.g, a.e_w, a.m_w, a.v_w
// point at that worker's d-vectors; a.wcodes/a.wscales at its message).
template <int C, bool VEC>
__global__ __launch_bounds__(kBlock) void worker_kernel(StepArgs a)
{
    __shared__ float lut_w[kLutSize];
    fill_lut(a.qw, lut_w);
    __syncthreads();
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    const int lane = lane_id();
    const bool wglobal = has_scale(a.qw) && a.qw.cpb == 0;
    float4 p[C], dq[C];
    worker_input<C, VEC>(a, a.g, a.e_w, a.m_w, a.v_w, t.base, t.nch, true, p);
    const float gs = wglobal ? a.wscales[0] : 0.0f;
    quantize_tile<C>(a.qw, lut_w, p, t.base, t.nch, a.d, a.k0, a.k1, a.t, (uint32_t)a.worker, gs, a.wcodes,
                     a.wscales, dq);
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (ch >= t.nch) continue;
        float4 r = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (a.qw.ef) r = make_float4(p[ch].x - dq[ch].x, p[ch].y - dq[ch].y, p[ch].z - dq[ch].z, p[ch].w - dq[ch].w);
        st4<VEC>(a.e_w, t.base + (int64_t)ch * kChunk + 4 * lane, a.d, r);
    }
}

// Split call: dequantize the N worker messages, average in ascending worker
// order, run Adam at the server if placed there; result in a.ubuf.
template <int C, bool VEC>
__global__ __launch_bounds__(kBlock) void aggregate_kernel(StepArgs a)
{
    __shared__ float lut_w[kLutSize];
    fill_lut(a.qw, lut_w);
    __syncthreads();
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    const int lane = lane_id();
    float4 acc[C], dq[C], u[C];
#pragma unroll
    for (int ch = 0; ch < C; ++ch) acc[ch] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int i = 0; i < a.N; ++i) {
        dequant_tile<C, VEC>(a.qw, lut_w, a.wcodes + (int64_t)i * a.qw.words,
                             a.wscales + (int64_t)i * a.qw.nscales, t.base, t.nch, a.d, dq);
#pragma unroll
        for (int ch = 0; ch < C; ++ch)
            acc[ch] = make_float4(acc[ch].x + dq[ch].x, acc[ch].y + dq[ch].y, acc[ch].z + dq[ch].z,
                                  acc[ch].w + dq[ch].w);
    }
    server_input<C, VEC>(a, acc, t.base, t.nch, u);
#pragma unroll
    for (int ch = 0; ch < C; ++ch)
        if (ch < t.nch) st4<VEC>(a.ubuf, t.base + (int64_t)ch * kChunk + 4 * lane, a.d, u[ch]);
}

// Server compression from u (a.ubuf) and e_s; optionally also x -= message.
template <int C, bool VEC>
__global__ __launch_bounds__(kBlock) void server_kernel(StepArgs a)
{
    __shared__ float lut_s[kLutSize];
    fill_lut(a.qs, lut_s);
    __syncthreads();
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    const int lane = lane_id();
    const bool sglobal = has_scale(a.qs) && a.qs.cpb == 0;
    float4 q[C], dq[C];
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        q[ch] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (ch >= t.nch) continue;
        const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
        const float4 uv = ld4<VEC>(a.ubuf, n, a.d);
        const float4 es = ld4<VEC>(a.e_s, n, a.d);
        q[ch] = make_float4(uv.x + es.x, uv.y + es.y, uv.z + es.z, uv.w + es.w);
    }
    const float gs = sglobal ? a.sscales[0] : 0.0f;
    quantize_tile<C>(a.qs, lut_s, q, t.base, t.nch, a.d, a.k0, a.k1, a.t, kServerStream, gs, a.scodes,
                     a.sscales, dq);
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (ch >= t.nch) continue;
        const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
        float4 r = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        if (a.qs.ef) r = make_float4(q[ch].x - dq[ch].x, q[ch].y - dq[ch].y, q[ch].z - dq[ch].z, q[ch].w - dq[ch].w);
        st4<VEC>(a.e_s, n, a.d, r);
        if (a.apply) {
            const float4 xv = ld4<VEC>(a.x, n, a.d);
            st4<VEC>(a.x, n, a.d, make_float4(xv.x - dq[ch].x, xv.y - dq[ch].y, xv.z - dq[ch].z, xv.w - dq[ch].w));
        }
    }
}

// Split call: x -= dequantized server message.
template <int C, bool VEC>
__global__ __launch_bounds__(kBlock) void apply_kernel(StepArgs a)
{
    __shared__ float lut_s[kLutSize];
    fill_lut(a.qs, lut_s);
    __syncthreads();
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    const int lane = lane_id();
    float4 dq[C];
    dequant_tile<C, VEC>(a.qs, lut_s, a.scodes, a.sscales, t.base, t.nch, a.d, dq);
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (ch >= t.nch) continue;
        const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
        const float4 xv = ld4<VEC>(a.x, n, a.d);
        st4<VEC>(a.x, n, a.d, make_float4(xv.x - dq[ch].x, xv.y - dq[ch].y, xv.z - dq[ch].z, xv.w - dq[ch].w));
    }
}

__global__ void fill_kernel(float* __restrict__ p, int64_t n, float value)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = value;
}

int64_t grid_of(const StepArgs& a)
{
    return (a.ntiles + kWavesPerBlock - 1) / kWavesPerBlock;
}

// Dispatch on (C, VEC) to a kernel template instance.
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

}  // namespace

hipError_t launch_step(const StepArgs& a, int C, bool vec, hipStream_t s)
{
    EA_DISPATCH(step_kernel, C, vec, grid_of(a), s, a);
    return hipGetLastError();
}

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

hipError_t launch_worker(const StepArgs& a, int C, bool vec, hipStream_t s)
{
    EA_DISPATCH(worker_kernel, C, vec, grid_of(a), s, a);
    return hipGetLastError();
}

hipError_t launch_aggregate(const StepArgs& a, int C, bool vec, hipStream_t s)
{
    EA_DISPATCH(aggregate_kernel, C, vec, grid_of(a), s, a);
    return hipGetLastError();
}

hipError_t launch_server(const StepArgs& a, int C, bool vec, hipStream_t s)
{
    EA_DISPATCH(server_kernel, C, vec, grid_of(a), s, a);
    return hipGetLastError();
}

hipError_t launch_apply(const StepArgs& a, int C, bool vec, hipStream_t s)
{
    EA_DISPATCH(apply_kernel, C, vec, grid_of(a), s, a);
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
