// ea_device.hpp -- device-side building blocks of one Efficient-Adam round on
// CDNA4 (gfx950): counter-based stochastic-rounding draws, wave64 bucket
// reductions, the element rules of each quantizer, and ballot bit-plane
// packing.  Every routine is wave-synchronous: one wave64 owns one tile of
// C chunks of 256 elements; lane l holds elements 4l..4l+3 of each chunk.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ea {

constexpr int kWave = 64;
constexpr int kChunk = 256;          // elements per chunk: 64 lanes x 4
constexpr int kWavesPerBlock = 4;
constexpr int kBlock = kWave * kWavesPerBlock;
constexpr int kLutSize = 512;        // largest code table (POW2 with 9-bit codes)
constexpr uint32_t kServerStream = 0xFFFFFFFFu;

enum : int32_t { Q_NONE = 0, Q_SCALED_SIGN = 1, Q_STOCH = 2, Q_DET = 3, Q_POW2 = 4 };
enum : int32_t { S_L1 = 0, S_L2 = 1, S_MAX = 2 };
enum : int32_t { AT_SERVER = 0, AT_WORKER = 1 };

// Device-side description of one quantizer (prepared by the host API).
struct QDev {
    int32_t kind;
    int32_t norm;       // S_L1 / S_L2 / S_MAX: which bucket norm gives the scale
    int32_t bits;       // code width b (32 for Q_NONE)
    int32_t ef;         // error feedback on/off
    int32_t cpb;        // chunks per bucket; 0 = one bucket over the whole vector
    int32_t L;          // STOCH: 2^b - 1 levels-1; DET: 2^(b-1) - 1
    int32_t kmin;       // POW2: smallest exponent
    int32_t kmax;       // POW2: largest exponent
    int64_t B;          // bucket length in elements (d for one bucket)
    int64_t nscales;    // scales per message
    int64_t words;      // uint64 words per message
};

__device__ __forceinline__ bool has_scale(const QDev& q)
{
    return q.kind == Q_SCALED_SIGN || q.kind == Q_STOCH || q.kind == Q_DET;
}

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 32x32->64 multiplies by fixed odd constants, with Weyl key increments.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint4 philox10(uint4 c, uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t a = (uint64_t)0xD2511F53u * c.x;
        const uint64_t b = (uint64_t)0xCD9E8D57u * c.z;
        c = make_uint4((uint32_t)(b >> 32) ^ c.y ^ k0, (uint32_t)b,
                       (uint32_t)(a >> 32) ^ c.w ^ k1, (uint32_t)a);
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return c;
}

// 24-bit uniform in [0, 1), exact in binary32.
__device__ __forceinline__ float u24(uint32_t r)
{
    return (float)(r >> 8) * 0x1p-24f;
}

// ---------------------------------------------------------------------------
// wave64 butterfly reductions: every lane ends with the same bits (addition
// and max are commutative, so partner lanes compute identical values).
// ---------------------------------------------------------------------------
__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ float wave_max(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

// Per-lane partial of a bucket norm over one float4 of elements (those with
// valid index only); binary64 for sums, binary32 (exact) for the maximum.
struct Partial {
    double sum;
    float mx;
};

__device__ __forceinline__ void partial_add(Partial& a, int32_t norm, float x)
{
    if (norm == S_L1) a.sum += (double)fabsf(x);
    else if (norm == S_L2) a.sum += (double)x * (double)x;
    else a.mx = fmaxf(a.mx, fabsf(x));
}

__device__ __forceinline__ void partial_add4(Partial& a, int32_t norm, float4 x, int nvalid)
{
    if (nvalid > 0) partial_add(a, norm, x.x);
    if (nvalid > 1) partial_add(a, norm, x.y);
    if (nvalid > 2) partial_add(a, norm, x.z);
    if (nvalid > 3) partial_add(a, norm, x.w);
}

// Scale of a bucket from its reduced norm (n = elements in the bucket).
__device__ __forceinline__ float scale_from(int32_t norm, double sum, float mx, int64_t n)
{
    if (norm == S_L1) return (float)(sum / (double)n);
    if (norm == S_L2) return sqrtf((float)sum);
    return mx;
}

// ---------------------------------------------------------------------------
// Code tables.  value = scale * lut[code] for SCALED_SIGN / STOCH / DET,
// value = lut[code] for POW2.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float lut_entry(const QDev& q, int32_t c)
{
    switch (q.kind) {
    case Q_SCALED_SIGN:
        return c == 0 ? 1.0f : -1.0f;
    case Q_STOCH:
        return c <= q.L ? (float)(2 * c - q.L) / (float)q.L : 0.0f;
    case Q_DET:
        return c <= 2 * q.L ? (float)(c - q.L) / (float)q.L : 0.0f;
    case Q_POW2: {
        if (c >= (1 << q.bits)) return 0.0f;
        const int32_t mag = c & ((1 << (q.bits - 1)) - 1);
        if (mag > q.kmax - q.kmin) return 0.0f;          // the zero code (and unused codes)
        const float v = __uint_as_float((uint32_t)(mag + q.kmin + 127) << 23);
        return (c >> (q.bits - 1)) ? -v : v;
    }
    default:
        return 0.0f;
    }
}

__device__ __forceinline__ void fill_lut(const QDev& q, float* lut)
{
    for (int c = threadIdx.x; c < kLutSize; c += blockDim.x) lut[c] = lut_entry(q, c);
}

// ---------------------------------------------------------------------------
// Element rules.  `ok` says the bucket scale is positive and finite; `inv` is
// 1/scale.  `u` is the element's uniform draw (STOCH only).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t code_of(const QDev& q, float p, float inv, bool ok, float u)
{
    switch (q.kind) {
    case Q_SCALED_SIGN:
        return p < 0.0f ? 1u : 0u;
    case Q_STOCH: {
        if (!ok) return 0u;
        const float Lf = (float)q.L;
        float y = (p * inv + 1.0f) * (Lf * 0.5f);
        y = y < 0.0f ? 0.0f : y;
        y = y > Lf ? Lf : y;
        const float lo = floorf(y);
        uint32_t c = (uint32_t)lo + (u < y - lo ? 1u : 0u);
        return c > (uint32_t)q.L ? (uint32_t)q.L : c;
    }
    case Q_DET: {
        if (!ok) return (uint32_t)q.L;
        const float Lf = (float)q.L;
        float a = fabsf(p) * inv * Lf;
        a = a > Lf ? Lf : a;
        int32_t i = (int32_t)floorf(a);
        if (a - (float)i > 0.5f) i += 1;
        return (uint32_t)((p < 0.0f ? -i : i) + q.L);
    }
    case Q_POW2: {
        const uint32_t bitsv = __float_as_uint(p);
        if ((bitsv & 0x7FFFFFFFu) == 0u) return (uint32_t)(q.kmax - q.kmin + 1);
        const int32_t ex = (int32_t)((bitsv >> 23) & 0xFFu);
        const uint32_t frac = bitsv & 0x7FFFFFu;
        int32_t e = ex == 0 ? -127 : ex - 127 + (frac > 0x400000u ? 1 : 0);
        e = e < q.kmin ? q.kmin : e;
        e = e > q.kmax ? q.kmax : e;
        return ((bitsv >> 31) << (q.bits - 1)) | (uint32_t)(e - q.kmin);
    }
    default:
        return __float_as_uint(p);
    }
}

__device__ __forceinline__ float deq_of(const QDev& q, const float* lut, uint32_t c, float p, float s, bool ok)
{
    switch (q.kind) {
    case Q_NONE:
        return p;
    case Q_POW2:
        return lut[c];
    case Q_SCALED_SIGN:
        return s * lut[c];
    default:
        return ok ? s * lut[c] : 0.0f;
    }
}

// ---------------------------------------------------------------------------
// Vector access with tail masking.  VEC: rows are 16-byte aligned.
// ---------------------------------------------------------------------------
template <bool VEC>
__device__ __forceinline__ float4 ld4(const float* __restrict__ p, int64_t n, int64_t lim)
{
    if (VEC && n + 4 <= lim) return *reinterpret_cast<const float4*>(p + n);
    float4 r = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (n < lim) r.x = p[n];
    if (n + 1 < lim) r.y = p[n + 1];
    if (n + 2 < lim) r.z = p[n + 2];
    if (n + 3 < lim) r.w = p[n + 3];
    return r;
}

template <bool VEC>
__device__ __forceinline__ void st4(float* __restrict__ p, int64_t n, int64_t lim, float4 v)
{
    if (VEC && n + 4 <= lim) {
        *reinterpret_cast<float4*>(p + n) = v;
        return;
    }
    if (n < lim) p[n] = v.x;
    if (n + 1 < lim) p[n + 1] = v.y;
    if (n + 2 < lim) p[n + 2] = v.z;
    if (n + 3 < lim) p[n + 3] = v.w;
}

__device__ __forceinline__ float comp(const float4& v, int k)
{
    return k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w;
}

__device__ __forceinline__ void set_comp(float4& v, int k, float x)
{
    if (k == 0) v.x = x;
    else if (k == 1) v.y = x;
    else if (k == 2) v.z = x;
    else v.w = x;
}

__device__ __forceinline__ int lane_id()
{
    return (int)(threadIdx.x & (kWave - 1));
}

// v_writelane_b32: write a wave-uniform 32-bit value into one lane of a VGPR.
extern "C" __device__ int ea_writelane_i32(int value, int lane, int old) __asm("llvm.amdgcn.writelane.i32");

// Collects 64-bit ballot words into lanes (word j of a group of 64 lands in
// lane j) and writes each full group with one coalesced store.
struct WordSink {
    uint64_t* __restrict__ out;
    uint32_t lo, hi;
    int filled;

    __device__ __forceinline__ void put(uint64_t w)
    {
        lo = (uint32_t)ea_writelane_i32((int)(uint32_t)w, filled, (int)lo);
        hi = (uint32_t)ea_writelane_i32((int)(uint32_t)(w >> 32), filled, (int)hi);
        if (++filled == kWave) flush();
    }
    __device__ __forceinline__ void flush()
    {
        if (filled == 0) return;
        if (lane_id() < filled) out[lane_id()] = ((uint64_t)hi << 32) | lo;
        out += filled;
        filled = 0;
    }
};

}  // namespace ea
