// ea_device.hpp -- device-side building blocks of one Efficient-Adam round on
// CDNA4 (gfx950): counter-based stochastic-rounding draws, wave64 bucket
// reductions, the element rules of each quantizer, and ballot bit-plane
// packing.  Every routine is wave-synchronous: one wave64 owns one tile of
// C chunks of 256 elements; lane l holds elements 4l..4l+3 of each chunk.
//
// Quantizer parameters reach the device code through a traits class: QRt
// reads them from the runtime description (any configuration), QCt<...>
// fixes them at compile time so that a specialized kernel carries no
// per-kind control flow.
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

__device__ __forceinline__ int lane_id()
{
    return (int)(threadIdx.x & (kWave - 1));
}

enum : int32_t { Q_NONE = 0, Q_SCALED_SIGN = 1, Q_STOCH = 2, Q_DET = 3, Q_POW2 = 4, Q_TOPK = 5, Q_RANDK = 6 };
enum : int32_t { S_L1 = 0, S_L2 = 1, S_MAX = 2 };
enum : int32_t { AT_SERVER = 0, AT_WORKER = 1 };

// Device-side description of one quantizer (prepared by the host API).
struct QDev {
    int32_t kind;
    int32_t norm;       // S_L1 / S_L2 / S_MAX: which bucket norm gives the scale
    int32_t bits;       // code width b (32 for Q_NONE)
    int32_t ef;         // error feedback on/off
    int32_t cpb;        // chunks per bucket; 0 = one bucket over the whole vector
    int32_t cpb_shift;  // log2(cpb) (bucket sizes are 256 times a power of two)
    int32_t L;          // STOCH: 2^b - 1; DET: 2^(b-1) - 1
    int32_t kmin;       // POW2: smallest exponent
    int32_t kmax;       // POW2: largest exponent
    int32_t keep;       // TOPK, RANDK: elements kept per bucket
    int64_t B;          // bucket length in elements (d for one bucket)
    int64_t nscales;    // scales per message
    int64_t words;      // uint64 words per message
};

// Quantizer parameters read at run time.
struct QRt {
    static constexpr bool fixed = false;
    __device__ static int kind(const QDev& q) { return q.kind; }
    __device__ static int bits(const QDev& q) { return q.bits; }
    __device__ static int norm(const QDev& q) { return q.norm; }
    __device__ static int cpb(const QDev& q) { return q.cpb; }
    __device__ static int cpb_shift(const QDev& q) { return q.cpb_shift; }
};

// Quantizer parameters fixed at compile time (kind, code bits, norm, chunks
// per bucket); L, kmin, kmax, ef still come from the description.
template <int K, int B, int NM, int CPB>
struct QCt {
    static constexpr bool fixed = true;
    __host__ __device__ static constexpr int kind(const QDev&) { return K; }
    __host__ __device__ static constexpr int bits(const QDev&) { return B; }
    __host__ __device__ static constexpr int norm(const QDev&) { return NM; }
    __host__ __device__ static constexpr int cpb(const QDev&) { return CPB; }
    __host__ __device__ static constexpr int cpb_shift(const QDev&)
    {
        return CPB >= 8 ? 3 : CPB >= 4 ? 2 : CPB >= 2 ? 1 : 0;
    }
};

template <class QT>
__device__ __forceinline__ bool has_scale(const QDev& q)
{
    const int k = QT::kind(q);
    return k == Q_SCALED_SIGN || k == Q_STOCH || k == Q_DET;
}

// Definition 3 sparsifiers: a kept-mask code plus `keep` values per bucket.
template <class QT>
__device__ __forceinline__ bool is_sparse(const QDev& q)
{
    const int k = QT::kind(q);
    return k == Q_TOPK || k == Q_RANDK;
}

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 32x32->64 multiplies by fixed odd constants, with Weyl key increments.
// The two three-way XORs of a round are one v_bitop3_b32 each.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c)
{
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

__device__ __forceinline__ uint4 philox10(uint4 c, uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t a = (uint64_t)0xD2511F53u * c.x;
        const uint64_t b = (uint64_t)0xCD9E8D57u * c.z;
        c = make_uint4(xor3((uint32_t)(b >> 32), c.y, k0), (uint32_t)b,
                       xor3((uint32_t)(a >> 32), c.w, k1), (uint32_t)a);
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
// wave64 reductions without LDS: DPP quad permutes and row mirrors inside each
// row of 16 lanes, then the gfx950 row swaps (permlane16/32_swap) across
// rows.  Every step combines a lane with a partner holding the mirror value
// and the operations are commutative, so all 64 lanes end with the same bits.
// ---------------------------------------------------------------------------
constexpr int kDppXor1 = 0xB1;          // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;          // quad_perm [2,3,0,1]
constexpr int kDppRowMirror = 0x140;    // lane i <- 15 - i within a row
constexpr int kDppHalfMirror = 0x141;   // lane i <- 7 - i within half a row

template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}

template <int CTRL>
__device__ __forceinline__ double dpp_partner(double v)
{
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint64_t r = ((uint64_t)dpp<CTRL>((uint32_t)(b >> 32)) << 32) | dpp<CTRL>((uint32_t)b);
    return __longlong_as_double((long long)r);
}

// Values of the lane 16 (ROWS=16) or 32 (ROWS=32) positions away, as the
// pair (own-side, other-side) in a fixed order that all partner lanes share.
__device__ __forceinline__ void row_swap16(uint32_t x, uint32_t& a, uint32_t& b)
{
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    a = r[0];
    b = r[1];
}

__device__ __forceinline__ void row_swap32(uint32_t x, uint32_t& a, uint32_t& b)
{
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    a = r[0];
    b = r[1];
}

__device__ __forceinline__ double join(uint32_t hi, uint32_t lo)
{
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

__device__ __forceinline__ double wave_sum(double v)
{
    v = v + dpp_partner<kDppXor1>(v);
    v = v + dpp_partner<kDppXor2>(v);
    v = v + dpp_partner<kDppHalfMirror>(v);
    v = v + dpp_partner<kDppRowMirror>(v);
    uint64_t b = (uint64_t)__double_as_longlong(v);
    uint32_t a_lo, b_lo, a_hi, b_hi;
    row_swap16((uint32_t)b, a_lo, b_lo);
    row_swap16((uint32_t)(b >> 32), a_hi, b_hi);
    v = join(a_hi, a_lo) + join(b_hi, b_lo);
    b = (uint64_t)__double_as_longlong(v);
    row_swap32((uint32_t)b, a_lo, b_lo);
    row_swap32((uint32_t)(b >> 32), a_hi, b_hi);
    return join(a_hi, a_lo) + join(b_hi, b_lo);
}

__device__ __forceinline__ float wave_max(float v)
{
    v = fmaxf(v, __uint_as_float(dpp<kDppXor1>(__float_as_uint(v))));
    v = fmaxf(v, __uint_as_float(dpp<kDppXor2>(__float_as_uint(v))));
    v = fmaxf(v, __uint_as_float(dpp<kDppHalfMirror>(__float_as_uint(v))));
    v = fmaxf(v, __uint_as_float(dpp<kDppRowMirror>(__float_as_uint(v))));
    uint32_t a, b;
    row_swap16(__float_as_uint(v), a, b);
    v = fmaxf(__uint_as_float(a), __uint_as_float(b));
    row_swap32(__float_as_uint(v), a, b);
    return fmaxf(__uint_as_float(a), __uint_as_float(b));
}

// A value every lane holds identically, made visibly wave-uniform.
__device__ __forceinline__ float uniform(float v)
{
    return __uint_as_float((uint32_t)__builtin_amdgcn_readfirstlane((int)__float_as_uint(v)));
}

// Per-lane partial of a bucket norm; binary64 for sums, binary32 (exact) for
// the maximum.  (double)x*(double)x is exact in binary64, so one fused
// multiply-add rounds exactly like a separate product and sum.
struct Partial {
    double sum;
    float mx;
};

__device__ __forceinline__ void partial_add(Partial& a, int norm, float x)
{
    if (norm == S_L1) {
        a.sum += (double)fabsf(x);
    } else if (norm == S_L2) {
        const double xd = (double)x;
        a.sum = fma(xd, xd, a.sum);
    } else {
        a.mx = fmaxf(a.mx, fabsf(x));
    }
}

__device__ __forceinline__ void partial_add4(Partial& a, int norm, float4 x, int nvalid)
{
    if (nvalid > 0) partial_add(a, norm, x.x);
    if (nvalid > 1) partial_add(a, norm, x.y);
    if (nvalid > 2) partial_add(a, norm, x.z);
    if (nvalid > 3) partial_add(a, norm, x.w);
}

// Scale of a bucket from its reduced norm (n = elements in the bucket).
__device__ __forceinline__ float scale_from(int norm, double sum, float mx, int64_t n)
{
    if (norm == S_L1) return (float)(sum / (double)n);
    if (norm == S_L2) return sqrtf((float)sum);
    return mx;
}

// ---------------------------------------------------------------------------
// Code tables.  value = scale * lut[code] for SCALED_SIGN / STOCH / DET,
// value = lut[code] for POW2.
// ---------------------------------------------------------------------------
template <class QT>
__device__ __forceinline__ float lut_entry(const QDev& q, int32_t c)
{
    switch (QT::kind(q)) {
    case Q_SCALED_SIGN:
        return c == 0 ? 1.0f : -1.0f;
    case Q_STOCH:
        return c <= q.L ? (float)(2 * c - q.L) / (float)q.L : 0.0f;
    case Q_DET:
        return c <= 2 * q.L ? (float)(c - q.L) / (float)q.L : 0.0f;
    case Q_POW2: {
        const int bits = QT::bits(q);
        if (c >= (1 << bits)) return 0.0f;
        const int32_t mag = c & ((1 << (bits - 1)) - 1);
        if (mag > q.kmax - q.kmin) return 0.0f;          // the zero code (and unused codes)
        const float v = __uint_as_float((uint32_t)(mag + q.kmin + 127) << 23);
        return (c >> (bits - 1)) ? -v : v;
    }
    default:
        return 0.0f;
    }
}

// Whole-block table (any code width); the caller synchronizes the block.
// Only the 2^bits entries a code can select are filled.
__device__ __forceinline__ void fill_lut(const QDev& q, float* lut)
{
    const int n = q.bits < 9 ? (1 << q.bits) : kLutSize;
    for (int c = threadIdx.x; c < n; c += blockDim.x) lut[c] = lut_entry<QRt>(q, c);
}

// Tables of specialized quantizers with codes below 64 are built per wave:
// lane l writes entry l of its own wave's table, and only that wave reads it,
// so no block barrier is needed.
template <class QT>
struct WaveTable {
    static constexpr bool value = false;
};
template <int K, int B, int NM, int CPB>
struct WaveTable<QCt<K, B, NM, CPB>> {
    static constexpr bool value = B <= 6;
};

template <class QT>
__device__ __forceinline__ void fill_wave_table(const QDev& q, float* tab)
{
    tab[lane_id()] = lut_entry<QT>(q, lane_id());
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---------------------------------------------------------------------------
// Element rules.  `inv` is 1/scale for a positive finite scale (any finite
// value otherwise: the caller then replaces code and value, see
// zero_code_of).  `r` is the element's 32-bit Philox word (STOCH only).
// ---------------------------------------------------------------------------
template <class QT>
__device__ __forceinline__ uint32_t code_of(const QDev& q, float p, float inv, uint32_t r)
{
    switch (QT::kind(q)) {
    case Q_SCALED_SIGN:
        return p < 0.0f ? 1u : 0u;
    case Q_STOCH: {
        const float Lf = (float)q.L;
        // clamp to [0, L]; y never reaches L with a positive fraction, so
        // lo + 1 never exceeds L.
        const float y = __builtin_amdgcn_fmed3f((p * inv + 1.0f) * (Lf * 0.5f), 0.0f, Lf);
        // y >= 0: truncation is the floor, and y - floor(y) is exact.
        return (uint32_t)y + (u24(r) < __builtin_amdgcn_fractf(y) ? 1u : 0u);
    }
    case Q_DET: {
        const float Lf = (float)q.L;
        float a = fabsf(p) * inv * Lf;
        a = a > Lf ? Lf : a;
        int32_t i = (int32_t)a;                            // a >= 0: the floor
        if (__builtin_amdgcn_fractf(a) > 0.5f) i += 1;
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
        return ((bitsv >> 31) << (QT::bits(q) - 1)) | (uint32_t)(e - q.kmin);
    }
    default:
        return __float_as_uint(p);
    }
}

// Code sent for every element of a bucket whose scale is zero or not finite
// (the bucket is sent as zeros).
template <class QT>
__device__ __forceinline__ uint32_t zero_code_of(const QDev& q)
{
    return QT::kind(q) == Q_DET ? (uint32_t)q.L : 0u;
}

// Whether a bucket's scale can make the bucket all zeros.
template <class QT>
__device__ __forceinline__ bool scale_gated(const QDev& q)
{
    return QT::kind(q) == Q_STOCH || QT::kind(q) == Q_DET;
}

template <class QT>
__device__ __forceinline__ float deq_of(const QDev& q, const float* lut, uint32_t c, float p, float s)
{
    switch (QT::kind(q)) {
    case Q_NONE:
        return p;
    case Q_POW2:
        return lut[c];
    case Q_SCALED_SIGN:
        return c ? -s : s;
    default:
        return s * lut[c];
    }
}

// ---------------------------------------------------------------------------
// Vector access with tail masking.  VEC: rows are 16-byte aligned.  FULL:
// the float4 lies inside the vector (no checks).
// ---------------------------------------------------------------------------
// Every vector the round touches is streamed once per round and is far larger
// than the caches, so loads and stores carry the non-temporal hint.
#ifndef EA_NONTEMPORAL
#define EA_NONTEMPORAL 1
#endif
typedef float ea_f4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float4 ldv(const float* p)
{
#if EA_NONTEMPORAL
    const ea_f4v v = __builtin_nontemporal_load(reinterpret_cast<const ea_f4v*>(p));
    return make_float4(v.x, v.y, v.z, v.w);
#else
    return *reinterpret_cast<const float4*>(p);
#endif
}

__device__ __forceinline__ void stv(float* p, float4 v)
{
#if EA_NONTEMPORAL
    const ea_f4v w = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(w, reinterpret_cast<ea_f4v*>(p));
#else
    *reinterpret_cast<float4*>(p) = v;
#endif
}

template <class T>
__device__ __forceinline__ T ld1(const T* p)
{
#if EA_NONTEMPORAL
    return __builtin_nontemporal_load(p);
#else
    return *p;
#endif
}

template <class T>
__device__ __forceinline__ void st1(T* p, T v)
{
#if EA_NONTEMPORAL
    __builtin_nontemporal_store(v, p);
#else
    *p = v;
#endif
}

template <bool VEC, bool FULL = false>
__device__ __forceinline__ float4 ld4(const float* __restrict__ p, int64_t n, int64_t lim)
{
    if (FULL || (VEC && n + 4 <= lim)) return ldv(p + n);
    float4 r = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (n < lim) r.x = ld1(p + n);
    if (n + 1 < lim) r.y = ld1(p + n + 1);
    if (n + 2 < lim) r.z = ld1(p + n + 2);
    if (n + 3 < lim) r.w = ld1(p + n + 3);
    return r;
}

template <bool VEC, bool FULL = false>
__device__ __forceinline__ void st4(float* __restrict__ p, int64_t n, int64_t lim, float4 v)
{
    if (FULL || (VEC && n + 4 <= lim)) {
        stv(p + n, v);
        return;
    }
    if (n < lim) st1(p + n, v.x);
    if (n + 1 < lim) st1(p + n + 1, v.y);
    if (n + 2 < lim) st1(p + n + 2, v.z);
    if (n + 3 < lim) st1(p + n + 3, v.w);
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

__device__ __forceinline__ float4 add4(float4 a, float4 b)
{
    return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

__device__ __forceinline__ float4 sub4(float4 a, float4 b)
{
    return make_float4(a.x - b.x, a.y - b.y, a.z - b.z, a.w - b.w);
}

__device__ __forceinline__ float4 zero4()
{
    return make_float4(0.0f, 0.0f, 0.0f, 0.0f);
}

// Number of set bits of a wave mask that belong to lanes below this one.
__device__ __forceinline__ uint32_t lanes_below(uint64_t m)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
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
        if (lane_id() < filled) st1(out + lane_id(), ((uint64_t)hi << 32) | lo);
        out += filled;
        filled = 0;
    }
};

}  // namespace ea
