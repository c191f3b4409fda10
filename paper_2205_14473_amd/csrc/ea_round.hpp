// ea_round.hpp -- the fused Efficient-Adam round for gfx950 as templates:
// the quantizer and sparsifier tile routines, the worker and server phases,
// and step_kernel.  Every translation unit that instantiates a step_kernel
// includes it (the generic and fully specialized kernels in ea_kernels.hip,
// the worker-specialized ones in ea_half_c*.hip) and gets its own copies.
//
// Work decomposition.  A tile is C chunks of 256 elements; a wave64 holds a
// tile of one vector, four consecutive elements per lane.  Bucket norms are
// reduced inside the wave (no LDS, no barrier); codes are bit-plane packed
// with one ballot per 64-element plane word.
//
// The fused round (step_kernel) gives a block K consecutive tiles and one
// wave per worker: each wave compresses its worker on the block's tiles and
// hands the dequantized values over through LDS; then wave k adds the
// handoffs of tile k in ascending worker order and runs the server's Adam,
// quantization and the update of x on that tile (Algorithms 1-2, Section IV).
// The split calls use blocks of 4 independent waves, one tile each.
//
// Every kernel is a template over the quantizer traits of both sides and the
// Adam placement: QRt / placement -1 give the generic kernels used for any
// configuration, QCt<...> the specialized ones for common shapes.  Tiles
// that lie wholly inside d go to kernels without per-element bounds checks.
#pragma once

#include "ea_launch.hpp"

namespace ea {

namespace {

// Largest number of waves in a block of the fused round (one worker each):
// wide tiles need more registers per wave, so their blocks are narrower.
#ifndef EA_WIDE_TILE_WAVES
#define EA_WIDE_TILE_WAVES 8
#endif
#ifndef EA_NARROW_TILE_WAVES
#define EA_NARROW_TILE_WAVES 16
#endif
#ifndef EA_ROUND_MIN_WAVES
#define EA_ROUND_MIN_WAVES 5
#endif
#ifndef EA_EDGE_MIN_WAVES
#define EA_EDGE_MIN_WAVES 5
#endif
__host__ __device__ constexpr int max_round_waves(int C)
{
    return C <= 2 ? EA_NARROW_TILE_WAVES : (C == 4 ? 8 : EA_WIDE_TILE_WAVES);
}

// One-chunk tiles with Adam at the server launch narrower blocks (more of
// them per CU): a worker's tile there is little work per wave, and 16-wave
// blocks left the CUs waiting on block boundaries (BERT-sized, 16 workers:
// stochastic 4-bit L2 with 256-element buckets 5.95 -> 4.81 ms, top-8 of 256
// 7.05 -> 4.88 ms).  With Adam at the workers 16 waves stay faster.
#ifndef EA_C1_SERVER_WAVES
#define EA_C1_SERVER_WAVES 4
#endif

// Tiles per block of the fused round.  Lean kernels (whole tiles, Adam at
// the server) take two consecutive tiles per block; the others one.
#ifndef EA_TILES_PER_BLOCK
#define EA_TILES_PER_BLOCK 2
#endif
__host__ __device__ constexpr int round_tiles_per_block(int C, bool lean)
{
    return C <= 2 && lean ? EA_TILES_PER_BLOCK : 1;
}

// Minimum waves per SIMD the compiler must leave room for (caps VGPRs).
// Kernels over whole tiles with Adam at the server have no per-element
// bounds checks and no worker moments, and need fewer registers than the
// others.
#ifndef EA_C4_MIN_WAVES
#define EA_C4_MIN_WAVES 1
#endif
#ifndef EA_C8_MIN_WAVES
#define EA_C8_MIN_WAVES 3
#endif
__host__ __device__ constexpr int round_min_waves(int C, bool lean)
{
    return C <= 2 ? (lean ? EA_ROUND_MIN_WAVES : EA_EDGE_MIN_WAVES)
                  : (lean ? (C == 4 ? EA_C4_MIN_WAVES : EA_C8_MIN_WAVES) : 1);
}

// Kernels specialized for the worker quantizer only (the server quantizer
// and the placement read at run time) take one-chunk tiles two to a block
// (5.58 -> 4.86 ms on a BERT-sized round with 256-element sign buckets).
// Loading their wide tiles' server rows after the last barrier, or capping
// their registers for more waves, measured slower.
#ifndef EA_HALF_C1_TILES
#define EA_HALF_C1_TILES 2
#endif
__host__ __device__ constexpr int kernel_tiles(int C, bool full, int pl, bool half)
{
    return half && full && C == 1 ? EA_HALF_C1_TILES : round_tiles_per_block(C, full && pl == AT_SERVER);
}
template <class QW, class QS, int PL>
__host__ __device__ constexpr bool half_kernel()
{
    return QW::fixed && !QS::fixed && PL < 0;
}

// Number of valid elements among a lane's float4 at element n.
__device__ __forceinline__ int nvalid4(int64_t n, int64_t d)
{
    const int64_t r = d - n;
    return r <= 0 ? 0 : (r >= 4 ? 4 : (int)r);
}

template <int PL>
__device__ __forceinline__ int placement_of(const StepArgs& a)
{
    return PL < 0 ? a.placement : PL;
}

// The launch's arguments with the step taken from the device when the round
// reads it there (a.t_dev), and lr, beta2 from the schedule at that step
// (Assumption 2: alpha/sqrt(T), 1 - theta/T; step decay: alpha * factor^k,
// k = (t-1)/period, factor^k by square-and-multiply from the lowest bit).
__device__ __forceinline__ StepArgs with_step(const StepArgs& in)
{
    StepArgs a = in;
    if (a.t_dev == nullptr) return a;
    const uint32_t t = *a.t_dev;
    a.t = t;
    if (a.sched_kind == EA_SCHED_ASSUMPTION2) {
        const float Tf = (float)a.sched_T;
        a.lr = a.sched_alpha / sqrtf(Tf);
        a.beta2 = 1.0f - a.sched_theta / Tf;
    } else if (a.sched_kind == EA_SCHED_STEP_DECAY) {
        int64_t k = ((int64_t)t - 1) / a.sched_period;
        float r = 1.0f, b = a.sched_factor;
        while (k > 0) {
            if (k & 1) r = r * b;
            b = b * b;
            k >>= 1;
        }
        a.lr = a.sched_alpha * r;
    }
    return a;
}

// ---------------------------------------------------------------------------
// Quantize one tile: scales (reduced per bucket inside the wave, or given for
// a one-bucket quantizer), codes, bit-plane packing and the dequantized
// values.  codes/scales point at the start of the message.  The code words go
// to `sink`, which the caller opens at the tile's first word (message_sink)
// and flushes; consecutive tiles may share one sink, since their words are
// consecutive in the message.
// ---------------------------------------------------------------------------
template <class QT>
__device__ __forceinline__ WordSink message_sink(const QDev& q, uint64_t* codes, int64_t base)
{
    WordSink sink;
    sink.out = codes + (base >> 8) * 4 * QT::bits(q);
    sink.lo = 0u;
    sink.hi = 0u;
    sink.filled = 0;
    return sink;
}

// Sparsifier tuning: how many of each lane's largest keys a first threshold
// search runs on (0: none), for tiles of up to 2 chunks and for wider ones
// (more keys per lane, so more of the kept ones can fall in one lane), and
// whether the searches skip the bits that all lane maxima share (1).
#ifndef EA_SPARSE_SUBSET
#define EA_SPARSE_SUBSET 3
#endif
// Tiles of 4 and 8 chunks: 8 keys per lane, so the first search covers k <=
// 128 (BERT-sized round, top-128 of 2048: 9.19 -> 7.35 ms against 5 keys per
// lane; top-64 of 2048 6.92 -> 7.13, random-64 of 2048 7.57 -> 7.63, top-100
// of 1024 unchanged).  Choosing 5 or 8 per bucket from k kept both gains on
// paper but the second search path slowed the first (top-64 7.19 ms).
#ifndef EA_SPARSE_SUBSET_WIDE
#define EA_SPARSE_SUBSET_WIDE 8
#endif
__host__ __device__ constexpr int sparse_subset(int C)
{
    return C >= 4 ? EA_SPARSE_SUBSET_WIDE : EA_SPARSE_SUBSET;
}
#ifndef EA_SPARSE_PREFIX
#define EA_SPARSE_PREFIX 1
#endif

// Threshold search over values the wave counts with count(c) = how many are
// >= c (non-increasing in c): the largest T with count(T) >= kk, built bit by
// bit from `top` down above a prefix T0 whose bits from `top` down are zero
// and which the answer is known to share; or, as soon as some accepted
// candidate is reached by exactly kk values, that candidate with exact set.
// Each step is one ballot per counted value slot; the loop is kept rolled
// (unrolling it measured no faster and multiplies the code).
struct Selected {
    uint32_t T;
    bool exact;
};
template <class Count>
__device__ __forceinline__ Selected bit_select(const Count& count, uint32_t kk, int top, uint32_t T0)
{
    Selected r{T0, false};
#pragma nounroll
    for (int bit = top; bit >= 0; --bit) {
        const uint32_t cand = r.T | (1u << bit);
        const uint32_t n = count(cand);
        if (n >= kk) {
            r.T = cand;
            if (n == kk) {
                r.exact = true;
                break;
            }
        }
    }
    return r;
}

__device__ __forceinline__ uint32_t wave_count(bool pred)
{
    return (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(pred));
}

// Bitwise OR over the wave of vo and AND of va (same steps as wave_max).
__device__ __forceinline__ void wave_or_and(uint32_t vo, uint32_t va, uint32_t& o, uint32_t& a)
{
    o = vo;
    a = va;
    o |= dpp<kDppXor1>(o);
    a &= dpp<kDppXor1>(a);
    o |= dpp<kDppXor2>(o);
    a &= dpp<kDppXor2>(a);
    o |= dpp<kDppHalfMirror>(o);
    a &= dpp<kDppHalfMirror>(a);
    o |= dpp<kDppRowMirror>(o);
    a &= dpp<kDppRowMirror>(a);
    uint32_t x, y;
    row_swap16(o, x, y);
    o = x | y;
    row_swap16(a, x, y);
    a = x & y;
    row_swap32(o, x, y);
    o = x | y;
    row_swap32(a, x, y);
    a = x & y;
}

// Definition 3 sparsifiers (TOPK, RANDK) on one tile.  Each bucket keeps
// its k = min(keep, n) highest-ranked elements by a 32-bit key, larger keys
// first and lower element indices first among equal keys: the magnitude's
// bit pattern (TOPK) or the element's 24-bit draw word (RANDK).
//
// The k-th largest key T is found by a bitwise search (bit_select) that
// counts with ballots; the search is the costly part, so three things cut its
// steps and ballots.  (1) For k <= 64 r, T lies between the smallest of the
// lanes' r-th largest keys and the largest key, so the search starts below
// the bits those keys all share (for magnitudes, typically the sign and most
// of the exponent); r runs up to S below.  (2)
// For k <= 16 S it first runs on each lane's S largest keys only (S ballots a
// step instead of 4 per chunk; S = 3 for tiles of up to 2 chunks, 8 for wider
// ones) and keeps that answer when a full count confirms it; else it runs
// again over every key.  A lane then holds k/64 <= S/4 of the k largest keys
// on average, so few buckets have a lane with more than S of them; for larger
// k most do, and the first search would mostly be wasted.  (3) It stops as soon as exactly k keys reach a candidate,
// which then splits the bucket without ties.  Otherwise the keys equal to T
// are ranked by element index (element n = 256c + 4l + s comes after every
// element of lower chunks, of lower lanes of its chunk, and of lower slots of
// its lane).  The kept
// values are listed in element order at positions counted the same way.
// Elements past d get key 0 and the highest indices, so they rank below
// every element of the vector and are never kept.
//
// FLAGS (random-k on wide tiles, whose keys do not depend on p): only the
// code words are sent, and the lane's kept flags are returned,
// bit 4j + k for its element in chunk j, slot k; sparse_values then writes
// the values from p, which is not read here.
template <int C, bool FULL, class QT, bool FLAGS = false>
__device__ __forceinline__ uint32_t sparsify_tile(const QDev& q, const float4 (&p)[C], int64_t base, int nch,
                                                  int64_t d, uint32_t k0, uint32_t k1, uint32_t step, uint32_t sid,
                                                  float* __restrict__ vals, WordSink& sink, float4 (&deq)[C])
{
    static_assert(!FLAGS || (C >= 4 && QT::fixed && QT::kind(QDev{}) == Q_RANDK), "flags first: wide random-k only");
    uint32_t kbits_out = 0u;
    const int lane = lane_id();
    const int cpb = QT::cpb(q);
    const bool topk = QT::kind(q) == Q_TOPK;
    const int top = topk ? 31 : 23;   // keys below 2^31 (TOPK) or 2^24 (RANDK)
    if (FULL) nch = C;

    // On tiles of 4 or more chunks a top-k key fixed at compile time is
    // formed from p where it is used (one AND), so the tile's keys take no
    // registers of their own.  (On narrower tiles registers are not short,
    // and held keys measured faster.)
    constexpr bool kKeyOfP = C >= 4 && QT::fixed && QT::kind(QDev{}) == Q_TOPK;
    uint32_t keys[kKeyOfP ? 1 : C][4];
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        deq[ch] = zero4();
        if constexpr (!kKeyOfP) {
            const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
            const int nv = FULL ? 4 : (ch < nch ? nvalid4(n, d) : 0);
            uint4 r = make_uint4(0u, 0u, 0u, 0u);
            if (!topk && (FULL || ch < nch)) {
                const uint64_t j = (uint64_t)n >> 2;
                r = philox10(make_uint4((uint32_t)j, (uint32_t)(j >> 32), step, sid), k0, k1);
            }
            const uint32_t rr[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t kv = topk ? (__float_as_uint(comp(p[ch], k)) & 0x7FFFFFFFu) : (rr[k] >> 8);
                keys[ch][k] = (FULL || k < nv) ? kv : 0u;
            }
        }
    }
    const auto key = [&](int j, int k) -> uint32_t {
        if constexpr (kKeyOfP) {
            uint32_t kv;
            asm volatile("v_and_b32 %0, 0x7fffffff, %1" : "=v"(kv) : "v"(comp(p[j], k)));
            if constexpr (FULL) return kv;
            else return j < nch && k < nvalid4(base + (int64_t)j * kChunk + 4 * lane, d) ? kv : 0u;
        } else {
            return keys[j][k];
        }
    };

    const int64_t chunk0 = base >> 8;
#pragma unroll
    for (int b0 = 0; b0 < C; ++b0) {
        if ((b0 & (cpb - 1)) != 0) continue;
        if (!FULL && b0 >= nch) continue;
        const int64_t e0 = base + (int64_t)b0 * kChunk;
        const int64_t nb = FULL ? q.B : ((d - e0) < q.B ? (d - e0) : q.B);
        const uint32_t kk = (uint32_t)(nb < q.keep ? nb : q.keep);

        // Threshold T: the kk-th largest key of the bucket.
        const auto count_all = [&](uint32_t c) {
            uint32_t n = 0u;
#pragma unroll
            for (int j = 0; j < C; ++j) {
                if (j < b0 || j >= b0 + cpb) continue;
#pragma unroll
                for (int k = 0; k < 4; ++k) n += wave_count(key(j, k) >= c);
            }
            return n;
        };
        uint32_t T = 0u, gt = 0u;
        bool exact = false, found = false, have_gt = false;
        // Each lane's S largest keys, m[0] the largest.
        constexpr int S = sparse_subset(C);
        uint32_t m[S > 0 ? S : 1];
#pragma unroll
        for (int r = 0; r < (S > 0 ? S : 1); ++r) m[r] = 0u;
#pragma unroll
        for (int j = 0; j < C; ++j) {
            if (j < b0 || j >= b0 + cpb) continue;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t x = key(j, k);
#pragma unroll
                for (int r = (S > 0 ? S : 1) - 1; r > 0; --r) m[r] = max(m[r], min(m[r - 1], x));
                m[0] = max(m[0], x);
            }
        }
        // With kk <= 64 r (r <= S) the threshold lies between the smallest
        // r-th largest key of a lane (64 r keys reach it) and the largest
        // key, so it has the bits that all lanes' largest and r-th largest
        // keys share above the highest bit where two of them differ.
        int hi = top;
        uint32_t prefix = 0u;
        constexpr int R = S > 0 ? S : 1;
        if (EA_SPARSE_PREFIX && kk <= (uint32_t)(R * kWave)) {
            uint32_t mr = m[0];
#pragma unroll
            for (int r = 1; r < R; ++r)
                if (kk > (uint32_t)(r * kWave)) mr = m[r];
            uint32_t o, n;
            wave_or_and(m[0] | mr, m[0] & mr, o, n);
            o = (uint32_t)__builtin_amdgcn_readfirstlane((int)o);
            n = (uint32_t)__builtin_amdgcn_readfirstlane((int)n);
            // bits above h: all of them for h < 0, none for h >= 31
            const auto above = [](int h) { return h < 0 ? 0xFFFFFFFFu : (h >= 31 ? 0u : ~((2u << h) - 1u)); };
            hi = o == n ? -1 : 31 - __builtin_clz(o ^ n);
            if (hi > top) hi = top;
            prefix = n & above(hi);
        }
        if (S > 0 && kk <= (uint32_t)(S * kWave / 4)) {
            // First on the keys that are among their lane's S
            // largest.  Its answer Tr holds for the bucket when the counts
            // agree: every key above Tr is among them (Tr is then the kk-th
            // largest of all), or, when exactly kk of them reach Tr, exactly
            // kk keys of the bucket do.
            const auto count_sub = [&](uint32_t c) {
                uint32_t n = 0u;
#pragma unroll
                for (int r = 0; r < S; ++r) n += wave_count(m[r] >= c);
                return n;
            };
            const Selected sr = bit_select(count_sub, kk, hi, prefix);
            const uint32_t Tr = sr.T;
            if (sr.exact) {
                found = exact = count_all(Tr) == kk;
            } else {
                gt = count_all(Tr + 1u);
                found = have_gt = gt == count_sub(Tr + 1u);
            }
            T = Tr;
        }
        if (!found) {
            const Selected sa = bit_select(count_all, kk, hi, prefix);
            T = sa.T;
            exact = sa.exact;
        }

        // Keys equal to T are kept in element order until kk are kept in all:
        // need of them after the gt keys above T.
        const auto need_of = [&]() {
            if (!have_gt) {
                gt = 0u;
#pragma unroll
                for (int j = 0; j < C; ++j) {
                    if (j < b0 || j >= b0 + cpb) continue;
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        gt += (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(key(j, k) > T));
                }
            }
            return kk - gt;
        };

        // Then the kept flags, the code words, the values in element order
        // and the dequantized tile.  A plain store for the values: the caches
        // merge the bucket's scattered 4-byte stores.
        float* vb = vals + ((chunk0 + b0) >> QT::cpb_shift(q)) * (int64_t)q.keep;
        if constexpr (C <= 2) {
            // Kept flags first, bit 4j + k of a lane for its element in chunk
            // j, slot k; then the rest.  (For wider tiles the flag word takes
            // a register per bit constant past 64.)
            uint32_t kbits = 0u;
            if (exact) {
#pragma unroll
                for (int j = 0; j < C; ++j) {
                    if (j < b0 || j >= b0 + cpb) continue;
#pragma unroll
                    for (int k = 0; k < 4; ++k) kbits |= (key(j, k) >= T ? 1u : 0u) << (4 * j + k);
                }
            } else {
                const uint32_t need = need_of();
                uint32_t before = 0;
#pragma unroll
                for (int j = 0; j < C; ++j) {
                    if (j < b0 || j >= b0 + cpb) continue;
                    uint32_t below = 0, tot = 0;
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const uint64_t em = __builtin_amdgcn_ballot_w64(key(j, k) == T);
                        below += lanes_below(em);
                        tot += (uint32_t)__builtin_popcountll(em);
                    }
                    uint32_t own = 0;
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const bool eq = key(j, k) == T;
                        const bool kept = key(j, k) > T || (eq && before + below + own < need);
                        kbits |= (kept ? 1u : 0u) << (4 * j + k);
                        own += eq ? 1u : 0u;
                    }
                    before += tot;
                }
            }
            uint32_t before = 0;
#pragma unroll
            for (int j = 0; j < C; ++j) {
                if (j < b0 || j >= b0 + cpb) continue;
                if (!FULL && j >= nch) continue;
                uint64_t km[4];
                uint32_t below = 0, tot = 0;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    km[k] = __builtin_amdgcn_ballot_w64(((kbits >> (4 * j + k)) & 1u) != 0u);
                    below += lanes_below(km[k]);
                    tot += (uint32_t)__builtin_popcountll(km[k]);
                }
                uint32_t own = 0;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const bool kept = ((kbits >> (4 * j + k)) & 1u) != 0u;
                    const float x = comp(p[j], k);
                    const uint32_t pos = before + below + own;   // < kk by construction; guarded all the same
                    if (kept && pos < (uint32_t)q.keep) vb[pos] = x;
                    own += kept ? 1u : 0u;
                    set_comp(deq[j], k, kept ? x : 0.0f);
                    sink.put(km[k]);
                }
                before += tot;
            }
        } else {
            // Chunk by chunk, each chunk's flags just before its output (the
            // same steps; the output loop is written out in both branches
            // because sharing it measured slower on these tiles: random-64 of
            // 2048 5.7 -> 6.4 ms).  Chunks past d come last in element
            // order, so skipping them leaves the ranks of the others as they
            // are.
            const uint32_t need = exact ? 0u : need_of();
            uint32_t eq_before = 0, kept_before = 0;
#pragma unroll
            for (int j = 0; j < C; ++j) {
                if (j < b0 || j >= b0 + cpb) continue;
                if (!FULL && j >= nch) continue;
                bool kept[4];
                if (exact) {
#pragma unroll
                    for (int k = 0; k < 4; ++k) kept[k] = key(j, k) >= T;
                } else {
                    uint32_t below = 0, tot = 0;
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const uint64_t em = __builtin_amdgcn_ballot_w64(key(j, k) == T);
                        below += lanes_below(em);
                        tot += (uint32_t)__builtin_popcountll(em);
                    }
                    uint32_t own = 0;
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const bool eq = key(j, k) == T;
                        kept[k] = key(j, k) > T || (eq && eq_before + below + own < need);
                        own += eq ? 1u : 0u;
                    }
                    eq_before += tot;
                }
                if constexpr (FLAGS) {
                    uint32_t nib = (kept[0] ? 1u : 0u) | (kept[1] ? 2u : 0u) | (kept[2] ? 4u : 0u) |
                                   (kept[3] ? 8u : 0u);
                    // kept opaque, so the shift below is not folded into
                    // selects of constants (a register per constant)
                    asm volatile("" : "+v"(nib));
                    kbits_out |= nib << (4 * j);
#pragma unroll
                    for (int k = 0; k < 4; ++k) sink.put(__builtin_amdgcn_ballot_w64(kept[k]));
                    continue;
                }
                uint64_t km[4];
                uint32_t below = 0, tot = 0;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    km[k] = __builtin_amdgcn_ballot_w64(kept[k]);
                    below += lanes_below(km[k]);
                    tot += (uint32_t)__builtin_popcountll(km[k]);
                }
                uint32_t own = 0;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const float x = comp(p[j], k);
                    const uint32_t pos = kept_before + below + own;   // < kk by construction; guarded all the same
                    if (kept[k] && pos < (uint32_t)q.keep) vb[pos] = x;
                    own += kept[k] ? 1u : 0u;
                    set_comp(deq[j], k, kept[k] ? x : 0.0f);
                    sink.put(km[k]);
                }
                kept_before += tot;
            }
        }
        // A bucket shorter than keep: the remaining value slots are zero.
        if (!FULL && !FLAGS)
            for (uint32_t sl = kk + (uint32_t)lane; sl < (uint32_t)q.keep; sl += kWave) vb[sl] = 0.0f;
    }
    return kbits_out;
}

// The values of a sparsified tile whose kept flags are known (bit 4j + k of
// a lane for its element in chunk j, slot k, from sparsify_tile<..., true>,
// which has sent the code words): per bucket the kept values in element
// order, zeros in the value slots past a short bucket's kk, and the
// dequantized tile.
template <int C, bool FULL, class QT>
__device__ __forceinline__ void sparse_values(const QDev& q, const float4 (&p)[C], uint32_t kbits, int64_t base,
                                              int nch, int64_t d, float* __restrict__ vals, float4 (&deq)[C])
{
    const int lane = lane_id();
    const int cpb = QT::cpb(q);
    if (FULL) nch = C;
    const int64_t chunk0 = base >> 8;
#pragma unroll
    for (int ch = 0; ch < C; ++ch) deq[ch] = zero4();
#pragma unroll
    for (int b0 = 0; b0 < C; ++b0) {
        if ((b0 & (cpb - 1)) != 0) continue;
        if (!FULL && b0 >= nch) continue;
        const int64_t e0 = base + (int64_t)b0 * kChunk;
        const int64_t nb = FULL ? q.B : ((d - e0) < q.B ? (d - e0) : q.B);
        const uint32_t kk = (uint32_t)(nb < q.keep ? nb : q.keep);
        float* vb = vals + ((chunk0 + b0) >> QT::cpb_shift(q)) * (int64_t)q.keep;
        uint32_t kept_before = 0;
#pragma unroll
        for (int j = 0; j < C; ++j) {
            if (j < b0 || j >= b0 + cpb) continue;
            if (!FULL && j >= nch) continue;
            uint32_t below = 0, tot = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint64_t km = __builtin_amdgcn_ballot_w64(((kbits >> (4 * j + k)) & 1u) != 0u);
                below += lanes_below(km);
                tot += (uint32_t)__builtin_popcountll(km);
            }
            uint32_t own = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const bool kept = ((kbits >> (4 * j + k)) & 1u) != 0u;
                const float x = comp(p[j], k);
                const uint32_t pos = kept_before + below + own;   // < kk by construction; guarded all the same
                if (kept && pos < (uint32_t)q.keep) vb[pos] = x;
                own += kept ? 1u : 0u;
                set_comp(deq[j], k, kept ? x : 0.0f);
            }
            kept_before += tot;
        }
        if (!FULL)
            for (uint32_t sl = kk + (uint32_t)lane; sl < (uint32_t)q.keep; sl += kWave) vb[sl] = 0.0f;
    }
}

// Sparsifiers whose selection runs before the values exist: random-k on
// 8-chunk tiles (its keys are draws).  The draws and the selection then do
// not hold registers beside the tile's values (random-64 of 2048 5.7 -> 5.0
// ms); on 4-chunk tiles, which have registers to spare, it measured slower
// (random-32 of 1024 4.7 -> 5.0 ms).
#ifndef EA_SELECT_FIRST_MIN_C
#define EA_SELECT_FIRST_MIN_C 8
#endif
template <class QT, int C>
__host__ __device__ constexpr bool select_first()
{
    return C >= EA_SELECT_FIRST_MIN_C && QT::fixed && QT::kind(QDev{}) == Q_RANDK;
}

template <int C, bool FULL, class QT>
__device__ __forceinline__ void quantize_tile(const QDev& q, const float* lut, const float4 (&p)[C],
                                              int64_t base, int nch, int64_t d, uint32_t k0, uint32_t k1,
                                              uint32_t step, uint32_t sid, float given_scale,
                                              uint64_t* __restrict__ codes, float* __restrict__ scales,
                                              WordSink& sink, float4 (&deq)[C])
{
    if (is_sparse<QT>(q)) {
        sparsify_tile<C, FULL, QT>(q, p, base, nch, d, k0, k1, step, sid, scales, sink, deq);
        return;
    }
    const int lane = lane_id();
    const int kind = QT::kind(q);
    const int norm = QT::norm(q);
    const int cpb = QT::cpb(q);
    const int bits = QT::bits(q);
    if (FULL) nch = C;

    const int64_t chunk0 = base >> 8;   // first chunk of the tile (tiles start on bucket boundaries)
    float s[C];
    if (has_scale<QT>(q)) {
        if (cpb == 0) {
#pragma unroll
            for (int ch = 0; ch < C; ++ch) s[ch] = given_scale;
        } else {
            Partial part[C];
#pragma unroll
            for (int ch = 0; ch < C; ++ch) {
                part[ch].sum = 0.0;
                part[ch].mx = 0.0f;
                if (ch < nch)
                    partial_add4(part[ch], norm, p[ch], FULL ? 4 : nvalid4(base + ch * kChunk + 4 * lane, d));
            }
#pragma unroll
            for (int ch = 0; ch < C; ++ch) {
                if ((ch & (cpb - 1)) == 0) {
                    if (ch < nch) {
                        Partial tot;
                        tot.sum = 0.0;
                        tot.mx = 0.0f;
#pragma unroll
                        for (int j = 0; j < C; ++j) {
                            if (j >= ch && j < ch + cpb) {
                                tot.sum += part[j].sum;
                                tot.mx = fmaxf(tot.mx, part[j].mx);
                            }
                        }
                        const int64_t b0 = base + (int64_t)ch * kChunk;
                        const int64_t nb = FULL ? q.B : ((d - b0) < q.B ? (d - b0) : q.B);
                        const double S = norm == S_MAX ? 0.0 : wave_sum(tot.sum);
                        const float M = norm == S_MAX ? wave_max(tot.mx) : 0.0f;
                        s[ch] = scale_from(norm, S, M, nb);
                        // A plain store: the caches merge the 4-byte scales of
                        // neighbouring tiles, where streaming stores reach HBM
                        // one partial line at a time.
                        if (lane == 0) scales[(chunk0 + ch) >> QT::cpb_shift(q)] = s[ch];
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

    const bool gated = scale_gated<QT>(q);
    if (kind == Q_NONE) {
        // Whole tiles: the raw message is 16-byte aligned (the launcher
        // requires it of messages sent as values before it takes them).
        float* raw = reinterpret_cast<float*>(codes);
#pragma unroll
        for (int ch = 0; ch < C; ++ch) {
            deq[ch] = p[ch];
            const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
            if (FULL) st4<true, true>(raw, n, d, p[ch]);
            else if (ch < nch) st4<false>(raw, n, d, p[ch]);
        }
        return;
    }
    // Codes are produced slot by slot and each code plane goes straight into
    // a ballot word, in message word order (4*chunk + slot)*bits + plane.
    // The scale, its reciprocal and the gate are wave-uniform and computed
    // once per bucket.  x/s is formed as x * (1/s); a scale below 2^-126
    // (whose reciprocal overflows) and x are first multiplied by 2^64, exact
    // for both.  That case takes a wave-uniform branch, so the common one does
    // no extra work per element.
    float sc = 0.0f, inv = 0.0f;
    bool ok = true, tiny = false;
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        const int nv = FULL ? 4 : (ch < nch ? nvalid4(n, d) : 0);
        if (ch == 0 || (cpb != 0 && (ch & (cpb - 1)) == 0)) {
            sc = uniform(s[ch]);
            ok = !gated || (sc > 0.0f && !isinf(sc));
            tiny = gated && sc < 0x1p-126f;
            inv = 1.0f / (tiny ? sc * 0x1p64f : sc);
        }
        if (!ok) {
            // Zero or non-finite scale (uniform over the wave): the chunk is
            // sent as zero codes and dequantizes to zero.
            const uint32_t zc = zero_code_of<QT>(q);
            deq[ch] = zero4();
            if (FULL || ch < nch) {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const bool valid = FULL || k < nv;
                    for (int pl = 0; pl < bits; ++pl)
                        sink.put(__builtin_amdgcn_ballot_w64(valid && ((zc >> pl) & 1u) != 0u));
                }
            }
            continue;
        }
        uint4 r = make_uint4(0u, 0u, 0u, 0u);
        if (kind == Q_STOCH && (FULL || ch < nch)) {
            const uint64_t j = (uint64_t)n >> 2;
            r = philox10(make_uint4((uint32_t)j, (uint32_t)(j >> 32), step, sid), k0, k1);
        }
        const uint32_t rr[4] = {r.x, r.y, r.z, r.w};
        uint32_t cc[4];
        if (tiny) {
#pragma unroll
            for (int k = 0; k < 4; ++k) cc[k] = code_of<QT>(q, comp(p[ch], k) * 0x1p64f, inv, rr[k]);
        } else {
#pragma unroll
            for (int k = 0; k < 4; ++k) cc[k] = code_of<QT>(q, comp(p[ch], k), inv, rr[k]);
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float x = comp(p[ch], k);
            float dv = deq_of<QT>(q, lut, cc[k], x, sc);
            if (!FULL && k >= nv) {
                cc[k] = 0u;
                dv = 0.0f;
            }
            set_comp(deq[ch], k, dv);
            if (FULL || ch < nch) {
                if constexpr (QT::fixed) {
                    // Codes are below 2^bits, so the top plane is a compare.
#pragma unroll
                    for (int pl = 0; pl < QT::bits(q); ++pl)
                        sink.put(__builtin_amdgcn_ballot_w64(pl == QT::bits(q) - 1 ? cc[k] >= (1u << pl)
                                                                                    : ((cc[k] >> pl) & 1u) != 0u));
                } else {
                    for (int pl = 0; pl < bits; ++pl)
                        sink.put(__builtin_amdgcn_ballot_w64(((cc[k] >> pl) & 1u) != 0u));
                }
            }
        }
    }
}

// Widest code the traits allow (9 bits: Example 2 with the widest exponent
// range).
template <class QT>
__host__ __device__ constexpr int max_code_bits()
{
    if constexpr (QT::fixed)
        return QT::bits(QDev{});
    else
        return 9;
}

// A bit-plane message's code words for one tile, spread for decoding.  Bit
// `lane` of a word lies in its low half for lanes 0-31 and in its high half
// for lanes 32-63; of each chunk's 4*bits words, lane l holds that half of
// word l mod 32 (x[ch][0]) and, for codes wider than 8 bits, of word
// 32 + l mod 32 (x[ch][1]).  Written to LDS in that order, the halves a
// lane needs are consecutive (decode_words).  Lanes past a chunk's words, and
// chunks past the tile's end, load a word that exists and decode to nothing:
// the loads take no branch, so the next worker's words stay in flight while
// the current worker's are decoded.  (The select on the chunk count also
// keeps the compiler from moving a prefetch's load into the next iteration,
// where it would be waited for at once.)
template <int C, class QT>
struct CodeWords {
    static constexpr int R = max_code_bits<QT>() > 8 ? 2 : 1;
    uint32_t x[C][R];
};

template <int C, class QT>
__device__ __forceinline__ void load_code_words(const QDev& q, const uint64_t* __restrict__ codes, int64_t base,
                                                int nch, CodeWords<C, QT>& w)
{
    const int lane = lane_id();
    const int nw = 4 * QT::bits(q);
    const uint32_t* __restrict__ c32 = reinterpret_cast<const uint32_t*>(codes);
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t chunk = (base >> 8) + (ch < nch ? ch : nch - 1);
#pragma unroll
        for (int r = 0; r < CodeWords<C, QT>::R; ++r) {
            const int j = 32 * r + (lane & 31);
            const uint32_t v = c32[(chunk * nw + (j < nw ? j : nw - 1)) * 2 + (lane >> 5)];
            w.x[ch][r] = ch < nch ? v : 0u;
        }
    }
}

// The scale of each chunk's bucket (1 for kinds without scales).
template <int C, class QT>
__device__ __forceinline__ void load_chunk_scales(const QDev& q, const float* __restrict__ scales, int64_t base,
                                                  int nch, float (&sc)[C])
{
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        sc[ch] = 1.0f;
        if (has_scale<QT>(q)) {
            const int64_t chunk = (base >> 8) + (ch < nch ? ch : nch - 1);
            const float v = scales[QT::cpb(q) == 0 ? 0 : (chunk >> QT::cpb_shift(q))];
            sc[ch] = ch < nch ? v : 1.0f;
        }
    }
}

// LDS a wave needs to decode a tile (decode_words): the spread words of its
// chunks.
template <int C, class QT>
__host__ __device__ constexpr int stage_words()
{
    return C * CodeWords<C, QT>::R * kWave;
}

// Byte rows, for code widths known at compile time: row r of a chunk holds
// byte r of each of the chunk's 4*bits words, in word order, padded to a
// multiple of 16 bytes.  Bit `lane` of a word is bit lane % 8 of its byte
// lane / 8, so lane l reads row l / 8 and finds the bits of its codes at bit
// l % 8 of consecutive bytes.
template <class QT>
__host__ __device__ constexpr int row_bytes()
{
    return 4 * max_code_bits<QT>() <= 16 ? 16 : (4 * max_code_bits<QT>() <= 32 ? 32 : 48);
}

// Weight of byte q of row dword i in the code (times 4) of slot k, for the
// planes below 6 (lo) or from 6 up (hi, in units of 256): 4 << p for the
// byte of plane p of slot k, else 0.
template <int B>
__host__ __device__ constexpr uint32_t dot_weights(int k, int i, bool hi)
{
    uint32_t w = 0;
    for (int q = 0; q < 4; ++q) {
        const int p = 4 * i + q - k * B;
        if (p >= 0 && p < B) {
            if (!hi && p < 6) w |= (4u << p) << (8 * q);
            if (hi && p >= 6) w |= (1u << (p - 6)) << (8 * q);
        }
    }
    return w;
}

// Decode through byte rows: a wave writes its words' bytes to `stage` (a lane
// holding a 32-bit half writes its four bytes), reads back its row and turns
// each group of four bytes into four bits with a shift and a mask; a packed
// dot product (v_dot4_u32_u8) then weighs the plane bits of a code straight
// into its byte offset in the code table.
template <int C, class QT, bool SUM, bool SCALED = false>
__device__ __forceinline__ void decode_words_rows(const QDev& q, const float* lut, const CodeWords<C, QT>& w,
                                                  const float (&scs)[C], int64_t base, int nch, int64_t d,
                                                  uint32_t* stage, float4 (&deq)[C], float* stab = nullptr)
{
    constexpr int R = CodeWords<C, QT>::R;
    constexpr int B = max_code_bits<QT>();
    constexpr int RS = row_bytes<QT>();
    constexpr int NW = 4 * B;
    const int lane = lane_id();
    uint8_t* sb = reinterpret_cast<uint8_t*>(stage);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    if constexpr (SCALED) {
        // One bucket per tile: the wave's own copy of the code table times
        // the bucket's scale (zero for a gated bucket), one entry per lane,
        // so each element takes its value in one read; every entry is the
        // product an element would form itself.
        static_assert(SUM && (1 << B) <= kWave && QT::cpb(QDev{}) == C, "one scale per tile, small table");
        const float sc = uniform(scs[0]);
        const bool ok = !scale_gated<QT>(q) || (sc > 0.0f && !isinf(sc));
        if (lane < (1 << B)) stab[lane] = (ok ? sc : 0.0f) * lut[lane];
        lut = stab;
    }
#pragma unroll
    for (int ch = 0; ch < C; ++ch)
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int j = 32 * r + (lane & 31);          // the word this lane holds half of
            if (j < NW) {
                const uint32_t v = w.x[ch][r];
                uint8_t* row = sb + (ch * 8 + 4 * (lane >> 5)) * RS + j;
#pragma unroll
                for (int b = 0; b < 4; ++b) row[b * RS] = (uint8_t)(v >> (8 * b));
            }
        }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int bl = lane & 7;
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        const float sc = uniform(scs[ch]);
        const bool ok = ch < nch && (!scale_gated<QT>(q) || (sc > 0.0f && !isinf(sc)));
        const int nv = nvalid4(n, d);
        const float se = ok ? sc : 0.0f;
        // the lane's row: B dwords of four word-bytes each, reduced to the
        // lane's bit of each byte
        const uint32_t* row = reinterpret_cast<const uint32_t*>(sb + (ch * 8 + (lane >> 3)) * RS);
        uint32_t t[(B + 3) / 4 * 4];
#pragma unroll
        for (int i4 = 0; i4 < B; i4 += 4) {
            const uint4 v = *reinterpret_cast<const uint4*>(row + i4);
            t[i4] = v.x;
            t[i4 + 1] = v.y;
            t[i4 + 2] = v.z;
            t[i4 + 3] = v.w;
        }
#pragma unroll
        for (int i = 0; i < B; ++i) t[i] = (t[i] >> bl) & 0x01010101u;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            uint32_t lo = 0, hi = 0;
#pragma unroll
            for (int i = 0; i < B; ++i) {
                if (4 * i + 3 < k * B || 4 * i >= (k + 1) * B) continue;
                lo = __builtin_amdgcn_udot4(t[i], dot_weights<B>(k, i, false), lo, false);
                if (B > 6) hi = __builtin_amdgcn_udot4(t[i], dot_weights<B>(k, i, true), hi, false);
            }
            const uint32_t c4 = lo + (hi << 8);
            const float tv = *reinterpret_cast<const float*>(reinterpret_cast<const char*>(lut) + c4);
            const int kind = QT::kind(q);
            const float s = SUM ? se : sc;
            const float dv = SCALED ? tv : kind == Q_SCALED_SIGN ? (c4 ? -s : s) : (kind == Q_POW2 ? tv : s * tv);
            set_comp(deq[ch], k, SUM || (ok && k < nv) ? dv : 0.0f);
        }
    }
}

// Decode one tile from its spread code words (load_code_words) and chunk
// scales: bit p of the code of slot k is bit `lane` of word k*bits + p.  The
// wave writes its words to `stage` (stage_words() dwords of its own) and reads
// back the halves that hold its bits, four words per 16-byte read; a rotate
// moves each bit to its place in the code.  One wave's LDS accesses complete
// in order, so only the compiler has to be kept from reordering them.
//
// SUM: the caller only adds the values to sums that start at +0 and never
// stores the lanes past d.  A gated bucket (zero or non-finite scale) then
// decodes to zeros of either sign, which leave such a sum's bits as +0 would,
// and the lanes past d or past the tile are not masked: no select per element.
template <int C, class QT, bool SUM = false, bool SCALED = false>
__device__ __forceinline__ void decode_words(const QDev& q, const float* lut, const CodeWords<C, QT>& w,
                                             const float (&scs)[C], int64_t base, int nch, int64_t d,
                                             uint32_t* stage, float4 (&deq)[C], float* stab = nullptr)
{
    // Byte rows for fixed widths of 2 bits and more; 1-bit codes read their
    // four words' halves in one 16-byte read per chunk here, which costs less
    // than writing bytes (ResNet-18-sized sign, 2048-element buckets: 58 against
    // 64 us).
    if constexpr (QT::fixed && max_code_bits<QT>() >= 2) {
        decode_words_rows<C, QT, SUM, SCALED>(q, lut, w, scs, base, nch, d, stage, deq, stab);
        return;
    }
    constexpr int R = CodeWords<C, QT>::R;
    const int lane = lane_id();
    const int bits = QT::bits(q);
    const int nw = 4 * bits;
    const int sh = lane & 31;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int ch = 0; ch < C; ++ch)
#pragma unroll
        for (int r = 0; r < R; ++r) stage[(ch * R + r) * kWave + lane] = w.x[ch][r];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        const float sc = uniform(scs[ch]);
        const bool ok = ch < nch && (!scale_gated<QT>(q) || (sc > 0.0f && !isinf(sc)));
        const int nv = nvalid4(n, d);
        // this lane's halves of the chunk's words (with the code width known
        // at compile time; else read one at a time below)
        const uint32_t* sl = stage + ch * R * kWave + (lane & 32);
        uint32_t hw[R * 32];
#pragma unroll
        for (int j4 = 0; j4 < R * 32; j4 += 4) {
            if (QT::fixed && j4 < nw) {
                const uint4 v = *reinterpret_cast<const uint4*>(sl + (j4 >> 5) * kWave + (j4 & 31));
                hw[j4] = v.x;
                hw[j4 + 1] = v.y;
                hw[j4 + 2] = v.z;
                hw[j4 + 3] = v.w;
            }
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            // the code times 4: its byte offset in the code table
            uint32_t c4 = 0;
#pragma unroll
            for (int pl = 0; pl < max_code_bits<QT>(); ++pl) {
                if (pl >= bits) break;
                const int j = k * bits + pl;
                const uint32_t h = QT::fixed ? hw[j] : sl[(j >> 5) * kWave + (j & 31)];
                // rotate bit sh of h to bit pl + 2, then insert it
                c4 |= __builtin_amdgcn_alignbit(h, h, (uint32_t)(sh - pl - 2) & 31u) & (4u << pl);
            }
            const float tv = *reinterpret_cast<const float*>(reinterpret_cast<const char*>(lut) + c4);
            const int kind = QT::kind(q);
            const float s = SUM ? (ok ? sc : 0.0f) : sc;
            const float dv = kind == Q_SCALED_SIGN ? (c4 ? -s : s) : (kind == Q_POW2 ? tv : s * tv);
            set_comp(deq[ch], k, SUM || (ok && k < nv) ? dv : 0.0f);
        }
    }
}

// Whether a message is bit planes (decoded with load_code_words and
// decode_words) rather than raw values or a sparsifier's mask and values.
template <class QT>
__device__ __forceinline__ bool plane_coded(const QDev& q)
{
    return !is_sparse<QT>(q) && QT::kind(q) != Q_NONE;
}

// Dequantize one tile of a message (the inverse of the code table).
template <int C, class QT>
__device__ __forceinline__ void dequant_tile(const QDev& q, const float* lut, const uint64_t* __restrict__ codes,
                                             const float* __restrict__ scales, int64_t base, int nch, int64_t d,
                                             uint32_t* stage, float4 (&deq)[C])
{
    const int lane = lane_id();
    if (is_sparse<QT>(q)) {
        // Kept elements take their bucket's values in element order; the
        // count of kept elements before a chunk restarts at each bucket.
        uint32_t before = 0;
#pragma unroll
        for (int ch = 0; ch < C; ++ch) {
            deq[ch] = zero4();
            if (ch >= nch) continue;
            const int64_t chunk = (base >> 8) + ch;
            if ((chunk & (QT::cpb(q) - 1)) == 0) before = 0;
            const uint64_t* w = codes + chunk * 4;
            const float* vb = scales + (chunk >> QT::cpb_shift(q)) * (int64_t)q.keep;
            uint64_t m[4];
            uint32_t below = 0, tot = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                m[k] = w[k];
                below += lanes_below(m[k]);
                tot += (uint32_t)__builtin_popcountll(m[k]);
            }
            uint32_t own = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                // A mask with more than keep bits in a bucket (not a message
                // this library wrote) reads no value past the bucket's slots.
                const bool kept = ((m[k] >> lane) & 1u) != 0u;
                const uint32_t pos = before + below + own;
                set_comp(deq[ch], k, kept && pos < (uint32_t)q.keep ? vb[pos] : 0.0f);
                own += kept ? 1u : 0u;
            }
            before += tot;
        }
        return;
    }
    if (plane_coded<QT>(q)) {
        CodeWords<C, QT> wv;
        float sc[C];
        load_code_words<C, QT>(q, codes, base, nch, wv);
        load_chunk_scales<C, QT>(q, scales, base, nch, sc);
        decode_words<C, QT>(q, lut, wv, sc, base, nch, d, stage, deq);
        return;
    }
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        deq[ch] = ch < nch ? ld4<false>(reinterpret_cast<const float*>(codes), n, d) : zero4();
    }
}

// Raw worker rows of one tile.
template <int C>
struct WorkerRows {
    float4 g[C], e[C], m[C], v[C];
};

template <int C, bool VEC, bool FULL, int PL>
__device__ __forceinline__ void load_worker(const StepArgs& a, const float* __restrict__ g,
                                            const float* __restrict__ e, const float* __restrict__ mw,
                                            const float* __restrict__ vw, int64_t base, int nch,
                                            WorkerRows<C>& r)
{
    const int lane = lane_id();
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        if (!FULL && ch >= nch) {
            r.g[ch] = r.e[ch] = r.m[ch] = r.v[ch] = zero4();
            continue;
        }
        r.g[ch] = ld4<VEC, FULL>(g, n, a.d);
        r.e[ch] = ld4<VEC, FULL>(e, n, a.d);
        if (placement_of<PL>(a) == AT_WORKER) {
            r.m[ch] = ld4<VEC, FULL>(mw, n, a.d);
            r.v[ch] = ld4<VEC, FULL>(vw, n, a.d);
        }
    }
}

// Adam's step lr * (m / sqrt(v)) (0 where v <= 0) on n values per lane, the
// square root and the division correctly rounded.  When every lane's values
// have v in [2^-96, 2^96] and |m| in [2^-60, 2^40] (a wave-uniform test),
// the square root needs no prescale and no special-value fixup, and the
// division no operand scaling and no fixup (the quotient and its operands
// stay normal and far from overflow), so each is computed from the hardware
// estimate and the same exact correction steps alone: the rounded square
// root is picked among s and its two neighbours by the signs of the fma
// residuals v - s'*s, and the quotient is refined from the reciprocal by
// fma residuals.  The results equal those of sqrtf and '/'; any other wave
// takes those.
template <int n>
__device__ __forceinline__ void adam_step(const float (&m)[n], const float (&v)[n], float lr, float (&u)[n])
{
    uint32_t vlo = 0xFFFFFFFFu, vhi = 0u;
    float mlo = __builtin_inff(), mhi = 0.0f;
#pragma unroll
    for (int i = 0; i < n; ++i) {
        vlo = min(vlo, __float_as_uint(v[i]));
        vhi = max(vhi, __float_as_uint(v[i]));
        mlo = fminf(mlo, fabsf(m[i]));
        mhi = fmaxf(mhi, fabsf(m[i]));
    }
    // v >= 0 by construction; a NaN or negative v (bit pattern above 2^96)
    // fails the test, and so does a NaN or infinite m, which makes v NaN or
    // infinite as well
    const bool ok = vlo >= 0x0F800000u && vhi <= 0x6F800000u && mlo >= 0x1p-60f && mhi <= 0x1p40f;
    if (__builtin_amdgcn_ballot_w64(!ok) == 0) {
#pragma unroll
        for (int i = 0; i < n; ++i) {
            float s = __builtin_amdgcn_sqrtf(v[i]);
            const float sdn = __uint_as_float(__float_as_uint(s) - 1u);
            const float sup = __uint_as_float(__float_as_uint(s) + 1u);
            const float rdn = fmaf(-sdn, s, v[i]);
            const float rup = fmaf(-sup, s, v[i]);
            s = rdn <= 0.0f ? sdn : s;
            s = rup > 0.0f ? sup : s;
            float r = __builtin_amdgcn_rcpf(s);
            r = fmaf(fmaf(-s, r, 1.0f), r, r);
            float q = m[i] * r;
            q = fmaf(fmaf(-s, q, m[i]), r, q);
            q = fmaf(fmaf(-s, q, m[i]), r, q);
            u[i] = lr * q;
        }
    } else {
#pragma unroll
        for (int i = 0; i < n; ++i) u[i] = v[i] > 0.0f ? lr * (m[i] / sqrtf(v[i])) : 0.0f;
    }
}

// p for a worker: g + e (Adam at the server) or lr*m/sqrt(v) + e after the
// moment update (Adam at the workers); updated moments are left in r.
template <int C, int PL>
__device__ __forceinline__ void worker_p(const StepArgs& a, WorkerRows<C>& r, float4 (&p)[C])
{
    const float omb1 = 1.0f - a.beta1, omb2 = 1.0f - a.beta2;
    if (placement_of<PL>(a) == AT_WORKER) {
        float mm[4 * C], vv[4 * C], uu[4 * C];
#pragma unroll
        for (int ch = 0; ch < C; ++ch) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float gk = comp(r.g[ch], k);
                const float vk = a.beta2 * comp(r.v[ch], k) + omb2 * (gk * gk);
                const float mk = a.beta1 * comp(r.m[ch], k) + omb1 * gk;
                set_comp(r.v[ch], k, vk);
                set_comp(r.m[ch], k, mk);
                mm[4 * ch + k] = mk;
                vv[4 * ch + k] = vk;
            }
        }
        adam_step<4 * C>(mm, vv, a.lr, uu);
#pragma unroll
        for (int ch = 0; ch < C; ++ch) {
#pragma unroll
            for (int k = 0; k < 4; ++k) set_comp(p[ch], k, uu[4 * ch + k] + comp(r.e[ch], k));
        }
    } else {
#pragma unroll
        for (int ch = 0; ch < C; ++ch) p[ch] = add4(r.g[ch], r.e[ch]);
    }
}

template <int C, bool VEC, bool FULL, int PL>
__device__ __forceinline__ void store_moments(const StepArgs& a, float* __restrict__ mw, float* __restrict__ vw,
                                              int64_t base, int nch, const WorkerRows<C>& r)
{
    if (placement_of<PL>(a) != AT_WORKER) return;
    const int lane = lane_id();
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (!FULL && ch >= nch) continue;
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        st4<VEC, FULL>(mw, n, a.d, r.m[ch]);
        st4<VEC, FULL>(vw, n, a.d, r.v[ch]);
    }
}

// The server's rows of one tile: Adam moments (Adam at the server), the
// server error and x.
template <int C>
struct ServerRows {
    float4 m[C], v[C], e[C], x[C];
};

template <int C, bool VEC, bool FULL, int PL>
__device__ __forceinline__ void load_server(const StepArgs& a, int64_t base, int nch, bool with_e, bool with_x,
                                            ServerRows<C>& r)
{
    const int lane = lane_id();
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        r.m[ch] = r.v[ch] = r.e[ch] = r.x[ch] = zero4();
        if (!FULL && ch >= nch) continue;
        if (placement_of<PL>(a) == AT_SERVER) {
            r.m[ch] = ld4<VEC, FULL>(a.m, n, a.d);
            r.v[ch] = ld4<VEC, FULL>(a.v, n, a.d);
        }
        if (with_e) r.e[ch] = ld4<VEC, FULL>(a.e_s, n, a.d);
        if (with_x) r.x[ch] = ld4<VEC, FULL>(a.x, n, a.d);
    }
}

// Average of the dequantized sum: a division by N, done as a multiplication
// by 1/N when N is a power of two (both are the correctly rounded x/N).
__device__ __forceinline__ float avg_of(float x, float fN, float invN, bool pow2)
{
    return pow2 ? x * invN : x / fN;
}

// Server input from the worker sum: Adam (at the server) or the average.
template <int C, bool VEC, bool FULL, int PL>
__device__ __forceinline__ void server_input(const StepArgs& a, const float4 (&acc)[C], int64_t base, int nch,
                                             ServerRows<C>& sr, float4 (&u)[C])
{
    const int lane = lane_id();
    const float fN = (float)a.N;
    const bool pow2 = (a.N & (a.N - 1)) == 0;
    const float invN = 1.0f / fN;
    const float omb1 = 1.0f - a.beta1, omb2 = 1.0f - a.beta2;
    float4 avg[C];
#pragma unroll
    for (int ch = 0; ch < C; ++ch)
        avg[ch] = make_float4(avg_of(acc[ch].x, fN, invN, pow2), avg_of(acc[ch].y, fN, invN, pow2),
                              avg_of(acc[ch].z, fN, invN, pow2), avg_of(acc[ch].w, fN, invN, pow2));
    if (placement_of<PL>(a) == AT_SERVER) {
        // the moments of every chunk (those past d are zero and unused)
        float mm[4 * C], vv[4 * C], uu[4 * C];
#pragma unroll
        for (int ch = 0; ch < C; ++ch) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float gk = comp(avg[ch], k);
                const float vk = a.beta2 * comp(sr.v[ch], k) + omb2 * (gk * gk);
                const float mk = a.beta1 * comp(sr.m[ch], k) + omb1 * gk;
                set_comp(sr.v[ch], k, vk);
                set_comp(sr.m[ch], k, mk);
                mm[4 * ch + k] = mk;
                vv[4 * ch + k] = vk;
            }
        }
        adam_step<4 * C>(mm, vv, a.lr, uu);
#pragma unroll
        for (int ch = 0; ch < C; ++ch) {
#pragma unroll
            for (int k = 0; k < 4; ++k) set_comp(avg[ch], k, uu[4 * ch + k]);
        }
    }
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        const int64_t n = base + (int64_t)ch * kChunk + 4 * lane;
        if (!FULL && ch >= nch) {
            u[ch] = zero4();
            continue;
        }
        if (placement_of<PL>(a) == AT_SERVER) {
            st4<VEC, FULL>(a.m, n, a.d, sr.m[ch]);
            st4<VEC, FULL>(a.v, n, a.d, sr.v[ch]);
        }
        u[ch] = avg[ch];
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
    t.tile = a.tile0 + (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x / kWave);
    if (t.tile >= a.ntiles) return false;
    t.base = t.tile * C * kChunk;
    const int64_t rem = (a.d - t.base + kChunk - 1) / kChunk;
    t.nch = rem < C ? (int)rem : C;
    return true;
}

// ---------------------------------------------------------------------------
// One worker's share of a tile: wave w compresses worker i and leaves its
// dequantized values in the handoff slot.
template <int C, bool VEC, bool FULL, int PL>
__device__ __forceinline__ void worker_load(const StepArgs& a, const TilePos& t, int i, WorkerRows<C>& r)
{
    const bool atw = placement_of<PL>(a) == AT_WORKER;
    const int64_t row = (int64_t)i * a.d;
    load_worker<C, VEC, FULL, PL>(a, a.g + row, a.e_w + row, atw ? a.m_w + row : nullptr,
                                  atw ? a.v_w + row : nullptr, t.base, t.nch, r);
}

template <int C, bool VEC, bool FULL, class QW, int PL>
__device__ __forceinline__ void worker_compute(const StepArgs& a, const TilePos& t, const float* lut_w, int i,
                                               WorkerRows<C>& r, WordSink& sink, float4* slot)
{
    const int lane = lane_id();
    const bool wglobal = has_scale<QW>(a.qw) && QW::cpb(a.qw) == 0;
    const bool atw = placement_of<PL>(a) == AT_WORKER;
    const int64_t row = (int64_t)i * a.d;
    float4 p[C], dq[C];
    if constexpr (select_first<QW, C>()) {
        // the selection and the code words first, while the rows arrive
        float4 none[C];
#pragma unroll
        for (int ch = 0; ch < C; ++ch) none[ch] = zero4();
        const uint32_t kb = sparsify_tile<C, FULL, QW, true>(a.qw, none, t.base, t.nch, a.d, a.k0, a.k1, a.t,
                                                             (uint32_t)i, nullptr, sink, dq);
        worker_p<C, PL>(a, r, p);
        if (atw) store_moments<C, VEC, FULL, PL>(a, a.m_w + row, a.v_w + row, t.base, t.nch, r);
        sparse_values<C, FULL, QW>(a.qw, p, kb, t.base, t.nch, a.d, a.wscales + (int64_t)i * a.qw.nscales, dq);
    } else {
        worker_p<C, PL>(a, r, p);
        if (atw) store_moments<C, VEC, FULL, PL>(a, a.m_w + row, a.v_w + row, t.base, t.nch, r);
        const float gs = wglobal ? a.wscales[(int64_t)i * a.qw.nscales] : 0.0f;
        quantize_tile<C, FULL, QW>(a.qw, lut_w, p, t.base, t.nch, a.d, a.k0, a.k1, a.t, (uint32_t)i, gs,
                                   a.wcodes + (int64_t)i * a.qw.words, a.wscales + (int64_t)i * a.qw.nscales, sink,
                                   dq);
    }
    float* e = a.e_w + row;
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (!FULL && ch >= t.nch) continue;
        const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
        st4<VEC, FULL>(e, n, a.d, a.qw.ef ? sub4(p[ch], dq[ch]) : zero4());
    }
#pragma unroll
    for (int ch = 0; ch < C; ++ch) slot[ch * kWave + lane] = dq[ch];
}

// Wave 0: add the cnt handoff slots of a group, in ascending worker order.
template <int C>
__device__ __forceinline__ void gather_group(const float4* slot, int cnt, float4 (&acc)[C])
{
    const int lane = lane_id();
    for (int j = 0; j < cnt; ++j) {
#pragma unroll
        for (int ch = 0; ch < C; ++ch) acc[ch] = add4(acc[ch], slot[(j * C + ch) * kWave + lane]);
    }
}

// Position of tile `tile` of C chunks.
template <int C>
__device__ __forceinline__ TilePos tile_at(const StepArgs& a, int64_t tile)
{
    TilePos t;
    t.tile = tile;
    t.base = tile * C * kChunk;
    const int64_t rem = (a.d - t.base + kChunk - 1) / kChunk;
    t.nch = rem < C ? (int)rem : C;
    return t;
}

// Worker i's rows of the block's nt consecutive tiles.
template <int C, int K, bool VEC, bool FULL, int PL>
__device__ __forceinline__ void worker_rows(const StepArgs& a, const TilePos (&tp)[K], int nt, int i,
                                            WorkerRows<C> (&r)[K])
{
#pragma unroll
    for (int k = 0; k < K; ++k)
        if (k < nt) worker_load<C, VEC, FULL, PL>(a, tp[k], i, r[k]);
}

// Worker i on the block's nt consecutive tiles, from rows loaded beforehand
// (worker_rows; all tiles' rows are loaded first, so the later tiles' loads
// are in flight while the first is compressed); the codes of the tiles leave
// through one sink, as one piece.  Tile k's dequantized values go to
// slots + (k*G + w)*C*64.
template <int C, int K, bool VEC, bool FULL, class QW, int PL>
__device__ __forceinline__ void worker_tiles(const StepArgs& a, const TilePos (&tp)[K], int nt, const float* lut_w,
                                             int i, WorkerRows<C> (&r)[K], float4* slots, int G, int w)
{
    WordSink sink = message_sink<QW>(a.qw, a.wcodes + (int64_t)i * a.qw.words, tp[0].base);
#pragma unroll
    for (int k = 0; k < K; ++k)
        if (k < nt)
            worker_compute<C, VEC, FULL, QW, PL>(a, tp[k], lut_w, i, r[k], sink,
                                                 slots + ((int64_t)k * G + w) * C * kWave);
    sink.flush();
}

// Worker i on the block's tiles: its rows are loaded, then compressed.  The
// two spellings take the same steps; the register allocator does better with
// the first on fully specialized whole-tile kernels (BERT-sized round 94 -> 89
// VGPRs, random-k 96 with a 24-byte spill -> 95 without) and with the second
// on the others (the generic 8-chunk kernel spills with the first).
template <int C, int K, bool VEC, bool FULL, class QW, int PL, bool INLINE>
__device__ __forceinline__ void worker_round(const StepArgs& a, const TilePos (&tp)[K], int nt, const float* lut_w,
                                             int i, float4* slots, int G, int w)
{
    WorkerRows<C> r[K];
    if constexpr (INLINE) {
#pragma unroll
        for (int k = 0; k < K; ++k)
            if (k < nt) worker_load<C, VEC, FULL, PL>(a, tp[k], i, r[k]);
        WordSink sink = message_sink<QW>(a.qw, a.wcodes + (int64_t)i * a.qw.words, tp[0].base);
#pragma unroll
        for (int k = 0; k < K; ++k)
            if (k < nt)
                worker_compute<C, VEC, FULL, QW, PL>(a, tp[k], lut_w, i, r[k], sink,
                                                     slots + ((int64_t)k * G + w) * C * kWave);
        sink.flush();
    } else {
        worker_rows<C, K, VEC, FULL, PL>(a, tp, nt, i, r);
        worker_tiles<C, K, VEC, FULL, QW, PL>(a, tp, nt, lut_w, i, r, slots, G, w);
    }
}

// 8-chunk tiles whose server bucket is the whole tile (a scaled or sign
// quantizer fixed at compile time): the server side runs on 8 waves, one
// chunk each, instead of one wave holding all eight chunks' rows (ResNet-18-
// sized round 0.315 -> 0.305 ms; BERT-sized, sign 2048, 16 workers 10.8 -> 5.0
// ms).  For 4-chunk tiles it measured slower (GPT-2-medium-sized 8.13 ->
// 8.36 ms): the waves that do not serve wait at its two barriers.
template <class QT, int C>
struct SplitServe {
    static constexpr bool value = false;
};
template <int K, int B, int NM, int CPB, int C>
struct SplitServe<QCt<K, B, NM, CPB>, C> {
    static constexpr bool value = C == 8 && CPB == C && (K == Q_SCALED_SIGN || K == Q_STOCH || K == Q_DET);
};
// The same quantizer with its scale given (computed by the waves together).
template <class QT>
struct GivenScale;
template <int K, int B, int NM, int CPB>
struct GivenScale<QCt<K, B, NM, CPB>> {
    using type = QCt<K, B, NM, 0>;
};

// Add chunk ch of the cnt handoff slots of a group (tiles of C chunks), in
// ascending worker order.
template <int C>
__device__ __forceinline__ void gather_chunk(const float4* slot, int cnt, int ch, float4& acc)
{
    const int lane = lane_id();
    for (int j = 0; j < cnt; ++j) acc = add4(acc, slot[(j * C + ch) * kWave + lane]);
}

// The server side of one tile on C waves: wave ch gathers chunk ch of the
// last group, runs Adam (at the server) and adds e_s on it; the lane partials
// of the bucket norm meet in `red` ([C][64], LDS) and every serving wave adds
// them in chunk order (the order of the one-wave round, so the scale has the
// same bits), then quantizes its chunk under that scale and applies it.
// Every wave of the block takes part in both barriers.  FULL = false: a
// ragged tile, served on the waves of its nch chunks, with bounds checks.
template <int C, bool VEC, bool FULL, class QS, int PL>
__device__ __forceinline__ void serve_split(const StepArgs& a, const TilePos& t, const float* lut_s,
                                            const float4* slots, int cnt, float4 acc, double* red)
{
    using QG = typename GivenScale<QS>::type;
    const int lane = lane_id();
    const int w = (int)(threadIdx.x / kWave);
    const int nch = FULL ? C : t.nch;
    const bool serving = w < nch;
    const int ch = serving ? w : 0;
    const int64_t base = t.base + (int64_t)ch * kChunk;
    const int norm = QS::norm(a.qs);
    ServerRows<1> sr;
    if (serving) load_server<1, VEC, FULL, PL>(a, base, 1, true, true, sr);
    __syncthreads();                           // the last group's handoff is complete
    float4 u[1], q[1], dq[1];
    if (serving) {
        gather_chunk<C>(slots, cnt, ch, acc);
        const float4 s1[1] = {acc};
        server_input<1, VEC, FULL, PL>(a, s1, base, 1, sr, u);
        q[0] = add4(u[0], sr.e[0]);
        Partial p;
        p.sum = 0.0;
        p.mx = 0.0f;
        partial_add4(p, norm, q[0], FULL ? 4 : nvalid4(base + 4 * lane, a.d));
        red[ch * kWave + lane] = norm == S_MAX ? (double)p.mx : p.sum;
    }
    __syncthreads();                           // every chunk's partial is in LDS
    if (!serving) return;
    double tot = 0.0;
    float mx = 0.0f;
#pragma unroll
    for (int j = 0; j < C; ++j) {
        if (!FULL && j >= nch) continue;
        if (norm == S_MAX) mx = fmaxf(mx, (float)red[j * kWave + lane]);
        else tot += red[j * kWave + lane];
    }
    const double S = norm == S_MAX ? 0.0 : wave_sum(tot);
    const float M = norm == S_MAX ? wave_max(mx) : 0.0f;
    const int64_t nb = FULL ? a.qs.B : ((a.d - t.base) < a.qs.B ? (a.d - t.base) : a.qs.B);
    const float scale = scale_from(norm, S, M, nb);
    if (ch == 0 && lane == 0) a.sscales[(t.base >> 8) >> QS::cpb_shift(a.qs)] = scale;
    WordSink sink = message_sink<QG>(a.qs, a.scodes, base);
    quantize_tile<1, FULL, QG>(a.qs, lut_s, q, base, 1, a.d, a.k0, a.k1, a.t, kServerStream, scale, a.scodes,
                               a.sscales, sink, dq);
    sink.flush();
    const int64_t n = base + 4 * lane;
    st4<VEC, FULL>(a.e_s, n, a.d, a.qs.ef ? sub4(q[0], dq[0]) : zero4());
    st4<VEC, FULL>(a.x, n, a.d, sub4(sr.x[0], dq[0]));
}

// 8-chunk tiles with a sparsifier on the server (top-k, random-k): the
// server's Adam runs on 8 waves, one chunk each, and one wave then selects
// and codes the whole tile (the threshold search needs every key of a
// bucket).  No wave holds all eight chunks' server rows, which kept these
// kernels at two waves per SIMD.
template <class QT, int C>
struct SparseServe {
    static constexpr bool value = false;
};
template <int K, int B, int NM, int CPB, int C>
struct SparseServe<QCt<K, B, NM, CPB>, C> {
    static constexpr bool value = C == 8 && (K == Q_TOPK || K == Q_RANDK);
};

// The server side of one tile for SparseServe: wave ch gathers chunk ch of
// the last group, runs Adam on it and adds e_s; it leaves q and x in the
// handoff slots of workers 0 and 1 of chunk ch, which no other wave reads.
// Wave 0 then sparsifies the tile's q and writes e_s and x.  Every wave of
// the block takes part in both barriers.  FULL = false: a ragged tile, with
// bounds checks.
template <int C, bool VEC, bool FULL, class QS, int PL>
__device__ __forceinline__ void serve_sparse(const StepArgs& a, const TilePos& t, const float* lut_s,
                                             float4* slots, int cnt, float4 acc)
{
    const int lane = lane_id();
    const int w = (int)(threadIdx.x / kWave);
    const int nch = FULL ? C : t.nch;
    const bool serving = w < nch;
    const int ch = serving ? w : 0;
    const int64_t base = t.base + (int64_t)ch * kChunk;
    ServerRows<1> sr;
    if (serving) load_server<1, VEC, FULL, PL>(a, base, 1, true, true, sr);
    __syncthreads();                           // the last group's handoff is complete
    if (serving) {
        gather_chunk<C>(slots, cnt, ch, acc);
        const float4 s1[1] = {acc};
        float4 u[1];
        server_input<1, VEC, FULL, PL>(a, s1, base, 1, sr, u);
        slots[ch * kWave + lane] = add4(u[0], sr.e[0]);
        slots[(C + ch) * kWave + lane] = sr.x[0];
    }
    __syncthreads();                           // q and x of every chunk are in LDS
    if (w != 0) return;
    float4 q[C], dq[C];
    WordSink sink = message_sink<QS>(a.qs, a.scodes, t.base);
    if constexpr (select_first<QS, C>()) {
#pragma unroll
        for (int j = 0; j < C; ++j) q[j] = zero4();
        const uint32_t kb = sparsify_tile<C, FULL, QS, true>(a.qs, q, t.base, t.nch, a.d, a.k0, a.k1, a.t,
                                                             kServerStream, nullptr, sink, dq);
#pragma unroll
        for (int j = 0; j < C; ++j) q[j] = (FULL || j < nch) ? slots[j * kWave + lane] : zero4();
        sparse_values<C, FULL, QS>(a.qs, q, kb, t.base, t.nch, a.d, a.sscales, dq);
    } else {
#pragma unroll
        for (int j = 0; j < C; ++j) q[j] = (FULL || j < nch) ? slots[j * kWave + lane] : zero4();
        quantize_tile<C, FULL, QS>(a.qs, lut_s, q, t.base, t.nch, a.d, a.k0, a.k1, a.t, kServerStream, 0.0f,
                                   a.scodes, a.sscales, sink, dq);
    }
    sink.flush();
#pragma unroll
    for (int j = 0; j < C; ++j) {
        if (!FULL && j >= nch) continue;
        const int64_t n = t.base + (int64_t)j * kChunk + 4 * lane;
        st4<VEC, FULL>(a.e_s, n, a.d, a.qs.ef ? sub4(q[j], dq[j]) : zero4());
        st4<VEC, FULL>(a.x, n, a.d, sub4(slots[(C + j) * kWave + lane], dq[j]));
    }
}

// ---------------------------------------------------------------------------
// The fused round on nt <= K consecutive tiles per block.  The block has
// G = min(N, 16) waves.  Workers are taken in groups of G: wave w compresses
// worker g0 + w on every tile of the block and hands its dequantized values
// over through LDS.  Wave k then serves tile k: it adds the handoffs in
// ascending worker order (the order of the average in Algorithm 1) and, after
// the last group, runs the server side on its tile.  Short-lived per-worker
// waves keep far more independent memory traffic in flight than one wave
// looping over all workers, and serving the tiles on separate waves keeps the
// server work off the workers' path.  The handoff is double-buffered over
// groups, so one barrier per group suffices: a buffer is rewritten only after
// the barrier that the serving waves reach once they have read the buffer's
// previous group.  The last group is peeled off so that the serving waves can
// issue the server's loads before the last barrier: their latency overlaps
// the wait for the workers, without the loaded rows being live during the
// earlier groups.
// ---------------------------------------------------------------------------
template <int C, int K, bool VEC, bool FULL, class QW, class QS, int PL>
__device__ __forceinline__ void round_tiles(const StepArgs& a, int64_t tile0, int nt, const float* lut_w,
                                            const float* lut_s, float4* xfer, int G, double* red)
{
    const int lane = lane_id();
    const int w = (int)(threadIdx.x / kWave);
    const bool sglobal = has_scale<QS>(a.qs) && QS::cpb(a.qs) == 0;
    // The server side on C waves, one chunk each (the launch gives the block
    // at least C waves); otherwise wave k serves tile k.
    constexpr bool kSparse = SparseServe<QS, C>::value && K == 1;
    constexpr bool kSplit = (SplitServe<QS, C>::value || kSparse) && K == 1;
    // Whole-tile launches give every block exactly K tiles.  With that known
    // at compile time, each wave's loads of all K tiles and its work on them
    // are straight-line code, so the compiler waits for each tile's rows
    // only before that tile's arithmetic.  (With the later tiles under a
    // branch it waited for every load, and for the stores issued since,
    // before the first tile and again before the second.)
    if constexpr (FULL) nt = K;

    TilePos tp[K];
#pragma unroll
    for (int k = 0; k < K; ++k) tp[k] = tile_at<C>(a, tile0 + k);

    constexpr int kAcc = kSplit ? 1 : C;
    float4 acc[kAcc];
#pragma unroll
    for (int ch = 0; ch < kAcc; ++ch) acc[ch] = zero4();
    const auto gather = [&](const float4* grp, int cnt) {
        if constexpr (kSplit) {
            if (w < C) gather_chunk<C>(grp, cnt, w, acc[0]);
        } else {
            if (w < nt) gather_group<C>(grp + (int64_t)w * G * C * kWave, cnt, acc);
        }
    };

    // Handoff layout: [group buffer][tile][wave][chunk][lane].  With more
    // workers than waves the groups alternate between two buffers, so one
    // barrier per group suffices; a single buffer (a.one_buffer, chosen by
    // the launcher when two buffers would leave a CU room for only one block)
    // takes a second barrier per group, after the gather.
    const int64_t per_buf = (int64_t)K * G * C * kWave;
    int buf = 0, g0 = 0;
    float4* slots;
    constexpr bool kInline = FULL && QW::fixed && QS::fixed;
    for (; g0 + G < a.N; g0 += G, buf ^= a.one_buffer ? 0 : 1) {
        slots = xfer + buf * per_buf;
        worker_round<C, K, VEC, FULL, QW, PL, kInline>(a, tp, nt, lut_w, g0 + w, slots, G, w);
        __syncthreads();
        gather(slots, G);
        if (a.one_buffer) __syncthreads();
    }
    slots = xfer + buf * per_buf;
    if (g0 + w < a.N) worker_round<C, K, VEC, FULL, QW, PL, kInline>(a, tp, nt, lut_w, g0 + w, slots, G, w);
    if constexpr (kSplit) {
        if constexpr (kSparse) serve_sparse<C, VEC, FULL, QS, PL>(a, tp[0], lut_s, slots, a.N - g0, acc[0]);
        else serve_split<C, VEC, FULL, QS, PL>(a, tp[0], lut_s, slots, a.N - g0, acc[0], red);
        return;
    } else {
    const TilePos t = tile_at<C>(a, tile0 + (w < nt ? w : 0));
    ServerRows<C> sr;
    if (w < nt) load_server<C, VEC, FULL, PL>(a, t.base, t.nch, true, !sglobal, sr);
    __syncthreads();
    if (w >= nt) return;
    gather_group<C>(slots + (int64_t)w * G * C * kWave, a.N - g0, acc);

    float4 u[C], q[C], dq[C];
    server_input<C, VEC, FULL, PL>(a, acc, t.base, t.nch, sr, u);
#pragma unroll
    for (int ch = 0; ch < C; ++ch) q[ch] = add4(u[ch], sr.e[ch]);
    if (sglobal) {
#pragma unroll
        for (int ch = 0; ch < C; ++ch)
            if (FULL || ch < t.nch) st4<VEC, FULL>(a.ubuf, t.base + (int64_t)ch * kChunk + 4 * lane, a.d, u[ch]);
        const double part = tile_partial<C>(a.qs, q, t.base, t.nch, a.d);
        if (lane == 0) a.spart[t.tile] = part;
        return;
    }
    WordSink sink = message_sink<QS>(a.qs, a.scodes, t.base);
    quantize_tile<C, FULL, QS>(a.qs, lut_s, q, t.base, t.nch, a.d, a.k0, a.k1, a.t, kServerStream, 0.0f, a.scodes,
                               a.sscales, sink, dq);
    sink.flush();
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (!FULL && ch >= t.nch) continue;
        const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
        st4<VEC, FULL>(a.e_s, n, a.d, a.qs.ef ? sub4(q[ch], dq[ch]) : zero4());
        st4<VEC, FULL>(a.x, n, a.d, sub4(sr.x[ch], dq[ch]));
    }
    }
}

// ---------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------

// Split call: worker a.worker compresses its row (a.g, a.e_w, a.m_w, a.v_w
// point at that worker's d-vectors; a.wcodes/a.wscales at its message).
// Blocks of 4 independent waves, one tile each; QW fixes the worker
// quantizer at compile time (by default it is read at run time).
template <int C, bool VEC, class QW = QRt>
__global__ __launch_bounds__(kBlock) void worker_kernel(StepArgs a)
{
    __shared__ float lut_w[kLutSize];
    fill_lut(a.qw, lut_w);
    __syncthreads();
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    const int lane = lane_id();
    const bool wglobal = has_scale<QW>(a.qw) && QW::cpb(a.qw) == 0;
    const bool atw = a.placement == AT_WORKER;
    WorkerRows<C> r;
    float4 p[C], dq[C];
    load_worker<C, VEC, false, -1>(a, a.g, a.e_w, a.m_w, a.v_w, t.base, t.nch, r);
    worker_p<C, -1>(a, r, p);
    if (atw) store_moments<C, VEC, false, -1>(a, a.m_w, a.v_w, t.base, t.nch, r);
    const float gs = wglobal ? a.wscales[0] : 0.0f;
    WordSink sink = message_sink<QW>(a.qw, a.wcodes, t.base);
    quantize_tile<C, false, QW>(a.qw, lut_w, p, t.base, t.nch, a.d, a.k0, a.k1, a.t, (uint32_t)a.worker, gs,
                                 a.wcodes, a.wscales, sink, dq);
    sink.flush();
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (ch >= t.nch) continue;
        st4<VEC>(a.e_w, t.base + (int64_t)ch * kChunk + 4 * lane, a.d, a.qw.ef ? sub4(p[ch], dq[ch]) : zero4());
    }
}

// Whether the aggregate decodes worker messages through a per-wave code
// table scaled by the bucket's scale: a scaled quantizer fixed at compile
// time, one bucket per tile, codes of 2 to 6 bits (byte-row decoding, a table
// of at most 64 entries, one per lane).
template <class QT, int C>
__host__ __device__ constexpr bool kScaledTable()
{
    if constexpr (QT::fixed) {
        constexpr QDev q{};
        return (QT::kind(q) == Q_STOCH || QT::kind(q) == Q_DET) && QT::cpb(q) == C && QT::bits(q) >= 2 &&
               QT::bits(q) <= 6;
    } else {
        return false;
    }
}

// Split call: dequantize the N worker messages, average in ascending worker
// order, run Adam at the server if placed there; result in a.ubuf.  FULL:
// every tile of the launch lies wholly inside d (no per-tile checks).
template <int C, bool VEC, class QW = QRt, bool FULL = false>
__global__ __launch_bounds__(kBlock) void aggregate_kernel(StepArgs a)
{
    static_assert(!FULL || VEC, "whole-tile kernels need aligned rows");
    __shared__ float lut_w[kLutSize];
    __shared__ __attribute__((aligned(16))) uint32_t stage_all[kWavesPerBlock][stage_words<C, QW>()];
    __shared__ float stab_all[kScaledTable<QW, C>() ? kWavesPerBlock : 1][kWave];
    fill_lut(a.qw, lut_w);
    __syncthreads();
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    const int nch = FULL ? C : t.nch;
    uint32_t* stage = stage_all[threadIdx.x / kWave];
    const int lane = lane_id();
    float4 acc[C], dq[C], u[C];
#pragma unroll
    for (int ch = 0; ch < C; ++ch) acc[ch] = zero4();
    // Bit-plane messages: the next worker's code words and scales are loaded
    // while the current worker's are decoded, into the other of two register
    // sets, so that each set is waited for only where it is decoded (with one
    // set copied forward each step, the copy waited for the load at once).
    const bool planes = plane_coded<QW>(a.qw);
    if (planes) {
        CodeWords<C, QW> wv0, wv1;
        float sc0[C], sc1[C];
        const auto load = [&](int64_t i, CodeWords<C, QW>& wv, float (&sc)[C]) {
            load_code_words<C, QW>(a.qw, a.wcodes + i * a.qw.words, t.base, nch, wv);
            load_chunk_scales<C, QW>(a.qw, a.wscales + i * a.qw.nscales, t.base, nch, sc);
        };
        const auto add = [&](const CodeWords<C, QW>& wv, const float (&sc)[C]) {
            decode_words<C, QW, true, kScaledTable<QW, C>()>(a.qw, lut_w, wv, sc, t.base, nch, a.d, stage, dq,
                                                              stab_all[threadIdx.x / kWave]);
#pragma unroll
            for (int ch = 0; ch < C; ++ch) acc[ch] = add4(acc[ch], dq[ch]);
        };
        load(0, wv0, sc0);
        for (int i = 0; i < a.N; i += 2) {
            load(i + 1 < a.N ? i + 1 : i, wv1, sc1);
            add(wv0, sc0);
            if (i + 1 < a.N) {
                load(i + 2 < a.N ? i + 2 : i + 1, wv0, sc0);
                add(wv1, sc1);
            }
        }
    } else {
        for (int i = 0; i < a.N; ++i) {
            dequant_tile<C, QW>(a.qw, lut_w, a.wcodes + (int64_t)i * a.qw.words,
                                 a.wscales + (int64_t)i * a.qw.nscales, t.base, nch, a.d, stage, dq);
#pragma unroll
            for (int ch = 0; ch < C; ++ch) acc[ch] = add4(acc[ch], dq[ch]);
        }
    }
    // The server's rows load after the decoding: held through it, they cost
    // occupancy (BERT-sized 4-bit, 16 workers: 843 -> 817 us).
    ServerRows<C> sr;
    load_server<C, VEC, FULL, -1>(a, t.base, nch, false, false, sr);
    server_input<C, VEC, FULL, -1>(a, acc, t.base, nch, sr, u);
#pragma unroll
    for (int ch = 0; ch < C; ++ch)
        if (FULL || ch < nch) st4<VEC, FULL>(a.ubuf, t.base + (int64_t)ch * kChunk + 4 * lane, a.d, u[ch]);
}


// Split call: the server's compression of u (a.ubuf) plus e_s; with a.apply
// also x -= its message.  QS: the server quantizer's traits.
template <int C, bool VEC, class QS = QRt>
__global__ __launch_bounds__(kBlock) void server_kernel(StepArgs args)
{
    const StepArgs a = with_step(args);
    __shared__ float lut_s[kLutSize];
    fill_lut(a.qs, lut_s);
    __syncthreads();
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    const int lane = lane_id();
    const bool sglobal = has_scale<QS>(a.qs) && QS::cpb(a.qs) == 0;
    float4 q[C], dq[C];
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        q[ch] = zero4();
        if (ch >= t.nch) continue;
        const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
        q[ch] = add4(ld4<VEC>(a.ubuf, n, a.d), ld4<VEC>(a.e_s, n, a.d));
    }
    const float gs = sglobal ? a.sscales[0] : 0.0f;
    WordSink sink = message_sink<QS>(a.qs, a.scodes, t.base);
    quantize_tile<C, false, QS>(a.qs, lut_s, q, t.base, t.nch, a.d, a.k0, a.k1, a.t, kServerStream, gs, a.scodes,
                                a.sscales, sink, dq);
    sink.flush();
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (ch >= t.nch) continue;
        const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
        st4<VEC>(a.e_s, n, a.d, a.qs.ef ? sub4(q[ch], dq[ch]) : zero4());
        if (a.apply) st4<VEC>(a.x, n, a.d, sub4(ld4<VEC>(a.x, n, a.d), dq[ch]));
    }
}

// Split call: x -= the dequantized server message.
template <int C, bool VEC, class QS = QRt>
__global__ __launch_bounds__(kBlock) void apply_kernel(StepArgs a)
{
    __shared__ float lut_s[kLutSize];
    __shared__ __attribute__((aligned(16))) uint32_t stage_all[kWavesPerBlock][stage_words<C, QS>()];
    fill_lut(a.qs, lut_s);
    __syncthreads();
    TilePos t;
    if (!tile_pos<C>(a, t)) return;
    const int lane = lane_id();
    float4 dq[C];
    dequant_tile<C, QS>(a.qs, lut_s, a.scodes, a.sscales, t.base, t.nch, a.d, stage_all[threadIdx.x / kWave], dq);
#pragma unroll
    for (int ch = 0; ch < C; ++ch) {
        if (ch >= t.nch) continue;
        const int64_t n = t.base + (int64_t)ch * kChunk + 4 * lane;
        st4<VEC>(a.x, n, a.d, sub4(ld4<VEC>(a.x, n, a.d), dq[ch]));
    }
}

// Floats of the code-table region of a fused-round block with G waves: room
// for both block-wide tables or for two 64-entry tables per wave.
__host__ __device__ constexpr int table_floats(int G)
{
    return 2 * kLutSize > 2 * kWave * G ? 2 * kLutSize : 2 * kWave * G;
}

// Dynamic LDS of a fused-round block with G waves: the code tables plus the
// handoff of G workers' tiles (bufs buffers when N > G).
inline size_t round_lds_bytes(int N, int C, int G, int K, int bufs = 2)
{
    const int nbuf = N > G ? bufs : 1;
    return table_floats(G) * sizeof(float) + (size_t)nbuf * K * G * C * kWave * sizeof(float4);
}

// Handoff buffers of a block with more workers than waves: two, unless two
// would leave a CU (whose LDS is the per-block limit on gfx950) room for only
// one block; then one, and the next block starts beside the serving waves
// (ResNet-50-sized round, 32 workers, 136 KB -> 72 KB per block: 2.110 ->
// 2.098 ms).
inline int handoff_bufs(int N, int C, int G, int K, size_t lds_limit)
{
    if (N <= G) return 1;
    return 2 * round_lds_bytes(N, C, G, K, 2) <= lds_limit ? 2 : 1;
}

// Waves per block: one per worker up to the tile's limit, fewer if the LDS
// would exceed what a block may use.
inline int round_waves(int N, int C, int K, size_t lds_limit, int placement)
{
    const int cap = C == 1 && placement == AT_SERVER ? EA_C1_SERVER_WAVES : max_round_waves(C);
    int G = N < cap ? N : cap;
    while (G > 1 && round_lds_bytes(N, C, G, K) > lds_limit) G = (G + 1) / 2;
    return G;
}

// Per-block LDS limit of the current device (queried once per device).
[[maybe_unused]] size_t lds_limit_bytes()
{
    static size_t cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 64 * 1024;
    if (cached[dev] == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= 0)
            v = 64 * 1024;
        cached[dev] = (size_t)v;
    }
    return cached[dev];
}

// The block's place in the launch's run of tiles.  The hardware deals
// consecutive blocks to the 8 XCDs in turn.  With xcd_run = R > 1, the
// blocks of each whole group of 8R take the group's tiles XCD-major: the
// R blocks an XCD receives there take R adjacent slots, so a cache line
// that two adjacent tiles share (rows whose length is not a multiple of
// 128 bytes) is fetched into one L2 instead of two, while the tiles in
// flight across the GPU stay one contiguous window.
__device__ __forceinline__ int64_t block_slot(const StepArgs& a)
{
    const int64_t b = blockIdx.x;
    const int64_t R = a.xcd_run;
    if (R <= 1) return b;
    const int64_t grp = 8 * R;
    const int64_t g = b / grp;
    if ((g + 1) * grp > (int64_t)gridDim.x) return b;     // the last, partial group as dealt
    const int64_t i = b - g * grp;
    return g * grp + (i % 8) * R + i / 8;
}

// The fused round.  With a one-bucket Q_w the worker scales are read from
// wscales (computed beforehand); with a one-bucket Q_s the block stops after
// the server input, which it leaves in ubuf with per-tile partial norms.
//
// MW > 0 overrides the minimum waves per SIMD of the launch bounds (the
// register cap).
//
// FULL kernels (rows 16-byte aligned) take the tiles that lie wholly inside d
// and carry no bounds checks; the others take any tile.  A launch covers
// tiles [a.tile0, a.tile1); block b works on the K tiles from
// a.tile0 + b*K.
template <int C, bool VEC, bool FULL, class QW, class QS, int PL, int MW = 0>
__global__ __launch_bounds__(max_round_waves(C) * kWave,
                             MW > 0 ? MW : round_min_waves(C, FULL && PL == AT_SERVER)) void step_kernel(
    StepArgs args)
{
    const StepArgs a = with_step(args);
    static_assert(!FULL || VEC, "whole-tile kernels need aligned rows");
    extern __shared__ float4 smem[];
    const int G = (int)(blockDim.x / kWave);
    float* lut_w;
    float* lut_s;
    if constexpr (WaveTable<QW>::value && WaveTable<QS>::value) {
        float* tab = reinterpret_cast<float*>(smem) + (threadIdx.x / kWave) * 2 * kWave;
        fill_wave_table<QW>(a.qw, tab);
        fill_wave_table<QS>(a.qs, tab + kWave);
        lut_w = tab;
        lut_s = tab + kWave;
    } else {
        lut_w = reinterpret_cast<float*>(smem);
        lut_s = lut_w + kLutSize;
        fill_lut(a.qw, lut_w);
        fill_lut(a.qs, lut_s);
        __syncthreads();
    }
    float4* xfer = smem + table_floats(G) / 4;
    constexpr int K = kernel_tiles(C, FULL, PL, half_kernel<QW, QS, PL>());
    __shared__ double red[SplitServe<QS, C>::value && K == 1 ? C * kWave : 1];
    const int64_t first = a.tile0 + block_slot(a) * K;
    const int64_t left = a.tile1 - first;
    round_tiles<C, K, VEC, FULL, QW, QS, PL>(a, first, left < K ? (int)left : K, lut_w, lut_s, xfer, G, red);
}

}  // namespace

}  // namespace ea
