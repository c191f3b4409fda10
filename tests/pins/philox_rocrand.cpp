// Test pin: exposes rocRAND's Philox4x32-10 block function (a library
// implementation of Salmon et al., SC'11) so that the oracle's own Philox can
// be checked against it.  Host-only; compiled with g++ by the test suite.
#include <rocrand/rocrand_philox4x32_10.h>

namespace {
struct philox_block : rocrand_device::philox4x32_10_engine {
    static uint4 apply(uint4 ctr, uint2 key) { philox_block b; return b.ten_rounds(ctr, key); }
};
}  // namespace

extern "C" void pin_philox4x32_10(const unsigned* ctr, const unsigned* key, unsigned* out, long n)
{
    for (long i = 0; i < n; ++i) {
        uint4 r = philox_block::apply(make_uint4(ctr[4 * i], ctr[4 * i + 1], ctr[4 * i + 2], ctr[4 * i + 3]),
                                      make_uint2(key[2 * i], key[2 * i + 1]));
        out[4 * i] = r.x; out[4 * i + 1] = r.y; out[4 * i + 2] = r.z; out[4 * i + 3] = r.w;
    }
}

// rocRAND's Philox4x32-10 generator state, seeded with `seed`, at
// subsequence stream * 2^32 + t and offset n0: the successive 32-bit outputs
// from there, each taken as a 24-bit uniform (word >> 8) * 2^-24.
extern "C" void pin_uniforms(unsigned long long seed, unsigned t, unsigned stream, long long n0, long long len,
                             float* out)
{
    rocrand_state_philox4x32_10 st;
    rocrand_init(seed, ((unsigned long long)stream << 32) | t, (unsigned long long)n0, &st);
    for (long long i = 0; i < len; ++i) out[i] = (float)(rocrand(&st) >> 8) * (1.0f / 16777216.0f);
}
