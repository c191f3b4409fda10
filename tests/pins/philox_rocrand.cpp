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
