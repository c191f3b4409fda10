// ea_half_c4.hip -- fused-round and split-call kernels for buckets of 1024 elements
// (4 chunks per tile) with the worker quantizer fixed at compile time: scaled
// sign, stochastic uniform with 1, 2, 4 or 8 bits and an L2 or max-norm
// scale, top-k, random-k, Example 1 with 2 or 3 bits, and (with no bucket,
// so at any tile size) Example 2 with 4-bit codes and full precision.  The
// server quantizer and the Adam placement are read at run time.  The
// workers' per-element work is N times the server's, so these kernels run
// close to the fully specialized ones.
#include "ea_round.hpp"

namespace ea {

namespace {

template <class QW>
constexpr HalfKernel half()
{
    return HalfKernel{4, QW::kind(QDev{}), QW::bits(QDev{}), QW::norm(QDev{}), QW::cpb(QDev{}),
                      step_kernel<4, true, true, QW, QRt, -1>, kernel_tiles(4, true, -1, true),
                      worker_kernel<4, true, QW>, aggregate_kernel<4, true, QW>, aggregate_kernel<4, true, QW, true>,
                      server_kernel<4, true, QW>, apply_kernel<4, true, QW>};
}

const HalfKernel kHalf[] = {
    half<QCt<Q_SCALED_SIGN, 1, S_L1, 4>>(),
    half<QCt<Q_STOCH, 1, S_L2, 4>>(),
    half<QCt<Q_STOCH, 1, S_MAX, 4>>(),
    half<QCt<Q_STOCH, 2, S_L2, 4>>(),
    half<QCt<Q_STOCH, 2, S_MAX, 4>>(),
    half<QCt<Q_STOCH, 4, S_L2, 4>>(),
    half<QCt<Q_STOCH, 4, S_MAX, 4>>(),
    half<QCt<Q_STOCH, 8, S_L2, 4>>(),
    half<QCt<Q_STOCH, 8, S_MAX, 4>>(),
    half<QCt<Q_TOPK, 1, S_MAX, 4>>(),
    half<QCt<Q_RANDK, 1, S_MAX, 4>>(),
    half<QCt<Q_DET, 2, S_MAX, 4>>(),
    half<QCt<Q_DET, 3, S_MAX, 4>>(),
    half<QCt<Q_POW2, 4, S_MAX, 0>>(),
    half<QCt<Q_NONE, 32, S_MAX, 0>>(),
};

}  // namespace

const HalfKernel* half_kernels_c4(int* n)
{
    *n = (int)(sizeof(kHalf) / sizeof(kHalf[0]));
    return kHalf;
}

}  // namespace ea
