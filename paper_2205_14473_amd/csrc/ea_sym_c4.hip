// ea_sym_c4.hip -- fully specialized fused-round kernels for buckets of
// 1024 elements with the same quantizer on both sides and Adam at the server:
// scaled sign, stochastic uniform with 1, 2, 4 or 8 bits and an L2 or
// max-norm scale, top-k and random-k.  With tiles this wide a run-time server
// quantizer needs most of the registers of the block, so the worker-specialized
// kernels run about half as fast as these.
#include "ea_round.hpp"

namespace ea {

namespace {

template <class Q>
constexpr SymKernel sym()
{
    return SymKernel{4, Q::kind(QDev{}), Q::bits(QDev{}), Q::norm(QDev{}), Q::cpb(QDev{}),
                     step_kernel<4, true, true, Q, Q, AT_SERVER>, round_tiles_per_block(4, true),
                     step_kernel<4, true, false, Q, Q, AT_SERVER>};
}

const SymKernel kSym[] = {
    sym<QCt<Q_SCALED_SIGN, 1, S_L1, 4>>(),
    sym<QCt<Q_STOCH, 1, S_L2, 4>>(),
    sym<QCt<Q_STOCH, 1, S_MAX, 4>>(),
    sym<QCt<Q_STOCH, 2, S_L2, 4>>(),
    sym<QCt<Q_STOCH, 2, S_MAX, 4>>(),
    sym<QCt<Q_STOCH, 4, S_L2, 4>>(),
    sym<QCt<Q_STOCH, 4, S_MAX, 4>>(),
    sym<QCt<Q_STOCH, 8, S_L2, 4>>(),
    sym<QCt<Q_STOCH, 8, S_MAX, 4>>(),
    sym<QCt<Q_TOPK, 1, S_MAX, 4>>(),
    sym<QCt<Q_RANDK, 1, S_MAX, 4>>(),
};

}  // namespace

const SymKernel* sym_kernels_c4(int* n)
{
    *n = (int)(sizeof(kSym) / sizeof(kSym[0]));
    return kSym;
}

}  // namespace ea
