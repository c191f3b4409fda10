// ea_sym_c8.hip -- fully specialized fused-round kernels for buckets of
// 2048 elements with the same quantizer on both sides and Adam at the server:
// scaled sign, stochastic uniform with 1, 2, 4 or 8 bits and an L2 or
// max-norm scale, top-k and random-k.  With tiles this wide a run-time server
// quantizer needs most of the registers of the block, so the worker-specialized
// kernels run about half as fast as these.
#include "ea_round.hpp"

namespace ea {

namespace {

// Two waves per SIMD (up to 256 VGPRs): capped at 168 for a third wave, these
// kernels spill 30 to 70 VGPRs and run up to 1.6x slower on a BERT-sized
// round.
#ifndef EA_SYM_C8_MIN_WAVES
#define EA_SYM_C8_MIN_WAVES 2
#endif
// The sparsifiers' whole-tile kernels serve on eight waves and select on one
// (SparseServe), and fit in fewer registers.
#ifndef EA_SYM_C8_TOPK_MIN_WAVES
#define EA_SYM_C8_TOPK_MIN_WAVES 4
#endif
#ifndef EA_SYM_C8_RANDK_MIN_WAVES
#define EA_SYM_C8_RANDK_MIN_WAVES 3
#endif

template <class Q, int MW = EA_SYM_C8_MIN_WAVES>
constexpr SymKernel sym()
{
    return SymKernel{8, Q::kind(QDev{}), Q::bits(QDev{}), Q::norm(QDev{}), Q::cpb(QDev{}),
                     step_kernel<8, true, true, Q, Q, AT_SERVER, MW>,
                     round_tiles_per_block(8, true), step_kernel<8, true, false, Q, Q, AT_SERVER, EA_SYM_C8_MIN_WAVES>};
}

const SymKernel kSym[] = {
    sym<QCt<Q_SCALED_SIGN, 1, S_L1, 8>>(),
    sym<QCt<Q_STOCH, 1, S_L2, 8>>(),
    sym<QCt<Q_STOCH, 1, S_MAX, 8>>(),
    sym<QCt<Q_STOCH, 2, S_L2, 8>>(),
    sym<QCt<Q_STOCH, 2, S_MAX, 8>>(),
    sym<QCt<Q_STOCH, 4, S_L2, 8>>(),
    sym<QCt<Q_STOCH, 4, S_MAX, 8>>(),
    sym<QCt<Q_STOCH, 8, S_L2, 8>>(),
    sym<QCt<Q_STOCH, 8, S_MAX, 8>>(),
    sym<QCt<Q_TOPK, 1, S_MAX, 8>, EA_SYM_C8_TOPK_MIN_WAVES>(),
    sym<QCt<Q_RANDK, 1, S_MAX, 8>, EA_SYM_C8_RANDK_MIN_WAVES>(),
};

}  // namespace

const SymKernel* sym_kernels_c8(int* n)
{
    *n = (int)(sizeof(kSym) / sizeof(kSym[0]));
    return kSym;
}

}  // namespace ea
