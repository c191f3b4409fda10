"""Efficient-Adam oracle: a plain single-threaded C reference and its ctypes wrapper.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` import this package.  It shares no code
with the HIP path.  See ``eao.h`` for the definitions and their sources in the
paper (Section IV, Algorithms 1-2; Section III, Examples 1-2 and the
Definition 3 compressors).
"""
from .eao import (  # noqa: F401
    Q_NONE, Q_SCALED_SIGN, Q_STOCH_UNIFORM, Q_DET_UNIFORM, Q_POW2, Q_TOPK, Q_RANDK,
    SCALE_L1, SCALE_L2, SCALE_MAX, ADAM_AT_SERVER, ADAM_AT_WORKER,
    SCHED_CONSTANT, SCHED_ASSUMPTION2, SCHED_STEP_DECAY, Schedule, schedule_at, toy_grad,
    Quant, Config, lib, philox, uniforms, code_bits, bucket_len, num_scales,
    msg_words, quantize, quantize_bucket, dequantize, pack, unpack, adam_moments, adam_update,
    State, step,
)
