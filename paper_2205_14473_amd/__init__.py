"""Efficient-Adam (Chen, Shen, Liu, Luo) data-parallel round on MI355X.

The work runs in ``libea.so`` (hand-written HIP kernels for gfx950 behind the
C ABI of ``include/ea.h``); this package only binds it.  ``state`` allocates
the device buffers one round needs (PyTorch provides memory and streams).
"""
from ._binding import (  # noqa: F401
    EA_OK, EA_ERR_ARG, EA_ERR_ALIGN, EA_ERR_HIP, EA_ERR_UNSUPPORTED,
    EA_Q_NONE, EA_Q_SCALED_SIGN, EA_Q_STOCH_UNIFORM, EA_Q_DET_UNIFORM, EA_Q_POW2,
    EA_SCALE_L1, EA_SCALE_L2, EA_SCALE_MAX, EA_ADAM_AT_SERVER, EA_ADAM_AT_WORKER,
    EA_SCHED_CONSTANT, EA_SCHED_ASSUMPTION2, EA_SCHED_STEP_DECAY,
    Quant, Config, Schedule, EAError, lib, LIB_PATH,
    ea_code_bits, ea_msg_words, ea_msg_scales, ea_msg_bits, ea_workspace_bytes, ea_validate,
    ea_last_error, ea_state_init, ea_worker_compress, ea_server_aggregate_adam, ea_server_compress,
    ea_worker_apply, ea_step, ea_schedule_at, ea_step_scheduled, ea_run,
)
