"""Efficient-Adam (Chen, Shen, Liu, Luo) data-parallel round on MI355X.

The work runs in ``libea.so`` (hand-written HIP kernels for gfx950 behind the
C ABI of ``include/ea.h``); this package only binds it.  ``state`` allocates
the device buffers one round needs (PyTorch provides memory and streams).

The binding is loaded on first use of any of its names, so that the ``build``
submodule can be imported (and the library compiled) before the library
exists; using a name with no library built raises ImportError.
"""
_EXPORTS = (
    "EA_OK", "EA_ERR_ARG", "EA_ERR_ALIGN", "EA_ERR_HIP", "EA_ERR_UNSUPPORTED",
    "EA_Q_NONE", "EA_Q_SCALED_SIGN", "EA_Q_STOCH_UNIFORM", "EA_Q_DET_UNIFORM", "EA_Q_POW2", "EA_Q_TOPK", "EA_Q_RANDK",
    "EA_SCALE_L1", "EA_SCALE_L2", "EA_SCALE_MAX", "EA_ADAM_AT_SERVER", "EA_ADAM_AT_WORKER",
    "EA_SCHED_CONSTANT", "EA_SCHED_ASSUMPTION2", "EA_SCHED_STEP_DECAY", "EA_NOALLOC_SCRATCH_BYTES",
    "Quant", "Config", "Schedule", "EAError", "lib", "LIB_PATH",
    "ea_code_bits", "ea_msg_words", "ea_msg_scales", "ea_msg_bits", "ea_workspace_bytes", "ea_validate",
    "ea_last_error", "ea_state_init", "ea_worker_compress", "ea_server_aggregate_adam", "ea_server_compress",
    "ea_worker_apply", "ea_step", "ea_step_noalloc", "ea_schedule_at", "ea_step_scheduled", "ea_run", "ea_toy_workspace_bytes",
    "ea_toy_grad", "ea_toy_step",
)
__all__ = list(_EXPORTS)


def __getattr__(name):
    if name in _EXPORTS:
        from . import _binding
        return getattr(_binding, name)
    raise AttributeError(f"module {__name__!r} has no attribute {name!r}")


def __dir__():
    return sorted(list(globals()) + list(_EXPORTS))
