"""ctypes binding of libea's C ABI (include/ea.h): argument marshalling only.

Every function has the name of the C entry point it calls.  Tensor arguments
must be contiguous device tensors of the documented dtype (or None where the
header allows NULL); streams are torch streams, raw hipStream_t integers, or
None for torch's current stream.  There is no fallback: if the shared library
is missing the import fails.
"""
import ctypes as C
import os

PKG = os.path.dirname(os.path.abspath(__file__))
# EA_LIB names another build of the same sources to load instead (the host
# code built with sanitizers, for the CPU tests); it must exist.
LIB_PATH = os.environ.get("EA_LIB") or os.path.join(PKG, "libea.so")

EA_OK, EA_ERR_ARG, EA_ERR_ALIGN, EA_ERR_HIP, EA_ERR_UNSUPPORTED = 0, -1, -2, -3, -4
EA_Q_NONE, EA_Q_SCALED_SIGN, EA_Q_STOCH_UNIFORM, EA_Q_DET_UNIFORM, EA_Q_POW2, EA_Q_TOPK, EA_Q_RANDK = 0, 1, 2, 3, 4, 5, 6
EA_SCALE_L1, EA_SCALE_L2, EA_SCALE_MAX = 0, 1, 2
EA_ADAM_AT_SERVER, EA_ADAM_AT_WORKER = 0, 1
EA_SCHED_CONSTANT, EA_SCHED_ASSUMPTION2, EA_SCHED_STEP_DECAY = 0, 1, 2
EA_NOALLOC_SCRATCH_BYTES = 16 << 20


class Quant(C.Structure):
    """ea_quant_t"""
    _fields_ = [("kind", C.c_int32), ("scale", C.c_int32), ("bits", C.c_int32),
                ("error_feedback", C.c_int32), ("bucket", C.c_int64),
                ("pow2_kmin", C.c_int32), ("pow2_kmax", C.c_int32), ("keep", C.c_int32),
                ("reserved", C.c_int32)]


class Config(C.Structure):
    """ea_config_t"""
    _fields_ = [("d", C.c_int64), ("N", C.c_int32), ("placement", C.c_int32),
                ("beta1", C.c_float), ("beta2", C.c_float), ("lr", C.c_float), ("eps", C.c_float),
                ("seed", C.c_uint64), ("qw", Quant), ("qs", Quant)]


class Schedule(C.Structure):
    """ea_schedule_t"""
    _fields_ = [("kind", C.c_int32), ("alpha", C.c_float), ("theta", C.c_float), ("factor", C.c_float),
                ("T", C.c_int64), ("period", C.c_int64)]


assert C.sizeof(Quant) == 40 and C.sizeof(Config) == 120 and C.sizeof(Schedule) == 32


class EAError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libea error {code}: {msg}")
        self.code = code


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2205_14473_amd.build` "
                          "(hipcc --offload-arch=gfx950) first")
    L = C.CDLL(LIB_PATH)
    P, I32, I64 = C.c_void_p, C.c_int32, C.c_int64
    QP, CP, SP = C.POINTER(Quant), C.POINTER(Config), C.POINTER(Schedule)
    sig = {
        "ea_code_bits": (I32, [QP]),
        "ea_msg_words": (I64, [QP, I64]),
        "ea_msg_scales": (I64, [QP, I64]),
        "ea_msg_bits": (I64, [QP, I64]),
        "ea_workspace_bytes": (I64, [CP]),
        "ea_validate": (C.c_int, [CP]),
        "ea_last_error": (C.c_char_p, []),
        "ea_state_init": (C.c_int, [CP, P, P, P, P, P, P, P]),
        "ea_worker_compress": (C.c_int, [CP, I32, I64, P, P, P, P, P, P, P, P]),
        "ea_server_aggregate_adam": (C.c_int, [CP, I64, P, P, P, P, P, P]),
        "ea_server_compress": (C.c_int, [CP, I64, P, P, P, P, P, P]),
        "ea_worker_apply": (C.c_int, [CP, P, P, P, P]),
        "ea_step": (C.c_int, [CP, I64] + [P] * 14),
        "ea_step_noalloc": (C.c_int, [CP, I64] + [P] * 13),
        "ea_schedule_at": (C.c_int, [CP, SP, I64, P, P]),
        "ea_step_scheduled": (C.c_int, [CP, SP] + [P] * 15),
        "ea_run": (C.c_int, [CP, SP, I64, I64, P, I64] + [P] * 13),
        "ea_toy_workspace_bytes": (I64, [I64]),
        "ea_toy_grad": (C.c_int, [I64, I32] + [P] * 8),
        "ea_toy_step": (C.c_int, [CP, I64] + [P] * 16),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype, f.argtypes = res, args
    return L


lib = _load()


def ea_last_error() -> str:
    return lib.ea_last_error().decode()


def _check(rc: int) -> int:
    if rc < 0:
        raise EAError(rc, ea_last_error())
    return rc


def _ptr(t, dtype=None):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("libea needs device tensors")
    if not t.is_contiguous():
        raise ValueError("libea needs contiguous tensors")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"expected {dtype}, got {t.dtype}")
    return t.data_ptr()


def _stream(stream):
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _f32():
    import torch
    return torch.float32


def _u64():
    import torch
    return torch.uint64


def ea_code_bits(q: Quant) -> int:
    return _check(lib.ea_code_bits(C.byref(q)))


def ea_msg_words(q: Quant, d: int) -> int:
    return _check(lib.ea_msg_words(C.byref(q), d))


def ea_msg_scales(q: Quant, d: int) -> int:
    return _check(lib.ea_msg_scales(C.byref(q), d))


def ea_msg_bits(q: Quant, d: int) -> int:
    return _check(lib.ea_msg_bits(C.byref(q), d))


def ea_workspace_bytes(cfg: Config) -> int:
    return _check(lib.ea_workspace_bytes(C.byref(cfg)))


def ea_validate(cfg: Config) -> int:
    return lib.ea_validate(C.byref(cfg))


def ea_state_init(cfg, m, v, e_s, e_w, m_w, v_w, stream=None):
    f = _f32()
    return _check(lib.ea_state_init(C.byref(cfg), _ptr(m, f), _ptr(v, f), _ptr(e_s, f), _ptr(e_w, f),
                                    _ptr(m_w, f), _ptr(v_w, f), _stream(stream)))


def ea_worker_compress(cfg, i, t, g, e_w, m_w, v_w, codes, scales, workspace=None, stream=None):
    f, u = _f32(), _u64()
    return _check(lib.ea_worker_compress(C.byref(cfg), i, t, _ptr(g, f), _ptr(e_w, f), _ptr(m_w, f),
                                         _ptr(v_w, f), _ptr(codes, u), _ptr(scales, f), _ptr(workspace),
                                         _stream(stream)))


def ea_server_aggregate_adam(cfg, t, wcodes, wscales, m, v, u_out, stream=None):
    f, u = _f32(), _u64()
    return _check(lib.ea_server_aggregate_adam(C.byref(cfg), t, _ptr(wcodes, u), _ptr(wscales, f), _ptr(m, f),
                                               _ptr(v, f), _ptr(u_out, f), _stream(stream)))


def ea_server_compress(cfg, t, u_in, e_s, codes, scales, workspace=None, stream=None):
    f, u = _f32(), _u64()
    return _check(lib.ea_server_compress(C.byref(cfg), t, _ptr(u_in, f), _ptr(e_s, f), _ptr(codes, u),
                                         _ptr(scales, f), _ptr(workspace), _stream(stream)))


def ea_worker_apply(cfg, codes, scales, x, stream=None):
    f, u = _f32(), _u64()
    return _check(lib.ea_worker_apply(C.byref(cfg), _ptr(codes, u), _ptr(scales, f), _ptr(x, f),
                                      _stream(stream)))


def ea_step(cfg, t, g, e_w, m_w, v_w, m, v, e_s, x, wcodes, wscales, scodes, sscales, workspace=None,
            stream=None):
    f, u = _f32(), _u64()
    return _check(lib.ea_step(C.byref(cfg), t, _ptr(g, f), _ptr(e_w, f), _ptr(m_w, f), _ptr(v_w, f),
                              _ptr(m, f), _ptr(v, f), _ptr(e_s, f), _ptr(x, f), _ptr(wcodes, u),
                              _ptr(wscales, f), _ptr(scodes, u), _ptr(sscales, f), _ptr(workspace),
                              _stream(stream)))


def ea_step_noalloc(cfg, t, g, e_w, m_w, v_w, m, v, e_s, x, wcodes, wscales, scodes, sscales, stream=None):
    f, u = _f32(), _u64()
    return _check(lib.ea_step_noalloc(C.byref(cfg), t, _ptr(g, f), _ptr(e_w, f), _ptr(m_w, f), _ptr(v_w, f),
                                      _ptr(m, f), _ptr(v, f), _ptr(e_s, f), _ptr(x, f), _ptr(wcodes, u),
                                      _ptr(wscales, f), _ptr(scodes, u), _ptr(sscales, f), _stream(stream)))


def ea_schedule_at(cfg, sched, t):
    """(lr_t, beta2_t) of the schedule at step t, as Python floats of binary32 values."""
    lr, b2 = C.c_float(), C.c_float()
    _check(lib.ea_schedule_at(C.byref(cfg), C.byref(sched), t, C.byref(lr), C.byref(b2)))
    return lr.value, b2.value


def _ptr_u32(t):
    if t is None or isinstance(t, int):
        return t
    if t.element_size() != 4 or t.is_floating_point():
        raise ValueError("t_dev must be a 4-byte integer tensor")
    return _ptr(t)


def ea_step_scheduled(cfg, sched, t_dev, g, e_w, m_w, v_w, m, v, e_s, x, wcodes, wscales, scodes, sscales,
                      workspace=None, stream=None):
    f, u = _f32(), _u64()
    return _check(lib.ea_step_scheduled(C.byref(cfg), C.byref(sched), _ptr_u32(t_dev), _ptr(g, f), _ptr(e_w, f),
                                        _ptr(m_w, f), _ptr(v_w, f), _ptr(m, f), _ptr(v, f), _ptr(e_s, f),
                                        _ptr(x, f), _ptr(wcodes, u), _ptr(wscales, f), _ptr(scodes, u),
                                        _ptr(sscales, f), _ptr(workspace), _stream(stream)))


def ea_run(cfg, sched, t0, steps, g, g_step_stride, e_w, m_w, v_w, m, v, e_s, x, wcodes, wscales, scodes,
           sscales, workspace=None, stream=None):
    f, u = _f32(), _u64()
    return _check(lib.ea_run(C.byref(cfg), C.byref(sched), t0, steps, _ptr(g, f), g_step_stride, _ptr(e_w, f),
                             _ptr(m_w, f), _ptr(v_w, f), _ptr(m, f), _ptr(v, f), _ptr(e_s, f), _ptr(x, f),
                             _ptr(wcodes, u), _ptr(wscales, f), _ptr(scodes, u), _ptr(sscales, f),
                             _ptr(workspace), _stream(stream)))


def ea_toy_workspace_bytes(d):
    return _check(lib.ea_toy_workspace_bytes(d))


def ea_toy_grad(d, N, A, x_star, xi, x, g, grad_sq, workspace, stream=None):
    import torch
    f = _f32()
    return _check(lib.ea_toy_grad(d, N, _ptr(A, f), _ptr(x_star, f), _ptr(xi, f), _ptr(x, f), _ptr(g, f),
                                  _ptr(grad_sq, torch.float64), _ptr(workspace), _stream(stream)))


def ea_toy_step(cfg, t, A, x_star, xi, e_w, m_w, v_w, m, v, e_s, x, wcodes, scodes, grad_sq, g_out, workspace,
                stream=None):
    import torch
    f, u = _f32(), _u64()
    return _check(lib.ea_toy_step(C.byref(cfg), t, _ptr(A, f), _ptr(x_star, f), _ptr(xi, f), _ptr(e_w, f),
                                  _ptr(m_w, f), _ptr(v_w, f), _ptr(m, f), _ptr(v, f), _ptr(e_s, f), _ptr(x, f),
                                  _ptr(wcodes, u), _ptr(scodes, u), _ptr(grad_sq, torch.float64), _ptr(g_out, f),
                                  _ptr(workspace), _stream(stream)))
