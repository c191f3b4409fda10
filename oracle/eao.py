"""ctypes wrapper of the C oracle (``eao.c``).  Test infrastructure only.

Arrays are numpy; every wrapper only marshals arguments.  The arithmetic is
in ``eao.c`` (Section IV, Algorithms 1-2 of the paper; Examples 1-2 and
Definition 3 of Section III).
"""
import ctypes as C
from dataclasses import dataclass
from typing import Optional

import numpy as np

from .build import ensure_built

Q_NONE, Q_SCALED_SIGN, Q_STOCH_UNIFORM, Q_DET_UNIFORM, Q_POW2, Q_TOPK, Q_RANDK = 0, 1, 2, 3, 4, 5, 6
SCALE_L1, SCALE_L2, SCALE_MAX = 0, 1, 2
ADAM_AT_SERVER, ADAM_AT_WORKER = 0, 1
SCHED_CONSTANT, SCHED_ASSUMPTION2, SCHED_STEP_DECAY = 0, 1, 2


class Quant(C.Structure):
    _fields_ = [("kind", C.c_int32), ("scale", C.c_int32), ("bits", C.c_int32),
                ("error_feedback", C.c_int32), ("bucket", C.c_int64),
                ("pow2_kmin", C.c_int32), ("pow2_kmax", C.c_int32), ("keep", C.c_int32),
                ("reserved", C.c_int32)]


class Config(C.Structure):
    _fields_ = [("d", C.c_int64), ("N", C.c_int32), ("placement", C.c_int32),
                ("beta1", C.c_float), ("beta2", C.c_float), ("lr", C.c_float),
                ("eps", C.c_float), ("seed", C.c_uint64), ("qw", Quant), ("qs", Quant)]


class Schedule(C.Structure):
    _fields_ = [("kind", C.c_int32), ("alpha", C.c_float), ("theta", C.c_float), ("factor", C.c_float),
                ("T", C.c_int64), ("period", C.c_int64)]


assert C.sizeof(Quant) == 40 and C.sizeof(Config) == 120 and C.sizeof(Schedule) == 32

_lib = None


def lib():
    global _lib
    if _lib is None:
        L = C.CDLL(ensure_built())
        P = C.c_void_p
        L.eao_philox4x32_10.argtypes = [P, P, P]
        L.eao_uniforms.argtypes = [C.c_uint64, C.c_uint32, C.c_uint32, C.c_int64, C.c_int64, P]
        L.eao_code_bits.argtypes = [C.POINTER(Quant)]
        L.eao_code_bits.restype = C.c_int32
        L.eao_bucket_len.argtypes = [C.POINTER(Quant), C.c_int64]
        L.eao_bucket_len.restype = C.c_int64
        L.eao_num_scales.argtypes = [C.POINTER(Quant), C.c_int64, C.c_int64]
        L.eao_num_scales.restype = C.c_int64
        L.eao_msg_words.argtypes = [C.POINTER(Quant), C.c_int64]
        L.eao_msg_words.restype = C.c_int64
        L.eao_quantize.argtypes = [C.POINTER(Quant), C.c_int64, C.c_int64, P, P, P, P, P]
        L.eao_quantize.restype = C.c_int
        L.eao_quantize_bucket.argtypes = [C.POINTER(Quant), C.c_int64, P, P, C.c_float, P, P]
        L.eao_quantize_bucket.restype = C.c_int
        L.eao_dequantize.argtypes = [C.POINTER(Quant), C.c_int64, C.c_int64, P, P, P]
        L.eao_dequantize.restype = C.c_int
        L.eao_pack.argtypes = [C.c_int32, C.c_int64, P, P]
        L.eao_unpack.argtypes = [C.c_int32, C.c_int64, P, P]
        L.eao_adam_moments.argtypes = [C.c_float, C.c_float, P, P, C.c_float]
        L.eao_adam_update.argtypes = [C.c_float, C.c_float, C.c_float]
        L.eao_adam_update.restype = C.c_float
        L.eao_step.argtypes = [C.POINTER(Config), C.c_uint32, C.c_int64, C.c_int64] + [P] * 15
        L.eao_step.restype = C.c_int
        L.eao_schedule_at.argtypes = [C.POINTER(Schedule), C.c_float, C.c_float, C.c_int64, P, P]
        L.eao_schedule_at.restype = C.c_int
        L.eao_toy_grad.argtypes = [C.c_int64, C.c_int32, P, P, P, P, P, P]
        _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data


def philox(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, np.uint32)
    lib().eao_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def uniforms(seed: int, t: int, stream: int, n0: int, length: int) -> np.ndarray:
    u = np.empty(length, np.float32)
    lib().eao_uniforms(seed, t, stream, n0, length, _ptr(u))
    return u


def code_bits(q: Quant) -> int:
    return lib().eao_code_bits(C.byref(q))


def bucket_len(q: Quant, d: int) -> int:
    return lib().eao_bucket_len(C.byref(q), d)


def num_scales(q: Quant, d: int, length: int) -> int:
    return lib().eao_num_scales(C.byref(q), d, length)


def msg_words(q: Quant, length: int) -> int:
    return lib().eao_msg_words(C.byref(q), length)


def quantize(q: Quant, p: np.ndarray, d: Optional[int] = None, u: Optional[np.ndarray] = None):
    """Quantize a bucket-aligned segment; returns (codes, deq, scales)."""
    p = np.ascontiguousarray(p, dtype=np.float32)
    n = p.size
    d = n if d is None else d
    codes = np.zeros(n, np.uint32)
    deq = np.zeros(n, np.float32)
    scales = np.zeros(max(num_scales(q, d, n), 1), np.float32)
    if u is not None:
        u = np.ascontiguousarray(u, dtype=np.float32)
    rc = lib().eao_quantize(C.byref(q), d, n, _ptr(p), _ptr(u), _ptr(codes), _ptr(deq), _ptr(scales))
    if rc != 0:
        raise ValueError("eao_quantize rejected the quantizer description")
    return codes, deq, scales[:num_scales(q, d, n)]


def quantize_bucket(q: Quant, p: np.ndarray, scale: float, u: Optional[np.ndarray] = None):
    """One bucket coded under the given scale instead of its own norm;
    returns (codes, deq)."""
    p = np.ascontiguousarray(p, dtype=np.float32)
    codes = np.zeros(p.size, np.uint32)
    deq = np.zeros(p.size, np.float32)
    if u is not None:
        u = np.ascontiguousarray(u, dtype=np.float32)
    rc = lib().eao_quantize_bucket(C.byref(q), p.size, _ptr(p), _ptr(u), float(np.float32(scale)),
                                   _ptr(codes), _ptr(deq))
    if rc != 0:
        raise ValueError("eao_quantize_bucket rejected its arguments")
    return codes, deq


def dequantize(q: Quant, codes: np.ndarray, scales: np.ndarray, d: Optional[int] = None) -> np.ndarray:
    codes = np.ascontiguousarray(codes, dtype=np.uint32)
    scales = np.ascontiguousarray(scales if scales.size else np.zeros(1), dtype=np.float32)
    n = codes.size
    d = n if d is None else d
    out = np.zeros(n, np.float32)
    rc = lib().eao_dequantize(C.byref(q), d, n, _ptr(codes), _ptr(scales), _ptr(out))
    if rc != 0:
        raise ValueError("eao_dequantize rejected the quantizer description")
    return out


def pack(bits: int, codes: np.ndarray) -> np.ndarray:
    codes = np.ascontiguousarray(codes, dtype=np.uint32)
    n = codes.size
    nw = (n + 1) // 2 if bits == 32 else ((n + 255) // 256) * 4 * bits
    words = np.zeros(nw, np.uint64)
    lib().eao_pack(bits, n, _ptr(codes), _ptr(words))
    return words


def unpack(bits: int, words: np.ndarray, n: int) -> np.ndarray:
    words = np.ascontiguousarray(words, dtype=np.uint64)
    codes = np.zeros(n, np.uint32)
    lib().eao_unpack(bits, n, _ptr(words), _ptr(codes))
    return codes


def adam_moments(beta1: float, beta2: float, m: float, v: float, g: float):
    mm = np.array([m], np.float32)
    vv = np.array([v], np.float32)
    lib().eao_adam_moments(beta1, beta2, _ptr(mm), _ptr(vv), g)
    return float(mm[0]), float(vv[0])


def schedule_at(s: Schedule, lr0: float, beta2_0: float, t: int):
    """(lr_t, beta2_t) as binary32 numpy scalars; ValueError for an invalid
    schedule (Assumption 2; Section V-B step decay)."""
    lr = np.zeros(1, np.float32)
    b2 = np.zeros(1, np.float32)
    if lib().eao_schedule_at(C.byref(s), lr0, beta2_0, t, _ptr(lr), _ptr(b2)) != 0:
        raise ValueError("invalid schedule")
    return lr[0], b2[0]


def toy_grad(A: np.ndarray, x_star: np.ndarray, xi: np.ndarray, x: np.ndarray, want_norm: bool = True):
    """Section V-A toy problem: g[N][d] = 2 A^T (A x - x* - xi_i) in binary32
    and the full gradient's squared norm (binary64)."""
    A = np.ascontiguousarray(A, np.float32)
    d = A.shape[0]
    xi = np.ascontiguousarray(xi, np.float32).reshape(-1, d)
    N = xi.shape[0]
    g = np.zeros((N, d), np.float32)
    gs = np.zeros(1, np.float64)
    lib().eao_toy_grad(d, N, _ptr(A), _ptr(np.ascontiguousarray(x_star, np.float32)), _ptr(xi),
                       _ptr(np.ascontiguousarray(x, np.float32)), _ptr(g), _ptr(gs) if want_norm else None)
    return g, float(gs[0])


def adam_update(lr: float, m: float, v: float) -> float:
    return float(lib().eao_adam_update(lr, m, v))


@dataclass
class State:
    """Optimizer state of one segment of the d-vector (Algorithms 1-2)."""
    e_w: np.ndarray                 # [N, len] worker residuals
    e_s: np.ndarray                 # [len] server residual
    x: np.ndarray                   # [len] parameters
    m: Optional[np.ndarray] = None  # [len] server moments (Adam at the server)
    v: Optional[np.ndarray] = None
    m_w: Optional[np.ndarray] = None  # [N, len] worker moments (Adam at the workers)
    v_w: Optional[np.ndarray] = None

    @staticmethod
    def init(cfg: Config, length: int, x1: Optional[np.ndarray] = None) -> "State":
        """m = 0, v = eps, e = 0 (initialization lines of Algorithms 1-2)."""
        N = cfg.N
        x = np.zeros(length, np.float32) if x1 is None else np.array(x1, np.float32, copy=True)
        st = State(e_w=np.zeros((N, length), np.float32), e_s=np.zeros(length, np.float32), x=x)
        if cfg.placement == ADAM_AT_WORKER:
            st.m_w = np.zeros((N, length), np.float32)
            st.v_w = np.full((N, length), cfg.eps, np.float32)
        else:
            st.m = np.zeros(length, np.float32)
            st.v = np.full(length, cfg.eps, np.float32)
        return st

    def copy(self) -> "State":
        cp = lambda a: None if a is None else a.copy()  # noqa: E731
        return State(cp(self.e_w), cp(self.e_s), cp(self.x), cp(self.m), cp(self.v),
                     cp(self.m_w), cp(self.v_w))


def step(cfg: Config, t: int, g: np.ndarray, st: State, n0: int = 0, want_srv_in: bool = False,
         want_inputs: bool = False):
    """One round on segment [n0, n0+len) in place; returns the messages (and,
    with want_inputs, the quantizer inputs "p_w" [N][len] and "q_s" [len])."""
    g = np.ascontiguousarray(g, dtype=np.float32)
    N = cfg.N
    length = g.shape[1]
    assert g.shape == (N, length)
    ww, sw = msg_words(cfg.qw, length), msg_words(cfg.qs, length)
    nsw, nss = num_scales(cfg.qw, cfg.d, length), num_scales(cfg.qs, cfg.d, length)
    out = {
        "wcodes": np.zeros((N, ww), np.uint64),
        "wscales": np.zeros((N, max(nsw, 1)), np.float32),
        "scodes": np.zeros(sw, np.uint64),
        "sscales": np.zeros(max(nss, 1), np.float32),
        "srv_in": np.zeros(length, np.float32) if want_srv_in else None,
        "p_w": np.zeros((N, length), np.float32) if want_inputs else None,
        "q_s": np.zeros(length, np.float32) if want_inputs else None,
    }
    rc = lib().eao_step(C.byref(cfg), t, n0, length, _ptr(g), _ptr(st.e_w), _ptr(st.m_w), _ptr(st.v_w),
                        _ptr(st.m), _ptr(st.v), _ptr(st.e_s), _ptr(st.x),
                        _ptr(out["wcodes"]), _ptr(out["wscales"]), _ptr(out["scodes"]),
                        _ptr(out["sscales"]), _ptr(out["srv_in"]), _ptr(out["p_w"]), _ptr(out["q_s"]))
    if rc != 0:
        raise ValueError("eao_step rejected its arguments")
    out["wscales"] = out["wscales"][:, :nsw]
    out["sscales"] = out["sscales"][:nss]
    return out
