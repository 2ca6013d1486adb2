"""ctypes binding of the CPU oracle (test infrastructure only).

Only tests, the smoke check and the benchmark's CPU-baseline leg import this
module. It loads oracle/libzo_oracle.so (built by oracle/build.py) and exposes
numpy-friendly wrappers. Nothing here performs any of the method's arithmetic.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libzo_oracle.so")


class RefConfig(C.Structure):
    _fields_ = [
        ("n_layers", C.c_int32),
        ("vocab", C.c_int32),
        ("embed", C.c_int32),
        ("hidden", C.c_int32),
        ("wdtype", C.c_int32),
        ("probe", C.c_int32),
    ]


LOSS_FN = C.CFUNCTYPE(C.c_double, C.POINTER(C.c_double), C.c_uint64, C.c_void_p)

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            import importlib.util
            spec = importlib.util.spec_from_file_location("_zo_oracle_build", os.path.join(HERE, "build.py"))
            mod = importlib.util.module_from_spec(spec)
            spec.loader.exec_module(mod)
            mod.build()
        _lib = C.CDLL(LIB_PATH)
        _declare(_lib)
    return _lib


def _declare(L):
    u32p = C.POINTER(C.c_uint32)
    f32p = C.POINTER(C.c_float)
    f64p = C.POINTER(C.c_double)
    i32p = C.POINTER(C.c_int32)
    u8p = C.POINTER(C.c_uint8)
    u64p = C.POINTER(C.c_uint64)
    cfgp = C.POINTER(RefConfig)
    L.zo_ref_threads.restype = C.c_int
    L.zo_ref_philox4x32_10.argtypes = [u32p, u32p, u32p]
    L.zo_ref_log_f32.argtypes = [C.c_float]
    L.zo_ref_log_f32.restype = C.c_float
    L.zo_ref_log_f32_array.argtypes = [f32p, C.c_uint64, f32p]
    L.zo_ref_sincos_2pi_array.argtypes = [u32p, C.c_uint64, f32p, f32p]
    L.zo_ref_gauss_pairs.argtypes = [u32p, C.c_uint64, f32p]
    L.zo_ref_probe_value.argtypes = [C.c_int32, C.c_uint64, C.c_uint32, C.c_uint64]
    L.zo_ref_probe_value.restype = C.c_float
    L.zo_ref_probe.argtypes = [C.c_int32, C.c_uint64, C.c_uint32, C.c_uint64, C.c_uint64, f32p]
    L.zo_ref_param_count.argtypes = [cfgp]
    L.zo_ref_param_count.restype = C.c_uint64
    L.zo_ref_layout.argtypes = [cfgp, u64p, C.c_int32]
    L.zo_ref_init.argtypes = [cfgp, C.c_void_p, C.c_uint64]
    L.zo_ref_materialise.argtypes = [cfgp, C.c_void_p, C.c_uint64, C.c_uint32, C.c_double, C.c_int32, f64p]
    L.zo_ref_lstm_loss.argtypes = [cfgp, f64p, i32p, u8p, C.c_int32, C.c_int32, C.c_int32, f64p]
    L.zo_ref_lstm_loss.restype = C.c_double
    L.zo_ref_perturbed_losses_ex.argtypes = [cfgp, C.c_void_p, C.c_uint64, C.c_float, C.c_int32,
                                             C.c_uint32, i32p, u8p, C.c_int32, C.c_int32, C.c_int32,
                                             f64p, f64p]
    L.zo_ref_perturbed_losses.argtypes = [cfgp, C.c_void_p, C.c_uint64, C.c_float, C.c_int32,
                                          C.c_uint32, i32p, u8p, C.c_int32, C.c_int32, f32p, f32p]
    L.zo_ref_update_coeff.argtypes = [C.c_float, C.c_int32, C.c_float, C.c_float, C.c_float]
    L.zo_ref_update_coeff.restype = C.c_float
    L.zo_ref_fd_losses.argtypes = [cfgp, C.c_void_p, C.c_uint64, C.c_float, C.c_int32, C.c_uint32,
                                   C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p]
    L.zo_ref_fd_update_coeff.argtypes = [C.c_float, C.c_int32, C.c_float, C.c_float, C.c_float]
    L.zo_ref_fd_update_coeff.restype = C.c_float
    L.zo_ref_fd_update.argtypes = [cfgp, C.c_void_p, C.c_uint64, C.c_float, C.c_float, C.c_int32,
                                   C.c_uint32, C.c_void_p, C.c_float]
    L.zo_ref_update.argtypes = [cfgp, C.c_void_p, C.c_uint64, C.c_float, C.c_float, C.c_int32,
                                C.c_uint32, f32p, f32p]
    L.zo_ref_update_sampled.argtypes = [cfgp, C.c_void_p, C.c_uint64, C.c_float, C.c_float, C.c_int32,
                                        C.c_uint32, f32p, f32p, u64p, C.c_uint64, C.c_void_p]
    L.zo_ref_cd_losses_generic.argtypes = [C.c_uint64, f64p, C.c_int32, C.c_uint64, C.c_double,
                                           C.c_int32, C.c_uint32, C.c_int32, LOSS_FN, C.c_void_p,
                                           f64p, f64p]
    L.zo_ref_cd_gradient.argtypes = [C.c_uint64, C.c_int32, C.c_uint64, C.c_double, C.c_int32,
                                     C.c_uint32, f64p, f64p, f64p]


def _p(a, ct):
    return a.ctypes.data_as(C.POINTER(ct))


def cfg_struct(cfg) -> RefConfig:
    return RefConfig(cfg["n_layers"], cfg["vocab"], cfg["embed"], cfg["hidden"],
                     cfg["wdtype"], cfg["probe"])


def theta_dtype(cfg):
    return np.uint16 if cfg["wdtype"] == 1 else np.float32


# ---------------------------------------------------------------------------
def threads() -> int:
    return int(lib().zo_ref_threads())


def philox(ctr, key) -> np.ndarray:
    c = np.asarray(ctr, dtype=np.uint32)
    k = np.asarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().zo_ref_philox4x32_10(_p(c, C.c_uint32), _p(k, C.c_uint32), _p(out, C.c_uint32))
    return out


def log_f32(u: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(u, dtype=np.float32)
    out = np.empty_like(u)
    lib().zo_ref_log_f32_array(_p(u, C.c_float), u.size, _p(out, C.c_float))
    return out


def sincos_2pi(k24: np.ndarray):
    k = np.ascontiguousarray(k24, dtype=np.uint32)
    s = np.empty(k.shape, np.float32)
    c = np.empty(k.shape, np.float32)
    lib().zo_ref_sincos_2pi_array(_p(k, C.c_uint32), k.size, _p(s, C.c_float), _p(c, C.c_float))
    return s, c


def gauss_pairs(words: np.ndarray) -> np.ndarray:
    w = np.ascontiguousarray(words, dtype=np.uint32)
    out = np.empty(w.size, np.float32)
    lib().zo_ref_gauss_pairs(_p(w, C.c_uint32), w.size // 2, _p(out, C.c_float))
    return out


def probe(kind: int, seed: int, i: int, j0: int, n: int) -> np.ndarray:
    out = np.empty(n, np.float32)
    lib().zo_ref_probe(kind, seed, i, j0, n, _p(out, C.c_float))
    return out


def probe_value(kind: int, seed: int, i: int, j: int) -> float:
    return lib().zo_ref_probe_value(kind, seed, i, j)


def param_count(cfg) -> int:
    s = cfg_struct(cfg)
    return int(lib().zo_ref_param_count(C.byref(s)))


def layout(cfg) -> np.ndarray:
    s = cfg_struct(cfg)
    n = 3 * cfg["n_layers"] + 4
    off = np.zeros(n, np.uint64)
    assert lib().zo_ref_layout(C.byref(s), _p(off, C.c_uint64), n) == 0
    return off


def init(cfg, seed: int) -> np.ndarray:
    s = cfg_struct(cfg)
    theta = np.zeros(param_count(cfg), theta_dtype(cfg))
    assert lib().zo_ref_init(C.byref(s), theta.ctypes.data_as(C.c_void_p), seed) == 0
    return theta


def materialise(cfg, theta: np.ndarray, seed: int, i: int, signed_eps: float, negate=False) -> np.ndarray:
    s = cfg_struct(cfg)
    w = np.empty(param_count(cfg), np.float64)
    st = lib().zo_ref_materialise(C.byref(s), theta.ctypes.data_as(C.c_void_p), seed, i,
                                  float(signed_eps), int(negate), _p(w, C.c_double))
    assert st == 0
    return w


def lstm_loss(cfg, w: np.ndarray, tokens: np.ndarray, mask=None, token_losses=False):
    s = cfg_struct(cfg)
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    B, C1 = tokens.shape
    Cn = C1 - 1
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    tl = np.zeros((B, Cn), np.float64) if token_losses else None
    L = lib().zo_ref_lstm_loss(C.byref(s), _p(np.ascontiguousarray(w, np.float64), C.c_double),
                               _p(tokens, C.c_int32), None if m is None else _p(m, C.c_uint8),
                               B, Cn, C1, None if tl is None else _p(tl, C.c_double))
    return (L, tl) if token_losses else L


def perturbed_losses(cfg, theta, seed, eps, N, tokens, mask=None, i0=0, negate=False, as_double=False):
    s = cfg_struct(cfg)
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    B, C1 = tokens.shape
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    if as_double or negate:
        lp = np.zeros(N, np.float64)
        lm = np.zeros(N, np.float64)
        st = lib().zo_ref_perturbed_losses_ex(C.byref(s), theta.ctypes.data_as(C.c_void_p), seed,
                                              eps, N, i0, _p(tokens, C.c_int32),
                                              None if m is None else _p(m, C.c_uint8), B, C1 - 1,
                                              int(negate), _p(lp, C.c_double), _p(lm, C.c_double))
    else:
        lp = np.zeros(N, np.float32)
        lm = np.zeros(N, np.float32)
        st = lib().zo_ref_perturbed_losses(C.byref(s), theta.ctypes.data_as(C.c_void_p), seed, eps, N,
                                           i0, _p(tokens, C.c_int32),
                                           None if m is None else _p(m, C.c_uint8), B, C1 - 1,
                                           _p(lp, C.c_float), _p(lm, C.c_float))
    if st != 0:
        raise ValueError(f"oracle perturbed_losses status {st}")
    return lp, lm


def update_coeff(lr, N, lp, lm, eps) -> float:
    return lib().zo_ref_update_coeff(lr, N, lp, lm, eps)


def update(cfg, theta: np.ndarray, seed, eps, lr, Lp, Lm, i0=0) -> int:
    """In-place update of theta; returns the status code."""
    s = cfg_struct(cfg)
    Lp = np.ascontiguousarray(Lp, np.float32)
    Lm = np.ascontiguousarray(Lm, np.float32)
    return lib().zo_ref_update(C.byref(s), theta.ctypes.data_as(C.c_void_p), seed, eps, lr, Lp.size,
                               i0, _p(Lp, C.c_float), _p(Lm, C.c_float))


def fd_losses(cfg, theta, seed, eps, N, tokens, mask=None, i0=0):
    """Forward differences: (L [N] at theta + eps z_{i0+n}, L0 at theta), fp64."""
    s = cfg_struct(cfg)
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    B, C1 = tokens.shape
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    L = np.zeros(N, np.float64)
    L0 = np.zeros(1, np.float64)
    st = lib().zo_ref_fd_losses(C.byref(s), theta.ctypes.data_as(C.c_void_p), seed, eps, N, i0,
                                _p(tokens, C.c_int32), None if m is None else _p(m, C.c_uint8), B, C1 - 1,
                                _p(L, C.c_double), _p(L0, C.c_double))
    if st != 0:
        raise ValueError(f"oracle fd_losses status {st}")
    return L, float(L0[0])


def fd_update_coeff(lr, N, L, L0, eps) -> float:
    return lib().zo_ref_fd_update_coeff(lr, N, L, L0, eps)


def fd_update(cfg, theta: np.ndarray, seed, eps, lr, L, L0, i0=0) -> int:
    """In-place forward-difference update of theta; returns the status code."""
    s = cfg_struct(cfg)
    L = np.ascontiguousarray(L, np.float32)
    return lib().zo_ref_fd_update(C.byref(s), theta.ctypes.data_as(C.c_void_p), seed, eps, lr, L.size, i0,
                                  _p(L, C.c_float), float(np.float32(L0)))


def update_sampled(cfg, theta, seed, eps, lr, Lp, Lm, idx, i0=0) -> np.ndarray:
    s = cfg_struct(cfg)
    Lp = np.ascontiguousarray(Lp, np.float32)
    Lm = np.ascontiguousarray(Lm, np.float32)
    idx = np.ascontiguousarray(idx, np.uint64)
    out = np.zeros(idx.size, theta_dtype(cfg))
    st = lib().zo_ref_update_sampled(C.byref(s), theta.ctypes.data_as(C.c_void_p), seed, eps, lr,
                                     Lp.size, i0, _p(Lp, C.c_float), _p(Lm, C.c_float),
                                     _p(idx, C.c_uint64), idx.size, out.ctypes.data_as(C.c_void_p))
    if st != 0:
        raise ValueError(f"oracle update_sampled status {st}")
    return out


def cd_losses_generic(theta: np.ndarray, loss, kind, seed, eps, N, i0=0, negate=False):
    theta = np.ascontiguousarray(theta, np.float64)
    P = theta.size

    def cb(wp, n, ctx):
        return float(loss(np.ctypeslib.as_array(wp, shape=(n,))))

    fn = LOSS_FN(cb)
    lp = np.zeros(N, np.float64)
    lm = np.zeros(N, np.float64)
    st = lib().zo_ref_cd_losses_generic(P, _p(theta, C.c_double), kind, seed, eps, N, i0, int(negate),
                                        fn, None, _p(lp, C.c_double), _p(lm, C.c_double))
    assert st == 0
    return lp, lm


def cd_gradient(P, kind, seed, eps, Lp, Lm, i0=0) -> np.ndarray:
    Lp = np.ascontiguousarray(Lp, np.float64)
    Lm = np.ascontiguousarray(Lm, np.float64)
    g = np.zeros(P, np.float64)
    lib().zo_ref_cd_gradient(P, kind, seed, eps, Lp.size, i0, _p(Lp, C.c_double), _p(Lm, C.c_double),
                             _p(g, C.c_double))
    return g


def bf16_to_f32(a: np.ndarray) -> np.ndarray:
    return (a.astype(np.uint32) << 16).view(np.float32)


def theta_as_f64(cfg, theta: np.ndarray) -> np.ndarray:
    if cfg["wdtype"] == 1:
        return bf16_to_f32(theta).astype(np.float64)
    return theta.astype(np.float64)
