"""Python binding of libzo.so (the HIP library of the CD-RGE step).

Argument marshalling only: every computation runs in the library's HIP
kernels. PyTorch supplies device memory (torch.cuda tensors) and the stream
(the current torch stream unless one is passed). The library must have been
built (paper_2505_17852_amd/build.py); there is no fallback of any kind.

Function names follow the C ABI in include/zo.h:
    param_count, workspace_bytes, workspace_bytes_min, init, perturbed_losses
    (zo_perturbed_losses / _ex), update, fd_losses (zo_fd_losses / _ex),
    fd_update, debug_probe, debug_gauss_pairs
A model configuration is a dict with the keys n_layers, vocab, embed,
hidden, wdtype (0 fp32, 1 bf16) and probe (0 Rademacher, 1 normal).
"""
from __future__ import annotations

import ctypes as C
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libzo.so")

ZO_OK, ZO_EINVAL, ZO_ESHAPE, ZO_EDEVICE, ZO_ENOMEM, ZO_ENONFINITE = 0, -1, -2, -3, -4, -5
FP32, BF16 = 0, 1
RADEMACHER, GAUSSIAN = 0, 1
# form of the perturbed products (bf16 weights: fused fp16(W + s eps z) or the
# two-stream A.W + A.(s eps z)); AUTO picks by eps
PRODUCTS_AUTO, PRODUCTS_FUSED, PRODUCTS_SPLIT = 0, 1, 2
BF16_FUSED_EPS_MIN = 2.0 ** -10  # ZO_BF16_FUSED_EPS_MIN
BF16_EPS_MIN = 2.0 ** -17        # ZO_BF16_EPS_MIN


class ZoError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"zo status {status}: {message}")
        self.status = status


class Config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("vocab", C.c_int32), ("embed", C.c_int32),
                ("hidden", C.c_int32), ("wdtype", C.c_int32), ("probe", C.c_int32)]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python paper_2505_17852_amd/build.py`")
        L = C.CDLL(LIB_PATH)
        vp, cfgp = C.c_void_p, C.POINTER(Config)
        L.zo_param_count.argtypes = [cfgp]
        L.zo_param_count.restype = C.c_size_t
        L.zo_workspace_bytes.argtypes = [cfgp, C.c_int32, C.c_int32, C.c_int32]
        L.zo_workspace_bytes.restype = C.c_size_t
        L.zo_workspace_bytes_min.argtypes = [cfgp, C.c_int32, C.c_int32, C.c_int32]
        L.zo_workspace_bytes_min.restype = C.c_size_t
        L.zo_init.argtypes = [cfgp, vp, C.c_uint64, vp]
        L.zo_perturbed_losses.argtypes = [cfgp, vp, C.c_uint64, C.c_float, C.c_int32, C.c_uint32,
                                          vp, vp, C.c_int32, C.c_int32, vp, vp, vp, C.c_size_t, vp]
        L.zo_update.argtypes = [cfgp, vp, C.c_uint64, C.c_float, C.c_float, C.c_int32, C.c_uint32,
                                vp, vp, vp, vp]
        L.zo_fd_losses.argtypes = [cfgp, vp, C.c_uint64, C.c_float, C.c_int32, C.c_uint32,
                                   vp, vp, C.c_int32, C.c_int32, vp, vp, vp, C.c_size_t, vp]
        L.zo_perturbed_losses_ex.argtypes = [cfgp, vp, C.c_uint64, C.c_float, C.c_int32, C.c_uint32,
                                             vp, vp, C.c_int32, C.c_int32, vp, vp, vp, C.c_size_t,
                                             C.c_int32, vp]
        L.zo_perturbed_losses_noalloc.argtypes = [cfgp, vp, C.c_uint64, C.c_float, C.c_int32, C.c_uint32,
                                                  vp, vp, C.c_int32, C.c_int32, vp, vp, vp]
        L.zo_fd_losses_ex.argtypes = [cfgp, vp, C.c_uint64, C.c_float, C.c_int32, C.c_uint32,
                                      vp, vp, C.c_int32, C.c_int32, vp, vp, vp, C.c_size_t, C.c_int32, vp]
        L.zo_probe_bits_offset.argtypes = [cfgp, C.c_int32, C.c_int32, C.c_int32]
        L.zo_probe_bits_offset.restype = C.c_size_t
        L.zo_update_cached.argtypes = [cfgp, vp, C.c_uint64, C.c_float, C.c_float, C.c_int32, C.c_uint32,
                                       vp, vp, vp, vp, vp]
        L.zo_fd_update.argtypes = [cfgp, vp, C.c_uint64, C.c_float, C.c_float, C.c_int32, C.c_uint32,
                                   vp, vp, vp, vp]
        L.zo_debug_probe.argtypes = [C.c_int32, C.c_uint64, C.c_uint32, C.c_uint64, C.c_uint64, vp, vp]
        L.zo_debug_gauss_pairs.argtypes = [vp, C.c_uint64, vp, vp]
        L.zo_profile_enable.argtypes = [C.c_int32]
        L.zo_profile_read.argtypes = [C.c_int32, C.POINTER(C.c_double), C.POINTER(C.c_int64),
                                      C.POINTER(C.c_int64)]
        L.zo_last_error.restype = C.c_char_p
        for f in ("zo_init", "zo_perturbed_losses", "zo_update", "zo_fd_losses", "zo_fd_update",
                  "zo_perturbed_losses_ex", "zo_fd_losses_ex", "zo_perturbed_losses_noalloc", "zo_update_cached",
                  "zo_debug_probe",
                  "zo_debug_gauss_pairs", "zo_profile_enable", "zo_profile_read"):
            getattr(L, f).restype = C.c_int
        _lib = L
    return _lib


def _cfg(cfg) -> Config:
    return Config(int(cfg["n_layers"]), int(cfg["vocab"]), int(cfg["embed"]), int(cfg["hidden"]),
                  int(cfg["wdtype"]), int(cfg["probe"]))


def _check(st: int):
    if st != ZO_OK:
        raise ZoError(st, lib().zo_last_error().decode())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _dev(t: torch.Tensor, dtype, name: str):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return C.c_void_p(t.data_ptr())


def theta_dtype(cfg):
    return torch.bfloat16 if int(cfg["wdtype"]) == BF16 else torch.float32


def _theta(cfg, theta: torch.Tensor):
    """theta's device pointer after checking its type and its length, P."""
    p = _dev(theta, theta_dtype(cfg), "theta")
    if theta.numel() != param_count(cfg):
        raise ValueError(f"theta has {theta.numel()} elements, the model has {param_count(cfg)}")
    return p


def param_count(cfg) -> int:
    c = _cfg(cfg)
    return int(lib().zo_param_count(C.byref(c)))


def workspace_bytes(cfg, N: int, B: int, C_: int) -> int:
    c = _cfg(cfg)
    return int(lib().zo_workspace_bytes(C.byref(c), N, B, C_))


def new_theta(cfg, device="cuda") -> torch.Tensor:
    return torch.empty(param_count(cfg), dtype=theta_dtype(cfg), device=device)


def init(cfg, theta: torch.Tensor, seed: int, stream=None):
    c = _cfg(cfg)
    _check(lib().zo_init(C.byref(c), _theta(cfg, theta), seed, _stream(stream)))


def workspace_bytes_min(cfg, N: int, B: int, C_: int) -> int:
    c = _cfg(cfg)
    return int(lib().zo_workspace_bytes_min(C.byref(c), N, B, C_))


def new_workspace(cfg, N: int, B: int, C_: int, device="cuda", probe_cache: bool = True) -> torch.Tensor:
    """Device workspace for zo_perturbed_losses; probe_cache=False gives the
    smallest one (normal probes then regenerated in every tile)."""
    n = workspace_bytes(cfg, N, B, C_) if probe_cache else workspace_bytes_min(cfg, N, B, C_)
    if n == 0:
        raise ValueError("invalid workspace request")
    return torch.empty(n, dtype=torch.uint8, device=device)


def perturbed_losses(cfg, theta: torch.Tensor, seed: int, eps: float, N: int,
                     tokens: torch.Tensor, mask: torch.Tensor | None = None, i0: int = 0,
                     Lplus: torch.Tensor | None = None, Lminus: torch.Tensor | None = None,
                     workspace: torch.Tensor | None = None, stream=None,
                     check_tokens: bool = True, products: int = PRODUCTS_AUTO):
    """Returns (L+, L-) as device fp32 tensors of N elements (asynchronous).

    The kernels never read memory by an id outside [0, vocab): such an id
    makes the affected losses non-finite (and zo_update then skips). With
    check_tokens (default) this wrapper rejects them first (one device
    sync). products: PRODUCTS_AUTO (zo_perturbed_losses), or PRODUCTS_FUSED /
    PRODUCTS_SPLIT (zo_perturbed_losses_ex, for measurement)."""
    c = _cfg(cfg)
    if tokens.dim() != 2:
        raise ValueError("tokens must be [B][C+1]")
    if check_tokens and tokens.numel():
        lo, hi = int(tokens.min()), int(tokens.max())
        if lo < 0 or hi >= int(cfg["vocab"]):
            raise ValueError(f"token ids must lie in [0, {cfg['vocab']}), got [{lo}, {hi}]")
    B, C1 = tokens.shape
    Cn = C1 - 1
    if mask is not None and tuple(mask.shape) != (B, Cn):
        raise ValueError("mask must be [B][C]")
    dev = theta.device
    if Lplus is None:
        Lplus = torch.empty(N, dtype=torch.float32, device=dev)
    if Lminus is None:
        Lminus = torch.empty(N, dtype=torch.float32, device=dev)
    if Lplus.numel() < N or Lminus.numel() < N:
        raise ValueError("loss buffers smaller than N")
    if workspace is None:
        workspace = new_workspace(cfg, N, B, Cn, device=dev)
    args = (C.byref(c), _theta(cfg, theta), seed, eps, N, i0,
            _dev(tokens, torch.int32, "tokens"),
            None if mask is None else _dev(mask, torch.uint8, "mask"), B, Cn,
            _dev(Lplus, torch.float32, "Lplus"), _dev(Lminus, torch.float32, "Lminus"),
            _dev(workspace, torch.uint8, "workspace"), workspace.numel())
    if products == PRODUCTS_AUTO:
        st = lib().zo_perturbed_losses(*args, _stream(stream))
    else:
        st = lib().zo_perturbed_losses_ex(*args, int(products), _stream(stream))
    _check(st)
    return Lplus, Lminus


NOALLOC_WORKSPACE_BYTES = 128 << 20  # ZO_NOALLOC_WORKSPACE_BYTES


def perturbed_losses_noalloc(cfg, theta: torch.Tensor, seed: int, eps: float, N: int,
                             tokens: torch.Tensor, mask: torch.Tensor | None, Lplus: torch.Tensor,
                             Lminus: torch.Tensor, i0: int = 0, stream=None):
    """zo_perturbed_losses_noalloc: the perturbed losses into the caller's
    Lplus / Lminus (device fp32, >= N elements) with the library's fixed
    device scratch as the workspace (nothing is allocated, here or in the
    library; token ids are not checked on the host)."""
    c = _cfg(cfg)
    if tokens.dim() != 2:
        raise ValueError("tokens must be [B][C+1]")
    B, C1 = tokens.shape
    Cn = C1 - 1
    if mask is not None and tuple(mask.shape) != (B, Cn):
        raise ValueError("mask must be [B][C]")
    if Lplus.numel() < N or Lminus.numel() < N:
        raise ValueError("loss buffers smaller than N")
    st = lib().zo_perturbed_losses_noalloc(
        C.byref(c), _theta(cfg, theta), seed, eps, N, i0, _dev(tokens, torch.int32, "tokens"),
        None if mask is None else _dev(mask, torch.uint8, "mask"), B, Cn,
        _dev(Lplus, torch.float32, "Lplus"), _dev(Lminus, torch.float32, "Lminus"), _stream(stream))
    _check(st)
    return Lplus, Lminus


def update(cfg, theta: torch.Tensor, seed: int, eps: float, lr: float, Lplus: torch.Tensor,
           Lminus: torch.Tensor, i0: int = 0, skipped: torch.Tensor | None = None, stream=None):
    """In-place update of theta (asynchronous)."""
    c = _cfg(cfg)
    N = Lplus.numel()
    if Lminus.numel() != N:
        raise ValueError("Lplus and Lminus differ in length")
    st = lib().zo_update(C.byref(c), _theta(cfg, theta), seed, eps, lr, N, i0,
                         _dev(Lplus, torch.float32, "Lplus"), _dev(Lminus, torch.float32, "Lminus"),
                         None if skipped is None else _dev(skipped, torch.int32, "skipped"),
                         _stream(stream))
    _check(st)


def probe_bits(cfg, N: int, B: int, C_: int, workspace: torch.Tensor) -> torch.Tensor | None:
    """The sign-probe cache inside a workspace of workspace_bytes() (a view of
    it as int32 words), or None when the shape has none."""
    c = _cfg(cfg)
    off = int(lib().zo_probe_bits_offset(C.byref(c), N, B, C_))
    if off == 0:
        return None
    P = param_count(cfg)
    nbytes = N * ((P + 127) // 128) * 4 * 4
    if workspace.numel() < off + nbytes:
        raise ValueError("the workspace does not hold the sign-probe cache")
    return workspace[off:off + nbytes].view(torch.int32)


def update_cached(cfg, theta: torch.Tensor, seed: int, eps: float, lr: float, Lplus: torch.Tensor,
                  Lminus: torch.Tensor, bits: torch.Tensor, i0: int = 0, skipped: torch.Tensor | None = None,
                  stream=None):
    """zo_update_cached: the update reading the probes' sign words from bits
    (probe_bits() of the workspace of the matching perturbed_losses call)."""
    c = _cfg(cfg)
    N = Lplus.numel()
    if Lminus.numel() != N:
        raise ValueError("Lplus and Lminus differ in length")
    if bits.numel() < N * ((param_count(cfg) + 127) // 128) * 4:
        raise ValueError("bits smaller than the N probes' sign words")
    st = lib().zo_update_cached(C.byref(c), _theta(cfg, theta), seed, eps, lr, N, i0,
                                _dev(Lplus, torch.float32, "Lplus"), _dev(Lminus, torch.float32, "Lminus"),
                                None if skipped is None else _dev(skipped, torch.int32, "skipped"),
                                _dev(bits, torch.int32, "bits"), _stream(stream))
    _check(st)


def fd_losses(cfg, theta: torch.Tensor, seed: int, eps: float, N: int, tokens: torch.Tensor,
              mask: torch.Tensor | None = None, i0: int = 0, L: torch.Tensor | None = None,
              L0: torch.Tensor | None = None, workspace: torch.Tensor | None = None, stream=None,
              check_tokens: bool = True, products: int = PRODUCTS_AUTO):
    """Forward differences: returns (L [N], L0 [1]) as device fp32 tensors
    (asynchronous): the losses at theta + eps z_n and at theta. products as
    for perturbed_losses (zo_fd_losses_ex when not PRODUCTS_AUTO)."""
    c = _cfg(cfg)
    if tokens.dim() != 2:
        raise ValueError("tokens must be [B][C+1]")
    if check_tokens and tokens.numel():
        lo, hi = int(tokens.min()), int(tokens.max())
        if lo < 0 or hi >= int(cfg["vocab"]):
            raise ValueError(f"token ids must lie in [0, {cfg['vocab']}), got [{lo}, {hi}]")
    B, C1 = tokens.shape
    Cn = C1 - 1
    if mask is not None and tuple(mask.shape) != (B, Cn):
        raise ValueError("mask must be [B][C]")
    dev = theta.device
    if L is None:
        L = torch.empty(N, dtype=torch.float32, device=dev)
    if L0 is None:
        L0 = torch.empty(1, dtype=torch.float32, device=dev)
    if L.numel() < N or L0.numel() < 1:
        raise ValueError("loss buffers too small")
    if workspace is None:
        workspace = new_workspace(cfg, N, B, Cn, device=dev)
    args = (C.byref(c), _theta(cfg, theta), seed, eps, N, i0,
            _dev(tokens, torch.int32, "tokens"),
            None if mask is None else _dev(mask, torch.uint8, "mask"), B, Cn,
            _dev(L, torch.float32, "L"), _dev(L0, torch.float32, "L0"),
            _dev(workspace, torch.uint8, "workspace"), workspace.numel())
    if products == PRODUCTS_AUTO:
        st = lib().zo_fd_losses(*args, _stream(stream))
    else:
        st = lib().zo_fd_losses_ex(*args, int(products), _stream(stream))
    _check(st)
    return L, L0


def fd_update(cfg, theta: torch.Tensor, seed: int, eps: float, lr: float, L: torch.Tensor,
              L0: torch.Tensor, i0: int = 0, skipped: torch.Tensor | None = None, stream=None):
    """In-place forward-difference update of theta (asynchronous)."""
    c = _cfg(cfg)
    N = L.numel()
    if L0.numel() < 1:
        raise ValueError("L0 must hold one loss")
    st = lib().zo_fd_update(C.byref(c), _theta(cfg, theta), seed, eps, lr, N, i0,
                            _dev(L, torch.float32, "L"), _dev(L0, torch.float32, "L0"),
                            None if skipped is None else _dev(skipped, torch.int32, "skipped"),
                            _stream(stream))
    _check(st)


def debug_probe(kind: int, seed: int, i: int, j0: int, n: int, device="cuda", stream=None):
    out = torch.empty(n, dtype=torch.float32, device=device)
    _check(lib().zo_debug_probe(kind, seed, i, j0, n, _dev(out, torch.float32, "out"), _stream(stream)))
    return out


def debug_gauss_pairs(words: torch.Tensor, stream=None) -> torch.Tensor:
    if words.numel() % 2:
        raise ValueError("words must hold whole pairs")
    out = torch.empty(words.numel(), dtype=torch.float32, device=words.device)
    _check(lib().zo_debug_gauss_pairs(_dev(words, torch.int32, "words") if words.dtype == torch.int32
                                      else _dev(words, torch.uint32, "words"),
                                      words.numel() // 2, _dev(out, torch.float32, "out"),
                                      _stream(stream)))
    return out


K_GATE, K_HEAD, K_EMBED, K_COMBINE, K_UPDATE, K_PROBE_CACHE, K_WEIGHTS16 = 0, 1, 2, 3, 4, 5, 6
KERNEL_CLASSES = {"gate": K_GATE, "head": K_HEAD, "embed": K_EMBED, "combine": K_COMBINE,
                  "update": K_UPDATE, "probe_cache": K_PROBE_CACHE, "weights16": K_WEIGHTS16}


def profile_enable(every: int = 1):
    """Start (and reset) event timing of every `every`-th launch of each
    kernel class (all launches are counted), or stop it with 0 / False."""
    _check(lib().zo_profile_enable(int(every)))


def profile_read() -> dict:
    """{class: (timed_ms, timed_launches, all_launches)} since the last
    profile_enable."""
    out = {}
    for name, k in KERNEL_CLASSES.items():
        ms, n, a = C.c_double(0.0), C.c_int64(0), C.c_int64(0)
        _check(lib().zo_profile_read(k, C.byref(ms), C.byref(n), C.byref(a)))
        out[name] = (ms.value, n.value, a.value)
    return out
