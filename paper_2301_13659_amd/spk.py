"""Python binding of libspk: argument marshalling only.

Each ``spk_*`` function takes torch tensors on an MI355X device, checks their
dtype, shape and contiguity, allocates outputs and workspaces with torch, and
calls the C entry point of the same name on torch's current stream.  Every
step of the computation runs in libspk's HIP kernels; there is no fallback.

``import torch`` must come before the library is loaded: torch ships the HIP
runtime that libspk then shares (same soname), so both use one runtime.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libspk.so")
NEVER = 255
MAX_T = 254

SPK_OK, SPK_E_ARG, SPK_E_SHAPE, SPK_E_UNSUPPORTED, SPK_E_WORKSPACE, SPK_E_HIP = range(6)
SPK_F32, SPK_F16 = 0, 1
SPK_CODE_RANK, SPK_CODE_LINEAR = 0, 1

# The ABI's spk_winner: {int32 c, y, x, t; float v} (20 bytes).
WINNER_DTYPE = np.dtype([("c", "<i4"), ("y", "<i4"), ("x", "<i4"), ("t", "<i4"), ("v", "<f4")])


class DogDesc(ctypes.Structure):
    _fields_ = [("ksize", ctypes.c_int32), ("sigma1", ctypes.c_double), ("sigma2", ctypes.c_double)]


class StdpConfig(ctypes.Structure):
    _fields_ = [("a_causal", ctypes.c_float), ("a_anticausal", ctypes.c_float),
                ("lower", ctypes.c_float), ("upper", ctypes.c_float), ("stabilize", ctypes.c_int32)]


class SpkError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"libspk status {status}: {message}")
        self.status = status


_P, _I, _F, _Z, _I64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t, ctypes.c_int64
_SIGNATURES = {
    "spk_version": ([], ctypes.c_char_p),
    "spk_last_error": ([], ctypes.c_char_p),
    "spk_out_extent": ([_I, _I, _I, _I], _I),
    "spk_dog_filter": ([_P, _I, _I, _I, _I, _P, _I, _I, _P, _P], _I),
    "spk_latency_code_workspace_size": ([_I, _I, _I, _I], _Z),
    "spk_latency_code": ([_P, _I, _I, _I, _I, _I, _F, _I, _P, _P, _P, _Z, _P], _I),
    "spk_dog_latency_code_workspace_size": ([_I, _I, _I, _I, _P, _I, _I], _Z),
    "spk_dog_latency_code": ([_P, _I, _I, _I, _I, _P, _I, _I, _I, _F, _P, _P, _P, _Z, _P], _I),
    "spk_conv_fire_workspace_size": ([_I] * 10 + [_F, _I], _Z),
    "spk_conv_fire": ([_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _I, _I, _I, _F, _P, _P, _P, _P,
                       _Z, _P], _I),
    "spk_conv_fire_noalloc": ([_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _I, _I, _I, _F, _P, _P, _P,
                               _P], _I),
    "spk_pool": ([_P, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P], _I),
    "spk_pool_conv_fire_workspace_size": ([_I] * 14 + [_F], _Z),
    "spk_pool_conv_fire": ([_P] + [_I] * 9 + [_P, _P, _I, _P] + [_I] * 5 + [_F, _P, _P, _P, _Z, _P],
                           _I),
    "spk_conv_packed_weights_size": ([_I] * 5, _Z),
    "spk_conv_pack_weights": ([_P, _I, _I, _I, _I, _I, _P, _Z, _P], _I),
    "spk_inhibit_winners_workspace_size": ([_I, _I, _I, _I], _Z),
    "spk_inhibit_winners": ([_P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _Z, _P],
                            _I),
    "spk_stdp_update_workspace_size": ([_I] * 6, _Z),
    "spk_stdp_update": ([_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _I, _I, _P, _P, _I, _P, _I, _P,
                         _P, _Z, _P], _I),
    "spk_rstdp_select": ([_P, _P, _I, _I, _P, _I, _P, _P], _I),
    "spk_frames_to_times": ([_P, _I, _I, _I64, _P, _P], _I),
    "spk_times_to_frames": ([_P, _I, _I, _I64, _P, _P], _I),
    "spk_cast_f16": ([_P, _P, _I64, _P], _I),
    "spk_fc_fire_workspace_size": ([_I, _I, _I, _I, _F, _I], _Z),
    "spk_fc_fire": ([_P, _I, _I, _I, _P, _I, _I, _F, _P, _P, _P, _P, _Z, _P], _I),
    "spk_fc_winners": ([_P, _P, _I, _I, _I, _I, _I, _I, _P, _P, _P], _I),
    "spk_fc_stdp_update_workspace_size": ([_I, _I, _I, _I], _Z),
    "spk_fc_stdp_update": ([_P, _P, _I, _I, _P, _I, _P, _P, _I, _P, _I, _P, _P, _Z, _P], _I),
    "spk_rate_code": ([_P, _P, _I, _I64, _I, _F, _P, _P, _Z, _P], _I),
    "spk_conv_if_rate_workspace_size": ([_I] * 11, _Z),
    "spk_conv_if_rate": ([_P, _I, _I, _I, _I, _I, _P, _I, _I, _I, _I, _I, _I, _F, _P, _P, _P, _Z, _P], _I),
    "spk_rate_pool": ([_P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P, _P], _I),
    "spk_rate_features": ([_P, _I64, _I, _P, _P], _I),
    "spk_log_filter": ([_P, _I, _I, _I, _I, _P, _I, _I, _I, _P, _P], _I),
    "spk_threshold": ([_P, _I64, _F, _F, _P], _I),
    "spk_fire": ([_P, _I, _I, _I64, _F, _P, _P, _P], _I),
    "spk_inhibit": ([_P, _P, _I, _I, _I, _I, _P, _P], _I),
    "spk_quantize": ([_P, _P, _I64, _F, _F, _F, _P], _I),
    "spk_gather": ([_P, _I64, _I, _P, _P], _I),
    "spk_times_to_spikes_workspace_size": ([_I] * 5, _Z),
    "spk_times_to_spikes": ([_P, _I, _I, _I, _I, _I, _I, _P, _P, _P, _Z, _P], _I),
    "spk_spikes_to_times": ([_P, _P, _I, _I, _I, _I, _I, _I, _P, _P], _I),
    "spk_conv_fire_sparse_workspace_size": ([_I] * 10 + [_I], _Z),
    "spk_conv_fire_sparse": ([_P, _P, _I, _I, _I, _I, _I, _I, _P, _I, _I, _I, _I, _I, _I, _F, _P,
                              _P, _P, _Z, _P], _I),
}

_lib = None


def load(path: str = LIB_PATH):
    """Load libspk (building it first only if no built library exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        from . import build as _build
        _build.build()
    L = ctypes.CDLL(path)
    for name, (args, res) in _SIGNATURES.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def symbols() -> list:
    return list(_SIGNATURES)


def _check(status: int):
    if status != SPK_OK:
        raise SpkError(status, load().spk_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor, dtype, name: str, ndim: int | None = None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name}: expected a tensor on the GPU")
    if t.dtype != dtype:
        raise ValueError(f"{name}: expected {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous tensor")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name}: expected {ndim} dimensions, got {t.dim()}")
    return t


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


_sentinel = False


def set_output_sentinel(on: bool) -> None:
    """Test aid: while on, every output and workspace these wrappers allocate
    is filled before the call (floats with NaN, every other type with 0xAB
    bytes), so an element a kernel fails to write cannot match a reference."""
    global _sentinel
    _sentinel = bool(on)


def _empty(shape, dtype, device) -> torch.Tensor:
    t = torch.empty(shape, dtype=dtype, device=device)
    if _sentinel:
        if t.is_floating_point():
            t.fill_(float("nan"))
        elif t.numel():
            t.view(torch.uint8).fill_(0xAB)
    return t


def _workspace(nbytes: int, device) -> torch.Tensor | None:
    return _empty(nbytes, dtype=torch.uint8, device=device) if nbytes else None


def out_extent(n: int, k: int, stride: int, pad: int) -> int:
    return load().spk_out_extent(n, k, stride, pad)


def version() -> str:
    return load().spk_version().decode()


# --------------------------------------------------------------------- calls

def spk_dog_filter(img, filters, pad: int = -1, out=None):
    _dev(img, torch.uint8, "img", 4)
    B, C, H, W = img.shape
    descs = (DogDesc * len(filters))(*[DogDesc(int(k), float(s1), float(s2)) for k, s1, s2 in filters])
    K0 = int(filters[0][0])
    Ho, Wo = (H, W) if pad < 0 else (H + 2 * pad - K0 + 1, W + 2 * pad - K0 + 1)
    if out is None:
        out = _empty((B, C * len(filters), Ho, Wo), dtype=torch.float32, device=img.device)
    _dev(out, torch.float32, "out", 4)
    _check(load().spk_dog_filter(_ptr(img), B, C, H, W, descs, len(filters), pad, _ptr(out),
                                 _stream(img.device)))
    return out


def spk_latency_code(x, T: int, min_value: float = 0.01, mode: int = SPK_CODE_RANK,
                     times=None, frames=False):
    _dev(x, torch.float32, "x", 4)
    B, C, H, W = x.shape
    if times is None:
        times = _empty((B, C, H, W), dtype=torch.uint8, device=x.device)
    _dev(times, torch.uint8, "times", 4)
    fr = None
    if frames is True:
        fr = _empty((B, T, C, H, W), dtype=torch.uint8, device=x.device)
    elif isinstance(frames, torch.Tensor):
        fr = _dev(frames, torch.uint8, "frames", 5)
    L = load()
    nbytes = L.spk_latency_code_workspace_size(B, C, H, W) if mode == SPK_CODE_RANK else 0
    ws = _workspace(nbytes, x.device)
    _check(L.spk_latency_code(_ptr(x), B, C, H, W, T, float(min_value), mode, _ptr(times),
                              _ptr(fr), _ptr(ws), nbytes, _stream(x.device)))
    return (times, fr) if fr is not None else times


def spk_dog_latency_code(img, filters, T: int, min_value: float = 0.01, pad: int = -1,
                         times=None, dog_out=None):
    """DoG filtering then rank-order coding in one call; dog_out: optional float
    tensor that also receives the filter outputs."""
    _dev(img, torch.uint8, "img", 4)
    B, C, H, W = img.shape
    descs = (DogDesc * len(filters))(*[DogDesc(int(k), float(s1), float(s2)) for k, s1, s2 in filters])
    K0 = int(filters[0][0])
    Ho, Wo = (H, W) if pad < 0 else (H + 2 * pad - K0 + 1, W + 2 * pad - K0 + 1)
    shape = (B, C * len(filters), Ho, Wo)
    if times is None:
        times = _empty(shape, dtype=torch.uint8, device=img.device)
    _dev(times, torch.uint8, "times", 4)
    if dog_out is not None:
        _dev(dog_out, torch.float32, "dog_out", 4)
    L = load()
    nbytes = L.spk_dog_latency_code_workspace_size(B, C, H, W, descs, len(filters), pad)
    ws = _workspace(nbytes, img.device)
    _check(L.spk_dog_latency_code(_ptr(img), B, C, H, W, descs, len(filters), pad, T, float(min_value),
                                  _ptr(times), _ptr(dog_out), _ptr(ws), nbytes, _stream(img.device)))
    return times


def spk_conv_fire(in_times, w, T: int, stride: int = 1, pad: int = 0, theta: float = math.inf,
                  potentials=False, out_times=None, out_vkey=None):
    """w: float32 master weights or float16 operand, Co x Ci x Kh x Kw."""
    _dev(in_times, torch.uint8, "in_times", 4)
    if w.dtype not in (torch.float32, torch.float16):
        raise ValueError("w: expected float32 or float16")
    _dev(w, w.dtype, "w", 4)
    B, Ci, Hi, Wi = in_times.shape
    Co, Ci2, Kh, Kw = w.shape
    if Ci != Ci2:
        raise ValueError(f"w has {Ci2} input channels, input has {Ci}")
    L = load()
    Ho, Wo = L.spk_out_extent(Hi, Kh, stride, pad), L.spk_out_extent(Wi, Kw, stride, pad)
    dev = in_times.device
    if out_times is None:
        out_times = _empty((B, Co, max(Ho, 1), max(Wo, 1)), dtype=torch.uint8, device=dev)
    if out_vkey is None:
        out_vkey = _empty((B, Co, max(Ho, 1), max(Wo, 1)), dtype=torch.float32, device=dev)
    _dev(out_times, torch.uint8, "out_times", 4)
    _dev(out_vkey, torch.float32, "out_vkey", 4)
    V = None
    if potentials is True:
        V = _empty((B, T, Co, Ho, Wo), dtype=torch.float32, device=dev)
    elif isinstance(potentials, torch.Tensor):
        V = _dev(potentials, torch.float32, "potentials", 5)
    nbytes = L.spk_conv_fire_workspace_size(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, float(theta),
                                            int(V is not None))
    ws = _workspace(nbytes, dev)
    dt = SPK_F16 if w.dtype == torch.float16 else SPK_F32
    _check(L.spk_conv_fire(_ptr(in_times), B, T, Ci, Hi, Wi, _ptr(w), dt, Co, Kh, Kw, stride, pad,
                           float(theta), _ptr(out_times), _ptr(out_vkey), _ptr(V), _ptr(ws), nbytes,
                           _stream(dev)))
    return (out_times, out_vkey, V) if V is not None else (out_times, out_vkey)


def spk_conv_fire_noalloc(in_times, w, T: int, stride: int = 1, pad: int = 0,
                          theta: float = math.inf, out_times=None, out_vkey=None):
    """spk_conv_fire with the library's static scratch instead of a workspace
    (for callers that cannot allocate): pass preallocated outputs to keep the
    call free of allocations."""
    _dev(in_times, torch.uint8, "in_times", 4)
    if w.dtype not in (torch.float32, torch.float16):
        raise ValueError("w: expected float32 or float16")
    _dev(w, w.dtype, "w", 4)
    B, Ci, Hi, Wi = in_times.shape
    Co, Ci2, Kh, Kw = w.shape
    if Ci != Ci2:
        raise ValueError(f"w has {Ci2} input channels, input has {Ci}")
    L = load()
    Ho, Wo = L.spk_out_extent(Hi, Kh, stride, pad), L.spk_out_extent(Wi, Kw, stride, pad)
    dev = in_times.device
    if out_times is None:
        out_times = _empty((B, Co, max(Ho, 1), max(Wo, 1)), dtype=torch.uint8, device=dev)
    if out_vkey is None:
        out_vkey = _empty((B, Co, max(Ho, 1), max(Wo, 1)), dtype=torch.float32, device=dev)
    _dev(out_times, torch.uint8, "out_times", 4)
    _dev(out_vkey, torch.float32, "out_vkey", 4)
    dt = SPK_F16 if w.dtype == torch.float16 else SPK_F32
    _check(L.spk_conv_fire_noalloc(_ptr(in_times), B, T, Ci, Hi, Wi, _ptr(w), dt, Co, Kh, Kw, stride,
                                   pad, float(theta), _ptr(out_times), _ptr(out_vkey), None,
                                   _stream(dev)))
    return out_times, out_vkey


def spk_pool_conv_fire(in_times, pool, w, T: int, stride: int = 1, pad: int = 0,
                       theta: float = math.inf, packed_w=None, keep_pooled: bool = True,
                       out_times=None, out_vkey=None):
    """Max-pooling then spk_conv_fire in one call.  pool: (k, stride, pad) of
    a square window (k may be a (kh, kw) pair).  packed_w: optional uint8
    tensor from spk_conv_pack_weights(w).  Returns (pooled, times, vkey), or
    (times, vkey) with keep_pooled=False."""
    _dev(in_times, torch.uint8, "in_times", 4)
    if w.dtype not in (torch.float32, torch.float16):
        raise ValueError("w: expected float32 or float16")
    _dev(w, w.dtype, "w", 4)
    k, pstride, ppad = pool
    pkh, pkw = (k, k) if isinstance(k, int) else k
    B, Ci, H0, W0 = in_times.shape
    Co, Ci2, Kh, Kw = w.shape
    if Ci != Ci2:
        raise ValueError(f"w has {Ci2} input channels, input has {Ci}")
    L = load()
    Hi, Wi = L.spk_out_extent(H0, pkh, pstride, ppad), L.spk_out_extent(W0, pkw, pstride, ppad)
    Ho = L.spk_out_extent(Hi, Kh, stride, pad) if Hi > 0 else -1
    Wo = L.spk_out_extent(Wi, Kw, stride, pad) if Wi > 0 else -1
    dev = in_times.device
    pooled = _empty((B, Ci, max(Hi, 1), max(Wi, 1)), dtype=torch.uint8, device=dev) if keep_pooled else None
    if out_times is None:
        out_times = _empty((B, Co, max(Ho, 1), max(Wo, 1)), dtype=torch.uint8, device=dev)
    if out_vkey is None:
        out_vkey = _empty((B, Co, max(Ho, 1), max(Wo, 1)), dtype=torch.float32, device=dev)
    _dev(out_times, torch.uint8, "out_times", 4)
    _dev(out_vkey, torch.float32, "out_vkey", 4)
    if packed_w is not None:
        _dev(packed_w, torch.uint8, "packed_w", 1)
    nbytes = L.spk_pool_conv_fire_workspace_size(B, T, Ci, H0, W0, pkh, pkw, pstride, ppad, Co, Kh, Kw,
                                                 stride, pad, float(theta))
    ws = _workspace(nbytes, dev)
    dt = SPK_F16 if w.dtype == torch.float16 else SPK_F32
    _check(L.spk_pool_conv_fire(_ptr(in_times), B, T, Ci, H0, W0, pkh, pkw, pstride, ppad,
                                _ptr(pooled), _ptr(w), dt, _ptr(packed_w), Co, Kh, Kw, stride, pad,
                                float(theta), _ptr(out_times), _ptr(out_vkey), _ptr(ws), nbytes,
                                _stream(dev)))
    return (pooled, out_times, out_vkey) if keep_pooled else (out_times, out_vkey)


def spk_conv_pack_weights(w, out=None):
    """The weights as the readout kernel's B fragments (a flat uint8 tensor)."""
    if w.dtype not in (torch.float32, torch.float16):
        raise ValueError("w: expected float32 or float16")
    _dev(w, w.dtype, "w", 4)
    Co, Ci, Kh, Kw = w.shape
    L = load()
    dt = SPK_F16 if w.dtype == torch.float16 else SPK_F32
    n = L.spk_conv_packed_weights_size(Co, Ci, Kh, Kw, dt)
    if out is None:
        out = _empty((max(n, 1),), dtype=torch.uint8, device=w.device)
    _dev(out, torch.uint8, "out", 1)
    _check(L.spk_conv_pack_weights(_ptr(w), dt, Co, Ci, Kh, Kw, _ptr(out), out.numel(),
                                   _stream(w.device)))
    return out


def spk_pool(in_times, k, stride: int | None = None, pad: int = 0, out=None):
    _dev(in_times, torch.uint8, "in_times", 4)
    kh, kw = (k, k) if isinstance(k, int) else k
    stride = kh if stride is None else stride
    B, C, Hi, Wi = in_times.shape
    L = load()
    Ho, Wo = L.spk_out_extent(Hi, kh, stride, pad), L.spk_out_extent(Wi, kw, stride, pad)
    if out is None:
        out = _empty((B, C, max(Ho, 1), max(Wo, 1)), dtype=torch.uint8, device=in_times.device)
    _dev(out, torch.uint8, "out", 4)
    _check(L.spk_pool(_ptr(in_times), B, C, Hi, Wi, kh, kw, stride, pad, _ptr(out),
                      _stream(in_times.device)))
    return out


def spk_inhibit_winners(times, vkey, T: int, k: int, radius: int, pointwise: bool = True,
                        readout: bool = False, inhibited=None, winners=None, n_winners=None):
    """Returns (winners int32 B x k x 5 [c, y, x, t, v bits], n_winners int32 B[, inhibited])."""
    _dev(times, torch.uint8, "times", 4)
    _dev(vkey, torch.float32, "vkey", 4)
    B, C, H, W = times.shape
    dev = times.device
    if winners is None:
        winners = _empty((B, k, 5), dtype=torch.int32, device=dev)
    if n_winners is None:
        n_winners = _empty((B,), dtype=torch.int32, device=dev)
    _dev(winners, torch.int32, "winners", 3)
    _dev(n_winners, torch.int32, "n_winners", 1)
    inh = None
    if inhibited is True:
        inh = _empty(times.shape, dtype=times.dtype, device=times.device)
    elif isinstance(inhibited, torch.Tensor):
        inh = _dev(inhibited, torch.uint8, "inhibited", 4)
    L = load()
    nbytes = L.spk_inhibit_winners_workspace_size(B, C, H, W) if pointwise else 0
    ws = _workspace(nbytes, dev)
    _check(L.spk_inhibit_winners(_ptr(times), _ptr(vkey), B, C, H, W, T, int(bool(pointwise)), k,
                                 radius, int(bool(readout)), _ptr(inh), _ptr(winners),
                                 _ptr(n_winners), _ptr(ws), nbytes, _stream(dev)))
    return (winners, n_winners, inh) if inh is not None else (winners, n_winners)


def spk_stdp_update(w, in_times, winners, n_winners, cfgs, stride: int = 1, pad: int = 0,
                    winner_cfg=None, w_f16=None):
    """In-place update of float32 master weights w (and of the half copy w_f16 if given).

    cfgs: iterable of (a_causal, a_anticausal, lower, upper, stabilize)."""
    _dev(w, torch.float32, "w", 4)
    _dev(in_times, torch.uint8, "in_times", 4)
    _dev(winners, torch.int32, "winners", 3)
    _dev(n_winners, torch.int32, "n_winners", 1)
    if w_f16 is not None:
        _dev(w_f16, torch.float16, "w_f16", 4)
    if winner_cfg is not None:
        _dev(winner_cfg, torch.int32, "winner_cfg")
    Co, Ci, Kh, Kw = w.shape
    B, Ci2, Hi, Wi = in_times.shape
    if Ci != Ci2:
        raise ValueError(f"w has {Ci} input channels, input has {Ci2}")
    k = winners.shape[1]
    cl = [tuple(c) for c in cfgs]
    arr = (StdpConfig * len(cl))(*[StdpConfig(float(a), float(b), float(lo), float(up), int(st))
                                   for a, b, lo, up, st in cl])
    L = load()
    nbytes = L.spk_stdp_update_workspace_size(Co, Ci, Kh, Kw, B, k)
    ws = _workspace(nbytes, w.device)
    _check(L.spk_stdp_update(_ptr(w), _ptr(w_f16), Co, Ci, Kh, Kw, stride, pad, _ptr(in_times), B,
                             Hi, Wi, _ptr(winners), _ptr(n_winners), k, arr, len(cl),
                             _ptr(winner_cfg), _ptr(ws), nbytes, _stream(w.device)))
    return w


def spk_rstdp_select(winners, n_winners, labels, group: int, out=None):
    _dev(winners, torch.int32, "winners", 3)
    _dev(n_winners, torch.int32, "n_winners", 1)
    _dev(labels, torch.int32, "labels", 1)
    B, k = winners.shape[:2]
    if out is None:
        out = _empty((B, k), dtype=torch.int32, device=winners.device)
    _check(load().spk_rstdp_select(_ptr(winners), _ptr(n_winners), B, k, _ptr(labels), group,
                                   _ptr(out), _stream(winners.device)))
    return out


def spk_frames_to_times(frames, out=None):
    _dev(frames, torch.uint8, "frames")
    B, T = frames.shape[:2]
    n = frames[0, 0].numel()
    if out is None:
        out = _empty((B,) + tuple(frames.shape[2:]), dtype=torch.uint8, device=frames.device)
    _check(load().spk_frames_to_times(_ptr(frames), B, T, n, _ptr(out), _stream(frames.device)))
    return out


def spk_times_to_frames(times, T: int, out=None):
    _dev(times, torch.uint8, "times")
    B = times.shape[0]
    n = times[0].numel()
    if out is None:
        out = _empty((B, T) + tuple(times.shape[1:]), dtype=torch.uint8, device=times.device)
    _check(load().spk_times_to_frames(_ptr(times), B, T, n, _ptr(out), _stream(times.device)))
    return out


def spk_cast_f16(x, out=None):
    _dev(x, torch.float32, "x")
    if out is None:
        out = _empty(x.shape, dtype=torch.float16, device=x.device)
    _check(load().spk_cast_f16(_ptr(x), _ptr(out), x.numel(), _stream(x.device)))
    return out


def spk_fc_fire(in_times, w, T: int, theta: float = math.inf, potentials=False):
    """Fully connected IF layer: in_times uint8 B x I, w float32 / float16 O x I."""
    _dev(in_times, torch.uint8, "in_times", 2)
    if w.dtype not in (torch.float32, torch.float16):
        raise ValueError("w: expected float32 or float16")
    _dev(w, w.dtype, "w", 2)
    B, I = in_times.shape
    O, I2 = w.shape
    if I != I2:
        raise ValueError(f"w has {I2} inputs, input has {I}")
    dev = in_times.device
    out_times = _empty((B, O), dtype=torch.uint8, device=dev)
    out_vkey = _empty((B, O), dtype=torch.float32, device=dev)
    V = _empty((B, T, O), dtype=torch.float32, device=dev) if potentials else None
    L = load()
    nbytes = L.spk_fc_fire_workspace_size(B, T, I, O, float(theta), int(V is not None))
    ws = _workspace(nbytes, dev)
    dt = SPK_F16 if w.dtype == torch.float16 else SPK_F32
    _check(L.spk_fc_fire(_ptr(in_times), B, T, I, _ptr(w), dt, O, float(theta), _ptr(out_times),
                         _ptr(out_vkey), _ptr(V), _ptr(ws), nbytes, _stream(dev)))
    return (out_times, out_vkey, V) if V is not None else (out_times, out_vkey)


def spk_fc_winners(times, vkey, T: int, k: int, radius: int, readout: bool = False):
    """fcwta: returns (winners int32 B x k x 5, n_winners int32 B)."""
    _dev(times, torch.uint8, "times", 2)
    _dev(vkey, torch.float32, "vkey", 2)
    B, O = times.shape
    dev = times.device
    winners = _empty((B, k, 5), dtype=torch.int32, device=dev)
    n_winners = _empty((B,), dtype=torch.int32, device=dev)
    _check(load().spk_fc_winners(_ptr(times), _ptr(vkey), B, O, T, k, radius, int(bool(readout)),
                                 _ptr(winners), _ptr(n_winners), _stream(dev)))
    return winners, n_winners


def spk_fc_stdp_update(w, in_times, winners, n_winners, cfgs, winner_cfg=None, w_f16=None):
    """In-place STDP of float32 FC weights w (O x I) from in_times (B x I)."""
    _dev(w, torch.float32, "w", 2)
    _dev(in_times, torch.uint8, "in_times", 2)
    _dev(winners, torch.int32, "winners", 3)
    _dev(n_winners, torch.int32, "n_winners", 1)
    if w_f16 is not None:
        _dev(w_f16, torch.float16, "w_f16", 2)
    if winner_cfg is not None:
        _dev(winner_cfg, torch.int32, "winner_cfg")
    O, I = w.shape
    B, I2 = in_times.shape
    if I != I2:
        raise ValueError(f"w has {I} inputs, input has {I2}")
    k = winners.shape[1]
    cl = [tuple(c) for c in cfgs]
    arr = (StdpConfig * len(cl))(*[StdpConfig(float(a), float(b), float(lo), float(up), int(st))
                                   for a, b, lo, up, st in cl])
    L = load()
    nbytes = L.spk_fc_stdp_update_workspace_size(O, I, B, k)
    ws = _workspace(nbytes, w.device)
    _check(L.spk_fc_stdp_update(_ptr(w), _ptr(w_f16), O, I, _ptr(in_times), B, _ptr(winners),
                                _ptr(n_winners), k, arr, len(cl), _ptr(winner_cfg), _ptr(ws), nbytes,
                                _stream(w.device)))
    return w


def winners_numpy(winners: torch.Tensor) -> np.ndarray:
    """Device winners (B x k x 5 int32) -> numpy structured array of WINNER_DTYPE."""
    a = winners.detach().cpu().contiguous().numpy()
    return a.view(np.uint8).reshape(a.shape[0], a.shape[1], 20).view(WINNER_DTYPE)[..., 0]


# ------------------------------------------------------- sparse interface

def spk_times_to_spikes(times, T: int, cap: int | None = None):
    """Spike list of a time map (B x C x H x W): (spikes uint32 as int32 B x cap,
    offsets int32 B x (T + 1)).  cap defaults to C*H*W (never truncates)."""
    _dev(times, torch.uint8, "times", 4)
    B, C, H, W = times.shape
    cap = C * H * W if cap is None else int(cap)
    dev = times.device
    spikes = _empty((B, cap), dtype=torch.int32, device=dev)
    offsets = _empty((B, T + 1), dtype=torch.int32, device=dev)
    L = load()
    nbytes = L.spk_times_to_spikes_workspace_size(B, C, H, W, T)
    ws = _workspace(max(nbytes, 1), dev)
    _check(L.spk_times_to_spikes(_ptr(times), B, C, H, W, T, cap, _ptr(spikes), _ptr(offsets),
                                 _ptr(ws), nbytes, _stream(dev)))
    return spikes, offsets


def spk_spikes_to_times(spikes, offsets, shape, T: int):
    """Time map B x shape (C, H, W) of a spike list."""
    _dev(spikes, torch.int32, "spikes", 2)
    _dev(offsets, torch.int32, "offsets", 2)
    B, cap = spikes.shape
    C, H, W = shape
    times = _empty((B, C, H, W), dtype=torch.uint8, device=spikes.device)
    _check(load().spk_spikes_to_times(_ptr(spikes), _ptr(offsets), cap, B, C, H, W, T, _ptr(times),
                                      _stream(spikes.device)))
    return times


def spk_conv_fire_sparse(spikes, offsets, in_shape, w, T: int, stride: int = 1, pad: int = 0,
                         theta: float = math.inf):
    """Conv + fire driven by a spike list over in_shape = (Ci, Hi, Wi):
    (out_times uint8, out_vkey float32), B x Co x Ho x Wo."""
    _dev(spikes, torch.int32, "spikes", 2)
    _dev(offsets, torch.int32, "offsets", 2)
    if w.dtype not in (torch.float32, torch.float16):
        raise ValueError("w: expected float32 or float16")
    _dev(w, w.dtype, "w", 4)
    B, cap = spikes.shape
    Ci, Hi, Wi = in_shape
    Co, Ci2, Kh, Kw = w.shape
    if Ci != Ci2:
        raise ValueError(f"w has {Ci2} input channels, input has {Ci}")
    Ho, Wo = out_extent(Hi, Kh, stride, pad), out_extent(Wi, Kw, stride, pad)
    dev = spikes.device
    out_times = _empty((B, Co, Ho, Wo), dtype=torch.uint8, device=dev)
    out_vkey = _empty((B, Co, Ho, Wo), dtype=torch.float32, device=dev)
    dt = SPK_F16 if w.dtype == torch.float16 else SPK_F32
    L = load()
    nbytes = L.spk_conv_fire_sparse_workspace_size(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, dt)
    ws = _workspace(max(nbytes, 1), dev)
    _check(L.spk_conv_fire_sparse(_ptr(spikes), _ptr(offsets), cap, B, T, Ci, Hi, Wi, _ptr(w), dt,
                                  Co, Kh, Kw, stride, pad, float(theta), _ptr(out_times),
                                  _ptr(out_vkey), _ptr(ws), nbytes, _stream(dev)))
    return out_times, out_vkey


# ------------------------------------------------ steps around the hot path

def spk_log_filter(img, stds, ksize: int, pad: int = -1):
    """LoG bank: img uint8 B x C x H x W -> float32 B x (C*2n) x Ho x Wo."""
    _dev(img, torch.uint8, "img", 4)
    B, C, H, W = img.shape
    n = len(stds)
    Ho = H if pad < 0 else H + 2 * pad - ksize + 1
    Wo = W if pad < 0 else W + 2 * pad - ksize + 1
    out = _empty((B, C * 2 * n, Ho, Wo), dtype=torch.float32, device=img.device)
    arr = (ctypes.c_float * n)(*[float(s) for s in stds])
    _check(load().spk_log_filter(_ptr(img), B, C, H, W, arr, n, ksize, pad, _ptr(out),
                                 _stream(img.device)))
    return out


def spk_threshold(x, threshold: float, value: float = 0.0):
    """In place: x = x if x > threshold else value (float32)."""
    _dev(x, torch.float32, "x")
    _check(load().spk_threshold(_ptr(x), x.numel(), float(threshold), float(value), _stream(x.device)))
    return x


def spk_quantize(w, lower: float, mid: float, upper: float, w_f16=None):
    """In place on float32 weights (and their half copy)."""
    _dev(w, torch.float32, "w")
    if w_f16 is not None:
        _dev(w_f16, torch.float16, "w_f16")
        if w_f16.numel() != w.numel():
            raise ValueError("w_f16 must match w")
    _check(load().spk_quantize(_ptr(w), _ptr(w_f16), w.numel(), float(lower), float(mid), float(upper),
                               _stream(w.device)))
    return w


def spk_gather(times, T: int):
    """Feature values of a time map: float32, T - t where fired, else 0."""
    _dev(times, torch.uint8, "times")
    out = _empty(times.shape, dtype=torch.float32, device=times.device)
    _check(load().spk_gather(_ptr(times), times.numel(), T, _ptr(out), _stream(times.device)))
    return out


# ------------------------------------------------------------ rate coding

def spk_rate_code(x, u, T: int, min_value: float = 0.01):
    """x float32 B x ... ; u float32 B x T x ... uniform draws -> frames uint8 B x T x ..."""
    _dev(x, torch.float32, "x")
    _dev(u, torch.float32, "u")
    B = x.shape[0]
    n = x[0].numel()
    if tuple(u.shape) != (B, T) + tuple(x.shape[1:]):
        raise ValueError("u must be B x T x (the shape of one sample of x)")
    frames = _empty(u.shape, dtype=torch.uint8, device=x.device)
    ws = _workspace(4 * B, x.device)
    _check(load().spk_rate_code(_ptr(x), _ptr(u), B, n, T, float(min_value), _ptr(frames), _ptr(ws),
                                4 * B, _stream(x.device)))
    return frames


def spk_conv_if_rate(frames, w, stride: int = 1, pad: int = 0, theta: float = 1.0):
    """IF with reset over frames uint8 B x T x Ci x Hi x Wi -> (frames, counts int32)."""
    _dev(frames, torch.uint8, "frames", 5)
    if w.dtype not in (torch.float32, torch.float16):
        raise ValueError("w: expected float32 or float16")
    _dev(w, w.dtype, "w", 4)
    B, T, Ci, Hi, Wi = frames.shape
    Co, Ci2, Kh, Kw = w.shape
    if Ci != Ci2:
        raise ValueError(f"w has {Ci2} input channels, frames have {Ci}")
    Ho, Wo = out_extent(Hi, Kh, stride, pad), out_extent(Wi, Kw, stride, pad)
    dev = frames.device
    out = _empty((B, T, Co, Ho, Wo), dtype=torch.uint8, device=dev)
    counts = _empty((B, Co, Ho, Wo), dtype=torch.int32, device=dev)
    dt = SPK_F16 if w.dtype == torch.float16 else SPK_F32
    L = load()
    nbytes = L.spk_conv_if_rate_workspace_size(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, dt)
    ws = _workspace(max(nbytes, 1), dev)
    _check(L.spk_conv_if_rate(_ptr(frames), B, T, Ci, Hi, Wi, _ptr(w), dt, Co, Kh, Kw, stride, pad,
                              float(theta), _ptr(out), _ptr(counts), _ptr(ws), nbytes, _stream(dev)))
    return out, counts


def spk_rate_pool(frames, counts, k, stride=None, pad: int = 0):
    _dev(frames, torch.uint8, "frames", 5)
    _dev(counts, torch.int32, "counts", 4)
    B, T, C, Hi, Wi = frames.shape
    kh, kw = (k, k) if isinstance(k, int) else k
    stride = kh if stride is None else stride
    Ho, Wo = out_extent(Hi, kh, stride, pad), out_extent(Wi, kw, stride, pad)
    out = _empty((B, T, C, Ho, Wo), dtype=torch.uint8, device=frames.device)
    oc = _empty((B, C, Ho, Wo), dtype=torch.int32, device=frames.device)
    _check(load().spk_rate_pool(_ptr(frames), _ptr(counts), B, T, C, Hi, Wi, kh, kw, stride, pad,
                                _ptr(out), _ptr(oc), _stream(frames.device)))
    return out, oc


def spk_rate_features(counts, T: int):
    _dev(counts, torch.int32, "counts")
    out = _empty(counts.shape, dtype=torch.float32, device=counts.device)
    _check(load().spk_rate_features(_ptr(counts), counts.numel(), T, _ptr(out), _stream(counts.device)))
    return out


def spk_fire(potentials, theta: float):
    """Fire over dense potentials B x T x ... -> (times uint8 B x ..., vkey float32 B x ...)."""
    _dev(potentials, torch.float32, "potentials")
    B, T = potentials.shape[:2]
    n = potentials[0, 0].numel()
    shape = (B,) + tuple(potentials.shape[2:])
    out_t = _empty(shape, dtype=torch.uint8, device=potentials.device)
    out_v = _empty(shape, dtype=torch.float32, device=potentials.device)
    _check(load().spk_fire(_ptr(potentials), B, T, n, float(theta), _ptr(out_t), _ptr(out_v),
                           _stream(potentials.device)))
    return out_t, out_v


def spk_inhibit(times, vkey, out=None):
    """Pointwise inhibition: a new (or the given, possibly `times` itself) uint8 map."""
    _dev(times, torch.uint8, "times", 4)
    _dev(vkey, torch.float32, "vkey", 4)
    B, C, H, W = times.shape
    if out is None:
        out = _empty(times.shape, dtype=times.dtype, device=times.device)
    _dev(out, torch.uint8, "out", 4)
    _check(load().spk_inhibit(_ptr(times), _ptr(vkey), B, C, H, W, _ptr(out), _stream(times.device)))
    return out
