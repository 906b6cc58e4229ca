"""CPU oracle for the spiking-conv pipeline -- TEST INFRASTRUCTURE.

ctypes wrappers over spk_oracle.c (plain C, fp64 where the paper leaves the
precision open).  Only the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package; the GPU library
never does, and the two share no code.  All arrays are numpy, C-contiguous.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

NEVER = 255
_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spk_oracle.c")
_LIB = os.path.join(_HERE, "liboracle_spk.so")

WINNER_DTYPE = np.dtype([("c", "<i4"), ("y", "<i4"), ("x", "<i4"), ("t", "<i4"), ("v", "<f4")])
STDP_DTYPE = np.dtype([("a_causal", "<f4"), ("a_anticausal", "<f4"), ("lower", "<f4"),
                       ("upper", "<f4"), ("stabilize", "<i4")])


def build() -> str:
    """Compile spk_oracle.c into liboracle_spk.so (plain gcc, no contraction)."""
    tmp = _LIB + ".tmp"
    subprocess.check_call(["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fPIC", "-shared",
                           "-Wall", "-o", tmp, _SRC, "-lm"])
    os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i, d, f, i64 = ctypes.c_int, ctypes.c_double, ctypes.c_float, ctypes.c_int64
        L.or_dog_kernel.argtypes = [i, d, d, P]
        L.or_dog_filter.argtypes = [P, i, i, i, i, P, P, P, i, i, P]
        L.or_latency_code.argtypes = [P, i, i64, i, f, i, P]
        L.or_times_to_frames.argtypes = [P, i, i, i64, P]
        L.or_frames_to_times.argtypes = [P, i, i, i64, P]
        L.or_conv_neuron.argtypes = [P, i, i, i, i, P, i, i, i, i, i, i, i, i, P]
        L.or_fire_neuron.argtypes = [P, i, d, P, P]
        L.or_conv_fire.argtypes = [P, i, i, i, i, i, P, i, i, i, i, i, d, P, P, P]
        L.or_pool.argtypes = [P, i, i, i, i, i, i, i, i, P]
        L.or_inhibit.argtypes = [P, P, i, i, i, i]
        L.or_kwta.argtypes = [P, P, i, i, i, i, i, i, i, i, P, P]
        L.or_stdp_update.argtypes = [P, i, i, i, i, i, i, P, i, i, i, P, P, i, P, i, P]
        L.or_stdp_update.restype = i
        L.or_rstdp_select.argtypes = [P, P, i, i, P, i, P]
        L.or_fc_wta.argtypes = [P, P, i, i, i, i, i, i, P, P]
        L.or_times_to_spikes.argtypes = [P, i, i64, i, i, P, P]
        L.or_threshold.argtypes = [P, i64, f, f]
        L.or_fire.argtypes = [P, i, i, i64, d, P, P]
        L.or_rate_code.argtypes = [P, P, i, i64, i, f, P]
        L.or_conv_if_rate.argtypes = [P, i, i, i, i, i, P, i, i, i, i, i, d, P, P]
        L.or_rate_pool.argtypes = [P, P, i, i, i, i, i, i, i, i, i, P, P]
        L.or_quantize.argtypes = [P, i64, f, f, f]
        L.or_gather.argtypes = [P, i64, i, P]
        L.or_spikes_to_times.argtypes = [P, P, i, i64, i, i, P]
        L.or_conv_fire_spikes.argtypes = [P, P, i, i, i, i, i, i, P, i, i, i, i, i, d, P, P]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    assert a.flags.c_contiguous
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ----------------------------------------------------------------------- DoG

def dog_kernel(ksize: int, sigma1: float, sigma2: float) -> np.ndarray:
    k = np.empty((ksize, ksize), np.float32)
    lib().or_dog_kernel(ksize, sigma1, sigma2, _p(k))
    return k


def dog_filter(img: np.ndarray, filters, pad: int = -1) -> np.ndarray:
    """img uint8 B x C x H x W; filters = [(K, sigma1, sigma2), ...]."""
    img = _c(img, np.uint8)
    B, C, H, W = img.shape
    ks = np.array([f[0] for f in filters], np.int32)
    s1 = np.array([f[1] for f in filters], np.float64)
    s2 = np.array([f[2] for f in filters], np.float64)
    F = len(filters)
    Ho = H if pad < 0 else H + 2 * pad - int(ks[0]) + 1
    Wo = W if pad < 0 else W + 2 * pad - int(ks[0]) + 1
    out = np.empty((B, C * F, Ho, Wo), np.float32)
    lib().or_dog_filter(_p(img), B, C, H, W, _p(ks), _p(s1), _p(s2), F, pad, _p(out))
    return out


# -------------------------------------------------------------- latency code

def latency_code(x: np.ndarray, T: int, min_value: float = 0.01, mode: int = 0) -> np.ndarray:
    x = _c(x, np.float32)
    B = x.shape[0]
    n = int(np.prod(x.shape[1:]))
    times = np.empty(x.shape, np.uint8)
    lib().or_latency_code(_p(x), B, n, T, min_value, mode, _p(times))
    return times


def times_to_frames(times: np.ndarray, T: int) -> np.ndarray:
    times = _c(times, np.uint8)
    B = times.shape[0]
    n = int(np.prod(times.shape[1:]))
    frames = np.empty((B, T) + times.shape[1:], np.uint8)
    lib().or_times_to_frames(_p(times), B, T, n, _p(frames))
    return frames


def frames_to_times(frames: np.ndarray) -> np.ndarray:
    frames = _c(frames, np.uint8)
    B, T = frames.shape[:2]
    n = int(np.prod(frames.shape[2:]))
    times = np.empty((B,) + frames.shape[2:], np.uint8)
    lib().or_frames_to_times(_p(frames), B, T, n, _p(times))
    return times


# -------------------------------------------------------------- conv + fire

def conv_neuron(in_times, w, T, stride, pad, b, o, y, x) -> np.ndarray:
    in_times = _c(in_times, np.uint8)
    w = _c(w, np.float32)
    _, Ci, Hi, Wi = in_times.shape
    _, _, Kh, Kw = w.shape
    V = np.empty(T, np.float64)
    lib().or_conv_neuron(_p(in_times), T, Ci, Hi, Wi, _p(w), Kh, Kw, stride, pad,
                         int(b), int(o), int(y), int(x), _p(V))
    return V


def fire_neuron(V: np.ndarray, theta: float):
    V = _c(V, np.float64)
    t = np.empty(1, np.uint8)
    v = np.empty(1, np.float64)
    lib().or_fire_neuron(_p(V), V.shape[0], theta, _p(t), _p(v))
    return int(t[0]), float(v[0])


def conv_fire(in_times, w, T, stride, pad, theta, potentials: bool = False):
    """Returns (t_f uint8 B x Co x Ho x Wo, V_key float32[, potentials float32 B x T x Co x Ho x Wo])."""
    in_times = _c(in_times, np.uint8)
    w = _c(w, np.float32)
    B, Ci, Hi, Wi = in_times.shape
    Co, Ci2, Kh, Kw = w.shape
    assert Ci == Ci2
    Ho = (Hi + 2 * pad - Kh) // stride + 1
    Wo = (Wi + 2 * pad - Kw) // stride + 1
    tf = np.empty((B, Co, Ho, Wo), np.uint8)
    vk = np.empty((B, Co, Ho, Wo), np.float32)
    V = np.empty((B, T, Co, Ho, Wo), np.float32) if potentials else None
    lib().or_conv_fire(_p(in_times), B, T, Ci, Hi, Wi, _p(w), Co, Kh, Kw, stride, pad,
                       float(theta), _p(tf), _p(vk), _p(V) if V is not None else None)
    return (tf, vk, V) if potentials else (tf, vk)


# --------------------------------------------------------------------- pool

def pool(in_times, k, stride, pad=0):
    in_times = _c(in_times, np.uint8)
    B, C, Hi, Wi = in_times.shape
    kh, kw = (k, k) if np.isscalar(k) else k
    Ho = (Hi + 2 * pad - kh) // stride + 1
    Wo = (Wi + 2 * pad - kw) // stride + 1
    out = np.empty((B, C, Ho, Wo), np.uint8)
    lib().or_pool(_p(in_times), B, C, Hi, Wi, kh, kw, stride, pad, _p(out))
    return out


# ------------------------------------------------------- inhibition / k-WTA

def inhibit(times, vkey) -> np.ndarray:
    t = np.array(times, np.uint8, copy=True, order="C")
    vkey = _c(vkey, np.float32)
    B, C, H, W = t.shape
    lib().or_inhibit(_p(t), _p(vkey), B, C, H, W)
    return t


def kwta(times, vkey, T, k, radius, readout=False):
    times = _c(times, np.uint8)
    vkey = _c(vkey, np.float32)
    B, C, H, W = times.shape
    win = np.zeros((B, max(k, 1)), WINNER_DTYPE)[:, :k].copy()
    nw = np.zeros(B, np.int32)
    lib().or_kwta(_p(times), _p(vkey), B, C, H, W, T, k, radius, int(bool(readout)),
                  _p(win), _p(nw))
    return win, nw


# --------------------------------------------------------------------- STDP

def stdp_configs(cfgs) -> np.ndarray:
    """cfgs: iterable of (a_causal, a_anticausal, lower, upper, stabilize)."""
    return np.array([tuple(c) for c in cfgs], STDP_DTYPE)


def stdp_update(w, in_times, winners, n_winners, cfgs, stride, pad, winner_cfg=None):
    w_new = np.array(w, np.float32, copy=True, order="C")
    in_times = _c(in_times, np.uint8)
    winners = _c(winners, WINNER_DTYPE)
    n_winners = _c(n_winners, np.int32)
    cfg = _c(cfgs if isinstance(cfgs, np.ndarray) else stdp_configs(cfgs), STDP_DTYPE)
    B, Ci, Hi, Wi = in_times.shape
    Co, Ci2, Kh, Kw = w_new.shape
    assert Ci == Ci2
    k = winners.shape[1]
    wc = None if winner_cfg is None else _c(winner_cfg, np.int32)
    rc = lib().or_stdp_update(_p(w_new), Co, Ci, Kh, Kw, stride, pad, _p(in_times), B, Hi, Wi,
                              _p(winners), _p(n_winners), k, _p(cfg), len(cfg),
                              _p(wc) if wc is not None else None)
    if rc != 0:
        raise ValueError("STDP configurations with different bounds in one update")
    return w_new


def rstdp_select(winners, n_winners, labels, group) -> np.ndarray:
    winners = _c(winners, WINNER_DTYPE)
    n_winners = _c(n_winners, np.int32)
    labels = _c(labels, np.int32)
    B, k = winners.shape
    out = np.empty((B, k), np.int32)
    lib().or_rstdp_select(_p(winners), _p(n_winners), B, k, _p(labels), group, _p(out))
    return out


# --------------------------------------------------------- fully connected

def fc_fire(in_times, w, T, theta, potentials: bool = False):
    """FC layer with IF neurons (§II-E.2): in_times B x I, w O x I.  The FC
    product is the convolution of a 1 x 1 kernel over I input channels."""
    in_times = _c(in_times, np.uint8)
    w = np.asarray(w)
    B, I = in_times.shape
    O = w.shape[0]
    r = conv_fire(in_times.reshape(B, I, 1, 1), w.reshape(O, I, 1, 1), T, 1, 0, theta,
                  potentials=potentials)
    if potentials:
        tf, vk, V = r
        return tf.reshape(B, O), vk.reshape(B, O), V.reshape(B, T, O)
    tf, vk = r
    return tf.reshape(B, O), vk.reshape(B, O)


def fc_wta(times, vkey, T, k, radius, readout=False):
    times = _c(times, np.uint8)
    vkey = _c(vkey, np.float32)
    B, O = times.shape
    win = np.zeros((B, max(k, 1)), WINNER_DTYPE)[:, :k].copy()
    nw = np.zeros(B, np.int32)
    lib().or_fc_wta(_p(times), _p(vkey), B, O, T, k, radius, int(bool(readout)), _p(win), _p(nw))
    return win, nw


def fc_stdp_update(w, in_times, winners, n_winners, cfgs, winner_cfg=None):
    """STDP / R-STDP of an FC layer: the convolution update with a 1 x 1 kernel."""
    w = np.asarray(w, np.float32)
    O, I = w.shape
    in_times = _c(in_times, np.uint8)
    B = in_times.shape[0]
    out = stdp_update(w.reshape(O, I, 1, 1), in_times.reshape(B, I, 1, 1), winners, n_winners,
                      cfgs, 1, 0, winner_cfg=winner_cfg)
    return out.reshape(O, I)


# --------------------------------------------------------- sparse interface

def times_to_spikes(times, T, cap=None):
    """Spike list of a time map (§II-B): (spikes uint32 B x cap, offsets int32
    B x (T + 1)).  Per sample, flat neuron indices grouped by step, ascending
    within a step; offsets[b, t] counts the spikes before step t."""
    times = _c(times, np.uint8)
    B = times.shape[0]
    n = int(np.prod(times.shape[1:]))
    cap = n if cap is None else int(cap)
    spikes = np.zeros((B, max(cap, 1)), np.uint32)[:, :cap].copy()
    offsets = np.empty((B, T + 1), np.int32)
    lib().or_times_to_spikes(_p(times), B, n, T, cap, _p(spikes), _p(offsets))
    return spikes, offsets


def spikes_to_times(spikes, offsets, shape, T):
    """The time map (B x shape) of a spike list; unstored spikes are absent."""
    spikes = _c(spikes, np.uint32)
    offsets = _c(offsets, np.int32)
    B, cap = spikes.shape
    n = int(np.prod(shape))
    times = np.empty((B,) + tuple(shape), np.uint8)
    lib().or_spikes_to_times(_p(spikes), _p(offsets), B, n, T, cap, _p(times))
    return times


def conv_fire_spikes(spikes, offsets, in_shape, w, T, stride, pad, theta):
    """Conv + fire driven by a spike list: in_shape = (Ci, Hi, Wi) of one
    sample.  Returns (t_f uint8 B x Co x Ho x Wo, V_key float32)."""
    spikes = _c(spikes, np.uint32)
    offsets = _c(offsets, np.int32)
    w = _c(w, np.float32)
    B, cap = spikes.shape
    Ci, Hi, Wi = in_shape
    Co, Ci2, Kh, Kw = w.shape
    assert Ci == Ci2 and offsets.shape == (B, T + 1)
    Ho = (Hi + 2 * pad - Kh) // stride + 1
    Wo = (Wi + 2 * pad - Kw) // stride + 1
    tf = np.empty((B, Co, Ho, Wo), np.uint8)
    vk = np.empty((B, Co, Ho, Wo), np.float32)
    lib().or_conv_fire_spikes(_p(spikes), _p(offsets), cap, B, T, Ci, Hi, Wi, _p(w), Co, Kh, Kw,
                              stride, pad, float(theta), _p(tf), _p(vk))
    return tf, vk


# ------------------------------------------ steps around the hot path (§IV)

def log_filters(stds, ksize):
    """The DoG pair that stands for each LoG deviation s (§II-C.3): on-centre
    (s/sqrt 2, s*sqrt 2), then off-centre (s*sqrt 2, s/sqrt 2), deviations
    held in float32 as a filter description carries them."""
    out = []
    for s in stds:
        s = float(np.float32(s))
        a = float(np.float32(s / math.sqrt(2.0)))
        b = float(np.float32(s * math.sqrt(2.0)))
        out += [(int(ksize), a, b), (int(ksize), b, a)]
    return out


def log_filter(img, stds, ksize, pad=-1):
    return dog_filter(img, log_filters(stds, ksize), pad)


def threshold(x, thr, value=0.0):
    x = _c(x, np.float32).copy()
    lib().or_threshold(_p(x), x.size, float(thr), float(value))
    return x


def quantize(w, lower, mid, upper):
    w = _c(w, np.float32).copy()
    lib().or_quantize(_p(w), w.size, float(lower), float(mid), float(upper))
    return w


def gather(times, T):
    times = _c(times, np.uint8)
    out = np.empty(times.shape, np.float32)
    lib().or_gather(_p(times), times.size, int(T), _p(out))
    return out


def lr_factor(samples_seen, a_causal, every=2000, factor=1.5, cap=0.15):
    """Learning-rate schedule of §IV's example: the rates grow by `factor`
    after every `every` samples, until the causal rate reaches `cap` (where it
    stays).  Returns the multiplier of both rates before a batch that starts
    after `samples_seen` samples."""
    k = samples_seen // every
    f = 1.0
    for _ in range(k):
        if a_causal * f >= cap:
            break
        f = min(f * factor, cap / a_causal)
    return f


# ------------------------------------------------- rate coding (§II-D.1)

def rate_code(x, u, T, min_value=0.01):
    """x float B x ... ; u float B x T x ... uniform draws -> frames uint8 B x T x ..."""
    x = _c(x, np.float32)
    B = x.shape[0]
    n = int(np.prod(x.shape[1:]))
    u = _c(u, np.float32)
    assert u.shape == (B, T) + x.shape[1:]
    frames = np.empty(u.shape, np.uint8)
    lib().or_rate_code(_p(x), _p(u), B, n, T, float(min_value), _p(frames))
    return frames


def conv_if_rate(frames, w, stride, pad, theta):
    """IF with reset over rate frames B x T x Ci x Hi x Wi -> (frames B x T x Co x Ho x Wo, counts)."""
    frames = _c(frames, np.uint8)
    w = _c(w, np.float32)
    B, T, Ci, Hi, Wi = frames.shape
    Co, Ci2, Kh, Kw = w.shape
    assert Ci == Ci2
    Ho = (Hi + 2 * pad - Kh) // stride + 1
    Wo = (Wi + 2 * pad - Kw) // stride + 1
    out = np.empty((B, T, Co, Ho, Wo), np.uint8)
    cnt = np.empty((B, Co, Ho, Wo), np.int32)
    lib().or_conv_if_rate(_p(frames), B, T, Ci, Hi, Wi, _p(w), Co, Kh, Kw, stride, pad, float(theta),
                          _p(out), _p(cnt))
    return out, cnt


def rate_pool(frames, counts, k, stride, pad=0):
    frames = _c(frames, np.uint8)
    counts = _c(counts, np.int32)
    B, T, C, Hi, Wi = frames.shape
    kh, kw = (k, k) if np.isscalar(k) else k
    Ho = (Hi + 2 * pad - kh) // stride + 1
    Wo = (Wi + 2 * pad - kw) // stride + 1
    out = np.empty((B, T, C, Ho, Wo), np.uint8)
    oc = np.empty((B, C, Ho, Wo), np.int32)
    lib().or_rate_pool(_p(frames), _p(counts), B, T, C, Hi, Wi, kh, kw, stride, pad, _p(out), _p(oc))
    return out, oc


def fire(V, theta):
    """Fire over dense potentials B x T x ... -> (times uint8 B x ..., vkey float32 B x ...)."""
    V = _c(V, np.float32)
    B, T = V.shape[:2]
    n = int(np.prod(V.shape[2:]))
    tf = np.empty((B,) + V.shape[2:], np.uint8)
    vk = np.empty((B,) + V.shape[2:], np.float32)
    lib().or_fire(_p(V), B, T, n, float(np.float32(theta)), _p(tf), _p(vk))
    return tf, vk
