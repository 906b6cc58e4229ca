"""spk_conv_fire_noalloc (the conv without a caller workspace, for callers
that cannot allocate) against spk_conv_fire, through the C ABI.  Both run the
same kernels, so their outputs must agree bit for bit.  Two calls in a row
share the GPU's static scratch; the second is smaller, so stale contents of
the first must not leak into it."""
import ctypes
import math

import numpy as np
import pytest
import torch

from parity import NEVER, gpu, np_
from paper_2301_13659_amd import spk, workloads

pytestmark = pytest.mark.gpu


def _noalloc(in_times, w, T, stride, pad, theta):
    """Direct C-ABI call; outputs preallocated with sentinels (0xAB, NaN)."""
    L = spk.load()
    B, Ci, Hi, Wi = in_times.shape
    Co, _, Kh, Kw = w.shape
    Ho, Wo = L.spk_out_extent(Hi, Kh, stride, pad), L.spk_out_extent(Wi, Kw, stride, pad)
    dev = in_times.device
    out_t = torch.full((B, Co, Ho, Wo), 0xAB, dtype=torch.uint8, device=dev)
    out_v = torch.full((B, Co, Ho, Wo), float("nan"), dtype=torch.float32, device=dev)
    dt = spk.SPK_F16 if w.dtype == torch.float16 else spk.SPK_F32
    st = L.spk_conv_fire_noalloc(ctypes.c_void_p(in_times.data_ptr()), B, T, Ci, Hi, Wi,
                                 ctypes.c_void_p(w.data_ptr()), dt, Co, Kh, Kw, stride, pad,
                                 float(theta), ctypes.c_void_p(out_t.data_ptr()),
                                 ctypes.c_void_p(out_v.data_ptr()), None,
                                 ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream))
    assert st == spk.SPK_OK, L.spk_last_error().decode()
    return out_t, out_v


def _compare(in_times, w, T, stride, pad, theta):
    g_t, g_v = _noalloc(in_times, w, T, stride, pad, theta)
    r_t, r_v = spk.spk_conv_fire(in_times, w, T, stride, pad, theta)
    torch.cuda.synchronize()
    a_t, a_v, b_t, b_v = np_(g_t), np_(g_v), np_(r_t), np_(r_v)
    assert np.all((a_t < T) | (a_t == NEVER))
    assert np.all(np.isfinite(a_v))
    np.testing.assert_array_equal(a_t, b_t)
    np.testing.assert_array_equal(a_v.view(np.uint32), b_v.view(np.uint32))


def _times(rng, shape, T, density):
    t = rng.integers(0, T, size=shape).astype(np.uint8)
    t[rng.random(shape) >= density] = NEVER
    return t


def test_noalloc_matches_workspace_call_twice():
    dev = gpu()
    # 1: the spike-input layer at full size (B = 128, 64 x 64 x 64, 128 maps,
    #    half weights, T = 30, 5 % input density): 34 MiB of scratch
    wl = workloads.get(5)
    s = wl.convs[0]
    t5 = torch.from_numpy(workloads.make_spike_times(wl, 1)).to(dev)
    w5 = torch.from_numpy(workloads.make_weights(wl, 1)).to(dev).to(torch.float16)
    _compare(t5, w5, wl.T, s.stride, s.pad, s.theta)
    # 2: a smaller layer right after it: 250 maps 3x3 over 30 x 14 x 14,
    #    float weights, B = 16, T = 15
    rng = np.random.default_rng(7)
    t2 = torch.from_numpy(_times(rng, (16, 30, 14, 14), 15, 0.8)).to(dev)
    w2 = torch.from_numpy(rng.normal(0.8, 0.05, (250, 30, 3, 3)).clip(0, 1).astype(np.float32)).to(dev)
    _compare(t2, w2, 15, 1, 1, 10.0)
    # 3: smaller still, a readout layer (theta = +inf: split-K partial sums in
    #    the scratch)
    t3 = torch.from_numpy(_times(rng, (4, 250, 5, 5), 15, 0.5)).to(dev)
    w3 = torch.from_numpy(rng.uniform(0, 1, (200, 250, 5, 5)).astype(np.float32)).to(dev)
    _compare(t3, w3, 15, 1, 2, math.inf)
