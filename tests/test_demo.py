"""The steps around the hot path in the paper's example network (§II-C.3
and §IV): LoG bank, threshold, quantize, gather and the learning-rate
schedule.  The oracle pinned on the CPU, then libspk against it on the GPU."""
import math

import numpy as np
import pytest
import torch

import oracle
from parity import gpu, np_
from paper_2301_13659_amd import spk
from paper_2301_13659_amd import workloads as wls
from paper_2301_13659_amd.workloads import random_times

NEVER = 255
STDS = (0.471, 1.099, 2.042)


# ----------------------------------------------------------- oracle pins

def test_oracle_log_pair_tracks_the_laplacian_of_gaussian():
    """Each on-centre channel is a DoG approximation of -LoG(s): on a smooth
    image it correlates with scipy's Gaussian Laplacian (negated) almost
    perfectly, and the off-centre channel is its exact negative."""
    from scipy.ndimage import gaussian_filter, gaussian_laplace
    rng = np.random.default_rng(3)
    img = np.clip(gaussian_filter(rng.uniform(0, 255, (64, 64)), 2.0) * 3 - 200, 0, 255).astype(np.uint8)
    out = oracle.log_filter(img[None, None], STDS, 15)
    assert out.shape == (1, 6, 64, 64)
    for i, s in enumerate(STDS):
        on, off = out[0, 2 * i], out[0, 2 * i + 1]
        np.testing.assert_array_equal(off, -on)
        ref = -gaussian_laplace(img.astype(np.float64) / 255.0, s, mode="constant")
        c = 8  # away from the border, where the truncated windows differ
        r = np.corrcoef(on[c:-c, c:-c].ravel(), ref[c:-c, c:-c].ravel())[0, 1]
        # below a pixel the sampled kernels of both sides stop being smooth,
        # so the smallest deviation only keeps the shape
        assert r > (0.8 if s < 1 else 0.995), (s, r)
        assert np.corrcoef(off[c:-c, c:-c].ravel(), ref[c:-c, c:-c].ravel())[0, 1] < -0.8


def test_oracle_log_filters_are_the_paper_pairs():
    f = oracle.log_filters([1.0], 7)
    assert f[0][0] == 7 and f[1][0] == 7
    assert math.isclose(f[0][1], 1 / math.sqrt(2), rel_tol=1e-7)
    assert math.isclose(f[0][2], math.sqrt(2), rel_tol=1e-7)
    assert f[1][1] == f[0][2] and f[1][2] == f[0][1]


def test_oracle_threshold_quantize_gather_closed_forms():
    x = np.array([-1.0, 0.0, 0.01, 0.0100001, 0.5, np.nan, np.inf], np.float32)
    got = oracle.threshold(x, 0.01, 0.0)
    np.testing.assert_array_equal(got, np.array([0, 0, 0, 0.0100001, 0.5, 0, np.inf], np.float32))
    w = np.array([0.0, 0.2, 0.4999, 0.5, 0.7, 1.0], np.float32)
    np.testing.assert_array_equal(oracle.quantize(w, 0.0, 0.5, 1.0), [0, 0, 0, 1, 1, 1])
    t = np.array([[0, 3, 14, NEVER, 15]], np.uint8)
    np.testing.assert_array_equal(oracle.gather(t, 15), [[15, 12, 1, 0, 0]])


@pytest.mark.parametrize("T", [1, 7, 30])
def test_oracle_gather_is_the_sum_of_the_frames(T):
    rng = np.random.default_rng(T)
    t = random_times(rng, (2, 3, 5, 4), T, 0.6)
    frames = oracle.times_to_frames(t, T)
    np.testing.assert_array_equal(oracle.gather(t, T), frames.sum(axis=1).astype(np.float32))


def test_oracle_learning_rate_schedule():
    a0 = 0.0004
    assert [oracle.lr_factor(n, a0) for n in (0, 1999, 2000, 3999, 4000, 6000)] == [1, 1, 1.5, 1.5, 2.25, 3.375]
    # 0.0004 * 1.5^14 = 0.1168 < 0.15 <= 0.0004 * 1.5^15: the fifteenth step stops at the cap
    assert math.isclose(oracle.lr_factor(14 * 2000, a0) * a0, a0 * 1.5 ** 14)
    assert math.isclose(oracle.lr_factor(15 * 2000, a0) * a0, 0.15)
    assert math.isclose(oracle.lr_factor(10 ** 6, a0) * a0, 0.15)


# ------------------------------------------------------ GPU against oracle

def _t(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


@pytest.mark.gpu
@pytest.mark.parametrize("B,C,H,W,stds,k,pad", [(3, 1, 28, 28, STDS, 7, -1), (2, 2, 33, 17, (0.8,), 5, 2),
                                                 (1, 1, 160, 250, (0.5, 1.0, 1.5, 2.0), 9, -1)])
def test_log_filter_bit_exact(B, C, H, W, stds, k, pad):
    dev = gpu()
    rng = np.random.default_rng(H)
    img = rng.integers(0, 256, size=(B, C, H, W), dtype=np.uint8)
    g = np_(spk.spk_log_filter(_t(img, dev), stds, k, pad))
    o = oracle.log_filter(img, stds, k, pad)
    np.testing.assert_array_equal(g.view(np.uint32), o.view(np.uint32))


@pytest.mark.gpu
def test_threshold_quantize_gather_bit_exact():
    dev = gpu()
    rng = np.random.default_rng(11)
    x = rng.normal(0, 0.05, size=(5, 6, 28, 28)).astype(np.float32)
    x.flat[:4] = [np.nan, np.inf, -np.inf, 0.01]
    g = spk.spk_threshold(_t(x, dev), 0.01, 0.0)
    np.testing.assert_array_equal(np_(g).view(np.uint32), oracle.threshold(x, 0.01, 0.0).view(np.uint32))
    w = rng.uniform(0, 1, size=(100, 6, 5, 5)).astype(np.float32)
    w.flat[:2] = [0.5, np.nextafter(np.float32(0.5), np.float32(0))]
    gw = _t(w, dev)
    g16 = gw.to(torch.float16)
    spk.spk_quantize(gw, 0.0, 0.5, 1.0, w_f16=g16)
    ref = oracle.quantize(w, 0.0, 0.5, 1.0)
    np.testing.assert_array_equal(np_(gw), ref)
    np.testing.assert_array_equal(np_(g16), ref.astype(np.float16))
    for T in (1, 15, 254):
        t = random_times(rng, (4, 200, 4, 4), T, 0.5)
        np.testing.assert_array_equal(np_(spk.spk_gather(_t(t, dev), T)), oracle.gather(t, T))


# ------------------------------------------------- the fire step on its own

@pytest.mark.parametrize("theta", [2.0, -0.5, math.inf])
def test_oracle_fire_matches_the_conv_firing(theta):
    """Fire over the conv's dense potentials gives the conv's own spikes."""
    rng = np.random.default_rng(9)
    t = random_times(rng, (2, 4, 9, 8), 10, 0.3)
    w = rng.uniform(-0.3, 1, size=(5, 4, 3, 3)).astype(np.float32)
    tf, vk, V = oracle.conv_fire(t, w, 10, 1, 1, theta, potentials=True)
    f_t, f_v = oracle.fire(V, theta)
    np.testing.assert_array_equal(f_t, tf)
    np.testing.assert_allclose(f_v, vk, rtol=1e-6, atol=1e-6)


def test_oracle_fire_closed_form():
    V = np.array([[[0.5], [1.5], [3.0]], [[0.1], [0.2], [0.3]]], np.float32)  # B = 2, T = 3, n = 1
    tf, vk = oracle.fire(V, 1.0)
    assert tf.ravel().tolist() == [1, NEVER] and vk.ravel().tolist() == [1.5, np.float32(0.3)]


@pytest.mark.gpu
@pytest.mark.parametrize("B,T,shape,theta", [(3, 15, (30, 28, 28), 6.0), (2, 7, (5, 3, 3), -0.1),
                                             (2, 30, (16, 8, 8), 20.0), (1, 4, (3,), 1.0)])
def test_fire_bit_exact(B, T, shape, theta):
    dev = gpu()
    rng = np.random.default_rng(T)
    V = np.cumsum(rng.uniform(-0.5, 2.0, size=(B, T) + shape), axis=1).astype(np.float32)
    g_t, g_v = spk.spk_fire(_t(V, dev), theta)
    o_t, o_v = oracle.fire(V, theta)
    np.testing.assert_array_equal(np_(g_t), o_t)
    np.testing.assert_array_equal(np_(g_v), o_v)
