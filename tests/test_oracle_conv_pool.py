"""Pins of the oracle's convolution + integrate-and-fire (Sec. II-E.1, Eq. 2) and
spike-time pooling (Sec. II-E.3, Eq. 3).

The potentials are checked against scipy's 2-D correlation of each cumulative
frame (a library routine), against exact integer counts (all-one weights), a
single input spike and the hand-worked 1-filter example; pooling against a
brute-force max over binary frames.
"""
import numpy as np
import pytest
from scipy.signal import correlate2d

import oracle
from conftest import load_golden
from paper_2301_13659_amd.workloads import random_times

NEVER = 255


def _frames(times, T):
    return np.stack([(times <= t) for t in range(T)], axis=1).astype(np.float64)


def _library_potentials(times, w, T, stride, pad):
    """V[b, t, o] = sum_c correlate2d(zero-padded S_t[b, c], W[o, c], 'valid')[::s, ::s]."""
    B, Ci, H, W = times.shape
    Co = w.shape[0]
    S = _frames(times, T)
    Sp = np.pad(S, ((0, 0), (0, 0), (0, 0), (pad, pad), (pad, pad)))
    out = None
    for b in range(B):
        for t in range(T):
            for o in range(Co):
                acc = sum(correlate2d(Sp[b, t, c], w[o, c].astype(np.float64), mode="valid")
                          for c in range(Ci))[::stride, ::stride]
                if out is None:
                    out = np.zeros((B, T, Co) + acc.shape)
                out[b, t, o] = acc
    return out


def test_conv_fire_hand_example():
    g = load_golden("h1_conv_stdp.json")
    times = np.array(g["in_times"], np.uint8)[None, None]
    w = np.array(g["weights"], np.float32)[None, None]
    tf, vk, V = oracle.conv_fire(times, w, g["T"], g["stride"], g["pad"], g["theta"], potentials=True)
    np.testing.assert_array_equal(V[0, :, 0], np.array(g["potentials_by_t"], np.float32))
    np.testing.assert_array_equal(tf[0, 0], np.array(g["t_f"], np.uint8))
    np.testing.assert_array_equal(vk[0, 0], np.array(g["v_key"], np.float32))


@pytest.mark.parametrize("stride,pad,K", [(1, 0, 3), (1, 2, 5), (2, 1, 3), (3, 2, 4), (1, 1, 2)])
def test_conv_potentials_match_library_correlation(stride, pad, K):
    rng = np.random.default_rng(10 * stride + pad + K)
    T = 5
    times = random_times(rng, (2, 3, 9, 8), T, 0.6)
    w = rng.uniform(-0.5, 1.0, size=(4, 3, K, K)).astype(np.float32)
    tf, vk, V = oracle.conv_fire(times, w, T, stride, pad, 1.0, potentials=True)
    ref = _library_potentials(times, w, T, stride, pad)
    assert V.shape == ref.shape
    assert V.shape[-2:] == ((9 + 2 * pad - K) // stride + 1, (8 + 2 * pad - K) // stride + 1)
    np.testing.assert_allclose(V, ref, rtol=1e-6, atol=1e-6)


def test_conv_all_one_weights_count_fired_inputs_exactly():
    rng = np.random.default_rng(5)
    T = 7
    times = random_times(rng, (1, 2, 6, 6), T, 0.5)
    w = np.ones((1, 2, 3, 3), np.float32)
    _, _, V = oracle.conv_fire(times, w, T, 1, 1, np.inf, potentials=True)
    Sp = np.pad(_frames(times, T), ((0, 0), (0, 0), (0, 0), (1, 1), (1, 1)))
    for t in range(T):
        for y in range(6):
            for x in range(6):
                assert V[0, t, 0, y, x] == Sp[0, t, :, y:y + 3, x:x + 3].sum()


def test_conv_single_spike_gives_the_weight():
    T = 4
    times = np.full((1, 1, 5, 5), NEVER, np.uint8)
    times[0, 0, 2, 3] = 2
    w = np.arange(9, dtype=np.float32).reshape(1, 1, 3, 3) / 16.0
    _, _, V = oracle.conv_fire(times, w, T, 1, 1, np.inf, potentials=True)
    assert not V[0, :2].any()
    for ky in range(3):
        for kx in range(3):
            y, x = 2 - ky + 1, 3 - kx + 1    # output whose window holds the spike at (ky, kx)
            if 0 <= y < 5 and 0 <= x < 5:
                assert V[0, 2, 0, y, x] == w[0, 0, ky, kx]
                assert V[0, 3, 0, y, x] == w[0, 0, ky, kx]


def test_fire_is_first_crossing_and_monotone_for_nonnegative_weights():
    rng = np.random.default_rng(6)
    T = 9
    times = random_times(rng, (2, 4, 7, 7), T, 0.4)
    w = rng.uniform(0.0, 1.0, size=(5, 4, 3, 3)).astype(np.float32)
    theta = 3.0
    tf, vk, V = oracle.conv_fire(times, w, T, 1, 1, theta, potentials=True)
    assert np.all(np.diff(V, axis=1) >= 0)
    Vd = np.moveaxis(V, 1, -1)  # B, Co, H, W, T
    for idx in np.ndindex(tf.shape):
        v = Vd[idx]
        above = np.flatnonzero(v > theta)
        if len(above):
            assert tf[idx] == above[0] and vk[idx] == v[above[0]]
        else:
            assert tf[idx] == NEVER and vk[idx] == v[-1]
    # single-neuron entry points agree with the layer
    b, o, y, x = 1, 3, 2, 5
    Vn = oracle.conv_neuron(times, w, T, 1, 1, b, o, y, x)
    np.testing.assert_allclose(Vn, V[b, :, o, y, x], rtol=1e-7)
    assert oracle.fire_neuron(Vn, theta)[0] == tf[b, o, y, x]


def test_fire_infinite_threshold_never_fires():
    rng = np.random.default_rng(8)
    times = random_times(rng, (1, 2, 5, 5), 4, 0.9)
    w = np.ones((2, 2, 3, 3), np.float32)
    tf, vk, V = oracle.conv_fire(times, w, 4, 1, 1, np.inf, potentials=True)
    assert np.all(tf == NEVER)
    np.testing.assert_array_equal(vk, V[:, -1])


# --------------------------------------------------------------------- pool

@pytest.mark.parametrize("k,s,p", [(2, 2, 0), (3, 3, 1), (7, 6, 0), (3, 1, 1)])
def test_pool_is_max_over_binary_frames(k, s, p):
    rng = np.random.default_rng(k * 10 + s + p)
    T = 6
    times = random_times(rng, (2, 3, 16, 13), T, 0.3)
    out = oracle.pool(times, k, s, p)
    Ho, Wo = (16 + 2 * p - k) // s + 1, (13 + 2 * p - k) // s + 1
    assert out.shape == (2, 3, Ho, Wo)
    S = np.pad(_frames(times, T), ((0, 0), (0, 0), (0, 0), (p, p), (p, p)))
    pooled = np.zeros((2, T, 3, Ho, Wo))
    for y in range(Ho):
        for x in range(Wo):
            pooled[..., y, x] = S[..., y * s:y * s + k, x * s:x * s + k].max(axis=(-1, -2))
    ref = np.where(pooled.any(axis=1), pooled.argmax(axis=1), NEVER)
    np.testing.assert_array_equal(out, ref.astype(np.uint8))
