"""Pins of the oracle's DoG filter (Sec. II-C.1, Eq. 1) and latency coding (Sec. II-D.3).

Each check rests on something other than the oracle itself: library routines
(scipy's Gaussian filter and 2-D correlation, numpy's lexsort), brute force on
tiny inputs, hand-worked examples and invariants.
"""
import numpy as np
import pytest
from scipy.ndimage import gaussian_filter
from scipy.signal import correlate2d

import oracle
from conftest import load_golden

NEVER = 255


# ---------------------------------------------------------------- DoG kernel

@pytest.mark.parametrize("K,s1,s2", [(7, 1.0, 2.0), (3, 3 / 7, 6 / 7), (13, 13 / 7, 26 / 7),
                                     (7, 0.5, 1.0), (5, 2.0, 1.0)])
def test_dog_kernel_is_difference_of_unit_sum_gaussians(K, s1, s2):
    # scipy's truncated Gaussian filter of an impulse is the unit-sum discrete
    # Gaussian of radius R = truncate * sigma (rounded); take R = (K-1)/2.
    R = (K - 1) // 2
    imp = np.zeros((K, K))
    imp[R, R] = 1.0
    g1 = gaussian_filter(imp, s1, truncate=(R + 0.25) / s1, mode="constant")
    g2 = gaussian_filter(imp, s2, truncate=(R + 0.25) / s2, mode="constant")
    k = oracle.dog_kernel(K, s1, s2)
    assert k.dtype == np.float32
    np.testing.assert_allclose(k, (g1 - g2).astype(np.float32), rtol=0, atol=2e-8)
    # zero sum (flat regions give ~0), symmetric under transposition and flips
    assert abs(float(k.astype(np.float64).sum())) < 1e-6
    np.testing.assert_array_equal(k, k.T)
    np.testing.assert_array_equal(k, k[::-1, :])


def test_dog_off_is_exact_negative_of_on():
    on = oracle.dog_kernel(7, 1.0, 2.0)
    off = oracle.dog_kernel(7, 2.0, 1.0)
    np.testing.assert_array_equal(off, -on)


# ---------------------------------------------------------------- DoG filter

def _dog_reference(img, filters):
    """float64 2-D correlation of the scaled image with each float32 kernel (scipy)."""
    B, C, H, W = img.shape
    out = np.zeros((B, C * len(filters), H, W))
    for f, (K, s1, s2) in enumerate(filters):
        k = oracle.dog_kernel(K, s1, s2).astype(np.float64)
        for b in range(B):
            for c in range(C):
                x = img[b, c].astype(np.float32) / np.float32(255.0)
                out[b, c * len(filters) + f] = correlate2d(x.astype(np.float64), k, mode="same")
    return out


def test_dog_filter_matches_library_correlation():
    rng = np.random.default_rng(0)
    img = rng.integers(0, 256, size=(2, 2, 11, 9), dtype=np.uint8)
    filters = [(3, 0.5, 1.0), (7, 1.0, 2.0), (5, 2.0, 1.0)]
    out = oracle.dog_filter(img, filters)
    assert out.shape == (2, 6, 11, 9) and out.dtype == np.float32
    ref = _dog_reference(img, filters)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-6)


def test_dog_filter_channel_order_is_c_times_F_plus_f():
    rng = np.random.default_rng(1)
    img = rng.integers(0, 256, size=(1, 3, 8, 8), dtype=np.uint8)
    filters = [(3, 0.5, 1.0), (5, 1.0, 2.0)]
    out = oracle.dog_filter(img, filters)
    for c in range(3):
        for f, flt in enumerate(filters):
            single = oracle.dog_filter(img[:, c:c + 1], [flt])
            np.testing.assert_array_equal(out[:, c * 2 + f], single[:, 0])


def test_dog_filter_zero_image_gives_zero_and_eq1_shape():
    img = np.zeros((1, 1, 10, 12), np.uint8)
    out = oracle.dog_filter(img, [(7, 1.0, 2.0)])
    assert not out.any()
    # Eq. 1 with an explicit padding: H_o = H + 2P - K + 1
    img = np.full((1, 1, 10, 12), 7, np.uint8)
    out = oracle.dog_filter(img, [(5, 1.0, 2.0)], pad=1)
    assert out.shape == (1, 1, 10 + 2 - 5 + 1, 12 + 2 - 5 + 1)
    out0 = oracle.dog_filter(img, [(5, 1.0, 2.0)], pad=0)
    # interior of a constant image under a zero-sum kernel is ~0
    assert np.abs(out0).max() < 1e-6


def test_dog_filter_off_channel_is_negated_on_channel():
    rng = np.random.default_rng(2)
    img = rng.integers(0, 256, size=(2, 1, 9, 9), dtype=np.uint8)
    out = oracle.dog_filter(img, [(7, 1.0, 2.0), (7, 2.0, 1.0)])
    np.testing.assert_array_equal(out[:, 1], -out[:, 0])


# ------------------------------------------------------------- latency code

def _brute_force_times(x, T, min_value):
    """O(N^2) rank counting per sample: r_i = #{greater} + #{equal with lower index}."""
    B = x.shape[0]
    flat = x.reshape(B, -1).astype(np.float32)
    out = np.full(flat.shape, NEVER, np.int64)
    for b in range(B):
        v = flat[b]
        elig = np.flatnonzero(v > np.float32(min_value))
        N = len(elig)
        for i in elig:
            r = 0
            for j in elig:
                if v[j] > v[i] or (v[j] == v[i] and j < i):
                    r += 1
            out[b, i] = (r * T) // N
    return out.reshape(x.shape)


def test_latency_code_hand_example():
    g = load_golden("h3_latency_code.json")
    v = np.array(g["values"], np.float32)[None]
    t2 = oracle.latency_code(v, 2, min_value=g["min_value"])
    t3 = oracle.latency_code(v, 3, min_value=g["min_value"])
    np.testing.assert_array_equal(t2[0], np.array(g["times_T2"], np.uint8))
    np.testing.assert_array_equal(t3[0], np.array(g["times_T3"], np.uint8))


@pytest.mark.parametrize("seed", range(6))
def test_latency_code_matches_brute_force_ranks(seed):
    rng = np.random.default_rng(seed)
    # coarse values force many exact ties, a few values sit at or below min_value
    x = (rng.integers(-3, 12, size=(3, 2, 5, 6)) / 8.0).astype(np.float32)
    for T in (1, 2, 7, 15, 30, 254):
        got = oracle.latency_code(x, T, min_value=0.01)
        np.testing.assert_array_equal(got, _brute_force_times(x, T, 0.01))


def test_latency_code_matches_library_sort_and_even_bins():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((2, 6, 28, 28)).astype(np.float32)
    x[:, :, :3] = np.round(x[:, :, :3], 1)  # ties
    T = 15
    got = oracle.latency_code(x, T, min_value=0.01)
    for b in range(2):
        v = x[b].ravel()
        idx = np.arange(v.size)
        elig = v > np.float32(0.01)
        order = np.lexsort((idx[elig], -v[elig]))     # value desc, index asc
        N = int(elig.sum())
        ref = np.full(v.size, NEVER, np.int64)
        ref[idx[elig][order]] = (np.arange(N) * T) // N
        np.testing.assert_array_equal(got[b].ravel(), ref)
        counts = np.bincount(got[b].ravel()[elig], minlength=T)
        assert set(counts.tolist()) <= {N // T, -(-N // T)}


def test_latency_code_frames_are_cumulative_and_round_trip():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 3, 7, 5)).astype(np.float32)
    T = 9
    times = oracle.latency_code(x, T)
    frames = oracle.times_to_frames(times, T)
    assert frames.shape == (2, T, 3, 7, 5)
    assert np.all(frames[:, 1:] >= frames[:, :-1])           # S_t subset of S_t+1
    np.testing.assert_array_equal(frames[:, -1] == 1, times != NEVER)
    np.testing.assert_array_equal(oracle.frames_to_times(frames), times)


def test_latency_code_nonfinite_and_empty_samples():
    x = np.array([[[[np.nan, 0.5, 0.0, -1.0]]], [[[0.0, 0.0, 0.0, 0.0]]]], np.float32)
    t = oracle.latency_code(x, 4, min_value=0.01)
    np.testing.assert_array_equal(t[0].ravel(), [NEVER, 0, NEVER, NEVER])
    assert np.all(t[1] == NEVER)


def test_latency_code_linear_mode_properties():
    rng = np.random.default_rng(4)
    T = 10
    vmax = np.float32(2.0)
    # values placed in the middle of each of the T linear bins land in that bin
    mids = (vmax * (1.0 - (np.arange(T) + 0.5) / T)).astype(np.float32)
    x = np.concatenate([[vmax], mids, rng.uniform(0.02, 2.0, size=40).astype(np.float32)])
    x = x.reshape(1, 1, 1, -1)
    t = oracle.latency_code(x, T, min_value=0.01, mode=1).ravel().astype(int)
    assert t[0] == 0
    np.testing.assert_array_equal(t[1:T + 1], np.arange(T))
    order = np.argsort(-x.ravel(), kind="stable")
    assert np.all(np.diff(t[order]) >= 0)                    # higher value never later
    assert t.max() <= T - 1
