"""Per-call parity of libspk against the CPU oracle on seeded random inputs.

Each call gets the same inputs on both sides (stage isolation); sizes span
several workgroup tiles with ragged tails, plus the edge cases of each
operation.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from conftest import load_golden
from parity import (NEVER, W_ABS, check_fire, check_potentials, excused_from_potentials, gpu,
                    np_, winners_list)
from paper_2301_13659_amd import spk
from paper_2301_13659_amd.workloads import random_times

pytestmark = pytest.mark.gpu


def _t(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


# ---------------------------------------------------------------------- DoG

@pytest.mark.parametrize("shape,filters,pad", [
    ((3, 2, 37, 70), [(7, 1.0, 2.0), (7, 2.0, 1.0)], -1),
    ((2, 1, 28, 28), [(3, 3 / 7, 6 / 7), (3, 6 / 7, 3 / 7), (7, 1.0, 2.0), (7, 2.0, 1.0),
                      (13, 13 / 7, 26 / 7), (13, 26 / 7, 13 / 7)], -1),
    ((1, 1, 160, 250), [(7, 0.5, 1.0), (7, 1.0, 0.5), (7, 1.0, 2.0), (7, 2.0, 1.0),
                        (7, 1.5, 3.0), (7, 3.0, 1.5)], -1),
    ((2, 3, 17, 9), [(5, 1.0, 2.0), (5, 0.7, 1.9)], 2),
    ((1, 1, 9, 11), [(5, 1.0, 2.0)], 0),
    ((1, 2, 5, 4), [(21, 3.0, 6.0), (1, 1.0, 2.0)], -1),
])
def test_dog_bit_exact(shape, filters, pad):
    dev = gpu()
    rng = np.random.default_rng(sum(shape))
    img = rng.integers(0, 256, size=shape, dtype=np.uint8)
    got = np_(spk.spk_dog_filter(_t(img, dev), filters, pad))
    ref = oracle.dog_filter(img, filters, pad)
    assert got.shape == ref.shape
    np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))


_DOG6 = [(3, 3 / 7, 6 / 7), (3, 6 / 7, 3 / 7), (7, 1.0, 2.0), (7, 2.0, 1.0),
         (13, 13 / 7, 26 / 7), (13, 26 / 7, 13 / 7)]


# fused (one workgroup per sample) and two-call cases: the three-layer net's
# input stage, an explicit pad, a 21x21 kernel beside a 1x1, more values per
# sample than the fused kernel ranks, and more coefficients than one block holds
@pytest.mark.parametrize("shape,filters,pad,T", [
    ((64, 1, 28, 28), _DOG6, -1, 15),
    ((2, 3, 17, 9), [(5, 1.0, 2.0), (5, 0.7, 1.9)], 2, 15),
    ((3, 1, 5, 4), [(21, 3.0, 6.0), (1, 1.0, 2.0)], -1, 4),
    ((3, 2, 37, 70), [(7, 1.0, 2.0), (7, 2.0, 1.0)], -1, 30),
    ((2, 1, 30, 20), [(13, 1.0, 2.0), (13, 2.0, 1.0), (13, 1.5, 3.0)], -1, 15),
])
def test_dog_latency_code_equals_filter_then_code(shape, filters, pad, T):
    dev = gpu()
    rng = np.random.default_rng(sum(shape) + T)
    img = rng.integers(0, 256, size=shape, dtype=np.uint8)
    img[1] = 0                                        # a sample with no eligible value
    ti = _t(img, dev)
    x = spk.spk_dog_filter(ti, filters, pad)
    ref = np_(spk.spk_latency_code(x, T, 0.01))
    np.testing.assert_array_equal(ref, oracle.latency_code(oracle.dog_filter(img, filters, pad), T, 0.01))
    times = torch.full(tuple(x.shape), 0xAB, dtype=torch.uint8, device=dev)
    d = torch.full(tuple(x.shape), float("nan"), dtype=torch.float32, device=dev)
    spk.spk_dog_latency_code(ti, filters, T, 0.01, pad, times=times, dog_out=d)
    np.testing.assert_array_equal(np_(times), ref)
    np.testing.assert_array_equal(np_(d).view(np.uint32), np_(x).view(np.uint32))
    alone = spk.spk_dog_latency_code(ti, filters, T, 0.01, pad)  # no filter outputs asked for
    np.testing.assert_array_equal(np_(alone), ref)


# ------------------------------------------------------------ latency code

@pytest.mark.parametrize("shape,T", [((5, 2, 28, 28), 15), ((3, 6, 28, 28), 15), ((2, 1, 1, 1), 4),
                                     ((2, 1, 90, 91), 30), ((2, 6, 160, 250), 30),
                                     ((1, 3, 57, 101), 254), ((4, 1, 1, 8192), 7)])
def test_latency_code_bit_exact(shape, T):
    dev = gpu()
    rng = np.random.default_rng(shape[-1] + T)
    x = rng.standard_normal(shape).astype(np.float32)
    x.reshape(shape[0], -1)[:, ::7] = np.round(x.reshape(shape[0], -1)[:, ::7], 1)  # ties
    if shape[0] > 1:
        x[1] = -1.0                                   # a sample with no eligible value
    x.reshape(-1)[::13] = -0.0
    got = np_(spk.spk_latency_code(_t(x, dev), T, 0.01))
    np.testing.assert_array_equal(got, oracle.latency_code(x, T, 0.01))


def test_latency_code_crowded_and_spread_samples():
    # bucketed ranks for spread values, the sort for samples with many equal values
    dev = gpu()
    rng = np.random.default_rng(21)
    x = rng.standard_normal((5, 6, 28, 28)).astype(np.float32)
    x[1] = 0.5                                        # one value: a single crowded bucket
    x[2] = np.where(rng.random((6, 28, 28)) < 0.5, 0.25, 2.0).astype(np.float32)
    x[3, :3] = 1.0                                    # half the sample tied, half spread
    x[4] = np.exp(rng.uniform(-20, 20, (6, 28, 28))).astype(np.float32)  # a wide span of exponents
    for T in (15, 30, 254):
        got = np_(spk.spk_latency_code(_t(x, dev), T, 0.01))
        np.testing.assert_array_equal(got, oracle.latency_code(x, T, 0.01))


def test_latency_code_large_samples_crowded_and_sparse():
    # samples over 8192 values: the boundary selection with one bucket holding
    # every key (ties ordered by index), two values, half tied, a wide span of
    # exponents, fewer eligible values than steps, one, and none
    dev = gpu()
    rng = np.random.default_rng(33)
    shape = (7, 6, 160, 250)
    x = rng.standard_normal(shape).astype(np.float32)
    x[0] = 0.5
    x[1] = np.where(rng.random(shape[1:]) < 0.5, 0.25, 2.0).astype(np.float32)
    x[2, :3] = 1.0
    x[3] = np.exp(rng.uniform(-20, 20, shape[1:])).astype(np.float32)
    x[4] = -1.0
    x[4].reshape(-1)[[3, 5, 100, 7000, 239999]] = [0.5, 1.0, 2.0, 2.0, 3.0]
    x[5] = -1.0
    x[5, 2, 80, 125] = 4.0
    x[6] = np.nan
    for T in (15, 30, 254):
        got = np_(spk.spk_latency_code(_t(x, dev), T, 0.01))
        np.testing.assert_array_equal(got, oracle.latency_code(x, T, 0.01))


def test_latency_code_frames_and_linear_mode():
    dev = gpu()
    rng = np.random.default_rng(11)
    x = rng.uniform(-0.5, 1.0, size=(3, 2, 19, 23)).astype(np.float32)
    T = 9
    times, frames = spk.spk_latency_code(_t(x, dev), T, 0.01, frames=True)
    ref = oracle.latency_code(x, T, 0.01)
    np.testing.assert_array_equal(np_(times), ref)
    np.testing.assert_array_equal(np_(frames), oracle.times_to_frames(ref, T))
    lin = spk.spk_latency_code(_t(x, dev), T, 0.01, mode=spk.SPK_CODE_LINEAR)
    np.testing.assert_array_equal(np_(lin), oracle.latency_code(x, T, 0.01, mode=1))


def test_latency_code_hand_example():
    dev = gpu()
    g = load_golden("h3_latency_code.json")
    v = np.array(g["values"], np.float32)[None]
    for T, key in ((2, "times_T2"), (3, "times_T3")):
        got = np_(spk.spk_latency_code(_t(v, dev), T, g["min_value"]))
        np.testing.assert_array_equal(got[0], np.array(g[key], np.uint8))


def test_frames_times_round_trip():
    dev = gpu()
    rng = np.random.default_rng(12)
    times = random_times(rng, (3, 4, 7, 9), 11, 0.6)
    fr = spk.spk_times_to_frames(_t(times, dev), 11)
    np.testing.assert_array_equal(np_(fr), oracle.times_to_frames(times, 11))
    back = spk.spk_frames_to_times(fr)
    np.testing.assert_array_equal(np_(back), times)


# ----------------------------------------------------------- conv + fire

CONV_CASES = [
    # B, Ci, Hi, Wi, Co, K, stride, pad, T, theta, density, dtype
    (3, 5, 19, 23, 37, 3, 1, 1, 7, 4.0, 0.4, "f32"),
    (2, 6, 28, 28, 30, 5, 1, 2, 15, 15.0, 0.3, "f32"),
    (2, 30, 14, 14, 65, 3, 1, 1, 15, 10.0, 0.2, "f32"),
    (1, 3, 33, 31, 9, 4, 2, 1, 5, 2.0, 0.5, "f32"),
    (2, 4, 26, 41, 20, 17, 1, 0, 6, 42.0, 0.5, "f32"),
    (2, 64, 12, 12, 128, 3, 1, 1, 30, 20.0, 0.05, "f16"),
    (2, 16, 9, 10, 33, 3, 1, 1, 12, 3.0, 0.3, "f16"),
    (1, 7, 5, 5, 11, 5, 1, 2, 15, math.inf, 0.6, "f32"),
    (3, 250, 5, 5, 200, 5, 1, 2, 15, math.inf, 0.3, "f32"),
    (2, 40, 6, 7, 24, 3, 1, 1, 9, math.inf, 0.5, "f16"),
    (1, 1, 3, 3, 1, 3, 3, 0, 1, 0.5, 1.0, "f32"),
    (2, 16, 11, 13, 40, 5, 1, 2, 10, 12.0, 0.3, "f32"),     # 13 subtiles: one row tile per wave
    (4, 2, 170, 250, 8, 3, 1, 1, 8, 2.5, 0.2, "f32"),       # several row groups per block, ragged
    (2, 8, 10, 10, 20, 3, 1, 1, 32, 5.0, 0.3, "f32"),       # T = 32
    (2, 8, 10, 10, 20, 3, 1, 1, 33, 5.0, 0.3, "f32"),       # T = 33
    (2, 30, 14, 14, 37, 3, 1, 1, 15, 3.0, 0.02, "f32"),     # sparse arrivals
    (2, 5, 9, 9, 7, 3, 1, 1, 5, -0.5, 0.3, "f32"),          # negative threshold
    (2, 6, 40, 40, 33, 5, 1, 2, 20, 6.0, 0.04, "f32"),      # unaligned channels, sparse, two column tiles
    (2, 3, 21, 19, 40, 3, 1, 0, 16, 1.5, 0.3, "f16"),       # unaligned channels, half weights, T = 16
    (2, 112, 6, 6, 40, 3, 1, 1, 12, 60.0, 0.3, "f16"),      # 1008 taps: exactly 32 subtiles of 32
    (3, 1000, 1, 1, 65, 1, 1, 0, 30, 60.0, 0.2, "f32"),     # 1 x 1 kernel over 1000 channels (an FC layer)
    (32, 30, 14, 14, 250, 3, 1, 1, 15, 10.0, 0.85, "f32"),  # the three-layer net's conv2 at B = 32: more
                                                            # than 64 positions per block range
    (2, 6, 160, 250, 4, 5, 1, 2, 30, 15.0, 0.05, "f32"),    # four maps: 2 x 4 position blocks, ragged x
    (2, 3, 21, 23, 5, 3, 2, 1, 12, 2.0, 0.4, "f32"),        # few maps, stride 2, ragged blocks
    (2, 8, 17, 19, 2, 5, 1, 2, 9, 3.0, 0.3, "f16"),         # two maps, half weights: 4 x 4 blocks
    (3, 12, 11, 20, 24, 3, 1, 1, 9, 4.0, 0.3, "f32"),       # 4 x 4 byte-transpose packing, padded channels
    (2, 4, 15, 16, 10, 3, 2, 1, 6, 2.0, 0.4, "f16"),        # the same with 4 channels and stride 2
    (2, 64, 12, 12, 96, 3, 1, 1, 30, 20.0, 0.05, "f16"),    # LDS-fed kernel: three column tiles (a pair
                                                            # with a zero second tile)
    (2, 64, 9, 13, 40, 3, 1, 1, 20, 12.0, 0.1, "f16"),      # LDS-fed kernel: 40 maps, T = 20, ragged
    (2, 6, 20, 22, 70, 5, 1, 2, 15, 16.0, 0.3, "f32"),      # LDS-fed kernel, 5x5 over 6 channels, float
                                                            # masters: three column tiles
    (2, 100, 14, 14, 200, 3, 1, 1, 15, 5.0, 0.3, "f32"),    # chunked LDS-fed kernel: 3x3 over 100
                                                            # channels, one kernel row of slices per chunk
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_fire_matches_oracle(case):
    dev = gpu()
    B, Ci, Hi, Wi, Co, K, s, p, T, theta, dens, dt = case
    rng = np.random.default_rng(B * 1000 + Ci * 10 + K)
    times = random_times(rng, (B, Ci, Hi, Wi), T, dens)
    w = rng.uniform(0.0, 1.0, size=(Co, Ci, K, K)).astype(np.float32)
    if dt == "f16":
        w = w.astype(np.float16).astype(np.float32)
    w_dev = _t(w, dev).to(torch.float16) if dt == "f16" else _t(w, dev)
    g_tf, g_vk, g_V = spk.spk_conv_fire(_t(times, dev), w_dev, T, s, p, theta, potentials=True)
    o_tf, o_vk, o_V = oracle.conv_fire(times, w, T, s, p, theta, potentials=True)
    check_potentials(np_(g_V), o_V)
    exc = excused_from_potentials(o_V, theta)
    check_fire(np_(g_tf), np_(g_vk), o_tf, o_vk, exc)
    # without the dense potentials the call takes the firing kernels (or, for a
    # readout layer, the single-frame GEMM): same rules against the oracle
    g_tf2, g_vk2 = spk.spk_conv_fire(_t(times, dev), w_dev, T, s, p, theta)
    if math.isinf(theta):
        assert np.all(np_(g_tf2) == NEVER)
        check_potentials(np_(g_vk2), o_vk, "readout v_key")
    else:
        check_fire(np_(g_tf2), np_(g_vk2), o_tf, o_vk, exc)


def test_conv_fire_hand_example():
    dev = gpu()
    g = load_golden("h1_conv_stdp.json")
    times = np.array(g["in_times"], np.uint8)[None, None]
    w = np.array(g["weights"], np.float32)[None, None]
    tf, vk, V = spk.spk_conv_fire(_t(times, dev), _t(w, dev), g["T"], 1, 0, g["theta"],
                                  potentials=True)
    np.testing.assert_array_equal(np_(V)[0, :, 0], np.array(g["potentials_by_t"], np.float32))
    np.testing.assert_array_equal(np_(tf)[0, 0], np.array(g["t_f"], np.uint8))
    np.testing.assert_array_equal(np_(vk)[0, 0], np.array(g["v_key"], np.float32))
    # the firing kernels (no dense potentials): dyadic values, exact in any order
    tf2, vk2 = spk.spk_conv_fire(_t(times, dev), _t(w, dev), g["T"], 1, 0, g["theta"])
    np.testing.assert_array_equal(np_(tf2)[0, 0], np.array(g["t_f"], np.uint8))
    np.testing.assert_array_equal(np_(vk2)[0, 0], np.array(g["v_key"], np.float32))


def test_conv_fire_silent_input_and_negative_weights():
    dev = gpu()
    rng = np.random.default_rng(21)
    times = np.full((2, 3, 8, 8), NEVER, np.uint8)
    times[1] = random_times(rng, (3, 8, 8), 6, 0.7)
    w = rng.uniform(-1.0, 1.0, size=(5, 3, 3, 3)).astype(np.float32)
    g_tf, g_vk, g_V = spk.spk_conv_fire(_t(times, dev), _t(w, dev), 6, 1, 1, 0.5, potentials=True)
    o_tf, o_vk, o_V = oracle.conv_fire(times, w, 6, 1, 1, 0.5, potentials=True)
    assert np.all(np_(g_tf)[0] == NEVER) and not np_(g_V)[0].any()
    check_potentials(np_(g_V), o_V)
    check_fire(np_(g_tf), np_(g_vk), o_tf, o_vk, excused_from_potentials(o_V, 0.5))
    g_tf2, g_vk2 = spk.spk_conv_fire(_t(times, dev), _t(w, dev), 6, 1, 1, 0.5)
    assert np.all(np_(g_tf2)[0] == NEVER) and not np_(g_vk2)[0].any()
    check_fire(np_(g_tf2), np_(g_vk2), o_tf, o_vk, excused_from_potentials(o_V, 0.5))


@pytest.mark.parametrize("case", [CONV_CASES[5], CONV_CASES[21]])
def test_conv_fire_unaligned_outputs(case):
    """Outputs off the 16-byte (V) and 4-byte (t) alignment the word stores
    need: the element stores give the same bits, and nothing outside the
    outputs is written."""
    dev = gpu()
    B, Ci, Hi, Wi, Co, K, s, p, T, theta, dens, dt = case
    rng = np.random.default_rng(7)
    times = _t(random_times(rng, (B, Ci, Hi, Wi), T, dens), dev)
    w = _t(rng.uniform(0.0, 1.0, size=(Co, Ci, K, K)).astype(np.float32), dev)
    w = w.to(torch.float16) if dt == "f16" else w
    tf, vk = spk.spk_conv_fire(times, w, T, s, p, theta)
    n = tf.numel()
    bt = torch.full((n + 2,), 0xAB, dtype=torch.uint8, device=dev)
    bv = torch.full((n + 2,), float("nan"), dtype=torch.float32, device=dev)
    tf2, vk2 = spk.spk_conv_fire(times, w, T, s, p, theta, out_times=bt[1:n + 1].view(tf.shape),
                                 out_vkey=bv[1:n + 1].view(vk.shape))
    np.testing.assert_array_equal(np_(tf2), np_(tf))
    np.testing.assert_array_equal(np_(vk2).view(np.uint32), np_(vk).view(np.uint32))
    assert int(bt[0]) == 0xAB and int(bt[-1]) == 0xAB
    assert math.isnan(float(bv[0])) and math.isnan(float(bv[-1]))


@pytest.mark.parametrize("shape", [(128, 10, 10, 128, 0.05), (128, 20, 20, 96, 0.1)])
def test_conv_fire_ranges_of_several_groups(shape):
    """Half weights, 3x3 over 64 channels, T = 30, B = 128 samples of 10x10 or
    20x20 (one sample per block range: two or seven 64-position groups, the
    last one ragged; 96 maps leave the second tile of a column pair empty).
    The oracle's event form gives the same bits (half weights sum exactly in
    any order)."""
    dev = gpu()
    B, H, W, Co, dens = shape
    T, theta = 30, 20.0
    rng = np.random.default_rng(H * 1000 + Co)
    times = random_times(rng, (B, 64, H, W), T, dens)
    w16 = rng.uniform(0.7, 0.9, size=(Co, 64, 3, 3)).astype(np.float16)
    tf, vk = spk.spk_conv_fire(_t(times, dev), _t(w16, dev), T, 1, 1, theta)
    sp, off = oracle.times_to_spikes(times, T)
    o_tf, o_vk = oracle.conv_fire_spikes(sp, off, times.shape[1:], w16.astype(np.float32), T, 1, 1, theta)
    np.testing.assert_array_equal(np_(tf), o_tf)
    np.testing.assert_array_equal(np_(vk), o_vk)


# --------------------------------------------------------------------- pool

@pytest.mark.parametrize("shape,k,s,p", [((3, 30, 28, 28), 2, 2, 0), ((2, 250, 14, 14), 3, 3, 1),
                                         ((2, 4, 160, 250), 7, 6, 0), ((1, 3, 5, 7), 3, 1, 1),
                                         ((1, 2, 4, 4), 5, 1, 2)])
def test_pool_bit_exact(shape, k, s, p):
    dev = gpu()
    rng = np.random.default_rng(shape[1])
    times = random_times(rng, shape, 15, 0.2)
    got = np_(spk.spk_pool(_t(times, dev), k, s, p))
    np.testing.assert_array_equal(got, oracle.pool(times, k, s, p))


# ------------------------------------------------------------ pool + conv

POOL_CONV_CASES = [
    # B, Ci, H0, W0, (pool k, stride, pad), Co, K, stride, pad, T, theta, density, dtype
    (4, 30, 28, 28, (2, 2, 0), 250, 3, 1, 1, 15, 10.0, 0.3, "f32"),    # three-layer net, conv2
    (3, 250, 14, 14, (3, 3, 1), 200, 5, 1, 2, 15, math.inf, 0.3, "f32"),  # and its readout
    (2, 40, 11, 13, (2, 2, 0), 24, 3, 1, 1, 9, math.inf, 0.5, "f16"),  # half readout, ragged
    (2, 4, 160, 250, (7, 6, 0), 20, 17, 1, 0, 30, 42.0, 0.05, "f32"),  # large-image conv2
    (2, 8, 12, 12, ((2, 3), 2, 1), 20, 3, 1, 1, 40, 5.0, 0.3, "f32"),  # 2 x 3 window, T = 40
    (2, 5, 9, 9, (1, 1, 0), 7, 3, 1, 1, 5, 2.0, 0.3, "f32"),           # 1 x 1 window: identity
    (1, 16, 100, 90, (2, 2, 0), 12, 3, 1, 1, 7, math.inf, 0.3, "f32"),  # readout, planes too big to stage
]


@pytest.mark.parametrize("case", POOL_CONV_CASES)
def test_pool_conv_fire_equals_pool_then_conv(case):
    """spk_pool_conv_fire pools inside the conv's packing pass (or with the
    pool kernel in front, on the paths that do not pack): its pooled map and
    outputs are bit-identical to spk_pool followed by spk_conv_fire, and they
    match the oracle's pool and conv."""
    dev = gpu()
    B, Ci, H0, W0, (pk, ps, pp), Co, K, s, p, T, theta, dens, dt = case
    rng = np.random.default_rng(B * 1000 + Ci * 10 + K + 7)
    times0 = random_times(rng, (B, Ci, H0, W0), T, dens)
    w = rng.uniform(0.0, 1.0, size=(Co, Ci, K, K)).astype(np.float32)
    if dt == "f16":
        w = w.astype(np.float16).astype(np.float32)
    w_dev = _t(w, dev).to(torch.float16) if dt == "f16" else _t(w, dev)
    t0 = _t(times0, dev)
    ref_pooled = spk.spk_pool(t0, pk, ps, pp)
    ref_tf, ref_vk = spk.spk_conv_fire(ref_pooled, w_dev, T, s, p, theta)
    pooled, tf, vk = spk.spk_pool_conv_fire(t0, (pk, ps, pp), w_dev, T, s, p, theta)
    np.testing.assert_array_equal(np_(pooled), np_(ref_pooled))
    np.testing.assert_array_equal(np_(tf), np_(ref_tf))
    np.testing.assert_array_equal(np_(vk), np_(ref_vk))
    tf1, vk1 = spk.spk_pool_conv_fire(t0, (pk, ps, pp), w_dev, T, s, p, theta, keep_pooled=False)
    np.testing.assert_array_equal(np_(tf1), np_(ref_tf))
    np.testing.assert_array_equal(np_(vk1), np_(ref_vk))
    if math.isinf(theta):
        # readout weights packed once, then read on every call
        packed = spk.spk_conv_pack_weights(w_dev)
        for _ in range(2):
            tf2, vk2 = spk.spk_pool_conv_fire(t0, (pk, ps, pp), w_dev, T, s, p, theta,
                                              packed_w=packed, keep_pooled=False)
            np.testing.assert_array_equal(np_(tf2), np_(ref_tf))
            np.testing.assert_array_equal(np_(vk2), np_(ref_vk))
    # and the oracle, from the raw map
    o_pooled = oracle.pool(times0, pk, ps, pp)
    np.testing.assert_array_equal(np_(pooled), o_pooled)
    o_tf, o_vk, o_V = oracle.conv_fire(o_pooled, w, T, s, p, theta, potentials=True)
    if math.isinf(theta):
        assert np.all(np_(tf) == NEVER)
        check_potentials(np_(vk), o_vk, "readout v_key")
    else:
        check_fire(np_(tf), np_(vk), o_tf, o_vk, excused_from_potentials(o_V, theta))


def test_packed_weights_follow_weight_updates():
    """A readout layer whose weights change: the packed fragments are rebuilt
    after the change and the readout matches a call that packs w itself."""
    dev = gpu()
    rng = np.random.default_rng(5)
    times0 = random_times(rng, (2, 250, 14, 14), 15, 0.3)
    w = _t(rng.uniform(0.0, 1.0, size=(200, 250, 5, 5)).astype(np.float32), dev)
    t0 = _t(times0, dev)
    packed = spk.spk_conv_pack_weights(w)
    w.mul_(0.5).add_(0.25)
    spk.spk_conv_pack_weights(w, out=packed)
    tf, vk = spk.spk_pool_conv_fire(t0, (3, 3, 1), w, 15, 1, 2, math.inf, packed_w=packed,
                                    keep_pooled=False)
    ref_tf, ref_vk = spk.spk_pool_conv_fire(t0, (3, 3, 1), w, 15, 1, 2, math.inf, keep_pooled=False)
    np.testing.assert_array_equal(np_(tf), np_(ref_tf))
    np.testing.assert_array_equal(np_(vk), np_(ref_vk))


# ------------------------------------------------------- inhibition + k-WTA

def test_inhibit_wta_hand_example():
    dev = gpu()
    g = load_golden("h2_inhibit_wta.json")
    times = np.array(g["times"], np.uint8)[None]
    vkey = np.array(g["v_key"], np.float32)[None]
    for key, r in (("k2_r0", 0), ("k2_r1", 1)):
        win, n, inh = spk.spk_inhibit_winners(_t(times, dev), _t(vkey, dev), g["T"], 2, r,
                                              inhibited=True)
        np.testing.assert_array_equal(np_(inh)[0], np.array(g["inhibited"], np.uint8))
        exp = [(e["c"], e["y"], e["x"], e["t"], e["v"]) for e in g[key]]
        assert winners_list(spk.winners_numpy(win), np_(n)) == [exp]


@pytest.mark.parametrize("B,C,H,W,k,r,dens,mode", [
    (4, 32, 28, 28, 5, 2, 0.05, "pointwise"), (3, 250, 14, 14, 8, 1, 0.1, "pointwise"),
    (2, 4, 160, 250, 1, 0, 0.01, "pointwise"), (2, 128, 64, 64, 16, 2, 0.02, "pointwise"),
    (3, 30, 9, 11, 40, 0, 0.3, "pointwise"), (3, 6, 7, 5, 4, 1, 0.3, "fired"),
    (4, 200, 5, 5, 1, 0, 0.0, "readout"), (2, 20, 6, 6, 5, 1, 0.0, "readout"),
    (2, 8, 8, 8, 0, 1, 0.3, "pointwise"), (2, 5, 6, 6, 3, 1, 0.0, "pointwise"),
    (2, 6, 80, 90, 6, 2, 0.05, "pointwise"), (2, 12, 20, 30, 7, 1, 0.2, "fired"),
    (2, 40, 16, 16, 3, 1, 0.0, "readout"), (2, 600, 6, 6, 3, 1, 0.2, "pointwise"),
])
def test_inhibit_wta_matches_oracle(B, C, H, W, k, r, dens, mode):
    dev = gpu()
    rng = np.random.default_rng(B * C + H + k)
    T = 15
    times = random_times(rng, (B, C, H, W), T, dens)
    vkey = (rng.integers(0, 40, size=times.shape) / 4).astype(np.float32)   # many ties
    readout = mode == "readout"
    pointwise = mode == "pointwise"
    win, n, inh = spk.spk_inhibit_winners(_t(times, dev), _t(vkey, dev), T, k, r,
                                          pointwise=pointwise, readout=readout, inhibited=True)
    cand = oracle.inhibit(times, vkey) if pointwise else times
    np.testing.assert_array_equal(np_(inh), cand)
    o_win, o_n = oracle.kwta(cand, vkey, T, k, r, readout)
    np.testing.assert_array_equal(np_(n), o_n)
    g = spk.winners_numpy(win)
    assert winners_list(g, np_(n)) == winners_list(o_win, o_n)
    for b in range(B):
        assert np.all(g[b, o_n[b]:]["c"] == -1)


def test_inhibit_in_place():
    dev = gpu()
    rng = np.random.default_rng(31)
    times = random_times(rng, (2, 9, 6, 7), 10, 0.4)
    vkey = rng.standard_normal(times.shape).astype(np.float32)
    tt = _t(times, dev)
    spk.spk_inhibit_winners(tt, _t(vkey, dev), 10, 3, 1, inhibited=tt)
    np.testing.assert_array_equal(np_(tt), oracle.inhibit(times, vkey))


@pytest.mark.parametrize("shape", [(2, 9, 6, 7), (3, 128, 8, 8), (2, 30, 28, 28), (1, 5, 3, 5), (2, 7, 2, 6),
                                   (2, 3, 202, 202), (2, 3, 256, 160), (2, 600, 6, 6)])
def test_inhibit_alone_matches_oracle(shape):
    """spk_inhibit: the vectorized pass (H*W % 4 == 0: the wide form for few
    locations, 4 or 8 locations per lane for many) and the per-location one,
    to a new map and in place, with ties in time and potential."""
    dev = gpu()
    rng = np.random.default_rng(sum(shape))
    times = random_times(rng, shape, 6, 0.5)
    vkey = np.round(rng.uniform(0, 3, size=shape), 1).astype(np.float32)
    ref = oracle.inhibit(times, vkey)
    np.testing.assert_array_equal(np_(spk.spk_inhibit(_t(times, dev), _t(vkey, dev))), ref)
    tt = _t(times, dev)
    spk.spk_inhibit(tt, _t(vkey, dev), out=tt)
    np.testing.assert_array_equal(np_(tt), ref)


# --------------------------------------------------------------------- STDP

def _winners_dev(win_np, dev):
    return _t(win_np.view(np.int32).reshape(win_np.shape + (5,)), dev)


def test_stdp_hand_example():
    dev = gpu()
    g = load_golden("h1_conv_stdp.json")
    times = _t(np.array(g["in_times"], np.uint8)[None, None], dev)
    win = np.zeros((1, 1), oracle.WINNER_DTYPE)
    win[0, 0] = (0, 0, 0, 0, 1.5)
    for key in ("stdp_reward", "stdp_punish"):
        c = g[key]
        w = _t(np.array(g["weights"], np.float32)[None, None], dev)
        spk.spk_stdp_update(w, times, _winners_dev(win, dev), _t(np.array([1], np.int32), dev),
                            [(c["a_causal"], c["a_anticausal"], c["lower"], c["upper"], 1)])
        np.testing.assert_allclose(np_(w)[0, 0], np.array(c["weights_after"]), rtol=0, atol=6e-8)


@pytest.mark.parametrize("Co,Ci,K,s,p,B,H,k,stab,ncfg", [
    (32, 2, 5, 1, 2, 8, 28, 5, 1, 1), (250, 30, 3, 1, 1, 16, 14, 8, 1, 1),
    (200, 250, 5, 1, 2, 64, 5, 1, 1, 2), (20, 4, 17, 1, 0, 6, 26, 1, 1, 1),
    (128, 64, 3, 1, 1, 8, 64, 16, 1, 1), (7, 3, 3, 2, 1, 300, 9, 3, 0, 2),
    (5, 8, 3, 1, 1, 400, 12, 3, 1, 2), (3, 30, 5, 1, 2, 200, 10, 2, 1, 1),
])
def test_stdp_matches_oracle(Co, Ci, K, s, p, B, H, k, stab, ncfg):
    dev = gpu()
    rng = np.random.default_rng(Co + Ci + B)
    T = 15
    times = random_times(rng, (B, Ci, H, H + 1), T, 0.3)
    Ho = (H + 2 * p - K) // s + 1
    Wo = (H + 1 + 2 * p - K) // s + 1
    w = np.clip(rng.normal(0.8, 0.05, size=(Co, Ci, K, K)), 0, 1).astype(np.float32)
    win = np.zeros((B, k), oracle.WINNER_DTYPE)
    n = rng.integers(0, k + 1, size=B).astype(np.int32)
    for b in range(B):
        maps = rng.permutation(Co)[:k]
        for sl in range(k):
            win[b, sl] = ((maps[sl], rng.integers(0, Ho), rng.integers(0, Wo), rng.integers(0, T),
                           1.0) if sl < n[b] else (-1, -1, -1, -1, 0.0))
    cfgs = [(0.004, -0.003, 0.0, 1.0, stab), (-0.0005, 0.004, 0.0, 1.0, stab)][:ncfg]
    wc = rng.integers(0, ncfg, size=(B, k)).astype(np.int32) if ncfg > 1 else None
    w_dev = _t(w, dev)
    w16 = w_dev.to(torch.float16)
    spk.spk_stdp_update(w_dev, _t(times, dev), _winners_dev(win, dev), _t(n, dev), cfgs, s, p,
                        winner_cfg=None if wc is None else _t(wc, dev), w_f16=w16)
    ref = oracle.stdp_update(w, times, win, n, cfgs, s, p, winner_cfg=wc)
    np.testing.assert_allclose(np_(w_dev), ref, rtol=0, atol=W_ABS)
    np.testing.assert_array_equal(np_(w16), np_(w_dev).astype(np.float16))
    # weights of maps without a winner are untouched, bit for bit
    won = {int(win[b, sl]["c"]) for b in range(B) for sl in range(n[b])}
    for o in range(Co):
        if o not in won:
            np.testing.assert_array_equal(np_(w_dev)[o], w[o])


def test_rstdp_select_matches_oracle():
    dev = gpu()
    rng = np.random.default_rng(41)
    B, k = 64, 2
    win = np.zeros((B, k), oracle.WINNER_DTYPE)
    win["c"] = rng.integers(0, 200, size=(B, k))
    n = rng.integers(0, k + 1, size=B).astype(np.int32)
    labels = rng.integers(0, 10, size=B).astype(np.int32)
    got = spk.spk_rstdp_select(_winners_dev(win, dev), _t(n, dev), _t(labels, dev), 20)
    np.testing.assert_array_equal(np_(got), oracle.rstdp_select(win, n, labels, 20))


def test_cast_f16():
    dev = gpu()
    x = np.random.default_rng(5).uniform(-2, 2, 1000).astype(np.float32)
    got = np_(spk.spk_cast_f16(_t(x, dev)))
    np.testing.assert_array_equal(got, x.astype(np.float16))
