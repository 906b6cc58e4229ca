"""Sparse interface (§II-B): spike lists and the conv driven by them.  The
oracle pinned on the CPU, then libspk against it on the GPU."""
import numpy as np
import pytest

import oracle
from paper_2301_13659_amd.workloads import random_times

NEVER = 255


# ----------------------------------------------------------- oracle pins

def test_oracle_spike_list_hand_example():
    # one sample, 1 x 2 x 3, T = 4: step 0 holds indices 2 and 4, step 1 index 3,
    # step 2 nothing, step 3 indices 0 and 5; index 1 never fires
    t = np.array([[[[3, NEVER, 0], [1, 0, 3]]]], np.uint8)
    s, o = oracle.times_to_spikes(t, 4)
    assert o.tolist() == [[0, 2, 3, 3, 5]]
    assert s[0, :5].tolist() == [2, 4, 3, 0, 5]
    s2, o2 = oracle.times_to_spikes(t, 4, cap=3)
    assert o2.tolist() == [[0, 2, 3, 3, 5]] and s2.tolist() == [[2, 4, 3]]
    back = oracle.spikes_to_times(s2, o2, (1, 2, 3), 4)
    assert back.tolist() == [[[[NEVER, NEVER, 0], [1, 0, NEVER]]]]


@pytest.mark.parametrize("seed", range(3))
def test_oracle_spike_list_is_a_stable_sort_by_time(seed):
    rng = np.random.default_rng(seed)
    B, C, H, W, T = 3, 4, 7, 9, 11
    t = random_times(rng, (B, C, H, W), T, 0.3)
    s, o = oracle.times_to_spikes(t, T)
    for b in range(B):
        flat = t[b].ravel()
        idx = np.nonzero(flat != NEVER)[0]
        order = idx[np.lexsort((idx, flat[idx]))]
        assert o[b, T] == len(order)
        assert s[b, :len(order)].tolist() == order.tolist()
        assert o[b].tolist() == [int((flat < k).sum()) for k in range(T + 1)]
    assert np.array_equal(oracle.spikes_to_times(s, o, (C, H, W), T), t)


CASES = [
    # B, Ci, Hi, Wi, Co, K, stride, pad, T, theta, density, signed weights
    (2, 3, 9, 8, 5, 3, 1, 1, 6, 1.5, 0.3, False),
    (2, 4, 11, 10, 7, 5, 2, 2, 9, 2.0, 0.2, True),
    (1, 2, 6, 6, 3, 3, 1, 0, 4, -0.5, 0.1, True),
    (3, 5, 7, 5, 4, 1, 1, 0, 12, 0.8, 0.5, False),
]


@pytest.mark.parametrize("case", CASES)
def test_oracle_spike_conv_equals_the_dense_conv(case):
    """The scatter from a spike list and the per-neuron gather over the time
    map are two independent forms of Eq. 2 with the same firing rule."""
    B, Ci, Hi, Wi, Co, K, s_, p_, T, theta, dens, signed = case
    rng = np.random.default_rng(Ci * 31 + K)
    t = random_times(rng, (B, Ci, Hi, Wi), T, dens)
    w = rng.uniform(-0.5 if signed else 0.0, 1.0, size=(Co, Ci, K, K)).astype(np.float32)
    sp, off = oracle.times_to_spikes(t, T)
    tf, vk = oracle.conv_fire_spikes(sp, off, (Ci, Hi, Wi), w, T, s_, p_, theta)
    d_tf, d_vk = oracle.conv_fire(t, w, T, s_, p_, theta)
    np.testing.assert_array_equal(tf, d_tf)
    np.testing.assert_allclose(vk, d_vk, rtol=1e-6, atol=1e-6)


def test_oracle_spike_conv_single_spike_and_truncation():
    # one spike at step 2 on channel 1, pixel (2, 3): with theta below its
    # weight, the neurons whose window holds it fire at 2 with V = w
    B, Ci, Hi, Wi, T = 1, 2, 5, 6, 5
    t = np.full((B, Ci, Hi, Wi), NEVER, np.uint8)
    t[0, 1, 2, 3] = 2
    t[0, 0, 0, 0] = 4
    w = np.arange(1, 2 * 2 * 3 * 3 + 1, dtype=np.float32).reshape(2, 2, 3, 3) / 8
    sp, off = oracle.times_to_spikes(t, T)
    tf, vk = oracle.conv_fire_spikes(sp, off, (Ci, Hi, Wi), w, T, 1, 1, 0.05)
    for o in range(2):
        for y in range(Hi):
            for x in range(Wi):
                ky, kx = 2 - y + 1, 3 - x + 1
                if 0 <= ky < 3 and 0 <= kx < 3:
                    assert tf[0, o, y, x] == 2 and vk[0, o, y, x] == w[o, 1, ky, kx]
                elif y <= 1 and x <= 1:
                    assert tf[0, o, y, x] == 4
                else:
                    assert tf[0, o, y, x] == NEVER and vk[0, o, y, x] == 0.0
    # a list truncated to its first spike is the input without the step-4 spike
    sp1, off1 = oracle.times_to_spikes(t, T, cap=1)
    tf1, _ = oracle.conv_fire_spikes(sp1, off1, (Ci, Hi, Wi), w, T, 1, 1, 0.05)
    assert tf1[0, 0, 0, 0] == NEVER and tf1[0, 0, 1, 2] == 2
