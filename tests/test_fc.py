"""Fully connected layer (§II-E.2), its winner selection fcwta (§II-F.3) and
STDP on it: the oracle pinned against independent forms on the CPU, then
libspk against the oracle on the GPU."""
import math

import numpy as np
import pytest
import torch

import oracle
from parity import W_ABS, check_fire, check_potentials, gpu, np_, winners_list
from paper_2301_13659_amd import spk
from paper_2301_13659_amd.workloads import random_times

NEVER = 255


# ----------------------------------------------------------- oracle pins

def _fc_direct(in_times, w, T, theta):
    """V_t = W @ [x <= t] per frame (a plain matrix product in float64), then
    the first crossing of theta; independent of the oracle's event scatter."""
    B, I = in_times.shape
    S = (in_times[:, None, :] <= np.arange(T)[None, :, None]).astype(np.float64)  # B x T x I
    V = S @ w.astype(np.float64).T                                                 # B x T x O
    fired = V > theta
    first = np.where(fired.any(axis=1), fired.argmax(axis=1), NEVER)
    last = V[:, -1, :]
    vkey = np.where(first != NEVER, np.take_along_axis(V, np.minimum(first, T - 1)[:, None, :], 1)[:, 0],
                    last)
    return first.astype(np.uint8), vkey, V


@pytest.mark.parametrize("B,I,O,T,theta,dens", [(3, 40, 7, 6, 4.0, 0.5), (2, 150, 33, 15, 20.0, 0.4),
                                                (1, 9, 4, 1, 0.5, 1.0), (2, 64, 5, 30, -1.0, 0.1)])
def test_oracle_fc_fire_is_a_matrix_product_per_frame(B, I, O, T, theta, dens):
    rng = np.random.default_rng(B * 100 + I)
    x = random_times(rng, (B, I), T, dens)
    w = rng.uniform(-0.2, 1.0, size=(O, I)).astype(np.float32)
    tf, vk, V = oracle.fc_fire(x, w, T, theta, potentials=True)
    d_tf, d_vk, d_V = _fc_direct(x, w, T, theta)
    np.testing.assert_allclose(V, d_V, rtol=1e-6, atol=1e-6)
    np.testing.assert_array_equal(tf, d_tf)
    np.testing.assert_allclose(vk, d_vk, rtol=1e-6, atol=1e-6)


def _fc_wta_sorted(times, vkey, T, k, radius, readout):
    """fcwta as a greedy scan of the fully sorted candidate list: a second,
    independent form of the iterative arg-min with masking."""
    out = []
    for b in range(times.shape[0]):
        O = times.shape[1]
        cand = [o for o in range(O) if readout or times[b, o] != NEVER]
        cand.sort(key=lambda o: ((0 if readout else int(times[b, o])), -float(vkey[b, o]), o))
        removed, win = set(), []
        for o in cand:
            if len(win) == k:
                break
            if o in removed:
                continue
            win.append((o, 0, 0, T - 1 if readout else int(times[b, o]), float(vkey[b, o])))
            removed.update(range(o - radius, o + radius + 1))
        out.append(win)
    return out


def test_oracle_fc_wta_hand_example():
    t = np.array([[2, 1, NEVER, 1, 3, 0]], np.uint8)
    v = np.array([[5.0, 4.0, 9.0, 6.0, 1.0, 2.0]], np.float32)
    win, n = oracle.fc_wta(t, v, 4, 3, 1)
    assert winners_list(win, n) == [[(5, 0, 0, 0, 2.0), (3, 0, 0, 1, 6.0), (1, 0, 0, 1, 4.0)]]
    win, n = oracle.fc_wta(t, v, 4, 3, 2)
    assert winners_list(win, n) == [[(5, 0, 0, 0, 2.0), (1, 0, 0, 1, 4.0)]]
    assert win[0, 2]["c"] == -1
    win, n = oracle.fc_wta(t, v, 4, 3, 1, readout=True)
    assert winners_list(win, n) == [[(2, 0, 0, 3, 9.0), (0, 0, 0, 3, 5.0), (5, 0, 0, 3, 2.0)]]


@pytest.mark.parametrize("seed", range(4))
def test_oracle_fc_wta_matches_sorted_scan(seed):
    rng = np.random.default_rng(seed)
    B, O, T = 3, int(rng.integers(5, 60)), 8
    t = random_times(rng, (B, O), T, 0.6)
    v = np.round(rng.uniform(0, 4, size=(B, O)), 1).astype(np.float32)  # ties on v too
    for k, r, ro in [(1, 0, False), (5, 2, False), (7, 0, True), (O, 3, False)]:
        win, n = oracle.fc_wta(t, v, T, k, r, ro)
        assert winners_list(win, n) == _fc_wta_sorted(t, v, T, k, r, ro)


def test_oracle_fc_stdp_single_winner_closed_form():
    rng = np.random.default_rng(7)
    B, I, O, T = 1, 30, 4, 10
    x = random_times(rng, (B, I), T, 0.7)
    w = rng.uniform(0.05, 0.95, size=(O, I)).astype(np.float32)
    win = np.zeros((B, 1), oracle.WINNER_DTYPE)
    win[0, 0] = (2, 0, 0, 4, 1.0)
    n = np.array([1], np.int32)
    ap, am = 0.004, -0.003
    got = oracle.fc_stdp_update(w, x, win, n, [(ap, am, 0.0, 1.0, 1)])
    ref = w.astype(np.float64).copy()
    a = np.where(x[0] <= 4, ap, am)
    ref[2] = np.clip(ref[2] + a * ref[2] * (1.0 - ref[2]), 0.0, 1.0)
    np.testing.assert_allclose(got, ref, atol=2e-7)
    assert np.array_equal(got[[0, 1, 3]], w[[0, 1, 3]])


# ------------------------------------------------------ GPU against oracle

def _t(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


FC_CASES = [
    # B, I, O, T, theta, density, dtype
    (5, 250, 200, 15, 40.0, 0.3, "f32"),
    (3, 6250, 200, 15, 600.0, 0.3, "f32"),
    (4, 1000, 65, 30, 60.0, 0.2, "f16"),
    (2, 37, 9, 7, 3.0, 0.5, "f32"),
    (3, 500, 40, 15, math.inf, 0.4, "f32"),
]


@pytest.mark.gpu
@pytest.mark.parametrize("case", FC_CASES)
def test_fc_fire_matches_oracle(case):
    dev = gpu()
    B, I, O, T, theta, dens, dt = case
    rng = np.random.default_rng(B * 1000 + I)
    x = random_times(rng, (B, I), T, dens)
    w = rng.uniform(0.0, 1.0, size=(O, I)).astype(np.float32)
    if dt == "f16":
        w = w.astype(np.float16).astype(np.float32)
    w_dev = _t(w, dev).to(torch.float16) if dt == "f16" else _t(w, dev)
    g_tf, g_vk, g_V = spk.spk_fc_fire(_t(x, dev), w_dev, T, theta, potentials=True)
    o_tf, o_vk, o_V = oracle.fc_fire(x, w, T, theta, potentials=True)
    check_potentials(np_(g_V), o_V)
    exc = ((np.abs(o_V.astype(np.float64) - theta) <= 1e-4 * abs(theta)).any(axis=1)
           if math.isfinite(theta) else np.zeros(o_tf.shape, bool))
    check_fire(np_(g_tf), np_(g_vk), o_tf, o_vk, exc)
    g_tf2, g_vk2 = spk.spk_fc_fire(_t(x, dev), w_dev, T, theta)
    if math.isinf(theta):
        assert np.all(np_(g_tf2) == NEVER)
        check_potentials(np_(g_vk2), o_vk, "readout v_key")
    else:
        check_fire(np_(g_tf2), np_(g_vk2), o_tf, o_vk, exc)


@pytest.mark.gpu
@pytest.mark.parametrize("B,O,k,r,readout", [(6, 200, 5, 3, False), (4, 1000, 16, 0, False),
                                             (3, 33, 40, 2, False), (5, 200, 1, 0, True),
                                             (2, 5000, 8, 100, True)])
def test_fc_winners_match_oracle(B, O, k, r, readout):
    dev = gpu()
    T = 15
    rng = np.random.default_rng(O + k)
    t = random_times(rng, (B, O), T, 0.4)
    v = np.round(rng.uniform(0, 30, size=(B, O)), 2).astype(np.float32)
    gw, gn = spk.spk_fc_winners(_t(t, dev), _t(v, dev), T, k, r, readout)
    ow, on = oracle.fc_wta(t, v, T, k, r, readout)
    np.testing.assert_array_equal(np_(gn), on)
    assert winners_list(spk.winners_numpy(gw), np_(gn)) == winners_list(ow, on)
    assert np.all(spk.winners_numpy(gw)["c"][np.arange(k)[None, :] >= np_(gn)[:, None]] == -1)


@pytest.mark.gpu
def test_fc_winners_hand_example():
    dev = gpu()
    t = np.array([[2, 1, NEVER, 1, 3, 0]], np.uint8)
    v = np.array([[5.0, 4.0, 9.0, 6.0, 1.0, 2.0]], np.float32)
    gw, gn = spk.spk_fc_winners(_t(t, dev), _t(v, dev), 4, 3, 1)
    assert winners_list(spk.winners_numpy(gw), np_(gn)) == [[(5, 0, 0, 0, 2.0), (3, 0, 0, 1, 6.0),
                                                             (1, 0, 0, 1, 4.0)]]


@pytest.mark.gpu
@pytest.mark.parametrize("B,I,O,k", [(8, 250, 200, 3), (4, 6250, 64, 2), (6, 40, 10, 5)])
def test_fc_layer_step_matches_oracle(B, I, O, k):
    """fire -> fcwta -> STDP of one FC layer, each stage against the oracle."""
    dev = gpu()
    T, theta = 15, 0.1 * I * 0.5
    rng = np.random.default_rng(I + O)
    x = random_times(rng, (B, I), T, 0.4)
    w = np.clip(rng.normal(0.8, 0.05, size=(O, I)), 0, 1).astype(np.float32)
    w_dev = _t(w, dev)
    g_tf, g_vk = spk.spk_fc_fire(_t(x, dev), w_dev, T, theta)
    gw, gn = spk.spk_fc_winners(g_tf, g_vk, T, k, 2)
    ow, on = oracle.fc_wta(np_(g_tf), np_(g_vk), T, k, 2)
    assert winners_list(spk.winners_numpy(gw), np_(gn)) == winners_list(ow, on)
    cfgs = [(0.004, -0.003, 0.0, 1.0, 1)]
    spk.spk_fc_stdp_update(w_dev, _t(x, dev), gw, gn, cfgs)
    ref = oracle.fc_stdp_update(w, x, spk.winners_numpy(gw), np_(gn), cfgs)
    assert np.abs(np_(w_dev) - ref).max() <= W_ABS
