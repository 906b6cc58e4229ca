"""Pins of the oracle's lateral inhibition and k-WTA (Sec. II-F.3) and of STDP /
R-STDP (Sec. II-F.1 Eq. 4-6, Sec. II-F.2 Eq. 7).

k-WTA is checked against the hand example and against a second, differently
built selection (sort every candidate once, then a greedy scan); STDP against
the hand-worked single-winner values, batch linearity, bounds and fixed points.
"""
import numpy as np
import pytest

import oracle
from conftest import load_golden
from paper_2301_13659_amd.workloads import random_times

NEVER = 255


def _w(rec):
    return (int(rec["c"]), int(rec["y"]), int(rec["x"]), int(rec["t"]), float(rec["v"]))


# ----------------------------------------------------------- inhibition

def test_inhibition_and_wta_hand_example():
    g = load_golden("h2_inhibit_wta.json")
    times = np.array(g["times"], np.uint8)[None]
    vkey = np.array(g["v_key"], np.float32)[None]
    inh = oracle.inhibit(times, vkey)
    np.testing.assert_array_equal(inh[0], np.array(g["inhibited"], np.uint8))
    for key, r in (("k2_r0", 0), ("k2_r1", 1)):
        win, n = oracle.kwta(inh, vkey, g["T"], 2, r)
        exp = [(e["c"], e["y"], e["x"], e["t"], e["v"]) for e in g[key]]
        assert n[0] == len(exp)
        assert [_w(win[0, s]) for s in range(n[0])] == exp
        assert all(win[0, s]["c"] == -1 for s in range(n[0], 2))


def test_inhibition_keeps_one_earliest_neuron_per_location():
    rng = np.random.default_rng(1)
    times = random_times(rng, (3, 6, 5, 7), 8, 0.5)
    vkey = rng.integers(0, 4, size=times.shape).astype(np.float32)  # many ties
    inh = oracle.inhibit(times, vkey)
    for b in range(3):
        for y in range(5):
            for x in range(7):
                t = times[b, :, y, x]
                fired = np.flatnonzero(t != NEVER)
                kept = np.flatnonzero(inh[b, :, y, x] != NEVER)
                if len(fired) == 0:
                    assert len(kept) == 0
                    continue
                assert len(kept) == 1
                c = kept[0]
                # brute force: lexicographic min of (t, -v, c)
                best = min(fired, key=lambda cc: (int(t[cc]), -float(vkey[b, cc, y, x]), cc))
                assert c == best and inh[b, c, y, x] == t[c]


# ----------------------------------------------------------------- k-WTA

def _kwta_by_sorting(times, vkey, T, k, r, readout):
    """Independent selection: sort all candidates once, then scan greedily."""
    B, C, H, W = times.shape
    out = []
    for b in range(B):
        cand = []
        for c in range(C):
            for y in range(H):
                for x in range(W):
                    t = int(times[b, c, y, x])
                    if readout or t != NEVER:
                        key = (0 if readout else t, -float(vkey[b, c, y, x]), (c * H + y) * W + x)
                        cand.append((key, c, y, x, T - 1 if readout else t, float(vkey[b, c, y, x])))
        cand.sort()
        won = []
        for _, c, y, x, t, v in cand:
            if len(won) == k:
                break
            if any(c == wc or (abs(y - wy) <= r and abs(x - wx) <= r) for wc, wy, wx, _, _ in won):
                continue
            won.append((c, y, x, t, v))
        out.append(won)
    return out


@pytest.mark.parametrize("seed,k,r,readout", [(0, 5, 2, False), (1, 8, 1, False), (2, 1, 0, False),
                                              (3, 16, 0, False), (4, 3, 1, True), (5, 1, 0, True),
                                              (6, 0, 1, False), (7, 40, 0, False)])
def test_kwta_matches_sorted_greedy_scan(seed, k, r, readout):
    rng = np.random.default_rng(seed)
    T = 6
    times = random_times(rng, (3, 5, 6, 7), T, 0.2 if not readout else 0.0)
    if readout:
        times[:] = NEVER
    vkey = rng.integers(0, 6, size=times.shape).astype(np.float32) / 2  # ties in V too
    win, n = oracle.kwta(times, vkey, T, k, r, readout)
    ref = _kwta_by_sorting(times, vkey, T, k, r, readout)
    for b in range(3):
        assert n[b] == len(ref[b])
        assert [_w(win[b, s]) for s in range(n[b])] == ref[b]
        # invariants: distinct maps, separated by more than r
        got = ref[b]
        for i in range(len(got)):
            for j in range(i):
                assert got[i][0] != got[j][0]
                assert max(abs(got[i][1] - got[j][1]), abs(got[i][2] - got[j][2])) > r


# ------------------------------------------------------------------- STDP

def _h1_winners():
    win = np.zeros((1, 1), oracle.WINNER_DTYPE)
    win[0, 0] = (0, 0, 0, 0, 1.5)
    return win, np.array([1], np.int32)


@pytest.mark.parametrize("key", ["stdp_reward", "stdp_punish"])
def test_stdp_hand_example(key):
    g = load_golden("h1_conv_stdp.json")
    cfg = g[key]
    times = np.array(g["in_times"], np.uint8)[None, None]
    w = np.array(g["weights"], np.float32)[None, None]
    win, n = _h1_winners()
    w2 = oracle.stdp_update(w, times, win, n,
                            [(cfg["a_causal"], cfg["a_anticausal"], cfg["lower"], cfg["upper"], 1)],
                            g["stride"], g["pad"])
    # the result is stored in float32: allow one float32 ulp at 0.5
    np.testing.assert_allclose(w2[0, 0], np.array(cfg["weights_after"]), rtol=0, atol=6e-8)


def test_stdp_batch_of_identical_samples_sums_the_changes():
    g = load_golden("h1_conv_stdp.json")
    times = np.array(g["in_times"], np.uint8)[None, None]
    w = np.array(g["weights"], np.float32)[None, None]
    cfg = [(0.004, -0.003, 0.0, 1.0, 1)]
    win, n = _h1_winners()
    one = oracle.stdp_update(w, times, win, n, cfg, 1, 0).astype(np.float64) - w
    B = 4
    two = oracle.stdp_update(w, np.repeat(times, B, 0), np.repeat(win, B, 0), np.repeat(n, B),
                             cfg, 1, 0).astype(np.float64) - w
    # each stored weight is rounded once to float32 (half an ulp is 2**-25 in [0.5, 1))
    np.testing.assert_allclose(two, B * one, rtol=0, atol=(B + 1) * 2.0 ** -25)


def test_stdp_without_stabiliser_adds_the_rate_and_clamps():
    times = np.array([[[[0, 5], [NEVER, 1]]]], np.uint8)
    w = np.array([[[[0.5, 0.5], [0.999, 0.0005]]]], np.float32)
    win = np.zeros((1, 1), oracle.WINNER_DTYPE)
    win[0, 0] = (0, 0, 0, 1, 2.0)
    w2 = oracle.stdp_update(w, times, win, np.array([1], np.int32),
                            [(0.004, -0.003, 0.0, 1.0, 0)], 1, 0)
    # t_pre 0 <= 1 causal, 5 > 1 anti, NEVER anti, 1 <= 1 causal
    np.testing.assert_allclose(w2[0, 0], [[0.504, 0.497], [0.996, 0.0045]], rtol=0, atol=6e-8)
    w3 = oracle.stdp_update(w, times, win, np.array([1], np.int32),
                            [(0.8, -0.8, 0.0, 1.0, 0)], 1, 0)
    assert w3[0, 0, 0, 0] == 1.0 and w3[0, 0, 0, 1] == 0.0          # clamped exactly to U and L
    np.testing.assert_allclose(w3[0, 0, 1], [0.199, 0.8005], rtol=0, atol=6e-8)


def test_stdp_bounds_fixed_points_and_untouched_weights():
    rng = np.random.default_rng(3)
    T = 5
    times = random_times(rng, (4, 3, 8, 8), T, 0.5)
    w = rng.uniform(0, 1, size=(6, 3, 3, 3)).astype(np.float32)
    w[0, 0, 0, 0], w[0, 0, 0, 1] = 0.0, 1.0
    win = np.zeros((4, 2), oracle.WINNER_DTYPE)
    n = np.array([2, 1, 0, 2], np.int32)
    for b in range(4):
        for s in range(2):
            win[b, s] = (s * 2 if b != 3 else s, rng.integers(0, 8), rng.integers(0, 8),
                         rng.integers(0, T), 1.0)
    cfg = [(0.3, -0.3, 0.0, 1.0, 1)]
    w2 = oracle.stdp_update(w, times, win, n, cfg, 1, 1)
    assert w2.min() >= 0.0 and w2.max() <= 1.0
    assert w2[0, 0, 0, 0] == 0.0 and w2[0, 0, 0, 1] == 1.0   # soft-bound fixed points
    winners_maps = {0, 1, 2}
    for o in range(6):
        if o not in winners_maps:
            np.testing.assert_array_equal(w2[o], w[o])
    # a reward configuration equal to the STDP rates is the same update
    w3 = oracle.stdp_update(w, times, win, n, [(0.3, -0.3, 0.0, 1.0, 1), (9.0, 9.0, 0.0, 1.0, 1)],
                            1, 1, winner_cfg=np.zeros((4, 2), np.int32))
    np.testing.assert_array_equal(w3, w2)
    with pytest.raises(ValueError):
        oracle.stdp_update(w, times, win, n, [(0.3, -0.3, 0.0, 1.0, 1), (0.3, -0.3, 0.1, 1.0, 1)],
                           1, 1)


def test_stdp_padding_is_a_silent_input():
    times = np.zeros((1, 1, 2, 2), np.uint8)   # every real input fires at t=0
    w = np.full((1, 1, 3, 3), 0.5, np.float32)
    win = np.zeros((1, 1), oracle.WINNER_DTYPE)
    win[0, 0] = (0, 0, 0, 0, 1.0)
    w2 = oracle.stdp_update(w, times, win, np.array([1], np.int32), [(0.004, -0.003, 0, 1, 1)], 1, 1)
    # receptive field of output (0,0) with pad 1: row 0 and column 0 are padding
    causal = np.zeros((3, 3), bool)
    causal[1:, 1:] = True
    np.testing.assert_allclose(w2[0, 0], np.where(causal, 0.501, 0.49925), rtol=0, atol=6e-8)


def test_rstdp_select_rewards_matching_class():
    win = np.zeros((3, 2), oracle.WINNER_DTYPE)
    win["c"] = [[45, 3], [19, -1], [-1, -1]]
    n = np.array([2, 1, 0], np.int32)
    sel = oracle.rstdp_select(win, n, np.array([2, 0, 5], np.int32), 20)
    np.testing.assert_array_equal(sel, [[0, 1], [0, 1], [1, 1]])
